"""Chunked verification attention (SpecMoEOff's verify step) for MI355X.

``verify_attn`` (chain drafts) and ``verify_attn_tree`` (tree drafts) run the HIP kernels of ``libspecmoe_verify.so`` through its
C-ABI; ``workloads`` draws the seeded synthetic inputs.
"""
from .binding import (Desc, SpecMoEError, alloc_workspace, desc_for, key_tile,  # noqa: F401
                      load_library, make_desc, status_str, verify_attn, verify_attn_tree, workspace_bytes)
