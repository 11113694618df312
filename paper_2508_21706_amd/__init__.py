"""Chunked verification attention (SpecMoEOff's verify step) for MI355X.

``verify_attn`` (chain drafts), ``verify_attn_tree`` (tree drafts),
``verify_attn_paged`` (a paged KV cache) and
``accept_greedy`` (the acceptance step after verification) run the HIP kernels
of ``libspecmoe_verify.so`` through its C-ABI; ``workloads`` draws the seeded
synthetic inputs.
"""
from .binding import (AcceptDesc, Desc, SpecMoEError, accept_desc, accept_greedy, accept_greedy_tree,  # noqa: F401
                      compact_accepted_kv,
                      alloc_accept_workspace, alloc_workspace, desc_for, key_tile, load_library, make_desc,
                      status_str, verify_attn, verify_attn_noalloc, verify_attn_paged, verify_attn_tree,
                      workspace_bytes,
                      workspace_status)
from . import binding  # noqa: F401
