"""fp64 CPU oracle for chunked verification attention.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only tests, the smoke check and
the benchmark's CPU-baseline leg may use it.  See ``oracle.reference``.
"""
from .reference import (bf16_bits_to_f64, chain_mask, chunked_attention,  # noqa: F401
                        f16_bits_to_f64, gather_pages, to_f64, tree_mask, verify_attn_ref)
from .acceptance import accept_greedy_ref, accept_tree_ref, compact_path_ref, tree_parent  # noqa: F401
