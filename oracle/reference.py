"""fp64 CPU oracle for chunked verification attention.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test-suite, the smoke
check and the CPU-baseline leg of the benchmark may import or run this module.
It shares no code with the HIP path (no kernels, headers, helpers, tables or
pre/post-processing) and imports nothing from it.

What it computes is the chunked-attention operator as the paper defines it
(Section 5.1, "Chunked Attention"), written out plainly in float64:

  * Q in R^{n x d} holds the queries of the n draft tokens of one sequence and
    one query head; K, V in R^{(l+n) x d} hold the keys/values of the l cached
    tokens followed by the n draft tokens.
  * The mask M in {-inf, 0}^{n x (l+n)} has M_ij = 0 where draft token i may
    attend to token j and -inf otherwise.  For a sequence (chain) draft, draft
    token i sees every cached token and draft tokens 0..i, i.e. j <= l + i.
  * Step one forms the scores S = scale * Q K^T + M; step two forms
    out = softmax(S) V, row by row.
  * lse is the natural log of the softmax denominator, log sum_j exp(S_ij),
    reported alongside out.

Grouped-query attention follows the paper's group factor g (Section 3.1,
"Model"): g query heads share one KV head; query head h reads KV head h // g.

Tree drafts (Section 2.3 on speculative decoding; Section 5.1, where only the
draft part of the mask is stored): the draft tokens of a tree are kept as a
sequence and an extra mask says which of them each draft token sees.  Here
that part is one bit word per draft token: bit k of word i set means draft
token i attends to draft token k (key position l + k).  Cached tokens are
always visible.

Readings where the paper is silent or garbled:
the printed mask set {-inf, 1} is read as {-inf, 0}; without a draft mask the
draft is a chain; the cached tokens come first in K/V, the chunk after; the
softmax scale is an argument; rows of a sequence beyond its chunk length are
padding and get out = 0, lse = -inf.  A draft mask is any set of bits (a tree's
ancestor sets are the intended use, but nothing requires it); bits k >= n are
ignored; a row that sees no key at all (l = 0 and no bit below n) gets out = 0,
lse = -inf, as a padding row does.

Parity pins (tests/test_oracle.py): a hand-worked golden example, the closed
form for q = 0 (uniform weights: lse = ln(l+i+1), out = mean of the visible V
rows), decode attention for n = 1 and full causal attention over the
concatenated sequence through torch's fp64 CPU scaled-dot-product attention,
n sequential decode steps, GQA equal to MHA with repeated KV heads, and
convex-hull / lse-bound / permutation invariants.  Draft masks: a chain's
words reproduce the chain mask, each row of a tree equals the chain
attention over its root path, arbitrary masks match torch's fp64 attention
with a boolean mask, q = 0 gives ln(#visible), and the all-ones mask is
bidirectional attention.
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode bf16 values stored as uint16 bit patterns into float64.

    A bf16 value is the upper half of the float32 with the same bits, so the
    float32 is the pattern shifted left by 16; float32 to float64 is exact.
    """
    bits = np.asarray(bits, dtype=np.uint16)
    as_f32 = (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return as_f32.astype(np.float64)


def f16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode IEEE binary16 values stored as uint16 bit patterns into float64
    (exact: every binary16 value is a float64 value)."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Input values as float64: ``dtype`` is "bf16" or "f16" (uint16 bits) or
    "f32"."""
    if dtype == "bf16":
        return bf16_bits_to_f64(x)
    if dtype == "f16":
        return f16_bits_to_f64(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def chain_mask(l: int, n: int) -> np.ndarray:
    """Additive mask M in {-inf, 0}^{n x (l+n)} of a chain draft (Section 5.1).

    Draft token i attends to every cached token j < l and to draft tokens
    0..i, i.e. to key positions j <= l + i.
    """
    M = np.full((n, l + n), -np.inf)
    for i in range(n):
        M[i, : l + i + 1] = 0.0
    return M


def tree_mask(l: int, n: int, words) -> np.ndarray:
    """Additive mask M in {-inf, 0}^{n x (l+n)} of a tree draft (Section 5.1).

    Every draft token sees all l cached tokens; draft token i sees draft token
    k (key position l + k) when bit k of ``words[i]`` is set.  Bits k >= n are
    ignored.
    """
    M = np.full((n, l + n), -np.inf)
    M[:, :l] = 0.0
    for i in range(n):
        for k in range(n):
            if (int(words[i]) >> k) & 1:
                M[i, l + k] = 0.0
    return M


def chunked_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, M: np.ndarray,
                      scale: float):
    """One sequence, one query head: out = softmax(scale * Q K^T + M) V.

    Q [n, d], K and V [l+n, d], M [n, l+n], all float64.  Returns out [n, d]
    and lse [n] (natural log of each row's softmax denominator).  The softmax
    subtracts the row maximum before exponentiating, which leaves the result
    unchanged and keeps exp() in range.  A row whose mask hides every key
    keeps out = 0, lse = -inf.
    """
    out = np.zeros((Q.shape[0], V.shape[1]))
    lse = np.full(Q.shape[0], -np.inf)
    seen = np.isfinite(M).any(axis=1)        # rows that see at least one key
    S = scale * (Q @ K.T) + M
    S = S[seen]
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    Z = E.sum(axis=1, keepdims=True)
    out[seen] = (E / Z) @ V
    lse[seen] = (m + np.log(Z))[:, 0]
    return out, lse


def gather_pages(pages: np.ndarray, block_table, page_size: int) -> np.ndarray:
    """A paged KV cache written out as the contiguous [B, Hkv, S_max, D] one.

    ``pages`` is [num_pages, Hkv, page_size, D]; ``block_table`` [B, P] lists
    each sequence's pages in order: token j of sequence b sits in page
    block_table[b, j // page_size] at row j % page_size, so S_max = P *
    page_size.  (Paged storage is not the paper's: Section 2.2 only cites KV
    cache managers; this layout is the build's own.)
    """
    table = np.asarray(block_table)
    B, P = table.shape
    _, Hkv, ps, D = pages.shape
    if ps != page_size:
        raise ValueError("pages and page_size disagree")
    out = np.empty((B, Hkv, P * ps, D), dtype=pages.dtype)
    for b in range(B):
        for t in range(P):
            out[b, :, t * ps:(t + 1) * ps] = pages[int(table[b, t])]
    return out


def verify_attn_ref(q, k_cache, v_cache, ctx_lens, chunk_lens, scale: float,
                    dtype: str, units=None, draft_mask=None):
    """Chunked verification attention for a batch of sequences, in float64.

    q        [B, C_max, Hq, D]      queries of each sequence's draft chunk
    k_cache  [B, Hkv, S_max, D]     rows [0, l_b) cached context, rows
    v_cache  [B, Hkv, S_max, D]     [l_b, l_b + c_b) the chunk's own K/V
    ctx_lens, chunk_lens  [B]       l_b and c_b
    dtype    "bf16" or "f16" (uint16 bit patterns) or "f32"
    units    optional iterable of (b, kv_head) pairs to compute; the others
             are left NaN (for sampled checks of large workloads)
    draft_mask  optional integer array [B, C_max] of draft-mask words (see
             tree_mask); None means a chain draft (chain_mask)

    Returns out [B, C_max, Hq, D] and lse [B, C_max, Hq] in float64.  Padding
    rows (i >= c_b) of computed units hold out = 0, lse = -inf.
    """
    B, C_max, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    if Hq % Hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    g = Hq // Hkv
    out = np.full((B, C_max, Hq, D), np.nan)
    lse = np.full((B, C_max, Hq), np.nan)
    if units is None:
        units = [(b, kvh) for b in range(B) for kvh in range(Hkv)]
    for b, kvh in units:
        l = int(ctx_lens[b])
        n = int(chunk_lens[b])
        K = to_f64(k_cache[b, kvh, : l + n], dtype)
        V = to_f64(v_cache[b, kvh, : l + n], dtype)
        M = chain_mask(l, n) if draft_mask is None else tree_mask(l, n, draft_mask[b])
        for h in range(kvh * g, (kvh + 1) * g):
            out[b, n:, h] = 0.0
            lse[b, n:, h] = -np.inf
            if n == 0:
                continue
            Q = to_f64(q[b, :n, h], dtype)
            o, s = chunked_attention(Q, K, V, M, scale)
            out[b, :n, h] = o
            lse[b, :n, h] = s
    return out, lse
