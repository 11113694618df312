"""Seeded synthetic workloads for chunked verification attention.

This module only draws inputs: lengths, and q / k / v values.  It holds none of
the attention arithmetic, so both the HIP path and the fp64 CPU oracle can take
their inputs from it without sharing any code of the method.

Shapes follow the paper's problem statement for the chunked-attention operator
(Section 5.1, "Chunked Attention"): per sequence, n draft tokens (the chunk)
attend to l cached tokens plus the chunk itself.  The KV cache is the paper's
4-D [b, h, s, d] tensor (Section 5.2, CPU/GPU separation), here
[B, Hkv, S_max, D]; rows [0, l_b) hold the cached context and rows
[l_b, l_b + c_b) the chunk's own K/V, already appended.  Queries are
token-major [B, C_max, Hq, D].

The workloads stand in for the paper's APPS and CNN/DailyMail runs of
Mixtral-8x7B (Section 6.1, dataset table): those datasets and model weights are
not used; lengths are drawn from distributions that cover their prefix lengths
(APPS mean 566 input tokens plus up to 1024 generated; CNN/DM mean 1006), and
Mixtral's attention shape (32 query heads, 8 KV heads, head_dim 128) is used.
The draft-side workload is the decode attention of the draft model's single
layer, one new token per sequence (chunk 1): its KV cache is 1/8 of the
target's 32 layers (Section 5.2: 17.75 GB against 142 GB), i.e. four times a
target layer's, which is 32 KV heads of head_dim 128 (multi-head, g = 1).

Recipe (all draws with numpy's PCG64 ``default_rng``):
  * lengths: ``default_rng(seed)``; context lengths first, then chunk lengths.
    Uniform integer ranges are inclusive.  Log-uniform is
    ``floor(exp(U(ln lo, ln hi)))``.
  * q: ``default_rng([seed, 0])``, N(0, 1) float32 of shape [B, C_max, Hq, D].
  * k slab of sequence b: ``default_rng([seed, 1, b])``, N(0, 1) float32 of
    shape [Hkv, T_b, D] written to rows [0, T_b); v likewise with
    ``[seed, 2, b]``.  Each sequence's slab can therefore be regenerated on its
    own, which lets a test check sampled sequences of a large workload.
  * bf16 (f16) workloads round each float32 value once, to nearest-even, to
    bf16 (binary16); the same bits feed the GPU and the oracle.
  * Rows that hold no valid data (cache rows >= T_b, query rows >= c_b) are
    filled with ``fill`` (NaN by default) so that any read of them shows up.
  * Paged caches (workloads with ``page_size`` > 0): the contiguous cache is
    cut into pages of ``page_size`` tokens, [num_pages, Hkv, page_size, D],
    placed in a pool of B * S_max / page_size + 8 pages at the positions of
    ``default_rng([seed, 5]).permutation``; the block table [B, S_max /
    page_size] lists each sequence's pages in order; unused pages hold
    ``fill``.
  * Tree drafts (workloads with ``draft="tree"``): the draft tokens of
    sequence b form a random recursive tree drawn with
    ``default_rng([seed, 3, b])``: token 0 is the root and token i >= 1 hangs
    under a parent drawn uniformly from the tokens before it.  The tree is
    handed over as draft-mask words: word i has bit k set for every token k
    on the path from the root to i (i itself included).  Words of rows
    i >= c_b are 0.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

BF16_NAN = np.uint16(0x7FC0)
F16_NAN = np.uint16(0x7E00)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int            # 1-based; also the RNG seed
    B: int
    Hq: int
    Hkv: int
    D: int
    dtype: str            # "f32", "bf16" or "f16"
    ctx: tuple            # ("fixed", [..]) | ("uniform", lo, hi) | ("loguniform", lo, hi)
    chunk: tuple          # ("fixed", n) | ("uniform", lo, hi)
    description: str
    draft: str = "chain"  # "chain", or "tree": a random tree with draft-mask words
    page_size: int = 0    # 0: contiguous KV cache; else tokens per page of a paged cache

    @property
    def group(self) -> int:
        return self.Hq // self.Hkv

    @property
    def C_max(self) -> int:
        kind = self.chunk[0]
        return self.chunk[1] if kind == "fixed" else self.chunk[2]

    @property
    def ctx_hi(self) -> int:
        kind = self.ctx[0]
        return max(self.ctx[1]) if kind == "fixed" else self.ctx[2]

    @property
    def S_max(self) -> int:
        return round_up(self.ctx_hi + self.C_max, 256)

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)

    @property
    def elt_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


WORKLOADS = [
    Workload("tiny_fp32", 1, B=2, Hq=4, Hkv=1, D=64, dtype="f32",
             ctx=("fixed", [128, 200]), chunk=("fixed", 4),
             description="tiny fp32: B=2, Hq=4, Hkv=1, D=64, ctx 128/200, chunk 4"),
    Workload("mixtral_b64", 2, B=64, Hq=32, Hkv=8, D=128, dtype="bf16",
             ctx=("uniform", 512, 2048), chunk=("fixed", 5),
             description="Mixtral-8x7B attention shape, bf16: B=64, Hq=32, Hkv=8, D=128, "
                         "ctx U[512,2048], chunk 5"),
    Workload("large_batch_b256", 3, B=256, Hq=32, Hkv=8, D=128, dtype="bf16",
             ctx=("uniform", 1024, 4096), chunk=("fixed", 8),
             description="large batch, bf16: B=256, Hq=32, Hkv=8, D=128, ctx U[1024,4096], chunk 8"),
    Workload("long_ctx_b32", 4, B=32, Hq=32, Hkv=8, D=128, dtype="bf16",
             ctx=("loguniform", 16384, 32768), chunk=("fixed", 4),
             description="long ragged contexts, bf16: B=32, Hq=32, Hkv=8, D=128, "
                         "ctx logU[16384,32768], chunk 4"),
    Workload("ragged_chunk_b128", 5, B=128, Hq=28, Hkv=4, D=128, dtype="bf16",
             ctx=("uniform", 256, 4096), chunk=("uniform", 1, 16),
             description="ragged chunks, wide GQA, bf16: B=128, Hq=28, Hkv=4, D=128, "
                         "ctx U[256,4096], chunk U[1,16]"),
    Workload("mixtral_tree_b64", 6, B=64, Hq=32, Hkv=8, D=128, dtype="bf16",
             ctx=("uniform", 512, 2048), chunk=("fixed", 16), draft="tree",
             description="Mixtral-8x7B attention shape with 16-token tree drafts, bf16: B=64, Hq=32, "
                         "Hkv=8, D=128, ctx U[512,2048], chunk 16, random recursive trees"),
    Workload("mixtral_f16_b64", 8, B=64, Hq=32, Hkv=8, D=128, dtype="f16",
             ctx=("uniform", 512, 2048), chunk=("fixed", 5),
             description="Mixtral-8x7B attention shape with an FP16 KV cache (the paper's precision): B=64, "
                         "Hq=32, Hkv=8, D=128, ctx U[512,2048], chunk 5"),
    Workload("mixtral_paged_b64", 9, B=64, Hq=32, Hkv=8, D=128, dtype="bf16",
             ctx=("uniform", 512, 2048), chunk=("fixed", 5), page_size=16,
             description="Mixtral-8x7B attention shape with a paged KV cache (16-token pages in a shuffled "
                         "pool), bf16: B=64, Hq=32, Hkv=8, D=128, ctx U[512,2048], chunk 5"),
    Workload("eagle_draft_b64", 7, B=64, Hq=32, Hkv=32, D=128, dtype="bf16",
             ctx=("uniform", 512, 2048), chunk=("fixed", 1),
             description="draft-model decode attention (one MHA layer of the EAGLE draft for Mixtral-8x7B), "
                         "bf16: B=64, Hq=Hkv=32, D=128, ctx U[512,2048], chunk 1"),
]
BY_NAME = {w.name: w for w in WORKLOADS}


def get(name_or_index) -> Workload:
    if isinstance(name_or_index, int):
        return next(w for w in WORKLOADS if w.index == name_or_index)
    return BY_NAME[name_or_index]


def draw_lengths(w: Workload):
    """Context and chunk lengths (int32 [B] each) of workload ``w``."""
    rng = np.random.default_rng(w.index)
    kind = w.ctx[0]
    if kind == "fixed":
        ctx = np.asarray(w.ctx[1], dtype=np.int64)
    elif kind == "uniform":
        ctx = rng.integers(w.ctx[1], w.ctx[2] + 1, size=w.B)
    elif kind == "loguniform":
        u = rng.uniform(math.log(w.ctx[1]), math.log(w.ctx[2]), size=w.B)
        ctx = np.floor(np.exp(u)).astype(np.int64)
        ctx = np.clip(ctx, w.ctx[1], w.ctx[2])
    else:
        raise ValueError(kind)
    kind = w.chunk[0]
    if kind == "fixed":
        chunk = np.full(w.B, w.chunk[1], dtype=np.int64)
    elif kind == "uniform":
        chunk = rng.integers(w.chunk[1], w.chunk[2] + 1, size=w.B)
    else:
        raise ValueError(kind)
    return ctx.astype(np.int32), chunk.astype(np.int32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns the uint16 bits.

    Input preparation only: the values are finite N(0, 1) draws or NaN fill.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded[nan] = BF16_NAN
    return rounded


def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to IEEE binary16 (numpy's conversion: nearest, ties to
    even); returns the uint16 bits.  Input preparation only."""
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def _encode(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "f16":
        return f32_to_f16_bits(x)
    return np.ascontiguousarray(x, np.float32)


def _fill_value(dtype: str, fill: float):
    if dtype == "bf16":
        return BF16_NAN if math.isnan(fill) else f32_to_bf16_bits(np.float32([fill]))[0]
    if dtype == "f16":
        return F16_NAN if math.isnan(fill) else f32_to_f16_bits(np.float32([fill]))[0]
    return np.float32(fill)


def kv_slab(w: Workload, b: int, T_b: int, which: str) -> np.ndarray:
    """N(0,1) K or V rows [Hkv, T_b, D] of sequence ``b`` (encoded dtype)."""
    stream = {"k": 1, "v": 2}[which]
    rng = np.random.default_rng([w.index, stream, b])
    x = rng.standard_normal((w.Hkv, T_b, w.D), dtype=np.float32)
    return _encode(x, w.dtype)


def make_inputs(w: Workload, fill: float = float("nan"),
                batches: Optional[Sequence[int]] = None,
                ctx_lens=None, chunk_lens=None, workers: int = 0):
    """Materialise workload ``w`` on the host.

    Returns a dict with q [B, C_max, Hq, D], k_cache / v_cache
    [B, Hkv, S_max, D] (uint16 bf16 bits, or float32), ctx_lens, chunk_lens
    (int32 [B]), scale, the workload itself, and draft_mask (uint64
    [B, C_max] words of a tree workload, else None).  ``batches`` restricts the
    cache fill to those sequences (others keep ``fill``), for sampled checks of
    large workloads.  ``ctx_lens`` / ``chunk_lens`` override the drawn lengths.
    ``workers`` > 1 draws the sequences' slabs in that many threads (each
    slab has its own generator, so the values do not depend on it).
    """
    ctx, chunk = draw_lengths(w)
    if ctx_lens is not None:
        ctx = np.asarray(ctx_lens, dtype=np.int32)
    if chunk_lens is not None:
        chunk = np.asarray(chunk_lens, dtype=np.int32)
    B, C, S = len(ctx), w.C_max, w.S_max
    fv = _fill_value(w.dtype, fill)
    store = np.float32 if w.dtype == "f32" else np.uint16

    qrng = np.random.default_rng([w.index, 0])
    q = _encode(qrng.standard_normal((B, C, w.Hq, w.D), dtype=np.float32), w.dtype)
    for b in range(B):
        q[b, chunk[b]:] = fv

    k = np.full((B, w.Hkv, S, w.D), fv, dtype=store)
    v = np.full((B, w.Hkv, S, w.D), fv, dtype=store)
    todo = range(B) if batches is None else batches

    def fill_seq(b):
        T_b = int(ctx[b]) + int(chunk[b])
        k[b, :, :T_b] = kv_slab(w, b, T_b, "k")
        v[b, :, :T_b] = kv_slab(w, b, T_b, "v")

    if workers > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill_seq, todo))
    else:
        for b in todo:
            fill_seq(b)
    draft_mask = tree_draft_masks(w.index, chunk, w.C_max) if w.draft == "tree" else None
    out = dict(q=q, k_cache=k, v_cache=v, ctx_lens=ctx, chunk_lens=chunk,
               scale=w.scale, workload=w, draft_mask=draft_mask)
    if w.page_size:
        out["k_pages"], out["block_table"] = paginate(k, w.page_size, w.index, fv)
        out["v_pages"], _ = paginate(v, w.page_size, w.index, fv)
    return out


def paginate(cache: np.ndarray, page_size: int, seed: int, fill, spare: int = 8):
    """Cut a contiguous [B, Hkv, S_max, D] cache into a shuffled pool of pages
    [B * S_max / page_size + spare, Hkv, page_size, D] and its block table
    [B, S_max / page_size] (int32): token j of sequence b lands in page
    table[b, j // page_size], row j % page_size.  The pool positions come
    from ``default_rng([seed, 5]).permutation``, the same for K and V; spare
    pages hold ``fill``.  Input preparation only."""
    B, Hkv, S, D = cache.shape
    if S % page_size:
        raise ValueError("S_max must be a multiple of page_size")
    P = S // page_size
    perm = np.random.default_rng([seed, 5]).permutation(B * P + spare)
    table = perm[: B * P].reshape(B, P).astype(np.int32)
    pages = np.full((B * P + spare, Hkv, page_size, D), fill, dtype=cache.dtype)
    for b in range(B):
        for t in range(P):
            pages[table[b, t]] = cache[b, :, t * page_size:(t + 1) * page_size]
    return pages, table


def tree_draft_masks(seed: int, chunk_lens, C_max: int) -> np.ndarray:
    """Draft-mask words [B, C_max] (uint64) of random recursive trees.

    Sequence b's tree comes from ``default_rng([seed, 3, b])``: token 0 is the
    root, token i >= 1 gets a parent drawn uniformly from 0..i-1, and word i
    holds the bits of the tokens on the root path of i, i itself included.
    Rows i >= c_b hold 0.
    """
    chunk = np.asarray(chunk_lens, np.int64)
    if C_max > 64:
        raise ValueError("draft-mask words hold at most 64 draft tokens")
    words = np.zeros((len(chunk), C_max), np.uint64)
    for b, n in enumerate(chunk):
        rng = np.random.default_rng([seed, 3, b])
        for i in range(int(n)):
            own = np.uint64(1) << np.uint64(i)
            words[b, i] = own if i == 0 else words[b, int(rng.integers(0, i))] | own
    return words


def random_draft_masks(rng: np.random.Generator, chunk_lens, C_max: int, density: float = 0.5,
                       self_bit: bool = True, junk_high_bits: bool = False) -> np.ndarray:
    """Arbitrary draft-mask words [B, C_max] (uint64), for edge cases.

    Each bit k < c_b of word i < c_b is set with probability ``density``;
    ``self_bit`` forces bit i of word i.  ``junk_high_bits`` also sets random
    bits k >= c_b, which the operator must ignore.  Rows i >= c_b hold 0.
    """
    chunk = np.asarray(chunk_lens, np.int64)
    words = np.zeros((len(chunk), C_max), np.uint64)
    for b, n in enumerate(chunk):
        n = int(n)
        for i in range(n):
            bits = rng.random(64) < density
            if not junk_high_bits:
                bits[n:] = False
            if self_bit:
                bits[i] = True
            words[b, i] = np.uint64(int(sum(1 << k for k in range(64) if bits[k])))
    return words


@dataclasses.dataclass(frozen=True)
class AcceptWorkload:
    """Inputs of the acceptance step: target logits for every chunk position
    and the chunk's token ids."""
    name: str
    index: int            # RNG seed
    B: int
    C_max: int            # chunk length (fixed)
    V: int                # vocabulary size
    dtype: str            # "f32" or "bf16" logits
    accept_prob: float    # chance that a draft token equals the planted prediction
    description: str
    tree: bool = False    # tree drafts: random recursive trees, tokens follow the parents' predictions

    @property
    def elt_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


ACCEPT_WORKLOADS = [
    AcceptWorkload("accept_mixtral_b64", 11, B=64, C_max=5, V=32000, dtype="bf16", accept_prob=0.7,
                   description="greedy acceptance after the Mixtral B=64 verification: chunk 5, "
                               "vocabulary 32000, bf16 logits"),
    AcceptWorkload("accept_large_b256", 12, B=256, C_max=8, V=32000, dtype="bf16", accept_prob=0.7,
                   description="greedy acceptance after the B=256 verification: chunk 8, vocabulary 32000, "
                               "bf16 logits"),
    AcceptWorkload("accept_tree_b64", 14, B=64, C_max=16, V=32000, dtype="bf16", accept_prob=0.7,
                   description="greedy acceptance of 16-node tree drafts after the Mixtral B=64 verification: "
                               "vocabulary 32000, bf16 logits", tree=True),
    AcceptWorkload("accept_tiny_f32", 13, B=3, C_max=4, V=1000, dtype="f32", accept_prob=0.6,
                   description="tiny f32 acceptance: B=3, chunk 4, vocabulary 1000"),
]
ACCEPT_BY_NAME = {w.name: w for w in ACCEPT_WORKLOADS}


def make_accept_inputs(w: AcceptWorkload, chunk_lens=None, ctx_lens=None, fill: float = float("nan")):
    """Logits [B, C_max, V], chunk token ids [B, C_max] (int32), ctx_lens and
    chunk_lens (int32 [B]) of an acceptance workload.

    Recipe (``default_rng([seed, 4])``): logits N(0, 1); in each valid row i
    a planted token p_i (uniform) gets the value 8 -- far above the N(0, 1)
    draws, so it is almost surely the row's maximum, though nothing relies on
    that.  Chunk token 0 is uniform; chunk token i + 1 is p_i with probability
    ``accept_prob``, else a uniform token other than p_i.  Context lengths are
    U[512, 2048] unless given; chunk lengths default to C_max.  Rows past c_b
    hold ``fill`` (logits) and -1 (tokens).
    """
    rng = np.random.default_rng([w.index, 4])
    B, C, V = w.B, w.C_max, w.V
    chunk = np.full(B, C, np.int32) if chunk_lens is None else np.asarray(chunk_lens, np.int32)
    ctx = rng.integers(512, 2049, size=B).astype(np.int32) if ctx_lens is None else np.asarray(ctx_lens, np.int32)
    x = rng.standard_normal((B, C, V), dtype=np.float32)
    planted = rng.integers(0, V, size=(B, C))
    x[np.arange(B)[:, None], np.arange(C)[None, :], planted] = 8.0
    tokens = np.full((B, C), -1, np.int32)
    tokens[:, 0] = rng.integers(0, V, size=B)
    hit = rng.random((B, C)) < w.accept_prob
    other = (planted + rng.integers(1, V, size=(B, C))) % V
    tokens[:, 1:] = np.where(hit[:, :-1], planted[:, :-1], other[:, :-1])
    for b in range(B):
        x[b, chunk[b]:] = fill
        tokens[b, chunk[b]:] = -1
    logits = _encode(x, w.dtype)
    words = None
    if w.tree:
        # tree drafts: node i's token is its parent's planted prediction with
        # probability accept_prob (the parent is the highest ancestor bit of
        # the node's root-path word below the node)
        words = tree_draft_masks(w.index, chunk, C)
        for b in range(B):
            for i in range(1, int(chunk[b])):
                par = (int(words[b, i]) & ~(1 << i)).bit_length() - 1
                tokens[b, i] = planted[b, par] if hit[b, i] else other[b, par]
    return dict(logits=logits, tokens=tokens, ctx_lens=ctx, chunk_lens=chunk, planted=planted, workload=w,
                draft_mask=words)


def algorithmic_kv_bytes(w: Workload, ctx_lens, chunk_lens) -> int:
    """K+V bytes of valid rows: sum_b Hkv * (l_b + c_b) * D * elt * 2.

    This is the attention row of the paper's cost table (Section 3.2): memory
    access 2*b*s*h/g elements, with h/g = Hkv*D the KV width per token, at the
    workload's element size, and s = l_b + c_b per sequence.
    """
    T = np.asarray(ctx_lens, np.int64) + np.asarray(chunk_lens, np.int64)
    return int(T.sum()) * w.Hkv * w.D * w.elt_bytes * 2


def useful_flops(w: Workload, ctx_lens, chunk_lens) -> int:
    """4 * sum_b c_b * g * Hkv * T_b * D: QK^T plus PV over all visible pairs.

    Counts every (row, key) pair up to T_b; the causal mask inside the chunk
    removes c*(c-1)/2 pairs per head, which this upper estimate keeps.
    """
    c = np.asarray(chunk_lens, np.int64)
    T = np.asarray(ctx_lens, np.int64) + c
    return int((c * T).sum()) * w.Hq * w.D * 4
