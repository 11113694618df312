"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's formula: each compares it with a
hand-worked example, a closed form, a library routine (torch's fp64 CPU
scaled-dot-product attention), a property of the definition (Section 5.1), or
brute force over the paper's rejected alternatives (Section 5.1, naive
solutions: per-draft-token decode attention and full prefill attention).
The mutation test at the end plants plausible mistakes in copies of the oracle
and checks that the pins catch every one of them.
"""
import math
import os
import types

import numpy as np
import pytest
import torch

from oracle import reference as oracle_mod
from paper_2508_21706_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- helpers

def _rand_case(rng, B=2, Hq=4, Hkv=2, D=8, ctx=(5, 9), chunk=(3, 4), C_max=None, S_pad=3):
    ctx = np.asarray(ctx, np.int32)
    chunk = np.asarray(chunk, np.int32)
    C_max = C_max or int(chunk.max())
    S_max = int((ctx + chunk).max()) + S_pad
    q = rng.standard_normal((B, C_max, Hq, D)).astype(np.float32)
    k = rng.standard_normal((B, Hkv, S_max, D)).astype(np.float32)
    v = rng.standard_normal((B, Hkv, S_max, D)).astype(np.float32)
    return q, k, v, ctx, chunk


def _parse_vals(tok):
    tok = tok.strip()
    if tok.startswith("ln(") and tok.endswith(")"):
        return float(np.float32(math.log(float(tok[3:-1]))))
    if tok == "-inf":
        return -math.inf
    return float(tok)


def _load_hand_example():
    rows = {}
    with open(os.path.join(GOLDEN, "hand_worked_example.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            key, rest = line.split(None, 1)
            rows[key] = rest
    def mat(s):       # "a b ; c d" -> [[a, b], [c, d]]
        return [[_parse_vals(t) for t in r.split()] for r in s.split(";")]
    def mat3(s):      # "a b , c d ; ..." -> [token][head][d]
        return [[[_parse_vals(t) for t in h.split()] for h in r.split(",")] for r in s.split(";")]
    k = np.array(mat(rows["k"]), np.float32)[None, None]          # [1, 1, 3, 2]
    v = np.array(mat(rows["v"]), np.float32)[None, None]
    q = np.array(mat3(rows["q"]), np.float32)[None]                 # [1, 3, 2, 2]
    ctx = np.array([int(rows["ctx"])], np.int32)
    chunk = np.array([int(rows["chunk"])], np.int32)
    lse = np.array(mat(rows["lse"]), np.float64)[None]              # [1, 3, 2]
    out = np.array(mat3(rows["out"]), np.float64)[None]             # [1, 3, 2, 2]
    return q, k, v, ctx, chunk, out, lse


def _sdpa(q, k, v, scale, causal):
    """torch fp64 CPU scaled-dot-product attention, [L, D] x [S, D]."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float64))[None, None]
    o = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), is_causal=causal, scale=scale)
    return o[0, 0].numpy()


# --------------------------------------------------------------------- pins
# Each pin takes the module under test, so the mutation test can run the same
# battery on planted-mistake copies.

def pin_bf16_decoding(m):
    bits = np.array([0x3F80, 0xC000, 0x4049, 0x0000, 0x8000, 0x7F80, 0x0001, 0x3C00], np.uint16)
    want = [1.0, -2.0, 3.140625, 0.0, -0.0, math.inf, 2.0 ** -133, 2.0 ** -7]
    got = m.bf16_bits_to_f64(bits)
    assert got.dtype == np.float64
    for g, w in zip(got, want):
        assert g == w, (g, w)
    assert math.copysign(1.0, got[4]) == -1.0


def pin_f16_decoding(m):
    """IEEE binary16 bit patterns decode exactly (the paper's KV precision,
    Section 3.3): normal, largest finite, subnormal, signed zero, infinity."""
    bits = np.array([0x3C00, 0xC000, 0x4248, 0x7BFF, 0x0001, 0x0400, 0x8000, 0x7C00, 0x3555], np.uint16)
    want = [1.0, -2.0, 3.140625, 65504.0, 2.0 ** -24, 2.0 ** -14, -0.0, math.inf, 0.333251953125]
    got = m.to_f64(bits, "f16")
    assert got.dtype == np.float64
    for g, w in zip(got, want):
        assert g == w, (g, w)
    assert math.copysign(1.0, got[6]) == -1.0


def pin_f16_path(m):
    """f16 inputs give the results of the f32 values they encode."""
    rng = np.random.default_rng(19)
    q, k, v, ctx, chunk = _rand_case(rng)
    qh, kh, vh = (a.astype(np.float16).view(np.uint16) for a in (q, k, v))
    back = lambda bits: bits.view(np.float16).astype(np.float32)
    o1, s1 = m.verify_attn_ref(qh, kh, vh, ctx, chunk, 0.3, "f16")
    o2, s2 = m.verify_attn_ref(back(qh), back(kh), back(vh), ctx, chunk, 0.3, "f32")
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(s1, s2)


def pin_hand_example(m):
    q, k, v, ctx, chunk, out, lse = _load_hand_example()
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 1.0, "f32")
    np.testing.assert_allclose(o, out, rtol=0, atol=1e-6)
    np.testing.assert_allclose(s, lse, rtol=0, atol=1e-6)


def pin_uniform_closed_form(m):
    """q = 0: every visible key weighs the same, so lse = ln(#visible) and
    out is the mean of the visible V rows (rows 0..l+i)."""
    rng = np.random.default_rng(11)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(0, 13), chunk=(4, 2))
    q[:] = 0.0
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.37, "f32")
    g = q.shape[2] // k.shape[1]
    for b in range(q.shape[0]):
        for i in range(int(chunk[b])):
            n_vis = int(ctx[b]) + i + 1
            for h in range(q.shape[2]):
                assert abs(s[b, i, h] - math.log(n_vis)) < 1e-12
                mean = v[b, h // g, :n_vis].astype(np.float64).mean(axis=0)
                np.testing.assert_allclose(o[b, i, h], mean, rtol=0, atol=1e-12)


def pin_decode_is_sdpa(m):
    """Chunk length 1 is plain decode attention over the l+1 keys (P1)."""
    rng = np.random.default_rng(12)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(7, 19), chunk=(1, 1), D=16)
    o, _ = m.verify_attn_ref(q, k, v, ctx, chunk, 0.25, "f32")
    g = q.shape[2] // k.shape[1]
    for b in range(2):
        T = int(ctx[b]) + 1
        for h in range(q.shape[2]):
            ref = _sdpa(q[b, :1, h], k[b, h // g, :T], v[b, h // g, :T], 0.25, causal=False)
            np.testing.assert_allclose(o[b, 0, h], ref[0], rtol=0, atol=1e-12)


def pin_chunk_is_causal_prefill(m):
    """A chunk equals the last n rows of full causal attention over the
    concatenated l+n sequence (P3, the prefill alternative)."""
    rng = np.random.default_rng(13)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(6, 0), chunk=(5, 3), D=16)
    o, _ = m.verify_attn_ref(q, k, v, ctx, chunk, 0.3, "f32")
    g = q.shape[2] // k.shape[1]
    for b in range(2):
        l, n = int(ctx[b]), int(chunk[b])
        for h in range(q.shape[2]):
            # prefill queries for the cached positions are arbitrary; only
            # the last n rows are compared
            qfull = np.concatenate([rng.standard_normal((l, 16)), q[b, :n, h]], axis=0)
            ref = _sdpa(qfull, k[b, h // g, :l + n], v[b, h // g, :l + n], 0.3, causal=True)
            np.testing.assert_allclose(o[b, :n, h], ref[l:], rtol=0, atol=1e-12)


def pin_sequential_decode(m):
    """A chunk of n equals n decode steps with the KV appended one token at a
    time (P2, the repeated-decode alternative)."""
    rng = np.random.default_rng(14)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(3, 10), chunk=(4, 2))
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.5, "f32")
    for i in range(4):
        live = chunk > i
        step_ctx = ctx + i
        step_chunk = live.astype(np.int32)
        o1, s1 = m.verify_attn_ref(q[:, i:i + 1], k, v, step_ctx, step_chunk, 0.5, "f32")
        for b in np.nonzero(live)[0]:
            np.testing.assert_allclose(o[b, i], o1[b, 0], rtol=0, atol=1e-12)
            np.testing.assert_allclose(s[b, i], s1[b, 0], rtol=0, atol=1e-12)


def pin_gqa_is_repeated_mha(m):
    rng = np.random.default_rng(15)
    q, k, v, ctx, chunk = _rand_case(rng, Hq=6, Hkv=2, ctx=(4, 8), chunk=(3, 3))
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.4, "f32")
    k_rep = np.repeat(k, 3, axis=1)        # head h reads kv head h // 3
    v_rep = np.repeat(v, 3, axis=1)
    o2, s2 = m.verify_attn_ref(q, k_rep, v_rep, ctx, chunk, 0.4, "f32")
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(s, s2, rtol=0, atol=1e-12)


def pin_invariants(m):
    rng = np.random.default_rng(16)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(20, 1), chunk=(3, 4), D=8)
    scale = 0.6
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, scale, "f32")
    g = q.shape[2] // k.shape[1]
    for b in range(2):
        l = int(ctx[b])
        for i in range(int(chunk[b])):
            for h in range(q.shape[2]):
                V = v[b, h // g, : l + i + 1].astype(np.float64)
                # rows are convex combinations of the visible V rows
                assert np.all(o[b, i, h] >= V.min(axis=0) - 1e-12)
                assert np.all(o[b, i, h] <= V.max(axis=0) + 1e-12)
                # max score <= lse <= max score + ln(#visible); the scores are
                # taken by brute force, one key at a time
                sc = [scale * float(np.dot(q[b, i, h].astype(np.float64),
                                           k[b, h // g, j].astype(np.float64)))
                      for j in range(l + i + 1)]
                assert max(sc) - 1e-12 <= s[b, i, h] <= max(sc) + math.log(len(sc)) + 1e-12
    # constant V rows give that constant
    v_const = np.broadcast_to(np.arange(8, dtype=np.float32), v.shape).copy()
    o_c, _ = m.verify_attn_ref(q, k, v_const, ctx, chunk, scale, "f32")
    for b in range(2):
        np.testing.assert_allclose(o_c[b, : chunk[b]], np.broadcast_to(np.arange(8.0), o_c[b, : chunk[b]].shape),
                                   rtol=0, atol=1e-12)
    # permuting the cached positions (K and V together) changes nothing
    perm_k, perm_v = k.copy(), v.copy()
    for b in range(2):
        p = rng.permutation(int(ctx[b]))
        perm_k[b, :, : ctx[b]] = k[b][:, p]
        perm_v[b, :, : ctx[b]] = v[b][:, p]
    o_p, s_p = m.verify_attn_ref(q, perm_k, perm_v, ctx, chunk, scale, "f32")
    np.testing.assert_allclose(o_p, o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(s_p, s, rtol=0, atol=1e-12)


def pin_one_hot(m):
    """One key with a dominant score makes the output that key's V row, for
    every head of its group and no other KV head."""
    B, Hq, Hkv, D, l, n = 1, 4, 2, 4, 6, 2
    q = np.zeros((B, n, Hq, D), np.float32)
    k = np.zeros((B, Hkv, l + n, D), np.float32)
    v = np.arange(B * Hkv * (l + n) * D, dtype=np.float32).reshape(B, Hkv, l + n, D)
    q[..., 0] = 1.0
    k[0, 1, 2, 0] = 200.0           # kv head 1, cached token 2
    o, s = m.verify_attn_ref(q, k, v, np.array([l]), np.array([n]), 1.0, "f32")
    for h in (2, 3):                # heads of kv head 1
        np.testing.assert_allclose(o[0, :, h], np.broadcast_to(v[0, 1, 2], (n, D)), rtol=0, atol=1e-9)
        np.testing.assert_allclose(s[0, :, h], 200.0, rtol=0, atol=1e-9)
    for h in (0, 1):                # kv head 0: all scores zero -> uniform
        np.testing.assert_allclose(s[0, 0, h], math.log(l + 1), atol=1e-12)


def pin_padding_and_poison(m):
    """Rows i >= c_b are padding (out 0, lse -inf); NaN in the unused cache
    rows and query rows must not reach any valid output."""
    rng = np.random.default_rng(17)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(5, 2), chunk=(1, 3), C_max=4)
    for b in range(2):
        q[b, chunk[b]:] = np.nan
        k[b, :, ctx[b] + chunk[b]:] = np.nan
        v[b, :, ctx[b] + chunk[b]:] = np.nan
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.3, "f32")
    for b in range(2):
        c = int(chunk[b])
        assert np.all(np.isfinite(o[b, :c])) and np.all(np.isfinite(s[b, :c]))
        assert np.all(o[b, c:] == 0.0) and np.all(s[b, c:] == -np.inf)
    # zero-length chunk: every row is padding
    o0, s0 = m.verify_attn_ref(q, k, v, ctx, np.array([0, 0], np.int32), 0.3, "f32")
    assert np.all(o0 == 0.0) and np.all(s0 == -np.inf)


def pin_bf16_path(m):
    """bf16 inputs decode to the same numbers as their f32 values."""
    rng = np.random.default_rng(18)
    q, k, v, ctx, chunk = _rand_case(rng)
    qb, kb, vb = (wl.f32_to_bf16_bits(a) for a in (q, k, v))
    back = lambda bits: (bits.astype(np.uint32) << 16).view(np.float32)
    o1, s1 = m.verify_attn_ref(qb, kb, vb, ctx, chunk, 0.3, "bf16")
    o2, s2 = m.verify_attn_ref(back(qb), back(kb), back(vb), ctx, chunk, 0.3, "f32")
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(s1, s2)


# ------------------------------------------------------- draft-mask pins

def _chain_words(n):
    return [(1 << (i + 1)) - 1 for i in range(n)]


def pin_tree_chain_words_are_causal(m):
    """The words of a chain (token i sees tokens 0..i) reproduce the chain
    mask: a tree draft that happens to be a sequence is the plain case."""
    rng = np.random.default_rng(21)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(7, 0), chunk=(5, 3), C_max=6)
    words = np.zeros((2, 6), np.uint64)
    for b in range(2):
        words[b, : chunk[b]] = _chain_words(int(chunk[b]))
    o1, s1 = m.verify_attn_ref(q, k, v, ctx, chunk, 0.3, "f32")
    o2, s2 = m.verify_attn_ref(q, k, v, ctx, chunk, 0.3, "f32", draft_mask=words)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(s1, s2)


def pin_tree_row_is_its_root_path(m):
    """In a tree draft, token i attends to the cached tokens and its root path
    only, so its row equals the last row of a chain draft made of that path
    (Section 2.3: the tree's tokens are kept as a sequence plus a mask)."""
    rng = np.random.default_rng(22)
    B, Hq, Hkv, D, C = 3, 4, 2, 8, 9
    ctx = np.array([6, 0, 11], np.int32)
    chunk = np.array([9, 7, 4], np.int32)
    q, k, v, _, _ = _rand_case(rng, B=B, Hq=Hq, Hkv=Hkv, D=D, ctx=ctx, chunk=chunk, C_max=C)
    words = wl.tree_draft_masks(5, chunk, C)
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.45, "f32", draft_mask=words)
    for b in range(B):
        l = int(ctx[b])
        assert np.all(o[b, chunk[b]:] == 0.0) and np.all(s[b, chunk[b]:] == -np.inf)
        for i in range(int(chunk[b])):
            path = [t for t in range(int(chunk[b])) if (int(words[b, i]) >> t) & 1]
            assert path[-1] == i and path[0] == 0
            rows = list(range(l)) + [l + t for t in path]
            kp = k[b:b + 1, :, rows]
            vp = v[b:b + 1, :, rows]
            qp = np.zeros((1, len(path), Hq, D), np.float32)
            qp[0, -1] = q[b, i]
            o1, s1 = m.verify_attn_ref(qp, kp, vp, np.array([l], np.int32),
                                       np.array([len(path)], np.int32), 0.45, "f32")
            np.testing.assert_allclose(o[b, i], o1[0, -1], rtol=0, atol=1e-12)
            np.testing.assert_allclose(s[b, i], s1[0, -1], rtol=0, atol=1e-12)


def pin_tree_matches_sdpa_boolean_mask(m):
    """Arbitrary draft masks (not trees) against torch's fp64 attention with a
    boolean mask over the l + n keys."""
    rng = np.random.default_rng(23)
    B, Hq, Hkv, D, C = 2, 6, 3, 16, 7
    ctx = np.array([5, 13], np.int32)
    chunk = np.array([7, 4], np.int32)
    q, k, v, _, _ = _rand_case(rng, B=B, Hq=Hq, Hkv=Hkv, D=D, ctx=ctx, chunk=chunk, C_max=C)
    words = wl.random_draft_masks(rng, chunk, C, density=0.4, self_bit=False, junk_high_bits=True)
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.21, "f32", draft_mask=words)
    g = Hq // Hkv
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float64))[None, None]
    for b in range(B):
        l, n = int(ctx[b]), int(chunk[b])
        allow = np.ones((n, l + n), bool)
        for i in range(n):
            for kk in range(n):
                allow[i, l + kk] = bool((int(words[b, i]) >> kk) & 1)
        for h in range(Hq):
            ref = torch.nn.functional.scaled_dot_product_attention(
                t(q[b, :n, h]), t(k[b, h // g, :l + n]), t(v[b, h // g, :l + n]),
                attn_mask=torch.from_numpy(allow)[None, None], scale=0.21)[0, 0].numpy()
            np.testing.assert_allclose(o[b, :n, h], ref, rtol=0, atol=1e-12)


def pin_tree_uniform_closed_form(m):
    """q = 0 under a draft mask: lse = ln(l + #set bits below n), out = mean
    of the visible V rows; with l = 0 an empty word leaves the row without
    keys (out 0, lse -inf).  Bits at or above n do not count."""
    rng = np.random.default_rng(24)
    B, Hq, Hkv, D, C = 3, 2, 1, 4, 6
    ctx = np.array([0, 3, 0], np.int32)
    chunk = np.array([6, 5, 2], np.int32)
    q, k, v, _, _ = _rand_case(rng, B=B, Hq=Hq, Hkv=Hkv, D=D, ctx=ctx, chunk=chunk, C_max=C)
    q[:] = 0.0
    words = np.zeros((B, C), np.uint64)
    words[0, :6] = [0b000001, 0, 0b101101, 0b111111, 0b010000 | (1 << 40), 1 << 63]
    words[1, :5] = [0, 0b10110, 0b11111, 0b01000, 1 << 5]
    words[2, :2] = [0b10, 0b100]
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.8, "f32", draft_mask=words)
    for b in range(B):
        l, n = int(ctx[b]), int(chunk[b])
        for i in range(n):
            vis = list(range(l)) + [l + t for t in range(n) if (int(words[b, i]) >> t) & 1]
            for h in range(Hq):
                if not vis:
                    assert s[b, i, h] == -np.inf and np.all(o[b, i, h] == 0.0)
                    continue
                assert abs(s[b, i, h] - math.log(len(vis))) < 1e-12
                mean = v[b, 0, vis].astype(np.float64).mean(axis=0)
                np.testing.assert_allclose(o[b, i, h], mean, rtol=0, atol=1e-12)
    assert s[0, 1, 0] == -np.inf and s[0, 5, 0] == -np.inf and s[2, 1, 0] == -np.inf


def pin_tree_all_ones_is_bidirectional(m):
    """Every bit set: each draft token sees all l + n keys, which is
    attention without a mask."""
    rng = np.random.default_rng(25)
    q, k, v, ctx, chunk = _rand_case(rng, ctx=(4, 9), chunk=(3, 5), C_max=5, D=16)
    words = np.full((2, 5), np.uint64(2 ** 64 - 1))
    o, s = m.verify_attn_ref(q, k, v, ctx, chunk, 0.3, "f32", draft_mask=words)
    g = q.shape[2] // k.shape[1]
    for b in range(2):
        T = int(ctx[b] + chunk[b])
        for h in range(q.shape[2]):
            ref = _sdpa(q[b, : chunk[b], h], k[b, h // g, :T], v[b, h // g, :T], 0.3, causal=False)
            np.testing.assert_allclose(o[b, : chunk[b], h], ref, rtol=0, atol=1e-12)


def pin_split_and_combine(m):
    """Attention over two complementary key sets, combined with log-sum-exp
    weights (lse = logaddexp of the parts, out = sum of exp(lse_part - lse) *
    out_part), equals attention over all keys: the merge the GPU applies to
    the pieces of a split key range (Section 5.2 notes that a sequence split
    needs this combine).  A part in which a row sees no key (lse -inf) drops
    out."""
    rng = np.random.default_rng(26)
    n, l, d = 4, 11, 8
    Q = rng.standard_normal((n, d))
    K = rng.standard_normal((l + n, d))
    V = rng.standard_normal((l + n, d))
    M = m.chain_mask(l, n)
    o, s = m.chunked_attention(Q, K, V, M, 0.7)
    for cut in (1, 5, l, l + 2):
        first = np.full_like(M, -np.inf)
        second = np.full_like(M, -np.inf)
        first[:, :cut] = M[:, :cut]
        second[:, cut:] = M[:, cut:]
        o1, s1 = m.chunked_attention(Q, K, V, first, 0.7)
        o2, s2 = m.chunked_attention(Q, K, V, second, 0.7)
        lse = np.logaddexp(s1, s2)
        w1 = np.where(np.isfinite(s1), np.exp(s1 - lse), 0.0)[:, None]
        w2 = np.where(np.isfinite(s2), np.exp(s2 - lse), 0.0)[:, None]
        np.testing.assert_allclose(lse, s, rtol=0, atol=1e-12)
        np.testing.assert_allclose(w1 * o1 + w2 * o2, o, rtol=0, atol=1e-12)


PINS = [pin_bf16_decoding, pin_f16_decoding, pin_f16_path, pin_hand_example, pin_uniform_closed_form, pin_decode_is_sdpa,
        pin_chunk_is_causal_prefill, pin_sequential_decode, pin_gqa_is_repeated_mha,
        pin_invariants, pin_one_hot, pin_padding_and_poison, pin_bf16_path, pin_split_and_combine,
        pin_tree_chain_words_are_causal, pin_tree_row_is_its_root_path, pin_tree_matches_sdpa_boolean_mask,
        pin_tree_uniform_closed_form, pin_tree_all_ones_is_bidirectional]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oracle_mod)


# ---------------------------------------------------------- planted mistakes

MUTATIONS = {
    "mask_excludes_self": ("M[i, : l + i + 1] = 0.0", "M[i, : l + i] = 0.0"),
    "mask_leaks_next": ("M[i, : l + i + 1] = 0.0", "M[i, : l + i + 2] = 0.0"),
    "mask_context_only": ("M[i, : l + i + 1] = 0.0", "M[i, : l + 1] = 0.0"),
    "no_scale": ("S = scale * (Q @ K.T) + M", "S = (Q @ K.T) + M"),
    "lse_drops_max": ("lse[seen] = (m + np.log(Z))[:, 0]", "lse[seen] = np.log(Z)[:, 0]"),
    "unnormalised": ("out[seen] = (E / Z) @ V", "out[seen] = E @ V"),
    "gqa_modulo": ("for h in range(kvh * g, (kvh + 1) * g):", "for h in range(kvh, Hq, Hkv):"),
    "k_shifted": ("K = to_f64(k_cache[b, kvh, : l + n], dtype)",
                  "K = to_f64(k_cache[b, kvh, 1 : l + n + 1], dtype)"),
    "v_from_k": ("V = to_f64(v_cache[b, kvh, : l + n], dtype)",
                 "V = to_f64(k_cache[b, kvh, : l + n], dtype)"),
    "bf16_shift": ("<< np.uint32(16)", "<< np.uint32(15)"),
    "f16_read_as_bf16": ("        return f16_bits_to_f64(x)", "        return bf16_bits_to_f64(x)"),
    "padding_lse_zero": ("lse[b, n:, h] = -np.inf", "lse[b, n:, h] = 0.0"),
    "q_wrong_token": ("Q = to_f64(q[b, :n, h], dtype)", "Q = to_f64(q[b, 1 : n + 1, h], dtype)"),
    "transposed_scores": ("out[seen] = (E / Z) @ V", "out[seen] = (E / Z) @ V[::-1]"),
    "tree_bits_reversed": ("if (int(words[i]) >> k) & 1:", "if (int(words[i]) >> (n - 1 - k)) & 1:"),
    "tree_transposed": ("if (int(words[i]) >> k) & 1:", "if (int(words[k]) >> i) & 1:"),
    "tree_no_offset": ("M[i, l + k] = 0.0", "M[i, k] = 0.0"),
    "tree_context_hidden": ("M[:, :l] = 0.0", "M[:, : max(l - 1, 0)] = 0.0"),
    "tree_high_bits_count": ("        for k in range(n):\n            if (int(words[i])",
                             "        for k in range(n):\n            if k == n - 1 or (int(words[i])"),
    "dead_row_lse_zero": ("lse = np.full(Q.shape[0], -np.inf)", "lse = np.zeros(Q.shape[0])"),
    "tree_ignored": ("M = chain_mask(l, n) if draft_mask is None else tree_mask(l, n, draft_mask[b])",
                     "M = chain_mask(l, n)"),
}


def _mutant(src, old, new):
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "<mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name):
    with open(oracle_mod.__file__) as f:
        src = f.read()
    mod = _mutant(src, *MUTATIONS[name])
    caught = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin(mod)
        except Exception:
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutation {name}"


# ------------------------------------------------- workload recipe checks

def test_workload_lengths_and_shapes():
    for w in wl.WORKLOADS:
        ctx, chunk = wl.draw_lengths(w)
        assert ctx.shape == (w.B,) and chunk.shape == (w.B,)
        assert np.all(ctx + chunk <= w.S_max)
        assert np.all(chunk >= 1) and np.all(chunk <= w.C_max)
        if w.ctx[0] == "fixed":
            assert list(ctx) == list(w.ctx[1])
        else:
            assert ctx.min() >= w.ctx[1] and ctx.max() <= w.ctx[2]
        # determinism: the recipe is a pure function of the workload
        ctx2, chunk2 = wl.draw_lengths(w)
        assert np.array_equal(ctx, ctx2) and np.array_equal(chunk, chunk2)
    assert wl.get(5).group == 7 and wl.get(2).S_max == 2304


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, np.nan], np.float32)
    bits = wl.f32_to_bf16_bits(x)
    # 1+2^-8 is a tie between 1 and 1+2^-7: even mantissa (1.0) wins;
    # 1+3*2^-8 ties between 1+2^-7 and 1+2^-6: even (1+2^-6) wins
    assert list(bits[:5]) == [0x3F80, 0x3F80, 0x3F82, 0x3F80, 0xC020]
    assert bits[5] == 0x7FC0


def test_sampled_batches_match_full_generation():
    w = wl.get(2)
    full = wl.make_inputs(wl.dataclasses.replace(w, B=4), fill=0.0)
    part = wl.make_inputs(wl.dataclasses.replace(w, B=4), fill=0.0, batches=[2])
    assert np.array_equal(full["k_cache"][2], part["k_cache"][2])
    assert np.array_equal(full["v_cache"][2], part["v_cache"][2])


def test_kv_accounting_matches_paper_cost_model():
    """Algorithmic KV bytes follow the cost table's 2*b*s*h/g (Section 3.2) and
    reproduce the paper's KV sizing (Section 3.3)."""
    vals = {}
    with open(os.path.join(GOLDEN, "paper_kv_sizing.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                k_, v_ = line.split()
                vals[k_] = int(v_)
    w = wl.Workload("mixtral_layer", 99, B=1, Hq=vals["q_heads"], Hkv=vals["kv_heads"],
                    D=vals["head_dim"], dtype="bf16", ctx=("fixed", [0]), chunk=("fixed", 1),
                    description="")
    s = vals["input_len"] + vals["output_len"]
    g = w.Hq // w.Hkv
    h = w.Hq * w.D
    for batch, gib in ((vals["batch_a30"], vals["kv_gib_a30"]),
                       (vals["batch_4090d"], vals["kv_gib_4090d"])):
        ctx = np.full(batch, s - 1)
        chunk = np.ones(batch)
        per_layer = wl.algorithmic_kv_bytes(w, ctx, chunk)
        assert per_layer == 2 * batch * s * h // g * vals["elt_bytes"]
        total_gib = per_layer * vals["layers"] / 2 ** 30
        assert abs(total_gib - gib) / gib < 1e-3, total_gib


def test_tree_masks_are_root_paths():
    """The tree recipe's words are root paths of a tree: word i holds bit i,
    bits only at or below i, and removing bit i leaves the word of i's parent
    (its highest remaining bit); rows past c_b are 0; draws repeat."""
    chunk = np.array([16, 1, 0, 9], np.int32)
    words = wl.tree_draft_masks(6, chunk, 16)
    assert words.dtype == np.uint64 and words.shape == (4, 16)
    for b, n in enumerate(chunk):
        for i in range(16):
            w = int(words[b, i])
            if i >= n:
                assert w == 0
                continue
            assert (w >> i) & 1 and w < (1 << (i + 1))
            if i == 0:
                assert w == 1
            else:
                rest = w & ~(1 << i)
                parent = rest.bit_length() - 1
                assert 0 <= parent < i and int(words[b, parent]) == rest
    assert np.array_equal(words, wl.tree_draft_masks(6, chunk, 16))
    w6 = wl.get("mixtral_tree_b64")
    inp = wl.make_inputs(wl.dataclasses.replace(w6, B=2), batches=[])
    assert inp["draft_mask"].shape == (2, 16) and inp["draft_mask"][0, 0] == 1
    assert wl.make_inputs(wl.dataclasses.replace(wl.get(1)))["draft_mask"] is None


# ------------------------------------------------------------ paged caches

def test_gather_pages_identity_and_shuffled():
    """Pages cut from a contiguous cache in order gather back to it exactly;
    a shuffled pool with its table gives the same attention results."""
    rng = np.random.default_rng(51)
    q, k, v, ctx, chunk = _rand_case(rng, B=3, ctx=(20, 3, 41), chunk=(4, 2, 3), C_max=4, S_pad=0)
    S = int((ctx + chunk).max())
    S = (S + 7) // 8 * 8
    k = np.pad(k, ((0, 0), (0, 0), (0, S - k.shape[2]), (0, 0)))
    v = np.pad(v, ((0, 0), (0, 0), (0, S - v.shape[2]), (0, 0)))
    ps, P = 8, S // 8
    ident = np.arange(3 * P, dtype=np.int32).reshape(3, P)
    pages = k.reshape(3, k.shape[1], P, ps, k.shape[3]).transpose(0, 2, 1, 3, 4).reshape(3 * P, k.shape[1], ps, -1)
    assert np.array_equal(oracle_mod.gather_pages(pages, ident, ps), k)
    kp, table = wl.paginate(k, ps, 7, np.float32(np.nan))
    vp, table_v = wl.paginate(v, ps, 7, np.float32(np.nan))
    assert np.array_equal(table, table_v) and len(np.unique(table)) == table.size
    assert np.all(np.isnan(np.delete(kp, table.ravel(), axis=0)))     # spare pages are poisoned
    o1, s1 = oracle_mod.verify_attn_ref(q, k, v, ctx, chunk, 0.3, "f32")
    o2, s2 = oracle_mod.verify_attn_ref(q, oracle_mod.gather_pages(kp, table, ps),
                                        oracle_mod.gather_pages(vp, table, ps), ctx, chunk, 0.3, "f32")
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(s1, s2)


@pytest.mark.parametrize("old,new", [
    ("pages[int(table[b, t])]", "pages[int(table[b, P - 1 - t])]"),          # pages out of order
    ("pages[int(table[b, t])]", "pages[int(table[b, t])][:, ::-1]"),         # rows reversed in a page
    ("pages[int(table[b, t])]", "pages[int(table[(b + 1) % B, t])]"),        # another sequence's table
])
def test_gather_pages_catches_planted_mistake(old, new):
    with open(oracle_mod.__file__) as f:
        src = f.read()
    _gather_pin(oracle_mod)
    mod = _mutant(src, old, new)
    with pytest.raises(AssertionError):
        _gather_pin(mod)


def _gather_pin(m):
    """Pages in order gather back to the cache they were cut from; so does a
    shuffled pool through its table."""
    rng = np.random.default_rng(52)
    k = rng.standard_normal((3, 2, 24, 4)).astype(np.float32)
    ps, P = 8, 3
    ident = np.arange(3 * P, dtype=np.int32).reshape(3, P)
    pages = k.reshape(3, 2, P, ps, 4).transpose(0, 2, 1, 3, 4).reshape(3 * P, 2, ps, 4)
    assert np.array_equal(m.gather_pages(pages, ident, ps), k)
    kp, table = wl.paginate(k, ps, 3, np.float32(np.nan))
    assert np.array_equal(m.gather_pages(kp, table, ps), k)
