"""Pins of the acceptance-step oracle (greedy verification of draft tokens).

Each pin checks the oracle against something it does not compute itself:
logits built so that every row's maximum is known, draft tokens chosen so
that the accepted length is known in advance, exact ties, the chunk of 1
(plain greedy decoding), bf16 against the f32 values it decodes to, and the
invariants that tie the outputs together.  Planted mistakes in copies of the
oracle must each be caught by some pin.
"""
import types

import numpy as np
import pytest

from oracle import acceptance as acc_mod
from paper_2508_21706_amd import workloads as wl


def _known_rows(rng, B, C, V, lo=-3.0, hi=3.0):
    """Logits whose row maxima are planted: every row has one entry at 10,
    the rest uniform in [lo, hi]; returns the logits and the planted ids."""
    x = rng.uniform(lo, hi, size=(B, C, V)).astype(np.float32)
    best = rng.integers(0, V, size=(B, C))
    x[np.arange(B)[:, None], np.arange(C)[None, :], best] = 10.0
    return x, best


def pin_known_acceptance_lengths(m):
    """Draft token i+1 equals row i's planted maximum for i < k_b and differs
    at i = k_b: exactly k_b drafts are accepted, the next token is row k_b's
    maximum and the context grows by k_b + 1."""
    rng = np.random.default_rng(31)
    B, C, V = 6, 5, 50
    x, best = _known_rows(rng, B, C, V)
    k = np.array([0, 1, 2, 3, 4, 2])
    tokens = np.zeros((B, C), np.int32)
    tokens[:, 0] = rng.integers(0, V, B)
    for b in range(B):
        for i in range(C - 1):
            tokens[b, i + 1] = best[b, i] if i < k[b] else (best[b, i] + 1 + i) % V
    ctx = np.array([0, 7, 100, 5, 1, 2048], np.int32)
    chunk = np.full(B, C, np.int32)
    r = m.accept_greedy_ref(x, tokens, ctx, chunk, "f32")
    assert list(r["accepted"]) == list(k)
    assert list(r["next_token"]) == [best[b, k[b]] for b in range(B)]
    assert list(r["new_ctx_lens"]) == list(ctx + k + 1)
    assert np.array_equal(r["argmax"], best)


def pin_rejection_stops_acceptance(m):
    """A rejected draft ends the accepted prefix even if later drafts would
    match their rows."""
    rng = np.random.default_rng(32)
    x, best = _known_rows(rng, 1, 6, 40)
    tokens = np.zeros((1, 6), np.int32)
    tokens[0, 1:] = best[0, :5]
    tokens[0, 3] = (best[0, 2] + 5) % 40          # reject the third draft only
    r = m.accept_greedy_ref(x, tokens, np.array([9]), np.array([6]), "f32")
    assert r["accepted"][0] == 2 and r["next_token"][0] == best[0, 2] and r["new_ctx_lens"][0] == 12


def pin_ties_take_lowest_id(m):
    """Equal maxima: the lowest token id wins (also for +0 against -0)."""
    x = np.zeros((1, 3, 12), np.float32)
    x[0, 0, [9, 4, 7]] = 2.5                      # tie at 4, 7, 9
    x[0, 1, :] = -1.0
    x[0, 1, [11, 3]] = 0.0                        # tie between +0 at 3 and 11
    x[0, 1, 3] = -0.0
    x[0, 2, :] = -7.0                             # all equal: id 0
    tokens = np.array([[5, 4, 3]], np.int32)
    r = m.accept_greedy_ref(x, tokens, np.array([3]), np.array([3]), "f32")
    assert list(r["argmax"][0]) == [4, 3, 0]
    assert r["accepted"][0] == 2 and r["next_token"][0] == 0 and r["new_ctx_lens"][0] == 6


def pin_chunk_of_one_is_greedy_decoding(m):
    """A chunk of 1 holds no draft: the step is one greedy decode."""
    rng = np.random.default_rng(33)
    x, best = _known_rows(rng, 4, 3, 30)
    tokens = rng.integers(0, 30, size=(4, 3)).astype(np.int32)
    r = m.accept_greedy_ref(x, tokens, np.array([1, 2, 3, 4]), np.array([1, 1, 1, 1]), "f32")
    assert np.all(r["accepted"] == 0)
    assert list(r["next_token"]) == list(best[:, 0])
    assert list(r["new_ctx_lens"]) == [2, 3, 4, 5]
    assert np.all(r["argmax"][:, 1:] == -1)


def pin_empty_chunk_takes_no_step(m):
    x = np.full((2, 2, 8), np.nan, np.float32)    # never read
    x[1, 0] = np.arange(8)
    r = m.accept_greedy_ref(x, np.zeros((2, 2), np.int32), np.array([5, 6]), np.array([0, 1]), "f32")
    assert r["accepted"][0] == 0 and r["next_token"][0] == -1 and r["new_ctx_lens"][0] == 5
    assert np.all(r["argmax"][0] == -1)
    assert r["next_token"][1] == 7 and r["new_ctx_lens"][1] == 7


def pin_all_accepted(m):
    """Every draft equal to its prediction: c - 1 accepted, the bonus token is
    the last row's prediction."""
    rng = np.random.default_rng(34)
    x, best = _known_rows(rng, 3, 4, 25)
    tokens = np.zeros((3, 4), np.int32)
    tokens[:, 1:] = best[:, :3]
    chunk = np.array([4, 3, 2], np.int32)
    r = m.accept_greedy_ref(x, tokens, np.array([0, 0, 0]), chunk, "f32")
    assert list(r["accepted"]) == [3, 2, 1]
    assert list(r["next_token"]) == [best[0, 3], best[1, 2], best[2, 1]]
    assert list(r["new_ctx_lens"]) == [4, 3, 2]


def pin_bf16_decodes_to_f32(m):
    w = wl.AcceptWorkload("t", 35, B=4, C_max=3, V=64, dtype="bf16", accept_prob=0.5, description="")
    inp = wl.make_accept_inputs(w, chunk_lens=[3, 2, 1, 3])
    back = (inp["logits"].astype(np.uint32) << 16).view(np.float32)
    r1 = m.accept_greedy_ref(inp["logits"], inp["tokens"], inp["ctx_lens"], inp["chunk_lens"], "bf16")
    r2 = m.accept_greedy_ref(back, inp["tokens"], inp["ctx_lens"], inp["chunk_lens"], "f32")
    for key in r1:
        assert np.array_equal(r1[key], r2[key]), key


def pin_invariants(m):
    """On random inputs: 0 <= a < c, the next token is row a's argmax, every
    accepted draft equals its prediction and the first rejected one does not,
    and the context grows by a + 1."""
    w = wl.AcceptWorkload("t", 36, B=40, C_max=6, V=97, dtype="f32", accept_prob=0.8, description="")
    chunk = np.random.default_rng(36).integers(0, 7, size=40)
    inp = wl.make_accept_inputs(w, chunk_lens=chunk)
    r = m.accept_greedy_ref(inp["logits"], inp["tokens"], inp["ctx_lens"], inp["chunk_lens"], "f32")
    for b in range(40):
        c, a = int(chunk[b]), int(r["accepted"][b])
        if c == 0:
            continue
        assert 0 <= a < c
        for i in range(c):       # each row's argmax is a maximum, and the first one
            row = inp["logits"][b, i].astype(np.float64)
            j = int(r["argmax"][b, i])
            assert row[j] == row.max() and not np.any(row[:j] == row.max())
        assert all(r["argmax"][b, i] == inp["tokens"][b, i + 1] for i in range(a))
        if a < c - 1:
            assert r["argmax"][b, a] != inp["tokens"][b, a + 1]
        assert r["next_token"][b] == r["argmax"][b, a]
        assert r["new_ctx_lens"][b] == inp["ctx_lens"][b] + a + 1


# ------------------------------------------------------------- tree drafts

def _tree_words(parents):
    """Root-path words of a tree given by parent indices (parents[0] = -1)."""
    words = []
    for i, par in enumerate(parents):
        words.append((1 << i) | (words[par] if par >= 0 else 0))
    return words


def pin_tree_chain_is_greedy(m):
    """Chain words make tree acceptance the chain acceptance, with the path
    of the first a + 1 tokens."""
    w = wl.AcceptWorkload("t", 37, B=12, C_max=6, V=53, dtype="f32", accept_prob=0.8, description="")
    chunk = np.random.default_rng(37).integers(0, 7, size=12)
    inp = wl.make_accept_inputs(w, chunk_lens=chunk)
    words = np.zeros((12, 6), np.uint64)
    for b in range(12):
        words[b, : chunk[b]] = [(1 << (i + 1)) - 1 for i in range(int(chunk[b]))]
    r1 = m.accept_greedy_ref(inp["logits"], inp["tokens"], inp["ctx_lens"], chunk, "f32")
    r2 = m.accept_tree_ref(inp["logits"], inp["tokens"], words, inp["ctx_lens"], chunk, "f32")
    for key in r1:
        assert np.array_equal(r1[key], r2[key]), key
    for b in range(12):
        want = (1 << (int(r1["accepted"][b]) + 1)) - 1 if chunk[b] else 0
        assert int(r2["path"][b]) == want


def pin_tree_known_branches(m):
    """Root 0; 1 and 2 under 0; 3 under 1; 4 under 2; 5 under 4.  Node 1
    misses, node 2 matches, node 3 matches its (rejected) parent's
    prediction, node 4 matches, node 5 misses: the path is 0-2-4."""
    rng = np.random.default_rng(38)
    x, best = _known_rows(rng, 1, 6, 40)
    words = np.array([_tree_words([-1, 0, 0, 1, 2, 4])], np.uint64)
    tok = np.zeros((1, 6), np.int32)
    tok[0, 1] = (best[0, 0] + 1) % 40
    tok[0, 2] = best[0, 0]
    tok[0, 3] = best[0, 1]
    tok[0, 4] = best[0, 2]
    tok[0, 5] = (best[0, 4] + 3) % 40
    r = m.accept_tree_ref(x, tok, words, np.array([10]), np.array([6]), "f32")
    assert int(r["path"][0]) == 0b10101 and r["accepted"][0] == 2
    assert r["next_token"][0] == best[0, 4] and r["new_ctx_lens"][0] == 13


def pin_tree_ties_take_lowest_index(m):
    """Two equally deep accepted nodes (siblings 1 and 2 carry the same
    token): the lower index wins; a deeper node beats both."""
    rng = np.random.default_rng(39)
    x, best = _known_rows(rng, 2, 4, 30)
    words = np.array([_tree_words([-1, 0, 0, 2]), _tree_words([-1, 0, 0, 2])], np.uint64)
    tok = np.zeros((2, 4), np.int32)
    tok[:, 1] = best[:, 0]
    tok[:, 2] = best[:, 0]
    tok[0, 3] = (best[0, 2] + 1) % 30      # node 3 (under 2) misses: depth-1 tie, node 1 wins
    tok[1, 3] = best[1, 2]                  # node 3 matches: depth 2 through node 2
    r = m.accept_tree_ref(x, tok, words, np.array([0, 0]), np.array([4, 4]), "f32")
    assert int(r["path"][0]) == 0b11 and r["next_token"][0] == best[0, 1]
    assert int(r["path"][1]) == 0b1101 and r["accepted"][1] == 2 and r["next_token"][1] == best[1, 3]


def pin_compaction_makes_the_path_a_chain(m):
    """After compaction, chain attention over the context plus the accepted
    path equals the tree attention of the path's nodes (the path's K/V rows
    are what its nodes attended to)."""
    from oracle import reference as ref
    rng = np.random.default_rng(40)
    B, Hq, Hkv, D, C = 2, 4, 2, 8, 6
    ctx = np.array([7, 3], np.int32)
    chunk = np.array([6, 5], np.int32)
    S = 16
    q = rng.standard_normal((B, C, Hq, D)).astype(np.float32)
    k = rng.standard_normal((B, Hkv, S, D)).astype(np.float32)
    v = rng.standard_normal((B, Hkv, S, D)).astype(np.float32)
    words = np.zeros((B, C), np.uint64)
    words[0, :6] = _tree_words([-1, 0, 0, 1, 2, 4])
    words[1, :5] = _tree_words([-1, 0, 1, 0, 3])
    paths = [0b10101, 0b11001]
    o_t, s_t = ref.verify_attn_ref(q, k, v, ctx, chunk, 0.4, "f32", draft_mask=words)
    kc = m.compact_path_ref(k, ctx, paths)
    vc = m.compact_path_ref(v, ctx, paths)
    for b in range(B):
        nodes = [i for i in range(C) if (paths[b] >> i) & 1]
        qp = np.zeros((1, C, Hq, D), np.float32)
        qp[0, : len(nodes)] = q[b, nodes]
        o_c, s_c = ref.verify_attn_ref(qp, kc[b:b + 1], vc[b:b + 1], ctx[b:b + 1],
                                       np.array([len(nodes)], np.int32), 0.4, "f32")
        np.testing.assert_allclose(o_c[0, : len(nodes)], o_t[b, nodes], rtol=0, atol=1e-12)
        np.testing.assert_allclose(s_c[0, : len(nodes)], s_t[b, nodes], rtol=0, atol=1e-12)
        # rows outside the moved range keep their values
        assert np.array_equal(kc[b, :, : ctx[b]], k[b, :, : ctx[b]])
        assert np.array_equal(kc[b, :, ctx[b] + len(nodes):], k[b, :, ctx[b] + len(nodes):])


PINS = [pin_known_acceptance_lengths, pin_rejection_stops_acceptance, pin_ties_take_lowest_id,
        pin_chunk_of_one_is_greedy_decoding, pin_empty_chunk_takes_no_step, pin_all_accepted,
        pin_bf16_decodes_to_f32, pin_invariants, pin_tree_chain_is_greedy, pin_tree_known_branches,
        pin_tree_ties_take_lowest_index, pin_compaction_makes_the_path_a_chain]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_accept_oracle_pin(pin):
    pin(acc_mod)


MUTATIONS = {
    "compares_same_position": ("argmax[b, a] == int(draft_tokens[b, a + 1])", "argmax[b, a] == int(draft_tokens[b, a])"),
    "last_of_ties": ("return int(np.argmax(row))", "return int(len(row) - 1 - np.argmax(row[::-1]))"),
    "ctx_without_bonus": ("new_ctx[b] = int(ctx_lens[b]) + a + 1", "new_ctx[b] = int(ctx_lens[b]) + a"),
    "next_after_prediction": ("next_token[b] = argmax[b, a]", "next_token[b] = argmax[b, min(a + 1, c - 1)]"),
    "accepts_one_more": ("while a < c - 1 and", "while a < c and a < C_max - 1 and"),
    "tree_parent_lowest_bit": ("    return rest.bit_length() - 1", "    return (rest & -rest).bit_length() - 1"),
    "tree_ignores_parent": ("ok[i] = ok[par] and argmax[b, par]", "ok[i] = argmax[b, par]"),
    "tree_ties_highest": ("key=lambda i: (depth[i], -i)", "key=lambda i: (depth[i], i)"),
    "compaction_reversed": ("for j, k in enumerate(nodes):", "for j, k in enumerate(nodes[::-1]):"),
    "keeps_going_after_reject": ("while a < c - 1 and argmax[b, a] == int(draft_tokens[b, a + 1]):\n            a += 1",
                                 "a = sum(int(argmax[b, i] == int(draft_tokens[b, i + 1])) for i in range(c - 1))"),
}


def _mutant(src, old, new):
    assert src.count(old) == 1, old
    mod = types.ModuleType("accept_mutant")
    mod.__dict__["__package__"] = "oracle"
    exec(compile(src.replace(old, new), "<mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_accept_pins_catch_planted_mistake(name):
    with open(acc_mod.__file__) as f:
        src = f.read()
    mod = _mutant(src, *MUTATIONS[name])
    caught = []
    for pin in PINS:
        try:
            pin(mod)
        except Exception:
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutation {name}"


def test_accept_workload_recipe():
    w = wl.ACCEPT_BY_NAME["accept_mixtral_b64"]
    inp = wl.make_accept_inputs(w)
    assert inp["logits"].shape == (64, 5, 32000) and inp["logits"].dtype == np.uint16
    assert inp["tokens"].shape == (64, 5) and inp["tokens"].dtype == np.int32
    assert np.all((inp["tokens"] >= 0) & (inp["tokens"] < 32000))
    inp2 = wl.make_accept_inputs(w)
    assert np.array_equal(inp["logits"], inp2["logits"]) and np.array_equal(inp["tokens"], inp2["tokens"])
    short = wl.make_accept_inputs(wl.ACCEPT_BY_NAME["accept_tiny_f32"], chunk_lens=[4, 0, 2])
    assert np.all(np.isnan(short["logits"][1])) and np.all(short["tokens"][1] == -1)
    assert np.all(np.isnan(short["logits"][2, 2:])) and np.all(short["tokens"][2, 2:] == -1)
