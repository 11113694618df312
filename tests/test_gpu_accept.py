"""GPU parity of the acceptance step (greedy verification of draft tokens)
against the CPU oracle, through the C-ABI.  Every output is an integer, so
the bar is bit-exact equality."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import accept_greedy_ref

pytestmark = pytest.mark.gpu


def dev():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a GPU")
    return torch.device("cuda:0")


def note(msg):
    print(msg, flush=True)


def logits_dev(x, dtype):
    if dtype in ("bf16", "f16"):
        t16 = torch.bfloat16 if dtype == "bf16" else torch.float16
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(t16).to(dev())
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(dev())


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev())


def run_accept(logits, tokens, ctx, chunk, dtype, split=0, workspace=None):
    d = dev()
    B, C = tokens.shape
    out = {k: torch.full(s, -7, dtype=torch.int32, device=d)
           for k, s in (("argmax", (B, C)), ("accepted", (B,)), ("next_token", (B,)), ("new_ctx_lens", (B,)))}
    pkg.accept_greedy(logits_dev(logits, dtype), i32(tokens), i32(ctx), i32(chunk), out=out, split=split,
                      workspace=workspace)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy().astype(np.int64) for k, v in out.items()}


def check(logits, tokens, ctx, chunk, dtype, label, split=0, workspace=None):
    note(f"case {label} split={split}")
    got = run_accept(logits, tokens, ctx, chunk, dtype, split, workspace)
    ref = accept_greedy_ref(logits, tokens, ctx, chunk, dtype)
    for k in ref:
        assert np.array_equal(got[k], ref[k]), f"{label}: {k} differs at {np.argwhere(got[k] != ref[k])[:5]}"
    note(f"[{label}] accepted histogram {np.bincount(ref['accepted']).tolist()}")
    return got


@pytest.mark.parametrize("name", ["accept_tiny_f32", "accept_mixtral_b64", "accept_large_b256"])
def test_accept_workloads(name):
    w = wl.ACCEPT_BY_NAME[name]
    inp = wl.make_accept_inputs(w)
    for split in (0, 2048, 4096 if w.dtype == "f32" else 8192, 32768):
        check(inp["logits"], inp["tokens"], inp["ctx_lens"], inp["chunk_lens"], w.dtype, name, split)


def test_accept_ragged_and_empty_chunks():
    w = dataclasses.replace(wl.ACCEPT_BY_NAME["accept_mixtral_b64"], B=9, C_max=7, V=4096, accept_prob=0.85)
    chunk = np.array([0, 1, 7, 3, 0, 2, 7, 5, 1], np.int32)
    inp = wl.make_accept_inputs(w, chunk_lens=chunk)
    for split in (0, 2048):
        check(inp["logits"], inp["tokens"], inp["ctx_lens"], chunk, "bf16", "ragged chunks", split)


def test_accept_ties_across_slices():
    """Equal maxima in different slices (and lanes, and waves): the lowest
    token id wins; +0 ties -0; a row of -inf elects token 0; a row of equal
    values elects token 0."""
    B, C, V = 2, 4, 8192
    x = np.random.default_rng(41).uniform(-4, 4, size=(B, C, V)).astype(np.float32)
    x[0, 0, [7000, 2049, 5000]] = 9.0                 # slices 3, 1, 2 at split 2048
    x[0, 1, :] = -1.0
    x[0, 1, [4095, 1, 4096]] = 0.0
    x[0, 1, 1] = -0.0                                  # -0 at the lowest id
    x[0, 2, :] = -np.inf
    x[0, 3, :] = 3.25
    x[1, 0, [8191, 8190]] = 20.0
    x[1, 1, [0, 8191]] = 20.0
    x[1, 2, 64 * 8 + 3] = 30.0                         # one lane apart
    x[1, 2, 64 * 8 + 2] = 30.0
    x[1, 3, [6000, 255]] = 11.0                       # different slices at split 2048
    tokens = np.array([[0, 2049, 1, 0], [5, 8190, 0, 514]], np.int32)
    for dtype in ("f32", "bf16"):
        lg = x if dtype == "f32" else wl.f32_to_bf16_bits(x)
        for split in (0, 2048, 4096):
            got = check(lg, tokens, np.array([10, 20]), np.array([4, 4]), dtype, f"ties {dtype}", split)
            assert list(got["argmax"][0]) == [2049, 1, 0, 0]
            assert list(got["argmax"][1]) == [8190, 0, 514, 255]


def test_accept_in_place_and_workspace_reuse():
    """ctx_lens updated in place; one workspace serves calls with different
    batches and slice widths, and its counters are left zero."""
    d = dev()
    w = wl.ACCEPT_BY_NAME["accept_mixtral_b64"]
    big = pkg.accept_desc(w.B, w.C_max, w.V, 1, 2048)
    ws = pkg.alloc_accept_workspace(big, d)
    for trial, (B, split) in enumerate([(64, 0), (17, 2048), (64, 8192), (3, 0)]):
        ww = dataclasses.replace(w, B=B, index=50 + trial)
        chunk = np.random.default_rng(trial).integers(0, w.C_max + 1, size=B).astype(np.int32)
        inp = wl.make_accept_inputs(ww, chunk_lens=chunk)
        ctx_d = i32(inp["ctx_lens"])
        note(f"case in-place trial {trial} B={B} split={split}")
        out = pkg.accept_greedy(logits_dev(inp["logits"], "bf16"), i32(inp["tokens"]), ctx_d, i32(chunk),
                                workspace=ws, split=split, in_place=True)
        torch.cuda.synchronize()
        ref = accept_greedy_ref(inp["logits"], inp["tokens"], inp["ctx_lens"], chunk, "bf16")
        assert out["new_ctx_lens"] is ctx_d
        for k in ref:
            assert np.array_equal(out[k].cpu().numpy(), ref[k]), (trial, k)
    counters = ws[: 65536 * 4].view(torch.int32).cpu()
    assert int(counters.abs().sum()) == 0


def test_accept_single_position_chunks():
    """C_max = 1: every step is plain greedy decoding."""
    w = dataclasses.replace(wl.ACCEPT_BY_NAME["accept_mixtral_b64"], B=33, C_max=1, V=2048)
    inp = wl.make_accept_inputs(w)
    got = check(inp["logits"], inp["tokens"], inp["ctx_lens"], inp["chunk_lens"], "bf16", "chunk of one")
    assert np.all(got["accepted"] == 0) and np.array_equal(got["new_ctx_lens"], inp["ctx_lens"] + 1)


def test_accept_rejects_bad_shapes():
    d = dev()
    x = torch.zeros((2, 3, 1001), dtype=torch.float32, device=d)
    t = torch.zeros((2, 3), dtype=torch.int32, device=d)
    n = torch.ones(2, dtype=torch.int32, device=d)
    with pytest.raises(pkg.SpecMoEError) as e:
        pkg.accept_greedy(x, t, n, n)
    assert e.value.status == -2


@pytest.mark.parametrize("B,C,V", [(5000, 1, 512), (3000, 2, 1024), (700, 3, 4096)])
def test_accept_many_short_sequences(B, C, V):
    """Many sequences of few short rows: workgroup ranges meet many sequences,
    both with arrivals counted per workgroup (through LDS) and, past 16
    sequences per workgroup range, per wave."""
    w = dataclasses.replace(wl.ACCEPT_BY_NAME["accept_mixtral_b64"], B=B, C_max=C, V=V, accept_prob=0.8,
                            index=60 + C)
    chunk = np.random.default_rng(B).integers(0, C + 1, size=B).astype(np.int32)
    inp = wl.make_accept_inputs(w, chunk_lens=chunk)
    for split in (0, 512):
        check(inp["logits"], inp["tokens"], inp["ctx_lens"], chunk, "bf16", f"short sequences B={B} C={C}", split)


# ------------------------------------------------------------- tree drafts

def _tree_case(seed, B, C, V, dtype, p_hit=0.75):
    """Random recursive trees with planted predictions; node i's token is its
    parent's planted prediction with probability p_hit."""
    from oracle import tree_parent
    w = wl.AcceptWorkload("tree", seed, B=B, C_max=C, V=V, dtype=dtype, accept_prob=0.0, description="")
    rng = np.random.default_rng(seed)
    chunk = rng.integers(0, C + 1, size=B).astype(np.int32)
    chunk[: max(1, B // 4)] = C
    inp = wl.make_accept_inputs(w, chunk_lens=chunk)
    words = wl.tree_draft_masks(seed, chunk, C)
    tokens = inp["tokens"].copy()
    for b in range(B):
        for i in range(1, int(chunk[b])):
            par = tree_parent(words[b], i)
            tokens[b, i] = inp["planted"][b, par] if rng.random() < p_hit else (inp["planted"][b, par] + 7) % V
    return inp, tokens, words, chunk


def run_tree(inp, tokens, words, chunk, dtype, split=0):
    d = dev()
    B, C = tokens.shape
    out = {k: torch.full(s, -7, dtype=torch.int32, device=d)
           for k, s in (("argmax", (B, C)), ("accepted", (B,)), ("next_token", (B,)), ("new_ctx_lens", (B,)))}
    out["path"] = torch.full((B,), -7, dtype=torch.int64, device=d)
    pkg.accept_greedy_tree(logits_dev(inp["logits"], dtype), i32(tokens), torch.from_numpy(words.view(np.int64)).to(d),
                           i32(inp["ctx_lens"]), i32(chunk), out=out, split=split)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy().astype(np.int64) for k, v in out.items()}


@pytest.mark.parametrize("B,C,V,dtype", [(64, 16, 32000, "bf16"), (40, 64, 4096, "f32"), (300, 5, 2048, "bf16"),
                                         (7, 1, 1024, "f32")])
def test_accept_tree_matches_oracle(B, C, V, dtype):
    from oracle import accept_tree_ref
    inp, tokens, words, chunk = _tree_case(70 + C, B, C, V, dtype)
    ref = accept_tree_ref(inp["logits"], tokens, words, inp["ctx_lens"], chunk, dtype)
    for split in (0, 512):
        note(f"case tree acceptance B={B} C={C} V={V} {dtype} split={split}")
        got = run_tree(inp, tokens, words, chunk, dtype, split)
        for k in ("argmax", "accepted", "next_token", "new_ctx_lens"):
            assert np.array_equal(got[k], ref[k]), (k, np.argwhere(got[k] != ref[k])[:5])
        assert [int(x) & ((1 << 64) - 1) for x in got["path"]] == [int(x) for x in ref["path"]]
    note(f"[tree acceptance] accepted histogram {np.bincount(ref['accepted']).tolist()}")


def test_accept_tree_chain_words_equal_chain_call():
    w = dataclasses.replace(wl.ACCEPT_BY_NAME["accept_mixtral_b64"], B=20, V=4096)
    chunk = np.random.default_rng(5).integers(0, w.C_max + 1, size=20).astype(np.int32)
    inp = wl.make_accept_inputs(w, chunk_lens=chunk)
    words = np.zeros((20, w.C_max), np.uint64)
    for b in range(20):
        words[b, : chunk[b]] = [(1 << (i + 1)) - 1 for i in range(int(chunk[b]))]
    # chain tokens: draft i + 1 follows position i; tree tokens: node i's own
    chain = run_accept(inp["logits"], inp["tokens"], inp["ctx_lens"], chunk, "bf16")
    tree = run_tree(inp, inp["tokens"], words, chunk, "bf16")
    for k in ("argmax", "accepted", "next_token", "new_ctx_lens"):
        assert np.array_equal(chain[k], tree[k]), k


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("f16", 64), ("f32", 128)])
def test_compact_accepted_kv_matches_oracle(dtype, D):
    """The accepted paths' K/V rows move after each context, overlapping
    moves included; every other row keeps its value."""
    from oracle import accept_tree_ref, compact_path_ref
    d = dev()
    B, Hkv, C = 9, 3, 12
    inp, tokens, words, chunk = _tree_case(90, B, C, 2048, "f32", p_hit=0.9)
    ref = accept_tree_ref(inp["logits"], tokens, words, inp["ctx_lens"], chunk, "f32")
    ctx = np.random.default_rng(91).integers(0, 300, B).astype(np.int32)
    S = 320
    kv = [np.random.default_rng(92 + t).standard_normal((B, Hkv, S, D)).astype(np.float32) for t in range(2)]
    enc = {"bf16": wl.f32_to_bf16_bits, "f16": wl.f32_to_f16_bits, "f32": lambda a: a}[dtype]
    k_h, v_h = enc(kv[0]), enc(kv[1])
    k_d = logits_dev(k_h, dtype) if dtype != "f32" else torch.from_numpy(k_h).to(d)
    v_d = logits_dev(v_h, dtype) if dtype != "f32" else torch.from_numpy(v_h).to(d)
    paths = np.array([int(x) for x in ref["path"]], dtype=np.uint64)
    note(f"case compaction {dtype} D={D}")
    pkg.compact_accepted_kv(k_d, v_d, i32(ctx), torch.from_numpy(paths.view(np.int64)).to(d))
    torch.cuda.synchronize()
    want_k = compact_path_ref(k_h, ctx, [int(x) for x in paths])
    want_v = compact_path_ref(v_h, ctx, [int(x) for x in paths])
    got_k = k_d.cpu().view(torch.int16).numpy().view(np.uint16) if dtype != "f32" else k_d.cpu().numpy()
    got_v = v_d.cpu().view(torch.int16).numpy().view(np.uint16) if dtype != "f32" else v_d.cpu().numpy()
    assert np.array_equal(got_k, want_k) and np.array_equal(got_v, want_v)
    assert any(bin(int(x)).count("1") > 2 and int(x) != (1 << bin(int(x)).count("1")) - 1 for x in paths), \
        "the case must hold paths with gaps"


def test_accept_tree_rejects_wide_chunks():
    d = dev()
    x = torch.zeros((1, 65, 512), dtype=torch.bfloat16, device=d)
    t = torch.zeros((1, 65), dtype=torch.int32, device=d)
    n = torch.ones(1, dtype=torch.int32, device=d)
    with pytest.raises(pkg.SpecMoEError) as e:
        pkg.accept_greedy_tree(x, t, torch.zeros((1, 65), dtype=torch.int64, device=d), n, n)
    assert e.value.status == -13
