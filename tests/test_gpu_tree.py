"""GPU parity of the tree-draft entry point (draft-mask words) against the
fp64 CPU oracle, through the C-ABI.

Same tolerances as the chain tests: f32 inputs 1e-4 on out and lse, bf16
inputs 1e-2 on out and 1e-3 on lse.  Rows the oracle leaves without any
visible key, and padding rows, must be exactly out = 0, lse = -inf.
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import verify_attn_ref
from test_gpu_parity import _custom, compare, dev, nan_outputs, note, run_gpu, to_dev

pytestmark = pytest.mark.gpu


def mask_dev(words):
    return torch.from_numpy(np.ascontiguousarray(words, np.uint64).view(np.int64)).to(dev())


def run_gpu_tree(inp, dtype, words, grid_blocks=0):
    out0, lse0 = nan_outputs(*inp["q"].shape)
    out, lse = pkg.verify_attn_tree(to_dev(inp["q"], dtype), to_dev(inp["k_cache"], dtype),
                                    to_dev(inp["v_cache"], dtype),
                                    torch.from_numpy(np.asarray(inp["ctx_lens"], np.int32)).to(dev()),
                                    torch.from_numpy(np.asarray(inp["chunk_lens"], np.int32)).to(dev()),
                                    mask_dev(words), inp["scale"], out=out0, lse=lse0, grid_blocks=grid_blocks,
                                    check_lengths=True)
    torch.cuda.synchronize()
    return out.cpu().double().numpy(), lse.cpu().double().numpy()


def check_tree(inp, dtype, words, label, grid_blocks=0):
    note(f"case {label} grid_blocks={grid_blocks}")
    o, s = run_gpu_tree(inp, dtype, words, grid_blocks)
    ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"],
                                   inp["chunk_lens"], inp["scale"], dtype, draft_mask=words)
    compare(o, s, ref_o, ref_l, dtype, label)
    return o, s


def test_tree_workload_reduced_batch():
    """Every row of a few sequences of the tree-draft workload."""
    w = dataclasses.replace(wl.get("mixtral_tree_b64"), B=6)
    inp = wl.make_inputs(w)
    for P in (0, 1, 5, 64, 300, 2048):
        check_tree(inp, w.dtype, inp["draft_mask"], f"{w.name}[B=6]", grid_blocks=P)


@pytest.mark.parametrize("name", ["ragged_chunk_b128", "mixtral_b64", "tiny_fp32"])
def test_chain_words_reproduce_chain_entry_point(name):
    """Chain words (token i sees tokens 0..i) through the tree entry point give
    the chain entry point's results bit for bit, and match the oracle."""
    w = dataclasses.replace(wl.get(name), B=min(8, wl.get(name).B))
    inp = wl.make_inputs(w)
    words = np.zeros((w.B, w.C_max), np.uint64)
    for b, n in enumerate(inp["chunk_lens"]):
        for i in range(int(n)):
            words[b, i] = (1 << (i + 1)) - 1
    for P in (0, 3):
        o_t, s_t = check_tree(inp, w.dtype, words, f"{name} chain words", grid_blocks=P)
        o_c, s_c = run_gpu(inp, w.dtype, grid_blocks=P)
        assert np.array_equal(o_t, o_c) and np.array_equal(s_t, s_c)


TREE_EDGE = {
    # name: (B, Hq, Hkv, D, dtype, ctx, chunk, C_max, mask kind)
    "random_trees_ragged_g7": (5, 28, 4, 128, "bf16", [700, 33, 1500, 2, 260], [10, 1, 16, 13, 7], 16, "tree"),
    # 64 draft tokens, one row block per KV head group of 1 (MHA), draft
    # region across a tile boundary
    "max_width_64_mha": (3, 4, 4, 128, "bf16", [100, 0, 191], [64, 64, 40], 64, "tree"),
    # f32, D = 128: 64-key tiles, so a 64-token draft fills a whole tile and
    # a unit cut at that tile has a piece made of draft keys only; every
    # third word is empty, so such a piece holds rows that see no key in it
    "f32_d128_draft_fills_tile": (3, 2, 1, 128, "f32", [64, 0, 128], [64, 64, 64], 64, "holes"),
    "bf16_d64_random": (3, 16, 4, 64, "bf16", [500, 0, 1], [5, 3, 5], 5, "random"),
    "f16_random_trees_g7": (5, 28, 4, 128, "f16", [700, 33, 1500, 2, 260], [10, 1, 16, 13, 7], 16, "tree"),
    "f32_d64_random_junk": (3, 12, 3, 64, "f32", [1000, 0, 640], [3, 8, 1], 8, "random_junk"),
    # no context and sparse masks: rows that see no key at all
    "empty_rows_no_context": (4, 8, 2, 128, "bf16", [0, 0, 0, 5], [6, 2, 9, 4], 9, "sparse"),
    "all_ones_bidirectional": (3, 8, 2, 128, "bf16", [300, 0, 129], [9, 5, 2], 9, "ones"),
}


def _edge_words(kind, chunk, C_max, rng):
    if kind == "tree":
        return wl.tree_draft_masks(11, chunk, C_max)
    if kind == "random":
        return wl.random_draft_masks(rng, chunk, C_max, density=0.5, self_bit=False)
    if kind == "random_junk":
        return wl.random_draft_masks(rng, chunk, C_max, density=0.5, self_bit=True, junk_high_bits=True)
    if kind == "sparse":
        return wl.random_draft_masks(rng, chunk, C_max, density=0.15, self_bit=False)
    if kind == "holes":
        words = wl.random_draft_masks(rng, chunk, C_max, density=0.5, self_bit=False)
        words[:, 1::3] = 0
        return words
    if kind == "ones":
        return wl.random_draft_masks(rng, chunk, C_max, density=1.0, junk_high_bits=True)
    raise ValueError(kind)


@pytest.mark.parametrize("name", sorted(TREE_EDGE))
def test_tree_edge_case(name):
    B, Hq, Hkv, D, dtype, ctx, chunk, C_max, kind = TREE_EDGE[name]
    inp = _custom(B, Hq, Hkv, D, dtype, ctx, chunk, C_max)
    words = _edge_words(kind, chunk, C_max, np.random.default_rng(len(name)))
    if kind in ("sparse", "holes"):
        ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"],
                                       inp["chunk_lens"], inp["scale"], dtype, draft_mask=words)
        valid_rows = np.arange(C_max)[None, :] < np.asarray(chunk)[:, None]
        assert np.any(np.isinf(ref_l[valid_rows])), "the case must hold rows without any visible key"
    for P in (0, 1, 2, 7, 33):
        check_tree(inp, dtype, words, name, grid_blocks=P)


def test_tree_mask_leak_is_visible():
    """Draft keys get scores far above the context's and one-hot V rows: a row
    that attended to a draft key outside its root path would move an output
    by O(1)."""
    B, Hq, Hkv, D, C = 2, 8, 2, 128, 12
    inp = _custom(B, Hq, Hkv, D, "bf16", [200, 333], [12, 9], C)
    words = wl.tree_draft_masks(3, inp["chunk_lens"], C)
    k = inp["k_cache"].view(np.uint16)
    qv = (inp["q"].astype(np.uint32) << 16).view(np.float32)
    for b in range(B):
        l, n = int(inp["ctx_lens"][b]), int(inp["chunk_lens"][b])
        for h in range(Hkv):
            direction = qv[b, :n, h * 4:(h + 1) * 4].reshape(-1, D).mean(axis=0)
            for j in range(n):
                k[b, h, l + j] = wl.f32_to_bf16_bits((direction * (8.0 + 2.0 * j)).astype(np.float32))
    v = inp["v_cache"]
    for b in range(B):
        l, n = int(inp["ctx_lens"][b]), int(inp["chunk_lens"][b])
        for j in range(n):
            row = np.zeros(D, np.float32)
            row[j] = 1.0
            v[b, :, l + j] = wl.f32_to_bf16_bits(row)
    for P in (0, 2):
        check_tree(inp, "bf16", words, "tree_mask_leak_structured", grid_blocks=P)


def test_tree_workspace_shared_with_chain_calls():
    """Chain and tree calls alternate on one workspace; each leaves its
    counters at zero for the next."""
    d = dev()
    w = dataclasses.replace(wl.get("ragged_chunk_b128"), B=6)
    q0 = torch.empty((w.B, w.C_max, w.Hq, w.D), dtype=torch.bfloat16)
    k0 = torch.empty((w.B, w.Hkv, w.S_max, w.D), dtype=torch.bfloat16)
    ws = pkg.alloc_workspace(pkg.desc_for(q0, k0, grid_blocks=64), d)
    rng = np.random.default_rng(9)
    for trial in range(4):
        ctx = rng.integers(0, 3000, w.B).astype(np.int32)
        chunk = rng.integers(0, w.C_max + 1, w.B).astype(np.int32)
        inp = wl.make_inputs(w, ctx_lens=ctx, chunk_lens=chunk)
        words = wl.tree_draft_masks(20 + trial, chunk, w.C_max) if trial % 2 else None
        note(f"case shared workspace trial {trial} ({'tree' if words is not None else 'chain'})")
        out, lse = nan_outputs(w.B, w.C_max, w.Hq, w.D)
        args = (to_dev(inp["q"], "bf16"), to_dev(inp["k_cache"], "bf16"), to_dev(inp["v_cache"], "bf16"),
                torch.from_numpy(ctx).to(d), torch.from_numpy(chunk).to(d))
        if words is None:
            pkg.verify_attn(*args, w.scale, out=out, lse=lse, workspace=ws, grid_blocks=64)
        else:
            pkg.verify_attn_tree(*args, mask_dev(words), w.scale, out=out, lse=lse, workspace=ws, grid_blocks=64)
        torch.cuda.synchronize()
        ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], ctx, chunk, w.scale, "bf16",
                                       draft_mask=words)
        compare(out.cpu().double().numpy(), lse.cpu().double().numpy(), ref_o, ref_l, "bf16",
                f"shared workspace {trial}")
    counters = ws[: 1024 * w.Hkv * 4].view(torch.int32).cpu()
    assert int(counters.abs().sum()) == 0


def test_tree_rejects_wide_masks_and_bad_mask_tensors():
    d = dev()
    q = torch.zeros((1, 65, 1, 128), dtype=torch.bfloat16, device=d)
    k = torch.zeros((1, 1, 256, 128), dtype=torch.bfloat16, device=d)
    lens = torch.ones(1, dtype=torch.int32, device=d)
    with pytest.raises(pkg.SpecMoEError) as e:
        pkg.verify_attn_tree(q, k, k, lens, lens, torch.zeros((1, 65), dtype=torch.int64, device=d), 0.1)
    assert e.value.status == -13
    with pytest.raises(TypeError):
        pkg.verify_attn_tree(q[:, :64], k, k, lens, lens, torch.zeros((1, 64), dtype=torch.int32, device=d), 0.1)
