"""GPU parity of the paged-KV entry point against the fp64 CPU oracle, which
gathers the pages into the contiguous cache and applies the same definition.
Tolerances as for the contiguous cache (f32 1e-4; bf16 and f16 1e-2 on out,
1e-3 on lse)."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import gather_pages, verify_attn_ref
from test_gpu_parity import _custom, compare, dev, nan_outputs, note, to_dev

pytestmark = pytest.mark.gpu


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev())


def check_paged(inp, dtype, page_size, label, grid_blocks=0, words=None, seed=3):
    fv = np.float32(np.nan) if dtype == "f32" else (wl.BF16_NAN if dtype == "bf16" else wl.F16_NAN)
    kp, table = wl.paginate(inp["k_cache"], page_size, seed, fv)
    vp, _ = wl.paginate(inp["v_cache"], page_size, seed, fv)
    note(f"case {label} page_size={page_size} grid_blocks={grid_blocks}")
    out, lse = nan_outputs(*inp["q"].shape)
    mask = None if words is None else torch.from_numpy(words.view(np.int64)).to(dev())
    pkg.verify_attn_paged(to_dev(inp["q"], dtype), to_dev(kp, dtype), to_dev(vp, dtype), i32(table),
                          i32(inp["ctx_lens"]), i32(inp["chunk_lens"]), inp["scale"], draft_mask=mask, out=out,
                          lse=lse, grid_blocks=grid_blocks, check_lengths=True)
    torch.cuda.synchronize()
    ref_o, ref_l = verify_attn_ref(inp["q"], gather_pages(kp, table, page_size), gather_pages(vp, table, page_size),
                                   inp["ctx_lens"], inp["chunk_lens"], inp["scale"], dtype, draft_mask=words)
    compare(out.cpu().double().numpy(), lse.cpu().double().numpy(), ref_o, ref_l, dtype, label)


def test_paged_workload_reduced_batch():
    w = dataclasses.replace(wl.get("mixtral_paged_b64"), B=6)
    inp = wl.make_inputs(w)
    for ps in (8, 16, 64, 128, 256):
        for P in (0, 5, 64):
            check_paged(inp, w.dtype, ps, f"{w.name}[B=6]", grid_blocks=P)


PAGED_EDGE = {
    # name: (B, Hq, Hkv, D, dtype, ctx, chunk, C_max, page sizes)
    "bf16_d64_256_key_tiles": (3, 16, 4, 64, "bf16", [500, 260, 1], [5, 3, 5], 5, (8, 32, 256)),
    "f32_d128_64_key_tiles": (2, 8, 2, 128, "f32", [300, 77], [4, 2], 4, (8, 64, 128)),
    "f32_d64": (3, 12, 3, 64, "f32", [1000, 5, 640], [3, 8, 1], 8, (8, 16)),
    "f16_tile_boundaries": (6, 8, 2, 128, "f16", [123, 127, 128, 129, 255, 507], [5, 1, 2, 5, 1, 5], 5, (8, 128)),
    "zero_chunk_and_zero_ctx": (4, 8, 2, 128, "bf16", [0, 300, 0, 17], [3, 0, 1, 4], 4, (8, 16)),
    "three_row_tiles_g7": (4, 28, 4, 128, "bf16", [700, 33, 1500, 2], [10, 12, 13, 16], 16, (16, 256)),
}


@pytest.mark.parametrize("name", sorted(PAGED_EDGE))
def test_paged_edge_case(name):
    B, Hq, Hkv, D, dtype, ctx, chunk, C_max, sizes = PAGED_EDGE[name]
    inp = _custom(B, Hq, Hkv, D, dtype, ctx, chunk, C_max)
    for ps in sizes:
        for P in (0, 2, 33):
            check_paged(inp, dtype, ps, name, grid_blocks=P)


def test_paged_tree_drafts():
    w = dataclasses.replace(wl.get("mixtral_tree_b64"), B=5)
    inp = wl.make_inputs(w)
    for ps in (8, 64):
        check_paged(inp, w.dtype, ps, "paged tree drafts", words=inp["draft_mask"])


def test_paged_table_entries_out_of_range_are_clamped():
    """Table entries outside the pool are clamped into it: the call completes
    and, with a finite pool, every valid row is finite."""
    d = dev()
    B, C, Hq, Hkv, D, ps, P = 3, 4, 8, 2, 128, 16, 8
    q = torch.randn((B, C, Hq, D), device=d).to(torch.bfloat16)
    kp = torch.randn((10, Hkv, ps, D), device=d).to(torch.bfloat16)
    vp = torch.randn((10, Hkv, ps, D), device=d).to(torch.bfloat16)
    table = torch.tensor([[0, 1, -5, 99, 3, 4, 5, 6], [7, 8, 9, 10 ** 6, 0, 1, 2, 3], [-1] * 8],
                         dtype=torch.int32, device=d)
    ctx = torch.tensor([100, 60, 120], dtype=torch.int32, device=d)
    chunk = torch.tensor([4, 3, 4], dtype=torch.int32, device=d)
    out, lse = pkg.verify_attn_paged(q, kp, vp, table, ctx, chunk, 0.088)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    assert torch.isfinite(lse[0, :4]).all() and torch.isfinite(lse[1, :3]).all()


def test_paged_geometry_errors():
    d = dev()
    q = torch.zeros((1, 2, 4, 128), dtype=torch.bfloat16, device=d)
    kp = torch.zeros((4, 1, 16, 128), dtype=torch.bfloat16, device=d)
    lens = torch.ones(1, dtype=torch.int32, device=d)
    for ps_pages, table_cols in (((4, 1, 12, 128), 4), ((4, 1, 4, 128), 4)):   # not a power of two; below 8
        bad = torch.zeros(ps_pages, dtype=torch.bfloat16, device=d)
        with pytest.raises(pkg.SpecMoEError) as e:
            pkg.verify_attn_paged(q, bad, bad, torch.zeros((1, table_cols), dtype=torch.int32, device=d),
                                  lens, lens, 0.1)
        assert e.value.status == -14
    out, _ = pkg.verify_attn_paged(q, kp, kp, torch.zeros((1, 4), dtype=torch.int32, device=d), lens, lens, 0.1)
    torch.cuda.synchronize()
    assert torch.isfinite(out[0, 0]).all()


def test_batches_past_one_launch():
    """More than 1024 sequences run as consecutive launches on the stream; the
    lengths, draft masks and block tables of every launch are offset to its
    sequences.  Chain, tree and paged calls on one batch of 1100 short
    sequences, every row against the oracle."""
    B, C = 1100, 4
    rng = np.random.default_rng(81)
    ctx = rng.integers(0, 200, B).astype(np.int32)
    chunk = rng.integers(0, C + 1, B).astype(np.int32)
    inp = _custom(B, 8, 2, 64, "bf16", ctx, chunk, C, seed=12)
    words = wl.random_draft_masks(rng, chunk, C, density=0.6)
    note("case 1100 sequences: chain, tree, paged")
    d = dev()
    q, k, v = to_dev(inp["q"], "bf16"), to_dev(inp["k_cache"], "bf16"), to_dev(inp["v_cache"], "bf16")
    for mode in ("chain", "tree", "paged"):
        out, lse = nan_outputs(*inp["q"].shape)
        if mode == "chain":
            pkg.verify_attn(q, k, v, i32(ctx), i32(chunk), inp["scale"], out=out, lse=lse)
            ref = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], ctx, chunk, inp["scale"], "bf16")
        elif mode == "tree":
            pkg.verify_attn_tree(q, k, v, i32(ctx), i32(chunk), torch.from_numpy(words.view(np.int64)).to(d),
                                 inp["scale"], out=out, lse=lse)
            ref = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], ctx, chunk, inp["scale"], "bf16",
                                  draft_mask=words)
        else:
            kp, table = wl.paginate(inp["k_cache"], 16, 4, wl.BF16_NAN)
            vp, _ = wl.paginate(inp["v_cache"], 16, 4, wl.BF16_NAN)
            pkg.verify_attn_paged(q, to_dev(kp, "bf16"), to_dev(vp, "bf16"), i32(table), i32(ctx), i32(chunk),
                                  inp["scale"], out=out, lse=lse)
            ref = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], ctx, chunk, inp["scale"], "bf16")
        torch.cuda.synchronize()
        compare(out.cpu().double().numpy(), lse.cpu().double().numpy(), ref[0], ref[1], "bf16",
                f"1100 sequences, {mode}")
