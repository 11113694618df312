"""Seeded random configurations through every attention entry point against
the oracle: element type, head dim, GQA group, batch, lengths, draft kind
(chain, tree, paged), page size and grid are drawn per case, so that the
combinations no hand-written case covers are exercised too."""
import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import verify_attn_ref
from test_gpu_parity import _custom, compare, dev, nan_outputs, note, to_dev

pytestmark = pytest.mark.gpu


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev())


def draw_case(seed):
    rng = np.random.default_rng(1000 + seed)
    dtype = ["bf16", "f16", "f32"][rng.integers(3)]
    D = [64, 128][rng.integers(2)]
    Hkv = [1, 2, 4][rng.integers(3)]
    g = [1, 2, 4, 7, 8][rng.integers(5)]
    C_max = int(rng.integers(1, min(64, 128 // g) + 1))
    B = int(rng.integers(1, 41))
    ctx = rng.integers(0, 3001, B).astype(np.int32)
    ctx[rng.random(B) < 0.15] = 0
    chunk = rng.integers(0, C_max + 1, B).astype(np.int32)
    mode = ["chain", "tree", "paged"][rng.integers(3)]
    page = [8, 16, 64, 256][rng.integers(4)]
    grid = [0, 1, 3, 17, 256, 700][rng.integers(6)]
    return dict(dtype=dtype, D=D, Hkv=Hkv, g=g, C_max=C_max, B=B, ctx=ctx, chunk=chunk, mode=mode, page=page,
                grid=grid, rng=rng)


@pytest.mark.parametrize("seed", range(24))
def test_random_configuration(seed):
    c = draw_case(seed)
    B, dtype, mode = c["B"], c["dtype"], c["mode"]
    label = (f"random {seed}: {dtype} D={c['D']} Hkv={c['Hkv']} g={c['g']} B={B} C_max={c['C_max']} "
             f"{mode} page={c['page']} grid={c['grid']}")
    note(f"case {label}")
    inp = _custom(B, c["Hkv"] * c["g"], c["Hkv"], c["D"], dtype, c["ctx"], c["chunk"], c["C_max"], seed=200 + seed)
    words = wl.random_draft_masks(c["rng"], c["chunk"], c["C_max"], density=0.5) if mode == "tree" else None
    q = to_dev(inp["q"], dtype)
    out, lse = nan_outputs(*inp["q"].shape)
    args = dict(out=out, lse=lse, grid_blocks=c["grid"], check_lengths=True)
    if mode == "chain":
        pkg.verify_attn(q, to_dev(inp["k_cache"], dtype), to_dev(inp["v_cache"], dtype), i32(c["ctx"]),
                        i32(c["chunk"]), inp["scale"], **args)
    elif mode == "tree":
        pkg.verify_attn_tree(q, to_dev(inp["k_cache"], dtype), to_dev(inp["v_cache"], dtype), i32(c["ctx"]),
                             i32(c["chunk"]), torch.from_numpy(words.view(np.int64)).to(dev()), inp["scale"],
                             **args)
    else:
        fv = np.float32(np.nan) if dtype == "f32" else (wl.BF16_NAN if dtype == "bf16" else wl.F16_NAN)
        kp, table = wl.paginate(inp["k_cache"], c["page"], seed, fv)
        vp, _ = wl.paginate(inp["v_cache"], c["page"], seed, fv)
        pkg.verify_attn_paged(q, to_dev(kp, dtype), to_dev(vp, dtype), i32(table), i32(c["ctx"]), i32(c["chunk"]),
                              inp["scale"], **args)
    torch.cuda.synchronize()
    ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], c["ctx"], c["chunk"], inp["scale"],
                                   dtype, draft_mask=words)
    o, s = out.cpu().double().numpy(), lse.cpu().double().numpy()
    if not np.isfinite(ref_l).any():
        assert np.all(o == 0.0) and np.all(s == -np.inf)
        return
    compare(o, s, ref_o, ref_l, dtype, label)
