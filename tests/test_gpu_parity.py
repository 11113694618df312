"""GPU parity: the HIP path through the C-ABI against the fp64 CPU oracle.

Tolerances (written here, applied to every valid row):
  * f32 inputs:  max |out - ref| <= 1e-4 and max |lse - ref| <= 1e-4
  * bf16 inputs: max |out - ref| <= 1e-2 and max |lse - ref| <= 1e-3
Padding rows (i >= c_b) must be exactly out = 0, lse = -inf.  Unused cache
rows and query rows are NaN-poisoned, so any read of them shows up as NaN.
"""
import ctypes
import dataclasses
import sys

import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import verify_attn_ref

pytestmark = pytest.mark.gpu

TOL = {"f32": (1e-4, 1e-4), "bf16": (1e-2, 1e-3), "f16": (1e-2, 1e-3)}
TORCH16 = {"bf16": torch.bfloat16, "f16": torch.float16}


def dev():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a GPU")
    return torch.device("cuda:0")


def to_dev(a, dtype):
    if dtype in TORCH16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(TORCH16[dtype]).to(dev())
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev())


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def nan_outputs(B, C_max, Hq, D):
    """Output buffers pre-filled with NaN, so that a row the kernel fails to
    write cannot pass for a result."""
    return (torch.full((B, C_max, Hq, D), float("nan"), device=dev()),
            torch.full((B, C_max, Hq), float("nan"), device=dev()))


def run_gpu(inp, dtype, grid_blocks=0):
    out0, lse0 = nan_outputs(*inp["q"].shape)
    out, lse = pkg.verify_attn(to_dev(inp["q"], dtype), to_dev(inp["k_cache"], dtype),
                               to_dev(inp["v_cache"], dtype),
                               torch.from_numpy(np.asarray(inp["ctx_lens"], np.int32)).to(dev()),
                               torch.from_numpy(np.asarray(inp["chunk_lens"], np.int32)).to(dev()),
                               inp["scale"], out=out0, lse=lse0, grid_blocks=grid_blocks, check_lengths=True)
    torch.cuda.synchronize()
    return out.cpu().double().numpy(), lse.cpu().double().numpy()


def compare(o, s, ref_o, ref_l, dtype, label, units=None):
    tol_o, tol_l = TOL[dtype]
    computed = ~np.isnan(ref_l)                 # rows of units the oracle computed
    valid = computed & np.isfinite(ref_l)
    pad = computed & ~np.isfinite(ref_l)
    assert valid.any()
    err_o = np.abs(o[valid] - ref_o[valid])
    err_l = np.abs(s[valid] - ref_l[valid])
    rms = np.sqrt(np.mean(ref_o[valid] ** 2))
    note(f"[{label}] rows={int(valid.sum())} max|dout|={err_o.max():.3e} "
         f"(rel RMS {err_o.max() / rms:.3e}) max|dlse|={err_l.max():.3e} pad_rows={int(pad.sum())}")
    assert np.all(np.isfinite(o[valid])), "non-finite output in a valid row"
    assert err_o.max() <= tol_o, f"{label}: out error {err_o.max():.3e} > {tol_o}"
    assert err_l.max() <= tol_l, f"{label}: lse error {err_l.max():.3e} > {tol_l}"
    assert np.all(o[pad] == 0.0), f"{label}: padding rows of out are not zero"
    assert np.all(s[pad] == -np.inf), f"{label}: padding rows of lse are not -inf"


def check_case(inp, dtype, label, grid_blocks=0):
    note(f"case {label} grid_blocks={grid_blocks}")
    o, s = run_gpu(inp, dtype, grid_blocks)
    ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"],
                                   inp["chunk_lens"], inp["scale"], dtype)
    compare(o, s, ref_o, ref_l, dtype, label)
    return o, s


# ------------------------------------------------------------- workloads

def test_tiny_fp32_full():
    w = wl.get("tiny_fp32")
    inp = wl.make_inputs(w)
    for P in (0, 1, 3):
        check_case(inp, w.dtype, w.name, grid_blocks=P)


@pytest.mark.parametrize("name", ["mixtral_b64", "large_batch_b256", "long_ctx_b32", "ragged_chunk_b128",
                                  "eagle_draft_b64", "mixtral_f16_b64"])
def test_workload_reduced_batch(name):
    """Every row of a few sequences drawn from each workload's distribution."""
    w = wl.get(name)
    nb = 3 if name == "long_ctx_b32" else 6
    w = dataclasses.replace(w, B=nb)
    inp = wl.make_inputs(w)
    for P in (0, 1, 5, 64, 300, 2048):
        check_case(inp, w.dtype, f"{name}[B={nb}]", grid_blocks=P)


# ------------------------------------------------------------- edge cases

def _custom(B, Hq, Hkv, D, dtype, ctx, chunk, C_max, seed=5):
    """Seeded inputs with the given lengths; capacity S_max = max(ctx) + C_max
    rounded up to 256, NaN beyond each sequence's valid rows."""
    ctx = np.asarray(ctx, np.int32)
    chunk = np.asarray(chunk, np.int32)
    w = wl.Workload("edge", seed, B=B, Hq=Hq, Hkv=Hkv, D=D, dtype=dtype, ctx=("fixed", list(ctx)),
                    chunk=("uniform", 0, C_max), description="edge case")
    return wl.make_inputs(w, ctx_lens=ctx, chunk_lens=chunk)


EDGE = {
    # name: (B, Hq, Hkv, D, dtype, ctx, chunk, C_max)
    "zero_chunk_and_zero_ctx": (4, 8, 2, 128, "bf16", [0, 300, 0, 17], [3, 0, 1, 4], 4),
    "single_key": (2, 4, 4, 128, "bf16", [0, 0], [1, 1], 1),
    "tile_boundaries": (6, 8, 2, 128, "bf16", [123, 127, 128, 129, 255, 507], [5, 1, 2, 5, 1, 5], 5),
    "three_row_tiles": (4, 28, 4, 128, "bf16", [700, 33, 1500, 2], [10, 12, 13, 16], 16),
    "max_rows_128": (2, 32, 4, 128, "bf16", [900, 64], [16, 16], 16),
    # 3 and 4 row blocks per unit: one wave per block, no key split
    "rows_three_four_blocks": (4, 32, 4, 128, "bf16", [300, 1000, 77, 129], [5, 8, 6, 7], 8),
    "f32_d64_three_blocks": (2, 16, 2, 64, "f32", [200, 150], [5, 6], 6),
    "mha_g1": (3, 8, 8, 128, "bf16", [400, 10, 1000], [4, 2, 3], 4),
    "bf16_d64": (3, 16, 4, 64, "bf16", [500, 260, 1], [5, 3, 5], 5),
    # f16 (the paper's KV precision): both head dims, ragged, three row blocks
    "f16_d64": (3, 16, 4, 64, "f16", [500, 260, 1], [5, 3, 5], 5),
    "f16_three_row_tiles": (4, 28, 4, 128, "f16", [700, 33, 1500, 2], [10, 12, 13, 16], 16),
    "f16_tile_boundaries": (6, 8, 2, 128, "f16", [123, 127, 128, 129, 255, 507], [5, 1, 2, 5, 1, 5], 5),
    "f32_d128": (2, 8, 2, 128, "f32", [300, 77], [4, 2], 4),
    "f32_d64_many": (3, 12, 3, 64, "f32", [1000, 5, 640], [3, 8, 1], 8),
    # chunks longer than a key tile (f32, D=128: 64-key tiles): some tiles
    # (and pieces) hold no key that an early row of the chunk may see
    "f32_chunk_longer_than_tile": (2, 4, 4, 128, "f32", [100, 5], [100, 70], 100),
    # bf16, D=128: a 128-key chunk fills a whole tile
    "bf16_chunk_fills_tile": (2, 2, 2, 128, "bf16", [50, 300], [128, 100], 128),
}


@pytest.mark.parametrize("name", sorted(EDGE))
def test_edge_case(name):
    B, Hq, Hkv, D, dtype, ctx, chunk, C_max = EDGE[name]
    inp = _custom(B, Hq, Hkv, D, dtype, ctx, chunk, C_max)
    for P in (0, 1, 2, 7, 33):
        check_case(inp, dtype, name, grid_blocks=P)


def test_mask_leak_is_visible():
    """Draft keys get scores far above the context's: a row that saw a key
    beyond its own position would be dominated by it."""
    B, Hq, Hkv, D, C = 2, 8, 2, 128, 5
    inp = _custom(B, Hq, Hkv, D, "bf16", [200, 333], [5, 4], C)
    k = inp["k_cache"].view(np.uint16)
    qv = (inp["q"].astype(np.uint32) << 16).view(np.float32)
    for b in range(B):
        l, n = int(inp["ctx_lens"][b]), int(inp["chunk_lens"][b])
        for h in range(Hkv):
            # draft key j aligned with every query of the sequence, scaled up
            direction = qv[b, :n, h * 4:(h + 1) * 4].reshape(-1, D).mean(axis=0)
            for j in range(n):
                k[b, h, l + j] = wl.f32_to_bf16_bits((direction * (8.0 + 4.0 * j)).astype(np.float32))
    # one-hot V rows for the draft keys expose the weights directly
    v = inp["v_cache"]
    for b in range(B):
        l, n = int(inp["ctx_lens"][b]), int(inp["chunk_lens"][b])
        for j in range(n):
            row = np.zeros(D, np.float32)
            row[j] = 1.0
            v[b, :, l + j] = wl.f32_to_bf16_bits(row)
    check_case(inp, "bf16", "mask_leak_structured")


def test_repeat_is_bitwise_deterministic():
    """The split of units into pieces depends only on the lengths and the
    grid, and pieces merge in a fixed order: repeated calls agree bit for bit."""
    w = dataclasses.replace(wl.get("ragged_chunk_b128"), B=16)
    inp = wl.make_inputs(w)
    ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"],
                                   inp["chunk_lens"], inp["scale"], w.dtype)
    for P in (0, 37):
        o1, s1 = run_gpu(inp, w.dtype, grid_blocks=P)
        compare(o1, s1, ref_o, ref_l, w.dtype, f"repeat grid {P}")
        for _ in range(3):
            o2, s2 = run_gpu(inp, w.dtype, grid_blocks=P)
            assert np.array_equal(o1, o2) and np.array_equal(s1, s2)


def test_lengths_outside_preconditions_stay_in_bounds():
    """Lengths that break the documented preconditions are clamped by the
    kernels: the call completes and padding/valid rows stay well formed."""
    B, Hq, Hkv, D, C = 3, 8, 2, 128, 4
    d = dev()
    ctx = torch.tensor([-5, 10 ** 6, 10], dtype=torch.int32, device=d)
    chunk = torch.tensor([2, 2, 99], dtype=torch.int32, device=d)
    # the whole cache holds finite values here, so clamped reads stay finite
    k = torch.randn((B, Hkv, 64, D), device=d).to(torch.bfloat16)
    v = torch.randn((B, Hkv, 64, D), device=d).to(torch.bfloat16)
    q = torch.randn((B, C, Hq, D), device=d).to(torch.bfloat16)
    out, lse = pkg.verify_attn(q, k, v, ctx, chunk, 0.088)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    assert torch.isfinite(lse[:, :2]).all()


def test_empty_batch():
    d = dev()
    q = torch.empty((0, 4, 8, 128), dtype=torch.bfloat16, device=d)
    k = torch.empty((0, 2, 64, 128), dtype=torch.bfloat16, device=d)
    e = torch.empty((0,), dtype=torch.int32, device=d)
    out, lse = pkg.verify_attn(q, k, k, e, e, 0.1)
    assert out.shape == (0, 4, 8, 128) and lse.shape == (0, 4, 8)


def test_workspace_reuse_across_calls():
    """One workspace serves many calls with different lengths and grids:
    every call leaves the counters at zero for the next.  Midway a fresh
    workspace on the same (recycled) memory is initialised and used."""
    d = dev()
    w = dataclasses.replace(wl.get("ragged_chunk_b128"), B=8)
    q0 = torch.empty((w.B, w.C_max, w.Hq, w.D), dtype=torch.bfloat16)
    k0 = torch.empty((w.B, w.Hkv, w.S_max, w.D), dtype=torch.bfloat16)
    desc = pkg.desc_for(q0, k0, grid_blocks=64)
    rng = np.random.default_rng(3)
    plan = [64, 13, 64, 1, 40, 64, 7, 64]
    ws = pkg.alloc_workspace(desc, d)
    for trial, P in enumerate(plan):
        if trial == 5:
            # drop the workspace and take a new one, on recycled memory
            del ws
            ws = pkg.alloc_workspace(desc, d)
        ctx = rng.integers(0, 3000, w.B).astype(np.int32)
        chunk = rng.integers(0, w.C_max + 1, w.B).astype(np.int32)
        inp = wl.make_inputs(w, ctx_lens=ctx, chunk_lens=chunk)
        note(f"case workspace reuse trial {trial} grid_blocks={P}")
        out, lse = nan_outputs(w.B, w.C_max, w.Hq, w.D)
        pkg.verify_attn(to_dev(inp["q"], "bf16"), to_dev(inp["k_cache"], "bf16"),
                        to_dev(inp["v_cache"], "bf16"), torch.from_numpy(ctx).to(d),
                        torch.from_numpy(chunk).to(d), w.scale, out=out, lse=lse, workspace=ws,
                        grid_blocks=P)
        torch.cuda.synchronize()
        ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], ctx, chunk, w.scale, "bf16")
        compare(out.cpu().double().numpy(), lse.cpu().double().numpy(), ref_o, ref_l, "bf16",
                f"workspace reuse {trial}")
    # the per-unit counters at the start of the workspace are back to zero
    counters = ws[: 1024 * w.Hkv * 4].view(torch.int32).cpu()
    assert int(counters.abs().sum()) == 0


def test_handoff_give_up_is_reported():
    """A call whose in-kernel waits are told to give up at once (the
    diagnostic flag; every kernel still ends normally and stays in bounds)
    leaves the sticky give-up bit in its workspace; the status query reports
    it until the workspace is initialised again, after which a normal call is
    correct and reports nothing."""
    d = dev()
    w = dataclasses.replace(wl.get("mixtral_b64"), B=8)
    inp = wl.make_inputs(w)
    args = (to_dev(inp["q"], "bf16"), to_dev(inp["k_cache"], "bf16"), to_dev(inp["v_cache"], "bf16"),
            torch.from_numpy(inp["ctx_lens"]).to(d), torch.from_numpy(inp["chunk_lens"]).to(d), w.scale)
    desc = pkg.desc_for(args[0], args[1], grid_blocks=16)
    ws = pkg.alloc_workspace(desc, d)
    assert pkg.workspace_status(ws) == 0
    note("case give-up forced from the host (flags = SPECMOE_FLAG_NO_WAIT), grid 16")
    pkg.verify_attn(*args, workspace=ws, grid_blocks=16, flags=pkg.binding.SPECMOE_FLAG_NO_WAIT)
    torch.cuda.synchronize()
    assert pkg.workspace_status(ws) == -15
    assert pkg.workspace_status(ws) == -15          # sticky
    # a give-up may also leave arrival counters set (a merge whose barrier
    # gave up is skipped): re-initialising clears the status word and them
    st = pkg.load_library().specmoe_verify_attn_workspace_init(
        ws.data_ptr(), ws.numel(), torch.cuda.current_stream(d).cuda_stream, ctypes.byref(desc))
    assert st == 0
    assert pkg.workspace_status(ws) == 0
    counters = ws[256: 256 + 1024 * w.Hkv * 4].view(torch.int32).cpu()
    assert int(counters.abs().sum()) == 0
    out, lse = nan_outputs(w.B, w.C_max, w.Hq, w.D)
    pkg.verify_attn(*args, out=out, lse=lse, workspace=ws, grid_blocks=16)
    torch.cuda.synchronize()
    assert pkg.workspace_status(ws) == 0
    ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"], inp["chunk_lens"],
                                   w.scale, "bf16")
    compare(out.cpu().double().numpy(), lse.cpu().double().numpy(), ref_o, ref_l, "bf16", "after a give-up")


def test_side_stream_without_workspace():
    """A call on a non-current stream without a workspace: the binding takes
    the workspace (and outputs) from that stream's pool, so allocations on
    the current stream right after the call cannot reuse the workspace while
    the kernel still runs."""
    d = dev()
    w = dataclasses.replace(wl.get("ragged_chunk_b128"), B=24)
    inp = wl.make_inputs(w)
    args = (to_dev(inp["q"], "bf16"), to_dev(inp["k_cache"], "bf16"), to_dev(inp["v_cache"], "bf16"),
            torch.from_numpy(inp["ctx_lens"]).to(d), torch.from_numpy(inp["chunk_lens"]).to(d), w.scale)
    ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"], inp["chunk_lens"],
                                   w.scale, "bf16")
    side = torch.cuda.Stream(device=d)
    side.wait_stream(torch.cuda.current_stream(d))
    for trial in range(3):
        note(f"case side stream, no workspace, trial {trial}")
        out, lse = pkg.verify_attn(*args, grid_blocks=64, stream=side)
        # the current stream allocates and fills buffers meanwhile
        junk = [torch.full((1 << 20,), 7, dtype=torch.int32, device=d) for _ in range(8)]
        del junk
        torch.cuda.synchronize()
        compare(out.cpu().double().numpy(), lse.cpu().double().numpy(), ref_o, ref_l, "bf16",
                f"side stream {trial}")
