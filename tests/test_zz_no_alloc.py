"""The allocation-free entry point (specmoe_verify_attn_noalloc) through the
C-ABI: on two calls in a row, the second with a smaller input of another
shape, its output equals the workspace entry point's bit for bit (the same
kernels, grid and schedule) and the oracle's within the bf16 tolerances
(max |dout| <= 1e-2, max |dlse| <= 1e-3)."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import verify_attn_ref
from test_gpu_parity import compare, dev, nan_outputs, note, to_dev

pytestmark = pytest.mark.gpu


def test_noalloc_matches_workspace_entry_point():
    d = dev()
    cases = [(wl.get("mixtral_b64"), 64), (wl.get("ragged_chunk_b128"), 12)]   # the second is smaller
    for w0, B in cases:
        w = dataclasses.replace(w0, B=B)
        note(f"case no-alloc entry point: {w.name} B={B}")
        inp = wl.make_inputs(w, workers=8)
        args = (to_dev(inp["q"], "bf16"), to_dev(inp["k_cache"], "bf16"), to_dev(inp["v_cache"], "bf16"),
                torch.from_numpy(inp["ctx_lens"]).to(d), torch.from_numpy(inp["chunk_lens"]).to(d), w.scale)
        out_ws, lse_ws = nan_outputs(w.B, w.C_max, w.Hq, w.D)
        pkg.verify_attn(*args, out=out_ws, lse=lse_ws)
        out_na, lse_na = nan_outputs(w.B, w.C_max, w.Hq, w.D)
        pkg.verify_attn_noalloc(*args, out=out_na, lse=lse_na)
        torch.cuda.synchronize()
        assert pkg.workspace_status(None) == 0
        assert torch.equal(out_ws, out_na) and torch.equal(lse_ws, lse_na)
        ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"], inp["chunk_lens"],
                                       w.scale, "bf16")
        compare(out_na.cpu().double().numpy(), lse_na.cpu().double().numpy(), ref_o, ref_l, "bf16",
                f"no-alloc {w.name} B={B}")


def test_noalloc_rejects_needs_beyond_the_scratch():
    d = dev()
    q = torch.zeros((2, 16, 32, 128), dtype=torch.bfloat16, device=d)    # 16 * 8 = 128 rows per KV head
    k = torch.zeros((2, 4, 256, 128), dtype=torch.bfloat16, device=d)
    lens = torch.zeros((2,), dtype=torch.int32, device=d)
    out = torch.zeros((2, 16, 32, 128), dtype=torch.float32, device=d)
    lse = torch.zeros((2, 16, 32), dtype=torch.float32, device=d)
    with pytest.raises(pkg.SpecMoEError) as e:
        pkg.verify_attn_noalloc(q, k, k, lens, lens, 0.088, out, lse, grid_blocks=2048)
    assert e.value.status == -8
