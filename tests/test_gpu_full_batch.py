"""GPU parity of whole batches at full size: every row of every sequence of
each attention workload, in the benchmark's launch configuration (default
grid, one workspace, the entry point the benchmark times), against the fp64
CPU oracle on the same seeded inputs.

Tolerances as in test_gpu_parity: f32 1e-4 on out and lse; bf16 and f16 1e-2
on out and 1e-3 on lse.  Each case logs max|dout|, max|dlse| and the largest
out error relative to the RMS of the reference output over the whole batch.
Unused cache rows and query rows hold NaN, so a read of them shows up.
"""
import os
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import gather_pages, verify_attn_ref
from test_gpu_parity import compare, dev, nan_outputs, note, to_dev

pytestmark = pytest.mark.gpu

WORKERS = min(16, len(os.sched_getaffinity(0)))


def oracle_whole_batch(inp, w, k_cache, v_cache):
    """The oracle over every (sequence, KV head) of the batch, the units
    spread over threads (each call computes its own units; the rest of its
    output stays NaN and is taken from the other calls)."""
    from threadpoolctl import threadpool_limits
    units = [(b, h) for b in range(w.B) for h in range(w.Hkv)]
    groups = [units[i::WORKERS] for i in range(WORKERS)]

    def part(us):
        return verify_attn_ref(inp["q"], k_cache, v_cache, inp["ctx_lens"], inp["chunk_lens"], w.scale, w.dtype,
                               units=us, draft_mask=inp["draft_mask"])

    with threadpool_limits(1), ThreadPoolExecutor(WORKERS) as ex:
        parts = list(ex.map(part, groups))
    out, lse = parts[0]
    for o, s in parts[1:]:
        have = ~np.isnan(s)
        out[have] = o[have]
        lse[have] = s[have]
    assert not np.isnan(lse).any(), "a unit was left out"
    return out, lse


@pytest.mark.parametrize("name", ["mixtral_b64", "large_batch_b256", "long_ctx_b32", "ragged_chunk_b128",
                                  "mixtral_tree_b64", "mixtral_f16_b64", "mixtral_paged_b64", "eagle_draft_b64"])
def test_whole_batch_full_size(name):
    w = wl.get(name)
    note(f"case {name} whole batch at full size: B={w.B} Hq={w.Hq} Hkv={w.Hkv} D={w.D} {w.dtype} "
         f"C_max={w.C_max} S_max={w.S_max} draft={w.draft} page_size={w.page_size}")
    t0 = time.time()
    inp = wl.make_inputs(w, workers=WORKERS)
    note(f"  inputs drawn in {time.time() - t0:.1f} s")
    d = dev()
    paged = w.page_size > 0
    q = to_dev(inp["q"], w.dtype)
    ctx = torch.from_numpy(inp["ctx_lens"]).to(d)
    chunk = torch.from_numpy(inp["chunk_lens"]).to(d)
    mask = None if inp["draft_mask"] is None else torch.from_numpy(inp["draft_mask"].view(np.int64)).to(d)
    out, lse = nan_outputs(w.B, w.C_max, w.Hq, w.D)
    if paged:
        kp, vp = to_dev(inp["k_pages"], w.dtype), to_dev(inp["v_pages"], w.dtype)
        table = torch.from_numpy(inp["block_table"]).to(d)
        ws = pkg.alloc_workspace(pkg.make_desc(w.B, w.Hq, w.Hkv, w.D, w.C_max, w.S_max, pkg.binding._dtype_code(q)), d)
        pkg.verify_attn_paged(q, kp, vp, table, ctx, chunk, w.scale, draft_mask=mask, out=out, lse=lse, workspace=ws)
    else:
        k, v = to_dev(inp["k_cache"], w.dtype), to_dev(inp["v_cache"], w.dtype)
        ws = pkg.alloc_workspace(pkg.desc_for(q, k), d)
        if mask is None:
            pkg.verify_attn(q, k, v, ctx, chunk, w.scale, out=out, lse=lse, workspace=ws)
        else:
            pkg.verify_attn_tree(q, k, v, ctx, chunk, mask, w.scale, out=out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    assert pkg.workspace_status(ws) == 0
    o = out.cpu().double().numpy()
    s = lse.cpu().double().numpy()
    note(f"  GPU call done; oracle over {w.B * w.Hkv} units in {WORKERS} threads")
    t0 = time.time()
    if paged:
        k_ref = gather_pages(inp["k_pages"], inp["block_table"], w.page_size)
        v_ref = gather_pages(inp["v_pages"], inp["block_table"], w.page_size)
    else:
        k_ref, v_ref = inp["k_cache"], inp["v_cache"]
    ref_o, ref_l = oracle_whole_batch(inp, w, k_ref, v_ref)
    note(f"  oracle done in {time.time() - t0:.1f} s")
    compare(o, s, ref_o, ref_l, w.dtype, f"{name} whole batch")
    del q, out, lse, ws
    torch.cuda.empty_cache()
