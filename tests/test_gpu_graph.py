"""The entry points under HIP graph capture: a serving loop captures the
verification call and the acceptance call once and replays them.  The
library issues no memset and no allocation (its workspace counters are left
zero by each call), so a captured call replays correctly.  Each replay is
separated by eager work on the same buffers and compared bit for bit with
the eager result."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2508_21706_amd as pkg
from paper_2508_21706_amd import workloads as wl
from oracle import accept_greedy_ref, verify_attn_ref
from test_gpu_parity import compare, dev, note, to_dev

pytestmark = pytest.mark.gpu


def test_verify_and_accept_replay_in_a_graph():
    d = dev()
    w = dataclasses.replace(wl.get("ragged_chunk_b128"), B=12)
    inp = wl.make_inputs(w)
    q, k, v = to_dev(inp["q"], "bf16"), to_dev(inp["k_cache"], "bf16"), to_dev(inp["v_cache"], "bf16")
    ctx = torch.from_numpy(inp["ctx_lens"]).to(d)
    chunk = torch.from_numpy(inp["chunk_lens"]).to(d)
    ws = pkg.alloc_workspace(pkg.desc_for(q, k, 64), d)
    out = torch.empty((w.B, w.C_max, w.Hq, w.D), dtype=torch.float32, device=d)
    lse = torch.empty((w.B, w.C_max, w.Hq), dtype=torch.float32, device=d)

    aw = dataclasses.replace(wl.ACCEPT_BY_NAME["accept_mixtral_b64"], B=12, C_max=w.C_max, V=8192)
    ainp = wl.make_accept_inputs(aw, chunk_lens=inp["chunk_lens"], ctx_lens=inp["ctx_lens"])
    logits = to_dev(ainp["logits"], "bf16")
    tokens = torch.from_numpy(ainp["tokens"]).to(d)
    aws = pkg.alloc_accept_workspace(pkg.accept_desc(aw.B, aw.C_max, aw.V, 1), d)
    aout = {"argmax": torch.empty((aw.B, aw.C_max), dtype=torch.int32, device=d),
            "accepted": torch.empty((aw.B,), dtype=torch.int32, device=d),
            "next_token": torch.empty((aw.B,), dtype=torch.int32, device=d),
            "new_ctx_lens": torch.empty((aw.B,), dtype=torch.int32, device=d)}

    # tree acceptance and the path compaction on a copy of the cache
    words = wl.tree_draft_masks(7, inp["chunk_lens"], w.C_max)
    mask = torch.from_numpy(words.view(np.int64)).to(d)
    tout = {"argmax": torch.empty((aw.B, aw.C_max), dtype=torch.int32, device=d),
            "accepted": torch.empty((aw.B,), dtype=torch.int32, device=d),
            "next_token": torch.empty((aw.B,), dtype=torch.int32, device=d),
            "new_ctx_lens": torch.empty((aw.B,), dtype=torch.int32, device=d),
            "path": torch.empty((aw.B,), dtype=torch.int64, device=d)}
    kc, vc = k.clone(), v.clone()

    def step(stream):
        pkg.verify_attn(q, k, v, ctx, chunk, w.scale, out=out, lse=lse, workspace=ws, grid_blocks=64,
                        stream=stream)
        pkg.accept_greedy(logits, tokens, ctx, chunk, out=aout, workspace=aws, stream=stream)
        kc.copy_(k)
        vc.copy_(v)
        pkg.accept_greedy_tree(logits, tokens, mask, ctx, chunk, out=tout, workspace=aws, stream=stream)
        pkg.compact_accepted_kv(kc, vc, ctx, tout["path"], stream=stream)

    # eager reference, checked against the oracles
    step(torch.cuda.current_stream(d))
    torch.cuda.synchronize()
    eager_o, eager_l = out.clone(), lse.clone()
    eager_a = {kk: vv.clone() for kk, vv in aout.items()}
    eager_t = {kk: vv.clone() for kk, vv in tout.items()}
    eager_kc, eager_vc = kc.clone(), vc.clone()
    ref_o, ref_l = verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"], inp["chunk_lens"],
                                   w.scale, "bf16")
    compare(eager_o.cpu().double().numpy(), eager_l.cpu().double().numpy(), ref_o, ref_l, "bf16", "graph eager")
    aref = accept_greedy_ref(ainp["logits"], ainp["tokens"], ainp["ctx_lens"], ainp["chunk_lens"], "bf16")
    for kk in aref:
        assert np.array_equal(eager_a[kk].cpu().numpy(), aref[kk]), kk

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream(d)
    side.wait_stream(torch.cuda.current_stream(d))
    with torch.cuda.stream(side):
        step(side)                       # warm up on the capture stream
    torch.cuda.current_stream(d).wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step(torch.cuda.current_stream(d))
    for rep in range(4):
        # eager work on the same buffers between replays
        out.fill_(float("nan"))
        lse.zero_()
        for t in aout.values():
            t.fill_(-9)
        step(torch.cuda.current_stream(d))
        torch.cuda.synchronize()
        out.fill_(float("nan"))
        for t in aout.values():
            t.fill_(-9)
        for t in tout.values():
            t.fill_(-9)
        kc.zero_()
        vc.zero_()
        graph.replay()
        torch.cuda.synchronize()
        note(f"graph replay {rep}")
        assert torch.equal(out, eager_o) and torch.equal(lse, eager_l), f"replay {rep}: attention differs"
        for kk, vv in aout.items():
            assert torch.equal(vv, eager_a[kk]), f"replay {rep}: {kk} differs"
        for kk, vv in tout.items():
            assert torch.equal(vv, eager_t[kk]), f"replay {rep}: tree {kk} differs"
        # bitwise (the caches hold NaN-poisoned rows past each sequence)
        assert torch.equal(kc.view(torch.int16), eager_kc.view(torch.int16)) and \
            torch.equal(vc.view(torch.int16), eager_vc.view(torch.int16)), f"replay {rep}: compaction differs"
    # the workspaces' counters are back to zero
    assert int(ws[: 1024 * w.Hkv * 4].view(torch.int32).abs().sum()) == 0
    assert int(aws[: 65536 * 4].view(torch.int32).abs().sum()) == 0
