"""Benchmark: chunked verification attention on one MI355X.

One step = one call of the whole hot path (the single persistent kernel that
streams the KV cache and merges split units) over one batch of the synthetic
workload, with every input already resident in HBM.  Prints ONE JSON line on stdout; progress goes to stderr.

    python bench.py [--steps K] [--warmup W] [--workload mixtral_b64]

The acceptance step that follows verification has workloads of its own
(``--workload accept_mixtral_b64`` etc.): one step is one greedy-acceptance
call over the batch's logits, and value = logits GB/s.

value = effective KV GB/s = sum_b Hkv*(l_b + c_b)*D*elt*2 / t_step, the K+V
bytes of every valid row (the attention row of the paper's cost table,
2*b*s*h/g elements, Section 3.2).  Input sets are rotated so that successive
steps read different HBM addresses and the KV cannot be served from the
256 MB Infinity Cache.  Before the warmup steps, steps run for --settle-ms of
sustained load (reported as settle_steps), so that the timed steps see the
GPU at its working clock rather than its ramp.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective KV HBM GB/s and verified draft tokens/sec, Mixtral shape B=64"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 / f16 matrix-core peak of an MI355X
MAIN_KERNEL = "verify_attn_kernel"
KERNEL_SOURCE = os.path.join(ROOT, "paper_2508_21706_amd", "csrc", "verify_attn.hip")
ACCEPT_METRIC = "acceptance step: logits HBM GB/s and accepted-token decisions per second"
ACCEPT_KERNEL = "accept_kernel"
ACCEPT_SOURCE = os.path.join(ROOT, "paper_2508_21706_amd", "csrc", "accept.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def source_digest(path: str = KERNEL_SOURCE) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def load_traffic(workload: str, kernel: str = MAIN_KERNEL, source: str = KERNEL_SOURCE):
    """HBM bytes per launch of a kernel from the committed rocprofv3 counter
    summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_sha256_16") != source_digest(source):
        return None
    return rec.get("hbm_bytes_per_launch")


def run_timed(step, args, stream):
    """Settle, warm up, then time exactly args.steps steps between two
    synchronisations; returns (ms per step, settle steps)."""
    import torch
    settle_steps = 0
    torch.cuda.synchronize()
    t_settle = time.time()
    while (time.time() - t_settle) * 1e3 < args.settle_ms:
        for _ in range(20):
            step(settle_steps)
            settle_steps += 1
        torch.cuda.synchronize()
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(args.steps):
        step(i)
    t_end.record(stream)
    torch.cuda.synchronize()
    return t_start.elapsed_time(t_end) / args.steps, settle_steps


def bench_accept(args):
    """The acceptance step: one greedy-acceptance launch per step over the
    batch's logits (rotated over enough copies that they come from HBM)."""
    import torch
    import paper_2508_21706_amd as pkg
    from paper_2508_21706_amd import workloads as wl

    w = wl.ACCEPT_BY_NAME[args.workload]
    dev = torch.device("cuda:0")
    inp = wl.make_accept_inputs(w)
    chunk = inp["chunk_lens"]
    rows = int(chunk.sum())
    logit_bytes = rows * w.V * w.elt_bytes
    # algorithmic bytes per launch: the valid logits rows, the chunk tokens and
    # lengths read, and the argmax / accepted / next / new-length outputs
    launch_bytes = logit_bytes + rows * 4 + w.B * 8 + w.B * w.C_max * 4 + w.B * 12
    if w.dtype == "bf16":
        x = torch.from_numpy(inp["logits"].view(np.int16)).view(torch.bfloat16).to(dev)
    else:
        x = torch.from_numpy(inp["logits"]).to(dev)
    n_sets = args.rotate or max(4, int(np.ceil(1.0e9 / x.numel() / x.element_size())))
    sets = [x] + [x.clone() for _ in range(n_sets - 1)]
    tokens = torch.from_numpy(inp["tokens"]).to(dev)
    ctx = torch.from_numpy(inp["ctx_lens"]).to(dev)
    chunk_d = torch.from_numpy(chunk).to(dev)
    desc = pkg.accept_desc(w.B, w.C_max, w.V, pkg.binding.SPECMOE_BF16 if w.dtype == "bf16" else 0)
    ws = pkg.alloc_accept_workspace(desc, dev)
    out = {"argmax": torch.empty((w.B, w.C_max), dtype=torch.int32, device=dev),
           "accepted": torch.empty((w.B,), dtype=torch.int32, device=dev),
           "next_token": torch.empty((w.B,), dtype=torch.int32, device=dev),
           "new_ctx_lens": torch.empty((w.B,), dtype=torch.int32, device=dev)}
    stream = torch.cuda.current_stream(dev)
    log(f"{n_sets} logits sets x {logit_bytes / 1e6:.1f} MB, {w.B} sequences x chunk {w.C_max}, vocabulary {w.V}")

    mask_d = torch.from_numpy(inp["draft_mask"].view(np.int64)).to(dev) if w.tree else None
    if w.tree:
        out["path"] = torch.empty((w.B,), dtype=torch.int64, device=dev)

    def step(i):
        if w.tree:
            pkg.accept_greedy_tree(sets[i % n_sets], tokens, mask_d, ctx, chunk_d, out=out, workspace=ws,
                                   stream=stream)
        else:
            pkg.accept_greedy(sets[i % n_sets], tokens, ctx, chunk_d, out=out, workspace=ws, stream=stream)

    ms, settle_steps = run_timed(step, args, stream)
    t = ms / 1e3
    value = logit_bytes / t / 1e9
    achieved = launch_bytes / t / 1e9
    log(f"step {ms * 1e3:.2f} us -> {value:.0f} GB/s of logits, {w.B / t / 1e6:.2f} M sequence decisions/s")
    cpu = None
    if args.cpu_budget > 0:
        from oracle import accept_greedy_ref, accept_tree_ref
        log("timing the oracle on the host ...")
        passes, t_total = 0, 0.0
        while t_total < args.cpu_budget:
            t0 = time.perf_counter()
            if w.tree:
                accept_tree_ref(inp["logits"], inp["tokens"], inp["draft_mask"], inp["ctx_lens"], chunk, w.dtype)
            else:
                accept_greedy_ref(inp["logits"], inp["tokens"], inp["ctx_lens"], chunk, w.dtype)
            t_total += time.perf_counter() - t0
            passes += 1
        cpu = {"value": passes * logit_bytes / t_total / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"{passes} passes over the whole batch ({w.B} sequences, {rows} logits rows), numpy "
                         f"oracle, {t_total:.1f} s"}
    traffic = load_traffic(w.name, ACCEPT_KERNEL, ACCEPT_SOURCE)
    rec = {
        "metric": ACCEPT_METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "settle_steps": settle_steps, "ms_per_step": round(ms, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "description": w.description, "B": w.B, "C_max": w.C_max, "V": w.V,
                   "tree": w.tree,
                   "input_sets": n_sets, "parallelism": "single GPU"},
        "sequence_decisions_per_s": round(w.B / t, 1),
        "roofline": {"bound": "hbm", "kernel": ACCEPT_KERNEL, "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "traffic_unit": "HBM bytes per launch",
                     "traffic_over_algorithmic": round(traffic / launch_bytes, 4) if traffic else None,
                     "algorithmic_bytes_per_launch": launch_bytes, "avg_launch_us": round(t * 1e6, 3)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


def measure_ceiling(args, sets, kv_bytes, stream):
    """Time the streaming-read probe (libspecmoe_probe.so, built beside the
    library; not part of it) over kv_bytes per step: half from the start of
    each input set's K, half from its V, rotating over the sets as the steps
    do.  Both load forms are timed; the faster is the measured ceiling."""
    import ctypes
    import torch
    from paper_2508_21706_amd import build as _build
    if not os.path.exists(_build.PROBE_OUTPUT):
        raise RuntimeError(f"{_build.PROBE_OUTPUT} is missing: run python paper_2508_21706_amd/build.py")
    lib = ctypes.CDLL(_build.PROBE_OUTPUT)
    lib.specmoe_probe_stream.restype = ctypes.c_int
    lib.specmoe_probe_stream.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_size_t,
                                         ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    half = kv_bytes // 2 // 1024 * 1024
    for k, v in sets:
        assert half <= k.numel() * k.element_size() and half <= v.numel() * v.element_size()
    grid = 256
    sink = torch.empty(grid, dtype=torch.int32, device=sets[0][0].device)
    res = {}
    for mode, name in ((0, "direct_to_lds"), (1, "registers")):
        def step(i, mode=mode):
            k, v = sets[i % len(sets)]
            st = lib.specmoe_probe_stream(k.data_ptr(), half, v.data_ptr(), half, mode, grid, sink.data_ptr(),
                                          stream.cuda_stream)
            if st != 0:
                raise RuntimeError(f"probe launch failed ({st})")
        ms, _ = run_timed(step, args, stream)
        res[name] = {"us": round(ms * 1e3, 3), "gbs": round(2 * half / (ms / 1e3) / 1e9, 2)}
        log(f"ceiling probe ({name}): {2 * half / 1e6:.1f} MB in {ms * 1e3:.1f} us -> {res[name]['gbs']:.0f} GB/s")
    best = max(res.values(), key=lambda r: r["gbs"])
    return {"gbs": best["gbs"], "bytes": 2 * half, "grid": grid, "forms": res,
            "what": "16-byte non-temporal reads of the same byte count, one persistent workgroup per CU, "
                    "~128 KB in flight per CU (libspecmoe_probe.so)"}


def cpu_baseline(inp, w, budget_s: float):
    """The fp64 oracle, timed on the host cores over a bounded sample of the
    same workload: whole sequences, in order (wrapping around the batch),
    until ~budget_s of work."""
    from oracle import verify_attn_ref
    from paper_2508_21706_amd import workloads as wl
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    done = []
    t_total = 0.0
    while t_total < budget_s:
        b = len(done) % w.B
        units = [(b, h) for h in range(w.Hkv)]
        t0 = time.perf_counter()
        verify_attn_ref(inp["q"], inp["k_cache"], inp["v_cache"], inp["ctx_lens"], inp["chunk_lens"],
                        w.scale, w.dtype, units=units, draft_mask=inp["draft_mask"])
        t_total += time.perf_counter() - t0
        done.append(b)
    ctx = inp["ctx_lens"][done]
    chunk = inp["chunk_lens"][done]
    kv = wl.algorithmic_kv_bytes(w, ctx, chunk)
    return {
        "value": kv / t_total / 1e9,
        "unit": "GB/s",
        "cores": int(blas_threads),
        "kind": "oracle",
        "sample": f"{len(done)} sequences (all KV heads; {len(done) / w.B:.1f} passes over the {w.B} of "
                  f"{w.name}), fp64 numpy oracle, {t_total:.1f} s; {int(chunk.sum())} draft tokens -> "
                  f"{chunk.sum() / t_total:.1f} verified tokens/s",
        "host": {"os_cpu_count": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)),
                 "cpu": platform.processor() or platform.machine()},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mixtral_b64")
    ap.add_argument("--grid-blocks", type=int, default=0, help="persistent workgroups (0: library default)")
    ap.add_argument("--rotate", type=int, default=0, help="input sets (0: enough for >= 1 GB)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work; 0 skips")
    ap.add_argument("--settle-ms", type=float, default=200.0,
                    help="before the warmup steps, run steps until the GPU has been busy this long "
                         "(its clocks ramp up over the first tens of ms of sustained load); 0 skips")
    ap.add_argument("--no-ceiling", dest="ceiling", action="store_false",
                    help="skip the streaming-read probe that measures the HBM read ceiling")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MB",
                    help="instead of the benchmark, run a plain elementwise copy of MB MiB (float32 read, "
                         "float32 write) 5 times: the known byte counts calibrate the HBM traffic counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the verification-attention kernel works on one "
              "GPU's share of the batch and has no multi-GPU component; run one process per GPU "
              "on disjoint sequences instead.", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe:
        n = args.copy_probe * (1 << 20) // 4
        x = torch.ones(n, dtype=torch.float32, device="cuda:0")
        y = torch.empty_like(x)
        for _ in range(5):
            torch.neg(x, out=y)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4, "launches": 5}))
        return
    import paper_2508_21706_amd as pkg
    from paper_2508_21706_amd import workloads as wl

    if args.workload in wl.ACCEPT_BY_NAME:
        bench_accept(args)
        return
    w = wl.get(args.workload)
    dev = torch.device("cuda:0")
    t0 = time.time()
    inp = wl.make_inputs(w)
    log(f"inputs for {w.name} drawn in {time.time() - t0:.1f} s")
    ctx, chunk = inp["ctx_lens"], inp["chunk_lens"]
    kv_bytes = wl.algorithmic_kv_bytes(w, ctx, chunk)
    tokens = int(chunk.sum())
    g = w.group
    elt = w.elt_bytes
    # algorithmic bytes of one main-kernel launch: K+V of valid rows, the valid
    # query rows, and the fp32 out + lse rows it produces (tree drafts: plus
    # the 8-byte draft-mask word of every valid row)
    tree = inp["draft_mask"] is not None
    launch_bytes = kv_bytes + int(chunk.sum()) * (w.Hq * (w.D * elt + (w.D + 1) * 4) + (8 if tree else 0))

    def to_dev(a):
        if w.dtype in ("bf16", "f16"):
            t16 = torch.bfloat16 if w.dtype == "bf16" else torch.float16
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(t16).to(dev)
        return torch.from_numpy(a).to(dev)

    paged = w.page_size > 0
    kname, vname = ("k_pages", "v_pages") if paged else ("k_cache", "v_cache")
    set_bytes = inp[kname].nbytes * 2
    n_sets = args.rotate or max(4, int(np.ceil(1.0e9 / set_bytes)))
    q = to_dev(inp["q"])
    k0, v0 = to_dev(inp[kname]), to_dev(inp[vname])
    table_d = torch.from_numpy(inp["block_table"]).to(dev) if paged else None
    sets = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(n_sets - 1)]
    ctx_d = torch.from_numpy(ctx).to(dev)
    chunk_d = torch.from_numpy(chunk).to(dev)
    mask_d = torch.from_numpy(inp["draft_mask"].view(np.int64)).to(dev) if tree else None
    desc = pkg.make_desc(w.B, w.Hq, w.Hkv, w.D, w.C_max, w.S_max, pkg.binding._dtype_code(q), args.grid_blocks)
    ws = pkg.alloc_workspace(desc, dev)
    out = torch.empty((w.B, w.C_max, w.Hq, w.D), dtype=torch.float32, device=dev)
    lse = torch.empty((w.B, w.C_max, w.Hq), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    log(f"{n_sets} input sets x {set_bytes / 1e6:.0f} MB, grid_blocks={args.grid_blocks or 'default'}, "
        f"KV bytes/step={kv_bytes / 1e6:.1f} MB, draft tokens/step={tokens}")

    def step(i):
        k, v = sets[i % n_sets]
        if paged:
            pkg.verify_attn_paged(q, k, v, table_d, ctx_d, chunk_d, w.scale, draft_mask=mask_d, out=out, lse=lse,
                                  workspace=ws, grid_blocks=args.grid_blocks, stream=stream)
        elif tree:
            pkg.verify_attn_tree(q, k, v, ctx_d, chunk_d, mask_d, w.scale, out=out, lse=lse, workspace=ws,
                                 grid_blocks=args.grid_blocks, stream=stream)
        else:
            pkg.verify_attn(q, k, v, ctx_d, chunk_d, w.scale, out=out, lse=lse, workspace=ws,
                            grid_blocks=args.grid_blocks, stream=stream)

    # settle (sustained load until the GPU runs at its working clock: a short
    # warmup alone measures the ramp, about 5% slower on this workload), warm
    # up, then the timed region: exactly K steps, bracketed by synchronisations
    ms_per_step, settle_steps = run_timed(step, args, stream)

    # Average launch duration of the main kernel: every step is one launch of
    # it on `stream`, so the timed region's HIP events divided by K give it
    # (an upper bound: gaps between launches are included).  As a diagnostic,
    # HIP events recorded on the same stream right before and after each
    # step give a per-launch spread; those add the events' own ~2 us to each
    # launch.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(ev):
        a.record(stream)
        step(i)
        b.record(stream)
    torch.cuda.synchronize()
    main_ms = np.array([a.elapsed_time(b) for a, b in ev])
    main_avg_ms = float(main_ms.mean())
    if pkg.workspace_status(ws, stream) != 0:
        raise RuntimeError("an in-kernel hand-off gave up during the benchmark: results are unspecified")

    # The measured streaming ceiling: the probe reads as many bytes as one
    # call's K and V rows (the first halves of K and V of the rotating input
    # sets), timed like the steps; the faster of its two load forms counts.
    ceiling = measure_ceiling(args, sets, kv_bytes, stream) if args.ceiling else None

    t = ms_per_step / 1e3
    value = kv_bytes / t / 1e9
    launch_s = t                   # average launch duration over the timed region
    achieved = launch_bytes / launch_s / 1e9
    # useful matrix work: Q K^T and P V over every valid (row, key) pair of
    # a unit, 2 FLOP per multiply-add: 4 c_b g T_b D per (sequence, KV head)
    useful_flop = 4.0 * w.Hq * w.D * float(np.sum(chunk.astype(np.int64) * (ctx.astype(np.int64) + chunk)))
    traffic = load_traffic(w.name)
    log(f"step {ms_per_step * 1e3:.1f} us -> {value:.0f} GB/s effective KV, {tokens / t / 1e6:.2f} M tok/s; "
        f"main kernel {launch_s * 1e6:.1f} us per launch -> {achieved:.0f} GB/s; event-bracketed per-launch "
        f"mean {main_avg_ms * 1e3:.1f} us (p10 {np.percentile(main_ms, 10) * 1e3:.1f}, "
        f"p90 {np.percentile(main_ms, 90) * 1e3:.1f})")

    cpu = None
    if args.cpu_budget > 0:
        log("timing the fp64 oracle on the host ...")
        cpu = cpu_baseline(inp, w, args.cpu_budget)

    rec = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_steps": settle_steps,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "description": w.description, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv,
                   "head_dim": w.D, "ctx_lens_sum": int(ctx.sum()), "chunk_lens_sum": tokens,
                   "C_max": w.C_max, "S_max": w.S_max, "draft": w.draft, "page_size": w.page_size,
                   "grid_blocks": args.grid_blocks or 256,
                   "input_sets": n_sets,
                   "parallelism": "single GPU"},
        "verified_tokens_per_s": round(tokens / t, 1),
        "kv_bytes_per_step": kv_bytes,
        "roofline": {"bound": "hbm", "kernel": MAIN_KERNEL, "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "traffic_unit": "HBM bytes per launch",
                     "traffic_over_algorithmic": round(traffic / launch_bytes, 4) if traffic else None,
                     "algorithmic_bytes_per_launch": launch_bytes,
                     "avg_launch_us": round(launch_s * 1e6, 3),
                     "event_bracketed_launch_us": round(main_avg_ms * 1e3, 3),
                     "event_bracketed_launch_us_p10_p50_p90": [round(float(np.percentile(main_ms, q_)) * 1e3, 3)
                                                              for q_ in (10, 50, 90)],
                     "measured_ceiling_gbs": round(ceiling["gbs"], 2) if ceiling else None,
                     "frac_of_ceiling": round(achieved / ceiling["gbs"], 4) if ceiling else None,
                     "ceiling_probe": ceiling},
        "mfma_util": {"useful_flop": useful_flop, "achieved_tflops": round(useful_flop / t / 1e12, 2),
                      "peak_tflops": MFMA_BF16_PEAK_TFLOPS if w.dtype != "f32" else 157.3,
                      "frac": round(useful_flop / t / 1e12 / (MFMA_BF16_PEAK_TFLOPS if w.dtype != "f32"
                                                             else 157.3), 5)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
