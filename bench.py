"""Outer-step benchmark: one JSON line on stdout.

A step is one pass of the whole hot path over one batch of synthetic input:
per-step edge masks and their Metropolis weights on the host, then the fused
kernel (outer gradient, Mix2, Mix1, Nesterov, consensus distance of every
intermediate) and the consensus finalize kernel.  Inputs are resident in HBM
before the timed region starts.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]

The default workload is 8 workers x 1.1e9 parameters with bf16 parameter
storage, float32 momentum and float32 arithmetic (global-mean Mix1, ring Mix2
with every edge dropped with probability 0.1 per step and Metropolis
reweighting).  Only one GPU is used.

The three arrays live in one buffer laid out by fgd_state_layout: the
momentum one range of physical memory past the parameter arrays (the fused
step runs about 17% longer when they share a range); --placement packed puts
them back to back instead.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
RESTORE_EVERY = 20      # timed steps between restores of the pristine inputs
METRIC = "outer-step HBM GB/s and % of MI355X HBM peak; params·workers/sec"


def read_traffic(workload, bytes_per_launch, step_hash, kernel="fused_step"):
    """HBM traffic per launch from the committed rocprofv3 counter summary,
    if it was taken with a library built from the same step sources as the
    loaded one (`step_hash`, the library's own fgd_source_hash); else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_hash") != step_hash:
        return None
    return {"fetch_bytes": t["fetch_bytes_per_launch"], "write_bytes": t["write_bytes_per_launch"],
            "total_bytes": t["fetch_bytes_per_launch"] + t["write_bytes_per_launch"],
            "ratio_to_algorithmic": (t["fetch_bytes_per_launch"] + t["write_bytes_per_launch"]) / bytes_per_launch,
            "kernel_source_hash": step_hash}


def host_cpu():
    model = platform.processor() or ""
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
    except Exception:
        pass
    return model, os.cpu_count()


def host_slice(tp, tl, v, dtype, p_slice):
    """Host copies of the first p_slice parameters of every worker row."""
    import numpy as np
    import torch

    if dtype == "bf16":
        h_tp = tp[:, :p_slice].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        h_tl = tl[:, :p_slice].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    else:
        h_tp = tp[:, :p_slice].contiguous().cpu().numpy()
        h_tl = tl[:, :p_slice].contiguous().cpu().numpy()
    return h_tp, h_tl, v[:, :p_slice].contiguous().cpu().numpy()


def cpu_baseline(sl, w, topo1, topo2):
    """The CPU oracle, single-threaded, on the first parameters of every worker
    row of the GPU's own first-step inputs (every parameter index is
    independent given W, so the work scales exactly with the slice)."""
    import oracle
    from synth import configs

    M = w["M"]
    h_tp, h_tl, h_v = sl
    p_slice = h_tp.shape[1]
    m1, m2 = oracle.Mix.from_topology(topo1), oracle.Mix.from_topology(topo2)
    segs = configs.subset_segments(w)
    if segs is not None:  # the subset restricted to the slice
        segs = [(b, min(e, p_slice)) for b, e in segs.tolist() if b < p_slice]
        if not segs:  # no subset parameter in the slice: Mix2 is the identity there
            m2, segs = oracle.Mix("identity"), None
    t0 = time.perf_counter()
    oracle.outer_step(h_tp, h_tl, h_v, m1, m2, lr=configs.OUTER_LR, mu=configs.MOMENTUM, dtype=w["dtype"],
                      mix1_state=bool(w.get("mix1_state")), subset=segs)
    dt = time.perf_counter() - t0
    gbs = configs.min_bytes_per_step(M, p_slice, w["dtype"]) / dt / 1e9
    model, ncpu = host_cpu()
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"first {p_slice} of {w['P']} parameters x {M} workers of the GPU's first-step inputs "
                      f"and topology, {dt:.2f} s single-threaded; GB/s from the same algorithmic byte count",
            "params_workers_per_s": round(M * p_slice / dt, 1), "host_cpu": model, "host_nproc": ncpu}


JS_WORKLOAD = dict(M=8, U=2048, K=128256, dtype="bf16", k=100, seed=0)


def js_bench(args, fgd, torch):
    """Jensen--Shannon functional distance (Appendix D.2): M workers' and the
    averaged model's logits over U tokens of a K-token vocabulary, resident in
    HBM; a step is one fgd_js_distance call (distances and their means)."""
    from synth import logits as slog

    w = dict(JS_WORKLOAD, dtype=args.js_dtype, k=args.js_topk)
    M, U, K, k = w["M"], w["U"], w["K"], w["k"]
    es = 2 if w["dtype"] == "bf16" else 4
    print(f"[bench] generating JS logits M={M} U={U} K={K}", file=sys.stderr, flush=True)
    A, W = slog.torch_logits(M, U, K, K, w["dtype"], seed=w["seed"])
    d = torch.empty((M, U), dtype=torch.float64, device=A.device)
    mean = torch.empty(M, dtype=torch.float64, device=A.device)
    ws = torch.empty(fgd.fgd_js_workspace_size(w["dtype"], M, U), dtype=torch.uint8, device=A.device)
    stream = torch.cuda.current_stream()

    def step():
        fgd.fgd_js_distance(A, W, w["dtype"], M, U, K, K, k, d, mean, None, ws, None, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(args.steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    nbytes = (M + 1) * U * K * es
    # The row kernel's access pattern without its arithmetic, on the same
    # logits, timed the same way right after the calls.
    pev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    pev[0].record(stream)
    for i in range(args.steps):
        fgd.fgd_stream_js_pattern(A, W, w["dtype"], M, U, K, K, ws, None, stream)
        pev[i + 1].record(stream)
    torch.cuda.synchronize()
    pat_ms = sum(pev[i].elapsed_time(pev[i + 1]) for i in range(args.steps)) / args.steps
    logits = (M + 1) * U * K
    ms = elapsed * 1e3 / args.steps
    avg = sum(step_ms) / len(step_ms)
    achieved = nbytes / (avg * 1e-3) / 1e9
    lib_hash = fgd.library_source_hash()
    wl = f"js_m{M}_u{U}_v{K}_{w['dtype']}"
    tr = read_traffic(wl[len("js_"):], nbytes, lib_hash["js"], kernel="js")
    out = {"metric": "JS distance: logits HBM GB/s and logits/s", "mode": "js", "value": round(nbytes / ms / 1e6, 2),
           "unit": "GB/s", "ms_per_step": round(ms, 4), "step_ms_median": round(step_ms[len(step_ms) // 2], 4),
           "step_ms_min": round(step_ms[0], 4), "steps": args.steps, "warmup": args.warmup,
           "pct_of_hbm_peak": round(100 * nbytes / ms / 1e6 / HBM_PEAK_GBS, 2),
           "logits_per_s": round(logits / (ms * 1e-3), 1), "tokens_workers_per_s": round(M * U / (ms * 1e-3), 1),
           "cd_js": float(mean.mean().item()),
           "config": {"workload": wl, "workers": M, "tokens": U, "vocab": K,
                      "top_k": k, "dtype": w["dtype"], "bytes_per_step": nbytes},
           # Bound: HBM.  Every logit is read once by the row kernel (all
           # M + 1 rows per token); the per-token kernel reads again only
           # the averaged rows' recorded vectors whose maxima reach its
           # threshold, and gathers the workers' logits of the selected
           # tokens.  Most bf16 logits cost a table read instead of a
           # float64 exp.
           "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(achieved / HBM_PEAK_GBS, 4),
                        "traffic": None if tr is None else tr["total_bytes"], "traffic_detail": tr,
                        "kernel": "one fgd_js_distance call (row kernel, per-token kernel, mean kernel)",
                        "kernel_avg_ms": round(avg, 4), "bytes_per_launch": nbytes},
           "kernel_source_hash": lib_hash["js"], "library_source_hash": lib_hash}
    out["pattern_reference"] = {"ms": round(pat_ms, 4), "gbs": round(nbytes / (pat_ms * 1e-3) / 1e9, 1),
                                "call_rate_vs_pattern": round(pat_ms / avg, 4),
                                "what": "the row kernel's loads (same grid, rows, lanes, cache hints, prefetch) "
                                        "without its arithmetic; the call adds the per-token kernels"}
    out["copy_reference_gbs"] = copy_reference(fgd, torch, A.device, args.copy_gb)
    if not args.no_cpu_baseline:
        from oracle import js as ojs

        n = 4
        za = A[:n].float().cpu().numpy()
        zw = W[:, :n].float().cpu().numpy()
        t0 = time.perf_counter()
        ojs.js_distances(zw, za, k)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round((M + 1) * n * K * es / dt / 1e9, 4), "unit": "GB/s", "cores": 1,
                               "kind": "oracle", "sample": f"first {n} of {U} tokens, all {M} workers, {dt:.2f} s",
                               "tokens_workers_per_s": round(M * n / dt, 2)}
    print(json.dumps(out))


def copy_reference(fgd, torch, dev, gb):
    """GB/s of a plain 16-byte streaming copy of `gb` GB (read and written),
    the practical streaming ceiling and the size reference against which the
    HBM traffic counters are calibrated; None for gb <= 0."""
    if gb <= 0:
        return None
    n = int(gb * 1e9) // 16 * 16
    a = torch.empty(n, dtype=torch.uint8, device=dev)
    b = torch.empty(n, dtype=torch.uint8, device=dev)
    fgd.fgd_stream_copy(b, a, n)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        fgd.fgd_stream_copy(b, a, n)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * n * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    return round(gbs, 1)


def consensus_bench(args, fgd, torch, w):
    """Standalone consensus distance (Sec. 4.4; Appendix D.1): S_m of the
    workload's theta_prev, resident in HBM; a step is one
    fgd_consensus_distance call (the streaming kernel and its finalize).  The
    scratch-free variant is timed beside it on the same array."""
    from synth import tensors

    M, P, dtype = w["M"], w["P"], w["dtype"]
    ld = -(-P // 8) * 8
    es = 2 if dtype == "bf16" else 4
    dev = torch.device("cuda:0")
    print(f"[bench] consensus: generating {args.workload} theta_prev", file=sys.stderr, flush=True)
    tp, tl, v = tensors.torch_inputs(M, P, ld=ld, dtype=dtype, prev_std=w["prev_std"], drift_std=w["drift_std"],
                                     mom_std=0.0, seed=w["seed"], device=dev)
    del tl, v
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    out = torch.zeros(M, dtype=torch.float64, device=dev)
    out2 = torch.zeros(M, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        t0 = time.perf_counter()
        ev[0].record(stream)
        for i in range(args.steps):
            fn()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return wall, sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))

    wall, ms = timed(lambda: eng.consensus_distance(tp, out, stream))
    _, ms2 = timed(lambda: fgd.fgd_consensus_distance_noalloc(M, P, ld, dtype, tp, out2, stream))
    nbytes = M * P * es
    avg = sum(ms) / len(ms)
    achieved = nbytes / (avg * 1e-3) / 1e9
    res = {"metric": "standalone consensus distance: HBM GB/s and % of MI355X HBM peak", "mode": "consensus",
           "value": round(nbytes * args.steps / wall / 1e9, 2), "unit": "GB/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(wall * 1e3 / args.steps, 4),
           "step_ms_median": round(ms[len(ms) // 2], 4), "step_ms_min": round(ms[0], 4),
           "higher_is_better": True, "dtype": "f32", "storage_dtype": dtype, "data": "synthetic",
           "config": {"workload": args.workload, "workers": M, "params_per_worker": P,
                      "what": "S_m = sum_p (x_m,p - mean_n x_n,p)^2 of theta_prev", "bytes_per_call": nbytes},
           "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(achieved / HBM_PEAK_GBS, 4),
                        "traffic": None, "kernel": "consensus_kernel + finalize_kernel (one call)",
                        "kernel_avg_ms": round(avg, 4), "bytes_per_launch": nbytes},
           "noalloc_ms_median": round(ms2[len(ms2) // 2], 4),
           "copy_reference_gbs": copy_reference(fgd, torch, dev, args.copy_gb),
           "noalloc_same_bits": bool(torch.equal(out, out2)),
           "kernel_source_hash": fgd.library_source_hash()["step"], "library_source_hash": fgd.library_source_hash()}
    t = read_traffic(args.workload, nbytes, fgd.library_source_hash()["step"], kernel="consensus")
    if t is not None:
        res["roofline"]["traffic"] = t["total_bytes"]
        res["roofline"]["traffic_detail"] = t
    if not args.no_cpu_baseline:
        import oracle

        p_slice = min(P, (1 << 27) // M)
        h = tp[:, :p_slice].contiguous()
        h = h.view(torch.int16).cpu().numpy().view("uint16") if dtype == "bf16" else h.cpu().numpy()
        t0 = time.perf_counter()
        oracle.consensus(h, P=p_slice, dtype=dtype)
        dt = time.perf_counter() - t0
        model, ncpu = host_cpu()
        res["cpu_baseline"] = {"value": round(M * p_slice * es / dt / 1e9, 4), "unit": "GB/s", "cores": 1,
                               "kind": "oracle", "sample": f"first {p_slice} of {P} parameters x {M} workers, "
                                                           f"{dt:.2f} s single-threaded",
                               "host_cpu": model, "host_nproc": ncpu}
    eng.close()
    print(json.dumps(res))


def split_round_bench(args, fgd, eng, torch, tp, tl, v, x, w, step_topos, placement):
    """Split execution of a round (Appendix A, Algorithm 1): the Mix1 half is
    launched on a side stream at the start of the round and overlaps a
    stand-in inner loop (bf16 matrix products on the main stream); the
    blocking half follows once both are done.  Reports each half alone, the
    inner loop alone and the overlapped round, and how much of the Mix1 half
    the inner loop hides.  One JSON line on stdout."""
    M, P = w["M"], w["P"]
    main_s = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    n1, n2 = eng.num_cd_rows_split()
    cd1 = torch.zeros((n1, M), dtype=torch.float64, device=tp.device)
    cd2 = torch.zeros((n2, M), dtype=torch.float64, device=tp.device)
    b1, b2 = eng.min_bytes_split(write_local=True)
    vmix = v if w.get("mix1_state") else None
    A = torch.randn(8192, 8192, device=tp.device, dtype=torch.bfloat16)
    B = torch.randn(8192, 8192, device=tp.device, dtype=torch.bfloat16)
    C = torch.empty_like(A)

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def set_masks(i):
        if step_topos is not None:
            eng.set_topology_dict("mix2", step_topos[i % len(step_topos)])

    def timed(fn, stream, reps):
        e0, e1 = ev(), ev()
        e0.record(stream)
        for i in range(reps):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    print("[bench] split: halves alone", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        eng.mix1(tp, x, vmix, cd1, main_s, num_blocks=args.mix1_blocks)
        set_masks(i)
        eng.outer_step_blocking(x, tp, tl, v, cd2, write_local=True, stream=main_s)
    torch.cuda.synchronize()
    nb = args.mix1_blocks
    t_mix1 = timed(lambda i: eng.mix1(tp, x, vmix, cd1, main_s, num_blocks=nb), main_s, args.steps)
    t_block = timed(lambda i: (set_masks(i), eng.outer_step_blocking(x, tp, tl, v, cd2, write_local=True,
                                                                     stream=main_s)), main_s, args.steps)
    timed(lambda i: torch.matmul(A, B, out=C), main_s, 3)  # library set-up outside the timing
    t_gemm = timed(lambda i: torch.matmul(A, B, out=C), main_s, 10)
    n_gemm = max(1, int(2.0 * t_mix1 / t_gemm + 0.999))
    t_inner = timed(lambda i: [torch.matmul(A, B, out=C) for _ in range(n_gemm)], main_s, 5)

    copy_gbs = copy_reference(fgd, torch, tp.device, args.copy_gb)
    print("[bench] split: overlapped rounds", file=sys.stderr, flush=True)
    rounds = []
    for r in range(args.steps):
        e0, e1 = ev(), ev()
        e0.record(main_s)
        side.wait_stream(main_s)
        with torch.cuda.stream(side):
            eng.mix1(tp, x, vmix, cd1, side, num_blocks=nb)
            done = torch.cuda.Event()
            done.record(side)
        for _ in range(n_gemm):
            torch.matmul(A, B, out=C)
        main_s.wait_event(done)
        set_masks(r)
        eng.outer_step_blocking(x, tp, tl, v, cd2, write_local=True, stream=main_s)
        e1.record(main_s)
        rounds.append((e0, e1))
    torch.cuda.synchronize()
    t_round = sorted(a.elapsed_time(b) for a, b in rounds)[len(rounds) // 2]
    exposed = max(0.0, t_round - t_inner - t_block)
    lib_hash = fgd.library_source_hash()
    tr1 = read_traffic(args.workload, b1, lib_hash["step"], kernel="split_mix1")
    tr2 = read_traffic(args.workload, b2, lib_hash["step"], kernel="split_blocking")
    out = {
        "metric": "split outer step: Mix1 half hidden under the inner loop; blocking-half HBM GB/s",
        "mode": "split", "workload": args.workload, "steps": args.steps, "warmup": args.warmup,
        "value": round(b2 / (t_block * 1e-3) / 1e9, 2), "unit": "GB/s",
        "mix1_ms": round(t_mix1, 4), "mix1_gbs": round(b1 / (t_mix1 * 1e-3) / 1e9, 1),
        "blocking_ms": round(t_block, 4), "blocking_gbs": round(b2 / (t_block * 1e-3) / 1e9, 1),
        "blocking_frac_of_peak": round(b2 / (t_block * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "bytes": {"mix1": b1, "blocking": b2}, "inner_standin": f"{n_gemm} bf16 GEMMs 8192^3 per round",
        "mix1_blocks": nb or "one per CU",
        "inner_ms": round(t_inner, 4), "round_ms_median": round(t_round, 4), "exposed_mix1_ms": round(exposed, 4),
        "mix1_hidden_fraction": round(1.0 - min(exposed, t_mix1) / t_mix1, 4),
        "config": {"workers": M, "params_per_worker": P, "dtype": w["dtype"], "write_back_theta_local": True,
                   "mix1_also_on_momentum": bool(w.get("mix1_state")), "placement": placement},
        "roofline": {"bound": "hbm", "achieved": round(b2 / (t_block * 1e-3) / 1e9, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(b2 / (t_block * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None if tr2 is None else tr2["total_bytes"], "traffic_detail": tr2,
                     "kernel": "blocking half (stream time of the call: kernel and consensus finalize)",
                     "bytes_per_launch": b2},
        "mix1_roofline": {"bound": "hbm", "achieved": round(b1 / (t_mix1 * 1e-3) / 1e9, 2), "peak": HBM_PEAK_GBS,
                          "unit": "GB/s", "frac": round(b1 / (t_mix1 * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "traffic": None if tr1 is None else tr1["total_bytes"], "traffic_detail": tr1,
                          "kernel": f"Mix1 half on {nb or 'one block per CU'} blocks (counter reset, kernel, "
                                    f"finalize)", "bytes_per_launch": b1},
        "copy_reference_gbs": copy_gbs,
        "kernel_source_hash": lib_hash["step"], "library_source_hash": lib_hash,
    }
    print(json.dumps(out))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="m8_p1100m_bf16")
    ap.add_argument("--cpu-slice", type=int, default=None,
                    help="parameters per worker in the CPU sample (default: 3 * 2^27 parameter-workers in all, "
                         "about 12 s of single-threaded oracle work)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-gb", type=float, default=8.0, help="size of the plain-copy reference, GB")
    ap.add_argument("--js-dtype", choices=["bf16", "f32"], default="bf16",
                    help="storage of the logits in --mode js (the benchmark workload is bf16)")
    ap.add_argument("--js-topk", type=int, default=100,
                    help="top-k tokens of --mode js (the paper's and the benchmark's 100; above 512 every "
                         "token takes the radix kernel)")
    ap.add_argument("--mode", choices=["fused", "split", "js", "consensus"], default="fused",
                    help="fused: one-pass outer step (the benchmark); split: Mix1 half on a side stream "
                         "overlapping a stand-in inner loop, then the blocking half; js: Jensen-Shannon "
                         "distance of 8 workers over 2048 tokens of a 128256-token vocabulary (bf16 logits); "
                         "consensus: the standalone consensus distance of the workload's theta_prev")
    ap.add_argument("--placement", choices=["spread", "packed"], default="spread",
                    help="spread: the momentum one physical-memory range past the parameter arrays "
                         "(fgd_state_layout; packed when memory is short); packed: the arrays back to back")
    ap.add_argument("--mix1-blocks", type=int, default=128,
                    help="split mode: blocks of the Mix1 half (0: one per CU); half the CUs gave the shortest "
                         "overlapped round in a sweep of 32-256")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the engine has no multi-GPU path "
              "(each parameter index is independent, so a P-sharded run needs no exchange); "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import __graft_entry__

    __graft_entry__.ensure_built()  # builds only when no library is present
    import paper_2606_22768_amd as fgd
    from synth import configs, tensors

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    if args.mode == "js":
        js_bench(args, fgd, torch)
        return
    w = configs.WORKLOADS[args.workload]
    if args.mode == "consensus":
        consensus_bench(args, fgd, torch, w)
        return
    M, P, dtype = w["M"], w["P"], w["dtype"]
    ld = -(-P // 8) * 8
    dev = torch.device("cuda:0")
    eng = fgd.Engine(M, P, ld, dtype, configs.OUTER_LR, configs.MOMENTUM, device=0,
                     mix1_state=bool(w.get("mix1_state")))
    split = args.mode == "split"
    spread = args.placement == "spread"
    if spread:
        # The spread layout leaves a gap; fall back to packed when the pool,
        # the pristine copies, the copy reference and the generator's
        # temporaries would not fit.
        es = 2 if dtype == "bf16" else 4
        _, total = eng.state_layout(spread=True, with_x=split)
        need = total + M * ld * (es + 4) + 2 * int(args.copy_gb * 1e9) + 8 * P + (4 << 30)
        spread = need <= torch.cuda.mem_get_info(dev)[0]
    free_before = torch.cuda.mem_get_info(dev)[0]
    st = eng.alloc_state(spread=spread, with_x=split)
    packed_mom = eng.state_layout(spread=False, with_x=split)[0][3]
    placement = ("momentum one physical-memory range (%.0f GiB) past theta_prev" % (st["offsets"][3] / 2**30)
                 if st["offsets"][3] != packed_mom else "packed")
    print(f"[bench] generating {args.workload} inputs ({placement}; {free_before / 2**30:.1f} GiB free before the "
          f"buffer)", file=sys.stderr, flush=True)
    tp, tl, v = tensors.torch_inputs(M, P, ld=ld, dtype=dtype, prev_std=w["prev_std"], drift_std=w["drift_std"],
                                     mom_std=w["mom_std"], seed=w["seed"], device=dev,
                                     out=(st["theta_prev"], st["theta_local"], st["momentum"]))
    sl = None if args.no_cpu_baseline else host_slice(tp, tl, v, dtype, min(args.cpu_slice or (3 << 27) // M, P))
    segs = configs.subset_segments(w)
    if segs is not None:
        eng.set_mix2_subset(segs)
    topo1 = configs.topology(w["mix1"], M, w["k1"], w["seed"])
    eng.set_topology_dict("mix1", topo1)
    per_step_masks = w["mix2"][1] == "metropolis" and w["mix2"][0] == "ring"

    def topo2_for(step):
        return configs.topology(w["mix2"], M, w["k2"], w["seed"], step=step)

    topo2 = topo2_for(0)
    eng.set_topology_dict("mix2", topo2)
    cd = torch.zeros((eng.num_cd_rows(), M), dtype=torch.float64, device=dev)
    # Mask tables for every step are drawn before timing (input generation);
    # the engine still builds the weights and uploads them inside each step.
    step_topos = [topo2_for(s) for s in range(args.warmup + args.steps)] if per_step_masks else None
    stream = torch.cuda.current_stream()

    def step(i):
        if step_topos is not None:
            eng.set_topology_dict("mix2", step_topos[i])
        eng.outer_step(tp, tl, v, cd, stream)

    if split:
        split_round_bench(args, fgd, eng, torch, tp, tl, v, st["x"], w, step_topos, placement)
        eng.close()
        return

    # Pristine copies of the arrays the step updates in place (allocated after
    # the inputs, so they do not change where the inputs live): restored before
    # the timed steps and between chunks of at most RESTORE_EVERY of them, so a
    # long run does not carry its inputs toward denormals.  Not timed.
    pristine = (tp.clone(), v.clone())

    def restore():
        tp.copy_(pristine[0])
        v.copy_(pristine[1])
        torch.cuda.synchronize()

    print("[bench] warmup", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    eng.enable_timing(True)
    print("[bench] timed steps", file=sys.stderr, flush=True)
    # Events on the launch stream bracket every step (median and min per step).
    step_ms, elapsed, done = [], 0.0, 0
    while done < args.steps:
        n = min(RESTORE_EVERY, args.steps - done)
        restore()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        t0 = time.perf_counter()
        ev[0].record(stream)
        for i in range(n):
            step(args.warmup + done + i)
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        elapsed += time.perf_counter() - t0
        step_ms += [ev[i].elapsed_time(ev[i + 1]) for i in range(n)]
        done += n
    step_ms.sort()
    del pristine
    kernel_ms, n_kernels = eng.read_timing()
    eng.enable_timing(False)

    bytes_step = eng.min_bytes_per_step()
    ms_step = elapsed * 1e3 / args.steps
    gbs = bytes_step * args.steps / elapsed / 1e9
    kernel_avg_ms = kernel_ms / max(n_kernels, 1)
    achieved = bytes_step / (kernel_avg_ms * 1e-3) / 1e9
    cd_host = cd.cpu().numpy()

    # The step's own access pattern without its arithmetic, on the same arrays
    # (they keep their bits): the practical ceiling of this read/write mix.
    pattern_ms = None
    if M in (1, 2, 4, 8, 16, 32, 64):
        eng.stream_step_pattern(tp, tl, v, stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(5):
            eng.stream_step_pattern(tp, tl, v, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        pattern_ms = e0.elapsed_time(e1) / 5

    copy_gbs = copy_reference(fgd, torch, dev, args.copy_gb)

    lib_hash = fgd.library_source_hash()
    traffic = read_traffic(args.workload, bytes_step, lib_hash["step"])  # counters of this library's sources
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "step_ms_median": round(step_ms[len(step_ms) // 2], 4),
        "step_ms_min": round(step_ms[0], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",  # the arithmetic type; storage_dtype gives the parameters' storage
        "storage_dtype": dtype,
        "data": "synthetic",
        "pct_of_hbm_peak": round(100.0 * gbs / HBM_PEAK_GBS, 2),
        "params_workers_per_s": round(M * P * args.steps / elapsed, 1),
        "config": {"workload": args.workload, "workers": M, "params_per_worker": P, "row_stride": ld,
                   "storage": "bf16 parameters, f32 momentum" if dtype == "bf16" else "f32 parameters and momentum",
                   "mix1": f"{w['mix1']} x{w['k1']}", "mix2": f"{w['mix2']} x{w['k2']}",
                   "mix1_also_on_momentum": bool(w.get("mix1_state")),
                   "mix2_subset_fraction": (None if segs is None else
                                            round(float(sum(e - b for b, e in segs.tolist())) / P, 4)),
                   "outer_lr": configs.OUTER_LR, "momentum": configs.MOMENTUM,
                   "consensus": "fused, every intermediate", "algorithmic_bytes_per_step": bytes_step,
                   "placement": placement,
                   "parallelism": "single GPU, workers simulated as rows"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None if traffic is None else traffic["total_bytes"],
                     "traffic_detail": traffic,
                     "kernel": "fused outer-step kernel", "kernel_avg_ms": round(kernel_avg_ms, 4),
                     "timed_launches": n_kernels, "bytes_per_launch": bytes_step},
        "pattern_reference": None if pattern_ms is None else {
            "ms": round(pattern_ms, 4), "gbs": round(bytes_step / (pattern_ms * 1e-3) / 1e9, 1),
            "kernel_rate_vs_pattern": round(pattern_ms / kernel_avg_ms, 4),
            "what": "the step's loads and stores (same tiles, launch shape, cache hints) without its arithmetic"},
        "copy_reference_gbs": None if copy_gbs is None else round(copy_gbs, 1),
        "consensus_last_step": {"rows": int(cd_host.shape[0]),
                                "cd_sq_mean_per_row": [float(x) for x in cd_host.mean(axis=1)]},
        "kernel_source_hash": lib_hash["step"],
        "library_source_hash": lib_hash,
    }
    if not args.no_cpu_baseline:
        print("[bench] CPU oracle baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(sl, w, topo1, topo2)
    else:
        out["cpu_baseline"] = None
    eng.close()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
