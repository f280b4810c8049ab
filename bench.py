"""Benchmark of the SAEF iteration on one MI355X.

One step = one whole iteration of Algorithm 1 (SAEF branch, double-way
compression) through the C ABI entry point saef_round: error averaging when
due, step ahead, worker compression of all K workers, server aggregation and
re-update.  The synthetic gradients of the iteration are already resident in
HBM when the timed region starts (two seeded gradient sets alternate).

Default workload: ResNet-50 shaped tensor list (161 tensors, d = 25,557,032),
K = 8 workers, lr 0.1, error averaging period 20.  --momentum MU runs the
momentum variant of the worker step (saef_round_momentum) instead.

Prints one JSON line (metric, value = parameters per second per K-worker
iteration, roofline of the dominant kernel, CPU oracle baseline).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0      # MI355X HBM3E
METRIC = "params/s per K-worker SAEF round + achieved HBM GB/s vs MI355X peak"
EVENT_EVERY = 4             # timed region: HIP events on every 4th dominant-kernel dispatch


def kernel_hash() -> str:
    """Hash of the kernel sources (the counters in profiles/ apply to it only)."""
    from paper_2008_05823_amd.profile_summary import kernel_source_hash
    return kernel_source_hash()


def traffic_from_profile(workload: str):
    """HBM bytes per compress launch from the committed rocprofv3 counter
    summary, when it was taken on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", f"compress_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha256_16") != kernel_hash():
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, grads_host, x0, rounds: int, keep=None) -> dict:
    """The CPU oracle (single thread) on the first `rounds` iterations of the
    same workload and inputs (Top-K with kept counts `keep` when given)."""
    import numpy as np
    from oracle import oracle as O
    off, n, d_pad = w.layout()
    orc = O.Oracle(off, n, d_pad)
    K, L = w.K, w.L
    x = x0.copy()
    e = np.zeros((K, d_pad), np.float32)
    e_srv = np.zeros(d_pad, np.float32)
    xh = np.zeros((K, d_pad), np.float32)
    signs = np.zeros((K, d_pad // 64), np.uint64)
    scales = np.zeros((K, L), np.float32)
    ss = np.zeros(d_pad // 64, np.uint64)
    sscales = np.zeros(L, np.float32)
    if keep is not None:
        total_keep = int(np.sum(keep))
        rank = np.zeros((K, d_pad // 64), np.uint32)
        vals = np.zeros((K, total_keep), np.float32)
        srank = np.zeros(d_pad // 64, np.uint32)
        svals = np.zeros(total_keep, np.float32)
    total = 0.0
    for t in range(rounds):
        g = grads_host[t % len(grads_host)]
        t0 = time.perf_counter()
        if keep is not None:
            rc = orc.topk_round(t, w.period, K, np.float32(w.lr), 0.0, w.mode, keep, g, None, e,
                                e_srv, x, xh, signs, rank, vals, ss, srank, svals)
        else:
            rc = orc.round(t, w.period, K, np.float32(w.lr), w.mode, g, e, e_srv, x, xh, signs,
                           scales, ss, sscales)
        total += time.perf_counter() - t0
        if rc != 0:
            raise RuntimeError(f"oracle returned {rc}")
    per_round = total / rounds
    return {"value": w.d / per_round, "unit": "params/s", "cores": 1, "kind": "oracle",
            "sample": f"{rounds} full iterations (t=0..{rounds - 1}) of the {w.name} workload, "
                      f"K={K}, single-threaded C oracle"
                      + (" (Top-K)" if keep is not None else "")
                      + f", {per_round:.2f} s per iteration",
            "host_cpu": host_cpu_model(), "host_threads": os.cpu_count()}


def host_cpu_model() -> str:
    """The host CPU's model name (Linux /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def stream_probe_gbps(n: int, reps: int = 10, in_place_copy: bool = False) -> float:
    """GB/s of the library's stream probe: c = a + b over n fp32 elements (2
    reads + 1 write, the worker compression's access pattern: the HBM ceiling
    the roofline fraction is also given against), or with in_place_copy
    a = a (1 read + 1 write in place, the server step's streams)."""
    import torch
    from paper_2008_05823_amd import saef
    a = torch.empty(n, dtype=torch.float32, device="cuda")
    a.fill_(1.0)
    if in_place_copy:
        b, c, nbytes = None, a, 8 * n
    else:
        b, c, nbytes = torch.empty_like(a), torch.empty_like(a), 12 * n
        b.fill_(2.0)
    for _ in range(2):
        saef.saef_stream_probe(a, b, c)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        saef.saef_stream_probe(a, b, c)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    del a, b, c
    return nbytes / (ms * 1e-3) / 1e9


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="resnet50",
                    help="flat64k | resnet56 | resnet50 | bert_base | flat256m")
    ap.add_argument("--cpu-rounds", type=int, default=2,
                    help="iterations of the CPU oracle baseline (0 = skip)")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the stream probe (the HBM ceiling of the compression's pattern)")
    ap.add_argument("--momentum", type=float, default=None,
                    help="momentum constant mu in [0, 1): time saef_round_momentum")
    ap.add_argument("--variant", choices=("saef", "ef"), default="saef",
                    help="saef: step ahead (default); ef: local error feedback, the gradient "
                         "is taken at x_t (saef_round_begin / saef_round_end)")
    ap.add_argument("--topk", type=float, default=None,
                    help="layer-wise Top-K compressor keeping this percent of every tensor "
                         "(saef_topk_round) instead of the scaled sign")
    ap.add_argument("--mismatch", action="store_true",
                    help="compute the gradient-mismatch bounds in every iteration")
    ap.add_argument("--kernel-events", choices=("on", "off"), default="on",
                    help="HIP events around each kernel in the timed region (roofline); "
                         "'off' times the iterations alone")
    ap.add_argument("--graph", action="store_true",
                    help="replay each iteration from a HIP graph (one captured per kind of "
                         "iteration: gradient buffer, error averaging or not); implies "
                         "--kernel-events off")
    args = ap.parse_args()
    if args.graph:
        args.kernel_events = "off"

    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (got --gpus {args.gpus}); the "
              "K workers are simulated on that GPU", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2008_05823_amd import saef
    from paper_2008_05823_amd import workloads as W

    w = W.get(args.workload)
    off, n, d_pad = w.layout()
    K, L, d = w.K, w.L, w.d
    torch.cuda.set_device(0)

    # synthetic inputs, resident in HBM before timing
    n_grad = 2
    grads_host = [W.gradients(w, t) for t in range(n_grad)]
    x0 = W.initial_x(w)
    f32 = dict(dtype=torch.float32, device="cuda")
    g_dev = [torch.from_numpy(g).cuda() for g in grads_host]
    x = torch.from_numpy(x0).cuda()
    e = torch.zeros((K, d_pad), **f32)
    e_srv = torch.zeros(d_pad, **f32)
    xh = torch.zeros((K, d_pad), **f32)
    signs = torch.zeros((K, d_pad // 64), dtype=torch.int64, device="cuda")
    scales = torch.zeros((K, L), **f32)
    srv_signs = torch.zeros(d_pad // 64, dtype=torch.int64, device="cuda")
    srv_scales = torch.zeros(L, **f32)
    layout = saef.Layout(off, n, d_pad, K)
    mu = args.momentum
    m = torch.zeros((K, d_pad), **f32) if mu is not None else None
    split = args.variant == "ef" or args.mismatch
    variant = saef.VARIANT_EF if args.variant == "ef" else saef.VARIANT_SAEF
    mism = torch.zeros(2 * L, dtype=torch.float64, device="cuda") if args.mismatch else None
    xh_arg = xh if variant == saef.VARIANT_SAEF else xh[0]
    topk = None
    if args.topk is not None:
        keep = W.topk_keep(w, args.topk)
        topk = saef.TopK(layout, keep)
        density = float(keep.sum()) / d
        W_ = d_pad // 64
        tk_rank = torch.zeros((K, W_), dtype=torch.int32, device="cuda")
        tk_vals = torch.zeros((K, topk.total), **f32)
        tk_srank = torch.zeros(W_, dtype=torch.int32, device="cuda")
        tk_svals = torch.zeros(topk.total, **f32)

    def step(t):
        if topk is not None and split:
            saef.saef_topk_round_begin(topk, t, w.period, K, w.mode, variant, e, signs, e_srv, x,
                                       xh_arg, mism)
            saef.saef_topk_round_end(topk, t, w.period, K, w.lr, 0.0 if mu is None else mu, w.mode,
                                     g_dev[t % n_grad], m, e, e_srv, x, signs, tk_rank, tk_vals,
                                     srv_signs, tk_srank, tk_svals)
        elif topk is not None:
            saef.saef_topk_round(topk, t, w.period, K, w.lr, 0.0 if mu is None else mu, w.mode,
                                 g_dev[t % n_grad], m, e, e_srv, x, xh, signs, tk_rank, tk_vals,
                                 srv_signs, tk_srank, tk_svals)
        elif split:
            saef.saef_round_begin(layout, t, w.period, K, w.mode, variant, e, e_srv, x, xh_arg,
                                  signs, scales, srv_signs, srv_scales, mism)
            saef.saef_round_end(layout, t, w.period, K, w.lr, 0.0 if mu is None else mu, w.mode,
                                g_dev[t % n_grad], m, e, e_srv, x, signs, scales, srv_signs,
                                srv_scales)
        elif mu is None:
            saef.saef_round(layout, t, w.period, K, w.lr, w.mode, g_dev[t % n_grad], e, e_srv, x,
                            xh, signs, scales, srv_signs, srv_scales)
        else:
            saef.saef_round_momentum(layout, t, w.period, K, w.lr, mu, w.mode, g_dev[t % n_grad],
                                     m, e, e_srv, x, xh, signs, scales, srv_signs, srv_scales)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    run = step
    if args.graph:
        # one graph per kind of iteration in the timed range; capturing
        # records the launches without running them
        if args.warmup < 1:
            print("bench.py: --graph needs --warmup >= 1 (t = 0 is the plain-state iteration)",
                  file=sys.stderr)
            return 2
        graphs = {}

        def kind(t):
            return (t % n_grad, bool(w.period and (t + 1) % w.period == 0))

        for t in range(args.warmup, args.warmup + args.steps):
            if kind(t) not in graphs:
                graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(graph):
                    step(t)
                graphs[kind(t)] = graph
        torch.cuda.synchronize()

        def run(t):
            graphs[kind(t)].replay()
    # timed region: K iterations; every EVENT_EVERY-th dispatch of the dominant
    # kernel (worker compression) stamps HIP events on the launch stream (a
    # stamped dispatch adds ~11 us of idle time around the kernel)
    if args.kernel_events == "on":
        saef.saef_profile_enable(layout, args.steps, kinds=("compress",), every=EVENT_EVERY)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        run(args.warmup + i)
    stop.record()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    prof = saef.saef_profile_read(layout)
    saef.saef_profile_enable(layout, 0)
    if saef.saef_status(layout) != saef.OK:
        print("bench.py: a value left the exact-sum range", file=sys.stderr)
        return 1
    ms_per_step = ms_total / args.steps

    timed_ts = range(args.warmup, args.warmup + args.steps)
    n_avg = sum(1 for t in timed_ts if w.period and (t + 1) % w.period == 0)
    if topk is not None:
        step_ahead = variant == saef.VARIANT_SAEF
        bytes_round = np.mean([W.topk_algorithmic_bytes_per_param(
            K, density, w.mode, averaging=bool(w.period and (t + 1) % w.period == 0))["round"]
            + (8 * K if mu is not None else 0)
            - (0 if step_ahead else (4 + 8 * K) - 8)
            + ((4 * K + (4 if w.mode == 1 else 0)) if args.mismatch else 0)
            for t in timed_ts]) * d
    else:
        bytes_round = np.mean([W.algorithmic_bytes_per_param(
            K, w.mode, averaging=bool(w.period and (t + 1) % w.period == 0),
            momentum=mu is not None, step_ahead=variant == saef.VARIANT_SAEF,
            mismatch=args.mismatch) for t in timed_ts]) * d

    # dominant kernel: worker compression (12 K + K/8 bytes per parameter,
    # 20 K + K/8 with momentum)
    c_count, c_ms = prof["compress"]
    # Top-K: the iteration end (compression and server step) runs pipelined
    # over tensor groups as one timed span when the plan pipelines it
    tk_pipelined = topk is not None and c_count > 0 and prof["aggregate"][0] == 0
    if topk is not None:
        tb = W.topk_algorithmic_bytes_per_param(K, density, w.mode)
        c_bytes = (tb["worker"] + (8 * K if mu is not None else 0)
                   + (tb["server"] if tk_pipelined else 0)) * d
    else:
        c_bytes = ((20 if mu is not None else 12) * K + K / 8) * d
    c_gbps = c_bytes / (c_ms / c_count * 1e-3) / 1e9 if c_count else None
    traffic = (traffic_from_profile(args.workload)
               if (mu is None and not split and topk is None) else None)

    # breakdown of every kernel, from a separate pass of the same length (each
    # timed dispatch costs a few microseconds, so it is kept out of the value)
    kernels = None
    if args.kernel_events == "on":
        saef.saef_profile_enable(layout, len(saef.PROFILE_KINDS) * args.steps)
        t0 = args.warmup + args.steps
        for i in range(args.steps):
            step(t0 + i)
        torch.cuda.synchronize()
        kernels = {k: {"launches": c, "avg_us": (ms / c * 1e3) if c else None}
                   for k, (c, ms) in saef.saef_profile_read(layout).items()}
        saef.saef_profile_enable(layout, 0)
    # the HBM ceiling of the dominant kernel's pattern: as many elements as
    # the compression streams per launch (K rows of d_pad)
    probe = None if args.no_probe else round(stream_probe_gbps(K * d_pad), 1)
    # and of the server step's: its error and weight rows, read and written in place
    probe_1r1w = None if args.no_probe else round(stream_probe_gbps(2 * d_pad,
                                                                    in_place_copy=True), 1)

    out = {
        "metric": METRIC,
        "value": d / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {L} tensors, d={d}, K={K} simulated workers, "
                               f"double-way, lr={w.lr}, error averaging period {w.period}"
                               + (f", momentum {mu}" if mu is not None else "")
                               + (", local error feedback" if args.variant == "ef" else "")
                               + (", mismatch bounds" if args.mismatch else "")
                               + (f", layer-wise Top-{args.topk}%" if topk is not None
                                  else ", scaled sign"),
                   "K": K, "d": d, "L": L, "period": w.period,
                   "mode": "DC" if w.mode == 1 else "SC",
                   **({"momentum": mu} if mu is not None else {}),
                   **({"variant": "ef"} if args.variant == "ef" else {}),
                   **({"mismatch": True} if args.mismatch else {}),
                   **({"topk_percent": args.topk} if topk is not None else {}),
                   **({"graph": True} if args.graph else {})},
        "worker_params_per_s": K * d / (ms_per_step * 1e-3),
        "round_hbm_gbps": bytes_round / (ms_per_step * 1e-3) / 1e9,
        "round_frac_of_peak": bytes_round / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "averaging_steps_timed": n_avg,
        "kernels": kernels,
        "kernels_note": "per-kernel averages from a second pass with every dispatch timed",
        "stream_probe_gbps": probe,
        "stream_probe_1r1w_gbps": probe_1r1w,
        "roofline": {"bound": "hbm",
                     "kernel": ("compress" if topk is None else
                                "topk_round_end (worker compression and server step, pipelined "
                                "over two tensor groups)" if tk_pipelined else
                                "topk_compress (all passes)"),
                     "achieved": c_gbps,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": c_gbps / HBM_PEAK_GBPS if c_gbps else None,
                     "traffic": traffic, "algorithmic_bytes_per_launch": c_bytes,
                     "launches_timed": c_count,
                     "achieved_source": f"HIP events on every {EVENT_EVERY}th compression "
                                        "dispatch of the timed region",
                     "traffic_source": (f"profiles/compress_{args.workload}_counters.txt "
                                        f"(rocprofv3 FETCH_SIZE + WRITE_SIZE, kernel source "
                                        f"sha256[:16] {kernel_hash()})") if traffic else None,
                     "stream_ceiling_gbps": probe,
                     "frac_of_stream": (c_gbps / probe) if (c_gbps and probe) else None},
    }
    if args.cpu_rounds > 0:
        if mu is not None or split:
            out["cpu_baseline"] = None  # the oracle baseline covers the default iteration
        else:
            out["cpu_baseline"] = cpu_baseline(w, grads_host, x0, args.cpu_rounds,
                                               keep=None if topk is None else W.topk_keep(
                                                   w, args.topk))
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
