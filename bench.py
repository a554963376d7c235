"""Benchmark: fused NA on the 2-D 7x7 fp16 workload (B=4, H=4, 56x56, D=32), one GPU.

A timed step is one pass of the fused path on that workload: na_forward then
na_backward (one launch: dK/dV and dQ workgroup roles, Delta in-kernel), inputs
resident in HBM; ms_per_step is the whole forward+backward step.  Three timed
regions, each K back-to-back calls with HIP events on the launch stream at its
two ends only: steps, forwards alone (fwd_ms), backwards alone (bwd_ms).  Each
region is timed --reps times and the median is reported (all repetitions are
listed too).  The reported value is the forward's useful throughput,
4*B*H*N*ell*D FLOPs (masked halo work is not credited) divided by fwd_ms.

A "cold" forward figure is measured beside it: single launches, each after a
512 MiB write that evicts the inputs from L2 and the MALL, timed one by one
with events (which adds the event overhead of one launch).  So are the K
forwards and K backwards replayed from HIP graphs (fwd_ms_graph,
bwd_ms_graph), as a serving loop that captures its launches would run them.

Beside the headline it reports, for every workload (bounded, about a minute in
all): the fused forward and backward against the unfused baseline of separate
PN / softmax / NN / IN launches that store the attention weights (the
paper's own comparison, with its A100 ratios as context), and the fp64 CPU
oracle's time per workload (median of 3).  Two measured ceilings stand beside
the spec peaks: a device-to-device copy's bandwidth and a large fp16 GEMM's
rate.

Prints one JSON line.  --gpus above 1 is refused: the benchmark runs on one GPU.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

import workloads  # noqa: E402

WORKLOAD = workloads.BENCH_WORKLOAD
PEAK_FP16_TFLOPS = 2516.6   # MI355X dense fp16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PMC_FILE = os.path.join(ROOT, "profiles", "na_fwd_kernel.2d_fp16_56x56_k7.pmc.txt")
FWD_SOURCES = ["na_fwd.hip", "na_common.h", "na_stage.h", "na_index.h", "na_fastdiv.h"]


def fwd_source_digest():
    h = hashlib.sha256()
    for name in FWD_SOURCES:
        with open(os.path.join(ROOT, "paper_2403_04690_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per forward launch from committed rocprofv3 counter runs, or None if stale."""
    if not os.path.exists(PMC_FILE):
        return None
    vals = {}
    with open(PMC_FILE) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                key, val = line.split(":", 1)
                vals[key.strip()] = val.strip()
    if vals.get("source_digest") != fwd_source_digest():
        return None
    try:
        return int(float(vals["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(problem, x, budget_s, single_thread_s):
    """The fp64 oracle's forward on the full workload, repeated for about budget_s seconds
    on all host threads, then for about single_thread_s seconds on one thread."""
    import oracle

    f = lambda t: t.double().numpy()
    q, k, v = f(x["q"]), f(x["k"]), f(x["v"])

    def run(budget):
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.forward(q, k, v, problem.kernel_size, problem.dilation,
                           problem.softmax_scale, causal=problem.causal_axes)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget or reps >= 10000:
                return reps, el

    threads = oracle.num_threads()
    reps, el = run(budget_s)
    out = {
        "value": problem.fwd_flops() * reps / el / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"full {problem.name} forward (all {problem.batch * problem.heads * problem.tokens}"
                  f" queries) x {reps} repetitions in {el:.1f} s, fp64",
        "cpu_model": cpu_model(),
        "ms_per_forward": round(el / reps * 1e3, 3),
    }
    if single_thread_s > 0:
        try:
            oracle.set_num_threads(1)
            reps1, el1 = run(single_thread_s)
        finally:
            oracle.set_num_threads(threads)
        out["single_thread"] = {"value": problem.fwd_flops() * reps1 / el1 / 1e12,
                                "ms_per_forward": round(el1 / reps1 * 1e3, 3),
                                "repetitions": reps1}
    return out


def oracle_per_config(max_run_s=5.0):
    """The fp64 oracle on every workload's full tensors: forward (and backward for the
    fwd+bwd workloads), median of 3 runs (one run when a run takes longer than max_run_s)."""
    import oracle

    rows = []
    for name in workloads.CONFIG_ORDER:
        p = workloads.CONFIGS[name]
        x = workloads.make_inputs(p, seed=0, with_grad=p.backward)
        f = {n: t.double().numpy() for n, t in x.items()}
        args = (p.kernel_size, p.dilation, p.softmax_scale)
        cz = p.causal_axes

        def med3(fn):
            ts = []
            for _ in range(3):
                t0 = time.perf_counter()
                fn()
                ts.append(time.perf_counter() - t0)
                if ts[-1] > max_run_s:
                    break
            ts.sort()
            return ts[len(ts) // 2] * 1e3, len(ts)

        fwd_ms, nf = med3(lambda: oracle.forward(f["q"], f["k"], f["v"], *args, causal=cz))
        row = {"workload": name, "fwd_ms": round(fwd_ms, 2), "fwd_runs": nf,
               "fwd_tflops": round(p.fwd_flops() / (fwd_ms * 1e-3) / 1e12, 4)}
        if p.backward:
            bwd_ms, nb = med3(lambda: oracle.backward(f["q"], f["k"], f["v"], f["dout"], *args,
                                                      causal=cz))
            row.update({"bwd_ms": round(bwd_ms, 2), "bwd_runs": nb})
        rows.append(row)
    return rows


# The paper's fused-over-naive speedups on an A100 (FP16, averages over its
# problem sweep; Tables "runtime_breakdown" and "runtime_breakdown_backward"),
# as the ratio t_naive / t_fused: context for the MI355X ratios, not a target.
PAPER_A100_FUSED_OVER_NAIVE = {
    1: {"fwd": 18.59, "fwd_bwd": 9.44},
    2: {"fwd": 10.58, "fwd_bwd": 4.85},
    3: {"fwd": 12.35, "fwd_bwd": 5.47},
}


def fused_vs_unfused(na, dev, spc, K=20, reps=3, names=None):
    """Fused forward/backward against the unfused baseline (separate PN, softmax, NN and IN
    launches storing the attention weights) on every workload (or those named): ms per call,
    median of reps regions of K back-to-back calls."""
    rows = []
    for name in names or workloads.CONFIG_ORDER:
        p = workloads.CONFIGS[name]
        x = workloads.make_inputs(p, seed=0, with_grad=True)
        q, k, v, g = (x[n].to(dev) for n in ("q", "k", "v", "dout"))
        del x
        args = (p.kernel_size, p.dilation, p.softmax_scale)
        cz = p.causal_axes if any(p.causal_axes) else None
        out, lse = torch.empty_like(q), torch.empty(q.shape[:-1], dtype=torch.float32, device=dev)
        dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
        w = torch.empty(tuple(q.shape[:-1]) + (p.window,), dtype=q.dtype, device=dev)
        gw = torch.empty_like(w)
        probs = {}

        def f_fwd():
            na.forward(q, k, v, *args, out=out, lse=lse, causal=cz)

        def f_bwd():
            na.backward(q, k, v, out, lse, g, *args, dq=dq, dk=dk, dv=dv, causal=cz)

        def u_fwd():
            o_, l_, probs["p"] = na.unfused_forward(q, k, v, *args, causal=cz, weights=w)

        def u_bwd():
            na.unfused_backward(q, k, v, probs["p"], g, *args, causal=cz, grad_weights=gw)

        def timed(fn):
            fn()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            one = time.perf_counter() - t0
            ts = []
            for _ in range(reps):
                torch.cuda._sleep(int(min(K * max(one, 50e-6) + 1e-3, 2.0) / spc))
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(K):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) / K)
            return sorted(ts)[len(ts) // 2]

        ff, uf = timed(f_fwd), timed(u_fwd)
        f_fwd()
        fb, ub = timed(f_bwd), timed(u_bwd)
        ctx = PAPER_A100_FUSED_OVER_NAIVE[p.rank]
        rows.append({
            "workload": name,
            "fused_fwd_ms": round(ff, 5), "unfused_fwd_ms": round(uf, 5),
            "fused_bwd_ms": round(fb, 5), "unfused_bwd_ms": round(ub, 5),
            "fwd_speedup": round(uf / ff, 2), "fwd_bwd_speedup": round((uf + ub) / (ff + fb), 2),
            "paper_a100_fp16_avg_speedup": ctx,
            "weights_bytes": w.numel() * w.element_size(),
        })
        del q, k, v, g, out, lse, dq, dk, dv, w, gw, probs
        torch.cuda.empty_cache()
    return rows


def measured_ceilings(dev):
    """Measured beside the spec peaks: a 1 GiB device copy (bytes read + written per
    second) and a 8192^3 fp16 GEMM (torch.matmul, the vendor library), each the best of 5."""
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, device=dev, dtype=torch.float16)
    b = torch.randn(8192, 8192, device=dev, dtype=torch.float16)
    copy_ms, gemm_ms = [], []
    for _ in range(5):
        dst.copy_(src)
        torch.matmul(a, b)
    torch.cuda.synchronize()
    for _ in range(5):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.matmul(a, b)
        e2.record()
        torch.cuda.synchronize()
        copy_ms.append(e0.elapsed_time(e1))
        gemm_ms.append(e1.elapsed_time(e2))
    del src, dst, a, b
    torch.cuda.empty_cache()
    return {"copy_gbs": round(2 * n / (min(copy_ms) * 1e-3) / 1e9, 1),
            "fp16_gemm_tflops": round(2 * 8192 ** 3 / (min(gemm_ms) * 1e-3) / 1e12, 1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--reps", type=int, default=5,
                    help="repetitions of each timed region (the median is reported)")
    ap.add_argument("--cold-launches", type=int, default=20,
                    help="single forward launches after a cache-evicting write (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--cpu-single-thread-seconds", type=float, default=3.0)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the CPU oracle baseline and the MFMA-bound side measurement "
                         "(profiling runs)")
    ap.add_argument("--workload", default=WORKLOAD, choices=workloads.CONFIG_ORDER,
                    help="profiling aid: run the same step on another workload (the reported "
                         "line is defined on the default one)")
    ap.add_argument("--no-graphs", dest="graphs", action="store_false",
                    help="skip the HIP-graph replay side measurement")
    ap.add_argument("--no-compare", dest="compare", action="store_false",
                    help="skip the per-workload fused-versus-unfused comparison, the measured "
                         "ceilings and the per-workload oracle timing")
    ap.add_argument("--tune", action="store_true",
                    help="run the library's tiling tuner (na_tune) on the workload before the "
                         "timed regions, so they use the tuned tilings")
    ap.add_argument("--tune-report", action="store_true",
                    help="only run the tuner on the workload and print its choice and timings")
    ap.add_argument("--tune-thorough", action="store_true",
                    help="let the tuner time every candidate tiling (not only the first 64)")
    ap.add_argument("--compare-workload", choices=workloads.CONFIG_ORDER, default=None,
                    help="profiling aid: only run the fused-versus-unfused comparison on this "
                         "workload and print its row")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="counter calibration: only run 5 device-to-device copies of this many "
                         "MiB (the HBM traffic of each is known) and exit")
    args = ap.parse_args()
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 5}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on exactly one GPU; --gpus {args.gpus} is not supported",
              file=sys.stderr)
        sys.exit(2)

    import paper_2403_04690_amd as na

    na.load_library()
    dev = torch.device("cuda", 0)
    if args.compare_workload:
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        torch.cuda._sleep(1_000_000)
        s1.record()
        torch.cuda.synchronize()
        spc = s0.elapsed_time(s1) * 1e-3 / 1_000_000
        print(json.dumps(fused_vs_unfused(na, dev, spc, names=[args.compare_workload])[0]),
              flush=True)
        return
    p = workloads.CONFIGS[args.workload]
    x = workloads.make_inputs(p, seed=0, with_grad=True)
    q, k, v, g = (x[n].to(dev) for n in ("q", "k", "v", "dout"))
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[:-1], dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ks, ds, sc = p.kernel_size, p.dilation, p.softmax_scale
    cz = p.causal_axes if any(p.causal_axes) else None

    tuning = None
    if args.tune or args.tune_report:
        na.tune_clear()
        bf, bb, tms = na.tune(q, k, v, g, ks, ds, sc, causal=cz, repeats=10, out=out, lse=lse,
                              dq=dq, dk=dk, dv=dv, thorough=args.tune_thorough)
        tuning = {"forward_tiling": list(bf), "backward_tiling": list(bb),
                  "fwd_ms_tuned": round(tms[0], 5), "bwd_ms_tuned": round(tms[1], 5),
                  "fwd_ms_heuristic": round(tms[2], 5), "bwd_ms_heuristic": round(tms[3], 5),
                  "candidates": [len(na.candidate_tilings(p.extents, ks, ds, p.batch, p.heads,
                                                          p.head_dim, q.dtype, forward=f))
                                 for f in (True, False)],
                  "thorough": args.tune_thorough}
        if args.tune_report:
            print(json.dumps({"workload": p.name, **tuning}), flush=True)
            return

    def fwd():
        na.forward(q, k, v, ks, ds, sc, out=out, lse=lse, causal=cz)

    def bwd():
        na.backward(q, k, v, out, lse, g, ks, ds, sc, dq=dq, dk=dk, dv=dv, causal=cz)

    def step():
        fwd()
        bwd()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # rate of the GPU-side spin used to give the host a head start
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record()
    torch.cuda._sleep(1_000_000)
    s1.record()
    torch.cuda.synchronize()
    spin_s_per_cycle = s0.elapsed_time(s1) * 1e-3 / 1_000_000
    # host cost of enqueueing one step: 100 steps behind a GPU-side spin, so
    # that the calls only enqueue (no synchronisation inside)
    n_host = 100
    torch.cuda._sleep(int(0.05 / max(spin_s_per_cycle, 1e-12)))
    t0 = time.perf_counter()
    for _ in range(n_host):
        step()
    host_step_s = (time.perf_counter() - t0) / n_host
    torch.cuda.synchronize()

    K = args.steps
    torch.cuda.synchronize()

    def timed(fn):
        """ms per call of fn over K back-to-back calls, HIP events at the two ends only.

        A GPU-side spin long enough for the host to enqueue all K calls runs
        first (outside the events), so the GPU then executes them back to back.
        """
        head_s = min(2.0 * K * host_step_s + 1e-3, 5.0)
        torch.cuda._sleep(int(head_s / max(spin_s_per_cycle, 1e-12)))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    def median(xs):
        ys = sorted(xs)
        n = len(ys)
        return ys[n // 2] if n % 2 else 0.5 * (ys[n // 2 - 1] + ys[n // 2])

    reps = max(args.reps, 1)
    step_reps, fwd_reps, bwd_reps = [], [], []
    for _ in range(reps):
        # Timed region 1: K forward + backward steps (the whole path).
        step_reps.append(timed(step))
        # Timed region 2: K forward launches (the forward kernel's steady-state
        # duration, which the metric and the roofline use).
        fwd_reps.append(timed(fwd))
        # Timed region 3: K backward launches.
        bwd_reps.append(timed(bwd))
    step_ms, fwd_ms, bwd_ms = median(step_reps), median(fwd_reps), median(bwd_reps)

    # The same K forwards and K backwards replayed from HIP graphs (what a
    # serving loop that captures its launches would see); context only.
    def graph_ms(fn):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            fn()
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                for _ in range(K):
                    fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            g0.record()
            graph.replay()
            g1.record()
            torch.cuda.synchronize()
            ts.append(g0.elapsed_time(g1) / K)
        del graph
        return median(ts)

    fwd_graph_ms = graph_ms(fwd) if args.graphs else None
    bwd_graph_ms = graph_ms(bwd) if args.graphs else None

    # Cold forward: each launch after a write of 512 MiB (beyond L2 and the
    # 256 MiB MALL), so Q, K and V come from HBM.
    cold_ms = None
    if args.cold_launches > 0:
        flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        cold = []
        for _ in range(args.cold_launches):
            flush.fill_(1)
            c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            c0.record()
            fwd()
            c1.record()
            torch.cuda.synchronize()
            cold.append(c0.elapsed_time(c1))
        del flush
        cold_ms = median(cold)

    def head_start(per_item_s):
        head_s = min(2.0 * K * per_item_s + 1e-3, 5.0)
        torch.cuda._sleep(int(head_s / max(spin_s_per_cycle, 1e-12)))

    fwd_tflops = p.fwd_flops() / (fwd_ms * 1e-3) / 1e12
    fwd_bytes = p.fwd_bytes()
    achieved_gbs = fwd_bytes / (fwd_ms * 1e-3) / 1e9
    traffic = measured_traffic()

    result = {
        "metric": "fused NA fwd TFLOP/s and % of MFMA peak (2-D 7x7 fp16); fwd+bwd ms",
        "value": round(fwd_tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"fp16": "f16", "bf16": "bf16", "fp32": "f32"}[p.dtype],
        "data": f"synthetic: iid N(0,1) q, k, v, dO (torch CPU generator, seed 0), rounded to "
                f"{p.dtype}",
        "config": {
            "workload": p.name,
            "rank": p.rank, "batch": p.batch, "heads": p.heads, "extents": list(p.extents),
            "head_dim": p.head_dim, "kernel_size": list(p.kernel_size),
            "dilation": list(p.dilation), "causal": list(p.causal_axes),
            "step": "na_forward + na_backward",
        },
        "fwd_ms": round(fwd_ms, 5),
        "bwd_ms": round(bwd_ms, 5),
        "fwd_bwd_ms": round(step_ms, 5),
        "reps": reps,
        "fwd_ms_reps": [round(t, 5) for t in fwd_reps],
        "bwd_ms_reps": [round(t, 5) for t in bwd_reps],
        "step_ms_reps": [round(t, 5) for t in step_reps],
        "fwd_ms_cold": None if cold_ms is None else round(cold_ms, 5),
        "fwd_ms_graph": None if fwd_graph_ms is None else round(fwd_graph_ms, 5),
        "bwd_ms_graph": None if bwd_graph_ms is None else round(bwd_graph_ms, 5),
        "tuned": tuning,
        "host_enqueue_ms_per_step": round(host_step_s * 1e3, 4),
        "mfma_peak_frac": round(fwd_tflops / PEAK_FP16_TFLOPS, 5),
        "roofline": {
            "kernel": "na_fwd_kernel",
            "bound": "hbm",
            "achieved": round(achieved_gbs, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved_gbs / PEAK_HBM_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": fwd_bytes,
        },
    }
    if args.compare:
        ceil = measured_ceilings(dev)
        result["measured_ceilings"] = ceil
        result["roofline"]["frac_of_measured_copy"] = round(achieved_gbs / ceil["copy_gbs"], 4)
        result["fused_vs_unfused"] = fused_vs_unfused(na, dev, spin_s_per_cycle)
    if not args.no_cpu_baseline:
        if p.name == workloads.BENCH_WORKLOAD:
            result["mfma_bound"] = mfma_bound_forward(na, dev, head_start, host_step_s)
            if args.compare:
                mb = result["mfma_bound"]
                mb["frac_of_measured_gemm"] = round(mb["tflops"] / ceil["fp16_gemm_tflops"], 4)
        result["cpu_baseline"] = cpu_baseline(p, x, args.cpu_seconds,
                                              args.cpu_single_thread_seconds)
        if args.compare:
            result["cpu_baseline"]["per_config"] = oracle_per_config()
            result["cpu_baseline"]["nproc"] = os.cpu_count()
    print(json.dumps(result), flush=True)


# The workload whose arithmetic intensity (about 507 FLOP/B) is above the fp16
# ridge point, so the forward's fraction of MFMA peak is meaningful there; the
# 2-D 7x7 workload is HBM- and latency-bound by its shape.
MFMA_BOUND_WORKLOAD = "1d_fp16_L32768_k1023_d4"


def mfma_bound_forward(na, dev, head_start, host_step_s, launches=100, reps=5):
    """Back-to-back forward launches on the MFMA-bound workload (side measurement,
    median of reps regions of `launches` launches)."""
    p = workloads.CONFIGS[MFMA_BOUND_WORKLOAD]
    x = workloads.make_inputs(p, seed=0, with_grad=False)
    q, k, v = (x[n].to(dev) for n in ("q", "k", "v"))
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[:-1], dtype=torch.float32, device=dev)
    args = (p.kernel_size, p.dilation, p.softmax_scale)
    for _ in range(10):
        na.forward(q, k, v, *args, out=out, lse=lse)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        head_start(host_step_s)
        f0.record()
        for _ in range(launches):
            na.forward(q, k, v, *args, out=out, lse=lse)
        f1.record()
        torch.cuda.synchronize()
        times.append(f0.elapsed_time(f1) / launches)
    ms = sorted(times)[len(times) // 2]
    tflops = p.fwd_flops() / (ms * 1e-3) / 1e12
    return {"workload": p.name, "launches": launches, "reps": reps, "fwd_ms": round(ms, 5),
            "tflops": round(tflops, 2), "mfma_peak_frac": round(tflops / PEAK_FP16_TFLOPS, 4)}


if __name__ == "__main__":
    main()
