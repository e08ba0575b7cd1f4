"""Benchmark: ISJL instance-steps per second on one MI355X.

One step = one fsched_simulate call over the whole batch of the
pareto_65536x2000 workload (65,536 instances x 2,000 jobs, heavy-tailed outputs, Poisson
arrivals, B = 512, M_kv = 1,048,576, alpha = 128, affine integer step cost):
ordering, event loop, admissions, Section 5 accounting and the per-instance
metrics, with the job tables already resident in HBM.  An instance-step is one
logical step of one instance, so a step contributes sum_i T_i instance-steps.

Prints one JSON line: the metric, the simulate kernel's position against the
int32 VALU peak (algorithmic lane operations per launch over the measured launch
time) and the oracle's rate on this host's cores (all of them, and one) on a
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "instance-steps/sec (ISJL, 1 MI355X) + fraction of gfx950 VALU/LDS/HBM roofline"
UNIT = "instance-steps/s"
# gfx950: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = int32 VALU lane operations per second
PEAK_ALU = 256 * 64 * 2.4e9
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "simulate_isjl_pareto_65536x2000_hbm.md")
KERNEL_SOURCES = ["sim_kernel.hpp", "sim_common.hpp", "regsort.hpp", "wave.hpp", "sim_isjl.hip",
                  "abi.cpp"]


def kernel_sources_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_02244_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    # the compiler flags are part of what the counters measured
    with open(os.path.join(ROOT, "paper_2608_02244_amd", "buildlib.py"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per launch from the committed counter summary, or None once the
    kernel sources differ from the ones the counters were taken with."""
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    vals = dict(line.split(": ", 1) for line in text.splitlines() if ": " in line and
                line.split(": ", 1)[0] in ("traffic_bytes_per_launch", "kernel_sources_sha256"))
    if vals.get("kernel_sources_sha256", "").strip() != kernel_sources_sha256():
        return None
    return int(vals["traffic_bytes_per_launch"])


COUNTS_FILE = os.path.join(ROOT, "tests", "golden", "roofline_counts.json")


def sort_compare_exchanges(n: int) -> int:
    """Compare-exchanges of a bitonic network over NP = 2^ceil(log2 n) keys
    (at least 64): NP/2 L (L + 1) / 2 with L = log2 NP."""
    NP = 64
    while NP < n:
        NP *= 2
    L = NP.bit_length() - 1
    return (NP // 2) * L * (L + 1) // 2


def unit_counts(workload_name: str, policy: str, alpha) -> dict:
    """The per-instance event and Phase ONE counts measured with the oracle on the
    workload's first instances (tests/golden/roofline_counts.json)."""
    key = "inf" if alpha in ("inf", 2**31 - 1) else alpha
    with open(COUNTS_FILE) as fh:
        for r in json.load(fh)["runs"]:
            if (r["workload"], r["policy"], r["alpha"]) == (workload_name, policy, key):
                return r
    raise KeyError(f"no unit counts for {workload_name} {policy} alpha={alpha}")


def algorithmic_ops(workload_name: str, n_inst: int, n: int, B: int, policy: str, alpha,
                    sorted_arrivals: bool) -> float:
    """Int32 lane operations the method needs per launch, from the three work
    terms of the hot path's measurement model:
      ordering     2 per compare-exchange of a bitonic network on the n keys
                   (a min and a max); none for FCFS over arrivals in index order;
      events       each job starts once and completes once; each of these 2n
                   events passes once over the active set S: ceil(|S| / 64)
                   wave operations of 64 lanes (mean sum per instance measured);
      Phase ONE    each pack candidate Algorithm 3 visits (from o_k on) is placed
                   first-fit by one ballot per 64 workers: ceil(B / 64) wave
                   operations (mean count per instance measured).
    The measured means come from the oracle (tests/golden/make_roofline_counts.py)."""
    c = unit_counts(workload_name, policy, alpha)
    needs_sort = policy != "fcfs" or not sorted_arrivals
    per_inst = (2 * sort_compare_exchanges(n) if needs_sort else 0) \
        + 64 * c["event_wave_ops_per_instance"] \
        + 64 * ((min(B, n) + 63) // 64) * c["pack_candidates_per_instance"]
    return float(n_inst) * per_inst


def profiled_valu_busy():
    """Fraction of the launch the SIMDs spent issuing VALU instructions (from the
    committed counter summary: SQ_INSTS_VALU x 4 cycles per wave64 instruction
    over 1,024 SIMDs at 2.4 GHz, divided by the traced launch time), or None once
    the kernel sources differ from the ones the counters were taken with."""
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    vals = dict(line.split(": ", 1) for line in text.splitlines() if ": " in line)
    if vals.get("kernel_sources_sha256", "").strip() != kernel_sources_sha256():
        return None
    v = vals.get("valu_busy_fraction")
    return None if v is None else float(v)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_baseline(np, a, p, o, m_gpu, fields, kw, seconds: float) -> dict:
    """The single-threaded C oracle timed on this host's cores: on one core over
    a leading sample, and on every core this process may use (one contiguous
    shard of instances per thread, at most 16) over a larger leading sample;
    both checked against the GPU's metrics."""
    import oracle
    n_inst = a.shape[0]
    c0 = time.perf_counter()
    oracle.simulate(a[:1], p[:1], o[:1], **kw)
    one = max(time.perf_counter() - c0, 1e-4)
    k1 = int(max(1, min(n_inst, seconds / 2 / one)))
    c0 = time.perf_counter()
    ref1 = oracle.simulate(a[:k1], p[:k1], o[:k1], **kw)
    s1 = time.perf_counter() - c0
    threads = oracle.host_threads()
    kn = int(max(k1, min(n_inst, k1 * threads)))
    c0 = time.perf_counter()
    refn = oracle.simulate_parallel(a[:kn], p[:kn], o[:kn], threads=threads, chunk=8, **kw)
    sn = time.perf_counter() - c0
    parity = all(np.array_equal(refn[f], m_gpu[f][:kn]) for f in fields) and \
        all(np.array_equal(ref1[f], m_gpu[f][:k1]) for f in fields)
    return {"value": float(refn["T"].sum()) / sn, "unit": UNIT, "cores": threads,
            "kind": "oracle",
            "sample": f"first {kn} instances on {threads} threads ({sn:.1f} s); one core: "
                      f"first {k1} instances ({s1:.1f} s)",
            "value_1core": float(ref1["T"].sum()) / s1, "nproc": os.cpu_count(),
            "cpu_model": cpu_model(), "parity_on_sample": parity}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="pareto_65536x2000")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--alpha", default=None,
                    help="sweep mode: a single fairness budget (an integer or 'inf')")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the per-alpha roofline lines of the fairness-budget sweep workload")
    ap.add_argument("--mode", default="simulate",
                    choices=["simulate", "copy", "decompose", "opt", "host", "profit",
                             "gamma", "robust", "efficiency", "prefill", "sweep", "configs"],
                    help="simulate: the benchmark line; copy: a plain device copy of known size "
                         "(calibrates the HBM byte counters); decompose / opt: time the other "
                         "two library calls (for profiles); host: host-buffer calls, "
                         "PCIe copies included; profit: the linear-pricing experiment; "
                         "gamma: the competitive-ratio experiment; robust: Robust-ISJL on "
                         "predicted sizes (pareto_65536x2000 and the guarantee on tiny "
                         "instances); efficiency: throughput and AEL of every policy on the "
                         "LMSYS-shaped workload; prefill: the prefill-at-admission variant "
                         "of every policy on pareto_65536x2000; sweep: the fairness-budget "
                         "sweep alone (--alpha to pick one budget, for counter runs); "
                         "configs: every named workload under each of its policies and "
                         "budgets, GPU rate, roofline fraction and the oracle on one and on "
                         "every host core (the results table of the baseline notes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the instances are "
              "independent, so more GPUs would each take a contiguous share of them, but "
              "only the one-GPU case is implemented and measured.", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    import workload
    import paper_2608_02244_amd as fs

    if args.mode == "copy":
        return copy_calibration(torch, args.steps)
    if args.mode == "decompose":
        return time_decompose(torch, np, workload, fs, args)
    if args.mode == "opt":
        return time_opt(torch, np, workload, fs, args)
    if args.mode == "host":
        return time_host(torch, np, workload, fs, args)
    if args.mode == "profit":
        return time_profit(args)
    if args.mode == "gamma":
        return time_gamma(args)
    if args.mode == "robust":
        return time_robust(torch, np, workload, fs, args)
    if args.mode == "efficiency":
        return time_efficiency(np, workload)
    if args.mode == "prefill":
        return time_prefill(torch, np, workload, fs, args)
    if args.mode == "configs":
        return time_configs(torch, np, workload, fs, args)
    if args.mode == "sweep":
        alphas = None
        if args.alpha is not None:
            alphas = [workload.ALPHA_INF if args.alpha == "inf" else int(args.alpha)]
        res = alpha_sweep(torch, np, workload, fs, torch.cuda.current_stream(),
                          reps=max(1, args.steps), alphas=alphas)
        print(json.dumps({"mode": "sweep", **res}))
        return 0
    w = workload.WORKLOADS[args.workload]
    alpha = w.alphas[0]
    policy = "isjl"
    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    a, p, o = workload.generate(w)
    gen_s = time.perf_counter() - t0
    sorted_arrivals = bool((np.diff(a, axis=1) >= 0).all())
    ta, tp, to = (torch.from_numpy(x).to(dev) for x in (a, p, o))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    kw = dict(policy=policy, B=w.B, alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c,
              cost_tau=w.cost_tau)

    raw, _, _ = fs.simulate(ta, tp, to, **kw)
    torch.cuda.synchronize()
    m = fs.metrics_view(raw)
    if (m["T"] < 0).any():
        raise RuntimeError("some instance reported an error marker")
    inst_steps = int(m["T"].sum())

    for _ in range(args.warmup):
        fs.simulate(ta, tp, to, **kw)
    torch.cuda.synchronize()
    ev_start = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev_end = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(args.steps):
        ev_start[k].record(stream)
        fs.simulate(ta, tp, to, **kw)
        ev_end[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    launch_ms = [s.elapsed_time(e) for s, e in zip(ev_start, ev_end)]
    avg_launch_s = sum(launch_ms) / len(launch_ms) / 1e3
    ms_per_step = wall / args.steps * 1e3
    value = inst_steps * args.steps / wall

    ops = algorithmic_ops(w.name, w.n_inst, w.n_jobs, w.B, policy, alpha, sorted_arrivals)
    achieved = ops / avg_launch_s
    roofline = {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_ALU / 1e12,
                "unit": "Tops/s (int32 lane operations)", "frac": achieved / PEAK_ALU,
                "traffic": measured_traffic(), "kernel": f"simulate_kernel<ISJL> ({w.n_inst} waves)",
                "avg_launch_ms": avg_launch_s * 1e3, "ops_per_launch": ops,
                "valu_busy_profiled": profiled_valu_busy()}

    out = {"metric": METRIC, "value": value, "unit": UNIT, "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
           "config": {"workload": w.name, "policy": policy, "n_inst": w.n_inst,
                      "n_jobs": w.n_jobs, "B": w.B, "alpha": alpha, "M_kv": w.M_kv,
                      "cost_c": w.cost_c, "cost_tau": w.cost_tau,
                      "instance_steps_per_step": inst_steps, "generate_s": round(gen_s, 3)},
           "roofline": roofline}

    if not args.no_sweep:
        out["alpha_sweep"] = alpha_sweep(torch, np, workload, fs, stream)

    if not args.no_cpu_baseline:
        kw_o = dict(policy=policy, B=w.B, alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c,
                    cost_tau=w.cost_tau)
        out["cpu_baseline"] = oracle_baseline(np, a, p, o, m, fs.METRIC_FIELDS, kw_o,
                                              args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


def _median_launch_ms(torch, fn, reps: int = 5) -> float:
    stream = torch.cuda.current_stream()
    fn()
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    return sorted(ms)[len(ms) // 2]


def time_configs(torch, np, workload, fs, args) -> int:
    """Every named workload of the benchmark target under each of its policies
    and fairness budgets: the sum of makespans, GPU instance-steps/s (HIP events,
    median of 5 launches over the whole table in HBM), the fraction of the ALU
    roofline under the three-term operation count, and the oracle's rate on one
    core and on every host core (leading samples, checked against the GPU)."""
    import oracle
    INF = workload.ALPHA_INF
    plan = [("uniform_256x64", [("fcfs", INF), ("ljf", 8), ("isjl", 8)]),
            ("lognormal_4096x1000", [("fcfs", INF), ("ljf", 64), ("isjl", 64)]),
            ("bimodal_sweep_4096x2000", [("isjl", al) for al in (0, 16, 64, 256, 1024, INF)]
             + [("fcfs", INF), ("ljf", 64)]),
            ("pareto_65536x2000", [("isjl", 128)])]
    rows = []
    threads = oracle.host_threads()
    secs = max(0.5, args.cpu_seconds / 8)
    for name, runs in plan:
        w = workload.WORKLOADS[name]
        a, p, o = workload.generate(w)
        sorted_arrivals = bool((np.diff(a, axis=1) >= 0).all())
        ta, tp, to = (torch.from_numpy(x).to("cuda:0") for x in (a, p, o))
        for pol, al in runs:
            kw = dict(policy=pol, B=w.B, alpha=al, M_kv=w.M_kv, cost_c=w.cost_c,
                      cost_tau=w.cost_tau)
            raw, _, _ = fs.simulate(ta, tp, to, **kw)
            torch.cuda.synchronize()
            m = fs.metrics_view(raw).copy()
            if (m["T"] < 0).any():
                raise RuntimeError(f"{name} {pol}: error marker")
            steps = int(m["T"].sum())
            ms = _median_launch_ms(torch, lambda: fs.simulate(ta, tp, to, **kw))
            try:
                ops = algorithmic_ops(name, w.n_inst, w.n_jobs, w.B, pol, al, sorted_arrivals)
                frac = ops / (ms / 1e3) / PEAK_ALU
            except KeyError:
                ops = frac = None
            cpu = oracle_baseline(np, a, p, o, m, fs.METRIC_FIELDS, kw, secs)
            row = {"workload": name, "policy": pol, "alpha": "inf" if al == INF else al,
                   "sum_T": steps, "gpu_ms": ms, "gpu_instance_steps_per_s": steps / (ms / 1e3),
                   "alu_frac": frac, "ops_per_launch": ops,
                   "oracle_1core": cpu["value_1core"], "oracle_all_cores": cpu["value"],
                   "oracle_threads": threads, "parity_on_samples": cpu["parity_on_sample"]}
            print(json.dumps(row), file=sys.stderr, flush=True)
            rows.append(row)
        del ta, tp, to
        torch.cuda.empty_cache()
    # the tiny workload: ISJL and the exact optimum for every (alpha, KV budget)
    w = workload.WORKLOADS["tiny_opt_1048576x8"]
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to("cuda:0") for x in (a, p, o))
    from fractions import Fraction
    for M in (w.M_kv, 0):
        for al in w.alphas:
            kw = dict(B=w.B, alpha=al, M_kv=M)
            raw, _, _ = fs.simulate(ta, tp, to, policy="isjl", cost_c=0, cost_tau=1, **kw)
            torch.cuda.synchronize()
            Ti = fs.metrics_view(raw)["T"].copy()
            ms_sim = _median_launch_ms(torch, lambda: fs.simulate(ta, tp, to, policy="isjl",
                                                                  **kw))
            To, _ = fs.bruteforce_opt(ta, tp, to, **kw)
            torch.cuda.synchronize()
            To = To.cpu().numpy()
            t0 = time.perf_counter()
            fs.bruteforce_opt(ta, tp, to, **kw)
            torch.cuda.synchronize()
            s_opt = time.perf_counter() - t0
            # makespans are below 2^8 here, so distinct ratios differ by far more than
            # a double's rounding: the argmin of the doubles is an exact minimum
            k = int(np.argmin(To / Ti))
            worst = Fraction(int(To[k]), int(Ti[k]))
            c0 = time.perf_counter()
            oracle.opt(a[:64], p[:64], o[:64], **kw)
            one = max((time.perf_counter() - c0) / 64, 1e-6)
            k1 = int(max(64, secs / 2 / one))
            c0 = time.perf_counter()
            r1 = oracle.opt(a[:k1], p[:k1], o[:k1], **kw)
            s1 = time.perf_counter() - c0
            kn = k1 * threads
            c0 = time.perf_counter()
            rn = oracle.opt_parallel(a[:kn], p[:kn], o[:kn], threads=threads, **kw)
            sn = time.perf_counter() - c0
            row = {"workload": w.name, "policy": "isjl+opt", "alpha": al, "M_kv": M,
                   "sum_T_isjl": int(Ti.sum()), "gpu_isjl_instance_steps_per_s":
                   float(Ti.sum()) / (ms_sim / 1e3), "gpu_opt_solves_per_s": w.n_inst / s_opt,
                   "oracle_opt_1core_solves_per_s": k1 / s1,
                   "oracle_opt_all_cores_solves_per_s": kn / sn, "oracle_threads": threads,
                   "min_T_opt_over_T_isjl": f"{worst.numerator}/{worst.denominator}",
                   "parity_on_samples": bool((r1 == To[:k1]).all() and (rn == To[:kn]).all())}
            print(json.dumps(row), file=sys.stderr, flush=True)
            rows.append(row)
    print(json.dumps({"mode": "configs", "cpu_model": cpu_model(), "nproc": os.cpu_count(),
                      "rows": rows}))
    return 0


def alpha_sweep(torch, np, workload, fs, stream, reps: int = 5, alphas=None) -> dict:
    """ISJL over the fairness-budget sweep workload (4,096 instances x 2,000 jobs,
    B = 128, M_kv = 262,144), one launch per alpha: instance-steps/s and the
    fraction of the ALU roofline, kernel time from HIP events (median of reps)."""
    w = workload.WORKLOADS["bimodal_sweep_4096x2000"]
    a, p, o = workload.generate(w)
    sorted_arrivals = bool((np.diff(a, axis=1) >= 0).all())
    ta, tp, to = (torch.from_numpy(x).to("cuda:0") for x in (a, p, o))
    rows = []
    for al in (w.alphas if alphas is None else alphas):
        ops = algorithmic_ops(w.name, w.n_inst, w.n_jobs, w.B, "isjl", al, sorted_arrivals)
        kw = dict(policy="isjl", B=w.B, alpha=al, M_kv=w.M_kv, cost_c=w.cost_c,
                  cost_tau=w.cost_tau)
        raw, _, _ = fs.simulate(ta, tp, to, **kw)
        torch.cuda.synchronize()
        steps = int(fs.metrics_view(raw)["T"].sum())
        ms = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fs.simulate(ta, tp, to, **kw)
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        t = sorted(ms)[len(ms) // 2] / 1e3
        rows.append({"alpha": "inf" if al == workload.ALPHA_INF else al, "ms": t * 1e3,
                     "instance_steps_per_s": steps / t, "ops_per_launch": ops,
                     "frac": ops / t / PEAK_ALU})
    return {"workload": w.name, "policy": "isjl", "B": w.B, "M_kv": w.M_kv,
            "bound": "alu", "results": rows}


def time_host(torch, np, workload, fs, args) -> int:
    """Host-buffer calls (the library stages the tables to the device and the
    metrics back): end-to-end rate including the PCIe copies."""
    w = workload.WORKLOADS[args.workload]
    a, p, o = workload.generate(w)
    kw = dict(policy="isjl", B=w.B, alpha=w.alphas[0], M_kv=w.M_kv, cost_c=w.cost_c,
              cost_tau=w.cost_tau)
    raw, _, _ = fs.simulate(a, p, o, **kw)
    steps = int(fs.metrics_view(raw)["T"].sum())
    for _ in range(args.warmup):
        fs.simulate(a, p, o, **kw)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        fs.simulate(a, p, o, **kw)
    dt = (time.perf_counter() - t0) / args.steps
    print(json.dumps({"mode": "host", "workload": w.name, "ms_per_call": dt * 1e3,
                      "instance_steps_per_s": steps / dt,
                      "table_bytes": int(a.nbytes + p.nbytes + o.nbytes)}))
    return 0


def time_profit(args) -> int:
    """The linear-pricing experiment (profit and cost decomposition, break-even
    overhead): 5 replications x 9 policies through the library, timed."""
    from paper_2608_02244_amd import profit
    profit.run_table(profit.gpu_simulate, replications=1)  # warm-up
    t0 = time.perf_counter()
    res = profit.run_table(profit.gpu_simulate, replications=5)
    dt = time.perf_counter() - t0
    # calibration replay of the fairness-budget sweep workload (4,096 x 2,000,
    # B = 128, M_kv = 262,144) on a grid alpha = delta * Q / O
    import workload
    w = workload.WORKLOADS["bimodal_sweep_4096x2000"]
    a, p, o = workload.generate(w)
    deltas = (0.0, 0.01, 0.02, 0.05, 0.1, 0.2, 0.5, 1.0)
    profit.calibrate_alpha(profit.gpu_simulate_batch, a[:64], p[:64], o[:64], deltas[:2],
                           B=w.B, M_kv=w.M_kv)  # warm-up
    t1 = time.perf_counter()
    cal = profit.calibrate_alpha(profit.gpu_simulate_batch, a, p, o, deltas, B=w.B,
                                 M_kv=w.M_kv, c=w.cost_c * 1e-6, tau=w.cost_tau * 1e-6)
    dcal = time.perf_counter() - t1
    print(json.dumps({"mode": "profit", "seconds": dt, "calls": 45,
                      "table": res["table"], "breakeven": {str(k): v for k, v in
                                                           res["breakeven"].items()},
                      "calibration": {"workload": w.name, "seconds": dcal, **cal}}))
    return 0


def time_gamma(args) -> int:
    """Exact optimum against ISJL over the tiny workload, B = 2, alpha = 1..19,
    binned by gamma = alpha / o_1, with beta = alpha and with beta*."""
    import workload
    from paper_2608_02244_amd import gamma_curve as gc
    n = 262144
    a, p, o = workload.generate("tiny_opt_1048576x8", n_inst=n)
    alphas = list(range(1, 20))
    out = {"mode": "gamma", "workload": "tiny_opt_1048576x8", "instances": n, "alphas": alphas}
    for bs in (False, True):
        t0 = time.perf_counter()
        res = gc.run(gc.gpu_pair, a, p, o, alphas, B=2, beta_star=bs)
        out["beta_star" if bs else "beta_alpha"] = {"seconds": time.perf_counter() - t0,
                                                    **gc.to_json(res)}
    print(json.dumps(out))
    return 0


def time_robust(torch, np, workload, fs, args) -> int:
    """Robust-ISJL: (1) the benchmark workload with upper bounds u = o + U * slack * o
    at several slacks, timed like the benchmark line, against ISJL on the true
    sizes (makespan and cost ratios, fairness); (2) the guarantee
    T_R <= 4/3 (T_OPT + Delta_pack), its corollary and the proof's first step on
    tiny offline instances."""
    from paper_2608_02244_amd import robust as rb
    w = workload.WORKLOADS[args.workload]
    alpha = w.alphas[0]
    dev = torch.device("cuda:0")
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to(dev) for x in (a, p, o))
    kw = dict(B=w.B, alpha=alpha, M_kv=w.M_kv, cost_c=w.cost_c, cost_tau=w.cost_tau)
    stream = torch.cuda.current_stream()
    base = fs.metrics_view(fs.simulate(ta, tp, to, policy="isjl", **kw)[0])
    rows = []
    for slack in (0.0, 0.25, 1.0, 3.0):
        tu = torch.from_numpy(workload.prediction_upper(o, slack, seed=1)).to(dev)
        m = fs.metrics_view(fs.simulate_robust(ta, tp, to, tu, **kw)[0])
        if (m["T"] < 0).any():
            raise RuntimeError("some instance reported an error marker")
        for _ in range(args.warmup):
            fs.simulate_robust(ta, tp, to, tu, **kw)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            fs.simulate_robust(ta, tp, to, tu, **kw)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        print(f"robust {w.name} slack={slack}: {ms:.2f} ms", file=sys.stderr, flush=True)
        rows.append({"slack": slack, "ms_per_launch": ms,
                     "instance_steps_per_s": float(m["T"].sum()) / (ms / 1e3),
                     "T_over_isjl": float(m["T"].sum() / base["T"].sum()),
                     "C_over_isjl": float(m["C"].sum() / base["C"].sum()),
                     "latency_over_isjl": float(m["sum_latency"].sum() /
                                                base["sum_latency"].sum()),
                     "unfair_steps": int(m["unfair_steps"].sum()),
                     "max_extent": int(m["max_extent"].max())})
        del tu
    out = {"mode": "robust", "workload": w.name, "alpha": alpha, "full_size": rows}
    # the exhaustive optimum gets much slower with B, so fewer instances there
    tiny = []
    for B, n in ((2, 32768), (3, 4096), (4, 1024)):
        a, p, o = workload.generate("tiny_opt_1048576x8", n_inst=n)
        for slack in (0.25, 1.0, 3.0):
            u = workload.prediction_upper(o, slack, seed=5)
            rows = []
            for al in (1, 2, 4, 7, 11):
                t0 = time.perf_counter()
                rows += rb.run(rb.gpu_quad, a, p, o, u, [al], B=B)["rows"]
                rows[-1]["seconds"] = time.perf_counter() - t0
                print(f"robust tiny B={B} n={n} slack={slack} alpha={al}: "
                      f"{rows[-1]['seconds']:.1f} s", file=sys.stderr, flush=True)
            tiny.append({"B": B, "instances": n, "slack": slack, "rows": rows})
    out["tiny"] = {"workload": "tiny_opt_1048576x8", "runs": tiny}
    print(json.dumps(out))
    return 0


def time_efficiency(np, workload) -> int:
    """Throughput and AEL of FCFS, SJF, LJF, ISJL(50/100/150) at B = 16 and 32 on
    the 256 instances of the LMSYS-shaped workload, with its Poisson releases and
    with every request released at step 0."""
    from paper_2608_02244_amd import efficiency as ef
    a, p, o = workload.generate("lmsys_shaped_256x2000")
    out = {"mode": "efficiency", "workload": "lmsys_shaped_256x2000"}
    ef.run_table(ef.gpu_simulate, a[:8], p[:8], o[:8], Bs=(16,))  # warm-up
    resume = lambda *x: ef.gpu_simulate(*x, resume_fill=True)  # noqa: E731
    for name, arr, sim in (("poisson", a, ef.gpu_simulate), ("offline", np.zeros_like(a),
                                                              ef.gpu_simulate),
                           ("poisson_resume_fill", a, resume),
                           ("offline_resume_fill", np.zeros_like(a), resume)):
        t0 = time.perf_counter()
        tab = ef.run_table(sim, arr, p, o)
        out[name] = {"seconds": time.perf_counter() - t0, "table": {str(B): r for B, r in
                                                                    tab.items()},
                     "markdown": ef.format_table(tab)}
        print(f"efficiency {name}: {out[name]['seconds']:.2f} s", file=sys.stderr, flush=True)
    print(json.dumps(out))
    return 0


def time_prefill(torch, np, workload, fs, args) -> int:
    """Every policy in the prefill-at-admission variant on the benchmark workload
    (the prompt is processed at admission, a job runs its output tokens), timed
    with HIP events, beside ISJL in the chunked reading."""
    w = workload.WORKLOADS[args.workload]
    alpha = w.alphas[0]
    dev = torch.device("cuda:0")
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to(dev) for x in (a, p, o))
    stream = torch.cuda.current_stream()
    rows = []
    for pol, pre in (("isjl", False), ("isjl", True), ("ljf", True), ("fcfs", True),
                     ("sjf", True)):
        kw = dict(policy=pol, B=w.B, alpha=alpha if pol in ("isjl", "ljf") else fs.ALPHA_INF,
                  M_kv=w.M_kv, cost_c=w.cost_c, cost_tau=w.cost_tau, prefill=pre)
        m = fs.metrics_view(fs.simulate(ta, tp, to, **kw)[0])
        if (m["T"] < 0).any():
            raise RuntimeError("some instance reported an error marker")
        for _ in range(args.warmup):
            fs.simulate(ta, tp, to, **kw)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            fs.simulate(ta, tp, to, **kw)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        print(f"prefill={pre} {pol}: {ms:.2f} ms", file=sys.stderr, flush=True)
        rows.append({"policy": pol, "prefill": pre, "ms_per_launch": ms,
                     "instance_steps_per_s": float(m["T"].sum()) / (ms / 1e3),
                     "mean_T": float(m["T"].mean()),
                     "tokens_per_step": float(m["O"].sum() / m["T"].sum()),
                     "mean_latency": float(m["sum_latency"].sum() / m["T"].size / w.n_jobs),
                     "W_over_T": float(m["W"].sum() / m["T"].sum()),
                     "unfair_steps": int(m["unfair_steps"].sum())})
    print(json.dumps({"mode": "prefill", "workload": w.name, "alpha": alpha, "rows": rows}))
    return 0


def copy_calibration(torch, steps: int) -> int:
    """A plain device-to-device copy of 1 GiB: 1 GiB read and 1 GiB written per
    dispatch, the reference for the FETCH_SIZE / WRITE_SIZE counters."""
    n = 1 << 28
    x = torch.arange(n, dtype=torch.int32, device="cuda:0")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(max(1, steps)):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"mode": "copy", "bytes_read_per_dispatch": 4 * n,
                      "bytes_written_per_dispatch": 4 * n, "dispatches": max(1, steps)}))
    return 0


def time_decompose(torch, np, workload, fs, args) -> int:
    """Re-score the ISJL schedules of the benchmark workload (fsched_cost_decompose)."""
    w = workload.WORKLOADS[args.workload]
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to("cuda:0") for x in (a, p, o))
    kw = dict(B=w.B, alpha=w.alphas[0], M_kv=w.M_kv, cost_c=w.cost_c, cost_tau=w.cost_tau)
    raw, st, _ = fs.simulate(ta, tp, to, policy="isjl", schedule=True, **kw)
    torch.cuda.synchronize()
    steps_per_call = int(fs.metrics_view(raw)["T"].sum())
    for _ in range(args.warmup):
        fs.cost_decompose(ta, tp, to, st, **kw)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        fs.cost_decompose(ta, tp, to, st, **kw)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / args.steps
    # algorithmic work: sorting the 2n start/end events (2 lane-ops per
    # compare-exchange of a bitonic network) and O(1) per event for the state
    # scans and span terms (4 lane-ops)
    NP2 = 64
    while NP2 < 2 * w.n_jobs:
        NP2 *= 2
    L = NP2.bit_length() - 1
    ops = float(w.n_inst) * (2 * (NP2 // 2) * L * (L + 1) // 2 + 4 * 2 * w.n_jobs)
    out = {"mode": "decompose", "workload": w.name, "ms_per_call": dt * 1e3,
           "instance_steps_per_s": steps_per_call / dt,
           "roofline": {"bound": "alu", "achieved": ops / dt / 1e12, "peak": PEAK_ALU / 1e12,
                        "frac": ops / dt / PEAK_ALU, "ops_per_launch": ops}}
    if not args.no_cpu_baseline:
        # the oracle's re-scorer on a bounded sample of the same schedules
        import oracle
        s_host = st.cpu().numpy()
        T = fs.metrics_view(raw)["T"]
        c0 = time.perf_counter()
        oracle.decompose(a[:1], p[:1], o[:1], s_host[:1], **kw)
        one = max(time.perf_counter() - c0, 1e-4)
        k = int(max(1, min(w.n_inst, args.cpu_seconds / 3 / one)))
        c0 = time.perf_counter()
        ref, _ = oracle.decompose(a[:k], p[:k], o[:k], s_host[:k], **kw)
        cpu_s = time.perf_counter() - c0
        out["cpu_baseline"] = {"value": float(T[:k].sum()) / cpu_s, "unit": "instance-steps/s",
                               "cores": 1, "kind": "oracle",
                               "sample": f"first {k} of {w.n_inst} schedules, {cpu_s:.1f} s",
                               "parity_on_sample": bool((ref["T"] == T[:k]).all())}
    print(json.dumps(out))
    return 0


def time_opt(torch, np, workload, fs, args) -> int:
    """Exact optima of the tiny adversarial workload (fsched_bruteforce_opt), one
    (alpha, M_kv) setting per call over every instance."""
    w = workload.WORKLOADS["tiny_opt_1048576x8"]
    a, p, o = workload.generate(w)
    ta, tp, to = (torch.from_numpy(x).to("cuda:0") for x in (a, p, o))
    res = {}
    for M in (w.M_kv, 0):
        for al in w.alphas:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(max(1, args.steps)):
                fs.bruteforce_opt(ta, tp, to, B=w.B, alpha=al, M_kv=M)
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t0) / max(1, args.steps)
            res[f"M_kv={M},alpha={al}"] = {"s_per_call": dt, "solves_per_s": w.n_inst / dt}
    out = {"mode": "opt", "workload": w.name, "results": res}
    if not args.no_cpu_baseline:
        # the oracle's exhaustive optimum on a bounded sample (first setting)
        import oracle
        al, M = w.alphas[0], w.M_kv
        c0 = time.perf_counter()
        oracle.opt(a[:64], p[:64], o[:64], B=w.B, alpha=al, M_kv=M)
        one = max((time.perf_counter() - c0) / 64, 1e-6)
        k = int(max(64, min(w.n_inst, args.cpu_seconds / 3 / one)))
        c0 = time.perf_counter()
        ref = oracle.opt(a[:k], p[:k], o[:k], B=w.B, alpha=al, M_kv=M)
        cpu_s = time.perf_counter() - c0
        T_gpu, _ = fs.bruteforce_opt(ta[:k], tp[:k], to[:k], B=w.B, alpha=al, M_kv=M)
        out["cpu_baseline"] = {"value": k / cpu_s, "unit": "exact solves/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"first {k} instances, M_kv={M}, alpha={al}, "
                                         f"{cpu_s:.1f} s",
                               "parity_on_sample": bool((T_gpu.cpu().numpy() == ref).all())}
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
