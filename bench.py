#!/usr/bin/env python3
"""Dion2 optimizer-step benchmark on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload 1b] [--alpha 0.25]

A step is one Dion2 update (Algorithm 1) of every matrix of a synthetic layer
stack with W, M, G resident in HBM: one batched call per same-shape group,
each on its own stream (forked from and joined into the timing stream), or
back to back on one stream with --streams 0. --calls grouped makes it one
dion2_step_groups call for the whole stack instead. The default is the paper's timing method
(Sec. 4.4): 100 steps, the mean of the final 20 reported (warmup 80,
steps 20). Prints one JSON line:
  value        mean ms per step at --alpha (lower is better)
  roofline     the dominant kernel phase against its roofline, measured with
               HIP events on the library's stream in a second timed pass
  cpu_baseline the CPU oracle timed on a bounded sample of the same stack
  per_alpha_ms the other fractions of the workload, timed the same way
  per_rule_ms  the l1 (Default) and Random selection rules at --alpha
  per_chain_ms the GRAM chain's storage: bf16 hi/lo pairs (the default) and
               the opt-in scaled fp16 (ns_chain), at every fraction
  per_master_ms X rounded once to bf16 (the default) against the opt-in fp32
               master (ns_master), at every fraction
"""
from __future__ import annotations

import argparse
import dataclasses
import glob
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import torch  # noqa: E402

from paper_2512_16928_amd import binding, profsum, workloads  # noqa: E402

METRIC = "Dion2 optimizer-step ms per layer stack at α=0.25/0.5/1; NS MFMA util %"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFS = 2500.0    # MI355X dense bf16 MFMA
RIDGE_FLOP_PER_BYTE = MFMA_BF16_PEAK_TFS * 1e12 / (HBM_PEAK_GBS * 1e9)
NS_PHASES = ("ns_gram", "ns_poly", "ns_update")
STREAMING_PHASES = ("momentum", "gather", "apply")


def mfma_per_alpha(workload, per_alpha, profiled):
    """{alpha: {phase: counter figures}} from the committed MFMA summaries, for
    the selection fractions this run timed (default Newton-Schulz settings only)."""
    out = {}
    if not profiled:
        return out
    paths = sorted(glob.glob(os.path.join(ROOT, "profiles", "*mfma*.txt")))
    for a in per_alpha:
        for p in NS_PHASES:
            for path in paths:
                hit = profsum.lookup_mfma(path, p, workload, float(a))
                if hit:
                    out.setdefault(a, {})[p] = {"mfma_util_pct": hit["mfma_util_pct"],
                                                "frac_of_peak": hit["frac_of_peak"]}
                    break
    return out


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def allocate(wl, dev, split=1):
    """The stack's tensors, one entry per library call: each shape group, or
    each of `split` equal sub-batches of it (views of the same storage)."""
    groups = []
    for gi, grp in enumerate(wl.groups):
        W, M, G = workloads.make_group(wl, gi, dev)
        n = max(1, min(split, grp.count))
        bounds = [grp.count * i // n for i in range(n + 1)]
        for lo, hi in zip(bounds[:-1], bounds[1:]):
            groups.append((grp, W[lo:hi], M[lo:hi], G[lo:hi]))
    torch.cuda.synchronize()
    return groups


NS_FORMS = {"auto": binding.NS_AUTO, "direct": binding.NS_DIRECT, "gram": binding.NS_GRAM}
SELECT_RULES = {"l1": binding.SELECT_L1, "random": binding.SELECT_RANDOM}
NS_FORM = binding.NS_AUTO
NS_CHAINS = {"hilo": binding.CHAIN_HILO, "f16": binding.CHAIN_F16}
NS_CHAIN = binding.CHAIN_HILO
NS_MASTERS = {"bf16": binding.MASTER_BF16, "fp32": binding.MASTER_FP32}
NS_MASTER = binding.MASTER_BF16
STEP = [0]      # optimizer step counter (the Random rule draws anew every step)
STREAMS = []    # one stream per shape group when the groups run concurrently
GROUPED = [False]   # one dion2_step_groups call for the whole stack
GROUP_STREAMS = [0]  # streams the grouped call may spread its groups over (0: library's choice)


def one_step(wl, groups, alpha, rule=binding.SELECT_L1):
    """One optimizer step over the whole stack: one library call per shape
    group. The groups are independent, so with STREAMS set each runs on its
    own stream (forked from and joined back into the current stream)."""
    STEP[0] += 1
    if GROUPED[0]:
        binding.dion2_step_groups([(W, M, G, grp.axis) for grp, W, M, G in groups], alpha, wl.mu,
                                  wl.lr, wl.ns_steps, ns_form=NS_FORM, select_rule=rule,
                                  rand_seed=1234, rand_step=STEP[0], rand_matrix0=0,
                                  group_streams=GROUP_STREAMS[0], ns_chain=NS_CHAIN,
                                  ns_master=NS_MASTER)
        return
    first = 0
    main = torch.cuda.current_stream()
    if STREAMS:
        fork = torch.cuda.Event()
        fork.record(main)
    for gi, (grp, W, M, G) in enumerate(groups):
        s = STREAMS[gi % len(STREAMS)] if STREAMS else main
        if STREAMS:
            s.wait_event(fork)
        with torch.cuda.stream(s):
            if (NS_FORM == binding.NS_AUTO and NS_CHAIN == binding.CHAIN_HILO
                    and NS_MASTER == binding.MASTER_BF16 and rule == binding.SELECT_L1):
                binding.dion2_step_strided(W, M, G, alpha, wl.mu, wl.lr, wl.ns_steps, grp.axis)
            else:
                binding.dion2_step_ex(W, M, G, alpha, wl.mu, wl.lr, wl.ns_steps, grp.axis,
                                      ns_form=NS_FORM, select_rule=rule, rand_seed=1234,
                                      rand_step=STEP[0], rand_matrix0=first, ns_chain=NS_CHAIN,
                                      ns_master=NS_MASTER)
        first += W.shape[0]
    for s in STREAMS:
        join = torch.cuda.Event()
        join.record(s)
        main.wait_event(join)


def time_steps(wl, groups, alpha, warmup, steps, rule=binding.SELECT_L1):
    for _ in range(warmup):
        one_step(wl, groups, alpha, rule)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(steps):
        one_step(wl, groups, alpha, rule)
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return per, wall


def profile_phases(wl, groups, alpha, steps):
    """Per-phase kernel time from events the library records around each
    launch on its stream, with the phase's algorithmic work. The groups run
    back to back here (one stream), so each phase is timed without other work
    beside it."""
    saved, saved_gs = STREAMS[:], GROUP_STREAMS[0]
    STREAMS.clear()
    GROUP_STREAMS[0] = 1
    binding.dion2_profile_reset()
    binding.dion2_profile_enable(True)
    try:
        for _ in range(steps):
            one_step(wl, groups, alpha)
        torch.cuda.synchronize()
        prof = binding.dion2_profile_read()
    finally:
        binding.dion2_profile_enable(False)
        STREAMS.extend(saved)
        GROUP_STREAMS[0] = saved_gs
    out = {}
    for ph, d in prof.items():
        if d["launches"] == 0:
            continue
        avg_ms = d["ms"] / d["launches"]       # per kernel launch
        flops, nbytes = d["flops"] / d["launches"], d["bytes"] / d["launches"]
        sec = avg_ms * 1e-3
        # the bound is the roofline's: MFMA where the phase's arithmetic
        # intensity reaches the ridge point, HBM below it
        if ph == "select":
            bound, ach, peak, unit = "latency", nbytes / sec / 1e9, HBM_PEAK_GBS, "GB/s"
        elif flops > 0 and flops / nbytes >= RIDGE_FLOP_PER_BYTE:
            bound, ach, peak, unit = "mfma", flops / sec / 1e12, MFMA_BF16_PEAK_TFS, "TFLOP/s"
        else:
            bound, ach, peak, unit = "hbm", nbytes / sec / 1e9, HBM_PEAK_GBS, "GB/s"
        out[ph] = dict(total_ms_per_step=d["ms"] / steps, avg_launch_ms=avg_ms,
                       launches_per_step=d["launches"] / steps, flops_per_launch=flops,
                       bytes_per_launch=nbytes, achieved=ach, peak=peak, unit=unit, bound=bound,
                       frac=ach / peak,
                       mfma_tflops=flops / sec / 1e12, hbm_gbs=nbytes / sec / 1e9)
    return out


def cpu_baseline(wl, alpha, seconds):
    """The oracle on a bounded sample: one matrix of each shape group per
    pass, repeated until `seconds` of CPU time have run, then scaled by the
    group counts to a whole-stack step."""
    import numpy as np

    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover - threadpoolctl is optional
        blas_threads = None
    dev = torch.device("cuda:0")
    per_group = [[] for _ in wl.groups]
    t_end = time.perf_counter() + seconds
    passes = 0
    while passes == 0 or time.perf_counter() < t_end:
        for gi, grp in enumerate(wl.groups):
            idx = passes % grp.count
            W, M, G = workloads.make_group(wl, gi, dev, first=idx, count=1)
            Wh = W[0].float().cpu().numpy().astype(np.float64)
            Mh = M[0].cpu().numpy()
            Gh = G[0].float().cpu().numpy()
            t0 = time.perf_counter()
            oracle.dion2_step(Wh, Mh, Gh, alpha, wl.mu, wl.lr, wl.ns_steps, grp.axis,
                              w_dtype=wl.w_dtype)
            per_group[gi].append(time.perf_counter() - t0)
        passes += 1
    est_s = sum(statistics.mean(t) * grp.count for t, grp in zip(per_group, wl.groups))
    cores = len(os.sched_getaffinity(0))
    return dict(value=est_s * 1e3, unit="ms", cores=blas_threads or cores, kind="oracle",
                host_cores=cores,
                sample=(f"{passes} pass(es) over one matrix of each of the {len(wl.groups)} "
                        f"shape groups ({sum(len(t) for t in per_group)} oracle steps, "
                        f"{sum(sum(t) for t in per_group):.1f} s), mean per group scaled by "
                        f"the group counts to the {wl.matrices()}-matrix stack"))


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=80)
    ap.add_argument("--workload", default="1b", choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--alpha", type=float, default=None,
                    help="selection fraction of the headline number (default: the workload's first)")
    ap.add_argument("--no-extra-alphas", action="store_true",
                    help="time only --alpha, not the workload's other fractions")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel event pass")
    ap.add_argument("--ns-form", default="auto", choices=sorted(NS_FORMS),
                    help="Newton-Schulz evaluation order (default: chosen by shape)")
    ap.add_argument("--ns-chain", default="hilo", choices=sorted(NS_CHAINS),
                    help="storage of the GRAM form's s x s matrices: bf16 hi/lo pairs "
                         "(default) or scaled fp16 (one MFMA pass per product, less "
                         "accurate on ill-conditioned inputs)")
    ap.add_argument("--ns-master", default="bf16", choices=sorted(NS_MASTERS),
                    help="X rounded once to bf16 (default), or kept as a bf16 hi/lo pair through "
                         "every product (fp32; runs in the GRAM order)")
    ap.add_argument("--ns-steps", type=int, default=None,
                    help="Newton-Schulz steps (default: the workload's, 5)")
    ap.add_argument("--split", type=int, default=1,
                    help="issue each shape group as this many sub-batch calls")
    ap.add_argument("--streams", type=int, default=-1,
                    help="run the shape groups on this many streams (0: all on the current "
                         "stream; default: one stream per group, the groups being independent)")
    ap.add_argument("--calls", default="per-group", choices=("grouped", "per-group"),
                    help="one dion2_step_groups call for the whole stack (groups of one padded "
                         "Newton-Schulz size share their s x s chain), or one call per shape "
                         "group on its own stream")
    ap.add_argument("--group-streams", type=int, default=0,
                    help="with --calls grouped: streams the library may spread the groups over "
                         "(0: its choice, 1: all on one stream)")
    ap.add_argument("--no-chain-compare", action="store_true",
                    help="skip timing the other GRAM chain storage (--ns-chain) at each fraction")
    ap.add_argument("--no-random-rule", action="store_true",
                    help="skip timing the Random selection rule at --alpha")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run plain 1 GiB device copies, the reference dispatches that "
                         "scale HBM byte counters (FETCH_SIZE / WRITE_SIZE) in a profiler run")
    args = ap.parse_args(argv)
    global NS_FORM, NS_CHAIN, NS_MASTER
    NS_FORM = NS_FORMS[args.ns_form]
    NS_CHAIN = NS_CHAINS[args.ns_chain]
    NS_MASTER = NS_MASTERS[args.ns_master]

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures the Dion2 step on one GPU only: there is no multi-GPU path "
              "(every matrix's step is independent, so several GPUs would each own whole "
              "shape groups); run it without --gpus or with --gpus 1.", file=sys.stderr)
        return 2
    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        return 2
    if not os.path.exists(binding.LIB_PATH):
        from paper_2512_16928_amd import build
        build.build()
    binding.load()

    if args.copy_calibration:
        # one elementwise kernel per copy (a device-to-device copy_ splits
        # into many smaller dispatches): 1 GiB read, 1 GiB written
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda:0").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log("[bench] ran 3 plain 1 GiB copies (torch.neg) for counter calibration")

    wl = workloads.WORKLOADS[args.workload]
    if args.ns_steps is not None:
        wl = dataclasses.replace(wl, ns_steps=args.ns_steps)
    alpha = args.alpha if args.alpha is not None else wl.alphas[0]
    GROUPED[0] = args.calls == "grouped"
    GROUP_STREAMS[0] = args.group_streams
    if GROUPED[0]:
        args.streams = 0
    if args.streams < 0:
        args.streams = len(wl.groups) * max(1, args.split)
    STREAMS.extend(torch.cuda.Stream() for _ in range(args.streams))   # default priority
    dev = torch.device("cuda:0")
    log(f"[bench] allocating workload {wl.name}: {wl.matrices()} matrices, "
        f"{wl.elements() / 1e6:.1f}M elements")
    groups = allocate(wl, dev, args.split)

    log(f"[bench] timing alpha={alpha}: warmup {args.warmup}, steps {args.steps}")
    per, wall = time_steps(wl, groups, alpha, args.warmup, args.steps)
    ms = statistics.mean(per)
    log(f"[bench] alpha={alpha}: {ms:.3f} ms/step (min {min(per):.3f})")

    # the committed counter summaries were taken with the default
    # Newton-Schulz settings; other settings run other kernels
    profiled = (args.ns_chain == "hilo" and args.ns_master == "bf16" and args.ns_form == "auto"
                and wl.ns_steps == workloads.WORKLOADS[args.workload].ns_steps)
    phases = {}
    roofline = None
    ns_frac = None
    mfma_counters = {}
    hbm_counters = {}
    if not args.no_profile:
        phases = profile_phases(wl, groups, alpha, args.steps)
        dom = max(phases, key=lambda p: phases[p]["total_ms_per_step"])
        d = phases[dom]
        traffic = None
        for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*traffic*.txt"))):
            traffic = traffic or (profsum.lookup_traffic(path, dom, wl.name, alpha) if profiled else None)
        for p in STREAMING_PHASES:
            for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*traffic*.txt"))):
                hit = profsum.lookup_hbm_rate(path, p, wl.name, alpha) if profiled else None
                if hit and p not in hbm_counters:
                    hbm_counters[p] = hit
        for p in NS_PHASES:
            for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*mfma*.txt"))):
                hit = profsum.lookup_mfma(path, p, wl.name, alpha) if profiled else None
                if hit and p not in mfma_counters:
                    mfma_counters[p] = hit
        roofline = dict(bound=d["bound"], achieved=round(d["achieved"], 3), peak=d["peak"],
                        unit=d["unit"], frac=round(d["frac"], 4),
                        traffic=None if traffic is None else round(traffic),
                        traffic_unit="bytes per launch", kernel=dom,
                        avg_launch_ms=round(d["avg_launch_ms"], 5),
                        algorithmic_per_launch=round(d["bytes_per_launch"] if d["unit"] == "GB/s"
                                                     else d["flops_per_launch"]),
                        algorithmic_unit="bytes" if d["unit"] == "GB/s" else "flops",
                        flops_per_launch=round(d["flops_per_launch"]),
                        bytes_per_launch=round(d["bytes_per_launch"]))
        ns_ms = sum(phases[p]["total_ms_per_step"] for p in NS_PHASES if p in phases)
        ns_work = sum(phases[p]["flops_per_launch"] * phases[p]["launches_per_step"]
                      for p in NS_PHASES if p in phases)
        if ns_ms > 0:
            ns_frac = ns_work / (ns_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS
        for p, d in phases.items():
            log(f"[bench]   {p:10s} {d['total_ms_per_step']:8.3f} ms/step  {d['bound']:7s} "
                f"{d['achieved']:9.1f} {d['unit']} ({100 * d['frac']:.1f}% of peak)"
                f"   [{d['hbm_gbs']:7.0f} GB/s, {d['mfma_tflops']:6.1f} TFLOP/s]")

    per_alpha = {str(alpha): round(ms, 4)}
    if not args.no_extra_alphas:
        for a in wl.alphas:
            if a == alpha:
                continue
            p2, _ = time_steps(wl, groups, a, args.warmup, args.steps)
            per_alpha[str(a)] = round(statistics.mean(p2), 4)
            log(f"[bench] alpha={a}: {per_alpha[str(a)]:.3f} ms/step")

    alphas = [alpha] if args.no_extra_alphas else list(dict.fromkeys([alpha, *wl.alphas]))
    per_chain, per_master = {}, {}
    if not args.no_chain_compare and NS_MASTER == binding.MASTER_BF16 and NS_FORM != binding.NS_DIRECT:
        # the other storage of the GRAM chain, and the fp32 master, at every fraction
        own = NS_CHAIN
        other = binding.CHAIN_F16 if own == binding.CHAIN_HILO else binding.CHAIN_HILO
        names = {v: k for k, v in NS_CHAINS.items()}
        per_chain[names[own]] = dict(per_alpha)
        per_chain[names[other]] = {}
        per_master = {"fp32": {}}
        try:
            for a in alphas:
                NS_CHAIN = other
                p4, _ = time_steps(wl, groups, a, args.warmup, args.steps)
                per_chain[names[other]][str(a)] = round(statistics.mean(p4), 4)
                log(f"[bench] alpha={a}, chain {names[other]}: {per_chain[names[other]][str(a)]:.3f} ms/step")
                NS_CHAIN = binding.CHAIN_HILO
                NS_MASTER = binding.MASTER_FP32
                p5, _ = time_steps(wl, groups, a, args.warmup, args.steps)
                per_master["fp32"][str(a)] = round(statistics.mean(p5), 4)
                log(f"[bench] alpha={a}, fp32 master: {per_master['fp32'][str(a)]:.3f} ms/step")
                NS_MASTER = binding.MASTER_BF16
        finally:
            NS_CHAIN = own
            NS_MASTER = binding.MASTER_BF16
        # the fp32 master runs the hi/lo chain: its reference is that chain's time
        per_master = {"bf16": per_chain[names[binding.CHAIN_HILO]], **per_master}

    per_rule = {"l1": round(ms, 4)}
    if not args.no_random_rule:
        p3, _ = time_steps(wl, groups, alpha, args.warmup, args.steps, binding.SELECT_RANDOM)
        per_rule["random"] = round(statistics.mean(p3), 4)
        log(f"[bench] alpha={alpha}, Random rule: {per_rule['random']:.3f} ms/step")

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] timing the CPU oracle for ~{args.cpu_seconds:.0f} s")
        cpu = cpu_baseline(wl, alpha, args.cpu_seconds)
        log(f"[bench] oracle: {cpu['value']:.1f} ms per stack step (estimated)")

    tail = per[-20:]
    line = {
        "metric": METRIC,
        "value": round(ms, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "alpha": alpha,
                   "matrices": wl.matrices(), "elements": wl.elements(),
                   "ns_steps": wl.ns_steps, "mu": wl.mu, "lr": wl.lr, "ns_form": args.ns_form,
                   "ns_chain": args.ns_chain, "ns_master": args.ns_master,
                   "parallelism": "single GPU, batched per shape group",
                   "calls": args.calls, "group_streams": args.group_streams,
                   "streams": args.streams, "split": args.split},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "per_alpha_ms": per_alpha,
        "per_rule_ms": per_rule,
        "per_chain_ms": per_chain,
        "per_master_ms": per_master,
        "ns_mfma_frac": None if ns_frac is None else round(ns_frac, 4),
        "ns_mfma_counters": mfma_counters or None,
        "ns_mfma_counters_per_alpha": mfma_per_alpha(wl.name, per_alpha, profiled) or None,
        "streaming_hbm_counters": hbm_counters or None,
        "step_ms_stats": {"mean": round(ms, 4), "median": round(statistics.median(per), 4),
                          "min": round(min(per), 4), "mean_last_20": round(statistics.mean(tail), 4),
                          "wall_s": round(wall, 3)},
        "phases": {p: {k: (round(v, 5) if isinstance(v, float) else v) for k, v in d.items()}
                   for p, d in phases.items()},
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
