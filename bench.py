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
  roofline     K4, the Newton-Schulz GEMMs, against the bf16 MFMA peak: the
               iteration's dense flop count T (4 s^2 l + 2 s^3) per matrix
               over the stack, divided by the Newton-Schulz kernels' time per
               step, measured with HIP events on the library's stream in a
               second timed pass; beside it rocprofv3's MFMA counters and the
               counted HBM bytes from the committed profiles
  step_frac    the step's roofline floor (the larger of the MFMA time of those
               flops and the HBM time of the step's algorithmic bytes) over
               the measured step time
  per_workload the other stacks (single matrix, column selection, 7B, MoE),
               each at its fractions, timed and measured the same way
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
import math
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


def num_selected(alpha, d_sel):
    """k = ceil(alpha * d_sel) with alpha as the fp32 value the library takes,
    clamped to [1, d_sel] (the fraction of lines Algorithm 1 selects)."""
    import numpy as np
    return int(min(d_sel, max(1, math.ceil(float(np.float32(alpha)) * d_sel))))


def floors(wl, alpha, ns_steps=None):
    """The step's algorithmic work and its roofline floors on one MI355X.

    Per matrix (rows x cols = fan-out x fan-in, N elements, k selected lines
    of length d_oth, s = min(k, d_oth), l = max(k, d_oth), T steps):
      Newton-Schulz flops   T (4 s^2 l + 2 s^3), the dense count of the
                            iteration A = X X^T, B = b A + c A^2, X <- a X + B X
      algorithmic bytes     N (4 + g + 4) + k d_oth (4 + 4 + 2 w): the momentum
                            read and written with the gradient read (every
                            element), then the selected lines of M read and
                            written and those of W read and written (g, w the
                            bytes per element of G and W)
    The compact matrix and the Newton-Schulz intermediates are implementation
    traffic, not counted here."""
    T = wl.ns_steps if ns_steps is None else ns_steps
    eb = 2.0 if wl.w_dtype == "bf16" else 4.0
    flops = nbytes = 0.0
    for g in wl.groups:
        axis = (0 if g.rows <= g.cols else 1) if g.axis == workloads.AXIS_AUTO else g.axis
        d_sel, d_oth = (g.rows, g.cols) if axis == 0 else (g.cols, g.rows)
        k = num_selected(alpha, d_sel)
        s_, l_ = min(k, d_oth), max(k, d_oth)
        n_el = float(g.rows) * g.cols
        flops += g.count * T * (4.0 * s_ * s_ * l_ + 2.0 * s_ ** 3)
        nbytes += g.count * (n_el * (8.0 + eb) + float(k) * d_oth * (8.0 + 2.0 * eb))
    ns_ms = flops / (MFMA_BF16_PEAK_TFS * 1e12) * 1e3
    hbm_ms = nbytes / (HBM_PEAK_GBS * 1e9) * 1e3
    return dict(ns_flops=flops, alg_bytes=nbytes, ns_ms_at_peak=ns_ms, hbm_ms_at_peak=hbm_ms,
                floor_ms=max(ns_ms, hbm_ms), bound="mfma" if ns_ms >= hbm_ms else "hbm")


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
                    and NS_MASTER == binding.MASTER_BF16 and rule == binding.SELECT_L1
                    and wl.w_dtype == "bf16"):
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
        # the Newton-Schulz GEMMs against the MFMA peak (their executed
        # flops, hi/lo passes included), the streaming kernels against HBM
        if ph == "select":
            bound, ach, peak, unit = "latency", nbytes / sec / 1e9, HBM_PEAK_GBS, "GB/s"
        elif ph in NS_PHASES:
            bound, ach, peak, unit = "mfma", flops / sec / 1e12, MFMA_BF16_PEAK_TFS, "TFLOP/s"
        else:
            bound, ach, peak, unit = "hbm", nbytes / sec / 1e9, HBM_PEAK_GBS, "GB/s"
        out[ph] = dict(total_ms_per_step=d["ms"] / steps, avg_launch_ms=avg_ms,
                       launches_per_step=d["launches"] / steps, flops_per_launch=flops,
                       bytes_per_launch=nbytes, achieved=ach, peak=peak, unit=unit, bound=bound,
                       frac=ach / peak,
                       mfma_tflops=flops / sec / 1e12, hbm_gbs=nbytes / sec / 1e9)
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(wl, alpha, seconds):
    """The oracle on a bounded sample: one matrix of each shape group per
    pass, repeated until `seconds` of CPU time have run, then scaled by the
    group counts to a whole-stack step. Also the single 256x256 matrix on
    one thread (its BLAS limited to one thread)."""
    import numpy as np

    import oracle
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover - threadpoolctl is optional
        threadpool_limits = None
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
    # the single fp32 256x256 matrix (alpha 0.25, rows) on one thread, in full
    single = workloads.WORKLOADS["single-256"]
    W, M, G = workloads.make_group(single, 0, dev)
    Wh, Mh, Gh = (W[0].double().cpu().numpy(), M[0].cpu().numpy(), G[0].cpu().numpy())
    c1 = []
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            for _ in range(5):
                t0 = time.perf_counter()
                oracle.dion2_step(Wh, Mh, Gh, 0.25, single.mu, single.lr, single.ns_steps,
                                  single.groups[0].axis, w_dtype=single.w_dtype)
                c1.append(time.perf_counter() - t0)
    return dict(value=est_s * 1e3, unit="ms", cores=blas_threads or 1, kind="oracle",
                host_cores=cores, blas_threads=blas_threads, cpu_model=cpu_model(),
                extrapolated=True,
                single_256_one_thread_ms=round(statistics.median(c1) * 1e3, 3) if c1 else None,
                sample=(f"{passes} pass(es) over one matrix of each of the {len(wl.groups)} "
                        f"shape groups ({sum(len(t) for t in per_group)} oracle steps, "
                        f"{sum(sum(t) for t in per_group):.1f} s), mean per group scaled by "
                        f"the group counts to the {wl.matrices()}-matrix stack; 'cores' is the "
                        f"BLAS thread count the oracle's matrix products ran on (its l1 sums "
                        f"are single-threaded); the single 256x256 fp32 matrix also ran in "
                        f"full on one thread (median of 5)"))


def ns_roofline(wl, alpha, phases, profiled):
    """K4 against the bf16 MFMA peak: the stack's dense Newton-Schulz flops
    per step over the Newton-Schulz kernels' event-timed time per step, with
    the committed counter figures for the same kernels beside it."""
    fl = floors(wl, alpha)
    ns_ms = sum(phases[p]["total_ms_per_step"] for p in NS_PHASES if p in phases)
    if ns_ms <= 0:
        return None
    ach = fl["ns_flops"] / (ns_ms * 1e-3) / 1e12
    executed = sum(phases[p]["flops_per_launch"] * phases[p]["launches_per_step"]
                   for p in NS_PHASES if p in phases)
    counters, traffic = {}, None
    if profiled:
        for p in NS_PHASES:
            for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*mfma*.txt"))):
                hit = profsum.lookup_mfma(path, p, wl.name, alpha)
                if hit and p not in counters:
                    counters[p] = hit
        tot = 0.0
        for p in NS_PHASES:
            if p not in phases:
                continue
            hit = None
            for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*traffic*.txt"))):
                hit = hit or profsum.lookup_traffic(path, p, wl.name, alpha)
            if hit is None:
                tot = None
                break
            tot += hit * phases[p]["launches_per_step"]
        traffic = None if tot is None else round(tot)
    util = None
    if counters and all(p in counters for p in NS_PHASES if p in phases):
        # duration-weighted over the Newton-Schulz phases
        w = {p: phases[p]["total_ms_per_step"] for p in NS_PHASES if p in phases}
        util = round(sum(counters[p]["mfma_util_pct"] * w[p] for p in w) / sum(w.values()), 2)
    return dict(bound="mfma", achieved=round(ach, 2), peak=MFMA_BF16_PEAK_TFS, unit="TFLOP/s",
                frac=round(ach / MFMA_BF16_PEAK_TFS, 4), traffic=traffic,
                traffic_unit="HBM bytes per step of the Newton-Schulz kernels (rocprofv3 "
                             "FETCH_SIZE + WRITE_SIZE, calibrated)",
                kernel="K4 Newton-Schulz GEMMs (ns_gram + ns_poly + ns_update)",
                unit_of_work="one step's Newton-Schulz over the whole stack",
                algorithmic_flops_per_step=fl["ns_flops"],
                ns_ms_per_step=round(ns_ms, 4),
                launches_per_step=round(sum(phases[p]["launches_per_step"] for p in NS_PHASES
                                            if p in phases), 2),
                executed_flops_per_step=executed,
                executed_tflops=round(executed / (ns_ms * 1e-3) / 1e12, 2),
                mfma_util_pct=util, mfma_counters=counters or None)


def measure_workload(name, alphas, warmup, steps, prof_steps, dev):
    """One other stack: allocated, timed at each fraction (one stream per
    shape group, as the headline), its Newton-Schulz phases event-timed in a
    second pass, then released."""
    wl = workloads.WORKLOADS[name]
    t0 = time.perf_counter()
    groups = allocate(wl, dev)
    log(f"[bench] workload {name}: {wl.matrices()} matrices, {wl.elements() / 1e6:.1f}M elements "
        f"(allocated in {time.perf_counter() - t0:.1f} s)")
    saved = STREAMS[:]
    STREAMS.clear()
    STREAMS.extend(torch.cuda.Stream() for _ in wl.groups)
    out = {}
    try:
        for a in alphas:
            w_, s_ = (warmup, steps) if not isinstance(warmup, dict) else (warmup[a], steps[a])
            per, _ = time_steps(wl, groups, a, w_, s_)
            ms = statistics.mean(per)
            phases = profile_phases(wl, groups, a, prof_steps if not isinstance(prof_steps, dict)
                                    else prof_steps[a])
            fl = floors(wl, a)
            roof = ns_roofline(wl, a, phases, True)
            out[str(a)] = dict(ms_per_step=round(ms, 4), steps=s_, warmup=w_,
                               floor_ms=round(fl["floor_ms"], 4), floor_bound=fl["bound"],
                               step_frac=round(fl["floor_ms"] / ms, 4),
                               ns_frac=None if roof is None else roof["frac"],
                               ns_ms_per_step=None if roof is None else roof["ns_ms_per_step"],
                               streaming_ms_per_step=round(sum(
                                   phases[p]["total_ms_per_step"] for p in
                                   ("momentum", "select", "gather", "apply") if p in phases), 4))
            log(f"[bench]   {name} alpha={a}: {ms:.3f} ms/step, floor {fl['floor_ms']:.3f} ms "
                f"({fl['bound']}), NS {out[str(a)]['ns_frac']} of MFMA peak")
    finally:
        STREAMS.clear()
        STREAMS.extend(saved)
        del groups
        torch.cuda.synchronize()
        binding.dion2_release_workspaces()
        torch.cuda.empty_cache()
    return {"description": wl.description, "matrices": wl.matrices(), "elements": wl.elements(),
            "per_alpha": out}


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
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other stacks (single matrix, column selection, MoE, 7B)")
    ap.add_argument("--workload-steps", type=int, default=10,
                    help="timed steps per fraction of each other stack (3 for 7B at alpha 1)")
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
    hbm_counters = {}
    if not args.no_profile:
        phases = profile_phases(wl, groups, alpha, args.steps)
        for p in STREAMING_PHASES:
            for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*traffic*.txt"))):
                hit = profsum.lookup_hbm_rate(path, p, wl.name, alpha) if profiled else None
                if hit and p not in hbm_counters:
                    hbm_counters[p] = hit
        roofline = ns_roofline(wl, alpha, phases, profiled)
        ns_ms = sum(phases[p]["total_ms_per_step"] for p in NS_PHASES if p in phases)
        ns_work = sum(phases[p]["flops_per_launch"] * phases[p]["launches_per_step"]
                      for p in NS_PHASES if p in phases)
        if ns_ms > 0:
            ns_frac = ns_work / (ns_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS
        for p, d in phases.items():
            log(f"[bench]   {p:10s} {d['total_ms_per_step']:8.3f} ms/step  {d['bound']:7s} "
                f"{d['achieved']:9.1f} {d['unit']} ({100 * d['frac']:.1f}% of peak)"
                f"   [{d['hbm_gbs']:7.0f} GB/s, {d['mfma_tflops']:6.1f} TFLOP/s]")
        if roofline:
            log(f"[bench] K4 roofline: {roofline['achieved']:.1f} TFLOP/s of dense Newton-Schulz "
                f"work = {100 * roofline['frac']:.1f}% of the bf16 MFMA peak "
                f"({roofline['ns_ms_per_step']:.3f} ms/step)")
    fl = floors(wl, alpha)
    step_frac = fl["floor_ms"] / ms

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

    per_workload = {}
    if not args.no_workloads and args.workload == "1b" and not GROUPED[0] and args.split == 1 \
            and NS_FORM == binding.NS_AUTO and NS_CHAIN == binding.CHAIN_HILO \
            and NS_MASTER == binding.MASTER_BF16 and wl.ns_steps == 5:
        # The other stacks of the measurement plan, one at a time (each
        # allocated, timed and released), with fewer steps: the 7B stack at
        # alpha = 1 takes about a second per step.
        n = args.workload_steps
        del groups
        torch.cuda.synchronize()
        binding.dion2_release_workspaces()
        torch.cuda.empty_cache()
        plan = [("single-256", (0.25,)), ("1b-colsel", (0.25,)), ("moe", (0.25,)),
                ("7b", (0.125, 0.25, 1.0))]
        for name, alist in plan:
            if name == "7b":
                warm = {0.125: 3, 0.25: 3, 1.0: 1}
                stp = {0.125: n, 0.25: n, 1.0: 3}
                prof = {0.125: 2, 0.25: 2, 1.0: 1}
            else:
                warm, stp, prof = 3, n, 2
            per_workload[name] = measure_workload(name, alist, warm, stp, prof, dev)
        groups = None

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
        "step_frac": round(step_frac, 4),
        "floors": {"floor_ms": round(fl["floor_ms"], 4), "bound": fl["bound"],
                   "ns_ms_at_mfma_peak": round(fl["ns_ms_at_peak"], 4),
                   "hbm_ms_at_peak": round(fl["hbm_ms_at_peak"], 4),
                   "ns_flops": fl["ns_flops"], "alg_bytes": fl["alg_bytes"],
                   "per_alpha_step_frac": {a: round(floors(wl, float(a))["floor_ms"] / v, 4)
                                           for a, v in per_alpha.items()}},
        "cpu_baseline": cpu,
        "per_alpha_ms": per_alpha,
        "per_rule_ms": per_rule,
        "per_chain_ms": per_chain,
        "per_master_ms": per_master,
        "ns_mfma_frac_executed": None if ns_frac is None else round(ns_frac, 4),
        "ns_mfma_counters_per_alpha": mfma_per_alpha(wl.name, per_alpha, profiled) or None,
        "streaming_hbm_counters": hbm_counters or None,
        "step_ms_stats": {"mean": round(ms, 4), "median": round(statistics.median(per), 4),
                          "min": round(min(per), 4), "mean_last_20": round(statistics.mean(tail), 4),
                          "wall_s": round(wall, 3)},
        "phases": {p: {k: (round(v, 5) if isinstance(v, float) else v) for k, v in d.items()}
                   for p, d in phases.items()},
        "per_workload": per_workload or None,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
