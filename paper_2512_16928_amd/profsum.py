"""Summaries of rocprofv3 CSV output for the Dion2 kernels.

    python -m paper_2512_16928_amd.profsum stats DIR
        per-kernel and per-phase launch statistics from a
        `rocprofv3 --kernel-trace --stats -f csv -d DIR` run
    python -m paper_2512_16928_amd.profsum traffic FETCH_DIR WRITE_DIR --workload W --alpha A [--stats DIR]
        HBM bytes per launch of every phase from two `--pmc FETCH_SIZE` and
        `--pmc WRITE_SIZE` runs, scaled by what the same counters read for
        the calibration copy (a single elementwise kernel, `torch.neg` of
        2^28 fp32 values: 1 GiB read, 1 GiB written); with the kernels'
        average durations from a `--kernel-trace --stats` run, also the
        counted HBM GB/s against the 8 TB/s peak

    python -m paper_2512_16928_amd.profsum mfma PMC_DIR STATS_DIR --workload W --alpha A
        MFMA utilisation of the Newton-Schulz phases from a `--pmc MfmaUtil
        MfmaFlopsBF16 MfmaFlopsF16` run (rocprofv3's derived counters: busy
        cycles of the matrix cores over active cycles of every SIMD, and 512
        flops per counted matrix op), with the kernels' average durations
        from a `--kernel-trace --stats` run of the same command
    python -m paper_2512_16928_amd.profsum gaps DIR [--split-us US]
        idle time between consecutive library kernels on each stream of a
        `--kernel-trace` run, and the share of the traced span during which
        some library kernel ran

The traffic and MFMA summaries end with one line per phase, tagged with a
hash of the kernel sources it was taken on; bench.py reports a phase's
figures only while those sources are unchanged.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import os
import re
import statistics
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")

# phase -> kernel source files whose text decides the phase's kernels
PHASE_SOURCES = {
    "momentum": ("k_momentum.hip",),
    "select": ("k_select.hip",),
    "gather": ("k_gather.hip",),
    "ns_gram": ("k_gemm.hip",),
    "ns_poly": ("k_gemm.hip",),
    "ns_update": ("k_gemm.hip",),
    "apply": ("k_apply.hip",),
}
CALIB_BYTES = float(1 << 30)   # the calibration copy reads and writes this much
CALIB_PATTERN = "neg_kernel"


_TOKENS = re.compile(r'"(?:\\.|[^"\\])*"|\'(?:\\.|[^\'\\])*\'|//[^\n]*|/\*.*?\*/', re.S)


def code_text(src: str) -> str:
    """Source text without comments and with whitespace collapsed: what the
    compiler sees, so that editing a comment does not count as a change."""
    out = _TOKENS.sub(lambda m: " " if m.group(0)[0] == "/" else m.group(0), src)
    return " ".join(out.split())


def source_hash(phase: str) -> str:
    h = hashlib.sha256()
    for f in PHASE_SOURCES[phase] + ("dion2_device.h", "dion2_api.hip"):
        with open(os.path.join(CSRC, f), encoding="utf-8") as fh:
            h.update(code_text(fh.read()).encode())
    return h.hexdigest()[:16]


def _local(kernel: str) -> str:
    """Demangled name without return type, namespaces and arguments."""
    k = kernel.replace("(anonymous namespace)::", "")
    k = k[5:] if k.startswith("void ") else k
    return k.split("dion2::", 1)[1] if k.startswith("dion2::") else k


def phase_of(kernel: str):
    """Library phase of a demangled kernel name, or None for other kernels."""
    if "dion2::" not in kernel:
        return None
    k = _local(kernel)
    if k.startswith("momentum"):
        return "momentum"
    if k.startswith("select"):
        return "select"
    if (k.startswith("gather") or k.startswith("update_cols") or k.startswith("decay_all")
            or k.startswith("colpass")):   # colpass_*: the end of the Random rule's single column pass
        return "gather"
    if k.startswith("apply"):
        return "apply"
    if k.startswith("transpose"):    # X^T for the Direct form's update
        return "ns_update"
    if k.startswith("chain_small"):  # the whole s x s chain of s <= 64 in one launch
        return "ns_poly"
    m = re.match(r"gemm<(\d+), (?:\(dion2::GemmEpi\))?(\d)", k)
    if m:
        npass, epi = int(m.group(1)), int(m.group(2))
        if epi in (2, 3, 5):         # update / final product with X (5: with the update step)
            return "ns_update"
        # X X^T: one pass on bf16 operands, stored as a hi / lo pair (0) or in
        # fp16 (6); the same epilogues on fp16 operands are s x s products
        f16_tile = re.search(r"Tile<[^>]*\btrue>", k) is not None
        if epi in (0, 6) and npass == 1 and not f16_tile:
            return "ns_gram"
        return "ns_poly"             # the s x s products
    return None


def short_name(kernel: str, width: int = 72) -> str:
    k = _local(kernel).replace("dion2::", "")
    k = k.split("(dion2", 1)[0] if "dion2::" in kernel else k
    return k if len(k) <= width else k[: width - 3] + "..."


def find_csv(d: str, suffix: str) -> str:
    hits = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not hits:
        sys.exit(f"no *{suffix} under {d}")
    return hits[-1]


def cmd_stats(args):
    path = find_csv(args.dir, "kernel_stats.csv")
    rows = list(csv.DictReader(open(path)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    phases = {}
    print(f"{'kernel':72s} {'calls':>7s} {'avg us':>9s} {'total ms':>9s} {'%':>6s}")
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name, calls, tot = r["Name"], int(r["Calls"]), float(r["TotalDurationNs"])
        ph = phase_of(name)
        if ph:
            p = phases.setdefault(ph, [0, 0.0])
            p[0] += calls
            p[1] += tot
        if tot / total < 0.001 and not ph:
            continue
        print(f"{short_name(name):72s} {calls:7d} {tot / calls / 1e3:9.2f} {tot / 1e6:9.3f} "
              f"{100 * tot / total:6.2f}")
    print()
    print(f"{'phase':12s} {'launches':>9s} {'avg us/launch':>14s} {'total ms':>9s}")
    for ph in PHASE_SOURCES:
        if ph in phases:
            n, t = phases[ph]
            print(f"{ph:12s} {n:9d} {t / n / 1e3:14.2f} {t / 1e6:9.3f}")


def read_counter(d: str, counter: str):
    """{dispatch id: (kernel name, grid size, value in bytes)} for one counter."""
    path = find_csv(d, "counter_collection.csv")
    out = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        did = int(r["Dispatch_Id"])
        name, grid, val = r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])
        prev = out.get(did)
        out[did] = (name, grid, val * 1024.0 + (prev[2] if prev else 0.0))
    return out


def cmd_traffic(args):
    fetch = read_counter(args.fetch_dir, "FETCH_SIZE")
    write = read_counter(args.write_dir, "WRITE_SIZE")

    def calib(data):
        v = [b for n, _, b in data.values() if CALIB_PATTERN in n]
        if not v:
            sys.exit(f"no calibration dispatch ({CALIB_PATTERN}) in the counter output")
        return statistics.median(v), len(v)

    cf, nf = calib(fetch)
    cw, nw = calib(write)
    f_fetch, f_write = CALIB_BYTES / cf, CALIB_BYTES / cw
    print(f"calibration copy (torch.neg, 2^28 fp32): FETCH_SIZE {cf / 2**30:.3f} GiB "
          f"({nf} dispatches), WRITE_SIZE {cw / 2**30:.3f} GiB ({nw} dispatches)")
    print(f"scale factors: fetch x{f_fetch:.3f}, write x{f_write:.3f}")
    print()

    def per_phase(data, factor):
        acc = {}
        for name, _, b in data.values():
            ph = phase_of(name)
            if ph:
                a = acc.setdefault(ph, {}).setdefault(short_name(name), [0, 0.0])
                a[0] += 1
                a[1] += b * factor
        return acc

    pf, pw = per_phase(fetch, f_fetch), per_phase(write, f_write)
    dur = kernel_durations(args.stats) if args.stats else {}
    print(f"{'kernel':72s} {'n':>5s} {'read MiB':>10s} {'write MiB':>10s}  (scaled, per dispatch)"
          + (f" {'avg us':>8s} {'GB/s':>8s}" if dur else ""))
    lines = []
    for ph in PHASE_SOURCES:
        if ph not in pf or ph not in pw:
            continue
        nf_tot = sum(n for n, _ in pf[ph].values())
        nw_tot = sum(n for n, _ in pw[ph].values())
        t_tot = 0.0   # ns over the phase's dispatches, from the stats run
        for k in pf[ph]:
            n, b = pf[ph][k]
            wn, wb = pw[ph].get(k, (1, 0.0))
            row = f"{k:72s} {n:5d} {b / n / 2**20:10.2f} {wb / max(wn, 1) / 2**20:10.2f}"
            if dur:
                ns = dur.get(k, float("nan"))
                t_tot += n * ns
                row += f" {ns / 1e3:8.2f} {(b / n + wb / max(wn, 1)) / ns:8.1f}"
            print(row)
        rd = sum(b for _, b in pf[ph].values()) / nf_tot
        wr = sum(b for _, b in pw[ph].values()) / nw_tot
        rate = ""
        if dur:
            gbs = (rd + wr) / (t_tot / nf_tot)
            rate = f" avg_launch_us={t_tot / nf_tot / 1e3:.2f} counted_gbs={gbs:.1f} frac_of_peak={gbs / HBM_PEAK_GBS:.4f}"
        lines.append(f"traffic phase={ph} workload={args.workload} alpha={args.alpha} "
                     f"sources={source_hash(ph)} read_bytes_per_launch={rd:.0f} "
                     f"write_bytes_per_launch={wr:.0f} bytes_per_launch={rd + wr:.0f} "
                     f"launches={nf_tot}{rate}")
    print()
    for ln in lines:
        print(ln)


MFMA_PEAK_FLOPS = {"bf16": 2.5e15, "f16": 2.5e15}   # dense matrix-core peaks of MI355X
HBM_PEAK_GBS = 8000.0                                 # MI355X HBM3E
NS_PHASES = ("ns_gram", "ns_poly", "ns_update")


def read_values(d: str, counters):
    """{dispatch id: (kernel name, {counter: [values]})} for the given counters."""
    path = find_csv(d, "counter_collection.csv")
    out = {}
    for r in csv.DictReader(open(path)):
        c = r["Counter_Name"]
        if c not in counters:
            continue
        ent = out.setdefault(int(r["Dispatch_Id"]), (r["Kernel_Name"], {}))
        ent[1].setdefault(c, []).append(float(r["Counter_Value"]))
    return out


def kernel_durations(d: str):
    """{short kernel name: average duration in ns} from a kernel-stats run."""
    rows = csv.DictReader(open(find_csv(d, "kernel_stats.csv")))
    return {short_name(r["Name"]): float(r["AverageNs"]) for r in rows if phase_of(r["Name"])}


def cmd_mfma(args):
    data = read_values(args.pmc_dir, ("MfmaUtil", "MfmaFlopsBF16", "MfmaFlopsF16"))
    dur = kernel_durations(args.stats_dir)
    acc = {}
    for name, vals in data.values():
        ph = phase_of(name)
        if ph not in NS_PHASES:
            continue
        k = short_name(name)
        a = acc.setdefault(ph, {}).setdefault(k, [0, 0.0, 0.0])
        a[0] += 1
        a[1] += statistics.mean(vals.get("MfmaUtil", [0.0]))
        a[2] += sum(vals.get("MfmaFlopsBF16", [0.0])) + sum(vals.get("MfmaFlopsF16", [0.0]))
    peak = MFMA_PEAK_FLOPS["bf16"]
    print(f"{'kernel':72s} {'n':>5s} {'MfmaUtil %':>10s} {'GFLOP/disp':>11s} {'avg us':>8s} {'TFLOP/s':>8s} {'of peak':>8s}")
    lines = []
    for ph in NS_PHASES:
        if ph not in acc:
            continue
        n_tot = t_tot = f_tot = u_w = 0.0
        for k, (n, u, f) in acc[ph].items():
            us = dur.get(k, float("nan")) / 1e3
            print(f"{k:72s} {n:5d} {u / n:10.1f} {f / n / 1e9:11.2f} {us:8.2f} "
                  f"{f / n / us / 1e6:8.1f} {f / n / us / 1e6 / (peak / 1e12):8.3f}")
            n_tot += n
            t_tot += n * us
            f_tot += f
            u_w += u * us          # utilisation weighted by each dispatch's duration
        util = u_w / t_tot
        tflops = f_tot / t_tot / 1e6
        lines.append(f"mfma phase={ph} workload={args.workload} alpha={args.alpha} "
                     f"sources={source_hash(ph)} mfma_util_pct={util:.2f} "
                     f"counted_flops_per_launch={f_tot / n_tot:.0f} avg_launch_us={t_tot / n_tot:.2f} "
                     f"counted_tflops={tflops:.1f} frac_of_peak={tflops * 1e12 / peak:.4f} "
                     f"launches={n_tot:.0f}")
    print()
    for ln in lines:
        print(ln)


def lookup_mfma(path: str, phase: str, workload: str, alpha: float):
    """The counter-based MFMA figures of `phase` from a committed summary, or
    None when absent or taken on other kernel sources."""
    kv = lookup_line(path, "mfma", phase, workload, alpha)
    if kv is None:
        return None
    return {"mfma_util_pct": float(kv["mfma_util_pct"]),
            "counted_flops_per_launch": float(kv["counted_flops_per_launch"]),
            "counted_tflops": float(kv["counted_tflops"]),
            "frac_of_peak": float(kv["frac_of_peak"])}


def lookup_line(path: str, kind: str, phase: str, workload: str, alpha: float):
    """The key=value fields of the `kind` line of `phase` in a committed
    summary, or None when absent or taken on other kernel sources."""
    if not os.path.exists(path):
        return None
    want = source_hash(phase)
    for ln in open(path):
        if not ln.startswith(kind + " "):
            continue
        kv = dict(x.split("=", 1) for x in ln.split()[1:])
        if (kv.get("phase") == phase and kv.get("workload") == workload
                and float(kv.get("alpha", "nan")) == alpha and kv.get("sources") == want):
            return kv
    return None


def lookup_traffic(path: str, phase: str, workload: str, alpha: float):
    """Scaled HBM bytes per launch of `phase` from a committed traffic summary,
    or None when absent or taken on other kernel sources."""
    kv = lookup_line(path, "traffic", phase, workload, alpha)
    return None if kv is None else float(kv["bytes_per_launch"])


def lookup_hbm_rate(path: str, phase: str, workload: str, alpha: float):
    """Counted HBM GB/s of `phase` (scaled counter bytes over the average
    launch duration) and its fraction of the peak, or None."""
    kv = lookup_line(path, "traffic", phase, workload, alpha)
    if kv is None or "counted_gbs" not in kv:
        return None
    return {"counted_gbs": float(kv["counted_gbs"]), "frac_of_peak": float(kv["frac_of_peak"])}


def cmd_gaps(args):
    """Idle time between consecutive library kernels on each stream of a
    kernel-trace run (the launch overhead that graph capture would remove),
    and how much of the traced span some library kernel was running."""
    path = find_csv(args.dir, "kernel_trace.csv")
    rows = [r for r in csv.DictReader(open(path)) if phase_of(r["Kernel_Name"])]
    if not rows:
        sys.exit(f"no library kernels in {path}")
    by_stream = {}
    for r in rows:
        by_stream.setdefault(r["Stream_Id"], []).append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    print(f"{'stream':>6s} {'kernels':>8s} {'gaps':>6s} {'median us':>10s} {'mean us':>8s} {'p95 us':>7s} "
          f"{'total ms':>9s}")
    for sid in sorted(by_stream, key=lambda x: int(x)):
        ks = sorted(by_stream[sid])
        # a gap longer than args.split_us separates two steps (host-side work, events)
        gaps = [b[0] - a[1] for a, b in zip(ks, ks[1:])]
        gaps = sorted(max(0, g) for g in gaps if g < args.split_us * 1e3)
        if not gaps:
            continue
        med, p95 = gaps[len(gaps) // 2], gaps[min(len(gaps) - 1, int(0.95 * len(gaps)))]
        print(f"{sid:>6s} {len(ks):8d} {len(gaps):6d} {med / 1e3:10.2f} {sum(gaps) / len(gaps) / 1e3:8.2f} "
              f"{p95 / 1e3:7.2f} {sum(gaps) / 1e6:9.3f}")
    ev = sorted([(int(r["Start_Timestamp"]), 1) for r in rows] + [(int(r["End_Timestamp"]), -1) for r in rows])
    busy, depth, last = 0, 0, ev[0][0]
    for t, d in ev:
        if depth > 0:
            busy += t - last
        depth += d
        last = t
    span = ev[-1][0] - ev[0][0]
    print(f"\nlibrary kernels running during {busy / 1e6:.3f} ms of the {span / 1e6:.3f} ms traced "
          f"({100 * busy / span:.1f}%)")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("--workload", required=True)
    t.add_argument("--alpha", type=float, required=True)
    t.add_argument("--stats", default=None)
    m = sub.add_parser("mfma")
    m.add_argument("pmc_dir")
    m.add_argument("stats_dir")
    m.add_argument("--workload", required=True)
    m.add_argument("--alpha", type=float, required=True)
    g = sub.add_parser("gaps")
    g.add_argument("dir")
    g.add_argument("--split-us", type=float, default=200.0,
                   help="gaps longer than this separate steps and are not counted")
    args = ap.parse_args(argv)
    {"stats": cmd_stats, "traffic": cmd_traffic, "mfma": cmd_mfma, "gaps": cmd_gaps}[args.cmd](args)


if __name__ == "__main__":
    main()
