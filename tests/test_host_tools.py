"""CPU tests of the host-side tools: the profile summariser's kernel-to-phase
mapping and the benchmark's single-GPU guard."""
import os
import subprocess
import sys

from paper_2512_16928_amd import profsum

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_phase_of_kernel_names():
    cases = {
        "void dion2::(anonymous namespace)::momentum_rows<4, unsigned short>(dion2::MatSet, long)": "momentum",
        "dion2::(anonymous namespace)::momentum_cols_final(double const*, int, long)": "momentum",
        "dion2::(anonymous namespace)::select_topk(dion2::SelectArgs)": "select",
        "void dion2::(anonymous namespace)::gather_rows<4>(dion2::GatherArgs)": "gather",
        "dion2::(anonymous namespace)::chain_small(dion2::SmallChainArgs)": "ns_poly",
        "void dion2::(anonymous namespace)::update_cols<4, unsigned short>(dion2::GatherArgs)": "gather",
        "void dion2::(anonymous namespace)::apply_cols<4, unsigned short>(dion2::ApplyArgs)": "apply",
        "void dion2::(anonymous namespace)::gemm<1, 0, dion2::(anonymous namespace)::Tile<1, 0, 128, 128, 32, 2, 2, 4>, true>(dion2::GemmArgs)": "ns_gram",
        "void dion2::(anonymous namespace)::gemm<3, 0, dion2::(anonymous namespace)::Tile<3, 0, 128, 128, 32, 4, 2, 2>, true>(dion2::GemmArgs)": "ns_poly",
        "void dion2::(anonymous namespace)::gemm<3, 4, dion2::(anonymous namespace)::Tile<3, 0, 128, 128, 32, 4, 2, 2>, true>(dion2::GemmArgs)": "ns_poly",
        "void dion2::(anonymous namespace)::gemm<3, 1, dion2::(anonymous namespace)::Tile<3, 0, 128, 128, 32, 4, 2, 2>, true>(dion2::GemmArgs)": "ns_poly",
        "void dion2::(anonymous namespace)::gemm<1, 6, dion2::(anonymous namespace)::Tile<1, 0, 256, 256, 32, 4, 2, 3, false>, true>(dion2::GemmArgs)": "ns_gram",
        "void dion2::(anonymous namespace)::gemm<1, 6, dion2::(anonymous namespace)::Tile<1, 0, 128, 128, 32, 2, 2, 4, true>, true>(dion2::GemmArgs)": "ns_poly",
        "void dion2::(anonymous namespace)::gemm<1, 0, dion2::(anonymous namespace)::Tile<1, 0, 128, 128, 32, 2, 2, 4, true>, true>(dion2::GemmArgs)": "ns_poly",
        "void dion2::(anonymous namespace)::gemm<1, 8, dion2::(anonymous namespace)::Tile<1, 0, 128, 128, 32, 2, 2, 4, true>, true>(dion2::GemmArgs)": "ns_poly",
        "void dion2::(anonymous namespace)::gemm<1, 2, dion2::(anonymous namespace)::Tile<1, 1, 128, 128, 32, 2, 2, 2>, false>(dion2::GemmArgs)": "ns_update",
        "void dion2::(anonymous namespace)::gemm<2, 3, dion2::(anonymous namespace)::Tile<2, 1, 128, 128, 32, 2, 2, 2>, false>(dion2::GemmArgs)": "ns_update",
        "void dion2::(anonymous namespace)::gemm<2, 5, dion2::(anonymous namespace)::Tile<2, 1, 128, 128, 32, 2, 2, 2>, false>(dion2::GemmArgs)": "ns_update",
        "dion2::transpose_bf16(unsigned short const*, unsigned short*, long, long, long)": "ns_update",
        "dion2::(anonymous namespace)::colpass_compact(dion2::ColpassArgs)": "gather",
        "dion2::(anonymous namespace)::colpass_fold(dion2::ColpassArgs)": "gather",
        "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda>": None,
    }
    for name, phase in cases.items():
        assert profsum.phase_of(name) == phase, name


def test_traffic_lookup_requires_matching_sources(tmp_path):
    good = profsum.source_hash("ns_poly")
    f = tmp_path / "t_traffic.txt"
    f.write_text(f"traffic phase=ns_poly workload=1b alpha=0.25 sources={good} "
                 "read_bytes_per_launch=1 write_bytes_per_launch=2 bytes_per_launch=3 launches=1\n"
                 "traffic phase=apply workload=1b alpha=0.25 sources=0000000000000000 "
                 "read_bytes_per_launch=1 write_bytes_per_launch=2 bytes_per_launch=3 launches=1\n")
    assert profsum.lookup_traffic(str(f), "ns_poly", "1b", 0.25) == 3.0
    assert profsum.lookup_traffic(str(f), "ns_poly", "1b", 0.5) is None     # other workload point
    assert profsum.lookup_traffic(str(f), "apply", "1b", 0.25) is None      # stale sources
    assert profsum.lookup_hbm_rate(str(f), "ns_poly", "1b", 0.25) is None   # no durations given
    good = profsum.source_hash("gather")
    f.write_text(f"traffic phase=gather workload=1b alpha=0.25 sources={good} read_bytes_per_launch=1 "
                 "write_bytes_per_launch=2 bytes_per_launch=3 launches=9 avg_launch_us=241.08 "
                 "counted_gbs=5758.4 frac_of_peak=0.7198\n")
    assert profsum.lookup_hbm_rate(str(f), "gather", "1b", 0.25) == {"counted_gbs": 5758.4,
                                                                       "frac_of_peak": 0.7198}


def test_mfma_lookup_requires_matching_sources(tmp_path):
    f = tmp_path / "m.txt"
    good = profsum.source_hash("ns_poly")
    f.write_text("kernel table ...\n"
                 f"mfma phase=ns_poly workload=1b alpha=0.25 sources={good} mfma_util_pct=16.5 "
                 "counted_flops_per_launch=2e10 avg_launch_us=35.0 counted_tflops=571.4 "
                 "frac_of_peak=0.2286 launches=126\n"
                 "mfma phase=ns_gram workload=1b alpha=0.25 sources=0000000000000000 mfma_util_pct=1 "
                 "counted_flops_per_launch=1 avg_launch_us=1 counted_tflops=1 frac_of_peak=0.1 launches=1\n")
    hit = profsum.lookup_mfma(str(f), "ns_poly", "1b", 0.25)
    assert hit == {"mfma_util_pct": 16.5, "counted_flops_per_launch": 2e10, "counted_tflops": 571.4,
                   "frac_of_peak": 0.2286}
    assert profsum.lookup_mfma(str(f), "ns_poly", "7b", 0.25) is None      # other workload
    assert profsum.lookup_mfma(str(f), "ns_gram", "1b", 0.25) is None      # stale sources


def test_mfma_summary_from_counter_csv(tmp_path, capsys):
    """profsum mfma: per-dispatch counters and the stats run's durations give
    the phase's counted TFLOP/s and duration-weighted MfmaUtil."""
    k_poly = "void dion2::(anonymous namespace)::gemm<3, 0, Tile<3, 0, 128, 128, 32, 4, 2, 2, false>, true>(dion2::GemmArgs)"
    k_mom = "void dion2::(anonymous namespace)::momentum_rows<4, unsigned short>(dion2::MatSet)"
    pmc = tmp_path / "pmc"
    st = tmp_path / "st"
    pmc.mkdir()
    st.mkdir()
    rows = ['"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value"']
    for d, util, fl in ((1, 10.0, 1e10), (2, 30.0, 3e10)):
        rows += [f'{d},"{k_poly}","MfmaUtil",{util}', f'{d},"{k_poly}","MfmaFlopsBF16",{fl}',
                 f'{d},"{k_poly}","MfmaFlopsF16",0']
    rows.append(f'3,"{k_mom}","MfmaUtil",0')
    (pmc / "run_counter_collection.csv").write_text("\n".join(rows) + "\n")
    (st / "run_kernel_stats.csv").write_text(
        '"Name","Calls","TotalDurationNs","AverageNs"\n'
        f'"{k_poly}",2,80000,40000\n"{k_mom}",1,1000,1000\n')
    profsum.main(["mfma", str(pmc), str(st), "--workload", "1b", "--alpha", "0.25"])
    out = capsys.readouterr().out
    line = [ln for ln in out.splitlines() if ln.startswith("mfma ")]
    assert len(line) == 1 and "phase=ns_poly" in line[0]
    kv = dict(x.split("=", 1) for x in line[0].split()[1:])
    assert float(kv["mfma_util_pct"]) == 20.0                   # equal durations: the plain mean
    assert float(kv["counted_flops_per_launch"]) == 2e10
    assert abs(float(kv["counted_tflops"]) - 500.0) < 1e-9     # 2e10 flops in 40 us
    assert abs(float(kv["frac_of_peak"]) - 0.2) < 1e-9



def test_launch_gaps_from_kernel_trace(tmp_path, capsys):
    """profsum gaps: per-stream idle time between consecutive library kernels
    (other kernels ignored, gaps past the step split left out) and the share
    of the span some library kernel ran."""
    k = "void dion2::(anonymous namespace)::gemm<3, 0, Tile<3, 0, 128, 128, 32, 4, 2, 2, false>, true>(dion2::GemmArgs)"
    other = "void at::native::vectorized_elementwise_kernel<4>(int)"
    rows = ['"Stream_Id","Kernel_Name","Start_Timestamp","End_Timestamp"']
    # stream 1: kernels at [0,10) [12,20) [20,30) (us) then one after a 1 ms step break
    for a, b in ((0, 10), (12, 20), (20, 30), (1030, 1040)):
        rows.append(f'1,"{k}",{a * 1000},{b * 1000}')
    rows.append(f'2,"{k}",{5 * 1000},{15 * 1000}')
    rows.append(f'1,"{other}",{10 * 1000},{12 * 1000}')
    (tmp_path / "run_kernel_trace.csv").write_text("\n".join(rows) + "\n")
    profsum.main(["gaps", str(tmp_path)])
    out = capsys.readouterr().out.splitlines()
    s1 = [ln.split() for ln in out if ln.split()[:1] == ["1"]][0]
    assert s1[1:3] == ["4", "2"]                   # 4 kernels, 2 gaps under the split
    assert float(s1[4]) == 1.0                     # mean of 2 us and 0 us
    assert float(s1[6]) == 0.002                   # 2 us in total
    # busy: [0,30) and [1030,1040) -> 40 us of a 1040 us span
    assert "0.040 ms of the 1.040 ms traced" in out[-1]

def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_source_hash_ignores_comments_only():
    """The traffic lines stay valid across comment edits, not code edits."""
    base = 'int f(int x) { return x + 1; } // add one\nconst char* s = "// kept";\n'
    same = '/* header */ int f(int x)  {  return x + 1; }\n// another note\nconst char* s = "// kept";'
    other = base.replace("x + 1", "x + 2")
    strings = base.replace('"// kept"', '"// changed"')
    assert profsum.code_text(base) == profsum.code_text(same)
    assert profsum.code_text(base) != profsum.code_text(other)
    assert profsum.code_text(base) != profsum.code_text(strings)


def test_bench_floors_match_the_measurement_plan():
    """bench.floors: the Newton-Schulz flops T (4 s^2 l + 2 s^3) and the
    algorithmic bytes N (8 + g) + k d_oth (8 + 2 w) of each stack, against
    the figures derived for the measurement plan from the Table 1 shapes
    (three significant digits), and the floors at 2.5 PFLOP/s and 8 TB/s."""
    sys.path.insert(0, ROOT)
    import bench
    from paper_2512_16928_amd import workloads as wls
    want = {("1b", 0.25): (2.19e12, 10.47e9), ("1b", 0.5): (9.28e12, 12.88e9),
            ("1b", 1.0): (4.12e13, 17.72e9), ("1b-colsel", 0.25): (9.02e12, 10.47e9),
            ("7b", 0.125): (8.59e12, 74.5e9), ("7b", 0.25): (3.56e13, 84.2e9),
            ("7b", 1.0): (6.84e14, 142.5e9), ("moe", 0.25): (1.21e13, 80.3e9),
            ("single-256", 0.25): (2.36e7, 1.05e6)}
    for (name, alpha), (flops, nbytes) in want.items():
        f = bench.floors(wls.WORKLOADS[name], alpha)
        assert abs(f["ns_flops"] / flops - 1) < 5e-3, (name, alpha, f["ns_flops"])
        assert abs(f["alg_bytes"] / nbytes - 1) < 5e-3, (name, alpha, f["alg_bytes"])
        assert abs(f["ns_ms_at_peak"] - f["ns_flops"] / 2.5e12) < 1e-9
        assert abs(f["hbm_ms_at_peak"] - f["alg_bytes"] / 8e9) < 1e-9
        assert f["floor_ms"] == max(f["ns_ms_at_peak"], f["hbm_ms_at_peak"])
    # one 2048x2048 matrix at alpha 0.25 by hand: k = 512 rows of 2048, s = 512, l = 2048
    one = wls.Workload("one", "t", (wls.Group("g", 2048, 2048, 1),), (0.25,))
    f = bench.floors(one, 0.25)
    assert f["ns_flops"] == 5 * (4 * 512 ** 2 * 2048 + 2 * 512 ** 3)
    assert f["alg_bytes"] == 2048 * 2048 * 10 + 512 * 2048 * 12
