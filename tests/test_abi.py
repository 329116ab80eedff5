"""CPU tests of the C ABI: the library loads, exports every declared symbol,
and rejects invalid arguments before touching HIP. No compute call is made
(these run without a GPU)."""
import ctypes
import os
import re

import pytest

import oracle
from paper_2512_16928_amd import binding
from paper_2512_16928_amd.binding import (AXIS_AUTO, AXIS_COLS, AXIS_ROWS,
                                          DION2_ERR_INVALID_ARG, DION2_ERR_UNSUPPORTED,
                                          DION2_ERR_WORKSPACE, DION2_OK, Options)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dion2.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        from paper_2512_16928_amd import build
        build.build()
    return binding.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dion2_[a-z_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(binding.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_layouts_match_the_header(tmp_path):
    """The ctypes mirrors of dion2_options and dion2_group have the header's
    field offsets and sizes (a C program built with gcc against
    include/dion2.h prints them)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    lines = []
    for struct, mirror in (("dion2_options", Options), ("dion2_group", binding.Group)):
        lines.append(f'printf("{struct} size %zu\\n", sizeof({struct}));')
        for name, _ in mirror._fields_:
            lines.append(f'printf("{struct} {name} %zu\\n", offsetof({struct}, {name}));')
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "dion2.h"\nint main(void) {\n'
                   + "\n".join(lines) + "\nreturn 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True, capture_output=True, timeout=120)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=60).stdout
    c_side = {tuple(ln.split()[:2]): int(ln.split()[2]) for ln in out.splitlines()}
    for struct, mirror in (("dion2_options", Options), ("dion2_group", binding.Group)):
        assert c_side[(struct, "size")] == ctypes.sizeof(mirror), struct
        for name, _ in mirror._fields_:
            assert c_side[(struct, name)] == getattr(mirror, name).offset, (struct, name)


def test_version_and_status_strings(lib):
    assert binding.dion2_version() == 1
    for st in (0, -1, -2, -3, -4):
        assert binding.dion2_status_string(st).startswith("DION2_")
    assert "unknown" in binding.dion2_status_string(7)


def test_options_defaults(lib):
    opt = Options()
    lib.dion2_options_init(ctypes.byref(opt))
    assert opt.w_dtype == binding.DTYPE_BF16 and opt.g_dtype == binding.DTYPE_BF16
    assert abs(opt.ns_eps - 1e-7) < 1e-12
    assert opt.decay_all == 0 and not opt.workspace and not opt.dbg_update
    assert not opt.ns_coeffs
    assert opt.ns_form == binding.NS_AUTO and opt.select_rule == binding.SELECT_L1
    assert opt.rand_seed == 0 and opt.rand_step == 0 and opt.rand_matrix0 == 0
    assert opt.ns_chain == binding.CHAIN_HILO and opt.ns_master == binding.MASTER_BF16
    assert not opt.dbg_compact and not opt.dbg_compact_lo


FAKE = 0x10000   # a 256-aligned non-null address; never dereferenced below


def call_step(lib, W=FAKE, M=FAKE, G=FAKE, rows=64, cols=64, alpha=0.25, mu=0.95, lr=0.02,
              ns=5, axis=AXIS_AUTO):
    return lib.dion2_step(W, M, G, rows, cols, alpha, mu, lr, ns, axis, None)


@pytest.mark.parametrize("kw,msg", [
    (dict(W=None), "NULL"), (dict(M=None), "NULL"), (dict(G=None), "NULL"),
    (dict(rows=0), "rows"), (dict(cols=-3), "rows"),
    (dict(alpha=0.0), "alpha"), (dict(alpha=1.5), "alpha"), (dict(alpha=float("nan")), "alpha"),
    (dict(alpha=-0.25), "alpha"),
    (dict(mu=float("inf")), "mu"), (dict(lr=float("nan")), "lr"),
    (dict(ns=-1), "ns_steps"), (dict(ns=17), "ns_steps"),
    (dict(axis=2), "axis"), (dict(axis=-2), "axis"),
    (dict(W=FAKE + 8), "aligned"), (dict(G=FAKE + 2), "aligned"),
])
def test_invalid_arguments_rejected(lib, kw, msg):
    assert call_step(lib, **kw) == DION2_ERR_INVALID_ARG
    assert msg in binding.dion2_last_error()


def test_unsupported_sizes(lib):
    assert call_step(lib, rows=1 << 21, cols=8) == DION2_ERR_UNSUPPORTED
    assert call_step(lib, rows=65536, cols=65536) == DION2_ERR_UNSUPPORTED


def test_strided_and_batched_validation(lib):
    st = lib.dion2_step_strided(FAKE, FAKE, FAKE, 0, 64, 64, 0.25, 0.95, 0.02, 5, -1, None)
    assert st == DION2_ERR_INVALID_ARG and "batch" in binding.dion2_last_error()
    st = lib.dion2_step_strided(FAKE, FAKE, FAKE, 70000, 64, 64, 0.25, 0.95, 0.02, 5, -1, None)
    assert st == DION2_ERR_INVALID_ARG
    arr = ctypes.c_void_p * 2
    good, bad = arr(FAKE, FAKE), arr(FAKE, None)
    st = lib.dion2_step_batched(good, good, bad, 2, 64, 64, 0.25, 0.95, 0.02, 5, -1, None)
    assert st == DION2_ERR_INVALID_ARG and "matrix 1" in binding.dion2_last_error()
    st = lib.dion2_step_batched(None, good, good, 2, 64, 64, 0.25, 0.95, 0.02, 5, -1, None)
    assert st == DION2_ERR_INVALID_ARG


def test_ex_options_validation(lib):
    def ex(**o):
        opt = Options()
        lib.dion2_options_init(ctypes.byref(opt))
        for k, v in o.items():
            setattr(opt, k, v)
        return lib.dion2_step_ex(FAKE, FAKE, FAKE, 1, 64, 64, 0.25, 0.95, 0.02, 2, -1,
                                 ctypes.byref(opt), None)
    assert ex(w_dtype=5) == DION2_ERR_INVALID_ARG
    assert ex(g_dtype=-1) == DION2_ERR_INVALID_ARG
    assert ex(ns_eps=-1.0) == DION2_ERR_INVALID_ARG
    assert ex(decay_all=3) == DION2_ERR_INVALID_ARG
    assert ex(ns_form=3) == DION2_ERR_INVALID_ARG and "ns_form" in binding.dion2_last_error()
    assert ex(ns_form=-1) == DION2_ERR_INVALID_ARG
    assert ex(select_rule=2) == DION2_ERR_INVALID_ARG and "select_rule" in binding.dion2_last_error()
    assert ex(select_rule=1, rand_matrix0=-1) == DION2_ERR_INVALID_ARG
    assert ex(select_rule=1, rand_matrix0=1 << 32) == DION2_ERR_INVALID_ARG   # batch of 1
    assert "2^32" in binding.dion2_last_error()
    assert ex(ns_chain=2) == DION2_ERR_INVALID_ARG and "ns_chain" in binding.dion2_last_error()
    assert ex(ns_chain=-1) == DION2_ERR_INVALID_ARG
    big = (ctypes.c_float * 6)(1e5, 0.0, 0.0, 1e5, 0.0, 0.0)   # A_1 = 1e10 A_0, T_1 = 1e15 A_0
    big_p = ctypes.cast(big, ctypes.POINTER(ctypes.c_float))
    assert ex(ns_chain=binding.CHAIN_F16, ns_coeffs=big_p) == DION2_ERR_UNSUPPORTED
    assert "fp16" in binding.dion2_last_error()
    assert ex(ns_master=2) == DION2_ERR_INVALID_ARG and "ns_master" in binding.dion2_last_error()
    assert ex(ns_master=1, ns_chain=binding.CHAIN_F16) == DION2_ERR_INVALID_ARG
    assert ex(ns_master=1, ns_form=binding.NS_DIRECT) == DION2_ERR_UNSUPPORTED
    # the fp32 master also keeps X's lo half: more workspace than the AUTO plan
    need_auto = binding.dion2_workspace_size_ex(1, 64, 64, 0.25, AXIS_AUTO, 2)
    assert ex(ns_master=1, workspace=FAKE, workspace_bytes=need_auto) == DION2_ERR_WORKSPACE
    # the lo halves of X exist only with the fp32 master and a Newton-Schulz step
    assert ex(dbg_compact_lo=FAKE) == DION2_ERR_INVALID_ARG
    assert "dbg_compact_lo" in binding.dion2_last_error()
    opt = Options()
    lib.dion2_options_init(ctypes.byref(opt))
    opt.ns_master, opt.dbg_compact_lo = 1, FAKE
    st = lib.dion2_step_ex(FAKE, FAKE, FAKE, 1, 64, 64, 0.25, 0.95, 0.02, 0, -1, ctypes.byref(opt), None)
    assert st == DION2_ERR_INVALID_ARG and "ns_steps" in binding.dion2_last_error()
    coeffs = (ctypes.c_float * 6)(1.0, 2.0, 3.0, 1.0, float("inf"), 0.0)
    assert ex(ns_coeffs=ctypes.cast(coeffs, ctypes.POINTER(ctypes.c_float))) == DION2_ERR_INVALID_ARG
    need = binding.dion2_workspace_size_ex(1, 64, 64, 0.25, AXIS_AUTO, 2)
    assert ex(workspace=FAKE, workspace_bytes=need - 1) == DION2_ERR_WORKSPACE
    assert ex(workspace=FAKE + 16, workspace_bytes=need) == DION2_ERR_INVALID_ARG


def test_direct_form_step_limit(lib):
    """DIRECT rounds X to bf16 after every step; past DION2_DIRECT_MAX_STEPS
    a forced DIRECT is refused (nothing launched), and the header and the
    binding agree on the limit."""
    text = open(HEADER).read()
    limit = int(re.search(r"#define DION2_DIRECT_MAX_STEPS (\d+)", text).group(1))
    assert limit == 6

    def ex(ns, **o):
        opt = Options()
        lib.dion2_options_init(ctypes.byref(opt))
        for k, v in o.items():
            setattr(opt, k, v)
        return lib.dion2_step_ex(FAKE, FAKE, FAKE, 1, 384, 384, 0.5, 0.95, 0.02, ns, -1,
                                 ctypes.byref(opt), None)
    for ns in (limit + 1, 16):
        assert ex(ns, ns_form=binding.NS_DIRECT) == DION2_ERR_UNSUPPORTED
        assert "DIRECT" in binding.dion2_last_error()
        assert binding.dion2_workspace_size_ex(1, 384, 384, 0.5, AXIS_AUTO, ns, ns_form=binding.NS_DIRECT) == 0
    # a step count beyond the maximum is an invalid argument under any form
    assert ex(17, ns_form=binding.NS_DIRECT) == DION2_ERR_INVALID_ARG


@pytest.mark.parametrize("rows,cols,alpha,axis", [
    (256, 256, 0.25, AXIS_AUTO), (2048, 8192, 0.25, AXIS_AUTO), (8192, 2048, 0.5, AXIS_AUTO),
    (2048, 8192, 0.25, AXIS_COLS), (11008, 4096, 0.125, AXIS_AUTO), (2048, 1408, 0.25, AXIS_AUTO),
    (1408, 2048, 0.25, AXIS_AUTO), (7, 5, 0.1, AXIS_AUTO), (100, 37, 1e-4, AXIS_ROWS),
    (300, 300, 1.0, AXIS_COLS), (1000, 3, 0.3, AXIS_AUTO),
])
def test_plan_matches_oracle_reading(lib, rows, cols, alpha, axis):
    k, ax = binding.dion2_plan_info(rows, cols, alpha, axis)
    ax_o = oracle.resolve_axis(rows, cols, axis)
    assert ax == ax_o
    assert k == oracle.num_selected(alpha, rows if ax_o == AXIS_ROWS else cols)


def test_workspace_size(lib):
    ws_ex = binding.dion2_workspace_size_ex
    assert binding.dion2_workspace_size(0, 64, 64, 0.25) == 0
    assert binding.dion2_workspace_size(1, 64, 64, 2.0) == 0
    assert ws_ex(0, 64, 64, 0.25) == 0 and ws_ex(1, 64, 64, 2.0) == 0
    assert ws_ex(1, 64, 64, 0.25, AXIS_AUTO, 17) == 0
    assert ws_ex(1, 64, 64, 0.25, ns_master=binding.MASTER_FP32, ns_chain=binding.CHAIN_F16) == 0
    a = ws_ex(1, 2048, 2048, 0.25)
    b = ws_ex(2, 2048, 2048, 0.25)
    c = ws_ex(1, 2048, 2048, 1.0)
    assert 0 < a < b and a < c
    assert a % 256 == 0
    # k = 512 of 2048 with l = 4 s: the GRAM form, one bf16 compact matrix,
    # the fp32 result and ten bf16 s x s buffers
    assert a >= 512 * 2048 * (2 + 4) + 10 * 512 * 512 * 2
    # alpha = 1 (s = l = 2048): the DIRECT form, two bf16 compact buffers and
    # two of X^T (the update's B operand as rows), three s x s
    assert c >= 2048 * 2048 * (4 * 2 + 4) + 3 * 2048 * 2048 * 2
    # the Random rule with column selection adds per-block partial sums
    r = ws_ex(1, 8192, 2048, 0.25, select_rule=binding.SELECT_RANDOM)
    assert r >= ws_ex(1, 8192, 2048, 0.25) + (8192 // 64) * 512 * 8
    # past the DIRECT form's step limit AUTO takes GRAM: ten s x s buffers
    c7 = ws_ex(1, 2048, 2048, 1.0, AXIS_AUTO, 7)
    assert c7 == ws_ex(1, 2048, 2048, 1.0, AXIS_AUTO, 5, ns_form=binding.NS_GRAM) and c7 > c
    assert c7 >= 2048 * 2048 * (2 + 4) + 10 * 2048 * 2048 * 2
    # the size without options covers every option and step count
    rnd = binding.SELECT_RANDOM
    for shape in ((1, 2048, 2048, 0.25), (2, 2048, 2048, 1.0), (3, 640, 256, 0.5), (1, 300, 200, 0.75),
                  (1, 2048, 8192, 1.0), (2, 8192, 2048, 1.0), (2, 8192, 2048, 0.25)):
        top = binding.dion2_workspace_size(*shape)
        for kw in (dict(), dict(ns_form=binding.NS_DIRECT), dict(ns_form=binding.NS_GRAM),
                   dict(ns_master=binding.MASTER_FP32), dict(ns_chain=binding.CHAIN_F16),
                   dict(w_dtype=torch_f32(), g_dtype=torch_f32()), dict(select_rule=rnd),
                   dict(select_rule=rnd, ns_form=binding.NS_DIRECT), dict(select_rule=rnd, ns_form=binding.NS_GRAM)):
            for ns in (0, 1, 5, 6, 16):
                need = ws_ex(*shape, AXIS_AUTO, ns, **kw)
                assert need <= top, (shape, kw, ns)
                refused = kw.get("ns_form") == binding.NS_DIRECT and (ns > 6 or one_tile(*shape))
                assert need > 0 or refused, (shape, kw, ns)


def one_tile(batch, rows, cols, alpha, axis=AXIS_AUTO):
    """The compact matrix fits one 128-line tile a side."""
    k, ax = binding.dion2_plan_info(rows, cols, alpha, axis)
    d_oth = cols if ax == binding.AXIS_ROWS else rows
    return min(k, d_oth) <= 128


def test_direct_form_needs_more_than_one_tile(lib):
    """On a compact matrix of one tile a side the DIRECT form's bf16 rounding
    of X after every step can exceed the 2e-2 bound, so a forced DIRECT is
    refused there (nothing launched) while AUTO and GRAM run; from 129 lines
    it is accepted, and the size without options still covers every plan."""
    def ex(rows, cols, alpha, form):
        opt = Options()
        lib.dion2_options_init(ctypes.byref(opt))
        opt.ns_form = form
        return lib.dion2_step_ex(FAKE, FAKE, FAKE, 1, rows, cols, alpha, 0.95, 0.02, 5, -1,
                                 ctypes.byref(opt), None)
    for rows, cols, alpha in ((256, 256, 0.25), (640, 256, 0.5), (12, 68, 0.3), (1, 40, 1.0)):
        assert one_tile(1, rows, cols, alpha)
        assert ex(rows, cols, alpha, binding.NS_DIRECT) == DION2_ERR_UNSUPPORTED
        assert "DIRECT" in binding.dion2_last_error() and "128" in binding.dion2_last_error()
        assert binding.dion2_workspace_size_ex(1, rows, cols, alpha, AXIS_AUTO, 5, ns_form=binding.NS_DIRECT) == 0
        for form in (binding.NS_AUTO, binding.NS_GRAM):
            assert binding.dion2_workspace_size_ex(1, rows, cols, alpha, AXIS_AUTO, 5, ns_form=form) > 0
        assert binding.dion2_workspace_size(1, rows, cols, alpha) > 0
    for rows, cols, alpha in ((200, 328, 0.75), (257, 129, 1.0), (384, 384, 0.5)):
        assert not one_tile(1, rows, cols, alpha)
        assert binding.dion2_workspace_size_ex(1, rows, cols, alpha, AXIS_AUTO, 5, ns_form=binding.NS_DIRECT) > 0


def torch_f32():
    import torch
    return torch.float32


def test_status_codes_match_header():
    text = open(HEADER).read()
    for name, val in (("DION2_OK", DION2_OK), ("DION2_ERR_INVALID_ARG", DION2_ERR_INVALID_ARG),
                      ("DION2_ERR_UNSUPPORTED", DION2_ERR_UNSUPPORTED),
                      ("DION2_ERR_WORKSPACE", DION2_ERR_WORKSPACE)):
        assert re.search(rf"{name}\s*=\s*{val}\b", text), name
    for name, val in (("DION2_AXIS_AUTO", AXIS_AUTO), ("DION2_AXIS_ROWS", AXIS_ROWS),
                      ("DION2_AXIS_COLS", AXIS_COLS)):
        assert re.search(rf"{name}\s*=\s*{val}\b", text), name


def groups_array(specs):
    arr = (binding.Group * max(len(specs), 1))()
    for i, kw in enumerate(specs):
        g = dict(W=FAKE, M=FAKE, G=FAKE, batch=2, rows=64, cols=64, axis=AXIS_AUTO)
        g.update(kw)
        arr[i] = binding.Group(g["W"], g["M"], g["G"], g["batch"], g["rows"], g["cols"], g["axis"])
    return arr


@pytest.mark.parametrize("specs,n,opt_kw,msg", [
    ([{}], 0, {}, "ngroups"),
    ([{}], 65, {}, "ngroups"),
    ([{}, {"W": None}], 2, {}, "NULL"),
    ([{}, {"G": FAKE + 4}], 2, {}, "aligned"),
    ([{"rows": 0}], 1, {}, "rows"),
    ([{}, {"axis": 5}], 2, {}, "axis"),
    ([{"batch": 0}], 1, {}, "batch"),
    ([{}], 1, {"workspace": FAKE, "workspace_bytes": 1 << 30}, "workspace"),
    ([{}], 1, {"dbg_norms": FAKE}, "debug"),
    ([{}], 1, {"dbg_compact": FAKE}, "debug"),
    ([{}], 1, {"dbg_compact_lo": FAKE, "ns_master": 1}, "debug"),
    ([{}], 1, {"select_rule": 7}, "select_rule"),
    ([{"batch": 3}, {"batch": 3}], 2, {"select_rule": 1, "rand_matrix0": (1 << 32) - 5}, "rand_matrix0"),
])
def test_groups_validation(lib, specs, n, opt_kw, msg):
    arr = groups_array(specs)
    opt = Options()
    lib.dion2_options_init(ctypes.byref(opt))
    for k, v in opt_kw.items():
        setattr(opt, k, v)
    st = binding.dion2_step_groups_raw(arr, n, 0.25, 0.95, 0.02, 5, opt, None)
    assert st == DION2_ERR_INVALID_ARG
    assert msg in binding.dion2_last_error()


def test_groups_null_array(lib):
    assert binding.dion2_step_groups_raw(None, 1, 0.25, 0.95, 0.02, 5, None, None) == DION2_ERR_INVALID_ARG


def test_groups_stream_count_validated(lib):
    arr = groups_array([{}])
    opt = Options()
    lib.dion2_options_init(ctypes.byref(opt))
    assert opt.group_streams == 0
    for bad in (-1, 9):
        opt.group_streams = bad
        assert binding.dion2_step_groups_raw(arr, 1, 0.25, 0.95, 0.02, 5, opt, None) == DION2_ERR_INVALID_ARG
        assert "group_streams" in binding.dion2_last_error()


def test_noalloc_validation(lib):
    """dion2_step_noalloc validates like dion2_step_ex, refuses a workspace of
    the caller's, and refuses a plan beyond its scratch array before any HIP
    call."""
    text = open(HEADER).read()
    assert re.search(r"#define DION2_NOALLOC_SCRATCH_BYTES \(\(size_t\)128 << 20\)", text)
    assert binding.NOALLOC_SCRATCH_BYTES == 128 << 20

    def na(rows=64, cols=64, batch=1, alpha=0.25, ns=5, **o):
        opt = Options()
        lib.dion2_options_init(ctypes.byref(opt))
        for k, v in o.items():
            setattr(opt, k, v)
        return lib.dion2_step_noalloc(FAKE, FAKE, FAKE, batch, rows, cols, alpha, 0.95, 0.02, ns, -1,
                                      ctypes.byref(opt), None)
    assert na(alpha=0.0) == DION2_ERR_INVALID_ARG
    assert na(ns=17) == DION2_ERR_INVALID_ARG
    assert na(workspace=FAKE, workspace_bytes=1 << 30) == DION2_ERR_INVALID_ARG
    assert "workspace" in binding.dion2_last_error()
    big = (16, 2048, 8192, 1.0)
    assert binding.dion2_workspace_size_ex(*big) > binding.NOALLOC_SCRATCH_BYTES
    assert na(rows=2048, cols=8192, batch=16, alpha=1.0) == DION2_ERR_WORKSPACE
    assert "scratch" in binding.dion2_last_error()


def _pad(n):
    return (n + 127) // 128 * 128


@pytest.mark.parametrize("rows,cols,alpha,steps", [
    (2048, 2048, 0.25, 5),    # s = 512, l = 2048 = 4 s: GRAM
    (2048, 2048, 0.5, 5),     # s = 1024, l = 2048: DIRECT
    (2048, 2048, 1.0, 5),     # s = l = 2048: DIRECT
    (2048, 2048, 1.0, 6),     # DIRECT up to DION2_DIRECT_MAX_STEPS
    (2048, 2048, 1.0, 7),     # past it: GRAM
    (8192, 2048, 0.25, 5),    # columns: s = 512, l = 8192
    (256, 256, 0.25, 5),      # s = 64: one tile, GRAM
    (300, 200, 0.75, 5),      # columns: s = 150, l = 300 (padded 256 and 384): DIRECT
    (129, 900, 1.0, 5),       # s = 129, l = 900 (padded 256 and 1024 >= 3 x 256): GRAM
])
def test_plan_form_auto(lib, rows, cols, alpha, steps):
    """AUTO takes GRAM where the padded compact matrix is at least three
    times as long as high, fits one tile a side, or the schedule is longer
    than DIRECT's limit, else DIRECT; host-only, as the step resolves it."""
    form, chain, fused = binding.dion2_plan_form(1, rows, cols, alpha, AXIS_AUTO, steps)
    k, ax = binding.dion2_plan_info(rows, cols, alpha, AXIS_AUTO)
    d_oth = cols if ax == AXIS_ROWS else rows
    s, l = _pad(min(k, d_oth)), _pad(max(k, d_oth))
    gram = l >= 3 * s or s <= 128 or steps > 6
    assert form == (binding.NS_GRAM if gram else binding.NS_DIRECT)
    assert chain == binding.CHAIN_HILO
    assert fused == int(gram and min(k, d_oth) <= 64)


@pytest.mark.parametrize("rows,cols,steps,want", [
    (664, 235, 5, False),     # l = 2.8 s (padded sides 768 = 3 x 256): hi/lo
    (1024, 256, 5, True),     # l = 4 s
    (256, 1100, 5, True),     # columns of the transpose, l = 4.3 s
    (1024, 256, 1, False),    # one step: no product to gain
    (1024, 60, 5, False),     # s = 60: the one-launch chain stays hi/lo
    (2048, 1024, 5, False),   # l = 2 s: DIRECT
])
def test_plan_form_f16_chain_rule(lib, rows, cols, steps, want):
    """An fp16-chain request is taken only by a chain of launches on a
    compact matrix at least four times as long as high (real sides)."""
    form, chain, fused = binding.dion2_plan_form(1, rows, cols, 1.0, AXIS_AUTO, steps,
                                                 ns_chain=binding.CHAIN_F16)
    assert chain == (binding.CHAIN_F16 if want else binding.CHAIN_HILO), (form, chain, fused)
    if want:
        assert form == binding.NS_GRAM and not fused


def test_plan_form_fused_chain_and_refusals(lib):
    """s <= 64 runs the chain as one launch unless one launch per product is
    asked for; no steps, no chain; a call the step would refuse raises the
    same status."""
    assert binding.dion2_plan_form(1, 256, 256, 0.25, AXIS_ROWS, 5) == (binding.NS_GRAM, binding.CHAIN_HILO, 1)
    assert binding.dion2_plan_form(1, 256, 256, 0.25, AXIS_ROWS, 5, ns_chain_per_product=True)[2] == 0
    assert binding.dion2_plan_form(1, 256, 256, 0.25, AXIS_ROWS, 0)[2] == 0
    assert binding.dion2_plan_form(1, 260, 1000, 0.25, AXIS_ROWS, 5)[2] == 0      # s = 65
    assert binding.dion2_plan_form(1, 2048, 2048, 1.0, AXIS_AUTO, 5,
                                   ns_master=binding.MASTER_FP32)[0] == binding.NS_GRAM
    refused = [
        (dict(ns_form=binding.NS_DIRECT), (1, 256, 256, 0.25, 5), DION2_ERR_UNSUPPORTED),   # one tile
        (dict(ns_form=binding.NS_DIRECT), (1, 2048, 2048, 1.0, 7), DION2_ERR_UNSUPPORTED),  # > 6 steps
        (dict(ns_master=binding.MASTER_FP32, ns_form=binding.NS_DIRECT), (1, 2048, 2048, 1.0, 5),
         DION2_ERR_UNSUPPORTED),
        (dict(ns_master=binding.MASTER_FP32, ns_chain=binding.CHAIN_F16), (1, 2048, 2048, 0.25, 5),
         DION2_ERR_INVALID_ARG),
        (dict(ns_chain=binding.CHAIN_F16, ns_coeffs=[(3e6, 0.0, 0.0)] * 5), (1, 1024, 256, 1.0, 5),
         DION2_ERR_UNSUPPORTED),   # the chain's values beyond fp16's range
        (dict(), (0, 256, 256, 0.25, 5), DION2_ERR_INVALID_ARG),
        (dict(), (1, 256, 256, 0.25, 17), DION2_ERR_INVALID_ARG),
    ]
    for kw, (batch, rows, cols, alpha, steps), status in refused:
        with pytest.raises(binding.Dion2Error) as ei:
            binding.dion2_plan_form(batch, rows, cols, alpha, AXIS_AUTO, steps, **kw)
        assert ei.value.status == status, (kw, ei.value)
