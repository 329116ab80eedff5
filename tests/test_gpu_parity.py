"""GPU parity: the HIP Dion2 step against the CPU oracle, element by element.

Acceptance (per matrix):
  * selected indices K equal the oracle's exactly (ties to the lower index);
  * the l1 line norms equal the oracle's exactly rounded sums bitwise;
  * the momentum M equals the oracle's fp32 result bitwise;
  * where a test asks for it (debug output dbg_compact), the compact bf16
    matrix X equals the oracle's normalised lines rounded in the kernel's
    precision, bitwise;
  * the Newton-Schulz output O (debug output, before the lr scale) is within
    relative Frobenius error 2e-2 of the oracle's fp64 result (bf16 and fp16
    MFMA);
  * W equals the oracle's update rule applied to the GPU's O bitwise, so
    unselected lines are untouched and the selected ones are rounded once.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2512_16928_amd import binding, workloads
from paper_2512_16928_amd.binding import AXIS_AUTO, AXIS_COLS, AXIS_ROWS, NS_DIRECT, NS_GRAM

pytestmark = pytest.mark.gpu

NS_TOL = 2e-2


def rel_fro(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def rounded_input_iteration(M, G, b, alpha, steps, axis, coeffs=None, eps=1e-7, rand=None):
    """The oracle's Newton-Schulz output for matrix b of the stack, and the
    exact iteration applied to its compact X / (||X||_F + eps) rounded once
    to bf16, the precision the default path takes X in (both in the compact
    matrix's own orientation; the second is None for a zero X or no steps)."""
    M0, Gb = M[b].cpu().numpy(), G[b].float().cpu().numpy()
    sel = dict(select="random", seed=rand[0], step=rand[1], matrix=rand[2] + b) if rand is not None else {}
    eps = float(np.float32(eps))
    out = oracle.dion2_step(np.zeros(M0.shape), M0, Gb, alpha, 0.95, 0.02, steps, axis, coeffs, eps=eps, **sel)
    X = oracle.gather(oracle.momentum_accumulate(M0, Gb), out["K"], out["axis"])
    nx = np.linalg.norm(X)
    if steps == 0 or not np.isfinite(nx) or nx == 0.0:
        return out["O"], None
    Z = oracle.round_bf16(X / (nx + eps))
    # eps chosen so that the oracle divides Z by exactly one, not by its norm
    return out["O"], oracle.newton_schulz(Z, steps, coeffs, eps=1.0 - np.linalg.norm(Z))


def rounding_floor(M, G, b, alpha, steps, axis, coeffs=None, eps=1e-7, rand=None):
    """The relative Frobenius distance between the exact iteration on matrix
    b's compact X and the exact iteration on X rounded once to bf16: the
    least error a path that rounds its input to bf16 can show. Compact
    matrices of a few lines with a small singular value, long quintic
    schedules and momentum of low rank plus a little noise can put it near
    or past the 2e-2 bound by itself."""
    O, Or = rounded_input_iteration(M, G, b, alpha, steps, axis, coeffs, eps, rand)
    return 0.0 if Or is None else rel_fro(Or, O)


FORMS = pytest.mark.parametrize("form", [NS_DIRECT, NS_GRAM], ids=["direct", "gram"])
CHAINS = pytest.mark.parametrize("chain", [binding.CHAIN_HILO, binding.CHAIN_F16], ids=["hilo", "f16"])


def run_gpu(W, M, G, alpha, ns_steps=5, axis=AXIS_AUTO, mu=0.95, lr=0.02, coeffs=None,
            decay_all=False, form=binding.NS_AUTO, rand=None, chain=binding.CHAIN_HILO,
            master=binding.MASTER_BF16, eps=1e-7, dbg_compact=None, dbg_compact_lo=None, norms=True,
            per_product=False):
    """One library call on stacks [B, rows, cols]; returns host copies and the
    debug outputs (norms=False leaves out the l1 norms, which the Random
    rule's single column pass does not compute)."""
    B, rows, cols = W.shape
    k, ax = binding.dion2_plan_info(rows, cols, alpha, axis)
    d_sel, d_oth = (rows, cols) if ax == AXIS_ROWS else (cols, rows)
    dev = W.device
    sel = torch.full((B, k), -1, dtype=torch.int32, device=dev)
    nrm = torch.full((B, d_sel), -1.0, dtype=torch.float64, device=dev)
    upd = torch.full((B, k, d_oth), float("nan"), dtype=torch.float32, device=dev)
    W0, M0 = W.cpu(), M.cpu()
    extra = {}
    if rand is not None:   # (seed, step, first matrix index): the Random rule
        extra = dict(select_rule=binding.SELECT_RANDOM, rand_seed=rand[0], rand_step=rand[1],
                     rand_matrix0=rand[2])
    binding.dion2_step_ex(W, M, G, alpha, mu, lr, ns_steps, axis, ns_coeffs=coeffs, ns_eps=eps,
                          decay_all=decay_all, dbg_sel_idx=sel, dbg_norms=nrm if norms else None, dbg_update=upd,
                          ns_form=form, ns_chain=chain, ns_master=master, dbg_compact=dbg_compact,
                          dbg_compact_lo=dbg_compact_lo, ns_chain_per_product=per_product, **extra)
    torch.cuda.synchronize()
    return dict(W=W.cpu(), M=M.cpu(), K=sel.cpu(), norms=nrm.cpu() if norms else None, O=upd.cpu(), W0=W0, M0=M0,
                G=G.cpu(), axis=ax, k=k)


def one_tile(rows, cols, alpha, axis=AXIS_AUTO):
    """The compact matrix fits one 128-line tile a side."""
    k, ax = binding.dion2_plan_info(rows, cols, alpha, axis)
    return min(k, cols if ax == AXIS_ROWS else rows) <= 128


def direct_refused(W, M, G, alpha, axis=AXIS_AUTO, form=NS_DIRECT):
    """A forced DIRECT on a compact matrix of one tile a side is refused before
    anything runs (its bf16 rounding of X can break the 2e-2 bar there). True
    after checking that; False where the call should run."""
    if form != NS_DIRECT or not one_tile(W.shape[-2], W.shape[-1], alpha, axis):
        return False
    W1, M1 = W.clone(), M.clone()
    with pytest.raises(binding.Dion2Error) as ei:
        binding.dion2_step_ex(W1, M1, G, alpha, 0.95, 0.02, 5, axis, ns_form=NS_DIRECT)
    assert ei.value.status == binding.DION2_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.equal(W1, W) and torch.equal(M1, M), "a refused call modified state"
    return True


def check_matrix(res, b, alpha, ns_steps=5, axis=AXIS_AUTO, mu=0.95, lr=0.02, coeffs=None,
                 decay_all=False, ns_tol=NS_TOL, rand=None, eps=1e-7, ns_ref=None):
    """K, the l1 norms, M and W (given O) against the oracle, and O within
    ns_tol of the oracle's exact iteration, or of ns_ref (the compact matrix's
    own orientation) where given."""
    wdt = "bf16" if res["W0"].dtype == torch.bfloat16 else "f32"
    W0 = res["W0"][b].float().numpy().astype(np.float64)
    M0 = res["M0"][b].numpy()
    G = res["G"][b].float().numpy()
    sel_kw = {}
    if rand is not None:
        sel_kw = dict(select="random", seed=rand[0], step=rand[1], matrix=rand[2] + b)
    out = oracle.dion2_step(W0, M0, G, alpha, mu, lr, ns_steps, axis, coeffs, eps=float(np.float32(eps)),
                            w_dtype=wdt, decay_all=decay_all, **sel_kw)
    assert out["axis"] == res["axis"] and out["k"] == res["k"]
    K = res["K"][b].numpy().astype(np.int64)
    np.testing.assert_array_equal(K, out["K"], err_msg="selected indices")
    if res["norms"] is not None:
        np.testing.assert_array_equal(res["norms"][b].numpy(), out["norms"], err_msg="l1 norms")
    np.testing.assert_array_equal(res["M"][b].numpy(), out["M"], err_msg="momentum")
    O_gpu = res["O"][b].numpy().astype(np.float64)          # [k, d_oth]
    O_ref = out["O"] if ns_ref is None else ns_ref
    O_ref = O_ref if out["axis"] == AXIS_ROWS else O_ref.T
    err = rel_fro(O_gpu, O_ref)
    assert err <= ns_tol, f"Newton-Schulz rel. Frobenius error {err:.3e} > {ns_tol}"
    O_paper = O_gpu if out["axis"] == AXIS_ROWS else O_gpu.T
    W_want = oracle.apply_update(W0, K, O_paper, lr, out["axis"], wdt)
    np.testing.assert_array_equal(res["W"][b].float().numpy().astype(np.float64), W_want,
                                  err_msg="weights")
    return err


def one_group_workload(rows, cols, count=1, axis=AXIS_AUTO, w_dtype="bf16", g_std=1e-3,
                       name="custom"):
    return workloads.Workload(name, "test", (workloads.Group("g", rows, cols, count, axis),),
                              (0.25,), w_dtype=w_dtype, g_std=g_std)


def test_single_256_fp32_full(hip_device):
    wl = workloads.WORKLOADS["single-256"]
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, 0.25, axis=AXIS_ROWS)
    assert res["k"] == 64
    check_matrix(res, 0, 0.25, axis=AXIS_ROWS)


@pytest.mark.parametrize("rows,cols,alpha,axis,wdt", [
    (200, 328, 0.25, AXIS_AUTO, "bf16"),     # rows, k = 50, ragged tiles
    (328, 200, 0.25, AXIS_AUTO, "bf16"),     # columns, k = 50
    (130, 75, 0.5, AXIS_AUTO, "bf16"),       # cols % 4 != 0: scalar paths
    (96, 1000, 0.5, AXIS_AUTO, "f32"),
    (257, 129, 1.0, AXIS_AUTO, "bf16"),      # alpha = 1 (Muon), columns
    (64, 256, 0.5, AXIS_COLS, "bf16"),       # k = 128 > d_oth = 64: iterate on L^T
    (300, 200, 0.75, AXIS_ROWS, "f32"),      # k = 225 > d_oth = 200, rows
    (1, 40, 1.0, AXIS_AUTO, "bf16"),         # a single row
    (384, 640, 0.1, AXIS_AUTO, "bf16"),      # alpha not a power of two
    (200, 96, 0.5, AXIS_AUTO, "f32"),        # columns, fp32 W, one row per wave
    (40, 4616, 0.5, AXIS_COLS, "bf16"),      # columns beyond 4096: 512-column strips
    (24, 4104, 0.25, AXIS_COLS, "f32"),      # the same with fp32 W, ragged last strip
    (64, 2048, 0.75, AXIS_COLS, "bf16"),     # k = 1536: one row per wave, two passes of ranks
    (48, 4096, 1.0, AXIS_COLS, "bf16"),      # k = 4096, the widest row of the LDS buffer
    (40, 2048, 0.6, AXIS_COLS, "f32"),       # fp32 W, k = 1229 (ragged last pass)
    (100, 250, 0.3, AXIS_ROWS, "bf16"),      # rows, cols % 4 != 0: scalar row apply
    (64, 100, 0.5, AXIS_ROWS, "bf16"),       # rows, cols % 8 = 4: vector row apply, no fused update
    (90, 154, 0.4, AXIS_ROWS, "f32"),        # rows, fp32 W, cols % 4 != 0
])
@FORMS
def test_ragged_shapes(hip_device, rows, cols, alpha, axis, wdt, form):
    wl = one_group_workload(rows, cols, axis=axis, w_dtype=wdt, name=f"r{rows}c{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    if direct_refused(W, M, G, alpha, axis, form):
        return
    res = run_gpu(W, M, G, alpha, axis=axis, form=form)
    check_matrix(res, 0, alpha, axis=axis)


@pytest.mark.parametrize("rows,cols,alpha,axis,wdt", [
    (200, 328, 0.75, AXIS_AUTO, "bf16"),     # rows, s = 150, ragged tiles both ways
    (328, 200, 0.75, AXIS_AUTO, "bf16"),     # columns, s = 150
    (330, 175, 0.9, AXIS_AUTO, "bf16"),      # columns, cols % 4 != 0: scalar paths
    (160, 1000, 1.0, AXIS_AUTO, "f32"),      # fp32 W
    (300, 200, 0.75, AXIS_ROWS, "f32"),      # k = 225 > d_oth = 200: iterate on L^T
    (140, 250, 1.0, AXIS_ROWS, "bf16"),      # rows, cols % 4 != 0: scalar row apply
    (136, 300, 1.0, AXIS_ROWS, "bf16"),      # rows, cols % 8 = 4: vector row apply, no fused update
    (150, 154, 1.0, AXIS_ROWS, "f32"),       # rows, fp32 W, cols % 4 != 0
])
def test_direct_ragged_shapes(hip_device, rows, cols, alpha, axis, wdt):
    """The DIRECT form on ragged shapes beyond one tile (it is refused on one)."""
    assert not one_tile(rows, cols, alpha, axis)
    wl = one_group_workload(rows, cols, axis=axis, w_dtype=wdt, name=f"dr{rows}c{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, alpha, axis=axis, form=NS_DIRECT)
    check_matrix(res, 0, alpha, axis=axis)


@pytest.mark.parametrize("axis", [AXIS_ROWS, AXIS_COLS])
def test_strided_batch(hip_device, axis):
    wl = one_group_workload(192, 320, count=3, axis=axis, name=f"batch{axis}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, 0.25, axis=axis)
    for b in range(3):
        check_matrix(res, b, 0.25, axis=axis)


def test_batched_pointer_tables_equal_strided(hip_device):
    wl = one_group_workload(256, 384, count=4, name="tables")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2 = W.clone(), M.clone()
    binding.dion2_step_strided(W, M, G, 0.25)
    binding.dion2_step_batched([W2[i] for i in range(4)], [M2[i] for i in range(4)],
                               [G[i] for i in range(4)], 0.25)
    torch.cuda.synchronize()
    assert torch.equal(W, W2) and torch.equal(M, M2)


def test_plain_entry_point_equals_ex(hip_device):
    wl = one_group_workload(256, 512, count=1, name="plain")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2 = W.clone(), M.clone()
    binding.dion2_step(W[0], M[0], G[0], 0.25)
    binding.dion2_step_ex(W2, M2, G, 0.25)
    torch.cuda.synchronize()
    assert torch.equal(W, W2) and torch.equal(M, M2)


@pytest.mark.parametrize("ns_steps,coeffs", [
    (0, None), (1, None), (3, [(1.5, -0.5, 0.0)] * 3),
    (4, [(3.0, -3.2, 1.2), (2.0, -1.5, 0.5), (1.5, -0.5, 0.0), (1.5, -0.5, 0.0)]),
])
@pytest.mark.parametrize("rows,cols", [(288, 768), (768, 288)], ids=["rowsel", "colsel"])
@FORMS
def test_ns_schedules(hip_device, ns_steps, coeffs, form, rows, cols):
    wl = one_group_workload(rows, cols, name=f"sched{ns_steps}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, 0.5, ns_steps=ns_steps, coeffs=coeffs, form=form)
    check_matrix(res, 0, 0.5, ns_steps=ns_steps, coeffs=coeffs)


@pytest.mark.parametrize("rows,cols,ns_steps", [
    (2048, 2176, 5),   # rows: l = 2176 (not a multiple of 256), update and fused apply on 256 x 128 tiles
    (2176, 2048, 5),   # columns: the final product writes O transposed, 256 x 128 tiles
    (2048, 2048, 1),   # one step: X_0^T straight into the final product
])
def test_direct_transposed_operand(hip_device, rows, cols, ns_steps):
    """From s = 2048 the DIRECT form keeps X^T beside X and runs the update
    B X with X^T as the B operand's rows (X_0^T from a transpose, later ones
    written by the update's epilogue)."""
    wl = one_group_workload(rows, cols, name=f"xrows{rows}c{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, 1.0, ns_steps=ns_steps, form=NS_DIRECT)
    assert res["k"] == 2048
    check_matrix(res, 0, 1.0, ns_steps=ns_steps)


@pytest.mark.parametrize("grow", [10, 21], ids=["fp16-scaled-down", "hilo-fallback"])
def test_direct_a_range(hip_device, grow):
    """The DIRECT form keeps A = X X^T in fp16 with a power-of-two scale bounded
    from the coefficients. A first step X <- 2^g X followed by a quintic step
    with b and c rescaled by 2^-2g and 2^-4g gives 2^g times one ordinary
    step. g = 10 puts A near 2^20 (stored scaled down by 2^-7); g = 21 takes A
    past the 2^40 that the fp16 path accepts, so A stays a bf16 hi/lo pair and
    A^2 takes three passes. Both match the oracle."""
    g = float(2 ** grow)
    coeffs = [(g, 0.0, 0.0), (3.4445, -4.7750 / g ** 2, 2.0315 / g ** 4)]
    wl = one_group_workload(160, 384, name=f"arange{grow}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, 1.0, ns_steps=2, coeffs=coeffs, form=NS_DIRECT)
    check_matrix(res, 0, 1.0, ns_steps=2, coeffs=coeffs)


@pytest.mark.parametrize("ns_steps,coeffs", [
    (2, None), (3, [(1.5, -0.5, 0.0)] * 3),
    (4, [(3.0, -3.2, 1.2), (2.0, -1.5, 0.5), (1.5, -0.5, 0.0), (1.5, -0.5, 0.0)]),
    (8, [(3.4445, -4.7750, 2.0315)] * 6 + [(1.875, -1.25, 0.375)] * 2),
])
def test_f16_chain_schedules(hip_device, ns_steps, coeffs):
    """The fp16 chain takes its scales from the coefficients: forced on a
    per-step schedule it stays within tolerance of the oracle."""
    wl = one_group_workload(160, 640, name=f"f16sched{ns_steps}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, 0.5, ns_steps=ns_steps, coeffs=coeffs, form=NS_GRAM,
                  chain=binding.CHAIN_F16)
    check_matrix(res, 0, 0.5, ns_steps=ns_steps, coeffs=coeffs)


def test_f16_chain_of_one_step_is_hilo(hip_device):
    """A chain of one step has no product to gain from fp16: it runs in hi/lo."""
    wl = one_group_workload(128, 512, count=2, name="f16one")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2 = W.clone(), M.clone()
    binding.dion2_step_ex(W, M, G, 0.5, 0.95, 0.02, 1, ns_form=NS_GRAM, ns_chain=binding.CHAIN_F16)
    binding.dion2_step_ex(W2, M2, G, 0.5, 0.95, 0.02, 1, ns_form=NS_GRAM, ns_chain=binding.CHAIN_HILO)
    torch.cuda.synchronize()
    assert torch.equal(W.view(torch.int16), W2.view(torch.int16)) and torch.equal(M, M2)


@pytest.mark.parametrize("rows,cols,taken", [
    (664, 235, False),   # s = 235, l = 664 = 2.8 s (padded 256 and 768: three times)
    (1024, 256, True),   # s = 256, l = 1024 = 4 s
    (256, 1100, True),   # columns of the transpose: s = 256, l = 1100
])
def test_f16_chain_needs_four_times_as_long(hip_device, rows, cols, taken):
    """The fp16 chain is taken only where the compact matrix is at least four
    times as long as it is high (real sides); elsewhere an fp16 request runs
    the hi/lo chain, bitwise."""
    wl = one_group_workload(rows, cols, name=f"f16w{rows}c{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    k, ax = binding.dion2_plan_info(rows, cols, 1.0, AXIS_AUTO)
    d_oth = cols if ax == AXIS_ROWS else rows
    assert (max(k, d_oth) >= 4 * min(k, d_oth)) == taken
    out = {}
    for chain in (binding.CHAIN_HILO, binding.CHAIN_F16):
        W1, M1 = W.clone(), M.clone()
        binding.dion2_step_ex(W1, M1, G, 1.0, 0.95, 0.02, 5, ns_form=NS_GRAM, ns_chain=chain)
        torch.cuda.synchronize()
        out[chain] = W1.view(torch.int16).cpu()
    assert torch.equal(out[binding.CHAIN_HILO], out[binding.CHAIN_F16]) != taken
    res = run_gpu(W, M, G, 1.0, axis=AXIS_AUTO, form=NS_GRAM, chain=binding.CHAIN_F16)
    check_matrix(res, 0, 1.0, axis=AXIS_AUTO)


@pytest.mark.parametrize("wl_name,gi,first,alpha,ratio", [
    ("1b", 0, 9, 0.25, 2.0),          # 2048x2048: s = 512, l = 2048
    ("1b", 1, 4, 0.25, 2.0),          # 8192x2048, columns: s = 512, l = 8192
    ("1b-colsel", 2, 3, 0.25, 2.0),   # 5% of the columns with x20 gradients
    ("moe", 0, 70, 0.25, 2.0),        # 2048x1408 expert: s = 352 padded to 384
    ("1b", 2, 4, 0.5, 2.0),           # 2048x8192, rows: s = 1024, l = 8192
    ("1b", 1, 6, 1.0, 4.0),           # 8192x2048, columns: s = 2048 (256 x 256 fp16 tiles)
])
def test_gram_chain_storage(hip_device, wl_name, gi, first, alpha, ratio):
    """Both storages of the GRAM chain against the oracle on one matrix of a
    benchmark shape. The fp16 chain keeps 11 significant bits where the hi/lo
    pairs keep about 16; on these wide, balanced matrices Z's own bf16
    rounding dominates both, and fp16 stays within twice the hi/lo error. At
    alpha = 1 the compact matrix is the whole momentum (smallest singular
    value 4.6e-3 of X / ||X||_F): fp16 measures 7.5e-3 against 2.3e-3 for
    hi/lo, still inside the 2e-2 bound that check_matrix applies."""
    wl = workloads.WORKLOADS[wl_name]
    grp = wl.groups[gi]
    W, M, G = workloads.make_group(wl, gi, hip_device, first=first, count=1)
    errs = {}
    for chain in (binding.CHAIN_HILO, binding.CHAIN_F16):
        res = run_gpu(W.clone(), M.clone(), G, alpha, axis=grp.axis, form=NS_GRAM, chain=chain)
        errs[chain] = check_matrix(res, 0, alpha, axis=grp.axis)
    assert errs[binding.CHAIN_F16] <= ratio * errs[binding.CHAIN_HILO] + 1e-3, errs


@pytest.mark.parametrize("rows,cols,alpha,axis", [
    (200, 328, 0.25, AXIS_AUTO),    # rows, s = 50, l = 328
    (328, 200, 0.25, AXIS_AUTO),    # columns, s = 50
    (130, 75, 0.5, AXIS_AUTO),      # columns, s = 38, l = 130
    (384, 640, 0.1, AXIS_AUTO),     # rows, s = 39
    (256, 1024, 0.5, AXIS_ROWS),    # s = 128: one whole tile
    (640, 1664, 0.3, AXIS_ROWS),    # s = 192 padded to 256: mirrored off-diagonal tiles
])
def test_f16_chain_ragged(hip_device, rows, cols, alpha, axis):
    """The fp16 chain on ragged wide shapes (padding inside the s x s tiles)."""
    wl = one_group_workload(rows, cols, axis=axis, name=f"f16r{rows}c{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, alpha, axis=axis, form=NS_GRAM, chain=binding.CHAIN_F16)
    check_matrix(res, 0, alpha, axis=axis)


MASTER_TOL = 2e-3   # fp32 master: X as a hi/lo pair, about 16 significant bits throughout

SCHEDULE = [(3.4445, -4.7750, 2.0315)] * 3 + [(1.5, -0.5, 0.0)] * 2


@pytest.mark.parametrize("rows,cols,alpha,axis,wdt,steps,coeffs,chain,master", [
    (200, 328, 0.25, AXIS_AUTO, "bf16", 5, None, binding.CHAIN_HILO, binding.MASTER_BF16),   # rows, s = 50
    (328, 200, 0.25, AXIS_AUTO, "bf16", 5, None, binding.CHAIN_HILO, binding.MASTER_BF16),   # columns, s = 50
    (256, 256, 0.25, AXIS_ROWS, "f32", 5, None, binding.CHAIN_HILO, binding.MASTER_BF16),    # fp32 W, s = 64
    (96, 1000, 0.25, AXIS_AUTO, "bf16", 5, None, binding.CHAIN_HILO, binding.MASTER_BF16),   # s = 24: one block
    (64, 256, 0.5, AXIS_COLS, "bf16", 5, None, binding.CHAIN_HILO, binding.MASTER_BF16),     # Z = L^T, s = 64
    (130, 75, 0.5, AXIS_AUTO, "bf16", 1, None, binding.CHAIN_HILO, binding.MASTER_BF16),     # P = Q_0
    (130, 75, 0.5, AXIS_AUTO, "bf16", 2, None, binding.CHAIN_HILO, binding.MASTER_BF16),
    (200, 328, 0.25, AXIS_AUTO, "bf16", 16, None, binding.CHAIN_HILO, binding.MASTER_BF16),  # the longest schedule
    (200, 328, 0.25, AXIS_AUTO, "bf16", 5, SCHEDULE, binding.CHAIN_HILO, binding.MASTER_BF16),
    (200, 328, 0.25, AXIS_AUTO, "bf16", 5, None, binding.CHAIN_F16, binding.MASTER_BF16),    # runs in hi / lo
    (200, 328, 0.25, AXIS_AUTO, "bf16", 5, None, binding.CHAIN_HILO, binding.MASTER_FP32),
])
def test_fused_small_chain(hip_device, rows, cols, alpha, axis, wdt, steps, coeffs, chain, master):
    """A GRAM chain with s <= 64 runs in one launch, its matrices in LDS: bitwise
    the chain with one launch per product (hi / lo, whatever ns_chain asks,
    since the fp16 storage only saves memory traffic), and within tolerance of
    the oracle."""
    wl = one_group_workload(rows, cols, axis=axis, w_dtype=wdt, name=f"fused{rows}x{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    fused = run_gpu(W.clone(), M.clone(), G, alpha, steps, axis, coeffs=coeffs, chain=chain, master=master)
    split = run_gpu(W.clone(), M.clone(), G, alpha, steps, axis, coeffs=coeffs, master=master, per_product=True)
    assert torch.equal(fused["O"], split["O"]), "O"
    assert torch.equal(fused["M"], split["M"]), "M"
    assert torch.equal(fused["W"].view(torch.int32 if wdt == "f32" else torch.int16),
                       split["W"].view(torch.int32 if wdt == "f32" else torch.int16)), "W"
    err = check_matrix(fused, 0, alpha, steps, axis, coeffs=coeffs,
                       ns_tol=MASTER_TOL if master == binding.MASTER_FP32 else NS_TOL)
    print(f"fused chain {rows}x{cols} alpha {alpha} steps {steps}: {err:.3e}")


def test_fused_small_chain_grouped(hip_device):
    """A grouped call gathers the groups with s <= 64 into one fused chain and
    keeps those with 64 < s <= 128 (the same padded size) on a chain of
    launches: bitwise the per-group calls, and bitwise the grouped call with
    one launch per product."""
    wl = workloads.Workload("gfused", "test",
                            (workloads.Group("a", 200, 328, 2), workloads.Group("b", 328, 200, 3),
                             workloads.Group("c", 96, 1000, 1), workloads.Group("d", 384, 640, 2),
                             workloads.Group("e", 256, 1024, 2, AXIS_ROWS)), (0.25,))
    stacks = [workloads.make_group(wl, gi, hip_device) for gi in range(len(wl.groups))]
    solo = [tuple(t.clone() for t in st) for st in stacks]
    split = [tuple(t.clone() for t in st) for st in stacks]
    for (W, M, G), grp in zip(solo, wl.groups):
        binding.dion2_step_ex(W, M, G, 0.25, 0.95, 0.02, 5, grp.axis)
    binding.dion2_step_groups([(W, M, G, grp.axis) for (W, M, G), grp in zip(stacks, wl.groups)], 0.25)
    binding.dion2_step_groups([(W, M, G, grp.axis) for (W, M, G), grp in zip(split, wl.groups)], 0.25,
                              ns_chain_per_product=True)
    torch.cuda.synchronize()
    for gi, ((W, M, _), (Ws, Ms, _), (Wp, Mp, _)) in enumerate(zip(stacks, solo, split)):
        assert torch.equal(M, Ms) and torch.equal(M, Mp), f"group {gi}: M"
        assert torch.equal(W.view(torch.int16), Ws.view(torch.int16)), f"group {gi}: W against its own call"
        assert torch.equal(W.view(torch.int16), Wp.view(torch.int16)), f"group {gi}: W against per-product"


@pytest.mark.parametrize("rows,cols,alpha,axis,wdt", [
    (200, 328, 0.25, AXIS_AUTO, "bf16"),     # rows, s = 50, Z = L
    (328, 200, 0.25, AXIS_AUTO, "bf16"),     # columns, Z = L
    (96, 1000, 0.5, AXIS_AUTO, "f32"),       # rows, fp32 W
    (300, 200, 0.75, AXIS_ROWS, "f32"),      # k = 225 > d_oth = 200: Z = L^T
    (64, 256, 0.5, AXIS_COLS, "bf16"),       # columns, k = 128 > d_oth = 64: Z = L^T
    (257, 129, 1.0, AXIS_AUTO, "bf16"),      # alpha = 1, square-ish
    (130, 75, 0.5, AXIS_AUTO, "bf16"),       # cols % 4 != 0
    (640, 1664, 0.3, AXIS_ROWS, "bf16"),     # s = 193: several tiles, ragged
])
def test_fp32_master_ragged(hip_device, rows, cols, alpha, axis, wdt):
    """X kept as a bf16 hi/lo pair through every product: the tolerance is a
    tenth of the bf16 one."""
    wl = one_group_workload(rows, cols, axis=axis, w_dtype=wdt, name=f"m{rows}c{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, alpha, axis=axis, master=binding.MASTER_FP32)
    check_matrix(res, 0, alpha, axis=axis, ns_tol=MASTER_TOL)


@pytest.mark.parametrize("noise", [1e-2, 1e-3])
def test_low_rank_plus_noise_takes_the_master(hip_device, noise):
    """Momentum of rank 32 plus a little noise (512 x 2048, row selection at
    alpha = 0.25, so X is 128 x 2048). The noise directions' singular values
    are so far below the signal's that rounding X once to bf16 moves them:
    the exact iteration on the rounded X lies about 0.1 from the exact
    result. The default path, which takes X in bf16, is held to 2e-2 of
    that iteration on the rounded X; the fp32 master, which carries X as a
    hi/lo pair, to 2e-2 of the exact result, at least ten times closer than
    the default."""
    rng = np.random.default_rng(2512 + int(-math.log10(noise)))
    rows, cols, r = 512, 2048, 32
    base = rng.standard_normal((rows, r)) @ rng.standard_normal((r, cols))
    Mh = 1e-3 * (base + noise * math.sqrt(r) * rng.standard_normal((rows, cols)))
    M = torch.from_numpy(Mh.astype(np.float32))[None].to(hip_device)
    G = torch.zeros((1, rows, cols), dtype=torch.bfloat16, device=hip_device)
    W = (0.02 * torch.from_numpy(rng.standard_normal((1, rows, cols)).astype(np.float32))).to(torch.bfloat16)
    W = W.to(hip_device)
    O_exact, O_rounded = rounded_input_iteration(M, G, 0, 0.25, 5, AXIS_ROWS)
    floor = rel_fro(O_rounded, O_exact)
    assert floor > 5 * NS_TOL, floor
    res = run_gpu(W.clone(), M.clone(), G, 0.25, axis=AXIS_ROWS)
    check_matrix(res, 0, 0.25, axis=AXIS_ROWS, ns_ref=O_rounded)
    err_bf16 = rel_fro(res["O"][0].numpy().astype(np.float64), O_exact)
    res = run_gpu(W.clone(), M.clone(), G, 0.25, axis=AXIS_ROWS, master=binding.MASTER_FP32)
    err_master = check_matrix(res, 0, 0.25, axis=AXIS_ROWS)
    assert err_master < 0.1 * err_bf16, (err_master, err_bf16)


@pytest.mark.parametrize("gi,sample", [(0, 21), (1, 5), (2, 12)])
def test_1b_stack_full_size_fp32_master(hip_device, gi, sample):
    """The fp32 master over a whole 1B-stack group in one batched call, one
    sampled matrix against the oracle: at least five times closer than the
    default's bound, and within 2e-4."""
    wl = workloads.WORKLOADS["1b"]
    W, M, G = workloads.make_group(wl, gi, hip_device)
    grp = wl.groups[gi]
    k, ax = binding.dion2_plan_info(grp.rows, grp.cols, 0.25, grp.axis)
    d_sel, d_oth = (grp.rows, grp.cols) if ax == AXIS_ROWS else (grp.cols, grp.rows)
    sel = torch.empty((grp.count, k), dtype=torch.int32, device=hip_device)
    nrm = torch.empty((grp.count, d_sel), dtype=torch.float64, device=hip_device)
    upd = torch.empty((grp.count, k, d_oth), dtype=torch.float32, device=hip_device)
    snap = (W[sample].cpu(), M[sample].cpu(), G[sample].cpu())
    binding.dion2_step_ex(W, M, G, 0.25, dbg_sel_idx=sel, dbg_norms=nrm, dbg_update=upd,
                          ns_master=binding.MASTER_FP32)
    torch.cuda.synchronize()
    res = dict(W0=snap[0][None], M0=snap[1][None], G=snap[2][None], W=W[sample].cpu()[None],
               M=M[sample].cpu()[None], K=sel[sample].cpu()[None], norms=nrm[sample].cpu()[None],
               O=upd[sample].cpu()[None], axis=ax, k=k)
    err = check_matrix(res, 0, 0.25, ns_tol=MASTER_TOL)
    assert err <= 2e-4, f"fp32 master at a 1B shape: {err:.3e}"


@pytest.mark.parametrize("chain", [binding.CHAIN_HILO, binding.CHAIN_F16], ids=["hilo", "f16"])
def test_batch_beyond_grid_z(hip_device, chain):
    """40000 matrices in one GRAM call: the dual s x s launches would need a
    grid z extent of 80000, beyond the hardware's 65535, and go out as
    consecutive launches over slices of the batch. Matrices on either side of
    the slice boundary are checked against the oracle and against calls over
    a few matrices."""
    n = 40000
    wl = one_group_workload(8, 64, count=n, name="bigbatch")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    picks = [0, 32766, 32767, 32768, n - 1]
    solo = {b: (W[b:b + 1].clone(), M[b:b + 1].clone(), G[b:b + 1].clone()) for b in picks}
    snap = {b: (W[b].cpu(), M[b].cpu(), G[b].cpu()) for b in picks}
    binding.dion2_step_ex(W, M, G, 0.5, ns_form=NS_GRAM, ns_chain=chain)
    for b in picks:
        Ws, Ms, Gs = solo[b]
        binding.dion2_step_ex(Ws, Ms, Gs, 0.5, ns_form=NS_GRAM, ns_chain=chain)
    torch.cuda.synchronize()
    for b in picks:
        assert torch.equal(W[b].view(torch.int16), solo[b][0][0].view(torch.int16)), f"matrix {b}: weights"
        assert torch.equal(M[b], solo[b][1][0]), f"matrix {b}: momentum"
        out = oracle.dion2_step(snap[b][0].float().numpy().astype(np.float64), snap[b][1].numpy(),
                                snap[b][2].float().numpy(), 0.5, 0.95, 0.02, 5, AXIS_AUTO, w_dtype="bf16")
        np.testing.assert_array_equal(M[b].cpu().numpy(), out["M"], err_msg=f"matrix {b}: momentum")
    del W, M, G
    binding.dion2_release_workspaces()


@pytest.mark.parametrize("rows,cols,alpha", [(256, 1024, 0.25), (1024, 256, 0.5), (384, 384, 0.5)],
                         ids=["rows-gram", "cols-gram", "square-direct"])
def test_caller_workspace(hip_device, rows, cols, alpha):
    """A caller-provided workspace of dion2_workspace_size_ex bytes gives
    bitwise the result of the library's own; one block short, or a plan that
    needs more (the fp32 master on a DIRECT shape), is refused before
    anything runs."""
    wl = one_group_workload(rows, cols, count=2, name=f"ws{rows}x{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2 = W.clone(), M.clone()
    need = binding.dion2_workspace_size_ex(2, rows, cols, alpha)
    assert need > 0
    ws = torch.empty(need, dtype=torch.uint8, device=hip_device)
    binding.dion2_step_ex(W, M, G, alpha, workspace=ws)
    binding.dion2_step_ex(W2, M2, G, alpha)
    torch.cuda.synchronize()
    assert torch.equal(W.view(torch.int16), W2.view(torch.int16)) and torch.equal(M, M2)
    W3, M3 = W.clone(), M.clone()
    with pytest.raises(binding.Dion2Error) as ei:
        binding.dion2_step_ex(W3, M3, G, alpha, workspace=ws[:need - 256])
    assert ei.value.status == binding.DION2_ERR_WORKSPACE
    k, _ = binding.dion2_plan_info(rows, cols, alpha, AXIS_AUTO)
    if rows == cols:   # AUTO is DIRECT here; the fp32 master's GRAM plan needs more
        with pytest.raises(binding.Dion2Error) as ei:
            binding.dion2_step_ex(W3, M3, G, alpha, workspace=ws, ns_master=binding.MASTER_FP32)
        assert ei.value.status == binding.DION2_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.equal(W3.view(torch.int16), W.view(torch.int16)) and torch.equal(M3, M), "refused calls modified state"


@pytest.mark.parametrize("kw", [dict(ns_form=NS_GRAM), dict(ns_master=binding.MASTER_FP32),
                                dict(ns_form=NS_DIRECT), dict(ns_form=NS_GRAM, ns_chain=binding.CHAIN_F16)],
                         ids=["gram", "fp32-master", "direct", "f16-chain"])
@pytest.mark.parametrize("rows,cols,alpha", [(384, 384, 0.5), (256, 1024, 0.25), (640, 256, 0.5)])
def test_caller_workspace_sized_for_options(hip_device, kw, rows, cols, alpha):
    """A caller workspace of exactly dion2_workspace_size_ex bytes for forced
    options gives bitwise the library workspace's result, one block less is
    refused (state untouched), and dion2_workspace_size (no options) covers
    it."""
    wl = one_group_workload(rows, cols, count=2, name=f"wsx{rows}x{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2, W3, M3 = W.clone(), M.clone(), W.clone(), M.clone()
    need = binding.dion2_workspace_size_ex(2, rows, cols, alpha, AXIS_AUTO, 5, **kw)
    if kw.get("ns_form") == NS_DIRECT and one_tile(rows, cols, alpha):   # DIRECT refused on one tile
        assert need == 0 and binding.dion2_workspace_size(2, rows, cols, alpha) > 0
        assert direct_refused(W, M, G, alpha)
        return
    assert 0 < need <= binding.dion2_workspace_size(2, rows, cols, alpha)
    ws = torch.empty(need, dtype=torch.uint8, device=hip_device)
    binding.dion2_step_ex(W, M, G, alpha, workspace=ws, **kw)
    binding.dion2_step_ex(W2, M2, G, alpha, **kw)
    with pytest.raises(binding.Dion2Error) as ei:
        binding.dion2_step_ex(W3, M3, G, alpha, workspace=ws[:need - 256], **kw)
    assert ei.value.status == binding.DION2_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.equal(W.view(torch.int16), W2.view(torch.int16)) and torch.equal(M, M2)
    W0, M0, _ = workloads.make_group(wl, 0, hip_device)
    assert torch.equal(W3.view(torch.int16), W0.view(torch.int16)) and torch.equal(M3, M0), \
        "a refused call modified state"


@pytest.mark.parametrize("rows,cols,alpha,kw", [
    (2048, 8192, 1.0, dict(ns_form=NS_DIRECT)),                    # X^T pair; l = 4 s
    (8192, 2048, 0.25, dict(select_rule=binding.SELECT_RANDOM)),  # column partials
], ids=["direct-xt", "random-columns"])
def test_caller_workspace_new_buffers(hip_device, rows, cols, alpha, kw):
    """The buffers the plan adds for the Direct form's X^T (from s = 2048) and
    the Random rule's single column pass: a caller workspace of exactly
    dion2_workspace_size_ex bytes gives bitwise the library workspace's
    result, one block less is refused, and dion2_workspace_size covers it."""
    wl = one_group_workload(rows, cols, count=1, name=f"wsn{rows}x{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2, W3, M3 = W.clone(), M.clone(), W.clone(), M.clone()
    need = binding.dion2_workspace_size_ex(1, rows, cols, alpha, AXIS_AUTO, 5, **kw)
    base = binding.dion2_workspace_size_ex(1, rows, cols, alpha, AXIS_AUTO, 5)
    assert base < need <= binding.dion2_workspace_size(1, rows, cols, alpha)
    ws = torch.empty(need, dtype=torch.uint8, device=hip_device)
    binding.dion2_step_ex(W, M, G, alpha, workspace=ws, **kw)
    binding.dion2_step_ex(W2, M2, G, alpha, **kw)
    with pytest.raises(binding.Dion2Error) as ei:
        binding.dion2_step_ex(W3, M3, G, alpha, workspace=ws[:need - 256], **kw)
    assert ei.value.status == binding.DION2_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.equal(W.view(torch.int16), W2.view(torch.int16)) and torch.equal(M, M2)
    W0, M0, _ = workloads.make_group(wl, 0, hip_device)
    assert torch.equal(W3.view(torch.int16), W0.view(torch.int16)) and torch.equal(M3, M0), \
        "a refused call modified state"


@pytest.mark.parametrize("eps", [0.0, 1.0], ids=["eps0", "eps-large"])
@FORMS
def test_normalisation_eps(hip_device, eps, form):
    """dion2_options.ns_eps reaches the normalisation X / (||X||_F + eps):
    with ||X||_F about 1.4 here, eps = 1 shrinks X by 40%, which moves O
    many times the tolerance away unless both sides use it."""
    wl = one_group_workload(128, 512, name="eps")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    if direct_refused(W, M, G, 0.25, form=form):
        return
    res = run_gpu(W, M, G, 0.25, form=form, eps=eps)
    check_matrix(res, 0, 0.25, eps=eps)


@pytest.mark.parametrize("wdt,gdt", [("bf16", "f32"), ("f32", "bf16")])
@pytest.mark.parametrize("axis", [AXIS_ROWS, AXIS_COLS])
def test_mixed_w_and_g_dtypes(hip_device, wdt, gdt, axis):
    """W and G in different storage types (dion2_options.w_dtype / g_dtype)."""
    wl = one_group_workload(192, 320, axis=axis, w_dtype="f32", name=f"mix{axis}")
    W, M, G = workloads.make_group(wl, 0, hip_device)   # fp32 W and G
    to = {"bf16": torch.bfloat16, "f32": torch.float32}
    W = W.to(to[wdt]).contiguous()
    G = G.to(to[gdt]).contiguous()
    res = run_gpu(W, M, G, 0.25, axis=axis)
    check_matrix(res, 0, 0.25, axis=axis)


def compact_x_want(M0, G, K, axis, eps):
    """X as K3 writes it, from the oracle's accumulated momentum and its
    Frobenius norm, with the rounding decisions taken in the kernel's
    precision: x = fl32(m * fl32(1 / (||M[K]||_F + eps))), hi = bf16(x),
    lo = bf16(x - hi). Also the fp64 quotient the definition rounds."""
    Macc = oracle.momentum_accumulate(M0, G)
    X = oracle.gather(Macc, K, axis)
    if axis == AXIS_COLS:
        X = X.T                                       # line p in row p
    q = X / (np.linalg.norm(X) + eps)                 # the oracle's normalisation
    sc = np.float32(1.0 / (np.linalg.norm(X) + eps))
    x32 = X.astype(np.float32) * sc
    hi = oracle.round_bf16(x32.astype(np.float64))
    lo = oracle.round_bf16((x32 - hi.astype(np.float32)).astype(np.float64))
    return hi, lo, q


@pytest.mark.parametrize("rows,cols,alpha,axis,gdt,form,steps", [
    (96, 256, 0.25, AXIS_ROWS, "bf16", binding.NS_AUTO, 5),     # L layout (GRAM)
    (640, 1024, 0.25, AXIS_ROWS, "bf16", NS_DIRECT, 5),         # L layout, DIRECT overwrites it
    (200, 64, 0.5, AXIS_ROWS, "f32", binding.NS_AUTO, 5),       # k > d_oth: L^T layout
    (256, 96, 0.25, AXIS_COLS, "bf16", NS_GRAM, 5),             # column gather (update_cols)
    (64, 200, 0.5, AXIS_COLS, "f32", binding.NS_AUTO, 5),       # columns, L^T layout
    (130, 70, 1.0, AXIS_AUTO, "bf16", binding.NS_AUTO, 0),      # ragged, no Newton-Schulz step
])
def test_compact_x_bitwise(hip_device, rows, cols, alpha, axis, gdt, form, steps):
    """K3: the compact matrix equals the oracle's normalised selected lines,
    rounded to bf16 in the kernel's precision, bit for bit, for every layout
    and both gathers; the decayed M and the rest of the step as usual."""
    wl = one_group_workload(rows, cols, count=3, axis=axis, w_dtype="f32", name=f"cx{rows}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W = W.to(torch.bfloat16).contiguous()
    G = G.to(torch.bfloat16 if gdt == "bf16" else torch.float32).contiguous()
    B = W.shape[0]
    k, ax = binding.dion2_plan_info(rows, cols, alpha, axis)
    d_oth = cols if ax == AXIS_ROWS else rows
    cx = torch.zeros((B, k, d_oth), dtype=torch.bfloat16, device=hip_device)
    M0, G0 = M.cpu().numpy(), G.float().cpu().numpy()
    res = run_gpu(W, M, G, alpha, ns_steps=steps, axis=axis, form=form, dbg_compact=cx)
    got = cx.float().cpu().numpy().astype(np.float64)
    eps = float(np.float32(1e-7))
    for b in range(B):
        check_matrix(res, b, alpha, ns_steps=steps, axis=axis)
        hi, _, q = compact_x_want(M0[b], G0[b], res["K"][b].numpy().astype(np.int64), ax, eps)
        np.testing.assert_array_equal(got[b], hi, err_msg=f"compact X, matrix {b}")
        # against the fp64 definition only rounding-boundary cases may differ, by one unit
        off = got[b] != oracle.round_bf16(q)
        assert off.mean() < 1e-3
        assert np.all(np.abs(got[b][off] - q[off]) <= 2.0 ** -7 * np.abs(q[off]))


@pytest.mark.parametrize("rows,cols,alpha,gdt,decay_all", [
    (600, 330, 0.25, "bf16", False),    # k = 83 <= d_oth: L layout, ragged tiles
    (300, 800, 1.0, "f32", False),      # k = 800 > d_oth = 300: L^T layout
    (1000, 512, 0.5, "bf16", True),     # decay-all
])
def test_random_rule_single_column_pass(hip_device, rows, cols, alpha, gdt, decay_all):
    """Column selection under the Random rule reads M and G once: K is drawn
    first, update_cols forms M + G, decays and copies the selected columns
    unscaled with per-block sums of squares, and ||X||_F and the compact
    matrix follow. Against the oracle (K, M, X bitwise; O; W given O), and
    bitwise the two-pass path the debug l1 norms select."""
    wl = one_group_workload(rows, cols, count=2, axis=AXIS_COLS, w_dtype="f32", name=f"cp{rows}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W = W.to(torch.bfloat16).contiguous()
    G = G.to(torch.bfloat16 if gdt == "bf16" else torch.float32).contiguous()
    B = W.shape[0]
    k, ax = binding.dion2_plan_info(rows, cols, alpha, AXIS_COLS)
    assert ax == AXIS_COLS
    rand = (21, 4, 7)
    M0, G0 = M.cpu().numpy(), G.float().cpu().numpy()
    W2, M2 = W.clone(), M.clone()
    cx = torch.zeros((B, k, rows), dtype=torch.bfloat16, device=hip_device)
    res = run_gpu(W, M, G, alpha, axis=AXIS_COLS, rand=rand, decay_all=decay_all, dbg_compact=cx,
                  norms=False)
    got = cx.float().cpu().numpy().astype(np.float64)
    eps = float(np.float32(1e-7))
    for b in range(B):
        check_matrix(res, b, alpha, axis=AXIS_COLS, rand=rand, decay_all=decay_all)
        if not decay_all:
            hi, _, _ = compact_x_want(M0[b], G0[b], res["K"][b].numpy().astype(np.int64), ax, eps)
            np.testing.assert_array_equal(got[b], hi, err_msg=f"compact X, matrix {b}")
    two = run_gpu(W2, M2, G, alpha, axis=AXIS_COLS, rand=rand, decay_all=decay_all)
    assert torch.equal(two["K"], res["K"]) and torch.equal(two["M"], res["M"])
    assert torch.equal(two["W"].view(torch.int16), res["W"].view(torch.int16))


@pytest.mark.parametrize("rows,cols,alpha,axis", [
    (160, 384, 0.25, AXIS_AUTO),     # rows, L layout
    (200, 64, 0.5, AXIS_ROWS),       # rows, L^T layout
    (64, 200, 0.5, AXIS_COLS),       # columns, L^T layout
])
def test_compact_x_lo_halves_fp32_master(hip_device, rows, cols, alpha, axis):
    """With the fp32 master K3 also writes the lo halves bf16(x - bf16(x)):
    both halves bitwise, and hi + lo within 2^-15 of the exact quotient
    (2^-16 from rounding lo, 2^-23 from the fp32 quotient)."""
    wl = one_group_workload(rows, cols, count=2, axis=axis, name=f"cxlo{rows}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    B = W.shape[0]
    k, ax = binding.dion2_plan_info(rows, cols, alpha, axis)
    d_oth = cols if ax == AXIS_ROWS else rows
    hi_t = torch.zeros((B, k, d_oth), dtype=torch.bfloat16, device=hip_device)
    lo_t = torch.zeros_like(hi_t)
    M0, G0 = M.cpu().numpy(), G.float().cpu().numpy()
    res = run_gpu(W, M, G, alpha, axis=axis, master=binding.MASTER_FP32, dbg_compact=hi_t,
                  dbg_compact_lo=lo_t)
    eps = float(np.float32(1e-7))
    for b in range(B):
        check_matrix(res, b, alpha, axis=axis, ns_tol=MASTER_TOL)
        hi, lo, q = compact_x_want(M0[b], G0[b], res["K"][b].numpy().astype(np.int64), ax, eps)
        gh = hi_t[b].float().cpu().numpy().astype(np.float64)
        gl = lo_t[b].float().cpu().numpy().astype(np.float64)
        np.testing.assert_array_equal(gh, hi, err_msg="hi halves")
        np.testing.assert_array_equal(gl, lo, err_msg="lo halves")
        assert np.all(np.abs(gh + gl - q) <= 2.0 ** -15 * np.abs(q))


@pytest.mark.parametrize("rows,cols,axis", [
    (1 << 20, 64, AXIS_AUTO),     # columns of a million entries: Gram over K = 2^20
    (1 << 20, 16, AXIS_ROWS),     # 2^20 lines to select from (keys beyond the LDS cache), L^T
    (16, 1 << 20, AXIS_AUTO),     # rows of a million entries: 8192 column tiles, fused update
])
def test_maximum_dimension(hip_device, rows, cols, axis):
    """A side of 2^20, the longest the library takes, against the whole
    oracle step (the oracle's exact l1 sums take about 15 s here)."""
    wl = one_group_workload(rows, cols, axis=axis, name=f"max{rows}x{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    k, ax = binding.dion2_plan_info(rows, cols, 0.25, axis)
    d_oth = cols if ax == AXIS_ROWS else rows
    cx = torch.zeros((1, k, d_oth), dtype=torch.bfloat16, device=hip_device)
    M0, G0 = M.cpu().numpy(), G.float().cpu().numpy()
    res = run_gpu(W, M, G, 0.25, axis=axis, dbg_compact=cx)
    check_matrix(res, 0, 0.25, axis=axis)
    hi, _, _ = compact_x_want(M0[0], G0[0], res["K"][0].numpy().astype(np.int64), ax,
                              float(np.float32(1e-7)))
    np.testing.assert_array_equal(cx[0].float().cpu().numpy().astype(np.float64), hi)


def sampled_column_step(hip_device, rows, cols, alpha, name, lr=0.02, mu=0.95):
    """One column-selection step on a matrix too large for the whole oracle
    step, checked by what holds at any size. Before the call, the oracle's
    accumulated momentum is formed chunk by chunk on the host: its column l1
    sums (fp64) give K, its column sums of squares the Frobenius norm of X.
    After it: K exactly (the k-th and next norms are apart by far more than
    the fp64 sums' error); the l1 norms of sampled columns against exact sums;
    M and W bitwise on sampled rows (W given the GPU's O); X bitwise on
    sampled rows; and every singular value of O inside the band the five
    quintic steps reach from a well-conditioned start, [0.68, 1.2] (Sec. 1),
    up to 2% for the bf16 arithmetic."""
    wl = one_group_workload(rows, cols, axis=AXIS_COLS, name=name)
    W, M, G = workloads.make_group(wl, 0, hip_device)
    k, ax = binding.dion2_plan_info(rows, cols, alpha, AXIS_COLS)
    assert ax == AXIS_COLS
    rng = np.random.default_rng(7)
    rs = np.unique(np.concatenate([[0, 1, rows - 1], rng.integers(0, rows, 61)]))
    cs = np.array([0, 1, cols // 2, cols - 1])
    rs_t = torch.from_numpy(rs).to(hip_device)
    col_l1 = np.zeros(cols)
    col_sq = np.zeros(cols)
    macc_cs = []
    for i in range(0, rows, 65536):
        macc = oracle.momentum_accumulate(M[0, i:i + 65536].cpu().numpy(),
                                          G[0, i:i + 65536].float().cpu().numpy())
        a64 = macc.astype(np.float64)
        col_l1 += np.abs(a64).sum(axis=0)
        col_sq += np.square(a64).sum(axis=0)
        macc_cs.append(macc[:, cs])
    macc_cs = np.concatenate(macc_cs)
    macc_rs = oracle.momentum_accumulate(M[0, rs_t].cpu().numpy(), G[0, rs_t].float().cpu().numpy())
    W0 = W[0, rs_t].float().cpu().numpy().astype(np.float64)
    order = np.lexsort((np.arange(cols), -col_l1))
    K = np.sort(order[:k])
    if k < cols:
        gap = col_l1[order[k - 1]] - col_l1[order[k]]
        assert gap > 1e-9 * col_l1[order[k - 1]], "near tie at the selection boundary"

    sel = torch.full((1, k), -1, dtype=torch.int32, device=hip_device)
    nrm = torch.full((1, cols), -1.0, dtype=torch.float64, device=hip_device)
    upd = torch.full((1, k, rows), float("nan"), dtype=torch.float32, device=hip_device)
    cx = torch.zeros((1, k, rows), dtype=torch.bfloat16, device=hip_device)
    binding.dion2_step_ex(W, M, G, alpha, mu, lr, 5, AXIS_COLS, dbg_sel_idx=sel, dbg_norms=nrm,
                          dbg_update=upd, dbg_compact=cx)
    torch.cuda.synchronize()

    np.testing.assert_array_equal(sel[0].cpu().numpy(), K, err_msg="selected columns")
    np.testing.assert_array_equal(nrm[0].cpu().numpy()[cs], oracle.l1_norms(macc_cs, AXIS_COLS))
    M_want = oracle.selective_decay(macc_rs, K, mu, AXIS_COLS)
    np.testing.assert_array_equal(M[0, rs_t].cpu().numpy(), M_want, err_msg="momentum rows")
    O_rows = upd[0][:, rs_t].cpu().numpy().astype(np.float64).T      # O[r, p], paper orientation
    W_want = W0.copy()
    W_want[:, K] = oracle.round_to(W0[:, K] - oracle.update_scale(lr, rows, cols) * O_rows, "bf16")
    np.testing.assert_array_equal(W[0, rs_t].float().cpu().numpy().astype(np.float64), W_want,
                                  err_msg="weight rows")
    sc = np.float32(1.0 / (math.sqrt(float(np.sum(col_sq[K]))) + float(np.float32(1e-7))))
    x_want = oracle.round_bf16((macc_rs[:, K].astype(np.float32) * sc).astype(np.float64))
    np.testing.assert_array_equal(cx[0][:, rs_t].float().cpu().numpy().astype(np.float64).T, x_want)
    O = upd[0].cpu().numpy()                                          # [k, rows] fp32
    ev = np.linalg.eigvalsh(O @ O.T)
    # the band, widened by 2% for the bf16 arithmetic
    assert (0.68 * 0.98) ** 2 <= ev.min() and ev.max() <= (1.2 * 1.02) ** 2, (ev.min(), ev.max())


def test_maximum_rows_column_step(hip_device):
    """2^20 rows x 1032 columns at alpha = 1 (1.08e9 elements): every column
    selected, the Gram product sums over K = 2^20, and the column update runs
    over 32768 blocks of 32 rows."""
    sampled_column_step(hip_device, 1 << 20, 1032, 1.0, "maxrows")


def test_near_2_31_elements_strip_kernel(hip_device):
    """524160 x 4097 (2^31 - 128 elements, the most a matrix may hold) at
    alpha = 0.25: rows wider than 8 KB take the 512-column strip kernel, here
    over 32760 row blocks, and element offsets reach the top of the signed
    32-bit range."""
    sampled_column_step(hip_device, 524160, 4097, 0.25, "near2p31")


CONCURRENT = workloads.Workload(
    "concurrent", "test", (workloads.Group("a", 256, 640, 3), workloads.Group("b", 640, 256, 2),
                           workloads.Group("c", 384, 384, 2)), (0.25,))


def test_concurrent_streams_and_threads(hip_device):
    """Calls on three streams at once (one workspace per stream), and calls
    from three host threads on one stream (serialised by the library), give
    bitwise the results of the same calls made one after another; two steps
    each, so a workspace reused across calls is covered too."""
    import threading
    stacks = [workloads.make_group(CONCURRENT, gi, hip_device) for gi in range(3)]
    seq = [tuple(t.clone() for t in st) for st in stacks]
    thr = [tuple(t.clone() for t in st) for st in stacks]
    for W, M, G in seq:
        for _ in range(2):
            binding.dion2_step_ex(W, M, G, 0.25)
    torch.cuda.synchronize()

    streams = [torch.cuda.Stream(device=hip_device) for _ in stacks]   # default priority
    for st, (W, M, G) in zip(streams, stacks):
        for _ in range(2):
            binding.dion2_step_ex(W, M, G, 0.25, stream=st)
    torch.cuda.synchronize()

    errors = []

    def worker(W, M, G):
        try:
            for _ in range(2):
                binding.dion2_step_ex(W, M, G, 0.25)
        except Exception as e:   # reported below, in the test's thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=t) for t in thr]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for gi in range(3):
        for got, name in ((stacks[gi], "streams"), (thr[gi], "threads")):
            assert torch.equal(got[1], seq[gi][1]), f"group {gi}, {name}: momentum"
            assert torch.equal(got[0].view(torch.int16), seq[gi][0].view(torch.int16)), \
                f"group {gi}, {name}: weights"


def test_decay_all_ablation(hip_device):
    wl = one_group_workload(128, 256, name="decayall")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res = run_gpu(W, M, G, 0.25, decay_all=True)
    check_matrix(res, 0, 0.25, decay_all=True)


def test_zero_state_selects_first_lines(hip_device):
    wl = one_group_workload(256, 256, count=2, name="zero")
    W, M, G = workloads.make_group(wl, 0, hip_device, m0_zero=True)
    G.zero_()
    res = run_gpu(W, M, G, 0.25)
    for b in range(2):
        assert res["K"][b].tolist() == list(range(64))
        assert torch.equal(res["W"][b], res["W0"][b])
        assert not torch.any(res["M"][b])
        assert not torch.any(res["O"][b])


@pytest.mark.parametrize("rows,cols,alpha,kw", [
    (200, 328, 0.25, {}),                                     # GRAM, one tile
    (200, 328, 0.75, dict(form=NS_DIRECT)),                   # DIRECT, s = 150
    (328, 200, 0.25, dict(rand=(5, 7, 0))),                   # Random rule, columns: the single column pass
    (200, 328, 0.25, dict(master=binding.MASTER_FP32)),       # X's lo halves too
], ids=["gram", "direct", "random-columns", "fp32-master"])
def test_zero_matrix_with_eps_zero(hip_device, rows, cols, alpha, kw):
    """With ns_eps = 0 a zero compact matrix leaves X / (||X||_F + eps) at
    0 / 0; it is taken at its limit as eps -> 0+, which is 0: O = 0 and W
    unchanged, no NaN, while the other matrix of the batch steps as usual."""
    wl = one_group_workload(rows, cols, count=2, name=f"zeps{rows}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    M[0] = 0.0
    G[0] = 0.0
    rand = kw.get("rand")
    res = run_gpu(W, M, G, alpha, eps=0.0, norms=rand is None, **kw)
    assert torch.all(torch.isfinite(res["O"])) and not torch.any(res["O"][0])
    assert torch.equal(res["W"][0].view(torch.int16), res["W0"][0].view(torch.int16))
    for b in range(2):
        check_matrix(res, b, alpha, eps=0.0, rand=rand,
                     ns_tol=MASTER_TOL if kw.get("master") == binding.MASTER_FP32 else NS_TOL)


@FORMS
def test_exact_ties_go_to_lower_index(hip_device, form):
    wl = one_group_workload(640, 768, name="ties")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    # rows 2j and 2j+1 identical: every norm appears twice
    M[0, 1::2] = M[0, 0::2]
    G[0, 1::2] = G[0, 0::2]
    res = run_gpu(W, M, G, 0.25, form=form)
    check_matrix(res, 0, 0.25)
    K = res["K"][0].tolist()
    assert all((i % 2 == 0) or (i - 1 in K) for i in K)


def test_nan_line_is_selected(hip_device):
    wl = one_group_workload(128, 256, name="nan")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    M[0, 77, 5] = float("nan")
    res = run_gpu(W, M, G, 0.125)
    assert 77 in res["K"][0].tolist()
    sel = set(res["K"][0].tolist())
    keep = [i for i in range(128) if i not in sel]
    assert torch.equal(res["W"][0][keep], res["W0"][0][keep])


def test_run_twice_bitwise(hip_device):
    wl = one_group_workload(512, 1024, count=2, name="det")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2 = W.clone(), M.clone()
    binding.dion2_step_strided(W, M, G, 0.5)
    binding.dion2_step_strided(W2, M2, G, 0.5)
    torch.cuda.synchronize()
    assert torch.equal(W, W2) and torch.equal(M, M2)


@FORMS
def test_two_steps_in_a_row(hip_device, form):
    wl = one_group_workload(640, 1024, name="twostep")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res1 = run_gpu(W, M, G, 0.25, form=form)
    check_matrix(res1, 0, 0.25)
    res2 = run_gpu(W, M, G, 0.25, form=form)   # continues from the updated state
    check_matrix(res2, 0, 0.25)


def test_gram_form_tracks_duplicate_lines(hip_device):
    """Duplicate selected lines make the Gram matrix singular; the GRAM form's
    accumulated polynomial is large on that null space, yet O stays within
    tolerance and duplicate lines of O stay equal to rounding."""
    wl = one_group_workload(256, 1024, name="dupgram")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    for j in range(0, 256, 8):
        M[0, j + 1:j + 4] = M[0, j]
        G[0, j + 1:j + 4] = G[0, j]
    res = run_gpu(W, M, G, 0.5, form=NS_GRAM)
    check_matrix(res, 0, 0.5)
    K = res["K"][0].tolist()
    O = res["O"][0]
    pos = {r: i for i, r in enumerate(K)}
    for j in range(0, 256, 8):
        rows = [pos[r] for r in range(j, j + 4) if r in pos]
        for r in rows[1:]:
            assert torch.allclose(O[r], O[rows[0]], rtol=0, atol=1e-3 * float(O[rows[0]].abs().max()))


@pytest.mark.parametrize("gi,alpha,samples", [(0, 0.25, (0, 63)), (1, 0.25, (7,)), (2, 0.25, (15,)),
                                              (0, 0.5, (31,)), (1, 0.5, (3,)), (2, 0.5, (10,)),
                                              (0, 1.0, (5,)), (1, 1.0, (12,)), (2, 1.0, (0,))])
def test_1b_stack_full_size_sampled(hip_device, gi, alpha, samples):
    """The whole group of the 1B-style stack in one batched call (the launch
    configuration the benchmark times) at every selection fraction the
    benchmark reports (the sweep of Sec. 4.1 and Muon's alpha = 1); sampled
    matrices checked in full. At alpha = 0.5 and 1 the 8192x2048 (columns)
    and 2048x8192 (rows) groups run the GRAM chain at s = 1024 and 2048, and
    the 2048x2048 group the DIRECT form."""
    wl = workloads.WORKLOADS["1b"]
    W, M, G = workloads.make_group(wl, gi, hip_device)
    grp = wl.groups[gi]
    k, ax = binding.dion2_plan_info(grp.rows, grp.cols, alpha, grp.axis)
    d_sel, d_oth = (grp.rows, grp.cols) if ax == AXIS_ROWS else (grp.cols, grp.rows)
    sel = torch.empty((grp.count, k), dtype=torch.int32, device=hip_device)
    nrm = torch.empty((grp.count, d_sel), dtype=torch.float64, device=hip_device)
    upd = torch.empty((grp.count, k, d_oth), dtype=torch.float32, device=hip_device)
    picks = list(samples)
    snap = {b: (W[b].cpu(), M[b].cpu(), G[b].cpu()) for b in picks}
    binding.dion2_step_ex(W, M, G, alpha, dbg_sel_idx=sel, dbg_norms=nrm, dbg_update=upd)
    torch.cuda.synchronize()
    for b in picks:
        res = dict(W0=snap[b][0][None], M0=snap[b][1][None], G=snap[b][2][None],
                   W=W[b].cpu()[None], M=M[b].cpu()[None], K=sel[b].cpu()[None],
                   norms=nrm[b].cpu()[None], O=upd[b].cpu()[None], axis=ax, k=k)
        check_matrix(res, 0, alpha)


@pytest.mark.parametrize("gi,sample", [(0, 40), (1, 11), (2, 2)])
def test_1b_stack_full_size_f16_chain(hip_device, gi, sample):
    """The opt-in fp16 chain over a whole 1B-stack group in one batched call
    (the configuration the benchmark's per_chain_ms times), one sampled
    matrix checked in full."""
    wl = workloads.WORKLOADS["1b"]
    W, M, G = workloads.make_group(wl, gi, hip_device)
    grp = wl.groups[gi]
    k, ax = binding.dion2_plan_info(grp.rows, grp.cols, 0.25, grp.axis)
    d_sel, d_oth = (grp.rows, grp.cols) if ax == AXIS_ROWS else (grp.cols, grp.rows)
    sel = torch.empty((grp.count, k), dtype=torch.int32, device=hip_device)
    nrm = torch.empty((grp.count, d_sel), dtype=torch.float64, device=hip_device)
    upd = torch.empty((grp.count, k, d_oth), dtype=torch.float32, device=hip_device)
    snap = (W[sample].cpu(), M[sample].cpu(), G[sample].cpu())
    binding.dion2_step_ex(W, M, G, 0.25, dbg_sel_idx=sel, dbg_norms=nrm, dbg_update=upd,
                          ns_chain=binding.CHAIN_F16)
    torch.cuda.synchronize()
    res = dict(W0=snap[0][None], M0=snap[1][None], G=snap[2][None], W=W[sample].cpu()[None],
               M=M[sample].cpu()[None], K=sel[sample].cpu()[None], norms=nrm[sample].cpu()[None],
               O=upd[sample].cpu()[None], axis=ax, k=k)
    err = check_matrix(res, 0, 0.25)
    assert err <= 5e-3, f"fp16 chain at a 1B shape: {err:.3e}"


def test_colsel_spikes_selected(hip_device):
    """Column selection on 2048x8192 with 5% of columns spiked x20: every
    spiked column is selected, and the sampled matrix matches the oracle."""
    wl = workloads.WORKLOADS["1b-colsel"]
    gi = 2
    W, M, G = workloads.make_group(wl, gi, hip_device, first=3, count=2)
    res = run_gpu(W, M, G, 0.25, axis=AXIS_COLS)
    check_matrix(res, 1, 0.25, axis=AXIS_COLS)
    # spiked columns have |G| ~ 20x the others: all of them land in K
    gabs = res["G"][1].float().abs().mean(dim=0)
    spiked = torch.nonzero(gabs > 5 * gabs.median()).flatten().tolist()
    assert len(spiked) == int(0.05 * 8192)
    assert set(spiked) <= set(res["K"][1].tolist())


@pytest.mark.parametrize("gi", [0, 1, 2], ids=["4096x4096", "11008x4096", "4096x11008"])
@pytest.mark.parametrize("alpha", [0.125, 0.25])
def test_7b_shapes_sampled(hip_device, gi, alpha):
    """7B-style shapes (the 11008x4096 group selects columns): two matrices of
    each group in one batched call, both checked in full."""
    wl = workloads.WORKLOADS["7b"]
    W, M, G = workloads.make_group(wl, gi, hip_device, first=5, count=2)
    res = run_gpu(W, M, G, alpha)
    for b in range(2):
        check_matrix(res, b, alpha)


def test_7b_square_muon(hip_device):
    """alpha = 1 (every line selected: Muon) on a 4096x4096 matrix."""
    wl = workloads.WORKLOADS["7b"]
    W, M, G = workloads.make_group(wl, 0, hip_device, first=9, count=1)
    res = run_gpu(W, M, G, 1.0)
    assert res["k"] == 4096
    check_matrix(res, 0, 1.0)


@pytest.mark.parametrize("gi", [1, 2], ids=["11008x4096", "4096x11008"])
def test_7b_tall_wide_muon(hip_device, gi):
    """alpha = 1 on one matrix of each non-square 7B group: every one of the
    4096 short-side lines is selected, so the orthogonalised block is the whole
    4096 x 11008 (or 11008 x 4096) momentum, the largest Newton-Schulz product
    the 7B stack runs."""
    wl = workloads.WORKLOADS["7b"]
    W, M, G = workloads.make_group(wl, gi, hip_device, first=9, count=1)
    res = run_gpu(W, M, G, 1.0)
    assert res["k"] == 4096
    check_matrix(res, 0, 1.0)


@pytest.mark.parametrize("gi", [0, 1], ids=["2048x1408", "1408x2048"])
@pytest.mark.parametrize("m0_zero", [True, False], ids=["m0-zero", "m0-drawn"])
def test_moe_experts_with_zero_gradients(hip_device, gi, m0_zero):
    """MoE expert shapes with 30% zero-gradient experts. With zero momentum a
    zero expert is all ties: K = first k lines, O = 0, W unchanged."""
    wl = workloads.WORKLOADS["moe"]
    zero = set(workloads.zero_gradient_matrices(wl, gi))
    # a window of 8 experts holding both kinds
    first = next(f for f in range(0, 57) if 0 < len(zero & set(range(f, f + 8))) < 8)
    W, M, G = workloads.make_group(wl, gi, hip_device, m0_zero=m0_zero, first=first, count=8)
    res = run_gpu(W, M, G, 0.25)
    for b in range(8):
        check_matrix(res, b, 0.25)
        if first + b in zero:
            assert not torch.any(res["G"][b])
            if m0_zero:
                assert res["K"][b].tolist() == list(range(res["k"]))
                assert torch.equal(res["W"][b], res["W0"][b])
                assert not torch.any(res["O"][b])


@pytest.mark.parametrize("rows,cols,axis", [(384, 640, AXIS_AUTO), (640, 384, AXIS_AUTO),
                                            (300, 200, AXIS_ROWS)], ids=["rowsel", "colsel", "rowsel-tall"])
@FORMS
def test_random_selection(hip_device, rows, cols, axis, form):
    """Random rule: the GPU draws the same Philox keys as the oracle, so K is
    identical; matrix b of the batch uses counter word rand_matrix0 + b."""
    wl = one_group_workload(rows, cols, count=3, axis=axis, name=f"rand{rows}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    rand = (0x1234_5678_9ABC_DEF0, 2**33 + 7, 41)
    res = run_gpu(W, M, G, 0.5, axis=axis, form=form, rand=rand)
    for b in range(3):
        check_matrix(res, b, 0.5, axis=axis, rand=rand)
    assert not torch.equal(res["K"][0], res["K"][1])   # each matrix draws its own subset


def test_random_selection_full_1b_group(hip_device):
    """The Random rule on the whole 2048x2048 group of the 1B-style stack."""
    wl = workloads.WORKLOADS["1b"]
    W, M, G = workloads.make_group(wl, 0, hip_device)
    k, ax = binding.dion2_plan_info(2048, 2048, 0.25, AXIS_AUTO)
    sel = torch.empty((64, k), dtype=torch.int32, device=hip_device)
    snap = {b: (W[b].cpu(), M[b].cpu(), G[b].cpu()) for b in (0, 63)}
    upd = torch.empty((64, k, 2048), dtype=torch.float32, device=hip_device)
    nrm = torch.empty((64, 2048), dtype=torch.float64, device=hip_device)
    binding.dion2_step_ex(W, M, G, 0.25, dbg_sel_idx=sel, dbg_norms=nrm, dbg_update=upd,
                          select_rule=binding.SELECT_RANDOM, rand_seed=5, rand_step=100)
    torch.cuda.synchronize()
    for b in (0, 63):
        res = dict(W0=snap[b][0][None], M0=snap[b][1][None], G=snap[b][2][None],
                   W=W[b].cpu()[None], M=M[b].cpu()[None], K=sel[b].cpu()[None],
                   norms=nrm[b].cpu()[None], O=upd[b].cpu()[None], axis=ax, k=k)
        check_matrix(res, 0, 0.25, rand=(5, 100, b))


# Several shape groups in one grouped call: five in the GRAM form (four of
# padded s = 128, one of 256: two shared chains) and one in the DIRECT form
# (600 x 640: s = 150, padded 256, and l = 640 < 3 s).
GROUPED = workloads.Workload(
    "grouped", "test", (workloads.Group("a", 256, 640, 2), workloads.Group("b", 640, 256, 3),
                        workloads.Group("c", 384, 384, 2), workloads.Group("d", 300, 200, 1),
                        workloads.Group("e", 600, 640, 2), workloads.Group("f", 1024, 2048, 1)),
    (0.25,))


@pytest.mark.parametrize("gs", [1, 0, 3], ids=["one-stream", "default-streams", "three-streams"])
@pytest.mark.parametrize("rand", [None, (11, 3, 5)], ids=["l1", "random"])
def test_groups_equal_per_group_calls(hip_device, rand, gs):
    """dion2_step_groups is bitwise the per-group dion2_step_ex calls on one
    stream or spread over several, its chains really are shared (s x s
    launches counted), and one group is tied to the oracle through the
    per-group call's debug outputs."""
    alpha = 0.25
    stacks = [workloads.make_group(GROUPED, gi, hip_device) for gi in range(len(GROUPED.groups))]
    solo = [tuple(t.clone() for t in s) for s in stacks]
    kw = {}
    if rand is not None:
        kw = dict(select_rule=binding.SELECT_RANDOM, rand_seed=rand[0], rand_step=rand[1])
    # per group, in order, with the Random rule's matrix indices continuing
    m0 = rand[2] if rand else 0
    for W, M, G in solo:
        binding.dion2_step_ex(W, M, G, alpha, rand_matrix0=m0, **kw)
        m0 += W.shape[0]
    binding.dion2_profile_reset()
    binding.dion2_profile_enable(True)
    binding.dion2_step_groups([(W, M, G, AXIS_AUTO) for W, M, G in stacks], alpha,
                              rand_matrix0=rand[2] if rand else 0, group_streams=gs, **kw)
    torch.cuda.synchronize()
    prof = binding.dion2_profile_read()
    binding.dion2_profile_enable(False)
    for gi, ((W, M, _), (Ws, Ms, _)) in enumerate(zip(stacks, solo)):
        assert torch.equal(M, Ms), f"group {gi}: momentum"
        assert torch.equal(W.view(torch.int16), Ws.view(torch.int16)), f"group {gi}: weights"
    # one launch for the fused chain of the groups with s <= 64 (a, b, d),
    # a chain of 14 launches (5 Newton-Schulz steps) for c (s = 96, the same
    # padded size) and one for f (s = 256), plus the DIRECT group's 5
    # polynomial products
    assert prof["ns_poly"]["launches"] == 1 + 2 * 14 + 5
    # the first group against the oracle (its own call, with debug outputs)
    W, M, G = workloads.make_group(GROUPED, 0, hip_device)
    res = run_gpu(W, M, G, alpha, rand=(rand[0], rand[1], rand[2]) if rand else None)
    assert torch.equal(res["W"].view(torch.int16), solo[0][0].cpu().view(torch.int16))
    check_matrix(res, 1, alpha, rand=rand)


def test_groups_with_direct_transposed_operand(hip_device):
    """A grouped call whose first group takes the DIRECT form with X^T kept
    beside X (2048 x 2048 at alpha = 1) is bitwise the per-group calls."""
    wl = workloads.Workload("gxr", "test", (workloads.Group("a", 2048, 2048, 2), workloads.Group("b", 256, 384, 3)),
                            (1.0,))
    stacks = [workloads.make_group(wl, gi, hip_device) for gi in range(2)]
    solo = [tuple(t.clone() for t in st) for st in stacks]
    for W, M, G in solo:
        binding.dion2_step_ex(W, M, G, 1.0)
    binding.dion2_step_groups([(W, M, G, AXIS_AUTO) for W, M, G in stacks], 1.0)
    torch.cuda.synchronize()
    for gi, ((W, M, _), (Ws, Ms, _)) in enumerate(zip(stacks, solo)):
        assert torch.equal(M, Ms), f"group {gi}: momentum"
        assert torch.equal(W.view(torch.int16), Ws.view(torch.int16)), f"group {gi}: weights"


def test_groups_single_group_equals_strided(hip_device):
    """One group through the grouped entry point equals dion2_step_strided."""
    wl = one_group_workload(2048, 2048, count=4, name="g1")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W2, M2, G2 = W.clone(), M.clone(), G.clone()
    binding.dion2_step_strided(W, M, G, 0.25)
    binding.dion2_step_groups([(W2, M2, G2, AXIS_AUTO)], 0.25)
    torch.cuda.synchronize()
    assert torch.equal(M, M2) and torch.equal(W.view(torch.int16), W2.view(torch.int16))


def test_groups_at_the_group_limit(hip_device):
    """64 groups (the most one call takes), of varied small shapes and axes, on
    the most streams a call may use: bitwise the per-group calls."""
    shapes = [(64 + 16 * (g % 7), 96 + 32 * (g % 5), (AXIS_AUTO, AXIS_ROWS, AXIS_COLS)[g % 3]) for g in range(64)]
    wl = workloads.Workload("limit", "test", tuple(workloads.Group(f"g{g}", r, c, 1 + g % 2, ax)
                                                   for g, (r, c, ax) in enumerate(shapes)), (0.25,))
    stacks = [workloads.make_group(wl, gi, hip_device) for gi in range(64)]
    solo = [tuple(t.clone() for t in st) for st in stacks]
    for gi, (W, M, G) in enumerate(solo):
        binding.dion2_step_ex(W, M, G, 0.3, 0.95, 0.02, 5, wl.groups[gi].axis)
    binding.dion2_step_groups([(W, M, G, wl.groups[gi].axis) for gi, (W, M, G) in enumerate(stacks)],
                              0.3, 0.95, 0.02, 5, group_streams=8)
    torch.cuda.synchronize()
    for gi, ((W, M, _), (Ws, Ms, _)) in enumerate(zip(stacks, solo)):
        assert torch.equal(M, Ms), f"group {gi}: momentum"
        assert torch.equal(W.view(torch.int16), Ws.view(torch.int16)), f"group {gi}: weights"


@pytest.mark.parametrize("rows,cols,alpha", [(160, 640, 0.5), (384, 384, 0.5), (300, 200, 0.75),
                                              (257, 129, 1.0)])
def test_sixteen_newton_schulz_steps(hip_device, rows, cols, alpha):
    """The most steps a call takes, on near-square compact matrices (where AUTO
    would take DIRECT at 5 steps). DIRECT rounds X to bf16 after every step,
    so its error grows with the step count and it is refused past
    DION2_DIRECT_MAX_STEPS; every path the library accepts at 16 steps meets
    the 2e-2 bar: AUTO (which takes GRAM), GRAM, and the fp32 master at a
    tenth of it."""
    wl = one_group_workload(rows, cols, name=f"ns16-{rows}x{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    W1, M1 = W.clone(), M.clone()
    with pytest.raises(binding.Dion2Error) as ei:
        binding.dion2_step_ex(W1, M1, G, alpha, 0.95, 0.02, 16, ns_form=NS_DIRECT)
    assert ei.value.status == binding.DION2_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.equal(W1.view(torch.int16), W.view(torch.int16)) and torch.equal(M1, M), \
        "a refused call modified state"
    errs = {}
    for name, kw, tol in (("auto", dict(), NS_TOL), ("gram", dict(form=NS_GRAM), NS_TOL),
                          ("master", dict(master=binding.MASTER_FP32), MASTER_TOL)):
        res = run_gpu(W.clone(), M.clone(), G, alpha, ns_steps=16, **kw)
        errs[name] = check_matrix(res, 0, alpha, ns_steps=16, ns_tol=tol)
        if name == "auto":
            O_auto = res["O"]
        if name == "gram":
            assert torch.equal(res["O"], O_auto), "AUTO at 16 steps is not the GRAM form"
    assert errs["master"] < errs["gram"], errs
    print("16-step errors", errs)


@pytest.mark.parametrize("rows,cols,alpha", [(160, 640, 0.5), (384, 384, 0.5), (300, 200, 0.75),
                                              (257, 129, 1.0), (2048, 2048, 0.5)])
def test_direct_form_at_its_step_limit(hip_device, rows, cols, alpha):
    """DIRECT at DION2_DIRECT_MAX_STEPS (6) steps, the most it takes, stays
    within 2e-2 on near-square compact matrices; with 6 steps AUTO still
    takes it where the compact matrix is more than one tile a side and
    l < 3 s (bitwise the forced DIRECT), and the GRAM form elsewhere
    (80 x 640: one tile, where a forced DIRECT is refused)."""
    wl = one_group_workload(rows, cols, name=f"direct6-{rows}x{cols}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    res_auto = run_gpu(W.clone(), M.clone(), G, alpha, ns_steps=6)
    res_gram = run_gpu(W.clone(), M.clone(), G, alpha, ns_steps=6, form=NS_GRAM)
    if direct_refused(W, M, G, alpha):
        assert torch.equal(res_auto["O"], res_gram["O"]), "AUTO on one tile is not the GRAM form"
        return
    res = run_gpu(W.clone(), M.clone(), G, alpha, ns_steps=6, form=NS_DIRECT)
    err = check_matrix(res, 0, alpha, ns_steps=6)
    k = res["k"]
    d_oth = cols if res["axis"] == AXIS_ROWS else rows
    pad = lambda x: -(-x // 128) * 128   # noqa: E731
    s_pad, l_pad = pad(min(k, d_oth)), pad(max(k, d_oth))
    want = res if (s_pad > 128 and l_pad < 3 * s_pad) else res_gram
    assert torch.equal(res_auto["O"], want["O"]), "AUTO at 6 steps took the other form"
    print(f"DIRECT, 6 steps, {rows}x{cols} alpha {alpha}: {err:.3e}")


@pytest.mark.parametrize("case", ["f32-decay-all-schedule", "forced-direct", "forced-gram", "no-steps",
                                  "f16-chain", "f16-chain-schedule", "fp32-master"])
def test_groups_options_equal_per_group_calls(hip_device, case):
    """Options reach every group of a grouped call as they reach dion2_step_ex:
    fp32 W and G, the decay-all ablation, a per-step coefficient schedule, a
    forced Newton-Schulz form, and zero steps (O = the scaled compact matrix)."""
    wdt = "f32" if case.startswith("f32") else "bf16"
    shapes = ((256, 640, 2), (640, 256, 2), (128, 160, 1))
    if case == "forced-direct":   # (DIRECT takes compact matrices of more than one tile)
        shapes = ((640, 1024, 2), (1024, 640, 2), (600, 520, 1))
    wl = workloads.Workload("grouped-opt", "test", tuple(workloads.Group(n, r, c, b) for n, (r, c, b)
                                                          in zip("abc", shapes)), (0.25,), w_dtype=wdt)
    kw = {}
    ns_steps = 5
    if case == "f32-decay-all-schedule":
        kw = dict(decay_all=True,
                  ns_coeffs=[(3.4445, -4.7750, 2.0315)] * 3 + [(1.5, -0.5, 0.0)] * 2)
    elif case == "forced-direct":
        kw = dict(ns_form=NS_DIRECT)
    elif case == "forced-gram":
        kw = dict(ns_form=NS_GRAM)
    elif case == "f16-chain":
        kw = dict(ns_form=NS_GRAM, ns_chain=binding.CHAIN_F16)
    elif case == "fp32-master":
        kw = dict(ns_master=binding.MASTER_FP32)
    elif case == "f16-chain-schedule":
        kw = dict(ns_form=NS_GRAM, ns_chain=binding.CHAIN_F16,
                  ns_coeffs=[(3.4445, -4.7750, 2.0315)] * 4 + [(1.5, -0.5, 0.0)])
    else:
        ns_steps = 0
    stacks = [workloads.make_group(wl, gi, hip_device) for gi in range(len(wl.groups))]
    solo = [tuple(t.clone() for t in s) for s in stacks]
    for W, M, G in solo:
        binding.dion2_step_ex(W, M, G, 0.25, 0.95, 0.02, ns_steps, **kw)
    binding.dion2_step_groups([(W, M, G, AXIS_AUTO) for W, M, G in stacks], 0.25, 0.95, 0.02,
                              ns_steps, **kw)
    torch.cuda.synchronize()
    iview = torch.int32 if wdt == "f32" else torch.int16
    for gi, ((W, M, _), (Ws, Ms, _)) in enumerate(zip(stacks, solo)):
        assert torch.equal(M, Ms), f"group {gi}: momentum"
        assert torch.equal(W.view(iview), Ws.view(iview)), f"group {gi}: weights"
