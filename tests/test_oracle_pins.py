"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these re-types an oracle formula: each compares the oracle with an
independent route to the same value (exact rational sums, brute-force sorts,
the SVD closed form of the Newton-Schulz polynomial, the polar factor, the
paper's own identities eq. (3) and eq. (4), a separately written Muon) or with
hand-worked special cases.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import AXIS_AUTO, AXIS_COLS, AXIS_ROWS, MUON_QUINTIC

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def scalar_ns(s, steps, coeffs=None):
    """The Newton-Schulz polynomial iterated on one scalar singular value."""
    coeffs = coeffs or [MUON_QUINTIC] * steps
    for t in range(steps):
        a, b, c = coeffs[t]
        s = a * s + b * s ** 3 + c * s ** 5
    return s


def svd_closed_form(X, steps, coeffs=None, eps=1e-7):
    """NS as a spectral function: U diag(p^T(sigma / (||X||_F + eps))) V^T."""
    U, S, Vt = np.linalg.svd(X, full_matrices=False)
    nf = math.sqrt(float(np.sum(S ** 2))) + eps
    P = np.array([scalar_ns(s / nf, steps, coeffs) for s in S])
    return (U * P) @ Vt


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


# ------------------------------------------------------------------ rounding

def _bf16_bits_rne(f32):
    """bf16 RNE of fp32 values by integer bit arithmetic (finite inputs)."""
    b = f32.view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def test_round_bf16_matches_bit_rounding():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(200000) * np.exp(rng.uniform(-60, 60, 200000))).astype(np.float32)
    np.testing.assert_array_equal(oracle.round_bf16(x.astype(np.float64)), _bf16_bits_rne(x))


def test_round_bf16_hand_cases():
    one = 1.0
    cases = {
        one + 2.0 ** -8: 1.0,                       # tie -> even (mantissa 0)
        one + 3 * 2.0 ** -8: one + 2.0 ** -6,       # tie -> even (round up)
        one + 2.0 ** -8 + 2.0 ** -30: one + 2.0 ** -7,  # just above the tie
        -(one + 2.0 ** -8): -1.0,
        2.0 ** -133: 2.0 ** -133,                   # smallest subnormal
        2.0 ** -134: 0.0,                           # tie to even (zero)
        3 * 2.0 ** -134: 2.0 ** -132,               # tie to even
        3.39e38: (2.0 - 2.0 ** -7) * 2.0 ** 127,    # rounds to the max finite
        3.4e38: math.inf,                           # past the midpoint to 2^128
    }
    for x, want in cases.items():
        assert oracle.round_bf16(np.float64(x)) == want, x


# ------------------------------------------------------- elementwise stages

def test_momentum_accumulate_is_single_fp32_rounding():
    # fl32(a + b) == float32(float64(a) + float64(b)) because fp64 carries
    # more than 2*24+2 bits (double rounding is innocuous for +).
    rng = np.random.default_rng(2)
    a = (rng.standard_normal(100000) * np.exp(rng.uniform(-40, 40, 100000))).astype(np.float32)
    b = (rng.standard_normal(100000) * np.exp(rng.uniform(-40, 40, 100000))).astype(np.float32)
    got = oracle.momentum_accumulate(a, b)
    assert got.dtype == np.float32
    want = (a.astype(np.float64) + b.astype(np.float64)).astype(np.float32)
    np.testing.assert_array_equal(got, want)


# ----------------------------------------------------------------- l1 norms

def test_l1_norm_is_exactly_rounded():
    rng = np.random.default_rng(3)
    M = (rng.standard_normal((7, 33)) * np.exp(rng.uniform(-30, 30, (7, 33)))).astype(np.float32)
    for axis in (AXIS_ROWS, AXIS_COLS):
        lines = M if axis == AXIS_ROWS else M.T
        want = [float(sum(Fraction(abs(float(v))) for v in line)) for line in lines]
        np.testing.assert_array_equal(oracle.l1_norms(M, axis), np.array(want))


def test_l1_norm_order_independent_where_naive_sum_is_not():
    # 2^60 followed by 200 ones: the exact sum 2^60 + 200 rounds to 2^60 + 256
    # in fp64, while a left-to-right fp64 sum stays at 2^60.
    row = np.array([2.0 ** 60] + [1.0] * 200, dtype=np.float32)[None, :]
    assert oracle.l1_norms(row, AXIS_ROWS)[0] == 2.0 ** 60 + 256
    assert oracle.l1_norms(row[:, ::-1], AXIS_ROWS)[0] == 2.0 ** 60 + 256


# ---------------------------------------------------------------- selection

def brute_topk(norms, k):
    key = [math.inf if math.isnan(v) else v for v in norms]
    order = sorted(range(len(key)), key=lambda i: (-key[i], i))
    return sorted(order[:k])


@pytest.mark.parametrize("seed", range(6))
def test_select_matches_bruteforce_with_ties(seed):
    rng = np.random.default_rng(seed)
    d = int(rng.integers(1, 300))
    norms = rng.integers(0, 12, d).astype(np.float64)   # many exact ties
    norms[rng.random(d) < 0.03] = np.nan
    norms[rng.random(d) < 0.03] = np.inf
    for k in {1, max(1, d // 4), max(1, d // 2), d}:
        assert list(oracle.select_top(norms, k)) == brute_topk(norms, k)


def test_select_hand_cases():
    assert list(oracle.select_top(np.zeros(8), 3)) == [0, 1, 2]
    assert list(oracle.select_top(np.ones(5), 5)) == [0, 1, 2, 3, 4]
    assert list(oracle.select_top(np.array([1.0, 5.0, 5.0, 2.0]), 1)) == [1]
    assert list(oracle.select_top(np.array([1.0, np.nan, 9.0]), 1)) == [1]
    assert list(oracle.select_top(np.array([3.0, 1.0, 2.0, 4.0]), 2)) == [0, 3]


def test_selection_ranks_by_l1_not_l2():
    # row 0: l1 = 3, l2 = 3; row 1: l1 = 4, l2 = 2 -> l1 picks row 1.
    M = np.array([[3, 0, 0, 0], [1, 1, 1, 1]], dtype=np.float32)
    out = oracle.dion2_step(np.zeros((2, 4)), M, np.zeros_like(M), alpha=0.5, ns_steps=0)
    assert list(out["K"]) == [1]


def test_num_selected_and_axis():
    assert oracle.num_selected(0.25, 256) == 64
    assert oracle.num_selected(1.0, 2048) == 2048
    assert oracle.num_selected(1e-6, 100) == 1
    assert oracle.num_selected(0.1, 2048) == 205   # fp32(0.1) > 0.1: ceil(204.8...)
    assert oracle.num_selected(0.125, 11008) == 1376
    with pytest.raises(ValueError):
        oracle.num_selected(0.0, 10)
    with pytest.raises(ValueError):
        oracle.num_selected(1.5, 10)
    assert oracle.resolve_axis(2048, 8192) == AXIS_ROWS
    assert oracle.resolve_axis(8192, 2048) == AXIS_COLS
    assert oracle.resolve_axis(2048, 2048) == AXIS_ROWS
    assert oracle.resolve_axis(2048, 8192, AXIS_COLS) == AXIS_COLS


# ------------------------------------------------------------ Newton-Schulz

@pytest.mark.parametrize("shape", [(16, 40), (40, 16), (33, 33), (64, 256), (5, 1)])
@pytest.mark.parametrize("steps", [0, 1, 5])
def test_ns_equals_spectral_closed_form(shape, steps):
    rng = np.random.default_rng(sum(shape) + steps)
    X = rng.standard_normal(shape) * np.exp(rng.standard_normal((shape[0], 1)))
    got = oracle.newton_schulz(X, steps)
    assert got.shape == X.shape
    assert rel(got, svd_closed_form(X, steps)) < 1e-12


def test_ns_custom_schedule_equals_closed_form():
    rng = np.random.default_rng(7)
    X = rng.standard_normal((24, 50))
    sched = [(3.0, -3.2, 1.2), (2.0, -1.5, 0.5), (1.5, -0.5, 0.0)]
    assert rel(oracle.newton_schulz(X, 3, sched), svd_closed_form(X, 3, sched)) < 1e-12


def test_ns_cubic_converges_to_polar_factor():
    # (a, b, c) = (1.5, -0.5, 0) is the classical cubic Newton-Schulz
    # iteration, whose limit is the polar factor U V^T.
    rng = np.random.default_rng(8)
    U, _ = np.linalg.qr(rng.standard_normal((30, 12)))
    V, _ = np.linalg.qr(rng.standard_normal((12, 12)))
    S = np.linspace(1.0, 0.05, 12)
    X = (U * S) @ V.T
    O = oracle.newton_schulz(X, 60, [(1.5, -0.5, 0.0)] * 60)
    assert rel(O, U @ V.T) < 1e-10


def test_ns_singular_values_in_polynomial_band():
    # The quintic maps normalised singular values in [2e-3, 1] into the band
    # spanned by p^5 over that interval; the matrix output must stay inside.
    grid = np.concatenate([np.linspace(2e-3, 1.0, 200001), [1.0]])
    img = np.array([scalar_ns(g, 5) for g in grid[::50]])
    lo, hi = img.min(), img.max()
    assert 0.68 < lo < 0.70 and 1.19 < hi < 1.21
    rng = np.random.default_rng(9)
    for shape in [(32, 128), (64, 64), (128, 40)]:
        U, _ = np.linalg.qr(rng.standard_normal((shape[0], min(shape))))
        V, _ = np.linalg.qr(rng.standard_normal((shape[1], min(shape))))
        S = np.exp(rng.uniform(np.log(0.05), 0, min(shape)))
        X = (U * S) @ V.T
        sv = np.linalg.svd(oracle.newton_schulz(X, 5), compute_uv=False)
        assert sv.min() >= lo - 1e-9 and sv.max() <= hi + 1e-9


def test_long_quintic_schedules_amplify_bf16_input_rounding():
    # Muon's quintic has no attracting fixed point: inside its band the slope
    # |p'| reaches about 1.58, so repeating it carries a perturbation of the
    # normalised input forward and enlarges it. The cubic step (1.5, -0.5, 0)
    # contracts toward 1 there. Rounding the input once to bf16 (the 16-bit
    # path's own first step) then moves the exact iteration's result by more
    # than 2e-2 after 16 quintic steps on compact matrices of a few lines,
    # while 5 quintic steps, or 5 followed by 11 cubic ones, stay well inside.
    band = np.linspace(0.68, 1.21, 2001)
    a, b, c = MUON_QUINTIC
    assert np.max(np.abs(a + 3 * b * band ** 2 + 5 * c * band ** 4)) > 1.5
    assert np.max(np.abs(1.5 - 1.5 * band ** 2)) < 1.0
    quintic = [MUON_QUINTIC] * 16
    tail = [MUON_QUINTIC] * 5 + [(1.5, -0.5, 0.0)] * 11
    for s in (3, 4):
        rng = np.random.default_rng(20 + s)
        worst = {"quintic16": 0.0, "tail16": 0.0, "quintic5": 0.0}
        for _ in range(24):
            X = rng.standard_normal((s, 40)) * np.exp(rng.standard_normal((s, 1)))
            Z = oracle.round_bf16(X / np.linalg.norm(X))
            for name, steps, sched in (("quintic16", 16, quintic), ("tail16", 16, tail),
                                       ("quintic5", 5, None)):
                e = rel(oracle.newton_schulz(Z, steps, sched, eps=0.0),
                        oracle.newton_schulz(X, steps, sched, eps=0.0))
                worst[name] = max(worst[name], e)
        assert worst["quintic16"] > 2e-2, (s, worst)
        assert worst["tail16"] < 5e-3 and worst["quintic5"] < 1e-2, (s, worst)


def test_ns_equivariance():
    rng = np.random.default_rng(10)
    X = rng.standard_normal((20, 48))
    P = rng.permutation(20)
    O = oracle.newton_schulz(X, 5)
    assert rel(oracle.newton_schulz(X[P], 5), O[P]) < 1e-12
    assert rel(oracle.newton_schulz(X.T, 5), O.T) < 1e-12
    # scale invariance is exact only without eps
    assert rel(oracle.newton_schulz(1e3 * X, 5, eps=0.0), oracle.newton_schulz(X, 5, eps=0.0)) < 1e-12


def test_ns_zero_matrix_gives_zero():
    assert not np.any(oracle.newton_schulz(np.zeros((4, 9)), 5))
    # with eps = 0 too: X / (||X||_F + eps) -> 0 as eps -> 0+ for X = 0, so no NaN
    out = oracle.newton_schulz(np.zeros((4, 9)), 5, eps=0.0)
    assert np.all(np.isfinite(out)) and not np.any(out)
    # and the step: W unchanged, M decayed on the first k lines (all tied)
    M = np.zeros((6, 8))
    res = oracle.dion2_step(np.ones((6, 8)), M, np.zeros_like(M), alpha=0.5, eps=0.0)
    assert np.array_equal(res["W"], np.ones((6, 8))) and not np.any(res["O"])


# --------------------------------------- paper identities: eq. (3), eq. (4)

@pytest.mark.parametrize("axis", [AXIS_ROWS, AXIS_COLS])
def test_compact_equals_masked_dense_eq3(axis):
    # eq. (3) with V a line selector: NS of the matrix with unselected lines
    # zeroed equals the compact NS result placed back, zeros elsewhere.
    rng = np.random.default_rng(11 + axis)
    M = rng.standard_normal((40, 56))
    d_sel = 40 if axis == AXIS_ROWS else 56
    K = np.sort(rng.choice(d_sel, 13, replace=False))
    dense = np.zeros_like(M)
    padded = np.zeros_like(M)
    O = oracle.newton_schulz(oracle.gather(M, K, axis), 5)
    if axis == AXIS_ROWS:
        dense[K, :] = M[K, :]
        padded[K, :] = O
    else:
        dense[:, K] = M[:, K]
        padded[:, K] = O
    assert rel(oracle.newton_schulz(dense, 5), padded) < 1e-12


@pytest.mark.parametrize("axis", [AXIS_ROWS, AXIS_COLS])
def test_selective_decay_is_error_feedback_eq4(axis):
    # eq. (4): M <- M - (1 - mu) M V V^T (columns; rows use V V^T M) with V
    # the selector of K reduces to the selective decay of eq. (2).
    rng = np.random.default_rng(12 + axis)
    M = rng.standard_normal((30, 45))
    d_sel = 30 if axis == AXIS_ROWS else 45
    K = np.sort(rng.choice(d_sel, 9, replace=False))
    V = np.zeros((d_sel, len(K)))
    V[K, np.arange(len(K))] = 1.0
    mu = 0.75   # exact in fp32, so the library's fp32 mu is this value
    ef = M - (1 - mu) * (V @ V.T @ M if axis == AXIS_ROWS else M @ V @ V.T)
    got = oracle.selective_decay(M, K, mu, axis, store="fp64")
    np.testing.assert_allclose(got, ef, rtol=1e-15, atol=1e-15)


# ---------------------------------------------------- whole-step properties

def make_case(rng, rows, cols, dtype="f32"):
    r = np.exp(rng.standard_normal((rows, 1)))
    G = (r * rng.standard_normal((rows, cols))).astype(np.float32)
    M = (r * rng.standard_normal((rows, cols))).astype(np.float32)
    W = oracle.round_to(0.02 * rng.standard_normal((rows, cols)), dtype)
    return W, M, G


@pytest.mark.parametrize("rows,cols,axis", [(48, 64, AXIS_AUTO), (64, 48, AXIS_AUTO),
                                            (40, 40, AXIS_COLS)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unselected_lines_untouched_and_momentum_exact(rows, cols, axis, dtype):
    rng = np.random.default_rng(rows * cols)
    W, M, G = make_case(rng, rows, cols, dtype)
    out = oracle.dion2_step(W, M, G, alpha=0.25, axis=axis, w_dtype=dtype)
    ax = out["axis"]
    d_sel = rows if ax == AXIS_ROWS else cols
    sel = np.zeros(d_sel, bool)
    sel[out["K"]] = True
    acc = (M.astype(np.float64) + G.astype(np.float64)).astype(np.float32)
    dec = (np.float64(np.float32(0.95)) * acc.astype(np.float64)).astype(np.float32)
    Wn, Mn = out["W"], out["M"]
    if ax == AXIS_COLS:
        W, Wn, Mn, acc, dec = W.T, Wn.T, Mn.T, acc.T, dec.T
    np.testing.assert_array_equal(Wn[~sel], W[~sel])
    np.testing.assert_array_equal(Mn[~sel], acc[~sel])
    np.testing.assert_array_equal(Mn[sel], dec[sel])
    assert np.all(Wn[sel] != W[sel]) or dtype == "bf16"
    assert len(out["K"]) == out["k"] == math.ceil(0.25 * d_sel)


def test_alpha_one_is_muon_trajectory():
    # Dion2 with alpha = 1 is Muon: B <- mu B + G, W <- W - lr sqrt(m/n) NS(B),
    # here with NS taken as the SVD closed form and fp64 state throughout.
    rng = np.random.default_rng(13)
    rows, cols, mu, lr = 24, 40, 0.95, 0.02
    W0 = 0.02 * rng.standard_normal((rows, cols))
    Wd, Md = W0.copy(), np.zeros((rows, cols))
    Wm, B = W0.copy(), np.zeros((rows, cols))
    for _ in range(5):
        G = rng.standard_normal((rows, cols))
        out = oracle.dion2_step(Wd, Md, G, alpha=1.0, mu=mu, lr=lr, w_dtype="f64", store="fp64")
        Wd, Md = out["W"], out["M"]
        B = np.float64(np.float32(mu)) * B + G
        Wm = Wm - float(np.float32(lr)) * math.sqrt(rows / cols) * svd_closed_form(B, 5)
        assert rel(Wd, Wm) < 1e-12


@pytest.mark.parametrize("rows,cols", [(24, 60), (60, 24)])
def test_update_spectral_norm_matches_eq1(rows, cols):
    rng = np.random.default_rng(14)
    W, M, G = make_case(rng, rows, cols)
    W = W.astype(np.float64)
    out = oracle.dion2_step(W, M, G, alpha=0.5, w_dtype="f64")
    dW = W - out["W"]
    X = oracle.gather(oracle.momentum_accumulate(M, G), out["K"], out["axis"])
    sv = np.linalg.svd(X, compute_uv=False)
    nf = math.sqrt(float(np.sum(sv ** 2))) + 1e-7
    want = float(np.float32(0.02)) * math.sqrt(rows / cols) * max(scalar_ns(s / nf, 5) for s in sv)
    assert abs(np.linalg.norm(dW, 2) - want) < 1e-12 * want


def test_column_mode_is_row_mode_of_transpose():
    rng = np.random.default_rng(15)
    W, M, G = make_case(rng, 36, 52)
    c = oracle.dion2_step(W, M, G, alpha=0.25, axis=AXIS_COLS, w_dtype="f64")
    r = oracle.dion2_step(W.T, M.T, G.T, alpha=0.25, axis=AXIS_ROWS, w_dtype="f64")
    assert list(c["K"]) == list(r["K"])
    np.testing.assert_array_equal(c["M"], r["M"].T)
    assert rel(c["O"], r["O"].T) < 1e-13
    ratio = math.sqrt(36 / 52) / math.sqrt(52 / 36)
    assert rel(W - c["W"], ratio * (W.T - r["W"]).T) < 1e-12


def test_zero_momentum_and_gradient():
    W = oracle.round_to(np.random.default_rng(16).standard_normal((8, 12)), "bf16")
    z = np.zeros((8, 12), np.float32)
    out = oracle.dion2_step(W, z, z, alpha=0.25, w_dtype="bf16")
    assert list(out["K"]) == [0, 1]
    np.testing.assert_array_equal(out["W"], W)
    assert not np.any(out["M"])


def test_nan_line_is_selected():
    rng = np.random.default_rng(17)
    W, M, G = make_case(rng, 16, 20)
    M[5, 3] = np.nan
    out = oracle.dion2_step(W, M, G, alpha=0.125)
    assert 5 in out["K"]


def test_decay_all_ablation():
    rng = np.random.default_rng(18)
    W, M, G = make_case(rng, 16, 20)
    out = oracle.dion2_step(W, M, G, alpha=0.25, decay_all=True)
    acc = oracle.momentum_accumulate(M, G)
    np.testing.assert_array_equal(out["M"], np.float32(0.95) * acc)


def test_ns_steps_zero_is_normalised_input():
    rng = np.random.default_rng(19)
    W, M, G = make_case(rng, 16, 24)
    out = oracle.dion2_step(W, M, G, alpha=0.5, ns_steps=0)
    X = oracle.gather(oracle.momentum_accumulate(M, G), out["K"], out["axis"])
    assert rel(out["O"], X / (np.linalg.norm(X) + 1e-7)) < 1e-15


def test_paper_constants_are_the_defaults():
    with open(os.path.join(GOLDEN, "paper_constants.json")) as f:
        pc = json.load(f)
    assert oracle.DEFAULT_MU == pc["mu"]["value"]
    assert oracle.DEFAULT_LR == pc["lr"]["value"]
    # the swept fractions give integer line counts at the paper's widths
    for a in pc["alphas_swept"]["value"]:
        for d in (1024, 2048):
            assert oracle.num_selected(a, d) == a * d


# ---- Random rule (Algorithm 1, selection step; Sec. 3.1) --------------------

# Published known-answer values of Philox-4x32-10 (Salmon et al., SC 2011):
# (counter words, key words) -> output words.
PHILOX_KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,want", PHILOX_KAT)
def test_philox_known_answers(ctr, key, want):
    got = tuple(int(x) for x in oracle.philox4x32_10(ctr, key))
    assert got == want


def test_philox_broadcasts_like_scalar_calls():
    ctr = np.array([[i, 7, 9, 11] for i in range(5)], dtype=np.uint32)
    batch = oracle.philox4x32_10(ctr, (3, 4))
    for i in range(5):
        assert tuple(batch[i]) == tuple(oracle.philox4x32_10(ctr[i], (3, 4)))


def test_random_selection_is_the_k_smallest_keys():
    """Brute force: sort (key, index) pairs with Python's sort."""
    for d, k, seed, step, m in [(37, 5, 1, 0, 0), (300, 75, 2**40 + 3, 2**33 + 1, 17), (8, 8, 5, 6, 7)]:
        keys = oracle.random_line_keys(d, seed, step, m)
        want = sorted(i for _, i in sorted((int(kk), i) for i, kk in enumerate(keys))[:k])
        assert oracle.select_random(d, k, seed, step, m).tolist() == want


def test_random_selection_valid_and_keyed():
    K = oracle.select_random(1000, 250, 42, 3, 5)
    assert len(K) == 250 and len(set(K.tolist())) == 250
    assert np.all(np.diff(K) > 0) and K[0] >= 0 and K[-1] < 1000
    assert np.array_equal(K, oracle.select_random(1000, 250, 42, 3, 5))       # deterministic
    for other in [(43, 3, 5), (42, 4, 5), (42, 3, 6)]:                          # seed, step, matrix
        assert not np.array_equal(K, oracle.select_random(1000, 250, *other))


def test_random_selection_is_uniform():
    """Each line's inclusion count over 3000 draws is Binomial(3000, k/d):
    within 5 standard deviations of its mean."""
    d, k, n = 40, 10, 3000
    counts = np.zeros(d)
    for step in range(n):
        counts[oracle.select_random(d, k, 99, step, 0)] += 1
    mean, sd = n * k / d, np.sqrt(n * (k / d) * (1 - k / d))
    assert np.all(np.abs(counts - mean) < 5 * sd)


def test_step_with_random_selection():
    rng = np.random.default_rng(23)
    W, M, G = make_case(rng, 32, 48)     # rows are selected: d_sel = 32, k = 8
    out = oracle.dion2_step(W, M, G, alpha=0.25, select="random", seed=7, step=2, matrix=1)
    K = out["K"]
    assert K.tolist() == oracle.select_random(32, 8, 7, 2, 1).tolist()
    keep = [i for i in range(32) if i not in set(K.tolist())]
    np.testing.assert_array_equal(out["W"][keep], W[keep])
    acc = oracle.momentum_accumulate(M, G)
    np.testing.assert_array_equal(out["M"][keep], acc[keep])
