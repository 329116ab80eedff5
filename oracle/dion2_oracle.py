"""Plain, slow CPU reference ("oracle") for the Dion2 optimizer step.

TEST INFRASTRUCTURE. Only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark may import this module. The product path (the HIP
library and its Python binding) never calls it, and this module imports
nothing from the product package.

What it computes follows the paper "Dion2: A Simple Method to Shrink Matrix in
Muon" (Ahn, Amsel, Langford):

  Algorithm 1 (row-selection version; columns analogous), per weight matrix W
  with momentum M and gradient G:
      M <- M + G                                   (accumulate)
      K <- Select_alpha(M)                         (alpha-fraction of lines)
      O <- NewtonSchulz(M[K, :])                   (orthonormalise submatrix)
      M[K, :] <- mu * M[K, :]                      (selective decay, eq. (2))
      W[K, :] <- W[K, :] - lr*sqrt(fan_out/fan_in)*O   (sparse update, eq. (1))

Precision: fp64 everywhere except where storage fixes the precision. The
momentum is stored in fp32, so the accumulate and the decay are fp32 IEEE
round-to-nearest-even operations (exactly what fp32 storage implies); W is
rounded once, round-to-nearest-even, to its storage type (fp32 or bf16).

Readings taken where the paper is silent (each one is listed with its reason
in the design notes):
  * Newton-Schulz: Muon's quintic p(x) = a x + b x^3 + c x^5 with
    (a, b, c) = (3.4445, -4.7750, 2.0315) at every step, input divided by
    (Frobenius norm + eps), eps = 1e-7, iterated on the orientation with the
    smaller Gram matrix (Sec. 1 and Algorithm 1 name the iteration but give
    neither coefficients, step count nor normalisation).
  * Select_alpha, Default rule: the k = ceil(alpha * d) lines of largest l1
    norm, ties to the lower index, NaN ranked as +inf, K returned ascending.
    The l1 norm is the exact sum of |M_ij| over the line, rounded once to
    fp64 (math.fsum), so it does not depend on a summation order.
  * Axis AUTO selects along the shorter dimension (Sec. 4, experimental
    details); a square matrix selects rows.
  * sqrt(fan_out/fan_in) uses the full W's rows/cols (y = W x, so
    fan_out = rows, fan_in = cols; Sec. 1, eq. (1)).
"""
from __future__ import annotations

import math

import numpy as np

AXIS_AUTO = -1
AXIS_ROWS = 0
AXIS_COLS = 1

# Muon's quintic Newton-Schulz coefficients (a, b, c); the paper cites Muon
# for the iteration (Sec. 1) without printing them.
MUON_QUINTIC = (3.4445, -4.7750, 2.0315)
DEFAULT_EPS = 1e-7
DEFAULT_MU = 0.95    # Algorithm 1, its momentum decay hyperparameter
DEFAULT_LR = 0.02    # Sec. 4, experimental details


# ---------------------------------------------------------------- rounding

def round_bf16(x):
    """Round fp64 values to bfloat16, round-to-nearest-even, returned as fp64.

    bfloat16 keeps 8 significant bits and fp32's exponent range. The value is
    written as an integer multiple of its quantum 2^q (q = exponent - 8, and
    never below the subnormal quantum 2^-133), the multiple is rounded with
    np.rint (ties to even), and overflow beyond the largest finite bf16 goes
    to +-inf. NaN propagates.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                        # x = m * 2^e, 0.5 <= |m| < 1
    q = np.maximum(e - 8, -133)
    r = np.ldexp(np.rint(np.ldexp(x, -q)), q)
    max_bf16 = (2.0 - 2.0 ** -7) * 2.0 ** 127
    r = np.where(np.abs(r) > max_bf16, np.copysign(np.inf, x), r)
    return np.where(np.isnan(x), x, r)


def round_to(x, dtype):
    """Round fp64 values to the storage type 'f32' or 'bf16' (RNE), as fp64;
    'f64' keeps them (used by identity checks that must not round)."""
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        return round_bf16(x)
    raise ValueError(f"unknown dtype {dtype!r}")


# ---------------------------------------------------------------- the steps

def resolve_axis(rows, cols, axis=AXIS_AUTO):
    """Selection axis. AUTO picks the shorter dimension (Sec. 4, details);
    a square matrix selects rows."""
    if axis == AXIS_AUTO:
        return AXIS_ROWS if rows <= cols else AXIS_COLS
    if axis not in (AXIS_ROWS, AXIS_COLS):
        raise ValueError(f"bad axis {axis}")
    return axis


def num_selected(alpha, d_sel):
    """k = ceil(alpha * d_sel), clamped to [1, d_sel]: the fraction alpha of
    lines that Algorithm 1 selects. alpha is taken as the fp32 value the
    library receives."""
    a = float(np.float32(alpha))
    if not (0.0 < a <= 1.0):
        raise ValueError(f"alpha must be in (0, 1], got {alpha}")
    return int(min(d_sel, max(1, math.ceil(a * d_sel))))


def momentum_accumulate(M, G):
    """M <- M + G (Algorithm 1, accumulate step), in fp32 arithmetic because the
    momentum is stored in fp32. G holds values exactly representable in fp32
    (fp32 or bf16 storage)."""
    return np.asarray(M, dtype=np.float32) + np.asarray(G, dtype=np.float32)


def l1_norms(M, axis):
    """l1 norm of every line along the selection axis (Select_alpha, Default
    rule of Algorithm 1 ranks lines by this norm). Each norm is the exact sum
    of absolute values, rounded once to fp64."""
    A = np.abs(np.asarray(M, dtype=np.float64))
    lines = A if axis == AXIS_ROWS else A.T
    return np.array([math.fsum(line.tolist()) for line in lines], dtype=np.float64)


def select_top(norms, k):
    """Select_alpha, Default rule: indices of the k largest norms, ties to the
    lower index, NaN ranked as +inf; returned in ascending index order."""
    key = np.where(np.isnan(norms), np.inf, norms)
    order = np.lexsort((np.arange(key.size), -key))
    return np.sort(order[:k]).astype(np.int64)


# Philox-4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers:
# as easy as 1, 2, 3", SC 2011): a keyed bijection on 128-bit counters made
# of ten rounds; each round multiplies two of the four words by fixed odd
# constants, swaps the halves and mixes in the round key, and the key is
# bumped by the Weyl constants between rounds.
PHILOX_M = (0xD2511F53, 0xCD9E8D57)     # round multipliers
PHILOX_W = (0x9E3779B9, 0xBB67AE85)     # key increments (golden ratio, sqrt(3) - 1)
_U32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(counter, key):
    """Philox-4x32-10 of uint32 arrays counter [..., 4] and key [..., 2]
    (broadcasting); returns uint32 [..., 4]."""
    counter = np.asarray(counter, dtype=np.uint64)
    key = np.asarray(key, dtype=np.uint64)
    c0, c1, c2, c3 = (counter[..., i] & _U32 for i in range(4))
    k0, k1 = key[..., 0] & _U32, key[..., 1] & _U32
    m0, m1 = np.uint64(PHILOX_M[0]), np.uint64(PHILOX_M[1])
    for r in range(10):
        if r:
            k0 = (k0 + np.uint64(PHILOX_W[0])) & _U32
            k1 = (k1 + np.uint64(PHILOX_W[1])) & _U32
        p0 = c0 * m0                       # 32 x 32 -> 64 bits, exact in uint64
        p1 = c2 * m1
        c0, c1, c2, c3 = ((p1 >> np.uint64(32)) ^ c1 ^ k0, p1 & _U32,
                          (p0 >> np.uint64(32)) ^ c3 ^ k1, p0 & _U32)
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def random_line_keys(d_sel, seed, step, matrix):
    """64-bit key of every line for the Random rule: Philox-4x32-10 of the
    counter (line, matrix, step low word, step high word) under the key
    (seed low word, seed high word); the first two output words, high first."""
    i = np.arange(d_sel, dtype=np.uint64)
    seed, step, matrix = int(seed), int(step), int(matrix)
    ctr = np.stack([i, np.full_like(i, matrix & 0xFFFFFFFF), np.full_like(i, step & 0xFFFFFFFF),
                    np.full_like(i, step >> 32)], axis=-1)
    out = philox4x32_10(ctr, [seed & 0xFFFFFFFF, seed >> 32]).astype(np.uint64)
    return (out[..., 0] << np.uint64(32)) | out[..., 1]


def select_random(d_sel, k, seed, step, matrix):
    """Select_alpha, Random rule (Algorithm 1, selection step: lines chosen
    uniformly at random; Sec. 3.1): the k lines with the smallest keys
    (i.i.d. uniform, so every k-subset is equally likely), ties to the lower
    index, returned ascending."""
    keys = random_line_keys(d_sel, seed, step, matrix)
    order = np.lexsort((np.arange(d_sel), keys))
    return np.sort(order[:k]).astype(np.int64)


def gather(M, K, axis):
    """The submatrix M[K, :] (rows) or M[:, K] (columns), in fp64."""
    M = np.asarray(M, dtype=np.float64)
    return M[K, :].copy() if axis == AXIS_ROWS else M[:, K].copy()


def newton_schulz(X, steps, coeffs=None, eps=DEFAULT_EPS):
    """Newton-Schulz orthonormalisation (Sec. 1; Algorithm 1, orthonormalisation step).

    X is divided by (||X||_F + eps); then each step t applies
        A = X X^T,  B = b_t A + c_t A^2,  X <- a_t X + B X,
    i.e. X <- p_t(X) for the odd polynomial p_t(x) = a x + b x^3 + c x^5
    acting on the singular values. The iteration runs on the orientation with
    the smaller Gram matrix (the result is the same spectral function either
    way). coeffs is a list of (a, b, c) per step, or None for Muon's quintic.
    """
    X = np.asarray(X, dtype=np.float64)
    if coeffs is None:
        coeffs = [MUON_QUINTIC] * steps
    if len(coeffs) < steps:
        raise ValueError("need one (a, b, c) per Newton-Schulz step")
    tall = X.shape[0] > X.shape[1]
    if tall:
        X = X.T
    # a zero X with eps = 0 leaves the normalisation 0 / 0; it is taken at its
    # limit as eps -> 0+, where X / (||X||_F + eps) = 0, so O = 0
    d = np.linalg.norm(X) + eps
    X = X / d if d > 0 else X
    for t in range(steps):
        a, b, c = coeffs[t]
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    return X.T.copy() if tall else X


def selective_decay(M, K, mu, axis, store="fp32", decay_all=False):
    """M[K, :] <- mu * M[K, :] (eq. (2); Algorithm 1, decay step), in the
    momentum's storage precision. decay_all=True is the ablation of Sec. 4.2
    (M <- mu * M)."""
    if store == "fp32":
        M = np.array(M, dtype=np.float32)
        m = np.float32(mu)
    else:
        M = np.array(M, dtype=np.float64)
        m = np.float64(np.float32(mu))   # mu as the fp32 value the library receives
    if decay_all:
        M = m * M
    elif axis == AXIS_ROWS:
        M[K, :] = m * M[K, :]
    else:
        M[:, K] = m * M[:, K]
    return M


def update_scale(lr, rows, cols):
    """lr * sqrt(fan_out / fan_in) for W in R^{fan_out x fan_in} (eq. (1)),
    lr taken as the fp32 value the library receives."""
    return float(np.float32(lr)) * math.sqrt(rows / cols)


def apply_update(W, K, O, lr, axis, w_dtype):
    """W[K, :] <- W[K, :] - lr*sqrt(fan_out/fan_in)*O (Algorithm 1, sparse update step;
    eq. (1)); columns analogously. Computed in fp64 and rounded once to W's
    storage type; lines outside K are left untouched."""
    W = np.array(W, dtype=np.float64)
    rows, cols = W.shape
    s = update_scale(lr, rows, cols)
    if axis == AXIS_ROWS:
        W[K, :] = round_to(W[K, :] - s * O, w_dtype)
    else:
        W[:, K] = round_to(W[:, K] - s * O, w_dtype)
    return W


def dion2_step(W, M, G, alpha, mu=DEFAULT_MU, lr=DEFAULT_LR, ns_steps=5,
               axis=AXIS_AUTO, coeffs=None, eps=DEFAULT_EPS, w_dtype="f32",
               store="fp32", decay_all=False, select="l1", seed=0, step=0, matrix=0):
    """One Dion2 step on one matrix (Algorithm 1). Inputs are not modified.

    W: (rows, cols) values of W's storage type w_dtype ('f32' | 'bf16').
    M: (rows, cols) momentum (fp32 storage; store='fp64' keeps it in fp64).
    G: (rows, cols) gradient values.
    Returns a dict with the new W (fp64 array of w_dtype values), the new M,
    the selected indices K (ascending), the Newton-Schulz output O in the
    submatrix's own orientation (k x cols for rows, rows x k for columns),
    the l1 norms, and the resolved axis. select='random' takes the Random
    rule keyed by (seed, step, matrix).
    """
    W = np.asarray(W)
    rows, cols = W.shape
    ax = resolve_axis(rows, cols, axis)
    d_sel = rows if ax == AXIS_ROWS else cols
    k = num_selected(alpha, d_sel)
    if store == "fp32":
        M1 = momentum_accumulate(M, G)
    else:
        M1 = np.asarray(M, dtype=np.float64) + np.asarray(G, dtype=np.float64)
    norms = l1_norms(M1, ax)
    if select == "l1":
        K = select_top(norms, k)
    elif select == "random":
        K = select_random(d_sel, k, seed, step, matrix)
    else:
        raise ValueError(select)
    X = gather(M1, K, ax)
    O = newton_schulz(X, ns_steps, coeffs, eps)
    M2 = selective_decay(M1, K, mu, ax, store, decay_all)
    W2 = apply_update(W, K, O, lr, ax, w_dtype)
    return {"W": W2, "M": M2, "K": K, "O": O, "norms": norms, "axis": ax,
            "k": k}
