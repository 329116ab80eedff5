"""Opt-in (DION2_FUZZ=<cases>): randomly drawn calls against the oracle --
shapes from 1 to 700 lines a side, selection fractions, axes, Newton-Schulz
forms and step counts, the fp32 master, fp32 W and G, the Random rule and
batches of one to three matrices -- each held to the same bar as the fixed
parity cases: K exact, M and the l1 norms bitwise, O within the tolerance of
its path, and W bitwise given O (or, for a forced DIRECT on a compact matrix
of one tile, the call refused). The draw is seeded, so case n is the same
call on every run."""
import os

import numpy as np
import pytest

from paper_2512_16928_amd import binding, workloads
from paper_2512_16928_amd.binding import AXIS_AUTO, AXIS_COLS, AXIS_ROWS, NS_AUTO, NS_DIRECT, NS_GRAM
from test_gpu_parity import MASTER_TOL, NS_TOL, check_matrix, direct_refused, one_group_workload, run_gpu

CASES = int(os.environ.get("DION2_FUZZ", "0") or 0)
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(CASES <= 0, reason="opt-in randomized sweep (set DION2_FUZZ=<cases>)")]

F16_TOL = 1e-1   # the fp16 chain loses the small directions of ill-conditioned Gram matrices


def draw(n):
    rng = np.random.default_rng([2512, 16928, n])
    small = rng.random() < 0.5
    hi = 130 if small else 700
    rows, cols = int(rng.integers(1, hi)), int(rng.integers(1, hi))
    alpha = float(rng.choice([0.01, 0.1, 0.25, 0.3, 0.5, 0.75, 1.0]))
    axis = int(rng.choice([AXIS_AUTO, AXIS_AUTO, AXIS_ROWS, AXIS_COLS]))
    master = binding.MASTER_FP32 if rng.random() < 0.15 else binding.MASTER_BF16
    form = NS_AUTO if master == binding.MASTER_FP32 else int(rng.choice([NS_AUTO, NS_AUTO, NS_DIRECT, NS_GRAM]))
    steps = int(rng.choice([0, 1, 2, 5, 5, 5, 6]))
    chain = binding.CHAIN_F16 if (form == NS_GRAM and steps >= 2 and rng.random() < 0.3) else binding.CHAIN_HILO
    wdt = "f32" if rng.random() < 0.25 else "bf16"
    rand = (int(rng.integers(0, 2**63)), int(rng.integers(0, 2**40)), int(rng.integers(0, 1000))) \
        if rng.random() < 0.2 else None
    batch = int(rng.integers(1, 4))
    return dict(rows=rows, cols=cols, alpha=alpha, axis=axis, form=form, steps=steps, chain=chain,
                master=master, wdt=wdt, rand=rand, batch=batch)


@pytest.mark.parametrize("n", range(max(CASES, 0)))
def test_random_call(hip_device, n):
    c = draw(n)
    print(f"case {n}: {c}", flush=True)
    wl = one_group_workload(c["rows"], c["cols"], count=c["batch"], axis=c["axis"], w_dtype=c["wdt"],
                            name=f"fuzz{n}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    if direct_refused(W, M, G, c["alpha"], c["axis"], c["form"]):
        return   # DIRECT on one tile: refused, nothing run
    res = run_gpu(W, M, G, c["alpha"], c["steps"], c["axis"], form=c["form"], rand=c["rand"],
                  chain=c["chain"], master=c["master"], norms=c["rand"] is None)
    tol = F16_TOL if c["chain"] == binding.CHAIN_F16 else (
        MASTER_TOL if c["master"] == binding.MASTER_FP32 else NS_TOL)
    for b in range(c["batch"]):
        check_matrix(res, b, c["alpha"], c["steps"], c["axis"], ns_tol=tol, rand=c["rand"])
