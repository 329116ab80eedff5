"""Opt-in (DION2_FULL_SWEEP=1, about four minutes on one MI355X): every
matrix of the 1B-style stack against the oracle at each selection fraction
the benchmark reports, each group in the one batched call the benchmark
times. The default suite checks sampled matrices of the same calls."""
import os

import pytest
import torch

from paper_2512_16928_amd import binding, workloads
from paper_2512_16928_amd.binding import AXIS_ROWS
from test_gpu_parity import check_matrix

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not os.environ.get("DION2_FULL_SWEEP"),
                                 reason="opt-in sweep over every matrix (set DION2_FULL_SWEEP=1)")]


@pytest.mark.parametrize("alpha", [0.25, 0.5, 1.0])
@pytest.mark.parametrize("gi", [0, 1, 2], ids=["2048x2048", "8192x2048", "2048x8192"])
def test_every_matrix_of_the_1b_stack(hip_device, gi, alpha):
    wl = workloads.WORKLOADS["1b"]
    grp = wl.groups[gi]
    W, M, G = workloads.make_group(wl, gi, hip_device)
    k, ax = binding.dion2_plan_info(grp.rows, grp.cols, alpha, grp.axis)
    d_sel, d_oth = (grp.rows, grp.cols) if ax == AXIS_ROWS else (grp.cols, grp.rows)
    sel = torch.empty((grp.count, k), dtype=torch.int32, device=hip_device)
    nrm = torch.empty((grp.count, d_sel), dtype=torch.float64, device=hip_device)
    upd = torch.empty((grp.count, k, d_oth), dtype=torch.float32, device=hip_device)
    W0, M0, G0 = W.cpu(), M.cpu(), G.cpu()
    binding.dion2_step_ex(W, M, G, alpha, dbg_sel_idx=sel, dbg_norms=nrm, dbg_update=upd)
    torch.cuda.synchronize()
    Wc, Mc, sc, nc, uc = W.cpu(), M.cpu(), sel.cpu(), nrm.cpu(), upd.cpu()
    for b in range(grp.count):
        res = dict(W0=W0[b][None], M0=M0[b][None], G=G0[b][None], W=Wc[b][None], M=Mc[b][None],
                   K=sc[b][None], norms=nc[b][None], O=uc[b][None], axis=ax, k=k)
        check_matrix(res, 0, alpha)
