"""The allocation-free entry point (dion2_step_noalloc) against dion2_step_ex:
the same kernels on the library's fixed scratch array instead of a
hipMalloc'd workspace, so every output is bitwise the same. Several calls
in a row with different, mostly smaller, inputs: the scratch keeps the
previous call's contents, and nothing in it may leak into the next result."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_16928_amd import binding, workloads
from paper_2512_16928_amd.binding import AXIS_AUTO, AXIS_COLS, AXIS_ROWS

pytestmark = pytest.mark.gpu


def wl_of(rows, cols, count, w_dtype="bf16", name="noalloc"):
    return workloads.Workload(name, "test", (workloads.Group("g", rows, cols, count),), (0.25,),
                              w_dtype=w_dtype)


# (rows, cols, batch, alpha, axis, options): each call smaller than the one
# before it, except the last, which runs the first shape again on the
# scratch the smaller calls left behind.
CALLS = [
    (2048, 2048, 4, 0.25, AXIS_AUTO, {}),                                    # rows, GRAM, fused update
    (640, 256, 3, 0.5, AXIS_AUTO, {}),                                       # columns, k > d_oth
    (384, 384, 2, 0.5, AXIS_ROWS, dict(ns_master=binding.MASTER_FP32)),     # fp32 master
    (200, 328, 1, 0.75, AXIS_AUTO, dict(ns_form=binding.NS_DIRECT)),        # DIRECT, ragged (s = 150)
    (2048, 2048, 1, 1.0, AXIS_AUTO, {}),                                     # DIRECT with X^T (s = 2048)
    (640, 256, 2, 0.25, AXIS_AUTO, dict(select_rule=binding.SELECT_RANDOM)),  # Random rule, one column pass
    (2048, 2048, 4, 0.25, AXIS_AUTO, {}),
]


def test_noalloc_equals_ex_calls_in_a_row(hip_device):
    assert binding.NOALLOC_SCRATCH_BYTES == 128 << 20
    for i, (rows, cols, batch, alpha, axis, kw) in enumerate(CALLS):
        need = binding.dion2_workspace_size_ex(batch, rows, cols, alpha, axis, 5, **kw)
        assert 0 < need <= binding.NOALLOC_SCRATCH_BYTES
        W, M, G = workloads.make_group(wl_of(rows, cols, batch, name=f"na{i}"), 0, hip_device)
        W2, M2 = W.clone(), M.clone()
        snap = (W[0].cpu(), M[0].cpu(), G[0].cpu())
        binding.dion2_step_noalloc(W, M, G, alpha, 0.95, 0.02, 5, axis, **kw)
        binding.dion2_step_ex(W2, M2, G, alpha, 0.95, 0.02, 5, axis, **kw)
        torch.cuda.synchronize()
        assert torch.equal(M, M2), f"call {i}: momentum"
        assert torch.equal(W.view(torch.int16), W2.view(torch.int16)), f"call {i}: weights"
        # and the first matrix against the oracle's momentum and selection
        rnd = dict(select="random", seed=0, step=0, matrix=0) if kw.get("select_rule") else {}
        out = oracle.dion2_step(snap[0].float().numpy().astype(np.float64), snap[1].numpy(),
                                snap[2].float().numpy(), alpha, 0.95, 0.02, 5, axis, w_dtype="bf16", **rnd)
        np.testing.assert_array_equal(M[0].cpu().numpy(), out["M"], err_msg=f"call {i}: momentum")
        sel = np.zeros(W.shape[1] if out["axis"] == AXIS_ROWS else W.shape[2], dtype=bool)
        sel[out["K"]] = True
        Wn, W0 = W[0].cpu(), snap[0]
        keep = ~sel
        if out["axis"] == AXIS_ROWS:
            assert torch.equal(Wn[keep], W0[keep]), f"call {i}: unselected rows written"
        else:
            assert torch.equal(Wn[:, keep], W0[:, keep]), f"call {i}: unselected columns written"


def test_noalloc_refusals_leave_state_untouched(hip_device):
    """A call beyond the scratch, and a call with a workspace of its own, are
    refused before anything runs."""
    rows, cols, batch = 2048, 8192, 16            # about 0.4 GB of workspace at alpha = 1
    assert binding.dion2_workspace_size_ex(batch, rows, cols, 1.0) > binding.NOALLOC_SCRATCH_BYTES
    W, M, G = workloads.make_group(wl_of(rows, cols, 2, name="na-big"), 0, hip_device)
    Wb = W.expand(batch // 2, 2, rows, cols).reshape(batch, rows, cols).contiguous()
    Mb = M.expand(batch // 2, 2, rows, cols).reshape(batch, rows, cols).contiguous()
    Gb = G.expand(batch // 2, 2, rows, cols).reshape(batch, rows, cols).contiguous()
    W0, M0 = Wb.clone(), Mb.clone()
    with pytest.raises(binding.Dion2Error) as ei:
        binding.dion2_step_noalloc(Wb, Mb, Gb, 1.0)
    assert ei.value.status == binding.DION2_ERR_WORKSPACE
    assert "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.equal(Wb.view(torch.int16), W0.view(torch.int16)) and torch.equal(Mb, M0)



def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


@pytest.mark.parametrize("name,rows,cols,batch,w_dtype,alpha,kw", [
    ("single-256", 256, 256, 1, "f32", 0.25, {}),              # one fp32 matrix: launch-bound
    ("bf16-group", 512, 1024, 4, "bf16", 0.25, {}),            # GRAM with the fused update
    ("random-cols", 640, 256, 2, "bf16", 0.25, dict(select_rule=binding.SELECT_RANDOM)),
])
def test_noalloc_step_in_a_hip_graph(hip_device, name, rows, cols, batch, w_dtype, alpha, kw):
    """dion2_step_noalloc captured in a HIP graph (it allocates nothing and
    issues only kernel launches) and replayed: every replay equals one eager
    dion2_step_ex step, bitwise, with other eager work and synchronisations
    between the replays."""
    wl = wl_of(rows, cols, batch, w_dtype=w_dtype, name=f"graph-{name}")
    W, M, G = workloads.make_group(wl, 0, hip_device)
    We, Me = W.clone(), M.clone()
    binding.dion2_step_noalloc(W, M, G, alpha, **kw)    # outside capture: the scratch address is taken
    binding.dion2_step_ex(We, Me, G, alpha, **kw)
    torch.cuda.synchronize()
    assert torch.equal(M, Me) and torch.equal(_bits(W), _bits(We))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        binding.dion2_step_noalloc(W, M, G, alpha, **kw)
    torch.cuda.synchronize()
    assert torch.equal(M, Me) and torch.equal(_bits(W), _bits(We)), "capture ran the step"
    for i in range(4):
        graph.replay()
        binding.dion2_step_ex(We, Me, G, alpha, **kw)
        junk = torch.randn(1 << 16, device=hip_device).square().sum()   # eager work between replays
        torch.cuda.synchronize()
        assert float(junk) > 0.0
        assert torch.equal(M, Me), f"replay {i}: momentum"
        assert torch.equal(_bits(W), _bits(We)), f"replay {i}: weights"
