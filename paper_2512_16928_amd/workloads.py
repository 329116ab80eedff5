"""Seeded synthetic optimizer states for the Dion2 step.

Shapes follow the paper's models (Table 1: d_model 2048, 16 layers for the
1.01B model) and the larger stacks the step is measured on. This module only
draws random numbers into tensors of those shapes; it holds none of the
step's arithmetic, so the HIP path and the CPU oracle can both be fed from
it.

Recipe (every workload):
  * W ~ N(0, 0.02^2), rounded to W's storage type.
  * per matrix and row i a scale r_i = exp(N(0, 1)) (log-normal), shared by
    the gradient and the prior momentum of that row;
  * G = r_i * N(0, g_std^2) and M0 = r_i * N(0, g_std^2), independent draws;
    G is stored like W (bf16, or fp32 for the single-matrix case), M0 in fp32.
  * optional: a seeded 5% of the lines along the group's (explicit) selection
    axis get G scaled by 20; a seeded 30% of the matrices in each block of
    experts get G = 0.
"""
from __future__ import annotations

import dataclasses
import zlib

import torch

AXIS_AUTO, AXIS_ROWS, AXIS_COLS = -1, 0, 1


@dataclasses.dataclass(frozen=True)
class Group:
    """`count` same-shape matrices [rows, cols] (rows = fan-out)."""
    name: str
    rows: int
    cols: int
    count: int
    axis: int = AXIS_AUTO
    spike_frac: float = 0.0     # lines (on `axis`) whose gradient is x20
    zero_frac: float = 0.0      # matrices per block of `zero_block` with G = 0
    zero_block: int = 0


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    description: str
    groups: tuple
    alphas: tuple
    w_dtype: str = "bf16"       # 'bf16' | 'f32' (W and G storage)
    g_std: float = 1e-3
    mu: float = 0.95
    lr: float = 0.02
    ns_steps: int = 5

    def matrices(self) -> int:
        return sum(g.count for g in self.groups)

    def elements(self) -> int:
        return sum(g.count * g.rows * g.cols for g in self.groups)


def _stack_1b(axis_up=AXIS_AUTO, axis_down=AXIS_AUTO, axis_attn=AXIS_AUTO, spike=0.0):
    L = 16
    return (Group("attn 2048x2048", 2048, 2048, 4 * L, axis_attn, spike),
            Group("mlp 8192x2048", 8192, 2048, L, axis_up, spike),
            Group("mlp 2048x8192", 2048, 8192, L, axis_down, spike))


WORKLOADS = {
    "single-256": Workload(
        "single-256", "one 256x256 fp32 matrix (fp32 W and G), rows, alpha 0.25",
        (Group("w 256x256", 256, 256, 1, AXIS_ROWS),), (0.25,), w_dtype="f32", g_std=1.0),
    "1b": Workload(
        "1b", "1B-style stack: 16 layers, d_model 2048, 4x 2048x2048 attention, "
        "8192x2048 + 2048x8192 MLP per layer; bf16 W/G, fp32 M; shorter-side selection",
        _stack_1b(), (0.25, 0.5, 1.0)),
    "1b-colsel": Workload(
        "1b-colsel", "1B-style stack, columns selected for 2048x8192 and rows elsewhere, "
        "5% of selection-axis lines with x20 gradients",
        _stack_1b(axis_up=AXIS_ROWS, axis_down=AXIS_COLS, axis_attn=AXIS_ROWS, spike=0.05),
        (0.25,)),
    "7b": Workload(
        "7b", "7B-style stack: 32 layers, d_model 4096, 4x 4096x4096 attention, "
        "2x 11008x4096 + 1x 4096x11008 SwiGLU MLP per layer",
        (Group("attn 4096x4096", 4096, 4096, 128),
         Group("mlp 11008x4096", 11008, 4096, 64),
         Group("mlp 4096x11008", 4096, 11008, 32)),
        (0.125, 0.25, 1.0)),
    "moe": Workload(
        "moe", "MoE-style stack: 16 layers x 64 experts of 2048x1408 and 1408x2048, "
        "plus 4x 2048x2048 attention per layer; 30% of experts with zero gradients",
        (Group("expert 2048x1408", 2048, 1408, 1024, zero_frac=0.3, zero_block=64),
         Group("expert 1408x2048", 1408, 2048, 1024, zero_frac=0.3, zero_block=64),
         Group("attn 2048x2048", 2048, 2048, 64)),
        (0.25,)),
}


def seed_for(*parts) -> int:
    """Stable 63-bit seed from a tuple of names and numbers."""
    return zlib.crc32(repr(parts).encode()) * 2654435761 % (2 ** 63 - 1)


def _gen(device, *parts):
    g = torch.Generator(device=device)
    g.manual_seed(seed_for(*parts))
    return g


def _storage(w_dtype):
    return torch.bfloat16 if w_dtype == "bf16" else torch.float32


def make_group(wl: Workload, gi: int, device="cuda", seed: int = 0, m0_zero: bool = False,
               first: int = 0, count: int | None = None):
    """W, M, G stacks [n, rows, cols] for group `gi` of workload `wl`.

    `first`/`count` select a sub-range of the group's matrices; every matrix
    is drawn from its own seed, so a sub-range equals the same slice of the
    full stack.
    """
    grp = wl.groups[gi]
    n = grp.count - first if count is None else count
    dt = _storage(wl.w_dtype)
    W = torch.empty((n, grp.rows, grp.cols), dtype=dt, device=device)
    M = torch.empty((n, grp.rows, grp.cols), dtype=torch.float32, device=device)
    G = torch.empty((n, grp.rows, grp.cols), dtype=dt, device=device)
    zero_set = set()
    if grp.zero_frac > 0:
        nz = round(grp.zero_frac * grp.zero_block)
        for blk in range(0, grp.count, grp.zero_block):
            perm = torch.randperm(grp.zero_block, generator=_gen("cpu", wl.name, gi, seed, "zero", blk))
            zero_set.update(int(blk + i) for i in perm[:nz])
    for j in range(n):
        idx = first + j
        g = _gen(device, wl.name, gi, seed, idx)
        W[j] = (0.02 * torch.randn((grp.rows, grp.cols), generator=g, device=device)).to(dt)
        r = torch.exp(torch.randn((grp.rows, 1), generator=g, device=device))
        gm = r * (wl.g_std * torch.randn((grp.rows, grp.cols), generator=g, device=device))
        mm = r * (wl.g_std * torch.randn((grp.rows, grp.cols), generator=g, device=device))
        if grp.spike_frac > 0:
            d_sel = grp.rows if grp.axis == AXIS_ROWS else grp.cols
            ns = int(grp.spike_frac * d_sel)
            lines = torch.randperm(d_sel, generator=_gen("cpu", wl.name, gi, seed, "spike", idx))[:ns]
            lines = lines.to(device)
            if grp.axis == AXIS_ROWS:
                gm[lines, :] *= 20.0
            else:
                gm[:, lines] *= 20.0
        if idx in zero_set:
            gm.zero_()
        G[j] = gm.to(dt)
        M[j] = 0.0 if m0_zero else mm
    return W, M, G


def zero_gradient_matrices(wl: Workload, gi: int, seed: int = 0):
    """Indices of the matrices of group `gi` whose gradient is zero."""
    grp = wl.groups[gi]
    out = set()
    if grp.zero_frac > 0:
        nz = round(grp.zero_frac * grp.zero_block)
        for blk in range(0, grp.count, grp.zero_block):
            perm = torch.randperm(grp.zero_block, generator=_gen("cpu", wl.name, gi, seed, "zero", blk))
            out.update(int(blk + i) for i in perm[:nz])
    return sorted(out)
