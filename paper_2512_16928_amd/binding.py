"""Thin Python binding of libdion2.so (the C ABI declared in include/dion2.h).

Argument marshalling only: torch tensors are turned into device pointers and
the current HIP stream, sizes are passed through, and a negative status is
raised as Dion2Error. Every step of the Dion2 update runs in the library's
HIP kernels; there is no fallback of any kind, and calling any entry point
without the built library raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import (POINTER, c_char_p, c_double, c_float, c_int, c_int64, c_size_t,
                    c_void_p)

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdion2.so")

DION2_OK = 0
DION2_ERR_INVALID_ARG = -1
DION2_ERR_UNSUPPORTED = -2
DION2_ERR_WORKSPACE = -3
DION2_ERR_HIP = -4

AXIS_AUTO = -1
AXIS_ROWS = 0
AXIS_COLS = 1

DTYPE_F32 = 0
DTYPE_BF16 = 1
NS_AUTO, NS_DIRECT, NS_GRAM = 0, 1, 2
CHAIN_HILO, CHAIN_F16 = 0, 1
MASTER_BF16, MASTER_FP32 = 0, 1
SELECT_L1, SELECT_RANDOM = 0, 1

MAX_NS_STEPS = 16

# Every function include/dion2.h declares (checked by the ABI tests).
EXPORTED = ("dion2_options_init", "dion2_step", "dion2_step_strided", "dion2_step_batched",
            "dion2_step_ex", "dion2_step_noalloc", "dion2_step_groups", "dion2_workspace_size",
            "dion2_workspace_size_ex", "dion2_plan_info", "dion2_plan_form",
            "dion2_release_workspaces", "dion2_status_string", "dion2_last_error",
            "dion2_version", "dion2_profile_enable", "dion2_profile_read", "dion2_profile_reset")

PHASES = ("momentum", "select", "gather", "ns_gram", "ns_poly", "ns_update", "apply")


class Dion2Error(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class Options(ctypes.Structure):
    """Mirror of struct dion2_options."""
    _fields_ = [
        ("w_dtype", c_int),
        ("g_dtype", c_int),
        ("ns_coeffs", POINTER(c_float)),
        ("ns_eps", c_float),
        ("decay_all", c_int),
        ("workspace", c_void_p),
        ("workspace_bytes", c_size_t),
        ("dbg_sel_idx", c_void_p),
        ("dbg_norms", c_void_p),
        ("dbg_update", c_void_p),
        ("ns_form", c_int),
        ("select_rule", c_int),
        ("rand_seed", ctypes.c_uint64),
        ("rand_step", ctypes.c_uint64),
        ("rand_matrix0", ctypes.c_int64),
        ("group_streams", c_int),
        ("ns_chain", c_int),
        ("ns_master", c_int),
        ("dbg_compact", c_void_p),
        ("dbg_compact_lo", c_void_p),
        ("ns_chain_per_product", c_int),
    ]


_lib = None


class Group(ctypes.Structure):
    """dion2_group: one same-shape stack of a grouped call."""
    _fields_ = [
        ("W", c_void_p),
        ("M", c_void_p),
        ("G", c_void_p),
        ("batch", c_int),
        ("rows", c_int64),
        ("cols", c_int64),
        ("axis", c_int),
    ]


def load(path: str = LIB_PATH):
    """Loads libdion2.so (once) and declares the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2512_16928_amd.build` "
            "(the Dion2 step has no non-HIP implementation)")
    lib = ctypes.CDLL(path)
    i64, vp = c_int64, c_void_p
    step_tail = [c_float, c_float, c_float, c_int, c_int]
    lib.dion2_options_init.argtypes = [POINTER(Options)]
    lib.dion2_options_init.restype = None
    lib.dion2_step.argtypes = [vp, vp, vp, i64, i64, *step_tail, vp]
    lib.dion2_step.restype = c_int
    lib.dion2_step_strided.argtypes = [vp, vp, vp, c_int, i64, i64, *step_tail, vp]
    lib.dion2_step_strided.restype = c_int
    lib.dion2_step_batched.argtypes = [POINTER(vp), POINTER(vp), POINTER(vp), c_int, i64, i64,
                                       *step_tail, vp]
    lib.dion2_step_batched.restype = c_int
    lib.dion2_step_ex.argtypes = [vp, vp, vp, c_int, i64, i64, *step_tail, POINTER(Options), vp]
    lib.dion2_step_ex.restype = c_int
    lib.dion2_step_noalloc.argtypes = [vp, vp, vp, c_int, i64, i64, *step_tail, POINTER(Options), vp]
    lib.dion2_step_noalloc.restype = c_int
    lib.dion2_step_groups.argtypes = [POINTER(Group), c_int, c_float, c_float, c_float, c_int,
                                      POINTER(Options), vp]
    lib.dion2_step_groups.restype = c_int
    lib.dion2_workspace_size.argtypes = [c_int, i64, i64, c_float, c_int]
    lib.dion2_workspace_size.restype = c_size_t
    lib.dion2_workspace_size_ex.argtypes = [c_int, i64, i64, c_float, c_int, c_int, POINTER(Options)]
    lib.dion2_workspace_size_ex.restype = c_size_t
    lib.dion2_plan_info.argtypes = [i64, i64, c_float, c_int, POINTER(c_int64), POINTER(c_int)]
    lib.dion2_plan_info.restype = c_int
    lib.dion2_plan_form.argtypes = [c_int, i64, i64, c_float, c_int, c_int, POINTER(Options),
                                    POINTER(c_int), POINTER(c_int), POINTER(c_int)]
    lib.dion2_plan_form.restype = c_int
    lib.dion2_release_workspaces.argtypes = []
    lib.dion2_release_workspaces.restype = None
    lib.dion2_status_string.argtypes = [c_int]
    lib.dion2_status_string.restype = c_char_p
    lib.dion2_last_error.argtypes = []
    lib.dion2_last_error.restype = c_char_p
    lib.dion2_version.argtypes = []
    lib.dion2_version.restype = c_int
    lib.dion2_profile_enable.argtypes = [c_int]
    lib.dion2_profile_enable.restype = c_int
    lib.dion2_profile_read.argtypes = [POINTER(c_double), POINTER(c_int64), POINTER(c_int64),
                                       POINTER(c_double), POINTER(c_double), c_int]
    lib.dion2_profile_read.restype = c_int
    lib.dion2_profile_reset.argtypes = []
    lib.dion2_profile_reset.restype = None
    _lib = lib
    return lib


def _check(status: int):
    if status != DION2_OK:
        lib = load()
        raise Dion2Error(status, lib.dion2_last_error().decode())


def _stream_ptr(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return c_void_p(stream.cuda_stream)


_DT = {torch.bfloat16: DTYPE_BF16, torch.float32: DTYPE_F32}


def _mats(W, M, G, ndim):
    for name, t in (("W", W), ("M", M), ("G", G)):
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
        if t.device.type != "cuda":
            raise ValueError(f"{name} must be a HIP device tensor, got {t.device}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.dim() != ndim:
            raise ValueError(f"{name} must have {ndim} dimensions, got {tuple(t.shape)}")
    if not (W.shape == M.shape == G.shape):
        raise ValueError(f"W {tuple(W.shape)}, M {tuple(M.shape)}, G {tuple(G.shape)} differ")
    if M.dtype != torch.float32:
        raise ValueError("M (momentum) must be float32")
    if W.dtype not in _DT or G.dtype not in _DT:
        raise ValueError("W and G must be bfloat16 or float32")
    if not (W.device == M.device == G.device):
        raise ValueError("W, M and G must be on one device")


def dion2_step(W, M, G, alpha, mu=0.95, lr=0.02, ns_steps=5, axis=AXIS_AUTO, stream=None):
    """One matrix, bf16 W and G, fp32 M (updated in place)."""
    _mats(W, M, G, 2)
    if W.dtype != torch.bfloat16 or G.dtype != torch.bfloat16:
        raise ValueError("dion2_step takes bf16 W and G; use dion2_step_ex for other dtypes")
    lib = load()
    rows, cols = W.shape
    _check(lib.dion2_step(W.data_ptr(), M.data_ptr(), G.data_ptr(), rows, cols, alpha, mu, lr,
                          ns_steps, axis, _stream_ptr(stream, W.device)))


def dion2_step_strided(W, M, G, alpha, mu=0.95, lr=0.02, ns_steps=5, axis=AXIS_AUTO,
                       stream=None):
    """Stacks [batch, rows, cols]: bf16 W and G, fp32 M."""
    _mats(W, M, G, 3)
    if W.dtype != torch.bfloat16 or G.dtype != torch.bfloat16:
        raise ValueError("dion2_step_strided takes bf16 W and G; use dion2_step_ex otherwise")
    lib = load()
    batch, rows, cols = W.shape
    _check(lib.dion2_step_strided(W.data_ptr(), M.data_ptr(), G.data_ptr(), batch, rows, cols,
                                  alpha, mu, lr, ns_steps, axis, _stream_ptr(stream, W.device)))


def dion2_step_batched(Ws, Ms, Gs, alpha, mu=0.95, lr=0.02, ns_steps=5, axis=AXIS_AUTO,
                       stream=None):
    """Lists of same-shape matrices (bf16 W and G, fp32 M)."""
    if not (len(Ws) == len(Ms) == len(Gs)) or len(Ws) == 0:
        raise ValueError("Ws, Ms, Gs must be non-empty lists of equal length")
    for W, M, G in zip(Ws, Ms, Gs):
        _mats(W, M, G, 2)
        if W.shape != Ws[0].shape:
            raise ValueError("all matrices of a batch must have one shape")
        if W.dtype != torch.bfloat16 or G.dtype != torch.bfloat16:
            raise ValueError("dion2_step_batched takes bf16 W and G")
    lib = load()
    n = len(Ws)
    arr = c_void_p * n
    tw = arr(*[t.data_ptr() for t in Ws])
    tm = arr(*[t.data_ptr() for t in Ms])
    tg = arr(*[t.data_ptr() for t in Gs])
    rows, cols = Ws[0].shape
    _check(lib.dion2_step_batched(tw, tm, tg, n, rows, cols, alpha, mu, lr, ns_steps, axis,
                                  _stream_ptr(stream, Ws[0].device)))


def dion2_step_ex(W, M, G, alpha, mu=0.95, lr=0.02, ns_steps=5, axis=AXIS_AUTO, *,
                  ns_coeffs=None, ns_eps=1e-7, decay_all=False, workspace=None,
                  dbg_sel_idx=None, dbg_norms=None, dbg_update=None, dbg_compact=None,
                  dbg_compact_lo=None, ns_form=NS_AUTO, select_rule=SELECT_L1, rand_seed=0,
                  rand_step=0, rand_matrix0=0, ns_chain=CHAIN_HILO, ns_master=MASTER_BF16,
                  ns_chain_per_product=False, stream=None):
    """Full control. W, M, G are [rows, cols] or [batch, rows, cols]; W and G
    may be bf16 or fp32. Debug outputs are preallocated device tensors:
    dbg_sel_idx int32 [batch, k], dbg_norms float64 [batch, d_sel],
    dbg_update float32 [batch, k, d_oth], dbg_compact and dbg_compact_lo
    bfloat16 [batch, k, d_oth] (X before Newton-Schulz, and with MASTER_FP32
    its lo halves). ns_form is NS_AUTO, NS_DIRECT or
    NS_GRAM (the Newton-Schulz evaluation order); ns_chain CHAIN_HILO or
    CHAIN_F16 (storage of the GRAM form's s x s matrices); ns_master
    MASTER_BF16 or MASTER_FP32 (X rounded once to bf16, or kept as a hi/lo
    pair through every product). ns_chain_per_product gives every s x s
    product its own launch even where s <= 64 (bitwise the same result).
    select_rule SELECT_RANDOM draws the lines from Philox keys of
    (rand_seed, rand_step, rand_matrix0 + b)."""
    if W.dim() == 2:
        W, M, G = W.unsqueeze(0), M.unsqueeze(0), G.unsqueeze(0)
    _mats(W, M, G, 3)
    lib = load()
    opt, coeff_buf = _options(W, G, ns_steps, ns_coeffs, ns_eps, decay_all, ns_form, select_rule,
                              rand_seed, rand_step, rand_matrix0, ns_chain, ns_master,
                              ns_chain_per_product)
    for name, t, dt in (("dbg_sel_idx", dbg_sel_idx, torch.int32),
                        ("dbg_norms", dbg_norms, torch.float64),
                        ("dbg_update", dbg_update, torch.float32),
                        ("dbg_compact", dbg_compact, torch.bfloat16),
                        ("dbg_compact_lo", dbg_compact_lo, torch.bfloat16)):
        if t is not None:
            if t.dtype != dt or not t.is_contiguous() or t.device != W.device:
                raise ValueError(f"{name} must be a contiguous {dt} tensor on {W.device}")
            setattr(opt, name, t.data_ptr())
    if workspace is not None:
        if workspace.device != W.device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on W's device")
        opt.workspace = workspace.data_ptr()
        opt.workspace_bytes = workspace.numel() * workspace.element_size()
    batch, rows, cols = W.shape
    _check(lib.dion2_step_ex(W.data_ptr(), M.data_ptr(), G.data_ptr(), batch, rows, cols, alpha,
                             mu, lr, ns_steps, axis, ctypes.byref(opt),
                             _stream_ptr(stream, W.device)))
    del coeff_buf


NOALLOC_SCRATCH_BYTES = 128 << 20


def dion2_step_noalloc(W, M, G, alpha, mu=0.95, lr=0.02, ns_steps=5, axis=AXIS_AUTO, *,
                       ns_coeffs=None, ns_eps=1e-7, decay_all=False, ns_form=NS_AUTO,
                       select_rule=SELECT_L1, rand_seed=0, rand_step=0, rand_matrix0=0,
                       ns_chain=CHAIN_HILO, ns_master=MASTER_BF16, ns_chain_per_product=False,
                       stream=None):
    """The step of dion2_step_ex without any device allocation: the library's
    fixed scratch array holds the workspace (NOALLOC_SCRATCH_BYTES per GPU).
    Calls that overlap on one GPU race."""
    if W.dim() == 2:
        W, M, G = W.unsqueeze(0), M.unsqueeze(0), G.unsqueeze(0)
    _mats(W, M, G, 3)
    lib = load()
    opt, coeff_buf = _options(W, G, ns_steps, ns_coeffs, ns_eps, decay_all, ns_form, select_rule,
                              rand_seed, rand_step, rand_matrix0, ns_chain, ns_master,
                              ns_chain_per_product)
    batch, rows, cols = W.shape
    _check(lib.dion2_step_noalloc(W.data_ptr(), M.data_ptr(), G.data_ptr(), batch, rows, cols,
                                  alpha, mu, lr, ns_steps, axis, ctypes.byref(opt),
                                  _stream_ptr(stream, W.device)))
    del coeff_buf


def _options(W, G, ns_steps, ns_coeffs, ns_eps, decay_all, ns_form, select_rule, rand_seed,
             rand_step, rand_matrix0, ns_chain=CHAIN_HILO, ns_master=MASTER_BF16,
             ns_chain_per_product=False):
    """Options struct (and the coefficient buffer it points to, kept alive by the caller)."""
    lib = load()
    opt = Options()
    lib.dion2_options_init(ctypes.byref(opt))
    opt.w_dtype = _DT[W.dtype]
    opt.g_dtype = _DT[G.dtype]
    coeff_buf = None
    if ns_coeffs is not None:
        flat = [float(v) for abc in ns_coeffs for v in abc]
        if len(flat) < 3 * ns_steps:
            raise ValueError("ns_coeffs needs one (a, b, c) per Newton-Schulz step")
        coeff_buf = (c_float * len(flat))(*flat)
        opt.ns_coeffs = ctypes.cast(coeff_buf, POINTER(c_float))
    opt.ns_eps = ns_eps
    opt.decay_all = 1 if decay_all else 0
    opt.ns_form = ns_form
    opt.select_rule = select_rule
    opt.rand_seed = rand_seed
    opt.rand_step = rand_step
    opt.rand_matrix0 = rand_matrix0
    opt.ns_chain = ns_chain
    opt.ns_master = ns_master
    opt.ns_chain_per_product = 1 if ns_chain_per_product else 0
    return opt, coeff_buf


def dion2_step_groups(groups, alpha, mu=0.95, lr=0.02, ns_steps=5, *, ns_coeffs=None,
                      ns_eps=1e-7, decay_all=False, ns_form=NS_AUTO, select_rule=SELECT_L1,
                      rand_seed=0, rand_step=0, rand_matrix0=0, group_streams=0,
                      ns_chain=CHAIN_HILO, ns_master=MASTER_BF16, ns_chain_per_product=False,
                      stream=None):
    """Several same-shape stacks in one call: groups is a list of (W, M, G, axis)
    with W, M, G [batch, rows, cols] on one device, W and G of one dtype pair
    across groups. Bitwise the result of dion2_step_ex per group; groups of one
    padded Newton-Schulz size share their chain of s x s products."""
    if not groups:
        raise ValueError("groups must be a non-empty list")
    arr = (Group * len(groups))()
    for i, (W, M, G, axis) in enumerate(groups):
        _mats(W, M, G, 3)
        if W.dtype != groups[0][0].dtype or G.dtype != groups[0][2].dtype:
            raise ValueError("every group must have the same W and G dtypes")
        if W.device != groups[0][0].device:
            raise ValueError("every group must be on one device")
        arr[i] = Group(W.data_ptr(), M.data_ptr(), G.data_ptr(), W.shape[0], W.shape[1],
                       W.shape[2], axis)
    W0, _, G0, _ = groups[0]
    opt, keep = _options(W0, G0, ns_steps, ns_coeffs, ns_eps, decay_all, ns_form, select_rule,
                         rand_seed, rand_step, rand_matrix0, ns_chain, ns_master, ns_chain_per_product)
    opt.group_streams = group_streams
    lib = load()
    _check(lib.dion2_step_groups(arr, len(groups), alpha, mu, lr, ns_steps, ctypes.byref(opt),
                                 _stream_ptr(stream, W0.device)))
    del keep


def dion2_step_groups_raw(group_array, ngroups, alpha, mu, lr, ns_steps, opt, stream):
    """The C call as is (for argument-validation tests): a ctypes Group array or
    None, an Options or None, a stream pointer."""
    lib = load()
    return lib.dion2_step_groups(group_array, ngroups, alpha, mu, lr, ns_steps,
                                 ctypes.byref(opt) if opt is not None else None, stream)


def dion2_workspace_size(batch, rows, cols, alpha, axis=AXIS_AUTO) -> int:
    """Workspace bytes that suffice for these arguments under any options."""
    return int(load().dion2_workspace_size(batch, rows, cols, alpha, axis))


def dion2_workspace_size_ex(batch, rows, cols, alpha, axis=AXIS_AUTO, ns_steps=5, *,
                            w_dtype=torch.bfloat16, g_dtype=torch.bfloat16, ns_form=NS_AUTO,
                            ns_chain=CHAIN_HILO, ns_master=MASTER_BF16, select_rule=SELECT_L1,
                            ns_coeffs=None) -> int:
    """Workspace bytes a dion2_step_ex call with exactly these options needs
    (0 where the call would be rejected)."""
    lib = load()
    opt = Options()
    lib.dion2_options_init(ctypes.byref(opt))
    opt.w_dtype = _DT[w_dtype]
    opt.g_dtype = _DT[g_dtype]
    keep = None
    if ns_coeffs is not None:
        flat = [float(v) for abc in ns_coeffs for v in abc]
        keep = (c_float * len(flat))(*flat)
        opt.ns_coeffs = ctypes.cast(keep, POINTER(c_float))
    opt.ns_form = ns_form
    opt.ns_chain = ns_chain
    opt.ns_master = ns_master
    opt.select_rule = select_rule
    n = int(lib.dion2_workspace_size_ex(batch, rows, cols, alpha, axis, ns_steps, ctypes.byref(opt)))
    del keep
    return n


def dion2_plan_form(batch, rows, cols, alpha, axis=AXIS_AUTO, ns_steps=5, *, ns_form=NS_AUTO,
                    ns_chain=CHAIN_HILO, ns_master=MASTER_BF16, ns_coeffs=None,
                    ns_chain_per_product=False):
    """(form, chain, fused) a dion2_step_ex call with these options would
    take: DIRECT or GRAM, the GRAM chain's storage, and whether it runs as one
    launch. Raises Dion2Error where the call would be rejected."""
    lib = load()
    opt = Options()
    lib.dion2_options_init(ctypes.byref(opt))
    keep = None
    if ns_coeffs is not None:
        flat = [float(v) for abc in ns_coeffs for v in abc]
        keep = (c_float * len(flat))(*flat)
        opt.ns_coeffs = ctypes.cast(keep, POINTER(c_float))
    opt.ns_form = ns_form
    opt.ns_chain = ns_chain
    opt.ns_master = ns_master
    opt.ns_chain_per_product = int(bool(ns_chain_per_product))
    form, chain, fused = c_int(-1), c_int(-1), c_int(-1)
    _check(lib.dion2_plan_form(batch, rows, cols, alpha, axis, ns_steps, ctypes.byref(opt),
                               ctypes.byref(form), ctypes.byref(chain), ctypes.byref(fused)))
    del keep
    return int(form.value), int(chain.value), int(fused.value)


def dion2_plan_info(rows, cols, alpha, axis=AXIS_AUTO):
    """(k, resolved_axis) for one matrix of this shape."""
    k = c_int64(0)
    ax = c_int(0)
    _check(load().dion2_plan_info(rows, cols, alpha, axis, ctypes.byref(k), ctypes.byref(ax)))
    return int(k.value), int(ax.value)


def dion2_release_workspaces():
    load().dion2_release_workspaces()


def dion2_status_string(status: int) -> str:
    return load().dion2_status_string(status).decode()


def dion2_last_error() -> str:
    return load().dion2_last_error().decode()


def dion2_version() -> int:
    return int(load().dion2_version())


def dion2_profile_enable(on: bool) -> bool:
    """Turns the per-phase event timing on or off; returns the previous state."""
    return bool(load().dion2_profile_enable(1 if on else 0))


def dion2_profile_read():
    """{phase: dict(ms, calls, launches, flops, bytes)} accumulated since the
    last reset."""
    n = len(PHASES)
    ms, flops, nbytes = (c_double * n)(), (c_double * n)(), (c_double * n)()
    calls, launches = (c_int64 * n)(), (c_int64 * n)()
    _check(load().dion2_profile_read(ms, calls, launches, flops, nbytes, n))
    return {p: dict(ms=ms[i], calls=calls[i], launches=launches[i], flops=flops[i],
                    bytes=nbytes[i]) for i, p in enumerate(PHASES)}


def dion2_profile_reset():
    load().dion2_profile_reset()
