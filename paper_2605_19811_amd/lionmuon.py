"""ctypes binding of ``liblionmuon.so`` (the C ABI in ``include/lionmuon.h``).

Argument marshalling only: every step of the optimizer runs in the library's
gfx950 kernels. PyTorch tensors provide device memory and the HIP stream.
There is no fallback: a missing library or a non-GPU tensor raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblionmuon.so")

LM_OK = 0
LM_ERR_INVALID_ARGUMENT = 1
LM_ERR_UNSUPPORTED = 2
LM_ERR_OUT_OF_MEMORY = 3
LM_ERR_WORKSPACE_TOO_SMALL = 4
LM_ERR_HIP = 5

LM_TENSOR_LION_ONLY = 1
LM_TENSOR_ADAMW = 2
LM_NS_BF16 = 0
LM_NS_FP32 = 1
LM_NS_SCALE_NONE = 0
LM_NS_SCALE_RMS02 = 1

PHASES = ("lion", "prep", "norm", "gram", "poly", "apply", "srank")
NOALLOC_SCRATCH_BYTES = 64 << 20     # LIONMUON_NOALLOC_SCRATCH_BYTES

EXPORTED = ("lionmuon_config_default", "lionmuon_step", "lionmuon_step_ex",
            "lionmuon_step_noalloc",
            "lionmuon_step_adaptive",
            "lionmuon_workspace_bytes", "lionmuon_ns", "lionmuon_plan_info",
            "lionmuon_profiling_enable", "lionmuon_profiling_read",
            "lionmuon_profiling_reset", "lionmuon_release",
            "lionmuon_status_string", "lionmuon_last_error", "lionmuon_abi_version")


class lm_shape(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("flags", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


class lm_config(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("ns_steps", ctypes.c_int32),
                ("ns_a", ctypes.c_double), ("ns_b", ctypes.c_double),
                ("ns_c", ctypes.c_double), ("ns_eps", ctypes.c_double),
                ("ns_precision", ctypes.c_int32), ("ns_scale_mode", ctypes.c_int32),
                ("lr_muon", ctypes.c_double), ("lr_lion", ctypes.c_double),
                ("ns_bf16_min_side", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("ns_schedule_steps", ctypes.c_int32), ("reserved2", ctypes.c_int32),
                ("ns_schedule", (ctypes.c_double * 3) * 16),
                ("adam_lr", ctypes.c_double), ("adam_beta1", ctypes.c_double),
                ("adam_beta2", ctypes.c_double), ("adam_eps", ctypes.c_double),
                ("adam_wd", ctypes.c_double),
                ("adaptive_alpha", ctypes.c_double), ("adaptive_power_steps", ctypes.c_int32),
                ("reserved3", ctypes.c_int32), ("adam_step", ctypes.c_int64)]


class lm_plan_info(ctypes.Structure):
    _fields_ = [("n_tensors", ctypes.c_int32), ("n_lion", ctypes.c_int32),
                ("n_adamw", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("n_muon", ctypes.c_int32), ("n_shape_classes", ctypes.c_int32),
                ("lion_elements", ctypes.c_int64), ("adamw_elements", ctypes.c_int64),
                ("muon_elements", ctypes.c_int64),
                ("gram_tiles", ctypes.c_int64), ("poly_tiles", ctypes.c_int64),
                ("apply_tiles", ctypes.c_int64), ("ns_flops", ctypes.c_double),
                ("ns_flops_dense", ctypes.c_double), ("lion_bytes", ctypes.c_double),
                ("workspace_bytes", ctypes.c_size_t), ("srank_bytes", ctypes.c_double)]


class lm_phase_times(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * 7), ("launches", ctypes.c_int64 * 7)]


class LionMuonError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(message)
        self.status = status


_lib = None


def library():
    """Load the built library (``__graft_entry__.build()`` builds it)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise LionMuonError(-1, f"{LIB_PATH} is not built: run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    i32, i64, f64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_size_t
    lib.lionmuon_config_default.argtypes = [P(lm_config)]
    lib.lionmuon_config_default.restype = None
    lib.lionmuon_step.argtypes = [vp, vp, vp, P(lm_shape), i32, i64, i32, f64, f64, f64, f64, vp]
    lib.lionmuon_step.restype = ctypes.c_int
    lib.lionmuon_step_ex.argtypes = [vp, vp, vp, vp, P(lm_shape), i32, i64, i32, f64, f64, f64,
                                     P(lm_config), vp, sz, vp]
    lib.lionmuon_step_ex.restype = ctypes.c_int
    lib.lionmuon_step_noalloc.argtypes = [vp, vp, vp, vp, P(lm_shape), i32, i64, i32, f64, f64,
                                          f64, P(lm_config), vp]
    lib.lionmuon_step_noalloc.restype = ctypes.c_int
    lib.lionmuon_step_adaptive.argtypes = [vp, vp, vp, vp, P(lm_shape), i32, i64, f64, f64, f64,
                                           P(lm_config), vp, sz, vp, vp, vp]
    lib.lionmuon_step_adaptive.restype = ctypes.c_int
    lib.lionmuon_workspace_bytes.argtypes = [P(lm_shape), i32, P(lm_config), P(sz)]
    lib.lionmuon_workspace_bytes.restype = ctypes.c_int
    lib.lionmuon_ns.argtypes = [vp, vp, i64, i64, i32, P(lm_config), vp, sz, vp]
    lib.lionmuon_ns.restype = ctypes.c_int
    lib.lionmuon_plan_info.argtypes = [P(lm_shape), i32, i64, i32, P(lm_config), P(lm_plan_info)]
    lib.lionmuon_plan_info.restype = ctypes.c_int
    lib.lionmuon_profiling_enable.argtypes = [i32]
    lib.lionmuon_profiling_enable.restype = ctypes.c_int
    lib.lionmuon_profiling_read.argtypes = [P(lm_phase_times)]
    lib.lionmuon_profiling_read.restype = ctypes.c_int
    lib.lionmuon_profiling_reset.argtypes = []
    lib.lionmuon_profiling_reset.restype = ctypes.c_int
    lib.lionmuon_release.argtypes = []
    lib.lionmuon_release.restype = None
    lib.lionmuon_status_string.argtypes = [ctypes.c_int]
    lib.lionmuon_status_string.restype = ctypes.c_char_p
    lib.lionmuon_last_error.argtypes = []
    lib.lionmuon_last_error.restype = ctypes.c_char_p
    lib.lionmuon_abi_version.argtypes = []
    lib.lionmuon_abi_version.restype = i32
    _lib = lib
    return lib


def _check(status, what):
    if status != LM_OK:
        lib = library()
        raise LionMuonError(status, f"{what}: {lib.lionmuon_status_string(status).decode()}: "
                                    f"{lib.lionmuon_last_error().decode()}")


def config(ns_steps=5, ns_coeffs=(3.4445, -4.7750, 2.0315), ns_eps=1e-7,
           ns_precision="bf16", ns_scale="none", lr_muon=0.0, lr_lion=0.0,
           ns_bf16_min_side=64, ns_schedule=None, adam_lr=1e-3, adam_betas=(0.8, 0.999),
           adam_eps=1e-8, adam_wd=0.0, adaptive_alpha=0.0, adaptive_power_steps=5,
           adam_step=0) -> lm_config:
    """lm_config with defaults; ``ns_schedule`` is an optional list of
    per-step (a, b, c) triples (its length sets ns_steps); ``adaptive_alpha``
    > 0 selects the stable-rank rule of Appendix G instead of the period;
    ``adam_step`` is the AdamW step count k >= 1 of the call's bias
    corrections (0: k = t + 1)."""
    cfg = lm_config()
    library().lionmuon_config_default(ctypes.byref(cfg))
    cfg.ns_steps = ns_steps
    cfg.ns_a, cfg.ns_b, cfg.ns_c = ns_coeffs
    cfg.ns_eps = ns_eps
    cfg.ns_precision = {"bf16": LM_NS_BF16, "fp32": LM_NS_FP32}[ns_precision]
    cfg.ns_scale_mode = {"none": LM_NS_SCALE_NONE, "rms02": LM_NS_SCALE_RMS02}[ns_scale]
    cfg.lr_muon = lr_muon
    cfg.lr_lion = lr_lion
    cfg.ns_bf16_min_side = ns_bf16_min_side
    cfg.adam_lr = adam_lr
    cfg.adam_beta1, cfg.adam_beta2 = adam_betas
    cfg.adam_eps = adam_eps
    cfg.adam_wd = adam_wd
    cfg.adaptive_alpha = adaptive_alpha
    cfg.adaptive_power_steps = adaptive_power_steps
    cfg.adam_step = int(adam_step)
    if ns_schedule is not None:
        sched = [tuple(float(v) for v in t) for t in ns_schedule]
        if not 1 <= len(sched) <= 16 or any(len(t) != 3 for t in sched):
            raise ValueError("ns_schedule needs 1..16 (a, b, c) triples")
        cfg.ns_steps = len(sched)
        cfg.ns_schedule_steps = len(sched)
        for k, t in enumerate(sched):
            for j in range(3):
                cfg.ns_schedule[k][j] = t[j]
    return cfg


def _flags(flag):
    """Tensor flags from a bool (Lion-only) or an int of LM_TENSOR_* bits."""
    if isinstance(flag, bool):
        return LM_TENSOR_LION_ONLY if flag else 0
    return int(flag)


def shape_of(t, lion_only=False) -> lm_shape:
    """rows x cols of a tensor: 1-D -> (1, n); k-D -> (shape[0], prod(rest)).
    ``lion_only`` is a bool or LM_TENSOR_* flag bits."""
    dims = tuple(t.shape)
    if len(dims) == 0:
        rows, cols = 1, 1
    elif len(dims) == 1:
        rows, cols = 1, dims[0]
    else:
        rows = dims[0]
        cols = 1
        for d in dims[1:]:
            cols *= d
    return lm_shape(rows, cols, _flags(lion_only), 0)


def shapes_array(specs):
    """lm_shape array from (rows, cols, flags) triples (flags: bool Lion-only
    or LM_TENSOR_* bits)."""
    arr = (lm_shape * max(len(specs), 1))()
    for i, (r, c, lo) in enumerate(specs):
        arr[i] = lm_shape(r, c, _flags(lo), 0)
    return arr


def _check_tensor(t, name):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise LionMuonError(LM_ERR_INVALID_ARGUMENT, f"{name} must be a GPU tensor")
    if t.dtype != torch.float32:
        raise LionMuonError(LM_ERR_INVALID_ARGUMENT, f"{name} must be float32")
    if not t.is_contiguous():
        raise LionMuonError(LM_ERR_INVALID_ARGUMENT, f"{name} must be contiguous")


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


class TensorList:
    """Marshalled pointer arrays of one (params, grads, momentum) list.

    ``lion_only``: per-tensor bool or LM_TENSOR_* flags; ``second_moment``:
    per-tensor AdamW second-moment tensors (None where not AdamW)."""

    def __init__(self, params, grads, momentum, lion_only=None, second_moment=None):
        n = len(params)
        if len(grads) != n or len(momentum) != n:
            raise ValueError("params, grads and momentum must have one length")
        lion_only = list(lion_only) if lion_only is not None else [False] * n
        second_moment = list(second_moment) if second_moment is not None else [None] * n
        if len(lion_only) != n:
            raise ValueError(f"lion_only has {len(lion_only)} entries for {n} tensors")
        if len(second_moment) != n:
            raise ValueError(f"second_moment has {len(second_moment)} entries for {n} tensors")
        for i, v in enumerate(second_moment):
            if v is not None:
                _check_tensor(v, f"second_moment[{i}]")
                if v.shape != params[i].shape:
                    raise ValueError(f"second_moment[{i}] has the wrong shape")
        for i in range(n):
            _check_tensor(params[i], f"params[{i}]")
            _check_tensor(grads[i], f"grads[{i}]")
            _check_tensor(momentum[i], f"momentum[{i}]")
            if params[i].shape != grads[i].shape or params[i].shape != momentum[i].shape:
                raise ValueError(f"tensor {i}: params, grads and momentum shapes differ")
        self.n = n
        k = max(n, 1)
        self.p = (ctypes.c_void_p * k)(*[t.data_ptr() for t in params])
        self.g = (ctypes.c_void_p * k)(*[t.data_ptr() for t in grads])
        self.m = (ctypes.c_void_p * k)(*[t.data_ptr() for t in momentum])
        self.v = (ctypes.c_void_p * k)(*[0 if t is None else t.data_ptr() for t in second_moment])
        self.shapes = (lm_shape * k)(*[shape_of(t, lo) for t, lo in zip(params, lion_only)])
        self._keep = (list(params), list(grads), list(momentum), second_moment)

    def set_grads(self, grads):
        if len(grads) != self.n:
            raise ValueError(f"{len(grads)} gradients for {self.n} tensors")
        for i, t in enumerate(grads):
            _check_tensor(t, f"grads[{i}]")
            if t.shape != self._keep[0][i].shape:
                raise ValueError(f"grads[{i}] has the wrong shape")
            self.g[i] = t.data_ptr()
        self._keep = (self._keep[0], list(grads), self._keep[2], self._keep[3])


def lionmuon_step(params, grads, momentum, t, P, beta1, beta2, lr, wd, stream=None,
                  lion_only=None, tensors: TensorList | None = None):
    """One LionMuon step (Algorithm 1) with eta_M = eta_L = lr, bf16 NS."""
    tl = tensors or TensorList(params, grads, momentum, lion_only)
    st = library().lionmuon_step(ctypes.cast(tl.p, ctypes.c_void_p), ctypes.cast(tl.g, ctypes.c_void_p),
                                 ctypes.cast(tl.m, ctypes.c_void_p), tl.shapes, tl.n, int(t), int(P),
                                 beta1, beta2, lr, wd, _stream_handle(stream))
    _check(st, "lionmuon_step")


def lionmuon_step_ex(params, grads, momentum, t, P, beta1, beta2, wd, cfg: lm_config,
                     workspace=None, stream=None, lion_only=None,
                     tensors: TensorList | None = None, second_moment=None):
    """One LionMuon step with an explicit lm_config; ``workspace`` is an
    optional uint8 GPU tensor (caller-owned workspace); ``second_moment``
    lists the AdamW second moments of LM_TENSOR_ADAMW tensors."""
    tl = tensors or TensorList(params, grads, momentum, lion_only, second_moment)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        if not workspace.is_cuda:
            raise LionMuonError(LM_ERR_INVALID_ARGUMENT, "workspace must be a GPU tensor")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    st = library().lionmuon_step_ex(ctypes.cast(tl.p, ctypes.c_void_p), ctypes.cast(tl.g, ctypes.c_void_p),
                                    ctypes.cast(tl.m, ctypes.c_void_p), ctypes.cast(tl.v, ctypes.c_void_p),
                                    tl.shapes, tl.n, int(t),
                                    int(P), beta1, beta2, wd, ctypes.byref(cfg), ws_ptr, ws_bytes,
                                    _stream_handle(stream))
    _check(st, "lionmuon_step_ex")


def lionmuon_step_noalloc(params, grads, momentum, t, P, beta1, beta2, wd, cfg: lm_config,
                          stream=None, lion_only=None, tensors: TensorList | None = None,
                          second_moment=None):
    """lionmuon_step_ex without a workspace, for callers that cannot allocate:
    the library allocates nothing and uses its static device scratch (at most
    NOALLOC_SCRATCH_BYTES per device; larger lists raise)."""
    tl = tensors or TensorList(params, grads, momentum, lion_only, second_moment)
    st = library().lionmuon_step_noalloc(ctypes.cast(tl.p, ctypes.c_void_p),
                                         ctypes.cast(tl.g, ctypes.c_void_p),
                                         ctypes.cast(tl.m, ctypes.c_void_p),
                                         ctypes.cast(tl.v, ctypes.c_void_p), tl.shapes, tl.n, int(t),
                                         int(P), beta1, beta2, wd, ctypes.byref(cfg),
                                         _stream_handle(stream))
    _check(st, "lionmuon_step_noalloc")


def lionmuon_step_adaptive(params, grads, momentum, t, beta1, beta2, wd, cfg: lm_config,
                           workspace=None, stream=None, lion_only=None,
                           tensors: TensorList | None = None, second_moment=None,
                           decisions=None, stable_rank=None):
    """One step of the adaptive variant (Appendix G); ``decisions`` (int32)
    and ``stable_rank`` (float64) are optional GPU tensors of one entry per
    tensor that receive the per-tensor branch and stable-rank estimate."""
    import torch
    tl = tensors or TensorList(params, grads, momentum, lion_only, second_moment)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        if not workspace.is_cuda:
            raise LionMuonError(LM_ERR_INVALID_ARGUMENT, "workspace must be a GPU tensor")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    outs = []
    for name, t_out, dtype in (("decisions", decisions, torch.int32),
                               ("stable_rank", stable_rank, torch.float64)):
        if t_out is None:
            outs.append(None)
            continue
        if not t_out.is_cuda or t_out.dtype != dtype or not t_out.is_contiguous() \
                or t_out.numel() < tl.n:
            raise LionMuonError(LM_ERR_INVALID_ARGUMENT,
                                f"{name} must be a contiguous GPU {dtype} tensor of n_tensors entries")
        outs.append(t_out.data_ptr())
    st = library().lionmuon_step_adaptive(
        ctypes.cast(tl.p, ctypes.c_void_p), ctypes.cast(tl.g, ctypes.c_void_p),
        ctypes.cast(tl.m, ctypes.c_void_p), ctypes.cast(tl.v, ctypes.c_void_p), tl.shapes, tl.n,
        int(t), beta1, beta2, wd, ctypes.byref(cfg), ws_ptr, ws_bytes, outs[0], outs[1],
        _stream_handle(stream))
    _check(st, "lionmuon_step_adaptive")


def lionmuon_ns(X, cfg: lm_config | None = None, out=None, stream=None):
    """O = kappa * NS_K(X) for X of shape (rows, cols) or (batch, rows, cols)."""
    import torch
    _check_tensor(X, "X")
    if X.dim() not in (2, 3):
        raise ValueError("X must be 2-D or 3-D")
    batch = 1 if X.dim() == 2 else X.shape[0]
    rows, cols = X.shape[-2], X.shape[-1]
    if out is None:
        out = torch.empty_like(X)
    _check_tensor(out, "out")
    if out.shape != X.shape or out.device != X.device:
        raise LionMuonError(LM_ERR_INVALID_ARGUMENT,
                            f"out must have X's shape {tuple(X.shape)} and device {X.device}")
    st = library().lionmuon_ns(X.data_ptr(), out.data_ptr(), rows, cols, batch,
                               ctypes.byref(cfg) if cfg is not None else None, None, 0,
                               _stream_handle(stream))
    _check(st, "lionmuon_ns")
    return out


def lionmuon_workspace_bytes(specs, cfg: lm_config | None = None) -> int:
    arr = shapes_array(specs)
    out = ctypes.c_size_t(0)
    st = library().lionmuon_workspace_bytes(arr, len(specs),
                                            ctypes.byref(cfg) if cfg is not None else None,
                                            ctypes.byref(out))
    _check(st, "lionmuon_workspace_bytes")
    return out.value


def lionmuon_plan_info(specs, t, P, cfg: lm_config | None = None) -> dict:
    arr = shapes_array(specs)
    info = lm_plan_info()
    st = library().lionmuon_plan_info(arr, len(specs), int(t), int(P),
                                      ctypes.byref(cfg) if cfg is not None else None,
                                      ctypes.byref(info))
    _check(st, "lionmuon_plan_info")
    return {name: getattr(info, name) for name, _ in lm_plan_info._fields_}


def lionmuon_profiling_enable(enable=True):
    _check(library().lionmuon_profiling_enable(1 if enable else 0), "lionmuon_profiling_enable")


def lionmuon_profiling_reset():
    _check(library().lionmuon_profiling_reset(), "lionmuon_profiling_reset")


def lionmuon_profiling_read() -> dict:
    t = lm_phase_times()
    _check(library().lionmuon_profiling_read(ctypes.byref(t)), "lionmuon_profiling_read")
    return {p: {"ms": t.ms[i], "launches": t.launches[i]} for i, p in enumerate(PHASES)}


def lionmuon_release():
    library().lionmuon_release()


def lionmuon_abi_version() -> int:
    return library().lionmuon_abi_version()
