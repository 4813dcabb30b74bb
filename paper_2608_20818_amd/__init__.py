"""Periodic Row-wise Muon optimizer step on AMD MI355X (gfx950).

Thin ctypes binding of ``libprm.so`` (C ABI in ``include/prm.h``).  The
functions and classes here only marshal arguments: every step of the
optimizer runs in the library's HIP kernels.  PyTorch is used, when given,
only to take device pointers and the current stream.  There is no fallback:
if ``libprm.so`` has not been built, loading it raises ``PRMError``.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "PRMError", "Config", "KernelStats", "Optimizer", "AdamWConfig", "AuxAdamW", "load",
    "config_default", "adamw_config_default",
    "schedule_is_refresh", "plan_workspace_bytes", "step_noalloc", "NOALLOC_SCRATCH_BYTES", "PRM_OK", "PRM_EINVAL", "PRM_EDTYPE", "PRM_EALIGN",
    "PRM_ENOMEM", "PRM_EHIP", "F32", "BF16", "KERNEL_CLASSES",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libprm.so")

PRM_OK, PRM_EINVAL, PRM_EDTYPE, PRM_EALIGN, PRM_ENOMEM, PRM_EHIP = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
SCALE_ONE, SCALE_SQRT_ASPECT, SCALE_RMS_0P2 = 0, 1, 2
NUM_KERNEL_CLASSES = 11
NOALLOC_SCRATCH_BYTES = 256 << 20  # PRM_NOALLOC_SCRATCH_BYTES
KERNEL_CLASSES = ("rw_wide", "rw_generic", "rw_tall_stats", "rw_tall_finalize", "rw_tall_apply",
                  "ns_prologue", "ns_alpha", "ns_gram", "ns_poly", "ns_apply", "ns_sprod")


class PRMError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libprm error {code}: {msg}")
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [
        ("K", ctypes.c_int32), ("beta", ctypes.c_float), ("lr", ctypes.c_float),
        ("wd", ctypes.c_float), ("gamma", ctypes.c_float), ("eps_rownorm", ctypes.c_float),
        ("eps_ns", ctypes.c_float), ("ns_a", ctypes.c_float), ("ns_b", ctypes.c_float),
        ("ns_c", ctypes.c_float), ("nesterov", ctypes.c_int32), ("ema_dampening", ctypes.c_int32),
        ("scale_mode", ctypes.c_int32), ("param_dtype", ctypes.c_int32),
        ("grad_dtype", ctypes.c_int32), ("never_refresh", ctypes.c_int32),
        ("gamma_on_refresh", ctypes.c_int32), ("ns_plain", ctypes.c_int32), ("ns_precise", ctypes.c_int32),
        ("workspace_budget_bytes", ctypes.c_uint64),
    ]


class AdamWConfig(ctypes.Structure):
    _fields_ = [
        ("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float), ("wd", ctypes.c_float), ("param_dtype", ctypes.c_int32),
        ("grad_dtype", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


class KernelStats(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("alg_bytes", ctypes.c_double),
                ("alg_flops", ctypes.c_double), ("exec_flops", ctypes.c_double)]


_lib = None


def load() -> ctypes.CDLL:
    """Load libprm.so (built in-tree by ``build.py``); raise loudly if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise PRMError(PRM_EHIP, f"{LIB_PATH} is not built; run paper_2608_20818_amd/build.py")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i64p = ctypes.POINTER(ctypes.c_int64)
    L.prm_config_default.argtypes = [ctypes.POINTER(Config)]
    L.prm_config_default.restype = None
    L.prm_init.argtypes = [ctypes.POINTER(P), ctypes.c_int32, i64p, i64p, ctypes.POINTER(Config), P]
    L.prm_init.restype = ctypes.c_int
    step_args = [P, ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(P), ctypes.c_int64,
                 ctypes.c_float, ctypes.POINTER(ctypes.c_int32)]
    L.prm_step.argtypes = step_args
    L.prm_step.restype = ctypes.c_int
    L.prm_step_debug.argtypes = step_args + [ctypes.POINTER(P)]
    L.prm_step_debug.restype = ctypes.c_int
    L.prm_is_refresh.argtypes = [P, ctypes.c_int64]
    L.prm_is_refresh.restype = ctypes.c_int
    L.prm_workspace_bytes.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    L.prm_workspace_bytes.restype = ctypes.c_int
    L.prm_schedule_is_refresh.argtypes = [ctypes.c_int64, ctypes.c_int32]
    L.prm_schedule_is_refresh.restype = ctypes.c_int
    L.prm_plan_workspace_bytes.argtypes = [ctypes.c_int32, i64p, i64p, ctypes.POINTER(Config),
                                           ctypes.POINTER(ctypes.c_uint64)]
    L.prm_plan_workspace_bytes.restype = ctypes.c_int
    L.prm_step_noalloc.argtypes = [ctypes.POINTER(Config), ctypes.c_int64, ctypes.c_int64, P, P, P,
                                   ctypes.c_int64, ctypes.c_float, ctypes.POINTER(ctypes.c_int32), P]
    L.prm_step_noalloc.restype = ctypes.c_int
    L.prm_profile_enable.argtypes = [P, ctypes.c_int32]
    L.prm_profile_enable.restype = ctypes.c_int
    L.prm_profile_read.argtypes = [P, ctypes.POINTER(KernelStats), ctypes.c_int32]
    L.prm_profile_read.restype = ctypes.c_int
    L.prm_destroy.argtypes = [P]
    L.prm_destroy.restype = ctypes.c_int
    L.prm_last_error.argtypes = []
    L.prm_last_error.restype = ctypes.c_char_p
    dp = ctypes.POINTER(ctypes.c_double)
    L.prm_peak_mfma.argtypes = [P, ctypes.c_int32, dp, dp]
    L.prm_peak_mfma.restype = ctypes.c_int
    L.prm_peak_hbm.argtypes = [P, ctypes.c_uint64, dp, dp, dp, dp]
    L.prm_peak_hbm.restype = ctypes.c_int
    L.prm_adamw_config_default.argtypes = [ctypes.POINTER(AdamWConfig)]
    L.prm_adamw_config_default.restype = None
    L.prm_adamw_init.argtypes = [ctypes.POINTER(P), ctypes.c_int32, i64p, ctypes.POINTER(AdamWConfig), P]
    L.prm_adamw_init.restype = ctypes.c_int
    L.prm_adamw_step.argtypes = [P, ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(P),
                                 ctypes.POINTER(P), ctypes.c_int64, ctypes.c_float]
    L.prm_adamw_step.restype = ctypes.c_int
    L.prm_adamw_destroy.argtypes = [P]
    L.prm_adamw_destroy.restype = ctypes.c_int
    _lib = L
    return L


def _check(rc: int) -> int:
    if rc < 0:
        raise PRMError(rc, load().prm_last_error().decode())
    return rc


def config_default(**overrides) -> Config:
    cfg = Config()
    load().prm_config_default(ctypes.byref(cfg))
    for k, v in overrides.items():
        if not hasattr(cfg, k):
            raise AttributeError(k)
        setattr(cfg, k, v)
    return cfg


def schedule_is_refresh(step: int, K: int) -> int:
    """rho_t = 1[t mod K = 0] without a context (prm_schedule_is_refresh)."""
    return _check(load().prm_schedule_is_refresh(step, K))


def _shape_arrays(shapes):
    n = len(shapes)
    rows = (ctypes.c_int64 * max(n, 1))(*[int(s[0]) for s in shapes])
    cols = (ctypes.c_int64 * max(n, 1))(*[int(s[1]) for s in shapes])
    return n, rows, cols


def plan_workspace_bytes(shapes, cfg: Config) -> int:
    """Device bytes prm_init would allocate (prm_plan_workspace_bytes)."""
    n, rows, cols = _shape_arrays(shapes)
    out = ctypes.c_uint64()
    _check(load().prm_plan_workspace_bytes(n, rows, cols, ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def _stream_handle(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream().cuda_stream
    if hasattr(stream, "cuda_stream"):  # a torch.cuda.Stream
        stream = stream.cuda_stream
    return ctypes.c_void_p(int(stream) if stream else 0)


def peak_mfma(iters: int = 20000, stream=None) -> dict:
    """Sustained bf16 MFMA rate and shader clock (calibration; see prm.h)."""
    t, g = ctypes.c_double(), ctypes.c_double()
    _check(load().prm_peak_mfma(_stream_handle(stream), int(iters), ctypes.byref(t), ctypes.byref(g)))
    return {"tflops": t.value, "clock_ghz": g.value}


def peak_hbm(nbytes: int = 4 << 30, stream=None) -> dict:
    """HBM read, write, copy and row-wise-traffic rates in GB/s (calibration; see prm.h)."""
    r, w, c, x = ctypes.c_double(), ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(load().prm_peak_hbm(_stream_handle(stream), int(nbytes), ctypes.byref(r), ctypes.byref(w),
                               ctypes.byref(c), ctypes.byref(x)))
    return {"read_gbs": r.value, "write_gbs": w.value, "copy_gbs": c.value, "rowwise_gbs": x.value}


def _ptr(x) -> int:
    return x if isinstance(x, int) else x.data_ptr()


def step_noalloc(cfg: Config, param, grad, momentum, step: int, lr: float = -1.0, stream=None) -> int:
    """One step of one matrix through prm_step_noalloc (no context, no device
    allocation; see prm.h); returns rho_t.  Tensors (or raw device pointers):
    contiguous W in ``cfg.param_dtype``, G in ``cfg.grad_dtype``, fp32 M, all of
    one shape (rows, cols)."""
    if not isinstance(param, int):
        shape = tuple(param.shape)
        for x, dt, what in ((param, _DT[cfg.param_dtype], "param"), (grad, _DT[cfg.grad_dtype], "grad"),
                            (momentum, "float32", "momentum")):
            if not x.is_cuda or tuple(x.shape) != shape or len(shape) != 2 or not x.is_contiguous() \
                    or str(x.dtype) != f"torch.{dt}":
                raise ValueError(f"{what}: need a contiguous 2-D {dt} device tensor of shape {shape}")
        rows, cols = shape
    else:
        raise ValueError("step_noalloc needs tensors (the shape comes from them)")
    rho = ctypes.c_int32(-1)
    _check(load().prm_step_noalloc(ctypes.byref(cfg), rows, cols, _ptr(param), _ptr(grad), _ptr(momentum),
                                   int(step), float(lr), ctypes.byref(rho), _stream_handle(stream)))
    return rho.value


_DT = {F32: "float32", BF16: "bfloat16"}


class Optimizer:
    """One libprm context: a fixed list of matrix shapes and a configuration.

    ``step`` takes lists of device tensors (or raw device pointers): weights in
    ``cfg.param_dtype``, gradients in ``cfg.grad_dtype``, fp32 momenta, each
    contiguous and shaped as given at construction.
    """

    def __init__(self, shapes, cfg: Config | None = None, stream=None):
        self.shapes = [(int(m), int(n)) for m, n in shapes]
        self.cfg = cfg if cfg is not None else config_default()
        h = _stream_handle(stream)
        self.stream = h.value or 0
        n, rows, cols = _shape_arrays(self.shapes)
        ctx = ctypes.c_void_p()
        _check(load().prm_init(ctypes.byref(ctx), n, rows, cols, ctypes.byref(self.cfg), h))
        self._ctx = ctx

    def _check_tensors(self, xs, dtype_name, what):
        if len(xs) != len(self.shapes):
            raise ValueError(f"{what}: expected {len(self.shapes)} entries, got {len(xs)}")
        for i, (x, s) in enumerate(zip(xs, self.shapes)):
            if x is None or isinstance(x, int):
                continue
            if not x.is_cuda:
                raise ValueError(f"{what}[{i}]: need a device tensor, got one on {x.device}")
            if tuple(x.shape) != s or not x.is_contiguous() or str(x.dtype) != f"torch.{dtype_name}":
                raise ValueError(f"{what}[{i}]: need contiguous {dtype_name} {s}, got "
                                 f"{x.dtype} {tuple(x.shape)} contiguous={x.is_contiguous()}")

    def step(self, params, grads, momenta, step: int, lr: float = -1.0, directions=None) -> int:
        """Enqueue optimizer step ``step``; returns rho_t (1 = NS5 refresh).
        ``directions`` (debug): fp32 tensors receiving D, None to skip a matrix."""
        self._check_tensors(params, _DT[self.cfg.param_dtype], "params")
        self._check_tensors(grads, _DT[self.cfg.grad_dtype], "grads")
        self._check_tensors(momenta, "float32", "momenta")
        n = len(self.shapes)
        arr = ctypes.c_void_p * max(n, 1)
        P = arr(*[_ptr(x) for x in params])
        G = arr(*[_ptr(x) for x in grads])
        M = arr(*[_ptr(x) for x in momenta])
        rho = ctypes.c_int32(-1)
        L = load()
        if directions is None:
            _check(L.prm_step(self._ctx, P, G, M, int(step), float(lr), ctypes.byref(rho)))
        else:
            self._check_tensors(directions, "float32", "directions")
            D = arr(*[0 if x is None else _ptr(x) for x in directions])
            _check(L.prm_step_debug(self._ctx, P, G, M, int(step), float(lr), ctypes.byref(rho), D))
        return rho.value

    def is_refresh(self, step: int) -> int:
        """rho_t of this context's schedule (prm_is_refresh)."""
        return _check(load().prm_is_refresh(self._ctx, int(step)))

    def workspace_bytes(self) -> int:
        """Device bytes this context holds (prm_workspace_bytes)."""
        out = ctypes.c_size_t()
        _check(load().prm_workspace_bytes(self._ctx, ctypes.byref(out)))
        return out.value

    def profile_enable(self, on: bool = True):
        _check(load().prm_profile_enable(self._ctx, 1 if on else 0))

    def profile_read(self) -> dict:
        out = (KernelStats * NUM_KERNEL_CLASSES)()
        _check(load().prm_profile_read(self._ctx, out, NUM_KERNEL_CLASSES))
        return {o.name.decode(): {"launches": o.launches, "total_ms": o.total_ms, "alg_bytes": o.alg_bytes,
                                  "alg_flops": o.alg_flops, "exec_flops": o.exec_flops} for o in out}

    def close(self):
        if getattr(self, "_ctx", None) is not None and self._ctx.value:
            _check(load().prm_destroy(self._ctx))
        self._ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def adamw_config_default(**overrides) -> AdamWConfig:
    """The paper's aux-AdamW settings (see prm.h), with keyword overrides."""
    c = AdamWConfig()
    load().prm_adamw_config_default(ctypes.byref(c))
    for k, v in overrides.items():
        setattr(c, k, v)
    return c


class AuxAdamW:
    """One fused-AdamW context over a fixed list of flat tensors (the non-matrix
    parameters).  ``step`` takes lists of device tensors (or raw pointers):
    parameters in ``cfg.param_dtype``, gradients in ``cfg.grad_dtype``, fp32
    first and second moments, each contiguous with the element count given at
    construction."""

    def __init__(self, numels, cfg: AdamWConfig | None = None, stream=None):
        self.numels = [int(n) for n in numels]
        self.cfg = cfg if cfg is not None else adamw_config_default()
        h = _stream_handle(stream)
        self.stream = h.value or 0
        n = len(self.numels)
        arr = (ctypes.c_int64 * max(n, 1))(*self.numels)
        ctx = ctypes.c_void_p()
        _check(load().prm_adamw_init(ctypes.byref(ctx), n, arr, ctypes.byref(self.cfg), h))
        self._ctx = ctx

    def _check_tensors(self, xs, dtype_name, what):
        if len(xs) != len(self.numels):
            raise ValueError(f"{what}: expected {len(self.numels)} entries, got {len(xs)}")
        for i, (x, k) in enumerate(zip(xs, self.numels)):
            if x is None or isinstance(x, int):
                continue
            if not x.is_cuda:
                raise ValueError(f"{what}[{i}]: need a device tensor, got one on {x.device}")
            if x.numel() != k or not x.is_contiguous() or str(x.dtype) != f"torch.{dtype_name}":
                raise ValueError(f"{what}[{i}]: need contiguous {dtype_name} with {k} elements, got "
                                 f"{x.dtype} {x.numel()} contiguous={x.is_contiguous()}")

    def step(self, params, grads, exp_avg, exp_avg_sq, t: int, lr: float = -1.0):
        """Enqueue the t-th AdamW update (t >= 1, this one included)."""
        self._check_tensors(params, _DT[self.cfg.param_dtype], "params")
        self._check_tensors(grads, _DT[self.cfg.grad_dtype], "grads")
        self._check_tensors(exp_avg, "float32", "exp_avg")
        self._check_tensors(exp_avg_sq, "float32", "exp_avg_sq")
        n = len(self.numels)
        arr = ctypes.c_void_p * max(n, 1)

        def ptrs(xs):
            return arr(*[0 if x is None else _ptr(x) for x in xs])
        _check(load().prm_adamw_step(self._ctx, ptrs(params), ptrs(grads), ptrs(exp_avg),
                                     ptrs(exp_avg_sq), int(t), float(lr)))

    def bind(self, params, grads, exp_avg, exp_avg_sq):
        """Validate and keep a fixed set of tensors so that ``step_bound`` costs
        one C call (for loops over persistent tensors)."""
        self._check_tensors(params, _DT[self.cfg.param_dtype], "params")
        self._check_tensors(grads, _DT[self.cfg.grad_dtype], "grads")
        self._check_tensors(exp_avg, "float32", "exp_avg")
        self._check_tensors(exp_avg_sq, "float32", "exp_avg_sq")
        arr = ctypes.c_void_p * max(len(self.numels), 1)

        def ptrs(xs):
            return arr(*[0 if x is None else _ptr(x) for x in xs])
        self._keep = (list(params), list(grads), list(exp_avg), list(exp_avg_sq))
        self._bound = (ptrs(params), ptrs(grads), ptrs(exp_avg), ptrs(exp_avg_sq))

    def step_bound(self, t: int, lr: float = -1.0):
        """``step`` on the tensors given to ``bind``."""
        _check(load().prm_adamw_step(self._ctx, *self._bound, int(t), float(lr)))

    def close(self):
        if getattr(self, "_ctx", None) is not None and self._ctx.value:
            _check(load().prm_adamw_destroy(self._ctx))
        self._ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def __getattr__(name):
    # the torch.optim adapter imports torch; load it on first use
    if name == "PRMOptimizer":
        from .torch_optim import PRMOptimizer
        return PRMOptimizer
    raise AttributeError(f"module {__name__!r} has no attribute {name!r}")
