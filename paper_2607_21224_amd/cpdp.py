"""Python binding of the CPDP C ABI (include/cpdp.h).

Argument marshalling only: every step of the path runs in the gfx950 kernels
of ``libcpdp.so``.  The functions carry the C names and argument order.
Pointer arguments accept a ``torch.Tensor`` (its ``data_ptr()``) or a plain
integer address; ``stream`` accepts ``None`` (the null stream), a
``torch.cuda.Stream`` or a raw ``hipStream_t`` integer.  A non-zero status is
raised as :class:`CpdpError` unless ``check=False``.

There is no fallback: if the library is not built, importing this module
raises ImportError.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcpdp.so")

CPDP_F32 = 0
CPDP_BF16 = 1

CPDP_OK = 0
CPDP_ERR_INVALID_ARG = 1
CPDP_ERR_NULL = 2
CPDP_ERR_MISALIGNED = 3
CPDP_ERR_OVERLAP = 4
CPDP_ERR_DTYPE = 5
CPDP_ERR_HIP = 6
CPDP_ERR_TOO_LARGE = 7
CPDP_PLAN_STATIC_BYTES = 262144

DTYPES = {"f32": CPDP_F32, "bf16": CPDP_BF16}

# every symbol declared in include/cpdp.h
EXPORTS = ("cpdp_state_init", "cpdp_local_step", "cpdp_reconcile",
           "cpdp_localsgd_sync", "cpdp_ddp_step", "cpdp_state_init_opt",
           "cpdp_local_step_opt", "cpdp_sync_step_opt", "cpdp_is_sync_step",
           "cpdp_period_for_epoch", "cpdp_lr_at", "cpdp_linear_scaled_lr",
           "cpdp_plan_bytes", "cpdp_plan_build", "cpdp_plan_build_static",
           "cpdp_state_init_plan", "cpdp_local_step_plan", "cpdp_sync_step_plan",
           "cpdp_step_table_bytes", "cpdp_step_table_fill", "cpdp_step_table_set_position",
           "cpdp_step_table_advance", "cpdp_step_table_position", "cpdp_local_step_table",
           "cpdp_sync_step_table", "cpdp_local_step_plan_table", "cpdp_sync_step_plan_table",
           "cpdp_count_unsynced", "cpdp_status_str")

CPDP_OPT_SGD = 0
CPDP_OPT_ADAMW = 1
CPDP_SYNC_CPDP = 0
CPDP_SYNC_LOCALSGD = 1
CPDP_SYNC_DDP = 2
SYNC_KINDS = {"cpdp": CPDP_SYNC_CPDP, "localsgd": CPDP_SYNC_LOCALSGD,
              "ddp": CPDP_SYNC_DDP}
CPDP_SYNC_WRITE_GRAD_MEAN = 1
CPDP_SYNC_AVERAGE_OPT_STATE = 2


class cpdp_plan(ctypes.Structure):
    """Mirror of the C struct cpdp_plan (include/cpdp.h)."""
    _fields_ = [("table", ctypes.c_void_p), ("W", ctypes.c_int), ("n_tensors", ctypes.c_int),
                ("param_dt", ctypes.c_int), ("has_mom2", ctypes.c_int),
                ("has_slow_mom", ctypes.c_int), ("has_anchor", ctypes.c_int),
                ("total_chunks", ctypes.c_int64), ("total_numel", ctypes.c_int64),
                ("seal", ctypes.c_uint64)]


class cpdp_step_table(ctypes.Structure):
    """Mirror of the C struct cpdp_step_table (include/cpdp.h)."""
    _fields_ = [("table", ctypes.c_void_p), ("n_steps", ctypes.c_int), ("update", ctypes.c_int),
                ("seal", ctypes.c_uint64)]


class cpdp_optimizer(ctypes.Structure):
    """Mirror of the C struct cpdp_optimizer (include/cpdp.h)."""
    _fields_ = [("kind", ctypes.c_int), ("lr", ctypes.c_float),
                ("momentum", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("step", ctypes.c_int64)]


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load a build of the C ABI and declare its signatures.  The module-level
    ``lib`` is the default build; tests load differently configured builds of
    the same sources (e.g. another block size) through this too."""
    # PyTorch ships its own HIP runtime.  Import it first so that libcpdp.so's
    # libamdhip64.so.7 dependency resolves to that already-loaded runtime: the
    # device memory and stream handles torch hands us belong to it, and a
    # second runtime instance in the process would not see the device.
    import torch  # noqa: F401
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is not built; run `python -m paper_2607_21224_amd.build` "
            "(the CPDP path has no CPU fallback)")
    lib = ctypes.CDLL(path)
    vp, i, i64, f = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
    lib.cpdp_state_init.argtypes = [vp, vp, vp, vp, vp, i, i64, i64, i, i, i, vp]
    lib.cpdp_local_step.argtypes = [vp, vp, vp, i, i64, i64, i, f, f, i, i, i, vp]
    lib.cpdp_reconcile.argtypes = [vp, vp, vp, vp, vp, i, i64, i64, i, f, f, f, f,
                                   i, i, i, vp]
    lib.cpdp_localsgd_sync.argtypes = [vp, vp, vp, vp, i, i64, i64, i, f, f, i, i, i, vp]
    lib.cpdp_ddp_step.argtypes = [vp, vp, vp, i, i64, i64, f, f, i, i, i, vp]
    op = ctypes.POINTER(cpdp_optimizer)
    lib.cpdp_state_init_opt.argtypes = [vp, vp, vp, vp, vp, vp, i, i64, i64, i, i, vp]
    lib.cpdp_local_step_opt.argtypes = [vp, vp, vp, vp, i, i64, i64, i, op, i, vp]
    lib.cpdp_sync_step_opt.argtypes = [i, vp, vp, vp, vp, vp, vp, i, i64, i64, i, op,
                                       f, f, ctypes.c_uint, i, vp]
    pp = ctypes.POINTER(cpdp_plan)
    lib.cpdp_plan_bytes.argtypes = [i, i]
    lib.cpdp_plan_bytes.restype = i64
    lib.cpdp_plan_build.argtypes = [pp, i64, i, i, ctypes.POINTER(i64), ctypes.POINTER(vp),
                                    ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                    ctypes.POINTER(vp), ctypes.POINTER(vp), i]
    lib.cpdp_plan_build.restype = i
    lib.cpdp_plan_build_static.argtypes = [pp, i, i, ctypes.POINTER(i64), ctypes.POINTER(vp),
                                           ctypes.POINTER(vp), ctypes.POINTER(vp),
                                           ctypes.POINTER(vp), ctypes.POINTER(vp),
                                           ctypes.POINTER(vp), i]
    lib.cpdp_plan_build_static.restype = i
    lib.cpdp_state_init_plan.argtypes = [pp, vp]
    lib.cpdp_state_init_plan.restype = i
    lib.cpdp_local_step_plan.argtypes = [pp, i, op, vp]
    lib.cpdp_local_step_plan.restype = i
    lib.cpdp_sync_step_plan.argtypes = [i, pp, i, op, f, f, ctypes.c_uint, vp]
    lib.cpdp_sync_step_plan.restype = i
    tp = ctypes.POINTER(cpdp_step_table)
    lib.cpdp_step_table_bytes.argtypes = [i]
    lib.cpdp_step_table_bytes.restype = i64
    lib.cpdp_step_table_fill.argtypes = [tp, i64, i, op, ctypes.POINTER(f), ctypes.POINTER(f)]
    lib.cpdp_step_table_set_position.argtypes = [tp, i64, vp]
    lib.cpdp_step_table_advance.argtypes = [tp, vp]
    lib.cpdp_step_table_position.argtypes = [tp, ctypes.POINTER(i64)]
    lib.cpdp_local_step_table.argtypes = [vp, vp, vp, vp, i, i64, i64, i, tp, i, vp]
    lib.cpdp_sync_step_table.argtypes = [i, vp, vp, vp, vp, vp, vp, i, i64, i64, i, tp,
                                         ctypes.c_uint, i, vp]
    for name in ("cpdp_step_table_fill", "cpdp_step_table_set_position",
                 "cpdp_step_table_advance", "cpdp_step_table_position",
                 "cpdp_local_step_table", "cpdp_sync_step_table"):
        getattr(lib, name).restype = i
    lib.cpdp_local_step_plan_table.argtypes = [pp, i, tp, vp]
    lib.cpdp_local_step_plan_table.restype = i
    lib.cpdp_sync_step_plan_table.argtypes = [i, pp, i, tp, ctypes.c_uint, vp]
    lib.cpdp_sync_step_plan_table.restype = i
    lib.cpdp_count_unsynced.argtypes = [vp, vp, i, i64, i64, i, vp, vp]
    lib.cpdp_count_unsynced.restype = i
    lib.cpdp_is_sync_step.argtypes = [i64, i, i64]
    lib.cpdp_period_for_epoch.argtypes = [i64, i64, i]
    lib.cpdp_period_for_epoch.restype = i
    lib.cpdp_lr_at.argtypes = [i64, i64, i64, f, f]
    lib.cpdp_lr_at.restype = f
    lib.cpdp_linear_scaled_lr.argtypes = [f, i64, i64]
    lib.cpdp_linear_scaled_lr.restype = f
    lib.cpdp_status_str.argtypes = [i]
    lib.cpdp_status_str.restype = ctypes.c_char_p
    for name in ("cpdp_state_init", "cpdp_local_step", "cpdp_reconcile",
                 "cpdp_localsgd_sync", "cpdp_ddp_step", "cpdp_state_init_opt",
                 "cpdp_local_step_opt", "cpdp_sync_step_opt", "cpdp_is_sync_step"):
        getattr(lib, name).restype = ctypes.c_int
    return lib


lib = load_library()


class CpdpError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {cpdp_status_str(status)}")


def _addr(x) -> int | None:
    """Device address of a buffer argument: None, an integer address, or a
    tensor.  A tensor must live on the GPU (a host tensor's address would be
    dereferenced by a kernel) and be contiguous (the ABI's layouts are dense
    rows of stride ld)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError(f"CPDP buffers must be device tensors, got one on {x.device}")
    if not x.is_contiguous():
        raise ValueError("CPDP buffers must be contiguous tensors")
    return int(x.data_ptr())


def _torch_dtypes():
    import torch
    return {CPDP_F32: torch.float32, CPDP_BF16: torch.bfloat16}


_TORCH_DTYPE = _torch_dtypes()


def _span(x, n_elems: int, dt, name: str):
    """Address of a buffer argument the call touches for n_elems elements of
    storage type dt.  A tensor must have that storage type, live on the GPU
    (a host tensor's address would be dereferenced by a kernel), be
    contiguous (the ABI's layouts are dense rows of stride ld) and hold at
    least those bytes: the ABI takes raw addresses and cannot see a buffer's
    size, so a short tensor would send the kernel past its end.  (An unknown
    storage-type code is left to the library, which rejects it before any
    launch.)"""
    if x is None or isinstance(x, int):
        return x
    code = DTYPES[dt] if isinstance(dt, str) else int(dt)
    want = _TORCH_DTYPE.get(code)
    if want is not None and x.dtype is not want:
        raise ValueError(f"{name}: storage type {want} expected, the tensor is {x.dtype}")
    if n_elems > 0:
        need = n_elems * (2 if code == CPDP_BF16 else 4)
        have = x.numel() * x.element_size()
        if have < need:
            raise ValueError(f"{name}: the call touches {need} bytes, the tensor holds {have}")
    if not x.is_cuda:
        raise ValueError(f"CPDP buffers must be device tensors, got one on {x.device}")
    if not x.is_contiguous():
        raise ValueError("CPDP buffers must be contiguous tensors")
    return x.data_ptr()


def _rows(x, W, P, ld, dt, name: str):
    """A W-row family (row stride ld, P coordinates per row)."""
    W, P, ld = int(W), int(P), int(ld)
    n = (W - 1) * ld + P if W >= 1 and P > 0 and ld >= P else 0
    return _span(x, n, dt, name)


def _vec(x, P, name: str, dt=CPDP_F32):
    return _span(x, int(P) if int(P) > 0 else 0, dt, name)


def _stream(s) -> int | None:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _dt(x) -> int:
    return DTYPES[x] if isinstance(x, str) else int(x)


def _done(status: int, where: str, check: bool) -> int:
    if check and status != CPDP_OK:
        raise CpdpError(status, where)
    return status


def cpdp_status_str(status: int) -> str:
    return lib.cpdp_status_str(int(status)).decode()


def cpdp_is_sync_step(t: int, K: int, T: int = 0) -> bool:
    r = lib.cpdp_is_sync_step(int(t), int(K), int(T))
    if r < 0:
        raise CpdpError(-r, "cpdp_is_sync_step")
    return bool(r)


def cpdp_state_init(theta0, params, mom, slow_mom, anchor, W, P, ld, K,
                    param_dt=CPDP_F32, mom_dt=CPDP_F32, stream=None, check=True):
    s = lib.cpdp_state_init(_vec(theta0, P, "theta0", param_dt),
                            _rows(params, W, P, ld, param_dt, "params"),
                            _rows(mom, W, P, ld, mom_dt, "mom"),
                            _vec(slow_mom, P, "slow_mom"), _vec(anchor, P, "anchor"), int(W), int(P),
                            int(ld), int(K), _dt(param_dt), _dt(mom_dt),
                            _stream(stream))
    return _done(s, "cpdp_state_init", check)


def cpdp_local_step(params, mom, grads, W, P, ld, K, lr, mu,
                    param_dt=CPDP_F32, grad_dt=CPDP_F32, mom_dt=CPDP_F32,
                    stream=None, check=True):
    s = lib.cpdp_local_step(_rows(params, W, P, ld, param_dt, "params"),
                            _rows(mom, W, P, ld, mom_dt, "mom"),
                            _rows(grads, W, P, ld, grad_dt, "grads"), int(W),
                            int(P), int(ld), int(K), float(lr), float(mu),
                            _dt(param_dt), _dt(grad_dt), _dt(mom_dt),
                            _stream(stream))
    return _done(s, "cpdp_local_step", check)


def cpdp_reconcile(params, mom, grads, slow_mom, anchor, W, P, ld, K, lr, mu,
                   beta, alpha, param_dt=CPDP_F32, grad_dt=CPDP_F32,
                   mom_dt=CPDP_F32, stream=None, check=True):
    s = lib.cpdp_reconcile(_rows(params, W, P, ld, param_dt, "params"),
                           _rows(mom, W, P, ld, mom_dt, "mom"),
                           _rows(grads, W, P, ld, grad_dt, "grads"),
                           _vec(slow_mom, P, "slow_mom"), _vec(anchor, P, "anchor"), int(W), int(P),
                           int(ld), int(K), float(lr), float(mu), float(beta),
                           float(alpha), _dt(param_dt), _dt(grad_dt),
                           _dt(mom_dt), _stream(stream))
    return _done(s, "cpdp_reconcile", check)


def cpdp_localsgd_sync(params, mom, grads, anchor, W, P, ld, K, lr, mu,
                       param_dt=CPDP_F32, grad_dt=CPDP_F32, mom_dt=CPDP_F32,
                       stream=None, check=True):
    s = lib.cpdp_localsgd_sync(_rows(params, W, P, ld, param_dt, "params"),
                               _rows(mom, W, P, ld, mom_dt, "mom"),
                               _rows(grads, W, P, ld, grad_dt, "grads"),
                               _vec(anchor, P, "anchor"), int(W), int(P), int(ld), int(K),
                               float(lr), float(mu), _dt(param_dt), _dt(grad_dt),
                               _dt(mom_dt), _stream(stream))
    return _done(s, "cpdp_localsgd_sync", check)


def cpdp_ddp_step(params, mom, grads, W, P, ld, lr, mu, param_dt=CPDP_F32,
                  grad_dt=CPDP_F32, mom_dt=CPDP_F32, stream=None, check=True):
    s = lib.cpdp_ddp_step(_rows(params, W, P, ld, param_dt, "params"),
                          _rows(mom, W, P, ld, mom_dt, "mom"),
                          _rows(grads, W, P, ld, grad_dt, "grads"), int(W),
                          int(P), int(ld), float(lr), float(mu), _dt(param_dt),
                          _dt(grad_dt), _dt(mom_dt), _stream(stream))
    return _done(s, "cpdp_ddp_step", check)


def _opt(opt):
    return None if opt is None else ctypes.byref(opt)


def cpdp_state_init_opt(theta0, params, mom, mom2, slow_mom, anchor, W, P, ld, K,
                        param_dt=CPDP_F32, stream=None, check=True):
    s = lib.cpdp_state_init_opt(_vec(theta0, P, "theta0", param_dt),
                                _rows(params, W, P, ld, param_dt, "params"),
                                _rows(mom, W, P, ld, CPDP_F32, "mom"),
                                _rows(mom2, W, P, ld, CPDP_F32, "mom2"),
                                _vec(slow_mom, P, "slow_mom"), _vec(anchor, P, "anchor"),
                                int(W), int(P), int(ld),
                                int(K), _dt(param_dt), _stream(stream))
    return _done(s, "cpdp_state_init_opt", check)


def cpdp_local_step_opt(params, mom, mom2, grads, W, P, ld, K, opt, param_dt=CPDP_F32,
                        stream=None, check=True):
    s = lib.cpdp_local_step_opt(_rows(params, W, P, ld, param_dt, "params"),
                                _rows(mom, W, P, ld, CPDP_F32, "mom"),
                                _rows(mom2, W, P, ld, CPDP_F32, "mom2"),
                                _rows(grads, W, P, ld, CPDP_F32, "grads"),
                                int(W), int(P), int(ld), int(K), _opt(opt),
                                _dt(param_dt), _stream(stream))
    return _done(s, "cpdp_local_step_opt", check)


def cpdp_sync_step_opt(strategy, params, mom, mom2, grads, slow_mom, anchor, W, P, ld, K,
                       opt, beta=0.0, alpha=1.0, flags=0, param_dt=CPDP_F32, stream=None,
                       check=True):
    strategy = SYNC_KINDS[strategy] if isinstance(strategy, str) else int(strategy)
    s = lib.cpdp_sync_step_opt(strategy, _rows(params, W, P, ld, param_dt, "params"),
                               _rows(mom, W, P, ld, CPDP_F32, "mom"),
                               _rows(mom2, W, P, ld, CPDP_F32, "mom2"),
                               _rows(grads, W, P, ld, CPDP_F32, "grads"),
                               _vec(slow_mom, P, "slow_mom"), _vec(anchor, P, "anchor"), int(W),
                               int(P), int(ld), int(K), _opt(opt), float(beta),
                               float(alpha), int(flags), _dt(param_dt), _stream(stream))
    return _done(s, "cpdp_sync_step_opt", check)


def cpdp_period_for_epoch(epoch: int, warmup_epochs: int, K: int) -> int:
    r = lib.cpdp_period_for_epoch(int(epoch), int(warmup_epochs), int(K))
    if r < 0:
        raise CpdpError(-r, "cpdp_period_for_epoch")
    return r


def cpdp_lr_at(step: int, total_steps: int, warmup_steps: int, base_lr: float,
               min_lr: float = 0.0) -> float:
    """Learning rate of 0-based ``step``; raises ValueError on invalid input."""
    import math
    r = lib.cpdp_lr_at(int(step), int(total_steps), int(warmup_steps), float(base_lr),
                       float(min_lr))
    if math.isnan(r):
        raise ValueError("cpdp_lr_at: invalid arguments")
    return r


def cpdp_linear_scaled_lr(base_lr: float, base_batch: int, global_batch: int) -> float:
    """base_lr scaled linearly with the global batch; raises ValueError on
    invalid input."""
    import math
    r = lib.cpdp_linear_scaled_lr(float(base_lr), int(base_batch), int(global_batch))
    if math.isnan(r):
        raise ValueError("cpdp_linear_scaled_lr: invalid arguments")
    return r


def cpdp_plan_bytes(W: int, n_tensors: int) -> int:
    return int(lib.cpdp_plan_bytes(int(W), int(n_tensors)))


def _ptr_array(xs):
    if xs is None:
        return None
    arr = (ctypes.c_void_p * len(xs))(*[_addr(x) for x in xs])
    return ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)), arr


def _plan_arrays(W, n_tensors, numel, params, mom, mom2, grads, slow_mom, anchor, param_dt):
    """The host arrays of a plan build, checked against the tensors they
    name.  Returns (numel array, [params, mom, mom2, grads, slow_mom, anchor]
    pointer arrays, the Python objects that must outlive the call)."""
    keep = []
    numel = [int(x) for x in numel]
    if len(numel) != int(n_tensors):
        raise ValueError(f"numel has {len(numel)} entries for {n_tensors} tensors")

    def arr(xs, dt, name, count):
        if xs is None:
            return None
        # the library reads exactly `count` addresses from the array
        if len(xs) != count:
            raise ValueError(f"{name}: {len(xs)} entries, the plan needs {count}")
        # every tensor must hold its model tensor's numel elements (the table
        # records raw addresses; the kernels trust numel)
        for k, x in enumerate(xs):
            _span(x, numel[k % len(numel)], dt, f"{name}[{k}]")
        r = _ptr_array(xs)
        keep.append(r[1])
        return r[0]
    wn = int(W) * len(numel) if int(W) > 0 else 0
    nm = (ctypes.c_int64 * len(numel))(*numel)
    ptrs = [arr(params, param_dt, "params", wn), arr(mom, CPDP_F32, "mom", wn),
            arr(mom2, CPDP_F32, "mom2", wn), arr(grads, CPDP_F32, "grads", wn),
            arr(slow_mom, CPDP_F32, "slow_mom", len(numel)),
            arr(anchor, CPDP_F32, "anchor", len(numel))]
    return nm, ptrs, keep


def cpdp_plan_build(plan: cpdp_plan, plan_bytes, W, n_tensors, numel, params, mom, mom2,
                    grads, slow_mom, anchor, param_dt=CPDP_F32, check=True):
    """numel: n ints; params/mom/grads/mom2: W*n tensors or addresses,
    replica-major ([i*n + t]); slow_mom/anchor: n tensors or None."""
    nm, ptrs, keep = _plan_arrays(W, n_tensors, numel, params, mom, mom2, grads, slow_mom,
                                  anchor, param_dt)
    s = lib.cpdp_plan_build(ctypes.byref(plan), int(plan_bytes), int(W), int(n_tensors), nm,
                            *ptrs, _dt(param_dt))
    del keep
    return _done(s, "cpdp_plan_build", check)


def cpdp_plan_build_static(plan: cpdp_plan, W, n_tensors, numel, params, mom, mom2, grads,
                           slow_mom, anchor, param_dt=CPDP_F32, check=True):
    """cpdp_plan_build into the library's own table on the current device
    (no allocation anywhere); sets plan.table.  Arguments as cpdp_plan_build."""
    nm, ptrs, keep = _plan_arrays(W, n_tensors, numel, params, mom, mom2, grads, slow_mom,
                                  anchor, param_dt)
    s = lib.cpdp_plan_build_static(ctypes.byref(plan), int(W), int(n_tensors), nm, *ptrs,
                                   _dt(param_dt))
    del keep
    return _done(s, "cpdp_plan_build_static", check)


def cpdp_state_init_plan(plan: cpdp_plan, stream=None, check=True):
    return _done(lib.cpdp_state_init_plan(ctypes.byref(plan), _stream(stream)),
                 "cpdp_state_init_plan", check)


def cpdp_local_step_plan(plan: cpdp_plan, K, opt, stream=None, check=True):
    s = lib.cpdp_local_step_plan(ctypes.byref(plan), int(K), _opt(opt), _stream(stream))
    return _done(s, "cpdp_local_step_plan", check)


def cpdp_sync_step_plan(strategy, plan: cpdp_plan, K, opt, beta=0.0, alpha=1.0, flags=0,
                        stream=None, check=True):
    strategy = SYNC_KINDS[strategy] if isinstance(strategy, str) else int(strategy)
    s = lib.cpdp_sync_step_plan(int(strategy), ctypes.byref(plan), int(K), _opt(opt),
                                float(beta), float(alpha), int(flags), _stream(stream))
    return _done(s, "cpdp_sync_step_plan", check)


def cpdp_step_table_bytes(n_steps: int) -> int:
    return int(lib.cpdp_step_table_bytes(int(n_steps)))


def cpdp_step_table_fill(t: cpdp_step_table, table_bytes, opts, betas=None, alphas=None,
                         check=True):
    """opts: a sequence of cpdp_optimizer (one per step); betas / alphas:
    sequences of floats or None."""
    n = len(opts)
    # ctypes would zero-fill a short list: every step needs its own values
    for name, xs in (("betas", betas), ("alphas", alphas)):
        if xs is not None and len(xs) != n:
            raise ValueError(f"{name}: {len(xs)} entries for {n} steps")
    arr = (cpdp_optimizer * n)(*opts)
    fb = (ctypes.c_float * n)(*[float(x) for x in betas]) if betas is not None else None
    fa = (ctypes.c_float * n)(*[float(x) for x in alphas]) if alphas is not None else None
    s = lib.cpdp_step_table_fill(ctypes.byref(t), int(table_bytes), n, arr, fb, fa)
    return _done(s, "cpdp_step_table_fill", check)


def cpdp_step_table_set_position(t: cpdp_step_table, position: int, stream=None, check=True):
    return _done(lib.cpdp_step_table_set_position(ctypes.byref(t), int(position), _stream(stream)),
                 "cpdp_step_table_set_position", check)


def cpdp_step_table_advance(t: cpdp_step_table, stream=None, check=True):
    return _done(lib.cpdp_step_table_advance(ctypes.byref(t), _stream(stream)),
                 "cpdp_step_table_advance", check)


def cpdp_step_table_position(t: cpdp_step_table) -> int:
    pos = ctypes.c_int64(-1)
    _done(lib.cpdp_step_table_position(ctypes.byref(t), ctypes.byref(pos)),
          "cpdp_step_table_position", True)
    return int(pos.value)


def cpdp_local_step_table(params, mom, mom2, grads, W, P, ld, K, t: cpdp_step_table,
                          param_dt=CPDP_F32, stream=None, check=True):
    s = lib.cpdp_local_step_table(_rows(params, W, P, ld, param_dt, "params"),
                                  _rows(mom, W, P, ld, CPDP_F32, "mom"),
                                  _rows(mom2, W, P, ld, CPDP_F32, "mom2"),
                                  _rows(grads, W, P, ld, CPDP_F32, "grads"), int(W),
                                  int(P), int(ld), int(K), ctypes.byref(t), _dt(param_dt),
                                  _stream(stream))
    return _done(s, "cpdp_local_step_table", check)


def cpdp_sync_step_table(strategy, params, mom, mom2, grads, slow_mom, anchor, W, P, ld, K,
                         t: cpdp_step_table, flags=0, param_dt=CPDP_F32, stream=None,
                         check=True):
    strategy = SYNC_KINDS[strategy] if isinstance(strategy, str) else int(strategy)
    s = lib.cpdp_sync_step_table(strategy, _rows(params, W, P, ld, param_dt, "params"),
                                 _rows(mom, W, P, ld, CPDP_F32, "mom"),
                                 _rows(mom2, W, P, ld, CPDP_F32, "mom2"),
                                 _rows(grads, W, P, ld, CPDP_F32, "grads"),
                                 _vec(slow_mom, P, "slow_mom"), _vec(anchor, P, "anchor"),
                                 int(W), int(P),
                                 int(ld), int(K), ctypes.byref(t), int(flags), _dt(param_dt),
                                 _stream(stream))
    return _done(s, "cpdp_sync_step_table", check)


def cpdp_count_unsynced(params, anchor, W, P, ld, count, param_dt=CPDP_F32, stream=None,
                        check=True):
    """Enqueue the count of coordinates where some replica differs from the
    reference model (stored type, bitwise) into ``count`` (a device uint64 /
    int64 tensor of one element)."""
    if hasattr(count, "data_ptr") and count.numel() * count.element_size() < 8:
        raise ValueError("count: the call writes 8 bytes, the tensor holds fewer")
    s = lib.cpdp_count_unsynced(_rows(params, W, P, ld, param_dt, "params"),
                                _vec(anchor, P, "anchor"), int(W), int(P), int(ld),
                                _dt(param_dt), _addr(count), _stream(stream))
    return _done(s, "cpdp_count_unsynced", check)


def cpdp_local_step_plan_table(plan: cpdp_plan, K, t: cpdp_step_table, stream=None, check=True):
    s = lib.cpdp_local_step_plan_table(ctypes.byref(plan), int(K), ctypes.byref(t),
                                       _stream(stream))
    return _done(s, "cpdp_local_step_plan_table", check)


def cpdp_sync_step_plan_table(strategy, plan: cpdp_plan, K, t: cpdp_step_table, flags=0,
                              stream=None, check=True):
    strategy = SYNC_KINDS[strategy] if isinstance(strategy, str) else int(strategy)
    s = lib.cpdp_sync_step_plan_table(int(strategy), ctypes.byref(plan), int(K),
                                      ctypes.byref(t), int(flags), _stream(stream))
    return _done(s, "cpdp_sync_step_plan_table", check)
