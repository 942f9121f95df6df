"""CPDP oracle: the plain CPU statement of the reconcile hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s CPU-baseline leg may import this package.  It shares no code
with the HIP library (``paper_2607_21224_amd``) and never imports it.

The arithmetic lives in ``cpdp_oracle.c`` (fp64, explicit rounding points);
this module compiles it with gcc, wraps it with ctypes, and adds the host
cadence of Sec. 3.2 / Sec. 3.1 (synchronisation indicator s_t and the forced
synchronisation at the end of an epoch) and the Algorithm 1 driver loop.

Storage types are named "f32", "bf16" or "f64" ("f64" = no rounding).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cpdp_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

_DT = {"f32": 0, "bf16": 1, "f64": 2}

_D = ctypes.POINTER(ctypes.c_double)


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc (IEEE double, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def load(path: str = _LIB_PATH) -> ctypes.CDLL:
    """Load a compiled oracle (building it first if nothing is built)."""
    if not os.path.exists(path):
        build(out=path)
    lib = ctypes.CDLL(path)
    i, i64, d = ctypes.c_int, ctypes.c_int64, ctypes.c_double
    lib.oracle_round.argtypes = [i, d]
    lib.oracle_round.restype = d
    lib.oracle_state_init.argtypes = [i, i64, i, i, _D, _D, _D, _D, _D]
    lib.oracle_state_init.restype = None
    lib.oracle_local_step.argtypes = [i, i64, i, i, _D, _D, _D, d, d]
    lib.oracle_local_step.restype = None
    lib.oracle_reconcile.argtypes = [i, i64, i, i, i, _D, _D, _D, _D, _D,
                                     d, d, d, d]
    lib.oracle_reconcile.restype = None
    lib.oracle_reconcile_vform.argtypes = [i, i64, i, i, i, _D, _D, _D, _D,
                                           _D, d, d, d]
    lib.oracle_reconcile_vform.restype = None
    lib.oracle_localsgd_sync.argtypes = [i, i64, i, i, i, _D, _D, _D, _D, d, d]
    lib.oracle_localsgd_sync.restype = None
    lib.oracle_ddp_step.argtypes = [i, i64, i, i, i, _D, _D, _D, d, d]
    lib.oracle_ddp_step.restype = None
    _OPTP = ctypes.POINTER(OracleOpt)
    lib.oracle_local_step_opt.argtypes = [i, i64, i, i, i, _D, _D, _D, _D, _OPTP]
    lib.oracle_local_step_opt.restype = None
    lib.oracle_sync_opt.argtypes = [i, i, i64, i, i, i, _D, _D, _D, _D, _D, _D,
                                    _OPTP, d, d, ctypes.c_uint]
    lib.oracle_sync_opt.restype = None
    return lib


class OracleOpt(ctypes.Structure):
    """Optimizer descriptor of the oracle: kind 0 = SGD (momentum mu, coupled
    weight decay wd), kind 1 = AdamW (beta1 = mu, beta2, eps, decoupled wd,
    1-based bias-correction step)."""
    _fields_ = [("kind", ctypes.c_int), ("lr", ctypes.c_double),
                ("mu", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("wd", ctypes.c_double),
                ("step", ctypes.c_int64)]


def sgd(lr, mu=0.0, wd=0.0) -> OracleOpt:
    return OracleOpt(0, float(lr), float(mu), 0.0, 0.0, float(wd), 0)


def adamw(lr, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0, step=1) -> OracleOpt:
    return OracleOpt(1, float(lr), float(beta1), float(beta2), float(eps),
                     float(wd), int(step))


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        _lib = load()
    return _lib


def _ptr(a: np.ndarray):
    assert a.dtype == np.float64 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(_D)


@dataclass
class OracleState:
    """State of Algorithm 1 for W workers over P coordinates (all float64).

    params, mom: (W, P); slow: (P,) holds u (u-form) or v (v-form);
    anchor: (P,) is the reference model theta_ref.
    """
    W: int
    P: int
    params: np.ndarray
    mom: np.ndarray
    slow: np.ndarray
    anchor: np.ndarray
    param_dt: str = "f32"
    mom_dt: str = "f32"
    aux_dt: str = "f32"
    lib: ctypes.CDLL | None = field(default=None, repr=False)

    def copy(self) -> "OracleState":
        return OracleState(self.W, self.P, self.params.copy(), self.mom.copy(),
                           self.slow.copy(), self.anchor.copy(), self.param_dt,
                           self.mom_dt, self.aux_dt, self.lib)

    @property
    def _l(self):
        return self.lib if self.lib is not None else lib()


def round_to(dt: str, x: float, use=None) -> float:
    return (use or lib()).oracle_round(_DT[dt], float(x))


def state_init(theta0, W: int, param_dt="f32", mom_dt="f32", aux_dt="f32",
               use=None) -> OracleState:
    """Algorithm 1 initialisation from theta0 (shape (P,))."""
    theta0 = np.ascontiguousarray(theta0, dtype=np.float64)
    P = theta0.shape[0]
    st = OracleState(W, P, np.empty((W, P)), np.empty((W, P)), np.empty(P),
                     np.empty(P), param_dt, mom_dt, aux_dt, use)
    st._l.oracle_state_init(W, P, _DT[param_dt], _DT[aux_dt], _ptr(theta0),
                            _ptr(st.params), _ptr(st.mom), _ptr(st.slow),
                            _ptr(st.anchor))
    return st


def _grads(st: OracleState, grads) -> np.ndarray:
    g = np.ascontiguousarray(grads, dtype=np.float64)
    assert g.shape == (st.W, st.P), (g.shape, st.W, st.P)
    return g


def local_step(st: OracleState, grads, lr: float, mu: float) -> None:
    """Local update phase (s_t = 0), in place."""
    g = _grads(st, grads)
    st._l.oracle_local_step(st.W, st.P, _DT[st.param_dt], _DT[st.mom_dt],
                            _ptr(st.params), _ptr(st.mom), _ptr(g),
                            float(lr), float(mu))


def reconcile(st: OracleState, grads, lr: float, mu: float, beta: float,
              alpha: float) -> None:
    """Synchronization phase (s_t = 1), u-form SlowMo, in place."""
    g = _grads(st, grads)
    st._l.oracle_reconcile(st.W, st.P, _DT[st.param_dt], _DT[st.mom_dt],
                           _DT[st.aux_dt], _ptr(st.params), _ptr(st.mom),
                           _ptr(g), _ptr(st.slow), _ptr(st.anchor), float(lr),
                           float(mu), float(beta), float(alpha))


def reconcile_vform(st: OracleState, grads, lr: float, mu: float,
                    beta: float) -> None:
    """Synchronization phase in the paper's v variables (st.slow holds v)."""
    g = _grads(st, grads)
    st._l.oracle_reconcile_vform(st.W, st.P, _DT[st.param_dt],
                                 _DT[st.mom_dt], _DT[st.aux_dt],
                                 _ptr(st.params), _ptr(st.mom), _ptr(g),
                                 _ptr(st.slow), _ptr(st.anchor), float(lr),
                                 float(mu), float(beta))


def localsgd_sync(st: OracleState, grads, lr: float, mu: float) -> None:
    """LocalSGD synchronisation step (Sec. 5.3): local optimizer step, then
    parameter averaging; the average is also written to st.anchor."""
    g = _grads(st, grads)
    st._l.oracle_localsgd_sync(st.W, st.P, _DT[st.param_dt], _DT[st.mom_dt],
                               _DT[st.aux_dt], _ptr(st.params), _ptr(st.mom),
                               _ptr(g), _ptr(st.anchor), float(lr), float(mu))


def ddp_step(st: OracleState, grads, lr: float, mu: float) -> None:
    """Synchronous DDP step (Sec. 3.1, Sec. 5.3): gradient mean, then the same
    optimizer step on every worker; no parameter averaging."""
    g = _grads(st, grads)
    st._l.oracle_ddp_step(st.W, st.P, _DT[st.param_dt], _DT[st.mom_dt],
                          _DT[st.aux_dt], _ptr(st.params), _ptr(st.mom), _ptr(g),
                          float(lr), float(mu))


METHODS = ("cpdp", "localsgd", "ddp")
_STRATEGY = {"cpdp": 0, "localsgd": 1, "ddp": 2}


def local_step_opt(st: OracleState, grads, opt: OracleOpt, mom2=None) -> None:
    """Local step with a general optimizer; ``mom2`` ((W, P) float64) holds
    AdamW's second moments and is updated in place."""
    g = _grads(st, grads)
    st._l.oracle_local_step_opt(st.W, st.P, _DT[st.param_dt], _DT[st.mom_dt],
                                _DT[st.aux_dt], _ptr(st.params), _ptr(st.mom),
                                _ptr(mom2) if mom2 is not None else None,
                                _ptr(g), ctypes.byref(opt))


SYNC_WRITE_GBAR = 1       # write the gradient mean back into every gradient row
SYNC_AVERAGE_STATE = 2    # optimizer-state reconciliation


def sync_opt(st: OracleState, method: str, grads, opt: OracleOpt, beta=0.0,
             alpha=1.0, mom2=None, write_anchor=True, flags: int = 0):
    """Synchronisation step of ``method`` with a general optimizer.  Returns
    the gradient array (updated in place when SYNC_WRITE_GBAR is set)."""
    g = np.array(grads, dtype=np.float64, order="C", copy=True)
    assert g.shape == (st.W, st.P)
    st._l.oracle_sync_opt(_STRATEGY[method], st.W, st.P, _DT[st.param_dt],
                          _DT[st.mom_dt], _DT[st.aux_dt], _ptr(st.params),
                          _ptr(st.mom), _ptr(mom2) if mom2 is not None else None,
                          _ptr(g), _ptr(st.slow),
                          _ptr(st.anchor) if write_anchor else None,
                          ctypes.byref(opt), float(beta), float(alpha), int(flags))
    return g


def run_opt(theta0, grad_fn, W: int, K: int, n_steps: int, make_opt, beta=0.0,
            alpha=1.0, T: int = 0, method="cpdp", param_dt="f32", mom_dt="f32",
            aux_dt="f32", callback=None, use=None, flags: int = 0):
    """Algorithm 1 (or a Sec. 5.3 baseline) with a general optimizer.
    make_opt(step) returns the OracleOpt of 1-based global step ``step`` (the
    AdamW step count advances on every step, local or synchronising).
    callback(step, kind, state, mom2) after every step.  Returns (state, mom2)."""
    if method not in METHODS:
        raise ValueError(method)
    st = state_init(theta0, W, param_dt, mom_dt, aux_dt, use)
    mom2 = np.zeros((W, st.P))
    for step in range(1, n_steps + 1):
        t = ((step - 1) % T) + 1 if T > 0 else step
        g = grad_fn(step, W, st.P)
        opt = make_opt(step)
        if method == "ddp" or is_sync_step(t, K, T):
            sync_opt(st, method, g, opt, beta, alpha, mom2, flags=flags)
            kind = "reconcile"
        else:
            local_step_opt(st, g, opt, mom2)
            kind = "local"
        if callback is not None:
            callback(step, kind, st, mom2)
    return st, mom2


def is_sync_step(t: int, K: int, T: int = 0) -> bool:
    """Synchronisation indicator.

    Sec. 3.2: s_t = 1 iff t mod K = 0, with t the 1-based step counter inside
    an epoch.  Sec. 3.1 / Sec. 4.2: when the epoch length T is not a multiple
    of K, its last step is also a synchronisation boundary.  T = 0 means the
    run has no epoch boundary.
    """
    if K < 1 or t < 1 or T < 0 or (T > 0 and t > T):
        raise ValueError("need K >= 1, t >= 1, T >= 0 and t <= T when T > 0")
    return t % K == 0 or (T > 0 and t == T)


def period_for_epoch(epoch: int, warmup_epochs: int, K: int) -> int:
    """Sec. 3.4 / Sec. 4.3 / Sec. 5.3: during the warmup epochs CPDP and
    LocalSGD synchronise every step (K = 1); afterwards the configured K."""
    if epoch < 0 or warmup_epochs < 0 or K < 1:
        raise ValueError("need epoch >= 0, warmup_epochs >= 0, K >= 1")
    return 1 if epoch < warmup_epochs else K


def lr_at(step: int, total_steps: int, warmup_steps: int, base_lr: float,
          min_lr: float = 0.0) -> float:
    """Sec. 4.3 cosine annealing with linear warmup (the curve is a reading):
    base_lr * (step+1)/warmup_steps during warmup, then
    min_lr + (base_lr - min_lr)(1 + cos(pi s/S))/2, s = step - warmup_steps,
    S = max(1, total_steps - warmup_steps).  Returned in double."""
    import math
    if not (0 <= step < total_steps and 0 <= warmup_steps <= total_steps
            and base_lr > 0 and 0 <= min_lr <= base_lr):
        raise ValueError("invalid schedule arguments")
    if step < warmup_steps:
        return base_lr * (step + 1) / warmup_steps
    S = max(1, total_steps - warmup_steps)
    return min_lr + (base_lr - min_lr) * (1 + math.cos(math.pi * (step - warmup_steps) / S)) / 2


def linear_scaled_lr(base_lr: float, base_batch: int, global_batch: int) -> float:
    """Sec. 4.3 / Sec. 5.3 linear scaling rule: the learning rate grows in
    proportion to the global batch, base_lr at base_batch.  Returned in double."""
    if not (base_lr > 0 and base_batch >= 1 and global_batch >= 1):
        raise ValueError("invalid scaling arguments")
    return base_lr * global_batch / base_batch


def run(theta0, grad_fn, W: int, K: int, n_steps: int, lr, mu: float,
        beta: float, alpha: float, T: int = 0, param_dt="f32", mom_dt="f32",
        aux_dt="f32", callback=None, use=None, method: str = "cpdp") -> OracleState:
    """Algorithm 1 driven for n_steps steps.

    grad_fn(step, W, P) returns the (W, P) gradients of 1-based global step
    ``step`` (the stand-in for the backward pass).  With T > 0 the within-epoch
    step counter restarts every T steps.  callback(step, kind, state) is called
    after every step with kind "local" or "reconcile".  ``lr`` is a number or
    a function of the 1-based step; ``K`` likewise may be a function of the
    0-based epoch (the warmup schedule).  ``method`` selects the
    synchronisation step: "cpdp" (Algorithm 1), "localsgd" (parameter
    averaging only) or "ddp" (gradient averaging at every step; K is ignored,
    DDP being the K = 1 schedule).
    """
    if method not in METHODS:
        raise ValueError(method)
    st = state_init(theta0, W, param_dt, mom_dt, aux_dt, use)
    for step in range(1, n_steps + 1):
        t = ((step - 1) % T) + 1 if T > 0 else step
        epoch = (step - 1) // T if T > 0 else 0
        k = K(epoch) if callable(K) else K
        lr_s = lr(step) if callable(lr) else lr
        g = grad_fn(step, W, st.P)
        if method == "ddp":
            ddp_step(st, g, lr_s, mu)
            kind = "reconcile"
        elif is_sync_step(t, k, T):
            if method == "cpdp":
                reconcile(st, g, lr_s, mu, beta, alpha)
            else:
                localsgd_sync(st, g, lr_s, mu)
            kind = "reconcile"
        else:
            local_step(st, g, lr_s, mu)
            kind = "local"
        if callback is not None:
            callback(step, kind, st)
    return st
