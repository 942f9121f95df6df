"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and rejects invalid arguments on the host before any GPU work.
Only argument combinations that fail validation are passed here, so no call
reaches HIP; the pointers are fake aligned addresses that are never read."""
import ctypes
import math
import re

import pytest

import oracle
from paper_2607_21224_amd import cpdp
from paper_2607_21224_amd.build import ROOT

HEADER = f"{ROOT}/include/cpdp.h"


def _gpu_visible() -> bool:
    import torch
    return torch.cuda.device_count() > 0


# These tests hand the library fake device addresses.  Every call is meant to
# fail validation, but if one ever passed it would launch a kernel on them:
# harmless without a GPU, a memory fault with one.  So they run only where no
# GPU is visible (the CPU suite).
pytestmark = pytest.mark.skipif(_gpu_visible(), reason="fake device addresses: CPU-only module")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cpdp_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert names == sorted(cpdp.EXPORTS)
    lib = ctypes.CDLL(cpdp.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for s in range(7):
        assert cpdp.cpdp_status_str(s).startswith("CPDP")
    assert "unknown" in cpdp.cpdp_status_str(99)


@pytest.mark.parametrize("K", range(1, 9))
def test_sync_indicator_matches_oracle_and_table2(K):
    for T in [0] + list(range(1, 30)):
        n = T if T else 40
        got = [cpdp.cpdp_is_sync_step(t, K, T) for t in range(1, n + 1)]
        want = [oracle.is_sync_step(t, K, T) for t in range(1, n + 1)]
        assert got == want
        if T:
            assert sum(got) == math.ceil(T / K)  # Table 2


@pytest.mark.parametrize("args", [(0, 2, 0), (1, 0, 0), (5, 2, 4), (1, 1, -1)])
def test_sync_indicator_invalid(args):
    with pytest.raises(cpdp.CpdpError):
        cpdp.cpdp_is_sync_step(*args)


# fake device addresses: 256-byte aligned, far apart, never dereferenced
A = 1 << 40
B = A + (1 << 36)
C = A + 2 * (1 << 36)
U = A + 3 * (1 << 36)
V = A + 4 * (1 << 36)
T0 = A + 5 * (1 << 36)

GOOD = dict(W=4, P=1000, ld=1024, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0)


def rec(**kw):
    a = dict(GOOD, params=A, mom=B, grads=C, slow=U, anchor=V, pdt=0, gdt=0, mdt=0)
    a.update(kw)
    return cpdp.cpdp_reconcile(a["params"], a["mom"], a["grads"], a["slow"],
                               a["anchor"], a["W"], a["P"], a["ld"], a["K"],
                               a["lr"], a["mu"], a["beta"], a["alpha"],
                               a["pdt"], a["gdt"], a["mdt"], None, check=False)


def loc(**kw):
    a = dict(GOOD, params=A, mom=B, grads=C, pdt=0, gdt=0, mdt=0)
    a.update(kw)
    return cpdp.cpdp_local_step(a["params"], a["mom"], a["grads"], a["W"],
                                a["P"], a["ld"], a["K"], a["lr"], a["mu"],
                                a["pdt"], a["gdt"], a["mdt"], None, check=False)


def ini(**kw):
    a = dict(GOOD, theta0=T0, params=A, mom=B, slow=U, anchor=V, pdt=0, mdt=0)
    a.update(kw)
    return cpdp.cpdp_state_init(a["theta0"], a["params"], a["mom"], a["slow"],
                                a["anchor"], a["W"], a["P"], a["ld"], a["K"],
                                a["pdt"], a["mdt"], None, check=False)


E = cpdp
SHAPE_CASES = [dict(W=0), dict(W=-3), dict(P=-1), dict(ld=999), dict(K=0),
               dict(P=(1 << 42), ld=(1 << 42)), dict(P=8, ld=(1 << 58))]


@pytest.mark.parametrize("kw", SHAPE_CASES)
@pytest.mark.parametrize("fn", [rec, loc, ini])
def test_bad_shape(fn, kw):
    assert fn(**kw) == E.CPDP_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [
    dict(lr=0.0), dict(lr=-0.1), dict(lr=float("nan")), dict(lr=float("inf")),
    dict(mu=-0.1), dict(mu=1.0), dict(mu=float("nan"))])
@pytest.mark.parametrize("fn", [rec, loc])
def test_bad_lr_mu(fn, kw):
    assert fn(**kw) == E.CPDP_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [
    dict(beta=1.0), dict(beta=-0.01), dict(beta=float("nan")), dict(alpha=0.0),
    dict(alpha=-1.0), dict(alpha=float("inf")), dict(alpha=float("nan"))])
def test_bad_slowmo(kw):
    assert rec(**kw) == E.CPDP_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(pdt=2), dict(gdt=2), dict(gdt=-1), dict(mdt=2),
                                dict(mdt=-1), dict(pdt=-1)])
def test_bad_dtype(kw):
    assert rec(**kw) == E.CPDP_ERR_DTYPE
    kl = {k: v for k, v in kw.items()}
    assert loc(**kl) == E.CPDP_ERR_DTYPE


def test_bf16_gradients_validated_at_two_bytes():
    """bf16 gradient rows (grad_dt = CPDP_BF16) pass the storage-type check of
    the momentum-SGD entry points and are checked at 2 bytes per element: an
    ld of 1028 elements makes 4112-byte rows in fp32 (16-byte multiples) but
    2056-byte rows in bf16, which the alignment rule rejects.  (Every call here
    fails validation, so none reaches a launch.)"""
    assert rec(gdt=0, ld=1028, slow=C) == E.CPDP_ERR_OVERLAP      # fp32: aligned
    assert rec(gdt=1, ld=1028) == E.CPDP_ERR_MISALIGNED
    assert loc(gdt=1, ld=1028) == E.CPDP_ERR_MISALIGNED
    # a buffer inside the bf16 gradient block still overlaps it
    W, ld = GOOD["W"], GOOD["ld"]
    assert rec(gdt=1, slow=C + 2 * ((W - 1) * ld + GOOD["P"]) - 16) == E.CPDP_ERR_OVERLAP


def test_bad_dtype_init():
    assert ini(pdt=3) == E.CPDP_ERR_DTYPE
    assert ini(mdt=2) == E.CPDP_ERR_DTYPE


@pytest.mark.parametrize("name", ["params", "mom", "grads", "slow", "anchor"])
def test_null(name):
    assert rec(**{name: None}) == E.CPDP_ERR_NULL


def test_null_init_and_local():
    assert ini(theta0=None) == E.CPDP_ERR_NULL
    assert loc(grads=None) == E.CPDP_ERR_NULL


@pytest.mark.parametrize("name", ["params", "mom", "grads", "slow", "anchor"])
def test_misaligned_pointer(name):
    base = dict(params=A, mom=B, grads=C, slow=U, anchor=V)[name]
    assert rec(**{name: base + 4}) == E.CPDP_ERR_MISALIGNED


def test_misaligned_stride():
    assert rec(P=1001, ld=1002) == E.CPDP_ERR_MISALIGNED  # 4008 B rows
    assert loc(P=1001, ld=1002) == E.CPDP_ERR_MISALIGNED
    # bf16 rows need ld % 8 == 0
    assert rec(P=1000, ld=1004, pdt=1) == E.CPDP_ERR_MISALIGNED


def test_overlap():
    row_bytes = 1024 * 4
    # grads starting inside the last used row of params
    assert rec(grads=A + 3 * row_bytes + 16) == E.CPDP_ERR_OVERLAP
    assert rec(anchor=U + 16) == E.CPDP_ERR_OVERLAP
    assert rec(mom=A) == E.CPDP_ERR_OVERLAP
    assert loc(mom=C) == E.CPDP_ERR_OVERLAP
    assert ini(theta0=A + 64) == E.CPDP_ERR_OVERLAP


def test_wrapping_range_rejected():
    """A buffer whose byte range would run past the end of the address space
    is rejected instead of being taken for an empty range (which no overlap
    test would catch)."""
    top = (1 << 64) - 4096          # 16 KB of params rows do not fit below 2^64
    assert rec(params=top) == E.CPDP_ERR_INVALID_ARG
    assert loc(grads=top) == E.CPDP_ERR_INVALID_ARG
    assert ini(theta0=top + 2048) == E.CPDP_ERR_INVALID_ARG   # 4000 B past the end


def test_p_zero_is_noop_without_pointers():
    assert rec(P=0, params=None, mom=None, grads=None, slow=None, anchor=None) == E.CPDP_OK
    assert loc(P=0, params=None, mom=None, grads=None) == E.CPDP_OK
    assert ini(P=0, theta0=None, params=None, mom=None, slow=None, anchor=None) == E.CPDP_OK


def test_binding_raises():
    with pytest.raises(cpdp.CpdpError, match="INVALID_ARG"):
        cpdp.cpdp_reconcile(A, B, C, U, V, 0, 10, 16, 1, 0.1, 0.9, 0.5, 1.0)


def lsgd(**kw):
    a = dict(GOOD, params=A, mom=B, grads=C, anchor=V, pdt=0, gdt=0, mdt=0)
    a.update(kw)
    return cpdp.cpdp_localsgd_sync(a["params"], a["mom"], a["grads"], a["anchor"],
                                   a["W"], a["P"], a["ld"], a["K"], a["lr"], a["mu"],
                                   a["pdt"], a["gdt"], a["mdt"], None, check=False)


def ddp(**kw):
    a = dict(GOOD, params=A, mom=B, grads=C, pdt=0, gdt=0, mdt=0)
    a.update(kw)
    return cpdp.cpdp_ddp_step(a["params"], a["mom"], a["grads"], a["W"], a["P"],
                              a["ld"], a["lr"], a["mu"], a["pdt"], a["gdt"], a["mdt"],
                              None, check=False)


@pytest.mark.parametrize("fn", [lsgd, ddp])
def test_baseline_validation(fn):
    assert fn(W=0) == E.CPDP_ERR_INVALID_ARG
    assert fn(ld=10) == E.CPDP_ERR_INVALID_ARG
    assert fn(lr=0.0) == E.CPDP_ERR_INVALID_ARG
    assert fn(mu=1.0) == E.CPDP_ERR_INVALID_ARG
    assert fn(pdt=7) == E.CPDP_ERR_DTYPE
    assert fn(params=None) == E.CPDP_ERR_NULL
    assert fn(mom=B + 8) == E.CPDP_ERR_MISALIGNED
    assert fn(grads=A) == E.CPDP_ERR_OVERLAP
    assert fn(P=0, params=None, mom=None, grads=None) == E.CPDP_OK


def test_localsgd_anchor_checks():
    assert lsgd(K=0) == E.CPDP_ERR_INVALID_ARG
    assert lsgd(anchor=V + 4) == E.CPDP_ERR_MISALIGNED
    assert lsgd(anchor=A + 64) == E.CPDP_ERR_OVERLAP


def opt_struct(kind=0, lr=0.1, momentum=0.9, beta2=0.999, eps=1e-8, wd=0.0, step=1):
    return cpdp.cpdp_optimizer(kind, lr, momentum, beta2, eps, wd, step)


M2 = A + 6 * (1 << 36)


def lopt(opt=None, **kw):
    a = dict(GOOD, params=A, mom=B, mom2=M2, grads=C, pdt=0)
    a.update(kw)
    return cpdp.cpdp_local_step_opt(a["params"], a["mom"], a["mom2"], a["grads"], a["W"],
                                    a["P"], a["ld"], a["K"], opt, a["pdt"], None, check=False)


def sopt(strategy=0, opt=None, **kw):
    a = dict(GOOD, params=A, mom=B, mom2=M2, grads=C, slow=U, anchor=V, pdt=0)
    a.update(kw)
    return cpdp.cpdp_sync_step_opt(strategy, a["params"], a["mom"], a["mom2"], a["grads"],
                                   a["slow"], a["anchor"], a["W"], a["P"], a["ld"], a["K"],
                                   opt, a["beta"], a["alpha"], a.get("flags", 0), a["pdt"],
                                   None, check=False)


BAD_OPTS = [dict(kind=2), dict(lr=0.0), dict(lr=float("nan")), dict(momentum=1.0),
            dict(wd=-1.0), dict(wd=float("inf")),
            dict(kind=1, beta2=1.0), dict(kind=1, eps=0.0), dict(kind=1, step=0),
            dict(kind=1, lr=1.0, wd=1.0), dict(kind=1, momentum=0.0, beta2=0.0, step=1,
                                               eps=float("nan"))]


@pytest.mark.parametrize("bad", BAD_OPTS)
def test_opt_validation(bad):
    o = opt_struct(**bad)
    assert lopt(o) == E.CPDP_ERR_INVALID_ARG
    assert sopt(0, o) == E.CPDP_ERR_INVALID_ARG


def test_opt_null_and_pointers():
    assert lopt(None) == E.CPDP_ERR_NULL
    assert sopt(0, None) == E.CPDP_ERR_NULL
    adam = opt_struct(kind=1)
    sgd = opt_struct(kind=0, wd=5e-4)
    assert lopt(adam, mom2=None) == E.CPDP_ERR_NULL
    assert sopt(1, adam, mom2=None) == E.CPDP_ERR_NULL
    assert sopt(0, sgd, slow=None) == E.CPDP_ERR_NULL
    assert sopt(0, sgd, anchor=None) == E.CPDP_ERR_NULL
    assert lopt(adam, mom2=B) == E.CPDP_ERR_OVERLAP
    assert lopt(adam, mom2=M2 + 4) == E.CPDP_ERR_MISALIGNED
    assert sopt(7, sgd) == E.CPDP_ERR_INVALID_ARG
    assert sopt(0, sgd, beta=1.0) == E.CPDP_ERR_INVALID_ARG
    assert sopt(0, sgd, pdt=5) == E.CPDP_ERR_DTYPE
    assert sopt(0, sgd, flags=4) == E.CPDP_ERR_INVALID_ARG
    assert sopt(0, sgd, flags=3, P=0) == E.CPDP_OK
    # SGD ignores mom2 and DDP ignores slow/anchor: only validated when used
    assert sopt(2, sgd, P=0) == E.CPDP_OK
    assert lopt(sgd, P=0, mom2=None) == E.CPDP_OK


def test_state_init_opt_validation():
    f = lambda **kw: cpdp.cpdp_state_init_opt(  # noqa: E731
        kw.get("theta0", T0), A, B, kw.get("mom2", M2), U, V, kw.get("W", 4), 1000, 1024, 2,
        kw.get("pdt", 0), None, check=False)
    assert f(W=0) == E.CPDP_ERR_INVALID_ARG
    assert f(pdt=3) == E.CPDP_ERR_DTYPE
    assert f(theta0=None) == E.CPDP_ERR_NULL
    assert f(mom2=A + 256) == E.CPDP_ERR_OVERLAP


def test_period_for_epoch_matches_oracle():
    for K in (1, 2, 4, 7):
        for warm in (0, 1, 3):
            for epoch in range(6):
                assert cpdp.cpdp_period_for_epoch(epoch, warm, K) == \
                    oracle.period_for_epoch(epoch, warm, K)
    for bad in [(-1, 0, 2), (0, -1, 2), (0, 0, 0)]:
        with pytest.raises(cpdp.CpdpError):
            cpdp.cpdp_period_for_epoch(*bad)


def test_lr_at_matches_oracle():
    import numpy as np
    for (total, warm, base, low) in [(100, 10, 0.1, 0.0), (37, 0, 0.4, 0.01), (5, 5, 1e-3, 0.0),
                                     (1, 0, 0.1, 0.1)]:
        for s in range(total):
            got = cpdp.cpdp_lr_at(s, total, warm, base, low)
            want = oracle.lr_at(s, total, warm, float(np.float32(base)), float(np.float32(low)))
            assert got == pytest.approx(want, rel=1e-6, abs=1e-12)
    for bad in [(-1, 10, 0, 0.1, 0.0), (10, 10, 0, 0.1, 0.0), (0, 10, 11, 0.1, 0.0),
                (0, 10, 0, 0.0, 0.0), (0, 10, 0, 0.1, 0.2), (0, 10, 0, 0.1, -1.0)]:
        with pytest.raises(ValueError):
            cpdp.cpdp_lr_at(*bad)


def test_plan_bytes():
    assert cpdp.cpdp_plan_bytes(8, 161) == 8 * (4 + 162 + 161 + 4 * 8 * 161 + 2 * 161)
    assert cpdp.cpdp_plan_bytes(0, 5) == 0


def _plan_args(W=2, n=3, numel=(100, 4, 8), **kw):
    base = A
    step = 1 << 30
    k = [0]

    def nxt():
        k[0] += 1
        return base + k[0] * step
    a = dict(params=[nxt() for _ in range(W * n)], mom=[nxt() for _ in range(W * n)],
             grads=[nxt() for _ in range(W * n)], mom2=None,
             slow=[nxt() for _ in range(n)], anchor=[nxt() for _ in range(n)], pdt=0,
             table=T0, bytes=cpdp.cpdp_plan_bytes(W, n))
    a.update(kw)
    plan = cpdp.cpdp_plan()
    plan.table = a["table"]
    return cpdp.cpdp_plan_build(plan, a["bytes"], W, n, list(numel), a["params"], a["mom"],
                                a["mom2"], a["grads"], a["slow"], a["anchor"], a["pdt"],
                                check=False)


def test_plan_build_validation():
    assert _plan_args(W=0) == E.CPDP_ERR_INVALID_ARG
    assert _plan_args(n=0, numel=()) == E.CPDP_ERR_INVALID_ARG
    assert _plan_args(bytes=64) == E.CPDP_ERR_INVALID_ARG
    assert _plan_args(numel=(100, -1, 8)) == E.CPDP_ERR_INVALID_ARG
    assert _plan_args(pdt=4) == E.CPDP_ERR_DTYPE
    assert _plan_args(table=None) == E.CPDP_ERR_NULL
    assert _plan_args(table=T0 + 4) == E.CPDP_ERR_MISALIGNED
    p = [A + (1 << 30) * (j + 1) for j in range(6)]
    assert _plan_args(params=[p[0] + 8] + p[1:]) == E.CPDP_ERR_MISALIGNED
    assert _plan_args(params=[None] + p[1:]) == E.CPDP_ERR_NULL
    q = list(p)
    q[1] = q[0] + 256          # second tensor starts inside the first (100 floats)
    assert _plan_args(params=q) == E.CPDP_ERR_OVERLAP
    far = A + (1 << 44)
    assert _plan_args(anchor=[A + (1 << 30), far, far + (1 << 30)]) == E.CPDP_ERR_OVERLAP
    # W x chunks blocks must fit one launch: 2 x 2^32 chunks of 256 coordinates
    # do not, and the running sum is checked before it could overflow
    assert _plan_args(n=2, numel=(1 << 40, 1 << 40)) == E.CPDP_ERR_INVALID_ARG
    assert _plan_args(W=1, n=3, numel=(1 << 57, 1 << 57, 1 << 57)) == E.CPDP_ERR_INVALID_ARG
    # a tensor range that wraps past the end of the address space
    top = (1 << 64) - 256
    assert _plan_args(params=[top] + p[1:]) == E.CPDP_ERR_INVALID_ARG


def test_plan_step_validation():
    plan = cpdp.cpdp_plan()
    sgd = opt_struct(kind=0)
    assert cpdp.cpdp_local_step_plan(plan, 2, sgd, check=False) == E.CPDP_ERR_NULL
    plan.table = T0
    plan.W, plan.n_tensors, plan.param_dt = 2, 3, 0
    plan.total_chunks = 3
    assert cpdp.cpdp_local_step_plan(plan, 0, sgd, check=False) == E.CPDP_ERR_INVALID_ARG
    assert cpdp.cpdp_local_step_plan(plan, 2, opt_struct(kind=1), check=False) == E.CPDP_ERR_NULL
    assert cpdp.cpdp_sync_step_plan(0, plan, 2, sgd, check=False) == E.CPDP_ERR_NULL
    assert cpdp.cpdp_sync_step_plan(5, plan, 2, sgd, check=False) == E.CPDP_ERR_INVALID_ARG
    assert cpdp.cpdp_sync_step_plan(2, plan, 2, sgd, flags=8, check=False) == E.CPDP_ERR_INVALID_ARG
    assert cpdp.cpdp_state_init_plan(plan, check=False) == E.CPDP_ERR_NULL
    plan.param_dt = 7
    assert cpdp.cpdp_sync_step_plan(2, plan, 2, sgd, check=False) == E.CPDP_ERR_DTYPE
    # a handle cpdp_plan_build did not seal never reaches a launch
    plan.param_dt = 0
    assert cpdp.cpdp_local_step_plan(plan, 2, sgd, check=False) == E.CPDP_ERR_INVALID_ARG
    assert cpdp.cpdp_sync_step_plan(2, plan, 2, sgd, check=False) == E.CPDP_ERR_INVALID_ARG


def test_binding_rejects_host_and_strided_tensors():
    """The binding never hands a kernel a host address or a strided view: a
    host tensor or a non-contiguous tensor raises before the library is called."""
    import torch
    host = torch.zeros(64)
    with pytest.raises(ValueError, match="device tensors"):
        cpdp.cpdp_local_step(host, host, host, 1, 64, 64, 1, 0.1, 0.9)
    with pytest.raises(ValueError, match="device tensors"):
        cpdp.cpdp_plan_build(cpdp.cpdp_plan(), 1 << 12, 1, 1, [64], [host], [host], None,
                             [host], None, None)


def test_binding_rejects_mistyped_tensors_and_short_lists():
    """A tensor whose dtype is not the declared storage type of its family
    would have its bits misread by the kernels; the binding raises instead.
    A per-step list shorter than the optimizer list would be zero-filled by
    ctypes; the binding raises instead.  Neither call reaches the library."""
    import torch
    f16 = torch.zeros(64, dtype=torch.float16)
    f32 = torch.zeros(64)
    with pytest.raises(ValueError, match="storage type"):
        cpdp.cpdp_local_step(f16, f32, f32, 1, 64, 64, 1, 0.1, 0.9, param_dt="bf16")
    with pytest.raises(ValueError, match="storage type"):
        cpdp.cpdp_reconcile(f32, f32, f32, f32, f32, 1, 64, 64, 1, 0.1, 0.9, 0.5, 1.0,
                            param_dt="bf16")
    with pytest.raises(ValueError, match="storage type"):
        cpdp.cpdp_state_init(f16, f32, f32, f32, f32, 1, 64, 64, 1)
    opts = [opt_struct() for _ in range(3)]
    with pytest.raises(ValueError, match="betas"):
        cpdp.cpdp_step_table_fill(cpdp.cpdp_step_table(), 1 << 12, opts, betas=[0.5, 0.5])
    with pytest.raises(ValueError, match="alphas"):
        cpdp.cpdp_step_table_fill(cpdp.cpdp_step_table(), 1 << 12, opts, alphas=[1.0] * 4)


def test_state_checks_shapes_before_the_library():
    """CpdpState validates buffer shapes, dtypes and devices itself: the ABI
    takes raw addresses and cannot see a too-small gradient buffer."""
    import torch
    from paper_2607_21224_amd.state import CpdpState, Hyper
    st = CpdpState(2, 8, ld=16, K=2, device="cpu")
    h = Hyper.fp32(0.1, 0.9, 0.5, 1.0)
    with pytest.raises(ValueError, match="shape"):
        st.local_step(torch.zeros(2, 8), h)
    with pytest.raises(ValueError, match="float32"):
        st.reconcile(torch.zeros(2, 16, dtype=torch.float64), h)
    with pytest.raises(ValueError, match="elements"):
        st.init(torch.zeros(4))
    with pytest.raises(ValueError, match="device tensors"):  # shapes fine, but host memory
        st.init(torch.zeros(8))
    with pytest.raises(ValueError, match="param_dt"):
        CpdpState(2, 8, ld=16, param_dt="fp16", device="cpu")


def test_rejected_optimizer_step_leaves_the_step_count():
    """A step the library rejects is not counted: AdamW's bias correction
    would otherwise be one step ahead after the caller fixes the call."""
    import torch
    from paper_2607_21224_amd.state import CpdpState, Optimizer
    st = CpdpState(2, 8, ld=16, K=2, device="cpu")
    opt = Optimizer("sgd", lr=0.1, momentum=0.9)
    with pytest.raises(ValueError, match="device tensors"):
        st.step_opt(1, torch.zeros(2, 16), opt)
    assert st.opt_step == 0


def test_linear_scaled_lr_matches_oracle():
    """cpdp_linear_scaled_lr is the oracle's rule rounded to fp32, for the
    Table 4 configurations and other batch ratios; invalid input raises."""
    import numpy as np
    for base_lr, base, glob in [(0.1, 256, 256), (0.1, 256, 384), (0.1, 256, 512),
                                (0.1, 256, 768), (0.1, 256, 1024), (5e-4, 64, 1024),
                                (0.05, 512, 64), (0.1, 3, 7)]:
        got = cpdp.cpdp_linear_scaled_lr(base_lr, base, glob)
        want = float(np.float32(oracle.linear_scaled_lr(float(np.float32(base_lr)), base, glob)))
        assert got == want, (base_lr, base, glob, got, want)
    for bad in [(0.0, 256, 512), (float("nan"), 256, 512), (0.1, 0, 512), (0.1, 256, 0),
                (float("inf"), 1, 1), (-0.1, 1, 1)]:
        with pytest.raises(ValueError):
            cpdp.cpdp_linear_scaled_lr(*bad)


def test_synth_device_wrappers_reject_host_and_small_tensors():
    """The device input generator and copy kernel never receive a host
    address or a size beyond the tensors (checked before the library)."""
    import torch
    from synth import device as sdev
    with pytest.raises(ValueError, match="GPU tensor"):
        sdev.fill_grads(torch.zeros(2, 16), 16, 1, 1)
    with pytest.raises(ValueError, match="GPU tensor"):
        sdev.copy_f32(torch.zeros(4), torch.zeros(4), 4)


def test_checkpoint_restore_rejects_mismatched_buffers():
    """from_state_dict copies only buffers of exactly the layout's shape and
    type: the kernels trust the state's W and ld, so a checkpoint buffer that
    is smaller, broadcastable or of another type must not reach them."""
    import torch
    from paper_2607_21224_amd.state import CpdpState
    st = CpdpState(2, 8, ld=16, K=2, device="cpu")
    for name in ("params", "mom", "slow_mom", "anchor"):
        getattr(st, name).copy_(torch.arange(getattr(st, name).numel(),
                                             dtype=torch.float32).view_as(getattr(st, name)))
    d = {"W": 2, "P": 8, "ld": 16, "K": 2, "param_dt": "f32", "opt_step": 3,
         "params": st.params.clone(), "mom": st.mom.clone(), "slow_mom": st.slow_mom.clone(),
         "anchor": st.anchor.clone(), "mom2": st.mom.clone()}
    back = CpdpState.from_state_dict(d, device="cpu")
    for name in ("params", "mom", "slow_mom", "anchor"):
        assert torch.equal(getattr(back, name), getattr(st, name))
    assert torch.equal(back.mom2, st.mom) and back.opt_step == 3
    bad = [("mom2", torch.zeros(2, 8)), ("mom2", torch.zeros(16)),
           ("mom", torch.zeros(2, 16, dtype=torch.float64)), ("anchor", torch.zeros(1)),
           ("params", [0.0] * 32)]
    for name, value in bad:
        with pytest.raises(ValueError, match=name):
            CpdpState.from_state_dict(dict(d, **{name: value}), device="cpu")


def test_binding_rejects_tensors_smaller_than_the_call_touches():
    """The ABI takes raw addresses, so the binding checks that every tensor
    argument holds the bytes the call will touch ((W-1)*ld + P elements of a
    row family, P of a vector, numel of a plan tensor): a short tensor never
    reaches a kernel.  (Integer addresses stand for the other buffers; they
    pass through unchecked, as in C.)"""
    import torch
    W, P, ld = 3, 100, 128
    a = [A + k * (1 << 30) for k in range(8)]
    full = torch.zeros(W * ld)
    short = torch.zeros(W * P)                      # rows of stride P, not ld
    short_vec = torch.zeros(P - 1)
    with pytest.raises(ValueError, match="grads"):
        cpdp.cpdp_local_step(a[0], a[1], short, W, P, ld, 1, 0.1, 0.9)
    with pytest.raises(ValueError, match="anchor"):
        cpdp.cpdp_reconcile(a[0], a[1], a[2], a[3], short_vec, W, P, ld, 2, 0.1, 0.9, 0.5, 1.0)
    with pytest.raises(ValueError, match="params"):  # bf16 rows: 2 bytes per element
        cpdp.cpdp_local_step(torch.zeros((W - 1) * ld + P - 1, dtype=torch.bfloat16), a[1], a[2],
                             W, P, ld, 1, 0.1, 0.9, param_dt="bf16")
    with pytest.raises(ValueError, match="theta0"):
        cpdp.cpdp_state_init(short_vec, a[1], a[2], a[3], a[4], W, P, ld, 1)
    with pytest.raises(ValueError, match="mom2"):
        cpdp.cpdp_local_step_opt(a[0], a[1], short, a[2], W, P, ld, 1,
                                 cpdp.cpdp_optimizer(1, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1))
    with pytest.raises(ValueError, match="count"):
        cpdp.cpdp_count_unsynced(a[0], a[1], W, P, ld, torch.zeros(1, dtype=torch.int32))
    # a right-sized host tensor gets past the size check and stops at the device check
    with pytest.raises(ValueError, match="device tensors"):
        cpdp.cpdp_local_step(a[0], a[1], full, W, P, ld, 1, 0.1, 0.9)
    # plans: the pointer arrays must have W*n (or n) entries, each tensor numel elements
    t63 = torch.zeros(63)
    with pytest.raises(ValueError, match="numel"):
        cpdp.cpdp_plan_build(cpdp.cpdp_plan(), 1 << 12, 1, 2, [64], a[:2], a[2:4], None,
                             a[4:6], None, None)
    with pytest.raises(ValueError, match="entries"):
        cpdp.cpdp_plan_build(cpdp.cpdp_plan(), 1 << 12, 2, 1, [64], a[:1], a[2:4], None,
                             a[4:6], None, None)
    with pytest.raises(ValueError, match=r"grads\[1\]"):
        cpdp.cpdp_plan_build(cpdp.cpdp_plan(), 1 << 12, 2, 1, [64], a[:2], a[2:4], None,
                             [a[4], t63], None, None)


def test_state_reserves_adamw_rows_when_asked():
    """adamw=True allocates the second-moment rows with the state (same shape
    and type as the momentum rows); by default they wait for init_opt."""
    from paper_2607_21224_amd.state import CpdpState
    st = CpdpState(3, 10, ld=16, K=2, device="cpu", adamw=True)
    assert st.mom2 is not None and st.mom2.shape == st.mom.shape
    assert st.mom2.dtype == st.mom.dtype
    assert CpdpState(3, 10, ld=16, K=2, device="cpu").mom2 is None
