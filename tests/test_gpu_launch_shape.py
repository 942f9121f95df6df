"""Results do not depend on the launch shape: the library built with 256-thread
blocks (a quarter of the blocks, four wavefronts each) gives bitwise the same
state as the default 64-thread build after every step.  The cross-replica sums run in a
fixed order inside one thread, so the grid only decides which thread owns which
four coordinates."""
import ctypes

import numpy as np
import pytest
import torch

from gpu_harness import log
from paper_2607_21224_amd import build, cpdp
from paper_2607_21224_amd.state import CpdpState, Hyper, Optimizer
from synth import device as sdev

pytestmark = pytest.mark.gpu

CASES = [
    # (W, P, K, param_dt, optimizer, flags, method)
    (8, 100_003, 3, "f32", None, 0, "cpdp"),          # compile-time W, ragged tail
    (5, 10_007, 2, "bf16", None, 0, "cpdp"),          # run-time W
    (4, 65_539, 2, "f32", "adamw", 3, "cpdp"),        # the variants' kernel
    (6, 4_099, 3, "f32", "sgd_wd", 0, "localsgd"),
    (3, 2_053, 1, "bf16", None, 0, "ddp"),
]


def _drive(lib, st, grads, s, h, opt, flags, method, stream):
    """One step of the period on library `lib` (the ABI calls, not the binding
    wrappers, so either build can be driven)."""
    vp = lambda x: ctypes.c_void_p(x.data_ptr())  # noqa: E731
    dt = 1 if st.param_dt == "bf16" else 0
    sync = method == "ddp" or cpdp.cpdp_is_sync_step(s, st.K, 0)
    ss = ctypes.c_void_p(stream.cuda_stream)
    if opt is None:
        if not sync:
            r = lib.cpdp_local_step(vp(st.params), vp(st.mom), vp(grads), st.W, st.P, st.ld,
                                    st.K, h.lr, h.mu, dt, 0, 0, ss)
        elif method == "cpdp":
            r = lib.cpdp_reconcile(vp(st.params), vp(st.mom), vp(grads), vp(st.slow_mom),
                                   vp(st.anchor), st.W, st.P, st.ld, st.K, h.lr, h.mu, h.beta,
                                   h.alpha, dt, 0, 0, ss)
        elif method == "localsgd":
            r = lib.cpdp_localsgd_sync(vp(st.params), vp(st.mom), vp(grads), vp(st.anchor),
                                       st.W, st.P, st.ld, st.K, h.lr, h.mu, dt, 0, 0, ss)
        else:
            r = lib.cpdp_ddp_step(vp(st.params), vp(st.mom), vp(grads), st.W, st.P, st.ld,
                                  h.lr, h.mu, dt, 0, 0, ss)
    else:
        c = opt.c_struct(s)
        m2 = vp(st.mom2) if st.mom2 is not None else None
        if not sync:
            r = lib.cpdp_local_step_opt(vp(st.params), vp(st.mom), m2, vp(grads), st.W, st.P,
                                        st.ld, st.K, ctypes.byref(c), dt, ss)
        else:
            strategy = {"cpdp": 0, "localsgd": 1, "ddp": 2}[method]
            r = lib.cpdp_sync_step_opt(strategy, vp(st.params), vp(st.mom), m2, vp(grads),
                                       vp(st.slow_mom), vp(st.anchor), st.W, st.P, st.ld, st.K,
                                       ctypes.byref(c), h.beta, h.alpha, flags, dt, ss)
    assert r == 0, cpdp.cpdp_status_str(r)


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"W{c[0]}-P{c[1]}-{c[3]}-{c[4]}-f{c[5]}-{c[6]}")
def test_block256_build_bitwise_equal(case):
    W, P, K, pdt, kind, flags, method = case
    log(f"[launch-shape] W={W} P={P} K={K} {pdt} {kind} flags={flags} {method}")
    lib256 = cpdp.load_library(build.LIB_CPDP_BLOCK256)
    stream = torch.cuda.Stream()
    h = Hyper.fp32(0.1, 0.9, 0.5, 1.0)
    opt = None
    if kind == "adamw":
        opt = Optimizer("adamw", 1e-2, 0.9, 0.99, 1e-6, 0.01)
    elif kind == "sgd_wd":
        opt = Optimizer("sgd", 0.1, 0.9, weight_decay=5e-4)
    states = [CpdpState(W, P, None, K, pdt, device="cuda") for _ in range(2)]
    with torch.cuda.stream(stream):
        th = torch.empty(P, dtype=torch.float32, device="cuda")
        sdev.fill_theta0(th, P, 7, 0.02, stream=stream)
        if pdt == "bf16":
            th = th.to(torch.bfloat16)
        for st in states:
            if opt is None:
                st.init(th, stream=stream)
            else:
                st.init_opt(th, opt, stream=stream)
        grads = [torch.empty((W, states[0].ld), dtype=torch.float32, device="cuda")
                 for _ in range(2)]
    for s in range(1, 3 * K + 1):
        with torch.cuda.stream(stream):
            sdev.fill_grads(grads[0], P, 7, s, 1e-3, 0.01, stream=stream)
            grads[1].copy_(grads[0])
        _drive(cpdp.lib, states[0], grads[0], s, h, opt, flags, method, stream)
        _drive(lib256, states[1], grads[1], s, h, opt, flags, method, stream)
        stream.synchronize()
        for fam in ("params", "mom", "mom2", "slow_mom", "anchor"):
            a, b = getattr(states[0], fam), getattr(states[1], fam)
            if a is None:
                continue
            a = a[..., :P] if a.dim() == 2 else a[:P]
            b = b[..., :P] if b.dim() == 2 else b[:P]
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32)), \
                (s, fam)
        assert torch.equal(grads[0][:, :P], grads[1][:, :P]), (s, "grads")
    log("[launch-shape] bitwise equal")
