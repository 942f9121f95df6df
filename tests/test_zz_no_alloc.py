"""The allocation-free plan build (cpdp_plan_build_static) against the
caller-table build (cpdp_plan_build): the same tensors stepped through a plan
on the library's own table and through a plan on a caller-allocated table
end bitwise equal, on two static builds in a row (the second smaller); a plan
from the first static build is refused once the second has replaced the
table; an oversized plan is refused before any runtime call."""
import numpy as np
import pytest
import torch

from gpu_harness import log

pytestmark = pytest.mark.gpu


def _flat(fam, W, n):
    return [fam[i][t] for i in range(W) for t in range(n)]


def _static(multi):
    """Rebuild multi's plan on the library's static table."""
    from paper_2607_21224_amd import cpdp
    plan = cpdp.cpdp_plan()
    adamw = multi.mom2 is not None
    cpdp.cpdp_plan_build_static(plan, multi.W, multi.n, multi.numels,
                                _flat(multi.params, multi.W, multi.n),
                                _flat(multi.mom, multi.W, multi.n),
                                _flat(multi.mom2, multi.W, multi.n) if adamw else None,
                                _flat(multi.grads, multi.W, multi.n), multi.slow_mom,
                                multi.anchor, multi.param_dt)
    assert plan.table not in (0, None) and plan.table != multi.table.data_ptr()
    multi.plan = plan
    return plan


def _state(multi):
    out = {}
    for fam in ("params", "mom", "mom2", "grads"):
        rows = getattr(multi, fam)
        if rows is None:
            continue
        out[fam] = [r[t][:multi.numels[t]].view(torch.int16 if r[t].dtype == torch.bfloat16
                                                else torch.int32).cpu()
                    for r in rows for t in range(multi.n)]
    for fam in ("slow_mom", "anchor"):
        out[fam] = [x[:multi.numels[t]].view(torch.int32).cpu()
                    for t, x in enumerate(getattr(multi, fam))]
    return out


def _run_pair(W, numels, param_dt, opt, steps, K, seed):
    """Two identical multi-tensor states, one on a caller table and one on
    the static table, stepped alike; returns the static state's plan."""
    from paper_2607_21224_amd.multi import CpdpMultiState
    log(f"[no-alloc] W={W} tensors={len(numels)} numel={sum(numels)} {param_dt} {opt.kind}")
    adamw = opt.kind == "adamw"
    a = CpdpMultiState(W, numels, K, param_dt, adamw)
    b = CpdpMultiState(W, numels, K, param_dt, adamw)
    plan = _static(b)
    rng = np.random.default_rng(seed)
    th = [torch.from_numpy(rng.normal(0, 0.02, x).astype(np.float32)).cuda() for x in numels]
    a.init(th)
    b.init(th)
    for s in range(1, steps + 1):
        for i in range(W):
            for t, x in enumerate(numels):
                g = torch.from_numpy(rng.normal(0, 1e-3, x).astype(np.float32)).cuda()
                a.grads[i][t][:x].copy_(g)
                b.grads[i][t][:x].copy_(g)
        ka = a.step(s, opt, 0.5, 1.0, flags=3 if s % K == 0 else 0)
        kb = b.step(s, opt, 0.5, 1.0, flags=3 if s % K == 0 else 0)
        assert ka == kb
        torch.cuda.synchronize()
        sa, sb = _state(a), _state(b)
        for fam in sa:
            for k, (x, y) in enumerate(zip(sa[fam], sb[fam])):
                assert torch.equal(x, y), f"step {s} ({ka}): {fam}[{k}] differs"
    return b, plan


def test_static_plan_equals_caller_table_plan_twice():
    from paper_2607_21224_amd import cpdp
    from paper_2607_21224_amd.state import Optimizer
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    adamw = Optimizer("adamw", f32(5e-4), f32(0.9), f32(0.999), f32(1e-8), f32(0.05))
    sgd = Optimizer("sgd", f32(0.1), f32(0.9), weight_decay=f32(5e-4))
    # first call: 8 replicas of a ragged 6-tensor model
    b1, plan1 = _run_pair(8, [5000, 0, 1027, 3, 8198, 4096], "f32", adamw, 6, 3, 1)
    # second call, smaller: 3 replicas of 3 tensors, bf16 parameters
    b2, plan2 = _run_pair(3, [1029, 7, 2048], "bf16", sgd, 4, 2, 2)
    # both static plans sit on the same array of this GPU
    assert plan1.table == plan2.table
    # the first static plan's handle is refused now that its table was replaced
    c = sgd.c_struct(1)
    s = cpdp.cpdp_local_step_plan(plan1, 3, c, check=False)
    assert s == cpdp.CPDP_ERR_INVALID_ARG
    assert cpdp.cpdp_local_step_plan(plan2, 2, c, check=False) == cpdp.CPDP_OK
    torch.cuda.synchronize()


def test_static_plan_refuses_oversized_tables():
    from paper_2607_21224_amd import cpdp
    W, n = 64, 200
    assert cpdp.cpdp_plan_bytes(W, n) > cpdp.CPDP_PLAN_STATIC_BYTES
    x = torch.zeros(64, device="cuda")
    fam = [x] * (W * n)
    plan = cpdp.cpdp_plan()
    s = cpdp.cpdp_plan_build_static(plan, W, n, [0] * n, fam, fam, None, fam, None, None,
                                    check=False)
    assert s == cpdp.CPDP_ERR_TOO_LARGE
