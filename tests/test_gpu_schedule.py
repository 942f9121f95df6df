"""Training-loop fidelity on the GPU path: warmup epochs at K = 1 followed by
the configured period, a per-step cosine learning rate with linear warmup, and
an epoch length that is not a multiple of K (forced epoch-end sync), all
against the oracle after every step."""
import numpy as np
import pytest
import torch

import oracle
from gpu_harness import Case, GpuRun, compare, oracle_inputs, state_from_grads
from paper_2607_21224_amd import cpdp
from paper_2607_21224_amd.state import Hyper

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("method", ["cpdp", "localsgd"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_warmup_and_lr_schedule(method, dt):
    T, warm_epochs, K, epochs = 10, 1, 4, 3
    total = T * epochs
    base, low, warm_steps = 0.1, 0.001, 5
    c = Case(W=8, P=30_011, K=K, lr=base, mu=0.9, beta=0.5, alpha=1.0, steps=total,
             param_dt=dt, T=T, method=method)
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    lr_oracle = [f32(oracle.lr_at(s, total, warm_steps, f32(base), f32(low))) for s in range(total)]
    lr_gpu = [cpdp.cpdp_lr_at(s, total, warm_steps, base, low) for s in range(total)]
    assert lr_gpu == lr_oracle

    refs = {}
    th0, grads = oracle_inputs(c, np.arange(c.P))
    oracle.run(th0, grads, c.W, lambda e: oracle.period_for_epoch(e, warm_epochs, K), total,
               lambda s: lr_oracle[s - 1], f32(0.9), f32(0.5), f32(1.0), T=T, param_dt=dt,
               method=method, callback=lambda s, k, st: refs.__setitem__(s, (k, st.copy())))
    g = GpuRun(c)
    from synth import device as sdev
    for s in range(1, total + 1):
        epoch, t = divmod(s - 1, T)
        g.st.K = cpdp.cpdp_period_for_epoch(epoch, warm_epochs, K)
        sdev.fill_grads(g.grads, c.P, c.seed, s, c.grad_sigma)
        h = Hyper.fp32(lr_gpu[s - 1], 0.9, 0.5, 1.0)
        kind = g.st.step(t + 1, g.grads, h, T, method=method)
        rk, ref = refs[s]
        assert kind == rk, (s, kind, rk)
        # the SlowMo state is gated as the velocity v = -lr*u at this step's lr:
        # during the warmup ramp (lr 0.02 ... 0.1) one fp32-ulp flip of one
        # replica moves u by ulp/(W*lr), at the edge of a 1e-6 relative gate
        compare(g.snapshot(), ref, dt, f"{method} step {s} ({kind})",
                velocity_lr=lr_gpu[s - 1], fp32_state=state_from_grads(None))
    torch.cuda.synchronize()
