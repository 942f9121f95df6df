"""GPU parity of the general optimizers (SGD with weight decay, AdamW; Table 3)
in all three strategies, against the oracle, after every step."""
import pytest

from gpu_harness import Case, run_parity, sample_indices
from synth import WORKLOADS

pytestmark = pytest.mark.gpu

SGD_WD = dict(kind="sgd", lr=0.1, momentum=0.9, weight_decay=5e-4)
ADAMW = dict(kind="adamw", lr=5e-4, momentum=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05)
ADAMW2 = dict(kind="adamw", lr=1e-2, momentum=0.8, beta2=0.99, eps=1e-6, weight_decay=0.0)

CASES = []
for method in ("cpdp", "localsgd", "ddp"):
    for opt in (SGD_WD, ADAMW):
        CASES += [
            Case(W=8, P=10_007, K=4, lr=opt["lr"], mu=0.9, beta=0.5, alpha=1.0, steps=8,
                 method=method, opt=opt),
            Case(W=32, P=3_001, K=4, lr=opt["lr"], mu=0.9, beta=0.5, alpha=1.0, steps=8,
                 param_dt="bf16", method=method, opt=opt),
            Case(W=5, P=1_027, K=3, lr=opt["lr"], mu=0.9, beta=0.3, alpha=1.5, steps=9,
                 method=method, opt=opt),
        ]
    CASES.append(Case(W=4, P=4_099, K=2, lr=1e-2, mu=0.8, beta=0.6, alpha=1.0, steps=8,
                      method=method, opt=ADAMW2))
    CASES.append(Case(W=16, P=2_053, K=8, lr=0.1, mu=0.9, beta=0.6, alpha=1.0, steps=16,
                      outlier_rate=0.01, method=method, opt=SGD_WD))


@pytest.mark.parametrize(
    "c", CASES, ids=lambda c: f"{c.method}-{c.opt['kind']}-wd{c.opt.get('weight_decay', 0)}"
    f"-W{c.W}-P{c.P}-{c.param_dt}")
def test_optimizer_parity(c):
    run_parity(c)


def test_vit_s_adamw_full_size_sampled():
    """The ViT-S-sized state with the paper's ViT-S optimizer (AdamW, lr 5e-4,
    weight decay 0.05) under CPDP, full size, sampled coordinates."""
    w = WORKLOADS["vit_s"]
    c = Case(W=w.W, P=w.P, K=w.K, lr=5e-4, mu=0.9, beta=w.beta, alpha=w.alpha, steps=8,
             ld=w.ld, opt=ADAMW)
    run_parity(c, sample_indices(w.P, w.boundaries()[1:], n_random=1 << 14, seed=3))


def test_r50_sgd_wd_full_size_sampled():
    w = WORKLOADS["r50_100"]
    c = Case(W=w.W, P=w.P, K=w.K, lr=w.lr, mu=w.mu, beta=w.beta, alpha=w.alpha, steps=8,
             ld=w.ld, opt=SGD_WD)
    run_parity(c, sample_indices(w.P, w.boundaries()[1:], n_random=1 << 14, seed=4))


AVG = 2  # optimizer-state reconciliation
WB = 1   # gradient-mean write-back

FLAG_CASES = []
for method in ("cpdp", "localsgd", "ddp"):
    for opt in (SGD_WD, ADAMW):
        FLAG_CASES.append(Case(W=8, P=4_099, K=4, lr=opt["lr"], mu=0.9, beta=0.5, alpha=1.0,
                               steps=8, method=method, opt=opt, flags=AVG))
        FLAG_CASES.append(Case(W=6, P=1_001, K=2, lr=opt["lr"], mu=0.9, beta=0.5, alpha=1.0,
                               steps=6, method=method, opt=opt, flags=AVG | WB,
                               param_dt="bf16"))


@pytest.mark.parametrize(
    "c", FLAG_CASES, ids=lambda c: f"{c.method}-{c.opt['kind']}-flags{c.flags}-W{c.W}-{c.param_dt}")
def test_sync_variants_parity(c):
    """Optimizer-state reconciliation (and write-back) variants, every step."""
    run_parity(c)


@pytest.mark.parametrize("method", ["cpdp", "localsgd", "ddp"])
def test_gradient_mean_write_back(method):
    """After a sync step with the write-back flag every gradient row holds the
    fp32 replica mean (CPDP, DDP); LocalSGD leaves the gradients untouched."""
    import numpy as np
    import torch

    import oracle
    from gpu_harness import GpuRun, oracle_inputs
    c = Case(W=8, P=20_003, K=1, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=1,
             method=method, opt=SGD_WD, flags=WB)
    g = GpuRun(c)
    g.step(1)
    torch.cuda.synchronize()
    got = g.grads[:, :c.P].cpu().numpy().astype(np.float64)
    th0, grads = oracle_inputs(c, np.arange(c.P))
    st = oracle.state_init(th0, c.W)
    o = c.opt32()
    want = oracle.sync_opt(st, method, grads(1, c.W, c.P),
                           oracle.sgd(o["lr"], o["momentum"], o["weight_decay"]), 0.5, 1.0,
                           flags=oracle.SYNC_WRITE_GBAR)
    assert np.allclose(got, want, rtol=1e-6, atol=1e-9)
    if method != "localsgd":
        assert (got == got[0:1]).all()
