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
