"""Every coordinate of the ResNet-50/CIFAR-100-sized workload (W=8,
P=23,712,932 in 161 tensors, K=4), of the ViT-S-sized one (W=8,
P=21,332,068, K=4) and of the ResNet-50/TinyImageNet-sized one (W=16,
P=23,917,832, K=8, gradients with 1 % outliers x100) for one whole period
(K-1 local steps and the reconcile) against the oracle, in the benchmark's
launch configuration.

Inputs come from the seeded generator: on the device for the HIP path, copied
to the host for the oracle (the generator is the one module both sides share;
a sample of each copy is re-derived here with the host generator, bit for
bit).  Nothing the HIP path computes feeds the oracle."""
import numpy as np
import pytest
import torch

import oracle
from gpu_harness import Case, GpuRun, compare, log
from synth import WORKLOADS, gen
from synth import device as sdev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["r50_100", "vit_s", "r50_200"])
def test_one_period_every_coordinate(name):
    w = WORKLOADS[name]
    c = Case(W=w.W, P=w.P, K=w.K, lr=w.lr, mu=w.mu, beta=w.beta, alpha=w.alpha, steps=w.K,
             ld=w.ld, seed=42, outlier_rate=w.outlier_rate)
    P, W = c.P, c.W
    lr, mu, beta, alpha = c.hyper32()
    rng = np.random.default_rng(0)
    sample = np.unique(np.concatenate([np.arange(64), P - 64 + np.arange(64),
                                       rng.integers(0, P, 4096)]))

    th = torch.empty(P, dtype=torch.float32, device="cuda")
    sdev.fill_theta0(th, P, c.seed, c.theta_sigma)
    th0 = th.cpu().numpy()
    assert np.array_equal(th0[sample].view(np.uint32),
                          gen.theta0(c.seed, sample, c.theta_sigma).view(np.uint32))
    ref = oracle.state_init(th0.astype(np.float64), W, "f32")
    del th

    g = GpuRun(c)
    for s in range(1, c.steps + 1):
        kind = g.step(s)  # fills g.grads with step s's gradients, then steps
        torch.cuda.synchronize()
        grads = g.grads[:, :P].cpu().numpy()
        assert np.array_equal(grads[:, sample].view(np.uint32),
                              gen.grads(c.seed, s, W, sample, c.grad_sigma,
                                        c.outlier_rate).view(np.uint32))
        g64 = grads.astype(np.float64)
        del grads
        if kind == "reconcile":
            oracle.reconcile(ref, g64, lr, mu, beta, alpha)
        else:
            oracle.local_step(ref, g64, lr, mu)
        del g64
        snap = g.snapshot()
        m = compare(snap, ref, "f32", f"{name} every coordinate, step {s} ({kind})", lr=lr)
        del snap
        log(f"[full-coords] {name} step {s} {kind}: {W}x{P} coordinates match; worst error / "
            f"tolerance " + ", ".join(f"{k} {v:.3g}" for k, v in m.items()))
    assert kind == "reconcile"
