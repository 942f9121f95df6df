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


STRESS_SLICE = 1 << 21


def _exact_f32(x64: np.ndarray) -> np.ndarray:
    f = x64.astype(np.float32)
    assert np.array_equal(f.astype(np.float64), x64, equal_nan=True), "not an fp32 value"
    return f


def _bf16_bits(x64: np.ndarray) -> np.ndarray:
    b = _exact_f32(x64).view(np.uint32)
    assert not (b & 0xFFFF).any(), "not a bf16 value"
    return (b >> 16).astype(np.uint16)


def _from_bits(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_stress_one_period_every_coordinate():
    """Stress (W=32 bf16 replicas, P=10^8, fp32 gradients, momentum, u and
    anchor, K=4): one whole period on every coordinate.  The fp64 oracle
    state of all coordinates would take about 50 GB of host memory, so the
    oracle keeps its state between steps in the storage types it rounds to
    at every store (bf16 parameters, fp32 momentum, u and anchor: lossless,
    asserted on every store-back) and steps slices of 2^21 coordinates in a
    thread pool; each slice is compared with the same slice of the GPU state
    after every step."""
    from concurrent.futures import ThreadPoolExecutor
    from gpu_harness import check_replicas_reconciled

    w = WORKLOADS["stress"]
    c = Case(W=w.W, P=w.P, K=w.K, lr=w.lr, mu=w.mu, beta=w.beta, alpha=w.alpha, steps=w.K,
             param_dt="bf16", ld=w.ld, seed=42)
    P, W = c.P, c.W
    lr, mu, beta, alpha = c.hyper32()
    th = torch.empty(P, dtype=torch.float32, device="cuda")
    sdev.fill_theta0(th, P, c.seed, c.theta_sigma)
    th0 = th.cpu().numpy()
    del th
    sample = np.array([0, 1, 4097, P // 2 + 3, P - 1])
    assert np.array_equal(th0[sample].view(np.uint32),
                          gen.theta0(c.seed, sample, c.theta_sigma).view(np.uint32))

    slices = [(lo, min(P, lo + STRESS_SLICE)) for lo in range(0, P, STRESS_SLICE)]
    bits = np.empty((W, P), dtype=np.uint16)
    mom = np.empty((W, P), dtype=np.float32)
    slow = np.empty(P, dtype=np.float32)
    anchor = np.empty(P, dtype=np.float32)

    def store(st, lo, hi):
        bits[:, lo:hi] = _bf16_bits(st.params)
        mom[:, lo:hi] = _exact_f32(st.mom)
        slow[lo:hi] = _exact_f32(st.slow)
        anchor[lo:hi] = _exact_f32(st.anchor)

    def init(sl):
        lo, hi = sl
        store(oracle.state_init(th0[lo:hi].astype(np.float64), W, "bf16"), lo, hi)

    oracle.lib()  # load once before the worker threads call into it
    g = GpuRun(c)
    workers = 12
    with ThreadPoolExecutor(workers) as pool:
        list(pool.map(init, slices))
        for s in range(1, c.steps + 1):
            kind = g.step(s)
            torch.cuda.synchronize()
            if s == 1:
                got = g.grads[:, sample].cpu().numpy()
                assert np.array_equal(got.view(np.uint32),
                                      gen.grads(c.seed, s, W, sample, c.grad_sigma).view(np.uint32))

            def work(sl, s=s, kind=kind):
                lo, hi = sl
                n = hi - lo
                g64 = g.grads[:, lo:hi].cpu().numpy().astype(np.float64)
                st = oracle.OracleState(W, n, _from_bits(bits[:, lo:hi]),
                                        mom[:, lo:hi].astype(np.float64),
                                        slow[lo:hi].astype(np.float64),
                                        anchor[lo:hi].astype(np.float64), "bf16", "f32", "f32")
                if kind == "reconcile":
                    oracle.reconcile(st, g64, lr, mu, beta, alpha)
                else:
                    oracle.local_step(st, g64, lr, mu)
                del g64
                store(st, lo, hi)
                snap = {"params": g.st.params[:, lo:hi].float().cpu().numpy().astype(np.float64),
                        "mom": g.st.mom[:, lo:hi].cpu().numpy().astype(np.float64),
                        "slow_mom": g.st.slow_mom[lo:hi].cpu().numpy().astype(np.float64),
                        "anchor": g.st.anchor[lo:hi].cpu().numpy().astype(np.float64)}
                tag = f"stress every coordinate, step {s} ({kind}), coords [{lo}, {hi})"
                m = compare(snap, st, "bf16", tag, lr=lr)
                if kind == "reconcile":
                    check_replicas_reconciled(snap, "bf16", tag)
                return m

            worst = {}
            for m in pool.map(work, slices):
                for k, v in m.items():
                    worst[k] = max(worst.get(k, 0.0), v)
            log(f"[full-coords] stress step {s} {kind}: {W}x{P} coordinates match; worst "
                f"error / tolerance " + ", ".join(f"{k} {v:.3g}" for k, v in worst.items()))
    assert kind == "reconcile"
