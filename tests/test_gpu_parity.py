"""GPU parity: the HIP path (through the C ABI) against the oracle, element by
element after every local step and every reconcile."""
import pytest

from gpu_harness import Case, run_parity, sample_indices
from synth import WORKLOADS

pytestmark = pytest.mark.gpu


def case_of(name, seed=42, steps=None):
    w = WORKLOADS[name]
    return Case(W=w.W, P=w.P, K=w.K, lr=w.lr, mu=w.mu, beta=w.beta,
                alpha=w.alpha, steps=steps or w.steps, param_dt=w.param_dt,
                seed=seed, ld=w.ld, theta_sigma=w.theta_sigma,
                grad_sigma=w.grad_sigma, outlier_rate=w.outlier_rate)


@pytest.mark.parametrize("seed", [42, 123, 777])
def test_tiny_every_coordinate(seed):
    """W=4, P=262,144, K=2, 10 periods: the whole state after every step."""
    run_parity(case_of("tiny", seed))


def test_stress_bf16_gradients_sampled():
    """The stress workload with bf16 gradient rows (bf16 parameters, bf16
    gradients, fp32 momentum, u and anchor), full size, sampled coordinates,
    one period."""
    w = WORKLOADS["stress"]
    c = case_of("stress", steps=w.K)
    c.grad_dt = "bf16"
    run_parity(c, sample_indices(w.P, n_random=1 << 15, seed=42))


def test_stress_all_bf16_replica_state_sampled():
    """The stress workload with every per-replica family in bf16 (parameters,
    gradients, momentum; u and anchor fp32), full size, sampled coordinates,
    one period."""
    w = WORKLOADS["stress"]
    c = case_of("stress", steps=w.K)
    c.grad_dt, c.mom_dt = "bf16", "bf16"
    run_parity(c, sample_indices(w.P, n_random=1 << 15, seed=7))


def test_tiny_long_horizon_every_coordinate():
    """200 periods (400 steps) of the tiny workload, every coordinate compared
    every 20 periods: the anchor accumulates across periods, so this checks
    that rounding differences between the fp32 kernel and the oracle stay
    bounded over a long run instead of drifting out of tolerance."""
    run_parity(case_of("tiny", steps=400), every=40)


@pytest.mark.parametrize("seed", [42, 123, 777])
@pytest.mark.parametrize("name", ["r50_100", "vit_s", "r50_200", "stress"])
def test_full_size_sampled(name, seed):
    """Full-size workloads in the benchmark's launch configuration, compared
    on both ends (ragged tail included), every tensor boundary and a random
    sample of coordinates (coordinates are independent), for the three seeds
    of the paper's runs (Sec. 5.1)."""
    w = WORKLOADS[name]
    idx = sample_indices(w.P, w.boundaries()[1:], n_random=1 << 15, seed=seed)
    run_parity(case_of(name, seed), idx)


SMALL = [
    # K = 1: every step reconciles (synchronous DDP cadence)
    Case(W=8, P=10_007, K=1, lr=0.1, mu=0.9, beta=0.3, alpha=1.0, steps=6),
    # plain SGD local steps, no outer momentum, alpha != 1, run-time W
    Case(W=5, P=4_099, K=3, lr=0.2, mu=0.0, beta=0.0, alpha=1.5, steps=9),
    # epoch boundary not a multiple of K: forced sync at t = T
    Case(W=4, P=3_001, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=12, T=6),
    Case(W=16, P=2_053, K=8, lr=0.1, mu=0.9, beta=0.6, alpha=1.0, steps=16,
         outlier_rate=0.01),
    Case(W=32, P=1_031, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=8),
    Case(W=32, P=5_003, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=8,
         param_dt="bf16"),
    Case(W=8, P=777, K=2, lr=0.05, mu=0.9, beta=0.7, alpha=0.75, steps=8,
         param_dt="bf16"),
    Case(W=3, P=1_000, K=2, lr=0.5, mu=0.5, beta=0.9, alpha=1.0, steps=10,
         theta_sigma=1.0, grad_sigma=0.1),
    Case(W=1, P=513, K=3, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=9),
    Case(W=2, P=64, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=6, ld=128),
    # bf16 gradient rows on the momentum-SGD entry points
    Case(W=8, P=10_007, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=8, grad_dt="bf16"),
    Case(W=5, P=4_099, K=3, lr=0.2, mu=0.9, beta=0.3, alpha=1.0, steps=9, grad_dt="bf16"),
    Case(W=16, P=2_053, K=8, lr=0.1, mu=0.9, beta=0.6, alpha=1.0, steps=16,
         outlier_rate=0.01, grad_dt="bf16"),
    Case(W=32, P=5_003, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=8,
         param_dt="bf16", grad_dt="bf16"),
    Case(W=4, P=3_001, K=2, lr=0.1, mu=0.9, beta=0.0, alpha=1.0, steps=6,
         method="localsgd", grad_dt="bf16"),
    Case(W=4, P=3_001, K=1, lr=0.1, mu=0.9, beta=0.0, alpha=1.0, steps=4,
         method="ddp", grad_dt="bf16"),
    # bf16 momentum buffers (with fp32 or bf16 gradients and parameters)
    Case(W=8, P=10_007, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=8, mom_dt="bf16"),
    Case(W=5, P=4_099, K=3, lr=0.2, mu=0.9, beta=0.3, alpha=1.0, steps=9, grad_dt="bf16",
         mom_dt="bf16"),
    Case(W=32, P=5_003, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=8,
         param_dt="bf16", grad_dt="bf16", mom_dt="bf16"),
    Case(W=4, P=3_001, K=2, lr=0.1, mu=0.9, beta=0.0, alpha=1.0, steps=6,
         method="localsgd", mom_dt="bf16"),
    Case(W=4, P=3_001, K=1, lr=0.1, mu=0.9, beta=0.0, alpha=1.0, steps=4,
         method="ddp", grad_dt="bf16", mom_dt="bf16"),
]


@pytest.mark.parametrize("c", SMALL, ids=lambda c: f"W{c.W}-P{c.P}-K{c.K}-{c.param_dt}"
                         + (f"-T{c.T}" if c.T else "")
                         + (f"-{c.method}" if c.method != "cpdp" else "")
                         + ("-bf16grads" if c.grad_dt == "bf16" else "")
                         + ("-bf16mom" if c.mom_dt == "bf16" else ""))
def test_small_variants(c):
    run_parity(c)
