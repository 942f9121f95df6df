"""The C ABI from a host program that uses only the HIP runtime (no PyTorch):
tests/consumer/abi_consumer allocates with hipMalloc, creates its own stream,
drives cpdp_state_init / cpdp_local_step / cpdp_reconcile on the cadence of
cpdp_is_sync_step and writes the final state, which must match the oracle.
The program also checks that the row padding it filled is untouched.

It runs as a child process; the module name sorts first among the GPU tests
so that the pytest process normally has not used the GPU yet when it starts."""
import os
import subprocess

import numpy as np
import pytest

from gpu_harness import Case, compare, log, run_oracle, state_from_grads
from synth import gen

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "consumer", "abi_consumer")

CASES = [
    Case(W=5, P=4_099, K=3, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=9),
    Case(W=8, P=1_027, K=4, lr=0.05, mu=0.9, beta=0.7, alpha=0.75, steps=10, T=6,
         param_dt="bf16"),
]


@pytest.mark.parametrize("c", CASES, ids=lambda c: f"W{c.W}-P{c.P}-K{c.K}-T{c.T}-{c.param_dt}")
def test_torch_free_consumer_matches_oracle(c, tmp_path):
    assert os.path.exists(BIN), "tests/consumer/abi_consumer is not built (run build())"
    idx = np.arange(c.P)
    th0 = gen.theta0(c.seed, idx, c.theta_sigma)
    if c.param_dt == "bf16":
        th0 = gen.bf16_round(th0)
        (th0.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16).tofile(
            tmp_path / "theta0.bin")
    else:
        th0.astype(np.float32).tofile(tmp_path / "theta0.bin")
    for s in range(1, c.steps + 1):
        gen.grads(c.seed, s, c.W, idx, c.grad_sigma, c.outlier_rate).astype(
            np.float32).tofile(tmp_path / f"grads_{s}.bin")

    refs = {}
    run_oracle(c, idx, lambda s, kind, st, m2: refs.__setitem__(s, (kind, st.copy())))

    lr, mu, beta, alpha = c.hyper32()
    args = [BIN, str(c.W), str(c.P), str(c.K), str(c.steps), str(c.T), repr(lr), repr(mu),
            repr(beta), repr(alpha), "1" if c.param_dt == "bf16" else "0", str(tmp_path)]
    log("[consumer] " + " ".join(args[1:-1]))
    r = subprocess.run(args, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, f"abi_consumer failed ({r.returncode}): {r.stdout}{r.stderr}"

    kinds = (tmp_path / "kinds.txt").read_text().split()
    assert kinds == [refs[s][0] for s in range(1, c.steps + 1)]
    if c.param_dt == "bf16":
        bits = np.fromfile(tmp_path / "params.bin", dtype=np.uint16).astype(np.uint32) << 16
        params = bits.view(np.float32)
    else:
        params = np.fromfile(tmp_path / "params.bin", dtype=np.float32)
    snap = {"params": params.reshape(c.W, c.P).astype(np.float64),
            "mom": np.fromfile(tmp_path / "mom.bin", dtype=np.float32).reshape(
                c.W, c.P).astype(np.float64),
            "slow_mom": np.fromfile(tmp_path / "slow.bin", dtype=np.float32).astype(np.float64),
            "anchor": np.fromfile(tmp_path / "anchor.bin", dtype=np.float32).astype(np.float64)}
    compare(snap, refs[c.steps][1], c.param_dt, f"consumer {c.param_dt} final", lr=lr,
            fp32_state=state_from_grads(None))
