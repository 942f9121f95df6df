"""Failure detection on the GPU: cpdp_count_unsynced counts the coordinates
at which some replica does not hold the reference model in the parameter
storage type.  The count is an integer, so it is compared exactly with a
recount on the host from the same state; it is 0 after every synchronisation
and flags a driver that skips a due synchronisation and single corrupted
coordinates."""
import numpy as np
import pytest
import torch

from gpu_harness import Case, GpuRun, log
from synth import gen

pytestmark = pytest.mark.gpu


def host_count(st) -> int:
    """The definition, on the host: coordinates p < P where some replica's
    stored bits differ from R(anchor) (a NaN matches a NaN)."""
    P = st.P
    a = st.anchor[:P].cpu().numpy().astype(np.float32)
    if st.param_dt == "bf16":
        a = gen.bf16_round(a)
    x = st.params[:, :P].float().cpu().numpy()
    same = (x.view(np.uint32) == a.view(np.uint32)[None, :]) | \
        (np.isnan(x) & np.isnan(a)[None, :])
    return int((~same.all(axis=0)).sum())


@pytest.mark.parametrize("method", ["cpdp", "localsgd"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_count_after_every_step(method, dt):
    c = Case(W=5, P=10_007, K=3, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=9,
             param_dt=dt, method=method, seed=3)
    log(f"[unsynced] {method} {dt} W={c.W} P={c.P} K={c.K}")
    g = GpuRun(c)
    assert g.st.count_unsynced() == 0 == host_count(g.st)  # after init
    for s in range(1, c.steps + 1):
        kind = g.step(s)
        n = g.st.count_unsynced()
        assert n == host_count(g.st), (s, kind)
        if kind == "reconcile":
            assert n == 0, (s, n)
        elif dt == "f32":
            assert n > 0.9 * c.P, (s, n)  # the replicas took different steps


def test_missed_synchronisation_is_detected():
    """A driver that runs a local step where the cadence asks for a
    reconcile leaves the replicas apart, and the count says so."""
    c = Case(W=4, P=65_537, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=4, seed=4)
    g = GpuRun(c)
    g.step(1)
    # step 2 is a synchronisation step; skip it
    from synth import device as sdev
    sdev.fill_grads(g.grads, c.P, c.seed, 2, c.grad_sigma, c.outlier_rate)
    g.st.local_step(g.grads, g.h)
    n = g.st.count_unsynced()
    assert n == host_count(g.st) and n > 0.9 * c.P
    g.step(3)
    g.step(4)  # the next synchronisation repairs it
    assert g.st.count_unsynced() == 0


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_single_coordinates(dt):
    c = Case(W=3, P=4_099, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=2, param_dt=dt,
             seed=6)
    g = GpuRun(c)
    g.step(1)
    g.step(2)
    st = g.st
    assert st.count_unsynced() == 0
    st.params[2, 123] = st.params[2, 123] * 2 + 1     # one replica, one coordinate
    assert st.count_unsynced() == 1 == host_count(st)
    st.params[0, 123] = st.params[0, 123] + 1         # same coordinate, another replica
    assert st.count_unsynced() == 1
    st.params[1, c.P - 1] = st.params[1, c.P - 1] + 1  # the ragged tail
    assert st.count_unsynced() == 2 == host_count(st)
    st.anchor[7] = float("nan")                       # NaN everywhere at p = 7: consistent
    st.params[:, 7] = float("nan")
    assert st.count_unsynced() == 2 == host_count(st)
    st.params[1, 7] = 0.0                             # a replica missing the NaN
    assert st.count_unsynced() == 3 == host_count(st)
