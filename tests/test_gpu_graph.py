"""A CPDP period captured into a HIP graph and replayed: every replay, with
eager work and synchronisations in between, equals the eager run bitwise."""
import numpy as np
import pytest
import torch

from gpu_harness import Case, GpuRun
from synth import device as sdev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("method", ["cpdp", "localsgd", "ddp"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_period_graph_replays_match_eager(method, dt):
    c = Case(W=4, P=262_144, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=2,
             param_dt=dt, method=method)
    eager, graphed = GpuRun(c), GpuRun(c)
    bufs = [torch.empty_like(graphed.grads) for _ in range(c.K)]
    graph, kinds = graphed.st.capture_period(bufs, graphed.h, method=method)
    torch.cuda.synchronize()
    # capturing ran nothing: the state is still the initial one
    assert torch.equal(graphed.st.params[:, :c.P], eager.st.params[:, :c.P])
    for period in range(4):
        for j in range(c.K):
            step = period * c.K + j + 1
            sdev.fill_grads(bufs[j], c.P, c.seed, step, c.grad_sigma)  # eager work
            kind = eager.step(step)
            assert kind == kinds[j]
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        a, b = eager.snapshot(), graphed.snapshot()
        for k in a:
            assert np.array_equal(a[k], b[k], equal_nan=True), (period, k)
