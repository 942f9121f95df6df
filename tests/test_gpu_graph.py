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


def test_state_methods_default_to_torchs_current_stream():
    """Without a stream argument the state methods launch on torch's current
    stream: steps called that way inside a graph capture on a side stream are
    captured, and the replay equals the same steps run eagerly, bitwise."""
    import torch
    from paper_2607_21224_amd.state import CpdpState, Hyper
    from synth import device as sdev
    W, P, K = 4, 20_011, 2
    h = Hyper.fp32(0.1, 0.9, 0.5, 1.0)
    th = torch.empty(P, dtype=torch.float32, device="cuda")
    sdev.fill_theta0(th, P, 42, 0.02)
    eager, graphed = CpdpState(W, P, K=K), CpdpState(W, P, K=K)
    grads = []
    for s in (1, 2):
        g = torch.empty((W, eager.ld), dtype=torch.float32, device="cuda")
        sdev.fill_grads(g, P, 42, s, 1e-3, 0.0)
        grads.append(g)
    eager.init(th)
    graphed.init(th)
    for s, g in zip((1, 2), grads):
        eager.step(s, g, h)
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            kinds = [graphed.step(s, g, h) for s, g in zip((1, 2), grads)]
    torch.cuda.current_stream().wait_stream(side)
    assert kinds == ["local", "reconcile"]
    graph.replay()
    torch.cuda.synchronize()
    for name in ("params", "mom", "slow_mom", "anchor"):
        a, b = getattr(eager, name), getattr(graphed, name)
        if a.dim() == 2:  # the row padding [P, ld) is never written
            a, b = a[:, :P], b[:, :P]
        assert torch.equal(a, b), name
