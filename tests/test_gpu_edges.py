"""Edge cases of the HIP path: ragged and empty sizes, row padding left
untouched, NaN/Inf propagation, determinism, and coordinate independence."""
import numpy as np
import pytest
import torch

import oracle
from gpu_harness import (Case, GpuRun, compare, log, oracle_inputs, run_parity,
                         state_from_grads, tolerance_regime)
from paper_2607_21224_amd import cpdp
from paper_2607_21224_amd.state import CpdpState, Hyper

pytestmark = pytest.mark.gpu

RAGGED = [(W, P) for W in (1, 2, 3, 5, 8, 32)
          for P in (1, 3, 4, 5, 7, 8, 9, 1023, 1025, 4097, (1 << 20) + 3)]


@pytest.mark.parametrize("W,P", RAGGED)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_ragged_sizes_and_pad_canaries(W, P, dt):
    """Every ragged size matches the oracle, and the padding columns
    [P, ld) of every row keep their canary bytes."""
    _ragged_case(W, P, dt, "f32")


RAGGED_BF16_GRADS = [(W, P) for W in (1, 3, 8, 32) for P in (1, 5, 1025, 4097, (1 << 20) + 3)]


@pytest.mark.parametrize("W,P", RAGGED_BF16_GRADS)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("mom_dt", ["f32", "bf16"])
def test_ragged_sizes_bf16_gradients(W, P, dt, mom_dt):
    """The same with bf16 gradient rows, and fp32 or bf16 momentum (the
    64-bit vector loads and stores and the scalar tails of the bf16 paths)."""
    _ragged_case(W, P, dt, "bf16", mom_dt)


def _ragged_case(W, P, dt, grad_dt, mom_dt="f32"):
    ld = ((P + 127) // 128) * 128 + 128
    c = Case(W=W, P=P, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=4,
             param_dt=dt, ld=ld, seed=P * 100 + W, grad_dt=grad_dt, mom_dt=mom_dt)
    log(f"[ragged] W={W} P={P} dt={dt} grads={grad_dt} mom={mom_dt}")
    refs = {}
    th0, grads = oracle_inputs(c, np.arange(P))
    oracle.run(th0, grads, W, c.K, c.steps, *c.hyper32(), param_dt=dt, mom_dt=mom_dt,
               callback=lambda s, k, st: refs.__setitem__(s, st.copy()))
    g = GpuRun(c)
    canary = torch.tensor(-1280.0, dtype=torch.float32)  # exact in bf16
    g.st.params[:, P:] = canary.to(g.st.params.dtype)
    g.st.mom[:, P:] = canary.to(g.st.mom.dtype)
    g.grads[:, P:] = canary
    for s in range(1, c.steps + 1):
        g.step(s)
        compare(g.snapshot(), refs[s], tolerance_regime(c), f"W={W} P={P} step {s}",
                lr=c.hyper32()[0], fp32_state=state_from_grads(None, mom_dt))
    torch.cuda.synchronize()
    assert (g.st.params[:, P:].float() == -1280.0).all()
    assert (g.st.mom[:, P:] == -1280.0).all()


def test_p_zero_is_noop():
    st = CpdpState(4, 0, ld=64)
    h = Hyper.fp32(0.1, 0.9, 0.5, 1.0)
    g = torch.zeros((4, 64), device="cuda")
    st.mom.fill_(7.0)
    st.init(torch.zeros(1, device="cuda"))
    st.local_step(g, h)
    st.reconcile(g, h)
    torch.cuda.synchronize()
    assert (st.mom == 7.0).all()


def test_nan_inf_propagation():
    """A NaN in one replica's gradient reaches every replica through the
    gradient mean at the next reconcile; an Inf likewise; positions match the
    oracle."""
    W, P, K = 4, 4096, 2
    c = Case(W=W, P=P, K=K, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=4)
    h = c.hyper32()
    th0, grads = oracle_inputs(c, np.arange(P))
    poison = {2: [(1, 17, np.nan), (3, 4095, np.inf)], 3: [(0, 100, -np.inf)]}

    def gfun(step, W_, P_):
        x = grads(step, W_, P_)
        for (i, p, v) in poison.get(step, []):
            x[i, p] = v
        return x

    refs = {}
    oracle.run(th0, gfun, W, K, c.steps, *h,
               callback=lambda s, k, st: refs.__setitem__(s, st.copy()))
    g = GpuRun(c)
    for s in range(1, c.steps + 1):
        from synth import device as sdev
        sdev.fill_grads(g.grads, P, c.seed, s, c.grad_sigma)
        for (i, p, v) in poison.get(s, []):
            g.grads[i, p] = float(v)
        t = s
        g.st.step(t, g.grads, g.h)
        snap = g.snapshot()
        compare(snap, refs[s], "f32", f"nan step {s}")
    assert np.isnan(snap["params"][:, 17]).all()


def test_bitwise_deterministic():
    c = Case(W=8, P=100_003, K=4, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=8)
    a, b = GpuRun(c), GpuRun(c)
    for s in range(1, c.steps + 1):
        a.step(s)
        b.step(s)
    sa, sb = a.snapshot(), b.snapshot()
    for k in sa:
        assert np.array_equal(sa[k], sb[k], equal_nan=True), k


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_subset_equals_full(dt):
    """Coordinates are independent: a run over the first P_sub coordinates
    (whose ragged tail takes the scalar path) is bitwise equal to the same
    coordinates of a run over P_full (vector path)."""
    full = Case(W=8, P=65_536, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0,
                steps=6, param_dt=dt)
    sub = Case(**{**full.__dict__, "P": 65_531})
    a, b = GpuRun(full), GpuRun(sub)
    for s in range(1, full.steps + 1):
        a.step(s)
        b.step(s)
    sa, sb = a.snapshot(), b.snapshot()
    for k in sa:
        x = sa[k][..., :sub.P]
        assert np.array_equal(x, sb[k], equal_nan=True), k


def test_streams():
    """Work enqueued on a non-default stream lands in order on that stream."""
    s = torch.cuda.Stream()
    c = Case(W=4, P=20_000, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=4)
    with torch.cuda.stream(s):
        run_parity(c, stream=s)


def test_invalid_call_leaves_state_untouched():
    st = CpdpState(2, 100)
    st.init(torch.ones(100, device="cuda"))
    torch.cuda.synchronize()
    before = st.params.clone()
    g = torch.zeros((2, st.ld), device="cuda")
    with pytest.raises(cpdp.CpdpError):
        st.reconcile(g, Hyper(0.1, 0.9, 1.5, 1.0))  # beta >= 1
    torch.cuda.synchronize()
    assert torch.equal(before, st.params)


@pytest.mark.parametrize("opt", [None, dict(kind="adamw", lr=5e-4, momentum=0.9,
                                            beta2=0.999, eps=1e-8, weight_decay=0.05)])
def test_checkpoint_resume_bitwise(tmp_path, opt):
    """Two periods, a checkpoint through a file, a fresh state restored from
    it, three more periods: bitwise equal to five uninterrupted periods."""
    c = Case(W=8, P=50_021, K=4, lr=0.1 if opt is None else 5e-4, mu=0.9, beta=0.5,
             alpha=1.0, steps=20, opt=opt)
    ref = GpuRun(c)
    for s in range(1, 21):
        ref.step(s)
    want = ref.snapshot()

    a = GpuRun(c)
    for s in range(1, 9):
        a.step(s)
    torch.cuda.synchronize()
    path = tmp_path / "cpdp_state.pt"
    torch.save(a.st.state_dict(), path)
    b = GpuRun(c)                       # fresh buffers, re-initialised
    b.st = CpdpState.from_state_dict(torch.load(path, weights_only=True))
    for s in range(9, 21):
        b.step(s)
    got = b.snapshot()
    for k in want:
        assert np.array_equal(got[k], want[k], equal_nan=True), k


HUGE = [
    # one row longer than 2^31 coordinates (fp32: 8.6 GB per row)
    dict(W=2, P=(1 << 31) + 1027, dt="f32", grad_dt="f32", mom_dt="f32", gib=80),
    # one row longer than 2^32 coordinates, every replica family in bf16
    dict(W=1, P=(1 << 32) + 517, dt="bf16", grad_dt="bf16", mom_dt="bf16", gib=110),
]


@pytest.mark.parametrize("h", HUGE, ids=lambda h: f"W{h['W']}-P{h['P']}-{h['dt']}")
def test_coordinates_beyond_32_bit_indices(h):
    """Coordinate indices past 2^31 and 2^32 inside one row: the device
    generator, every kernel's 64-bit index arithmetic and the ragged tail,
    compared with the oracle on both ends, on 2048 coordinates around each
    power-of-two boundary and on a random sample, over two periods."""
    free, _ = torch.cuda.mem_get_info()
    if free < h["gib"] << 30:
        pytest.skip(f"needs about {h['gib']} GiB of free device memory, {free >> 30} GiB free")
    P = h["P"]
    rng = np.random.default_rng(3)
    parts = [np.arange(2048), np.arange(P - 2048, P), rng.integers(0, P, 1 << 14)]
    for b in (1 << 31, 1 << 32):
        if b < P:
            parts.append(np.arange(b - 1024, min(b + 1024, P)))
    idx = np.unique(np.concatenate(parts)).astype(np.int64)
    c = Case(W=h["W"], P=P, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=4,
             param_dt=h["dt"], grad_dt=h["grad_dt"], mom_dt=h["mom_dt"])
    try:
        g = run_parity(c, idx)
        # the consistency check over the same rows: the run ended on a
        # reconcile, so every replica holds the reference model; one replica
        # changed at one coordinate past the last power-of-two boundary counts 1
        st = g.st
        assert st.count_unsynced() == 0
        p = P - 3
        i = c.W - 1
        old = st.params[i, p].clone()
        st.params[i, p] = old + 1.0
        assert st.count_unsynced() == 1
        st.params[i, p] = old
        assert st.count_unsynced() == 0
    finally:
        torch.cuda.empty_cache()
