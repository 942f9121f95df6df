"""Shared driver for the GPU parity tests: runs the same seeded CPDP schedule
through the C ABI on the GPU and through the oracle on the CPU, and compares
them after every step on a set of coordinates (all of them for small sizes).

Inputs: theta0 and gradients come from the seeded counter-based generator
(synth.gen on the host for the oracle, synth/synth.hip on the device for the
GPU path); the two generators are checked bit for bit in test_gpu_inputs.py.
No value computed by the HIP path ever feeds the oracle.
"""
from __future__ import annotations

import sys
from dataclasses import dataclass

import numpy as np
import torch

import oracle
from synth import device as sdev
from synth import gen

# fp32 tolerance of the reconcile path: |gpu - ref| <= ATOL + RTOL * |ref|
RTOL_F32, ATOL_F32 = 1e-6, 1e-7
# bf16 replica parameters: relative 1e-2 (atol only for exact-zero refs)
RTOL_BF16, ATOL_BF16 = 1e-2, 1e-5


@dataclass
class Case:
    W: int
    P: int
    K: int
    lr: float
    mu: float
    beta: float
    alpha: float
    steps: int
    param_dt: str = "f32"
    seed: int = 42
    ld: int | None = None
    T: int = 0
    theta_sigma: float = 0.02
    grad_sigma: float = 1e-3
    outlier_rate: float = 0.0
    method: str = "cpdp"

    def hyper32(self):
        f = lambda x: float(np.float32(x))  # noqa: E731
        return f(self.lr), f(self.mu), f(self.beta), f(self.alpha)


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def sample_indices(P: int, boundaries=(), n_random: int = 1 << 15, seed: int = 0,
                   edge: int = 2048) -> np.ndarray:
    """Coordinates to compare at full size: both ends (incl. the ragged tail),
    every tensor boundary +-2, and a random sample."""
    rng = np.random.default_rng(seed)
    parts = [np.arange(min(edge, P)), np.arange(max(0, P - edge), P),
             rng.integers(0, P, size=min(n_random, P))]
    b = np.asarray(boundaries, dtype=np.int64)
    if b.size:
        parts.append((b[:, None] + np.arange(-2, 3)[None, :]).ravel())
    idx = np.unique(np.concatenate(parts))
    return idx[(idx >= 0) & (idx < P)]


def oracle_inputs(c: Case, idx: np.ndarray):
    th0 = gen.theta0(c.seed, idx, c.theta_sigma).astype(np.float64)

    def grads(step, W, P):
        return gen.grads(c.seed, step, c.W, idx, c.grad_sigma,
                         c.outlier_rate).astype(np.float64)
    return th0, grads


def run_oracle(c: Case, idx: np.ndarray, on_step):
    """on_step(step, kind, oracle_state)"""
    h = c.hyper32()
    th0, grads = oracle_inputs(c, idx)
    oracle.run(th0, grads, c.W, c.K, c.steps, *h, T=c.T, param_dt=c.param_dt,
               mom_dt="f32", aux_dt="f32", callback=on_step, method=c.method)


class GpuRun:
    """The GPU side of a Case: state in HBM, inputs from the device generator."""

    def __init__(self, c: Case, stream=None):
        from paper_2607_21224_amd.state import CpdpState, Hyper
        self.c = c
        self.stream = stream
        self.st = CpdpState(c.W, c.P, c.ld, c.K, c.param_dt, device="cuda")
        self.h = Hyper(*c.hyper32())
        self.grads = torch.empty((c.W, self.st.ld), dtype=torch.float32,
                                 device="cuda")
        th = torch.empty(max(c.P, 1), dtype=torch.float32, device="cuda")
        sdev.fill_theta0(th, c.P, c.seed, c.theta_sigma, stream=stream)
        if c.param_dt == "bf16":
            th = th.to(torch.bfloat16)
        self.st.init(th, stream=stream)

    def step(self, step: int) -> str:
        c = self.c
        sdev.fill_grads(self.grads, c.P, c.seed, step, c.grad_sigma,
                        c.outlier_rate, stream=self.stream)
        t = ((step - 1) % c.T) + 1 if c.T > 0 else step
        return self.st.step(t, self.grads, self.h, c.T, stream=self.stream,
                            method=c.method)

    def snapshot(self, idx: np.ndarray | None = None):
        torch.cuda.synchronize()
        P = self.c.P
        sl = (slice(None), slice(0, P))
        if idx is None:
            get = lambda x: x[sl] if x.dim() == 2 else x[:P]  # noqa: E731
        else:
            ti = torch.from_numpy(idx).to("cuda")
            get = lambda x: x.index_select(x.dim() - 1, ti)  # noqa: E731
        out = {k: get(getattr(self.st, k)).float().cpu().numpy().astype(np.float64)
               for k in ("params", "mom", "slow_mom", "anchor")}
        return out


def compare(gpu: dict, ref: "oracle.OracleState", param_dt: str, tag: str):
    """Assert the GPU snapshot matches the oracle state within tolerance."""
    pairs = [("params", ref.params), ("mom", ref.mom), ("slow_mom", ref.slow),
             ("anchor", ref.anchor)]
    for name, want in pairs:
        got = gpu[name]
        assert got.shape == want.shape, (tag, name, got.shape, want.shape)
        if param_dt == "f32":
            rtol, atol = RTOL_F32, ATOL_F32
        elif name == "params":
            rtol, atol = RTOL_BF16, ATOL_BF16
        else:
            # fp32 state driven by bf16 replicas: a one-ulp bf16 flip of one
            # replica moves the mean by ulp/W, so scale atol with the data
            rms = float(np.sqrt(np.mean(want[np.isfinite(want)] ** 2))) if want.size else 0.0
            rtol, atol = RTOL_BF16, 1e-2 * rms + 1e-12
        nan_g, nan_w = np.isnan(got), np.isnan(want)
        assert np.array_equal(nan_g, nan_w), f"{tag} {name}: NaN positions differ"
        fin = ~nan_w
        err = np.abs(got[fin] - want[fin])
        lim = atol + rtol * np.abs(want[fin])
        bad = err > lim
        if bad.any():
            k = np.argmax(err - lim)
            raise AssertionError(
                f"{tag} {name}: {int(bad.sum())}/{bad.size} out of tolerance; worst "
                f"got {got[fin][k]!r} want {want[fin][k]!r} (rtol {rtol}, atol {atol})")


def check_replicas_reconciled(gpu: dict, param_dt: str, tag: str):
    """After a reconcile every replica holds exactly the anchor in the
    parameter storage type."""
    p = gpu["params"]
    assert (p == p[0:1]).all() or np.isnan(p).any(), f"{tag}: replicas differ"
    a = gpu["anchor"].astype(np.float32)
    if param_dt == "bf16":
        a = gen.bf16_round(a)
    same = (p[0] == a) | (np.isnan(p[0]) & np.isnan(a))
    assert same.all(), f"{tag}: replicas != storage(anchor)"


def run_parity(c: Case, idx: np.ndarray | None = None, stream=None):
    """Run a Case on both sides and compare after every step."""
    P = c.P
    sel = np.arange(P) if idx is None else idx
    log(f"[parity] {c.method} W={c.W} P={P} K={c.K} steps={c.steps} dt={c.param_dt} "
        f"seed={c.seed} ld={c.ld} coords={sel.size}")
    refs = {}
    run_oracle(c, sel, lambda s, kind, st: refs.__setitem__(s, (kind, st.copy())))
    g = GpuRun(c, stream)
    for s in range(1, c.steps + 1):
        kind = g.step(s)
        snap = g.snapshot(idx)
        rk, ref = refs[s]
        assert kind == rk, (s, kind, rk)
        compare(snap, ref, c.param_dt, f"step {s} ({kind})")
        if kind == "reconcile" and c.method != "ddp":
            check_replicas_reconciled(snap, c.param_dt, f"step {s}")
    log(f"[parity] ok: {c.steps} steps")
    return g
