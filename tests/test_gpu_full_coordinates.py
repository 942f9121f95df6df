"""Every coordinate of the four full-size workloads for one whole period (K-1
local steps and the reconcile) against the oracle, after every step, in the
benchmark's launch configuration (longer runs on request, below):
  r50_100  ResNet-50/CIFAR-100-sized, W=8, P=23,712,932 in 161 tensors, K=4
  vit_s    ViT-S-sized, W=8, P=21,332,068, K=4
  r50_200  ResNet-50/TinyImageNet-sized, W=16, P=23,917,832, K=8, gradients
           with 1 % outliers x100
  stress   W=32 bf16 replicas, P=10^8, fp32 gradients, momentum, u, anchor, K=4
and vit_s once more with AdamW, the optimizer the paper trains ViT-S with
(Table 3: lr 5e-4, betas 0.9 / 0.999, eps 1e-8, decoupled weight decay 0.05),
second moments included, r50_100 with the paper's ResNet optimizer (momentum
SGD with weight decay 5e-4, Table 3) through the general-optimizer path, and
r50_100 under the paper's two baselines (Sec. 5.3): the LocalSGD sync and the
synchronous DDP step.

Inputs come from the seeded generator: on the device for the HIP path, copied
to the host for the oracle (the generator is the one module both sides share;
a sample of each copy is re-derived here with the host generator, bit for
bit).  Nothing the HIP path computes feeds the oracle.

The fp64 oracle state of all coordinates would take up to about 50 GB of host
memory (stress), so between steps the oracle's state is kept in the storage
types it rounds to at every store (fp32 or bf16 parameters, fp32 momentum, u
and anchor).  That is lossless, and every store-back asserts it.  Coordinates
are independent, so slices of 2^21 coordinates are stepped in a thread pool
(the oracle's C calls and numpy release the GIL), each compared with the same
slice of the GPU state after every step.

By default each workload runs one period at seed 42.  Environment variables
widen the run (a whole configured run takes several minutes per workload):
  CPDP_FULL_PERIODS=all   the workload's configured number of periods
  CPDP_FULL_SEEDS=42,123,777   the seeds to run (comma-separated)
  CPDP_FULL_VARIANTS=1    also the stress state's other storage readings:
                          bf16 gradients, and bf16 gradients and momentum"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from gpu_harness import (Case, GpuRun, check_replicas_reconciled, compare, log,
                         state_from_grads, tolerance_regime)
from synth import WORKLOADS, gen
from synth import device as sdev

pytestmark = pytest.mark.gpu

SLICE = 1 << 21
WORKERS = 12

WHOLE_RUN = os.environ.get("CPDP_FULL_PERIODS", "1") == "all"
SEEDS = [int(x) for x in os.environ.get("CPDP_FULL_SEEDS", "42").split(",") if x]
ADAMW = dict(kind="adamw", lr=5e-4, momentum=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05)
SGD_WD = dict(kind="sgd", lr=0.1, momentum=0.9, weight_decay=5e-4)
# (workload, gradient storage, momentum storage, general optimizer, strategy)
CASES = [("r50_100", "f32", "f32", None, "cpdp"), ("vit_s", "f32", "f32", None, "cpdp"),
         ("r50_200", "f32", "f32", None, "cpdp"), ("stress", "f32", "f32", None, "cpdp"),
         ("vit_s", "f32", "f32", ADAMW, "cpdp"), ("r50_100", "f32", "f32", SGD_WD, "cpdp"),
         ("r50_100", "f32", "f32", None, "localsgd"),
         ("r50_100", "f32", "f32", None, "ddp")]
if os.environ.get("CPDP_FULL_VARIANTS") == "1":
    CASES += [("stress", "bf16", "f32", None, "cpdp"), ("stress", "bf16", "bf16", None, "cpdp")]


def _case_id(case) -> str:
    name, g, m, opt, method = case
    if method != "cpdp":
        return f"{name}-{method}"
    if opt is not None:
        return f"{name}-{'adamw' if opt['kind'] == 'adamw' else 'sgd_wd'}"
    return f"{name}-grads_{g}-mom_{m}"


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


class CompactState:
    """The oracle state of all coordinates in its storage types."""

    def __init__(self, W: int, P: int, param_dt: str, mom_dt: str = "f32", adamw: bool = False):
        self.W, self.param_dt, self.mom_dt = W, param_dt, mom_dt
        self.params = np.empty((W, P), dtype=np.uint16 if param_dt == "bf16" else np.float32)
        self.mom = np.empty((W, P), dtype=np.uint16 if mom_dt == "bf16" else np.float32)
        self.slow = np.empty(P, dtype=np.float32)
        self.anchor = np.empty(P, dtype=np.float32)
        # AdamW's second moments (fp32 storage), kept beside the oracle state
        self.mom2 = np.zeros((W, P), dtype=np.float32) if adamw else None

    def load_mom2(self, lo: int, hi: int) -> np.ndarray:
        return self.mom2[:, lo:hi].astype(np.float64)

    def store_mom2(self, m2: np.ndarray, lo: int, hi: int) -> None:
        self.mom2[:, lo:hi] = _exact_f32(m2)

    def load(self, lo: int, hi: int) -> oracle.OracleState:
        p = self.params[:, lo:hi]
        params = _from_bits(p) if self.param_dt == "bf16" else p.astype(np.float64)
        m = self.mom[:, lo:hi]
        mom = _from_bits(m) if self.mom_dt == "bf16" else m.astype(np.float64)
        return oracle.OracleState(self.W, hi - lo, params, mom,
                                  self.slow[lo:hi].astype(np.float64),
                                  self.anchor[lo:hi].astype(np.float64), self.param_dt,
                                  self.mom_dt, "f32")

    def store(self, st: oracle.OracleState, lo: int, hi: int) -> None:
        self.params[:, lo:hi] = (_bf16_bits(st.params) if self.param_dt == "bf16"
                                 else _exact_f32(st.params))
        self.mom[:, lo:hi] = (_bf16_bits(st.mom) if self.mom_dt == "bf16"
                              else _exact_f32(st.mom))
        self.slow[lo:hi] = _exact_f32(st.slow)
        self.anchor[lo:hi] = _exact_f32(st.anchor)


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("name,gdt,mdt,opt,method", CASES, ids=[_case_id(x) for x in CASES])
def test_every_coordinate(name, gdt, mdt, opt, method, seed):
    w = WORKLOADS[name]
    c = Case(W=w.W, P=w.P, K=w.K, lr=w.lr, mu=w.mu, beta=w.beta, alpha=w.alpha,
             steps=w.steps if WHOLE_RUN else w.K, param_dt=w.param_dt, ld=w.ld, seed=seed,
             theta_sigma=w.theta_sigma, grad_sigma=w.grad_sigma,
             outlier_rate=w.outlier_rate, grad_dt=gdt, mom_dt=mdt, opt=opt, method=method)
    P, W = c.P, c.W
    lr, mu, beta, alpha = c.hyper32()
    o = c.opt32() if opt is not None else None
    # the oracle's optimizer of 1-based global step s (AdamW's step count
    # advances on every step), with the fp32 values of the hyperparameters
    make_opt = None
    if o is not None and o["kind"] == "adamw":
        make_opt = lambda s: oracle.adamw(o["lr"], o["momentum"], o["beta2"], o["eps"],  # noqa: E731
                                          o["weight_decay"], s)
    elif o is not None:
        make_opt = lambda s: oracle.sgd(o["lr"], o["momentum"], o["weight_decay"])  # noqa: E731
    adamw = o is not None and o["kind"] == "adamw"
    rng = np.random.default_rng(0)
    sample = np.unique(np.concatenate([np.arange(64), P - 64 + np.arange(64),
                                       rng.integers(0, P, 4096)]))

    th = torch.empty(P, dtype=torch.float32, device="cuda")
    sdev.fill_theta0(th, P, c.seed, c.theta_sigma)
    th0 = th.cpu().numpy()
    del th
    assert np.array_equal(th0[sample].view(np.uint32),
                          gen.theta0(c.seed, sample, c.theta_sigma).view(np.uint32))

    slices = [(lo, min(P, lo + SLICE)) for lo in range(0, P, SLICE)]
    ref = CompactState(W, P, c.param_dt, c.mom_dt, adamw=adamw)
    oracle.lib()  # load once before the worker threads call into it

    def init(sl):
        lo, hi = sl
        ref.store(oracle.state_init(th0[lo:hi].astype(np.float64), W, c.param_dt, c.mom_dt),
                  lo, hi)

    g = GpuRun(c)
    with ThreadPoolExecutor(WORKERS) as pool:
        list(pool.map(init, slices))
        for s in range(1, c.steps + 1):
            kind = g.step(s)  # fills g.grads with step s's gradients, then steps
            torch.cuda.synchronize()
            got = g.grads[:, sample].cpu().numpy()
            assert np.array_equal(got.view(np.uint32),
                                  gen.grads(c.seed, s, W, sample, c.grad_sigma,
                                            c.outlier_rate).view(np.uint32))
            if c.grad_dt == "bf16":  # the rows the library read: RNE of the generated values
                gb = g.grads_bf16[:, sample].float().cpu().numpy()
                assert np.array_equal(gb.view(np.uint32), gen.bf16_round(got).view(np.uint32))

            def work(sl, s=s, kind=kind):
                lo, hi = sl
                g32 = g.grads[:, lo:hi].cpu().numpy()
                if c.grad_dt == "bf16":  # the oracle steps on the stored bf16 values
                    g32 = gen.bf16_round(g32)
                g64 = g32.astype(np.float64)
                del g32
                st = ref.load(lo, hi)
                m2 = None
                if make_opt is not None:
                    m2 = ref.load_mom2(lo, hi) if adamw else None
                    if kind == "reconcile":
                        oracle.sync_opt(st, "cpdp", g64, make_opt(s), beta, alpha, m2)
                    else:
                        oracle.local_step_opt(st, g64, make_opt(s), m2)
                    if adamw:
                        ref.store_mom2(m2, lo, hi)
                elif kind == "reconcile" and method == "localsgd":
                    oracle.localsgd_sync(st, g64, lr, mu)
                elif kind == "reconcile" and method == "ddp":
                    oracle.ddp_step(st, g64, lr, mu)
                elif kind == "reconcile":
                    oracle.reconcile(st, g64, lr, mu, beta, alpha)
                else:
                    oracle.local_step(st, g64, lr, mu)
                del g64
                ref.store(st, lo, hi)
                snap = {"params": g.st.params[:, lo:hi].float().cpu().numpy().astype(np.float64),
                        "mom": g.st.mom[:, lo:hi].float().cpu().numpy().astype(np.float64),
                        "slow_mom": g.st.slow_mom[lo:hi].cpu().numpy().astype(np.float64),
                        "anchor": g.st.anchor[lo:hi].cpu().numpy().astype(np.float64)}
                if m2 is not None:
                    snap["mom2"] = g.st.mom2[:, lo:hi].cpu().numpy().astype(np.float64)
                tag = (f"{name} {method} grads {c.grad_dt} mom {c.mom_dt} seed {c.seed} every coordinate, "
                       f"step {s} ({kind}), coordinates [{lo}, {hi})")
                exc = []
                if o is not None:  # as run_parity gates the general optimizers
                    m = compare(snap, st, tolerance_regime(c), tag, mom2=m2, scaled=True,
                                velocity_lr=o["lr"] if adamw else None, lr=o["lr"],
                                fp32_state=state_from_grads(c.opt, c.mom_dt), exceptions=exc)
                else:
                    m = compare(snap, st, tolerance_regime(c), tag, lr=lr,
                                fp32_state=state_from_grads(None, c.mom_dt), exceptions=exc)
                for fam, row, col, got_v, want_v, r_tight, r_loose in exc:
                    log(f"[full-coords] {name} seed {c.seed} step {s}: tight-tier exception "
                        f"{fam} replica {row} coordinate {lo + col}: got {got_v!r} want "
                        f"{want_v!r} ({r_tight:.3f} of the tight limit, {r_loose:.3f} of the "
                        f"loose one)")
                if kind == "reconcile" and method == "ddp":
                    # identical replicas stepped with the same mean gradient stay identical
                    p = snap["params"]
                    assert (p == p[0:1]).all(), f"{tag}: DDP replicas differ"
                elif kind == "reconcile":
                    check_replicas_reconciled(snap, c.param_dt, tag)
                return m

            worst = {}
            for m in pool.map(work, slices):
                for k, v in m.items():
                    worst[k] = max(worst.get(k, 0.0), v)
            log(f"[full-coords] {name} {method} {o['kind'] if o is not None else 'sgd'}"
                f"{'+wd' if o is not None and o['kind'] == 'sgd' else ''} grads {c.grad_dt} "
                f"mom {c.mom_dt} seed {c.seed} step {s} "
                f"{kind}: {W}x{P} coordinates match; worst "
                f"error / tolerance " + ", ".join(f"{k} {v:.3g}" for k, v in worst.items()))
    assert kind == "reconcile"
