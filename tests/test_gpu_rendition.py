"""The library's momentum-SGD local step and CPDP reconcile equal, bit for
bit, the fp32 rendition of their operation order (tests/kernel_rendition.py),
on the stress window where that rendition leaves the oracle's tight bf16 tier
(test_bf16_gate_evidence.py) and on fp32 parameters.  So the GPU's distance
from the fp64 oracle there is the rounding order the rendition spells out.
Inputs are the seeded generator's values for the window's global coordinates,
made on the host and copied to the device."""
import numpy as np
import pytest
import torch

from gpu_harness import log
from kernel_rendition import Rendition
from synth import WORKLOADS, gen

pytestmark = pytest.mark.gpu

STRESS = WORKLOADS["stress"]
COORD = 54_970_965       # u leaves the tight tier (seed 42)
COORD_777 = 53_890_736   # a broadcast flip (seed 777)


@pytest.mark.parametrize("param_dt,W,lo,n,seed", [
    ("bf16", 32, COORD - 2000, 4096 + 3, 42),      # the stress windows, ragged tail
    ("bf16", 32, COORD_777 - 1000, 2048 + 1, 777),
    ("f32", 8, 1_000_000, 3 * 1024 + 5, 42),       # fp32 replicas, r50_100's W
])
def test_library_equals_fp32_rendition(param_dt, W, lo, n, seed):
    from paper_2607_21224_amd.state import CpdpState, Hyper
    w = STRESS
    idx = np.arange(lo, lo + n, dtype=np.int64)
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    lr, mu, beta, alpha = f32(w.lr), f32(w.mu), f32(w.beta), f32(w.alpha)
    th0 = gen.theta0(seed, idx, w.theta_sigma)
    if param_dt == "bf16":
        th0 = gen.bf16_round(th0)
    log(f"[rendition] {param_dt} W={W} coordinates [{lo}, {lo + n}) seed {seed} "
        f"steps={w.steps}")
    R = Rendition(th0, W, param_dt)
    st = CpdpState(W, n, K=w.K, param_dt=param_dt, device="cuda")
    tdt = torch.bfloat16 if param_dt == "bf16" else torch.float32
    st.init(torch.from_numpy(th0).to("cuda").to(tdt))
    grads = torch.zeros((W, st.ld), dtype=torch.float32, device="cuda")
    h = Hyper(lr, mu, beta, alpha)
    for s in range(1, w.steps + 1):
        g = gen.grads(seed, s, W, idx, w.grad_sigma, w.outlier_rate)
        grads[:, :n].copy_(torch.from_numpy(g))
        kind = st.step(s, grads, h)
        if kind == "reconcile":
            R.reconcile(g, lr, mu, beta, alpha)
        else:
            R.local_step(g, lr, mu)
        torch.cuda.synchronize()
        got = {"params": st.params[:, :n].float().cpu().numpy(),
               "mom": st.mom[:, :n].cpu().numpy(),
               "slow_mom": st.slow_mom[:n].cpu().numpy(),
               "anchor": st.anchor[:n].cpu().numpy()}
        want = R.snapshot()
        for k, v in got.items():
            same = v.view(np.uint32) == want[k].astype(np.float32).view(np.uint32)
            assert same.all(), (f"step {s} ({kind}) {k}: {int((~same).sum())} values differ "
                                f"from the rendition")
