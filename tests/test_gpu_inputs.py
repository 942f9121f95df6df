"""The device input generator agrees bit for bit with the host generator."""
import numpy as np
import pytest
import torch

from synth import device as sdev
from synth import gen

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("outliers", [0.0, 0.01])
def test_generator_bitwise(outliers):
    W, P, ld = 3, 1_000_003, 1_000_064
    buf = torch.full((W, ld), -7.0, dtype=torch.float32, device="cuda")
    sdev.fill_grads(buf, P, 777, 5, 1e-3, outliers)
    rng = np.random.default_rng(4)
    idx = np.unique(np.concatenate([np.arange(100), np.arange(P - 100, P),
                                    rng.integers(0, P, 50_000)]))
    want = gen.grads(777, 5, W, idx, 1e-3, outliers)
    got = buf[:, torch.from_numpy(idx).cuda()].cpu().numpy()
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    assert (buf[:, P:] == -7.0).all()


def test_theta0_and_bf16_rounding():
    P = 300_001
    th = torch.empty(P, dtype=torch.float32, device="cuda")
    sdev.fill_theta0(th, P, 42)
    want = gen.theta0(42, np.arange(P))
    assert np.array_equal(th.cpu().numpy(), want)
    bf = th.to(torch.bfloat16).float().cpu().numpy()
    assert np.array_equal(bf, gen.bf16_round(want))
