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


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1023, 1024, 1025, 4097, 8 * 1024 + 4, (1 << 20) + 3])
def test_reference_copy_ragged_sizes(n):
    """The bandwidth-reference copy moves exactly src[:n] into dst[:n] (every
    block and the ragged tail) and leaves the bytes after n untouched."""
    src = torch.arange(n + 64, dtype=torch.float32, device="cuda") + 0.5
    dst = torch.full((n + 64,), -7.0, dtype=torch.float32, device="cuda")
    sdev.copy_f32(dst, src, n)
    torch.cuda.synchronize()
    assert torch.equal(dst[:n], src[:n])
    assert (dst[n:] == -7.0).all()
