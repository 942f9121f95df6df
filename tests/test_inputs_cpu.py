"""CPU pins of the synthetic inputs: the seeded generator against the published
SplitMix64 sequence and the statistics its definition fixes, and the workload
tensor layouts against an independent implementation of the two model
architectures (Hugging Face ``transformers``, built from configs offline, no
weights); and the parity harness's host-side check of sampled coordinates."""
import numpy as np
import pytest

from synth import WORKLOADS, gen
from synth.workloads import resnet50_tensors, vit_s_tensors

# First three outputs of SplitMix64 started from state 0 (Steele, Lea, Flood,
# OOPSLA 2014; the reference generator's published sequence).
SPLITMIX64_FROM_ZERO = (0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F)


def test_mix64_reproduces_splitmix64_sequence():
    for n, want in enumerate(SPLITMIX64_FROM_ZERO, 1):
        assert gen.mix64_int(n * gen.GAMMA) == want


def test_vectorised_mix64_equals_scalar():
    rng = np.random.default_rng(7)
    z = rng.integers(0, 2 ** 63, size=257, dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    with np.errstate(over="ignore"):
        got = gen._mix64(z)
    assert [int(x) for x in got] == [gen.mix64_int(int(x)) for x in z]


def test_normal_draw_is_the_stated_irwin_hall_sum():
    """Recompute one coordinate's draw from the definition with Python ints."""
    key = gen.stream_key(123, gen.KIND_GRAD, 3, 5)
    for p in (0, 1, 4097, 10 ** 8 - 1):
        s = 0
        for j in range(3):
            h = gen.mix64_int(key + (4 * p + j + 1) * gen.GAMMA)
            s += sum((h >> (16 * f)) & 0xFFFF for f in range(4))
        z = np.float32((s - 393210) * 2.0 ** -16)
        want = np.float32(z * np.float32(1e-3))
        got = gen.grads(123, 3, 6, np.array([p]), 1e-3)[5, 0]
        assert got.view(np.uint32) == want.view(np.uint32)


def test_normal_moments_and_range():
    n = 1 << 20
    for sigma in (0.02, 1e-3):
        v = gen.theta0(42, np.arange(n), sigma).astype(np.float64)
        assert abs(v.mean()) < 5 * sigma / np.sqrt(n)
        assert abs(v.std() / sigma - 1.0) < 0.01
        assert np.abs(v).max() <= 6 * sigma * (1 + 1e-6)
        # z is a multiple of 2^-16 and the value is one fp32 multiply of it:
        # the nearest grid point reproduces every draw bit for bit
        zg = (np.round(v / np.float32(sigma) * 65536) / 65536).astype(np.float32)
        again = (zg * np.float32(sigma)).astype(np.float32)
        assert np.array_equal(again, v.astype(np.float32))


def test_outlier_rate_and_scale():
    n = 1 << 20
    idx = np.arange(n)
    plain = gen.grads(42, 1, 2, idx, 1e-3)
    out = gen.grads(42, 1, 2, idx, 1e-3, outlier_rate=0.01)
    nz = plain != 0
    ratio = out[nz] / plain[nz]
    hit = np.isclose(ratio, 100.0, rtol=1e-6)
    assert np.all(hit | (ratio == 1.0))
    assert abs(hit.mean() - 0.01) < 0.001
    # outliers are exactly fp32(value * 100)
    assert np.array_equal(out[nz][hit], (plain[nz][hit] * np.float32(100.0)).astype(np.float32))


def test_streams_are_deterministic_and_distinct():
    idx = np.arange(4096)
    a = gen.grads(42, 2, 4, idx)
    assert np.array_equal(a.view(np.uint32), gen.grads(42, 2, 4, idx).view(np.uint32))
    others = [gen.grads(43, 2, 4, idx), gen.grads(42, 3, 4, idx), gen.theta0(42, idx)[None]]
    for o in others:
        assert np.mean(o[0] == a[0]) < 0.01
    # replicas draw independent streams
    assert abs(np.corrcoef(a[0], a[1])[0, 1]) < 0.05


def _transformers():
    return pytest.importorskip("transformers")


@pytest.mark.parametrize("classes,name", [(1000, None), (100, "r50_100"), (200, "r50_200")])
def test_resnet50_layout_matches_transformers(classes, name):
    tf = _transformers()
    m = tf.ResNetForImageClassification(tf.ResNetConfig(num_labels=classes))
    theirs = sorted(p.numel() for p in m.parameters())
    ours = sorted(n for _, n in resnet50_tensors(classes))
    assert ours == theirs
    if classes == 1000:
        assert sum(ours) == 25_557_032  # the published ResNet-50 parameter count
    else:
        assert WORKLOADS[name].P == sum(ours)
        assert list(WORKLOADS[name].tensors) == resnet50_tensors(classes)


def test_vit_s_layout_matches_transformers():
    tf = _transformers()
    cfg = tf.ViTConfig(hidden_size=384, num_hidden_layers=12, num_attention_heads=6,
                       intermediate_size=1536, num_labels=100)
    m = tf.ViTForImageClassification(cfg)
    blocks, head = {}, 0
    for n, p in m.named_parameters():
        parts = n.split(".")
        if "layers" in parts or "layer" in parts:
            k = parts.index("layers") if "layers" in parts else parts.index("layer")
            blocks[int(parts[k + 1])] = blocks.get(int(parts[k + 1]), 0) + p.numel()
        elif parts[0] == "classifier":
            head += p.numel()
    ours = vit_s_tensors(100)
    per_block = sum(n for t, n in ours if t.startswith("blocks.0."))
    assert sorted(blocks) == list(range(12))
    assert set(blocks.values()) == {per_block}
    assert sum(n for t, n in ours if t.startswith("head.")) == head
    assert WORKLOADS["vit_s"].P == 12 * per_block + head == sum(n for _, n in ours)


def test_parity_sample_outside_the_state_is_rejected_on_the_host():
    """A sampled coordinate at or past P is refused before any device work:
    u and the anchor have no padding, so torch's gather would hit its
    device-side bounds assertion (a GPU trap) on it."""
    import pytest
    from gpu_harness import Case, check_sample, run_parity
    c = Case(W=1, P=10, K=2, lr=0.1, mu=0.9, beta=0.5, alpha=1.0, steps=2)
    for bad in ([0, 9, 10], [-1, 3]):
        with pytest.raises(ValueError, match="outside"):
            run_parity(c, np.array(bad))
    check_sample(np.array([0, 9]), 10)
