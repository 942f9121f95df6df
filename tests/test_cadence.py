"""Host cadence of Sec. 3.2 / Sec. 3.1 against Table 2's counts (CPU only)."""
import math

import pytest

import oracle


@pytest.mark.parametrize("K", range(1, 11))
def test_table2_counts(K):
    # Table 2: CPDP performs ceil(T/K) gradient and ceil(T/K) parameter
    # synchronisations per epoch; K = 1 is DDP's T per epoch.
    for T in range(1, 61):
        syncs = sum(oracle.is_sync_step(t, K, T) for t in range(1, T + 1))
        assert syncs == math.ceil(T / K)
        if K == 1:
            assert syncs == T


@pytest.mark.parametrize("K", range(1, 9))
def test_at_most_k_minus_1_local_steps(K):
    # Sec. 5: up to K - 1 local updates between two synchronisation steps, and
    # the last step of every epoch synchronises (Sec. 3.1).
    for T in range(1, 40):
        run = 0
        for t in range(1, T + 1):
            if oracle.is_sync_step(t, K, T):
                run = 0
            else:
                run += 1
                assert run <= K - 1
        assert oracle.is_sync_step(T, K, T)


def test_no_epoch_boundary():
    assert [oracle.is_sync_step(t, 3) for t in range(1, 8)] == [
        False, False, True, False, False, True, False]


@pytest.mark.parametrize("bad", [(0, 2, 0), (1, 0, 0), (5, 2, 4), (1, 2, -1)])
def test_invalid(bad):
    with pytest.raises(ValueError):
        oracle.is_sync_step(*bad)


@pytest.mark.parametrize("K", [2, 3, 4, 8])
def test_warmup_then_table2_counts(K):
    # Sec. 3.4: Table 2's counts apply after warmup; during warmup CPDP and
    # LocalSGD synchronise every step.
    T, warm = 13, 2
    for epoch in range(5):
        k = oracle.period_for_epoch(epoch, warm, K)
        syncs = sum(oracle.is_sync_step(t, k, T) for t in range(1, T + 1))
        assert syncs == (T if epoch < warm else math.ceil(T / K))


def test_lr_schedule_shape():
    base, low, total, warm = 0.4, 0.001, 110, 10
    lrs = [oracle.lr_at(s, total, warm, base, low) for s in range(total)]
    assert lrs[0] == pytest.approx(base / warm)
    assert lrs[warm - 1] == pytest.approx(base)
    assert lrs[warm] == pytest.approx(base)            # cosine starts at base
    assert lrs[warm + 50] == pytest.approx((base + low) / 2)
    assert all(a > b for a, b in zip(lrs[warm:], lrs[warm + 1:]))   # decreasing
    assert all(a < b for a, b in zip(lrs[:warm - 1], lrs[1:warm]))  # increasing
    assert low < lrs[-1] < low + 1e-3
    with pytest.raises(ValueError):
        oracle.lr_at(total, total, warm, base, low)


def test_linear_lr_scaling_reproduces_table4():
    """The linear scaling rule gives the learning rates Table 4 prints for
    every intra-site configuration (64 per GPU, 0.1 at a global batch of 256)."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                    "table4_lr_scaling.json")))
    for row in g["rows"]:
        assert row["global_batch"] == 64 * row["gpus"]
        got = oracle.linear_scaled_lr(g["base_lr"], g["base_batch"], row["global_batch"])
        assert abs(got - row["lr"]) < 1e-12, row
    with pytest.raises(ValueError):
        oracle.linear_scaled_lr(0.0, 256, 512)
    with pytest.raises(ValueError):
        oracle.linear_scaled_lr(0.1, 0, 512)
