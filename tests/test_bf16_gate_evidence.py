"""Why the bf16 gate has a loose tier: a correct fp32 computation in the
kernels' operation order can leave the fp64 oracle by more than two bf16
flips' worth on a rare coordinate.

tests/kernel_rendition.py models the library's momentum-SGD steps in fp32
(exact fused multiply-adds, bf16 round-to-nearest-even, the kernels' order of
operations); test_gpu_rendition.py checks that the library equals it bit for
bit.  Here, on the CPU, the rendition and the oracle run the stress workload
(32 bf16 replicas, fp32 momentum / u / anchor, lr 0.1, mu 0.9, beta 0.5,
K = 4, seed 42) over its full 12 steps on a window of coordinates around
54,970,965.  A search of the 2M coordinates [54525952, 56623104) with the same
two programs (run_window over the whole range) finds that coordinate as the
only one whose u leaves the tight tier: after the second reconcile the
rendition's u is 1.22 times the two-flip allowance away from the oracle's,
and within the loose tier of four flips, until the third reconcile brings it
back inside the tight tier.  The GPU's u there is the
rendition's (test_gpu_rendition.py), so the gap is rounding order, not a
defect."""
import numpy as np

import oracle
from gpu_harness import BF16_LOOSE_FACTOR, compare
from kernel_rendition import Rendition
from synth import WORKLOADS, gen

STRESS = WORKLOADS["stress"]
COORD = 54_970_965
WINDOW = np.arange(COORD - 40, COORD + 24, dtype=np.int64)


def run_window(idx, seed=42, steps=None):
    """The stress workload on coordinates idx through the oracle and the
    rendition; yields (step, kind, oracle state, rendition snapshot)."""
    w = STRESS
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    lr, mu, beta, alpha = f32(w.lr), f32(w.mu), f32(w.beta), f32(w.alpha)
    th0 = gen.bf16_round(gen.theta0(seed, idx, w.theta_sigma))
    R = Rendition(th0, w.W)
    st = oracle.state_init(th0.astype(np.float64), w.W, "bf16")
    for s in range(1, (steps or w.steps) + 1):
        g = gen.grads(seed, s, w.W, idx, w.grad_sigma, w.outlier_rate)
        if oracle.is_sync_step(s, w.K):
            oracle.reconcile(st, g.astype(np.float64), lr, mu, beta, alpha)
            R.reconcile(g, lr, mu, beta, alpha)
            kind = "reconcile"
        else:
            oracle.local_step(st, g.astype(np.float64), lr, mu)
            R.local_step(g, lr, mu)
            kind = "local"
        yield s, kind, st, R.snapshot()


def _u_tiers(st, lr, W):
    """The harness's tight (two-flip) limit on u for every coordinate, and
    its loose one."""
    fa = st.anchor[np.isfinite(st.anchor)]
    a_rms = float(np.sqrt(np.mean(fa ** 2)))
    flip = (2.0 / W) * 2.0 ** -7 * np.maximum(np.abs(st.anchor), a_rms) / lr
    u_rms = float(np.sqrt(np.mean(st.slow ** 2)))
    tight = 1e-2 * u_rms + 1e-12 + flip + 1e-2 * np.abs(st.slow)
    return tight, tight + (BF16_LOOSE_FACTOR - 1.0) * flip


def test_rendition_leaves_tight_tier_only_where_the_search_found():
    lr = float(np.float32(STRESS.lr))
    j = int(np.nonzero(WINDOW == COORD)[0][0])
    seen = False
    for s, kind, st, snap in run_window(WINDOW):
        tight, loose = _u_tiers(st, lr, STRESS.W)
        err = np.abs(snap["slow_mom"] - st.slow)
        # every coordinate of the window stays inside the loose tier ...
        assert (err <= loose).all(), f"step {s}: u beyond the loose tier"
        # ... and the tight tier holds everywhere except at COORD from the
        # second reconcile (step 8) until the third (step 12) pulls u back
        others = np.delete(err / tight, j)
        assert (others <= 1).all(), f"step {s}: another coordinate leaves the tight tier"
        if 8 <= s < 12:
            seen = True
            assert err[j] / tight[j] > 1.0, f"step {s}: expected the tight tier to fail here"
            assert err[j] / loose[j] < 0.2
        else:
            assert err[j] <= tight[j]
        # the other families stay within the stated gates (fp32 momentum at the
        # fp32 tolerance: it never reads a parameter)
        rest = {k: v for k, v in snap.items() if k != "slow_mom"}
        rest["slow_mom"] = st.slow.copy()
        compare(rest, st, "bf16", f"rendition step {s} ({kind})", lr=lr, fp32_state=True)
    assert seen


# A second mechanism, located by the whole stress run's report of tight-tier
# exceptions at seed 777 (the location only; every value below is computed
# here).  At the first reconcile one replica's x_i lands one bf16 ulp away
# from the oracle's, which moves the rendition's anchor by about ulp / W; the
# oracle's anchor lies exactly on the bf16 rounding boundary between 2^-7 and
# the next bf16 value, so the two copy-backs round to different sides and all
# 32 replicas differ by one bf16 ulp ("broadcast flip": W flips at once).  The
# next reconcile's mean then moves by a whole ulp: u leaves the tight tier by
# almost 5x and stays at a third of the loose one (after the third reconcile
# 2.3x and a sixth), and replica 16's parameter leaves it at steps 10-11 (two
# ulps at the binade boundary).
COORD_777 = 53_890_736
WINDOW_777 = np.arange(COORD_777 - 40, COORD_777 + 24, dtype=np.int64)


def _p_tiers(st, W):
    """The harness's tight and loose limits on the bf16 parameters."""
    from gpu_harness import ATOL_BF16, RTOL_BF16
    fa = st.anchor[np.isfinite(st.anchor)]
    a_rms = float(np.sqrt(np.mean(fa ** 2)))
    flip = (2.0 / W) * 2.0 ** -7 * np.maximum(np.abs(st.anchor), a_rms)[None, :]
    tight = ATOL_BF16 + flip + RTOL_BF16 * np.abs(st.params)
    return tight, tight + (BF16_LOOSE_FACTOR - 1.0) * flip


def test_broadcast_flip_stays_inside_the_loose_tier():
    lr = float(np.float32(STRESS.lr))
    W = STRESS.W
    j = int(np.nonzero(WINDOW_777 == COORD_777)[0][0])
    for s, kind, st, snap in run_window(WINDOW_777, seed=777):
        if s == 4:
            ulp = np.spacing(np.float32(np.abs(st.params[0, j]))) * 2.0 ** 16  # bf16 spacing
            assert 0 < abs(snap["anchor"][j] - st.anchor[j]) < ulp / W
            d = snap["params"][:, j] - st.params[:, j]
            assert (np.abs(d) == ulp).all(), "every replica one bf16 ulp away"
        tight, loose = _u_tiers(st, lr, W)
        err_u = np.abs(snap["slow_mom"] - st.slow)
        assert (err_u <= loose).all(), f"step {s}: u beyond the loose tier"
        if 8 <= s < 12:  # the second reconcile's mean carries the whole-ulp shift
            assert 4 < err_u[j] / tight[j] and err_u[j] / loose[j] < 0.35, s
        elif s == 12:    # the third reconcile halves it, still outside the tight tier
            assert 1 < err_u[j] / tight[j] and err_u[j] / loose[j] < 0.2, s
        pt, pl = _p_tiers(st, W)
        err_p = np.abs(snap["params"] - st.params)
        assert (err_p <= pl).all(), f"step {s}: parameters beyond the loose tier"
        over = err_p > pt
        if s in (10, 11):
            assert over[16, j] and over.sum() == 1, s
        else:
            assert not over.any(), s
