"""Pins for the CPDP oracle: checks against things other than the oracle itself.

Each ``pin_*`` function takes ``use`` (a loaded oracle library, or None for the
default build) and raises AssertionError when the oracle disagrees with what
the paper or the mathematics fixes.  ``tests/test_oracle_pins.py`` runs them on
the real oracle; ``tests/test_oracle_mutants.py`` runs them on copies of the
oracle with planted mistakes and requires every mistake to be caught.
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import oracle
from brute_cpdp import run_exact

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _close(a, b, rtol, atol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    ok = np.abs(a - b) <= atol + rtol * np.abs(b)
    assert ok.all(), f"{what}: got {a[~ok][:4]} want {b[~ok][:4]}"


def pin_worked_example(use=None):
    """Hand-derived trajectory of Algorithm 1 (tests/golden), exact arithmetic."""
    fx = json.load(open(os.path.join(GOLDEN, "worked_example_w2_k2.json")))
    s = fx["setup"]
    grads = [np.array(g, dtype=np.float64) for g in fx["grads"]]
    snaps = {}

    def cb(step, kind, st):
        snaps[step] = (kind, st.copy())

    oracle.run(s["theta0"], lambda step, W, P: grads[step - 1], s["W"], s["K"],
               len(grads), s["lr"], s["mu"], s["beta"], s["alpha"],
               param_dt="f64", mom_dt="f64", aux_dt="f64", callback=cb, use=use)
    for e in fx["expected"]:
        kind, st = snaps[e["step"]]
        assert kind == e["kind"], (e["step"], kind)
        _close(st.mom[:, 0], e["mom"], 1e-12, 1e-12, f"mom step {e['step']}")
        _close(st.params[:, 0], e["params"], 1e-12, 1e-12,
               f"params step {e['step']}")
        _close(st.slow[0], e["u"], 1e-12, 1e-12, f"u step {e['step']}")
        _close(st.anchor[0], e["anchor"], 1e-12, 1e-12,
               f"anchor step {e['step']}")


def pin_worked_example_vform(use=None):
    """Same example through the paper's v variables (Sec. 3.3)."""
    fx = json.load(open(os.path.join(GOLDEN, "worked_example_w2_k2.json")))
    s = fx["setup"]
    st = oracle.state_init(s["theta0"], s["W"], "f64", "f64", "f64", use=use)
    for e, g in zip(fx["expected"], fx["grads"]):
        g = np.array(g, dtype=np.float64)
        if e["kind"] == "local":
            oracle.local_step(st, g, s["lr"], s["mu"])
        else:
            oracle.reconcile_vform(st, g, s["lr"], s["mu"], s["beta"])
        _close(st.slow[0], e["v"], 1e-12, 1e-12, f"v step {e['step']}")
        _close(st.anchor[0], e["anchor"], 1e-12, 1e-12,
               f"vform anchor step {e['step']}")
        _close(st.params[:, 0], e["params"], 1e-12, 1e-12,
               f"vform params step {e['step']}")


def _rand_dyadic(rng, shape, scale=8):
    return rng.integers(-4 * scale, 4 * scale + 1, size=shape) / scale


def pin_brute_force(use=None, cases=12, seed=5, methods=("cpdp",)):
    """Exact rational Algorithm 1 (tests/brute_cpdp.py) on tiny random inputs."""
    rng = np.random.default_rng(seed)
    for c in range(cases):
        W = int(rng.integers(1, 6))
        P = int(rng.integers(1, 9))
        K = int(rng.integers(1, 5))
        T = int(rng.choice([0, 0, 5, 7]))
        n = int(rng.integers(K, 3 * K + 3))
        lr = float(rng.choice([0.125, 0.25, 0.1, 0.05]))
        mu = float(rng.choice([0.0, 0.5, 0.9, 0.75]))
        beta = float(rng.choice([0.0, 0.5, 0.3, 0.875]))
        alpha = float(rng.choice([1.0, 1.0, 0.5, 1.5]))
        method = methods[c % len(methods)]
        theta0 = _rand_dyadic(rng, P)
        grads = [_rand_dyadic(rng, (W, P)) for _ in range(n)]
        exact = run_exact([Fraction(x) for x in theta0],
                          [[[Fraction(x) for x in r] for r in g] for g in grads],
                          W, K, Fraction(lr), Fraction(mu), Fraction(beta),
                          Fraction(alpha), T=T, method=method)
        snaps = []
        oracle.run(theta0, lambda step, W_, P_: grads[step - 1], W, K, n, lr,
                   mu, beta, alpha, T=T, param_dt="f64", mom_dt="f64",
                   aux_dt="f64", use=use, method=method,
                   callback=lambda step, kind, st: snaps.append((kind, st.copy())))
        for s, ((kind, st), ex) in enumerate(zip(snaps, exact)):
            tag = f"case {c} {method} step {s + 1} (W={W} P={P} K={K} T={T})"
            assert kind == ex["kind"], tag
            _close(st.params, [[float(x) for x in r] for r in ex["params"]],
                   1e-12, 1e-12, tag + " params")
            _close(st.mom, [[float(x) for x in r] for r in ex["mom"]], 1e-12,
                   1e-12, tag + " mom")
            _close(st.anchor, [float(x) for x in ex["ref"]], 1e-12, 1e-12,
                   tag + " anchor")
            # u-form state: v = -lr * u  (alpha does not enter v's recursion)
            _close(-lr * st.slow,
                   [float(x) for x in ex["v"]], 1e-12, 1e-12, tag + " u")


def pin_closed_form_slowmo(use=None):
    """Constant gradient c on every worker and step, mu = 0.

    Each period moves the average K*lr*c away from the reference, so
    u_n = K c (1 - beta^n) / (1 - beta) and
    ref_n = theta0 - alpha lr K c [n - beta (1 - beta^n)/(1 - beta)] / (1 - beta).
    Within a period, after j local steps, theta = ref - j lr c.
    """
    for (W, K, beta, alpha, lr, c) in [(3, 4, 0.5, 1.0, 0.1, 0.7),
                                       (2, 2, 0.3, 0.5, 0.25, -1.5),
                                       (5, 3, 0.875, 1.5, 0.05, 2.0),
                                       (1, 1, 0.6, 1.0, 0.1, 1.0)]:
        theta0 = np.array([0.3, -2.0, 5.5])
        P = theta0.size
        periods = 6
        rec = []
        oracle.run(theta0, lambda s, W_, P_: np.full((W_, P_), c), W, K,
                   periods * K, lr, 0.0, beta, alpha, param_dt="f64",
                   mom_dt="f64", aux_dt="f64", use=use,
                   callback=lambda s, kind, st: rec.append((s, kind, st.copy())))
        for s, kind, st in rec:
            n, j = divmod(s, K)
            if j == 0:
                u = K * c * (1 - beta ** n) / (1 - beta)
                ref = theta0 - alpha * lr * K * c * (
                    n - beta * (1 - beta ** n) / (1 - beta)) / (1 - beta)
                assert kind == "reconcile"
                _close(st.slow, np.full(P, u), 1e-12, 1e-12, f"u n={n}")
                _close(st.anchor, ref, 1e-12, 1e-12, f"ref n={n}")
                _close(st.params, np.tile(ref, (W, 1)), 1e-12, 1e-12,
                       f"params n={n}")
            else:
                assert kind == "local"
                ref = st.anchor
                _close(st.params, np.tile(ref - j * lr * c, (W, 1)), 1e-12,
                       1e-12, f"local j={j}")
            _close(st.mom, np.full((W, P), c), 1e-12, 1e-12, "mom = c")


def pin_closed_form_momentum(use=None):
    """beta = 0, alpha = 1, identical workers, constant gradient c.

    Averaging identical replicas is the identity and SlowMo with beta = 0,
    alpha = 1 returns the average, so the run is heavy-ball SGD with a constant
    gradient: buf_t = c (1 - mu^t)/(1 - mu) and
    theta_t = theta0 - lr c [t - mu (1 - mu^t)/(1 - mu)] / (1 - mu).
    """
    for (W, K, mu, lr, c) in [(4, 3, 0.9, 0.1, 1.0), (2, 1, 0.5, 0.25, -3.0),
                              (3, 5, 0.75, 0.05, 0.5)]:
        theta0 = np.array([1.0, -0.25])
        rec = []
        oracle.run(theta0, lambda s, W_, P_: np.full((W_, P_), c), W, K,
                   4 * K + 1, lr, mu, 0.0, 1.0, param_dt="f64", mom_dt="f64",
                   aux_dt="f64", use=use,
                   callback=lambda s, kind, st: rec.append((s, st.copy())))
        for t, st in rec:
            buf = c * (1 - mu ** t) / (1 - mu)
            th = theta0 - lr * c * (t - mu * (1 - mu ** t) / (1 - mu)) / (1 - mu)
            _close(st.mom, np.full(st.mom.shape, buf), 1e-12, 1e-12,
                   f"buf t={t}")
            _close(st.params, np.tile(th, (W, 1)), 1e-12, 1e-12, f"theta t={t}")


def _torch_reference(theta0, grads, W, K, lr, mu, method="cpdp"):
    """The three strategies of Sec. 5.3 written with torch.optim.SGD, one
    optimizer per worker (local momentum buffers, Sec. 4.2):
      cpdp (beta = 0, alpha = 1): averaged gradient on sync steps, then
        parameter averaging copied back into every worker;
      localsgd: local gradient on every step, parameter averaging on sync steps;
      ddp: averaged gradient on every step, no parameter averaging.
    """
    import torch
    ps = [torch.nn.Parameter(torch.tensor(theta0, dtype=torch.float64))
          for _ in range(W)]
    opts = [torch.optim.SGD([p], lr=lr, momentum=mu) for p in ps]
    out = []
    for s, g in enumerate(grads, start=1):
        sync = s % K == 0 or method == "ddp"
        use_gbar = sync and method in ("cpdp", "ddp")
        gbar = g.mean(axis=0)
        for i in range(W):
            ps[i].grad = torch.tensor(gbar if use_gbar else g[i])
            opts[i].step()
        if sync and method in ("cpdp", "localsgd"):
            avg = torch.stack([p.detach() for p in ps]).mean(0)
            for p in ps:
                p.data.copy_(avg)
        bufs = np.stack([
            opts[i].state[ps[i]]["momentum_buffer"].numpy().copy()
            if mu > 0 else (gbar if use_gbar else g[i]) for i in range(W)])
        out.append((np.stack([p.detach().numpy().copy() for p in ps]), bufs))
    return out


def pin_torch_sgd(use=None):
    """beta = 0: the run equals per-worker torch.optim.SGD with the averaged
    gradient on sync steps followed by parameter averaging; covers K = 1
    (synchronous DDP, Sec. 3.1) and W = 1 (plain momentum SGD)."""
    rng = np.random.default_rng(11)
    for (W, K, mu, lr) in [(4, 1, 0.9, 0.1), (1, 3, 0.9, 0.1), (3, 2, 0.5, 0.2),
                           (5, 4, 0.9, 0.05), (2, 3, 0.0, 0.1)]:
        P = 6
        n = 3 * K + 2
        theta0 = rng.normal(0, 1, P)
        grads = [rng.normal(0, 1, (W, P)) for _ in range(n)]
        ref = _torch_reference(theta0, grads, W, K, lr, mu)
        rec = []
        oracle.run(theta0, lambda s, W_, P_: grads[s - 1], W, K, n, lr, mu,
                   0.0, 1.0, param_dt="f64", mom_dt="f64", aux_dt="f64",
                   use=use, callback=lambda s, kind, st: rec.append(st.copy()))
        for s, (st, (p_ref, b_ref)) in enumerate(zip(rec, ref), start=1):
            _close(st.params, p_ref, 1e-12, 1e-12, f"W={W} K={K} params s={s}")
            _close(st.mom, b_ref, 1e-12, 1e-12, f"W={W} K={K} mom s={s}")


def pin_permutation(use=None):
    """Relabelling the workers permutes params/mom and leaves SlowMo state and
    the reference model unchanged."""
    rng = np.random.default_rng(3)
    W, P, K, n = 5, 7, 3, 10
    theta0 = rng.normal(0, 1, P)
    grads = [rng.normal(0, 1, (W, P)) for _ in range(n)]
    perm = np.array([3, 0, 4, 1, 2])
    a = oracle.run(theta0, lambda s, W_, P_: grads[s - 1], W, K, n - 1, 0.1,
                   0.9, 0.5, 1.0, param_dt="f64", mom_dt="f64", aux_dt="f64",
                   use=use)
    b = oracle.run(theta0, lambda s, W_, P_: grads[s - 1][perm], W, K, n - 1,
                   0.1, 0.9, 0.5, 1.0, param_dt="f64", mom_dt="f64",
                   aux_dt="f64", use=use)
    _close(b.params, a.params[perm], 1e-13, 1e-13, "perm params")
    _close(b.mom, a.mom[perm], 1e-13, 1e-13, "perm mom")
    _close(b.slow, a.slow, 1e-13, 1e-13, "perm u")
    _close(b.anchor, a.anchor, 1e-13, 1e-13, "perm anchor")


def pin_fixed_point(use=None):
    """Zero gradients from identical workers: nothing moves, u stays 0
    (averaging identical replicas is the identity, Sec. 3.2)."""
    theta0 = np.array([0.125, -3.0, 7.5, 0.0], dtype=np.float64)
    for dt in ("f32", "f64"):
        st = oracle.run(theta0, lambda s, W_, P_: np.zeros((W_, P_)), 4, 3, 9,
                        0.1, 0.9, 0.7, 1.3, param_dt=dt, mom_dt=dt,
                        aux_dt=dt, use=use)
        assert np.array_equal(st.params, np.tile(theta0, (4, 1))), dt
        assert np.array_equal(st.anchor, theta0), dt
        assert not st.slow.any() and not st.mom.any(), dt


def pin_identical_workers(use=None):
    """W identical workers behave exactly like one worker (power-of-two W keeps
    the means exact, so this holds bitwise in fp32 storage too)."""
    rng = np.random.default_rng(9)
    P, K, n = 16, 4, 12
    theta0 = rng.normal(0, 0.02, P).astype(np.float32).astype(np.float64)
    g1 = [rng.normal(0, 1e-3, (1, P)).astype(np.float32).astype(np.float64)
          for _ in range(n)]
    one = oracle.run(theta0, lambda s, W_, P_: g1[s - 1], 1, K, n, 0.1, 0.9,
                     0.5, 1.0, use=use)
    four = oracle.run(theta0, lambda s, W_, P_: np.repeat(g1[s - 1], 4, 0), 4,
                      K, n, 0.1, 0.9, 0.5, 1.0, use=use)
    assert np.array_equal(four.params, np.repeat(one.params, 4, 0))
    assert np.array_equal(four.mom, np.repeat(one.mom, 4, 0))
    assert np.array_equal(four.slow, one.slow)
    assert np.array_equal(four.anchor, one.anchor)


def pin_linearity(use=None):
    """Gradients do not depend on theta here, so the state after any number of
    steps is linear in (theta0, gradients): F(a + b) = F(a) + F(b)."""
    rng = np.random.default_rng(21)
    W, P, K, n = 3, 5, 3, 8
    ta, tb = rng.normal(0, 1, P), rng.normal(0, 1, P)
    ga = [rng.normal(0, 1, (W, P)) for _ in range(n)]
    gb = [rng.normal(0, 1, (W, P)) for _ in range(n)]

    def go(t0, gs):
        return oracle.run(t0, lambda s, W_, P_: gs[s - 1], W, K, n - 1, 0.1,
                          0.9, 0.5, 0.8, param_dt="f64", mom_dt="f64",
                          aux_dt="f64", use=use)

    a, b = go(ta, ga), go(tb, gb)
    ab = go(ta + tb, [x + y for x, y in zip(ga, gb)])
    for name in ("params", "mom", "slow", "anchor"):
        _close(getattr(ab, name), getattr(a, name) + getattr(b, name), 1e-11,
               1e-11, "linearity " + name)


def pin_rounding(use=None):
    """Storage rounding: fp32 = IEEE round-to-nearest-even (numpy's cast);
    bf16 = torch's float32 -> bfloat16 conversion (also nearest-even)."""
    import torch
    rng = np.random.default_rng(0)
    xs = np.concatenate([rng.normal(0, 1, 2000) * 10.0 ** rng.integers(-8, 8, 2000),
                         [0.0, -0.0, 1.0 + 2.0 ** -24, 1.0 + 2.0 ** -8,
                          1.0 + 3 * 2.0 ** -8, 3.4e38, -3.4e38, 1e39, np.inf,
                          -np.inf, 1e-40],
                         # exact bf16 ties on both parities of the kept bit
                         1.0 + (np.arange(1, 64) + 0.5) * 2.0 ** -7,
                         -(2.0 + (np.arange(1, 64) + 0.5) * 2.0 ** -6)])
    with np.errstate(over="ignore"):
        f32 = xs.astype(np.float32)
    bf = torch.from_numpy(f32).to(torch.bfloat16).to(torch.float64).numpy()
    for x, want32, want16 in zip(xs, f32.astype(np.float64), bf):
        got32 = oracle.round_to("f32", x, use=use)
        got16 = oracle.round_to("bf16", x, use=use)
        assert got32 == want32 or (np.isnan(got32) and np.isnan(want32)), x
        assert got16 == want16 or (np.isnan(got16) and np.isnan(want16)), x
    assert np.isnan(oracle.round_to("bf16", np.nan, use=use))
    assert oracle.round_to("f64", 0.1, use=use) == 0.1


ALL_PINS = [pin_worked_example, pin_worked_example_vform, pin_brute_force,
            pin_closed_form_slowmo, pin_closed_form_momentum, pin_torch_sgd,
            pin_permutation, pin_fixed_point, pin_identical_workers,
            pin_linearity, pin_rounding]


def pin_torch_baselines(use=None):
    """LocalSGD and DDP (Sec. 5.3) against per-worker torch.optim.SGD."""
    rng = np.random.default_rng(17)
    for method in ("localsgd", "ddp"):
        for (W, K, mu, lr) in [(4, 2, 0.9, 0.1), (3, 3, 0.5, 0.2), (1, 2, 0.9, 0.1),
                               (5, 4, 0.0, 0.05)]:
            P = 5
            n = 3 * K + 1
            theta0 = rng.normal(0, 1, P)
            grads = [rng.normal(0, 1, (W, P)) for _ in range(n)]
            ref = _torch_reference(theta0, grads, W, K, lr, mu, method)
            rec = []
            oracle.run(theta0, lambda s, W_, P_: grads[s - 1], W, K, n, lr, mu,
                       0.5, 1.0, param_dt="f64", mom_dt="f64", aux_dt="f64",
                       use=use, method=method,
                       callback=lambda s, kind, st: rec.append(st.copy()))
            for s, (st, (p_ref, b_ref)) in enumerate(zip(rec, ref), start=1):
                tag = f"{method} W={W} K={K} s={s}"
                _close(st.params, p_ref, 1e-12, 1e-12, tag + " params")
                _close(st.mom, b_ref, 1e-12, 1e-12, tag + " mom")
                assert not st.slow.any(), tag + ": SlowMo state must stay 0"


def pin_brute_force_baselines(use=None):
    pin_brute_force(use, cases=10, seed=8, methods=("localsgd", "ddp"))


def pin_localsgd_closed_form(use=None):
    """LocalSGD, mu = 0, worker i always sees the constant gradient c_i: every
    period moves the average by K lr mean(c), so after n periods all workers
    hold theta0 - n K lr mean(c); j local steps into a period, worker i holds
    that minus j lr c_i."""
    c = np.array([0.5, -1.25, 2.0])
    W, K, lr = 3, 4, 0.1
    theta0 = np.array([1.0, -2.0])
    rec = []
    oracle.run(theta0, lambda s, W_, P_: np.tile(c[:, None], (1, P_)), W, K,
               3 * K, lr, 0.0, 0.7, 1.0, param_dt="f64", mom_dt="f64",
               aux_dt="f64", use=use, method="localsgd",
               callback=lambda s, kind, st: rec.append((s, st.copy())))
    for s, st in rec:
        n, j = divmod(s, K)
        base = theta0 - n * K * lr * c.mean()
        want = base[None, :] - j * lr * c[:, None]
        _close(st.params, want, 1e-12, 1e-12, f"localsgd closed form s={s}")
        if j == 0:
            _close(st.anchor, base, 1e-12, 1e-12, f"localsgd anchor s={s}")


ALL_PINS += [pin_torch_baselines, pin_brute_force_baselines, pin_localsgd_closed_form]


def _torch_opt_reference(theta0, grads, W, K, method, make_torch_opt,
                         average_state=False):
    """Per-worker torch optimizers (fp64) driven like the Sec. 4.2
    implementation: averaged gradient on CPDP/DDP sync steps, local gradient
    otherwise; parameter averaging on CPDP (beta = 0, alpha = 1) and LocalSGD
    sync steps; optimizer states averaged across workers on sync steps only
    when ``average_state`` (the optimizer-state-reconciliation variant)."""
    import torch
    ps = [torch.nn.Parameter(torch.tensor(theta0, dtype=torch.float64)) for _ in range(W)]
    opts = [make_torch_opt([p]) for p in ps]
    out = []
    for s, g in enumerate(grads, start=1):
        sync = s % K == 0 or method == "ddp"
        use_gbar = sync and method in ("cpdp", "ddp")
        gbar = g.mean(axis=0)
        for i in range(W):
            ps[i].grad = torch.tensor(gbar if use_gbar else g[i])
            opts[i].step()
        if sync and method in ("cpdp", "localsgd"):
            avg = torch.stack([p.detach() for p in ps]).mean(0)
            for p in ps:
                p.data.copy_(avg)
        if sync and average_state:
            for key in opts[0].state[ps[0]]:
                if key == "step":
                    continue
                mean = torch.stack([opts[i].state[ps[i]][key] for i in range(W)]).mean(0)
                for i in range(W):
                    opts[i].state[ps[i]][key].copy_(mean)
        out.append(np.stack([p.detach().numpy().copy() for p in ps]))
    return out


def pin_torch_optimizers(use=None):
    """SGD with weight decay and AdamW (Table 3 optimizers) in every strategy
    against torch.optim.SGD / torch.optim.AdamW, one optimizer per worker."""
    import torch
    rng = np.random.default_rng(23)
    cfgs = [
        ("sgd", dict(lr=0.1, momentum=0.9, weight_decay=5e-4),
         lambda s: oracle.sgd(0.1, 0.9, 5e-4)),
        ("sgd", dict(lr=0.05, momentum=0.0, weight_decay=0.01),
         lambda s: oracle.sgd(0.05, 0.0, 0.01)),
        ("adamw", dict(lr=5e-4, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.05),
         lambda s: oracle.adamw(5e-4, 0.9, 0.999, 1e-8, 0.05, s)),
        ("adamw", dict(lr=1e-2, betas=(0.8, 0.99), eps=1e-6, weight_decay=0.0),
         lambda s: oracle.adamw(1e-2, 0.8, 0.99, 1e-6, 0.0, s)),
    ]
    for method in ("cpdp", "localsgd", "ddp"):
        for kind, tkw, mk in cfgs:
            W, K, P = 3, 3, 4
            n = 3 * K + 1
            theta0 = rng.normal(0, 1, P)
            grads = [rng.normal(0, 1, (W, P)) for _ in range(n)]
            topt = ((lambda ps: torch.optim.SGD(ps, **tkw)) if kind == "sgd"
                    else (lambda ps: torch.optim.AdamW(ps, **tkw)))
            ref = _torch_opt_reference(theta0, grads, W, K, method, topt)
            rec = []
            oracle.run_opt(theta0, lambda s, W_, P_: grads[s - 1], W, K, n, mk, 0.0,
                           1.0, method=method, param_dt="f64", mom_dt="f64",
                           aux_dt="f64", use=use,
                           callback=lambda s, k, st, m2: rec.append(st.copy()))
            for s, (st, p_ref) in enumerate(zip(rec, ref), start=1):
                _close(st.params, p_ref, 1e-11, 1e-12, f"{kind} {method} s={s}")


def pin_adamw_closed_form(use=None):
    """AdamW with a constant gradient c and no weight decay: the bias-corrected
    moments are exactly c and c^2, so every step moves theta by
    lr * c / (|c| + eps)."""
    c, lr, eps = -0.3, 0.01, 1e-8
    theta0 = np.array([0.5, -1.0])
    for method in ("cpdp", "localsgd", "ddp"):
        rec = []
        oracle.run_opt(theta0, lambda s, W_, P_: np.full((W_, P_), c), 2, 3, 7,
                       lambda s: oracle.adamw(lr, 0.9, 0.999, eps, 0.0, s), 0.0, 1.0,
                       method=method, param_dt="f64", mom_dt="f64", aux_dt="f64",
                       use=use, callback=lambda s, k, st, m2: rec.append((s, st.copy())))
        for s, st in rec:
            want = theta0 - s * lr * c / (abs(c) + eps)
            _close(st.params, np.tile(want, (2, 1)), 1e-12, 1e-12, f"adamw cf {method} s={s}")


def pin_sgd_weight_decay_closed_form(use=None):
    """SGD, mu = 0, weight decay wd, constant gradient c: theta_{t+1} =
    theta_t (1 - lr wd) - lr c, so theta_t = (theta0 + c/wd)(1 - lr wd)^t - c/wd."""
    c, lr, wd = 0.7, 0.1, 0.05
    theta0 = np.array([2.0, -3.0, 0.25])
    rec = []
    oracle.run_opt(theta0, lambda s, W_, P_: np.full((W_, P_), c), 4, 2, 9,
                   lambda s: oracle.sgd(lr, 0.0, wd), 0.0, 1.0, method="cpdp",
                   param_dt="f64", mom_dt="f64", aux_dt="f64", use=use,
                   callback=lambda s, k, st, m2: rec.append((s, st.copy())))
    for s, st in rec:
        want = (theta0 + c / wd) * (1 - lr * wd) ** s - c / wd
        _close(st.params, np.tile(want, (4, 1)), 1e-12, 1e-12, f"sgd wd cf s={s}")


def pin_general_sgd_matches_plain(use=None):
    """The general-optimizer path with plain SGD (no weight decay) is the same
    computation as the plain local step and reconcile (bitwise, fp32 storage)."""
    rng = np.random.default_rng(31)
    W, P, K, n = 4, 64, 3, 9
    theta0 = rng.normal(0, 0.02, P).astype(np.float32).astype(np.float64)
    grads = [rng.normal(0, 1e-3, (W, P)).astype(np.float32).astype(np.float64)
             for _ in range(n)]
    for method in ("cpdp", "localsgd", "ddp"):
        a = oracle.run(theta0, lambda s, W_, P_: grads[s - 1], W, K, n, 0.1, 0.9, 0.5,
                       1.0, method=method, use=use)
        b, _ = oracle.run_opt(theta0, lambda s, W_, P_: grads[s - 1], W, K, n,
                              lambda s: oracle.sgd(0.1, 0.9, 0.0), 0.5, 1.0,
                              method=method, use=use)
        for name in ("params", "mom", "slow", "anchor"):
            assert np.array_equal(getattr(a, name), getattr(b, name)), (method, name)


ALL_PINS += [pin_torch_optimizers, pin_adamw_closed_form,
             pin_sgd_weight_decay_closed_form, pin_general_sgd_matches_plain]


def pin_torch_state_averaging(use=None):
    """Optimizer-state reconciliation: momentum buffers (SGD) or both AdamW
    moments replaced by the worker mean on sync steps, against per-worker torch
    optimizers whose states are averaged the same way."""
    import torch
    rng = np.random.default_rng(29)
    for method in ("cpdp", "localsgd", "ddp"):
        for kind in ("sgd", "adamw"):
            W, K, P = 4, 2, 3
            n = 3 * K + 1
            theta0 = rng.normal(0, 1, P)
            grads = [rng.normal(0, 1, (W, P)) for _ in range(n)]
            if kind == "sgd":
                topt = lambda ps: torch.optim.SGD(ps, lr=0.1, momentum=0.9, weight_decay=1e-3)  # noqa: E731
                mk = lambda s: oracle.sgd(0.1, 0.9, 1e-3)  # noqa: E731
            else:
                topt = lambda ps: torch.optim.AdamW(ps, lr=1e-2, betas=(0.9, 0.99), eps=1e-6,  # noqa: E731
                                                    weight_decay=0.01)
                mk = lambda s: oracle.adamw(1e-2, 0.9, 0.99, 1e-6, 0.01, s)  # noqa: E731
            ref = _torch_opt_reference(theta0, grads, W, K, method, topt, average_state=True)
            rec = []
            oracle.run_opt(theta0, lambda s, W_, P_: grads[s - 1], W, K, n, mk, 0.0, 1.0,
                           method=method, param_dt="f64", mom_dt="f64", aux_dt="f64",
                           use=use, flags=oracle.SYNC_AVERAGE_STATE,
                           callback=lambda s, k, st, m2: rec.append(st.copy()))
            for s, (st, p_ref) in enumerate(zip(rec, ref), start=1):
                _close(st.params, p_ref, 1e-11, 1e-12, f"avg state {kind} {method} s={s}")


def pin_gradient_write_back(use=None):
    """With the write-back flag the gradient rows leave a CPDP or DDP sync
    holding the replica-mean gradient (what a DDP AllReduce leaves in .grad),
    LocalSGD leaves them untouched, and the rest of the state is unchanged."""
    rng = np.random.default_rng(37)
    W, P = 3, 5
    theta0 = rng.normal(0, 1, P)
    g = rng.normal(0, 1, (W, P))
    for method in ("cpdp", "localsgd", "ddp"):
        a = oracle.state_init(theta0, W, "f64", "f64", "f64", use=use)
        b = a.copy()
        ga = oracle.sync_opt(a, method, g, oracle.sgd(0.1, 0.9), 0.5, 1.0, flags=0)
        gb = oracle.sync_opt(b, method, g, oracle.sgd(0.1, 0.9), 0.5, 1.0,
                             flags=oracle.SYNC_WRITE_GBAR)
        assert np.array_equal(ga, g), method
        want = g if method == "localsgd" else np.tile(g.mean(axis=0), (W, 1))
        _close(gb, want, 1e-15, 1e-15, f"write-back {method}")
        for name in ("params", "mom", "slow", "anchor"):
            assert np.array_equal(getattr(a, name), getattr(b, name)), (method, name)


ALL_PINS += [pin_torch_state_averaging, pin_gradient_write_back]


# ---- storage-rounding points ---------------------------------------------------

def exact(expr: str):
    """Value of a fixture expression (numbers, + - * / and ** over exact
    rationals), e.g. "1 + 3*2**-9"."""
    import ast
    import operator as op
    ops = {ast.Add: op.add, ast.Sub: op.sub, ast.Mult: op.mul, ast.Div: op.truediv,
           ast.Pow: op.pow}

    def ev(n):
        if isinstance(n, ast.Expression):
            return ev(n.body)
        if isinstance(n, ast.Constant) and isinstance(n.value, int):
            return Fraction(n.value)
        if isinstance(n, ast.Constant) and isinstance(n.value, float):
            return Fraction(n.value)
        if isinstance(n, ast.UnaryOp) and isinstance(n.op, (ast.USub, ast.UAdd)):
            v = ev(n.operand)
            return -v if isinstance(n.op, ast.USub) else v
        if isinstance(n, ast.BinOp) and type(n.op) in ops:
            return ops[type(n.op)](ev(n.left), ev(n.right))
        raise ValueError(f"not an exact expression: {expr!r}")

    return ev(ast.parse(str(expr), mode="eval"))


def _f(expr) -> float:
    v = exact(expr)
    assert Fraction(float(v)) == v, f"{expr} is not a double"
    return float(v)


def _fixture_state(case, dts, use):
    """The case's input state as an OracleState (P = number of coordinates)."""
    W, cs = case["W"], case["coords"]
    P = len(cs)
    st = oracle.state_init(np.zeros(P), W, dts["param"], dts["mom"], dts["aux"], use=use)
    for p, c in enumerate(cs):
        for i in range(W):
            st.params[i, p] = _f(c["in"]["params"][i])
            st.mom[i, p] = _f(c["in"]["mom"][i])
        st.slow[p] = _f(c["in"]["u"])
        st.anchor[p] = _f(c["in"]["anchor"])
    mom2 = None
    if "mom2" in cs[0]["in"]:
        mom2 = np.array([[_f(c["in"]["mom2"][i]) for c in cs] for i in range(W)])
    g = np.array([[_f(c["grads"][i]) for c in cs] for i in range(W)])
    return st, mom2, g


def _check_fixture_out(case, st, mom2, tag):
    for p, c in enumerate(case["coords"]):
        want = c["out"]
        got = {"params": st.params[:, p], "mom": st.mom[:, p], "u": st.slow[p],
               "anchor": st.anchor[p]}
        if "mom2" in want:
            got["mom2"] = mom2[:, p]
        for k, w in want.items():
            w = [_f(x) for x in w] if isinstance(w, list) else _f(w)
            g = np.atleast_1d(got[k])
            assert np.array_equal(g, np.atleast_1d(w)), \
                f"{tag} coordinate {p} ({c['pins']}): {k} = {g.tolist()}, want {w}"


def pin_rounding_points(use=None):
    """Every storage-rounding point of init, the local steps and the three
    synchronisation steps, on the plain functions and on the general-optimizer
    ones, against the hand derivations of tests/golden/rounding_points_bf16.json
    (Algorithm 1 and Sec. 4.2: tensors are stored in their storage types where
    the implementation writes them)."""
    fx = json.load(open(os.path.join(GOLDEN, "rounding_points_bf16.json")))
    dts = fx["dtypes"]
    hp = {k: _f(v) for k, v in fx["hyper"].items()}
    lr, mu, beta, alpha = hp["lr"], hp["mu"], hp["beta"], hp["alpha"]
    for case in fx["cases"]:
        op = case["op"]
        if op == "init":
            cs = case["coords"]
            st = oracle.state_init(np.array([_f(c["theta0"]) for c in cs]), case["W"],
                                   dts["param"], dts["mom"], dts["aux"], use=use)
            _check_fixture_out(case, st, None, "init")
            continue
        if op == "reconcile_vform":  # the paper's own variables; st.slow holds v
            st, _, g = _fixture_state(case, dts, use)
            oracle.reconcile_vform(st, g, lr, mu, beta)
            _check_fixture_out(case, st, None, op)
            continue
        if op in ("local", "reconcile", "localsgd", "ddp"):
            # the plain momentum-SGD functions
            st, _, g = _fixture_state(case, dts, use)
            if op == "local":
                oracle.local_step(st, g, lr, mu)
            elif op == "reconcile":
                oracle.reconcile(st, g, lr, mu, beta, alpha)
            elif op == "localsgd":
                oracle.localsgd_sync(st, g, lr, mu)
            else:
                oracle.ddp_step(st, g, lr, mu)
            _check_fixture_out(case, st, None, op)
            # the general-optimizer functions with plain momentum SGD
            st, _, g = _fixture_state(case, dts, use)
            o = oracle.sgd(lr, mu, 0.0)
            if op == "local":
                oracle.local_step_opt(st, g, o)
            else:
                method = {"reconcile": "cpdp", "localsgd": "localsgd", "ddp": "ddp"}[op]
                oracle.sync_opt(st, method, g, o, beta, alpha)
            _check_fixture_out(case, st, None, op + " (general optimizer)")
            continue
        if op == "ddp_average_state":  # a variant of the general functions only
            st, _, g = _fixture_state(case, dts, use)
            oracle.sync_opt(st, "ddp", g, oracle.sgd(lr, mu, 0.0), beta, alpha,
                            flags=oracle.SYNC_AVERAGE_STATE)
            _check_fixture_out(case, st, None, op)
            continue
        o = {k: (_f(v) if isinstance(v, str) else v) for k, v in case["opt"].items()}
        st, mom2, g = _fixture_state(case, dts, use)
        if op == "local_sgd_wd":
            oracle.local_step_opt(st, g, oracle.sgd(o["lr"], o["mu"], o["wd"]))
        elif op == "local_adamw":
            mom2 = np.ascontiguousarray(mom2)
            oracle.local_step_opt(st, g, oracle.adamw(o["lr"], o["beta1"], o["beta2"],
                                                      o["eps"], o["wd"], o["step"]), mom2)
        else:
            raise ValueError(op)
        _check_fixture_out(case, st, mom2, op)


ALL_PINS.insert(0, pin_rounding_points)


def pin_brute_force_rounded(use=None, seed=41):
    """The oracle's stored state equals, bit for bit, an exact rational run of
    the same steps that rounds to the storage types only where a tensor is
    written (tests/brute_rounded.py), on tiny random inputs: every dtype
    combination the library takes, the three strategies, the plain momentum-
    SGD functions, the v-form, and the general functions with SGD + weight
    decay and AdamW, with and without the two sync-step variants."""
    import brute_rounded as br
    rng = np.random.default_rng(seed)
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    lr, mu, beta, alpha = f32(0.1), f32(0.9), f32(0.5), 1.0
    W, P, K, n = 3, 5, 3, 7
    combos = [("f32", "f32", "f32"), ("bf16", "f32", "f32"), ("bf16", "bf16", "f32"),
              ("f32", "bf16", "f32")]

    def compare(st, bst, tag, mom2=None):
        fl = lambda rows: np.array([[float(x) for x in r] for r in rows])  # noqa: E731
        for name, a, b in (("params", st.params, fl(bst.params)), ("mom", st.mom, fl(bst.mom)),
                           ("u", st.slow, np.array([float(x) for x in bst.u])),
                           ("anchor", st.anchor, np.array([float(x) for x in bst.ref]))):
            assert np.array_equal(a, b), f"{tag}: {name} {a.ravel()[:4]} want {b.ravel()[:4]}"
        if mom2 is not None:
            assert np.array_equal(mom2, fl(bst.mom2)), f"{tag}: mom2"

    for pdt, mdt, adt in combos:
        theta0 = rng.normal(0, 0.02, P).astype(np.float32).astype(np.float64)
        grads = [rng.normal(0, 1e-3, (W, P)).astype(np.float32).astype(np.float64)
                 for _ in range(n)]
        # plain momentum-SGD functions, and the v-form
        for method in ("cpdp", "localsgd", "ddp", "vform"):
            st = oracle.state_init(theta0, W, pdt, mdt, adt, use=use)
            bst = br.State(theta0, W, pdt, mdt, adt)
            o = br.Opt("sgd", lr, mu)
            for s in range(1, n + 1):
                g = grads[s - 1]
                tag = f"{method} {pdt}/{mdt}/{adt} step {s}"
                if method == "ddp":
                    oracle.ddp_step(st, g, lr, mu)
                    br.sync_step(bst, "ddp", g, o)
                elif s % K:
                    oracle.local_step(st, g, lr, mu)
                    br.local_step(bst, g, o)
                elif method == "cpdp":
                    oracle.reconcile(st, g, lr, mu, beta, alpha)
                    br.sync_step(bst, "cpdp", g, o, beta, alpha)
                elif method == "localsgd":
                    oracle.localsgd_sync(st, g, lr, mu)
                    br.sync_step(bst, "localsgd", g, o)
                else:
                    oracle.reconcile_vform(st, g, lr, mu, beta)
                    br.sync_vform(bst, g, o, beta)
                compare(st, bst, tag)
        # general-optimizer functions
        opts = [("sgd_wd", lambda t: oracle.sgd(lr, mu, f32(5e-4)),
                 lambda t: br.Opt("sgd", lr, mu, wd=f32(5e-4))),
                ("adamw", lambda t: oracle.adamw(f32(1e-2), mu, f32(0.999), f32(1e-8), f32(0.05), t),
                 lambda t: br.Opt("adamw", f32(1e-2), mu, f32(0.05), f32(0.999), f32(1e-8), t))]
        for method in ("cpdp", "localsgd", "ddp"):
            for oname, mk, bmk in opts:
                for flags in (0, 3):
                    st = oracle.state_init(theta0, W, pdt, mdt, adt, use=use)
                    bst = br.State(theta0, W, pdt, mdt, adt)
                    mom2 = np.zeros((W, P))
                    for s in range(1, n + 1):
                        g = grads[s - 1]
                        tag = f"{method} {oname} flags={flags} {pdt}/{mdt}/{adt} step {s}"
                        if method == "ddp" or s % K == 0:
                            gout = oracle.sync_opt(st, method, g, mk(s), beta, alpha, mom2,
                                                   flags=flags)
                            bg = br.sync_step(bst, method, g, bmk(s), beta, alpha, flags)
                            assert np.array_equal(gout, np.array([[float(x) for x in r]
                                                                  for r in bg])), tag + " grads"
                        else:
                            oracle.local_step_opt(st, g, mk(s), mom2)
                            br.local_step(bst, g, bmk(s))
                        compare(st, bst, tag, mom2)


ALL_PINS.append(pin_brute_force_rounded)


def _ulps(a, b):
    """|a - b| in units of the fp32 spacing at b (elementwise)."""
    b32 = np.asarray(b, dtype=np.float32)
    return np.abs(np.asarray(a, dtype=np.float64) - b32.astype(np.float64)) / \
        np.spacing(np.abs(b32)).astype(np.float64)


def pin_torch_fp32_optimizers(use=None):
    """fp32 storage against PyTorch's own fp32 optimizers (one worker, local
    steps): torch.optim.SGD (momentum, coupled weight decay) and
    torch.optim.AdamW on float32 parameters.  torch multiplies its fp32
    tensors by AdamW's decay factor 1 - lr*wd, step size lr/(1 - b1^t) and
    sqrt(1 - b2^t) as fp32 values, which is the oracle's reading.  The two
    differ only in the rounding of intermediate tensor operations (torch
    rounds after each of mul_, add_, lerp_, sqrt, div), so the parameters
    stay within 2 fp32 ulps over 24 steps (parameters of size 1..2, SGD
    gradients of size 0.01).  lr = 1e-3 and wd = 0.02 make
    1 - lr*wd lose 0.46 ulp in fp32; with the factor kept exact, parameters
    of size 1..2 drift by about a quarter to half an ulp per step."""
    import torch
    rng = np.random.default_rng(43)
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    P, n = 2048, 24
    theta0 = (rng.choice([-1.0, 1.0], P) * (1 + rng.random(P))).astype(np.float32)
    grads = {"adamw": [rng.normal(0, 1, (1, P)).astype(np.float32) for _ in range(n)],
             # SGD steps scale with the gradient: small ones keep theta in its
             # binade, so ulps at theta measure the update's rounding, not a
             # cancellation
             "sgd": [rng.normal(0, 1e-2, (1, P)).astype(np.float32) for _ in range(n)]}
    cfgs = [("adamw", dict(lr=f32(1e-3), betas=(f32(0.9), f32(0.999)), eps=f32(1e-8),
                           weight_decay=f32(0.02)),
             lambda t: oracle.adamw(f32(1e-3), f32(0.9), f32(0.999), f32(1e-8), f32(0.02), t)),
            ("sgd", dict(lr=f32(0.1), momentum=f32(0.9), weight_decay=f32(5e-4)),
             lambda t: oracle.sgd(f32(0.1), f32(0.9), f32(5e-4)))]
    for kind, tkw, mk in cfgs:
        p = torch.nn.Parameter(torch.from_numpy(theta0.copy()))
        opt = (torch.optim.AdamW([p], foreach=False, **tkw) if kind == "adamw"
               else torch.optim.SGD([p], foreach=False, **tkw))
        st = oracle.state_init(theta0.astype(np.float64), 1, "f32", "f32", "f32", use=use)
        mom2 = np.zeros((1, P))
        for t in range(1, n + 1):
            g = grads[kind][t - 1]
            p.grad = torch.from_numpy(g[0].copy())
            opt.step()
            oracle.local_step_opt(st, g.astype(np.float64), mk(t), mom2)
            d = _ulps(st.params[0], p.detach().numpy())
            assert d.max() <= 2, f"{kind} step {t}: {int((d > 2).sum())} parameters more " \
                                 f"than 2 ulps from torch (max {d.max():.1f})"


ALL_PINS.append(pin_torch_fp32_optimizers)


def _torch_bf16_cpdp(theta0, grads, W, K, lr, mu, beta, alpha):
    """CPDP with SlowMo written with torch tensor operations in the stress
    storage types: bf16 parameter tensors, fp32 momentum buffers, fp32 mean
    gradient, u and reference model.  In the order of Sec. 4.2: the local
    optimizer step writes each replica's bf16 parameter tensor; at a sync the
    mean gradient is formed, the optimizer step writes the parameter tensors,
    and only then are they averaged, SlowMo applied and the result copied
    back.  Returns the (params, mom, u, anchor) arrays after every step."""
    import torch
    bf, f32 = torch.bfloat16, torch.float32
    ps = [torch.tensor(theta0, dtype=f32).to(bf) for _ in range(W)]
    bufs = [torch.zeros(len(theta0), dtype=f32) for _ in range(W)]
    u = torch.zeros(len(theta0), dtype=f32)
    ref = ps[0].to(f32)
    out = []
    for s, g in enumerate(grads, start=1):
        gt = torch.tensor(g, dtype=f32)
        sync = s % K == 0
        gbar = gt.mean(0) if sync else None
        for i in range(W):
            bufs[i].mul_(mu).add_(gbar if sync else gt[i])
            ps[i].copy_((ps[i].to(f32) - lr * bufs[i]).to(bf))
        if sync:
            avg = torch.stack([p.to(f32) for p in ps]).mean(0)
            u = beta * u + (ref - avg) / lr
            ref = ref - alpha * lr * u
            for p in ps:
                p.copy_(ref.to(bf))
        out.append((np.stack([p.to(f32).numpy() for p in ps]).astype(np.float64),
                    np.stack([b.numpy() for b in bufs]).astype(np.float64),
                    u.numpy().astype(np.float64), ref.numpy().astype(np.float64)))
    return out


def pin_torch_bf16_params(use=None):
    """The stress storage types (bf16 parameters, fp32 momentum, u and
    anchor) against the torch rendition above.  torch rounds after every
    tensor operation where the oracle rounds once per stored tensor, so:
      * fp32 momentum agrees to a few ulps of the updates' operands (a result
        may cancel, so ulps are taken at the largest |m| or summed gradient
        the coordinate has seen so far);
      * a bf16 parameter may land one bf16 ulp away where such a difference
        meets a rounding boundary; that must stay rare (at most 1 % of the
        coordinates over the run) and be exactly one ulp;
      * until its first parameter flip, a coordinate's anchor and lr*u agree
        to a few fp32 ulps of the anchor (after a flip the mean and so the
        SlowMo state legitimately move by up to a bf16 ulp / W)."""
    rng = np.random.default_rng(47)
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    W, P, K, n = 4, 512, 2, 10
    lr, mu, beta, alpha = f32(0.1), f32(0.9), f32(0.5), 1.0
    theta0 = rng.normal(0, 0.02, P).astype(np.float32).astype(np.float64)
    grads = [rng.normal(0, 1e-3, (W, P)).astype(np.float32).astype(np.float64)
             for _ in range(n)]
    ref = _torch_bf16_cpdp(theta0, grads, W, K, lr, mu, beta, alpha)
    rec = []
    oracle.run(theta0, lambda s, W_, P_: grads[s - 1], W, K, n, lr, mu, beta, alpha,
               param_dt="bf16", mom_dt="f32", aux_dt="f32", use=use,
               callback=lambda s, kind, st: rec.append(st.copy()))
    sp = lambda x: np.spacing(np.abs(np.asarray(x)).astype(np.float32)).astype(np.float64)  # noqa: E731
    flipped = np.zeros(P, dtype=bool)
    m_scale = np.zeros((W, P))
    for s, (st, (p_ref, m_ref, u_ref, a_ref)) in enumerate(zip(rec, ref), start=1):
        tag = f"bf16 rendition step {s}"
        off = np.abs(st.params - p_ref)
        assert ((off == 0) | (off == sp(p_ref) * 2 ** 16)).all(), \
            tag + f": a parameter differs by other than one bf16 ulp ({off.max():.2e})"
        flipped |= (off > 0).any(axis=0)
        assert flipped.mean() <= 0.01, tag + f": {flipped.mean():.3f} of coordinates flipped"
        g = grads[s - 1]
        # operands of the buffer update: the gradient rows it sums (at a sync,
        # all W of them) and the buffer itself
        g_ops = np.tile(np.abs(g).max(axis=0), (W, 1)) if s % K == 0 else np.abs(g)
        m_scale = np.maximum(m_scale, np.maximum(np.abs(m_ref), g_ops))
        assert (np.abs(st.mom - m_ref) <= 4 * sp(m_scale)).all(), tag + ": mom"
        ok = ~flipped
        scale = sp(a_ref)
        assert (np.abs(st.anchor - a_ref) <= 8 * scale)[ok].all(), tag + ": anchor"
        assert (np.abs(lr * (st.slow - u_ref)) <= 8 * scale)[ok].all(), tag + ": lr*u"


ALL_PINS.append(pin_torch_bf16_params)
