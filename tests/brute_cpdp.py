"""Exact rational brute force of Algorithm 1 (CPDP with SlowMo) for tiny inputs.

A second, independent statement of the method used to pin the fp64 oracle.
It is written in the paper's own variables (Sec. 3.3): the SlowMo velocity v
and the reference model theta_ref, with the optimizer of Sec. 4.2 (SGD with a
local momentum buffer per worker) and the SlowMo step size alpha of the
original SlowMo formulation applied to the velocity (alpha = 1 is the paper's
theta_new = theta_ref + v).  Everything is a ``fractions.Fraction``: no
rounding anywhere, pure-Python loops, so only tiny sizes are practical.
"""
from __future__ import annotations

from fractions import Fraction


def run_exact(theta0, grads, W, K, lr, mu, beta, alpha=1, T=0, method="cpdp"):
    """Run Algorithm 1 exactly (method "cpdp"), or the two baselines of
    Sec. 5.3 with the same optimizer: "localsgd" (local steps; at a sync step
    each worker steps on its own gradient, then parameters are averaged, no
    SlowMo) and "ddp" (every step averages the gradient; no parameter
    averaging).

    theta0: list of P numbers; grads: list over steps of W lists of P numbers
    (grads[s][i][p] is g_{i, s+1}).  Returns a list with one snapshot per step:
    dict(kind, params, mom, v, ref) with exact Fractions.
    """
    F = Fraction
    lr, mu, beta, alpha = F(lr), F(mu), F(beta), F(alpha)
    P = len(theta0)
    theta = [[F(x) for x in theta0] for _ in range(W)]
    buf = [[F(0)] * P for _ in range(W)]
    v = [F(0)] * P
    ref = [F(x) for x in theta0]
    out = []
    for s, g_step in enumerate(grads):
        step = s + 1
        t = ((step - 1) % T) + 1 if T > 0 else step
        sync = (t % K == 0) or (T > 0 and t == T) or method == "ddp"
        g = [[F(x) for x in row] for row in g_step]
        if sync and method == "ddp":
            for p in range(P):
                gbar = sum(g[i][p] for i in range(W)) / W
                for i in range(W):
                    buf[i][p] = mu * buf[i][p] + gbar
                    theta[i][p] = theta[i][p] - lr * buf[i][p]
        elif sync and method == "localsgd":
            for p in range(P):
                for i in range(W):
                    buf[i][p] = mu * buf[i][p] + g[i][p]
                    theta[i][p] = theta[i][p] - lr * buf[i][p]
                avg = sum(theta[i][p] for i in range(W)) / W
                for i in range(W):
                    theta[i][p] = avg
                ref[p] = avg
        elif not sync:
            for i in range(W):
                for p in range(P):
                    buf[i][p] = mu * buf[i][p] + g[i][p]
                    theta[i][p] = theta[i][p] - lr * buf[i][p]
        else:
            for p in range(P):
                gbar = sum(g[i][p] for i in range(W)) / W
                for i in range(W):
                    buf[i][p] = mu * buf[i][p] + gbar
                    theta[i][p] = theta[i][p] - lr * buf[i][p]
                avg = sum(theta[i][p] for i in range(W)) / W
                delta = avg - ref[p]
                v[p] = beta * v[p] + delta
                new = ref[p] + alpha * v[p]
                for i in range(W):
                    theta[i][p] = new
                ref[p] = new
        out.append(dict(kind="reconcile" if sync else "local",
                        params=[row[:] for row in theta],
                        mom=[row[:] for row in buf], v=v[:], ref=ref[:]))
    return out
