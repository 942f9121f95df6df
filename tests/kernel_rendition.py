"""An fp32 model of the library's momentum-SGD local step and CPDP reconcile,
in the operation order of its gfx950 kernels, for the tests that explain the
bf16 tolerance (it is not the oracle and the oracle does not use it).

The kernels compute in fp32: fused multiply-adds round once, every other
operation rounds on its own (they are built with -ffp-contract=off), fp32
division is correctly rounded, and bf16 parameters are the round-to-nearest-
even bf16 of the fp32 value.  Per coordinate and replica:
  local step   m <- fma(mu, m, g);  theta <- bf16(fma(-lr, m, theta))
  reconcile    gbar = (((g_0 + g_1) + g_2) + ... + g_{W-1}) * (1/W)
               for i = 0..W-1:  m_i <- fma(mu, m_i, gbar)
                                x_i = bf16(fma(-lr, m_i, theta_i))
                                s <- s + (x_i - a)
               u <- fma(beta, u, -(s * (1/W)) / lr)
               a <- fma(-(alpha * lr), u, a);  theta_i <- bf16(a)
with 1/W and alpha*lr rounded to fp32 once (bf16() is the identity for fp32
parameters).  numpy's float32 arithmetic is
IEEE (correctly rounded); the fused multiply-add is emulated exactly below.
"""
from __future__ import annotations

import numpy as np

F32 = np.float32


def fma32(a, b, c) -> np.ndarray:
    """fp32 fused multiply-add: a*b + c rounded once to nearest-even fp32.
    a*b of two fp32 values is exact in double; the double sum s = a*b + c may
    round, and TwoSum gives its exact error e.  The fp32 rounding of s + e
    equals that of s unless s lies exactly halfway between two fp32 values,
    where the sign of e decides."""
    a64 = np.asarray(a, F32).astype(np.float64)
    b64 = np.asarray(b, F32).astype(np.float64)
    c64 = np.asarray(c, F32).astype(np.float64)
    p = a64 * b64
    s = p + c64
    bb = s - p
    e = (p - (s - bb)) + (c64 - bb)
    r = s.astype(F32)
    r64 = r.astype(np.float64)
    tie_candidates = (e != 0) & (r64 != s)
    if tie_candidates.any():
        away = np.where(s > r64, np.inf, -np.inf).astype(F32)
        other = np.nextafter(r, away)
        mid = (r64 + other.astype(np.float64)) / 2
        tie = tie_candidates & (s == mid)
        if tie.any():
            up = np.maximum(r, other)
            down = np.minimum(r, other)
            r = np.where(tie, np.where(e > 0, up, down), r)
    return r


def bf16(x) -> np.ndarray:
    """Round fp32 values to nearest-even bf16 (NaN kept quiet), as fp32."""
    b = np.asarray(x, F32).view(np.uint32).astype(np.uint64)
    nan = (b & 0x7FFFFFFF) > 0x7F800000
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    r = np.where(nan, b | 0x400000, r) & 0xFFFF0000
    return r.astype(np.uint32).view(F32)


class Rendition:
    """State of W replicas over a set of coordinates (all arrays fp32);
    param_dt "bf16" or "f32" is the parameters' storage type."""

    def __init__(self, theta0: np.ndarray, W: int, param_dt: str = "bf16"):
        th = np.asarray(theta0, F32)
        self.round = bf16 if param_dt == "bf16" else (lambda x: np.asarray(x, F32))
        assert np.array_equal(self.round(th), th), "theta0 must be a parameter-type value"
        self.W = W
        self.params = np.tile(th, (W, 1))
        self.mom = np.zeros_like(self.params)
        self.u = np.zeros_like(th)
        self.a = th.copy()

    def local_step(self, g: np.ndarray, lr: float, mu: float) -> None:
        g = np.asarray(g, F32)
        for i in range(self.W):
            self.mom[i] = fma32(F32(mu), self.mom[i], g[i])
            self.params[i] = self.round(fma32(F32(-F32(lr)), self.mom[i], self.params[i]))

    def reconcile(self, g: np.ndarray, lr: float, mu: float, beta: float,
                  alpha: float) -> None:
        g = np.asarray(g, F32)
        lr, mu, beta = F32(lr), F32(mu), F32(beta)
        inv_w = F32(1) / F32(self.W)
        alpha_lr = F32(alpha) * lr
        acc = np.zeros_like(self.a)
        for i in range(self.W):
            acc = acc + g[i]
        gbar = acc * inv_w
        s = np.zeros_like(self.a)
        for i in range(self.W):
            self.mom[i] = fma32(mu, self.mom[i], gbar)
            x = self.round(fma32(-lr, self.mom[i], self.params[i]))
            s = s + (x - self.a)
        drift = s * inv_w
        self.u = fma32(beta, self.u, (-drift) / lr)
        self.a = fma32(-alpha_lr, self.u, self.a)
        self.params[:] = self.round(self.a)[None, :]

    def snapshot(self) -> dict:
        return {"params": self.params.astype(np.float64), "mom": self.mom.astype(np.float64),
                "slow_mom": self.u.astype(np.float64), "anchor": self.a.astype(np.float64)}
