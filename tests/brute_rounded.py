"""Exact rational statement of the CPDP steps with the storage roundings,
for comparison with the oracle bit for bit on tiny inputs.

Written from the method, not from the oracle: Algorithm 1 (initialisation,
local update, synchronization), the Sec. 5.3 baselines (LocalSGD, DDP),
the Table 3 optimizers in the framework's semantics (SGD with momentum and
coupled weight decay, AdamW with decoupled decay and bias correction), and
the reading of Sec. 4.2 that every tensor the implementation writes is
stored in its storage type.  Arithmetic between stores is exact
(fractions.Fraction); square roots are computed to 2^-200 relative, far
below any rounding decision.  Rounding to fp32 and bf16 is written here from
the IEEE definition: round to nearest representable value of the format,
ties to the even significand; bf16 rounds the fp32 value.
"""
from __future__ import annotations

from fractions import Fraction
from math import isqrt

# (significand bits including the leading one, smallest normal exponent,
#  largest exponent) of the storage formats
FORMATS = {"f32": (24, -126, 127), "bf16": (8, -126, 127)}


def _rne(x: Fraction, p: int, emin: int, emax: int) -> Fraction:
    if x == 0:
        return Fraction(0)
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if a < Fraction(2) ** e:
        e -= 1
    elif a >= Fraction(2) ** (e + 1):
        e += 1
    e = max(e, emin)                 # subnormal range: fixed spacing
    q = Fraction(2) ** (e - (p - 1))  # spacing of representable values at a
    n = a / q
    k = n.numerator // n.denominator
    rem = n - k
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and k % 2 == 1):
        k += 1
    r = k * q
    if r >= Fraction(2) ** (emax + 1):
        raise OverflowError("value outside the format's range")
    return r if x > 0 else -r


def store(dt: str, x: Fraction) -> Fraction:
    """The value a tensor of storage type dt holds after x is written."""
    if dt == "f64":
        return x
    if dt == "f32":
        return _rne(x, *FORMATS["f32"])
    if dt == "bf16":
        return _rne(_rne(x, *FORMATS["f32"]), *FORMATS["bf16"])
    raise ValueError(dt)


def sqrt(x: Fraction, bits: int = 200) -> Fraction:
    if x < 0:
        raise ValueError("sqrt of a negative number")
    n, d = x.numerator, x.denominator
    return Fraction(isqrt(n * d * 4 ** bits), d * 2 ** bits)


class Opt:
    """kind "sgd": lr, mu, wd (coupled).  kind "adamw": lr, b1, b2, eps, wd
    (decoupled), t = 1-based update count.  All values exact rationals."""

    def __init__(self, kind, lr, mu=0, wd=0, b2=0, eps=0, t=1):
        self.kind = kind
        self.lr, self.mu, self.wd = Fraction(lr), Fraction(mu), Fraction(wd)
        self.b2, self.eps, self.t = Fraction(b2), Fraction(eps), int(t)


class State:
    """One coordinate column per list entry: params[i][p], mom[i][p],
    mom2[i][p] (AdamW second moments), u[p] (SlowMo state), ref[p] (anchor)."""

    def __init__(self, theta0, W, param_dt, mom_dt, aux_dt):
        self.pdt, self.mdt, self.adt = param_dt, mom_dt, aux_dt
        th = [store(param_dt, Fraction(x)) for x in theta0]
        self.params = [list(th) for _ in range(W)]
        self.mom = [[Fraction(0)] * len(th) for _ in range(W)]
        self.mom2 = [[Fraction(0)] * len(th) for _ in range(W)]
        self.u = [Fraction(0)] * len(th)
        self.ref = [store(aux_dt, x) for x in th]
        self.W, self.P = W, len(th)


def _update(st: State, o: Opt, i: int, p: int, g: Fraction) -> None:
    """One replica's optimizer step at one coordinate (framework semantics,
    each written tensor stored in its type)."""
    th, m = st.params[i][p], st.mom[i][p]
    if o.kind == "sgd":
        d = store(st.adt, g + o.wd * th) if o.wd != 0 else g   # gradient tensor
        m = store(st.mdt, o.mu * m + d)                        # momentum buffer
        th = store(st.pdt, th - o.lr * m)                      # parameter
    else:
        v = st.mom2[i][p]
        f32 = lambda x: store("f32", x)  # noqa: E731  fp32 scalars of the fp32 tensor ops
        if o.wd != 0:
            th = store(st.pdt, th * f32(1 - o.lr * o.wd))      # decoupled decay
        m = store(st.mdt, o.mu * m + (1 - o.mu) * g)           # first moment
        v = store(st.mdt, o.b2 * v + (1 - o.b2) * g * g)       # second moment
        step_size = f32(o.lr / (1 - o.mu ** o.t))
        sqrt_bc2 = f32(sqrt(1 - o.b2 ** o.t))
        th = store(st.pdt, th - step_size * m / (sqrt(v) / sqrt_bc2 + o.eps))
        st.mom2[i][p] = v
    st.params[i][p], st.mom[i][p] = th, m


def local_step(st: State, grads, o: Opt) -> None:
    for i in range(st.W):
        for p in range(st.P):
            _update(st, o, i, p, Fraction(grads[i][p]))


def sync_step(st: State, method: str, grads, o: Opt, beta=0, alpha=1, flags: int = 0,
              write_anchor: bool = True):
    """Synchronisation step; returns the gradient rows afterwards (the mean
    written back when flags & 1, CPDP and DDP only).  flags & 2 replaces every
    replica's optimizer state by the replica mean after the step."""
    beta, alpha = Fraction(beta), Fraction(alpha)
    W = st.W
    g = [[Fraction(x) for x in row] for row in grads]
    for p in range(st.P):
        gbar = None
        if method != "localsgd":
            gbar = store(st.adt, sum(g[i][p] for i in range(W)) / W)
        for i in range(W):
            _update(st, o, i, p, g[i][p] if method == "localsgd" else gbar)
        if flags & 1 and method != "localsgd":
            for i in range(W):
                g[i][p] = gbar
        if flags & 2:
            mm = store(st.mdt, sum(st.mom[i][p] for i in range(W)) / W)
            vm = store(st.mdt, sum(st.mom2[i][p] for i in range(W)) / W)
            for i in range(W):
                st.mom[i][p] = mm
                if o.kind == "adamw":
                    st.mom2[i][p] = vm
        if method == "ddp":
            continue
        avg = sum(st.params[i][p] for i in range(W)) / W
        if method == "cpdp":
            u = store(st.adt, beta * st.u[p] + (st.ref[p] - avg) / o.lr)
            new = store(st.adt, st.ref[p] - alpha * o.lr * u)
            st.u[p], st.ref[p] = u, new
        else:
            new = store(st.adt, avg)
            if write_anchor:
                st.ref[p] = new
        for i in range(W):
            st.params[i][p] = store(st.pdt, new)
    return g


def sync_vform(st: State, grads, o: Opt, beta) -> None:
    """CPDP synchronisation in the paper's own SlowMo variables (Sec. 3.3):
    Delta = mean - ref, v <- beta v + Delta, new = ref + v; st.u holds v."""
    beta = Fraction(beta)
    W = st.W
    for p in range(st.P):
        gbar = store(st.adt, sum(Fraction(grads[i][p]) for i in range(W)) / W)
        for i in range(W):
            _update(st, o, i, p, gbar)
        avg = sum(st.params[i][p] for i in range(W)) / W
        v = store(st.adt, beta * st.u[p] + (avg - st.ref[p]))
        new = store(st.adt, st.ref[p] + v)
        st.u[p], st.ref[p] = v, new
        for i in range(W):
            st.params[i][p] = store(st.pdt, new)
