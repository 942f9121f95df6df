"""Seeded synthetic inputs, host side (numpy).

This module holds none of the CPDP arithmetic: it only draws the numbers that
stand in for the initial model and for backward-pass gradients.  The same
generator is implemented for the device in ``synth/synth.hip``; both follow the
definition below, and a GPU test checks that they agree bit for bit.

Definition
----------
mix64(z)        SplitMix64 output function (Steele, Lea, Flood, "Fast
                splittable pseudorandom number generators", OOPSLA 2014):
                z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
                z *= 0x94D049BB133111EB; z ^= z >> 31   (all mod 2^64).
stream key      key(seed, kind, t, i) =
                mix64(mix64(mix64(seed ^ kind*C1) ^ t*C2) ^ i*C3)
                kind 0 = initial parameters, 1 = gradients; t = 1-based step;
                i = worker (replica) index.
word j of p     h_j(p) = mix64(key + (4p + j + 1) * GAMMA), j = 0..3,
                i.e. SplitMix64's sequence started at ``key``.
normal          S = sum of the twelve 16-bit fields of h_0, h_1, h_2;
                z = (S - 393210) * 2^-16  (Irwin-Hall, n = 12: mean 0, sd ~1,
                exact in fp32), value = fp32(z * fp32(sigma)) (one RNE multiply).
outlier         if the low 32 bits of h_3 are below round(rate * 2^32) the
                value becomes fp32(value * fp32(scale)).
"""
from __future__ import annotations

import numpy as np

M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
C1 = 0xD1B54A32D192ED03
C2 = 0xABC98388FB8FAC03
C3 = 0x8CB92BA72F3D8DD7
KIND_THETA0 = 0
KIND_GRAD = 1
IRWIN_HALL_MEAN = 393210  # 12 fields x mean 32767.5


def mix64_int(z: int) -> int:
    z &= M64
    z ^= z >> 30
    z = (z * 0xBF58476D1CE4E5B9) & M64
    z ^= z >> 27
    z = (z * 0x94D049BB133111EB) & M64
    z ^= z >> 31
    return z


def stream_key(seed: int, kind: int, t: int, i: int) -> int:
    k = mix64_int(seed ^ ((kind * C1) & M64))
    k = mix64_int(k ^ ((t * C2) & M64))
    return mix64_int(k ^ ((i * C3) & M64))


def _mix64(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * np.uint64(0xBF58476D1CE4E5B9)
    z = z ^ (z >> np.uint64(27))
    z = z * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def outlier_threshold(rate: float) -> int:
    return int(round(rate * 2.0 ** 32))


def normal(key: int, idx, sigma: float, outlier_rate: float = 0.0,
           outlier_scale: float = 100.0) -> np.ndarray:
    """fp32 draws for coordinates ``idx`` (any int array) of stream ``key``."""
    idx = np.asarray(idx, dtype=np.uint64)
    with np.errstate(over="ignore"):
        base = np.uint64(key) + (np.uint64(4) * idx) * np.uint64(GAMMA)
        s = np.zeros(idx.shape, dtype=np.int64)
        for j in range(3):
            h = _mix64(base + np.uint64(j + 1) * np.uint64(GAMMA))
            for f in range(4):
                s += ((h >> np.uint64(16 * f)) & np.uint64(0xFFFF)).astype(np.int64)
        z = ((s - IRWIN_HALL_MEAN).astype(np.float32)
             * np.float32(2.0 ** -16))
        v = z * np.float32(sigma)
        if outlier_rate > 0.0:
            h3 = _mix64(base + np.uint64(4) * np.uint64(GAMMA))
            hit = (h3 & np.uint64(0xFFFFFFFF)) < np.uint64(
                outlier_threshold(outlier_rate))
            v = np.where(hit, v * np.float32(outlier_scale), v).astype(np.float32)
    return v.astype(np.float32)


def theta0(seed: int, idx, sigma: float = 0.02) -> np.ndarray:
    return normal(stream_key(seed, KIND_THETA0, 0, 0), idx, sigma)


def grads(seed: int, step: int, W: int, idx, sigma: float = 1e-3,
          outlier_rate: float = 0.0, outlier_scale: float = 100.0) -> np.ndarray:
    """(W, len(idx)) fp32 gradients of 1-based step ``step``."""
    return np.stack([normal(stream_key(seed, KIND_GRAD, step, i), idx, sigma,
                            outlier_rate, outlier_scale) for i in range(W)])


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returned as fp32."""
    x = np.asarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    r = ((b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1)))
         & np.uint64(0xFFFF0000)).astype(np.uint32)
    out = r.view(np.float32)
    return np.where(np.isnan(x), x, out).astype(np.float32)
