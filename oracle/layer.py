"""Plain CPU statement of the layer epilogue: residual addition and RMSNorm
after the reduce-scatter.

TEST INFRASTRUCTURE ONLY (imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path).

The paper's layer-level evaluation (Section 5.2, "Layer-Level Performance")
runs the attention output projection's GEMM and ReduceScatter followed by a
residual addition and RMSNorm.  Reading used here, per output row i of the
rank's chunk (N columns), with O the reduced chunk, R the residual stream
(bf16), gamma the RMSNorm weight (bf16, length N) and eps > 0:

    h[i, :] = O[i, :] + R[i, :]                     (new residual stream)
    y[i, :] = h[i, :] / sqrt(mean_j h[i, j]^2 + eps) * gamma

evaluated in float64 with no reordering.  The device path produces h in
bfloat16 and computes y from that bfloat16 h (the normalisation of the stored
residual stream), so its error against these exact values is bounded by
``h_bound`` and ``y_bound`` below.
"""
from __future__ import annotations

import numpy as np

from .reduce_scatter import U_BF16, U_F32, bf16_to_f64, f32_to_bf16_rne_bits


def residual_add(O: np.ndarray, R_bits) -> np.ndarray:
    """h = O + R in float64."""
    return np.asarray(O, dtype=np.float64) + bf16_to_f64(R_bits)


def rmsnorm(h: np.ndarray, gamma_bits, eps: float) -> np.ndarray:
    """y = h / sqrt(mean of squares over the row + eps) * gamma, float64."""
    h = np.asarray(h, dtype=np.float64)
    ms = np.mean(h * h, axis=1, keepdims=True)
    return h / np.sqrt(ms + eps) * bf16_to_f64(gamma_bits)[None, :]


def layer(O: np.ndarray, R_bits, gamma_bits, eps: float):
    """(h, y) of the layer epilogue for the reduced rows O."""
    h = residual_add(O, R_bits)
    return h, rmsnorm(h, gamma_bits, eps)


def h_bound(sum_bound: np.ndarray, h: np.ndarray, R_bits) -> np.ndarray:
    """Elementwise bound on |h_device - h| for a path that adds the residual
    to the float32 reduction (whose own error is ``sum_bound`` before any
    final rounding), in float32, then rounds to bfloat16: the sum's error,
    one float32 addition and one bfloat16 rounding, doubled for second-order
    terms."""
    return sum_bound + 2 * U_F32 * (np.abs(h) + bf16_to_f64(R_bits)) + 2 * U_BF16 * np.abs(h)


def y_bound(h: np.ndarray, hb: np.ndarray, gamma_bits, eps: float) -> np.ndarray:
    """Elementwise bound on |y_device - y| given the exact h and a bound hb on
    the device's h error.

    y = gamma h r with r = (mean h^2 + eps)^(-1/2).  The device normalises its
    own bfloat16 h (error <= hb), forms the mean of squares in float32 over N
    terms (relative error <= (N + 2) u32), takes a reciprocal square root
    (a few float32 ulps) and rounds gamma * h * r to bfloat16.  A change dm of
    the mean changes r by at most r |dm| / (2 (m + eps)) to first order, and
    dm <= mean(2 |h| hb + hb^2).  All first-order terms are doubled."""
    h = np.asarray(h, dtype=np.float64)
    N = h.shape[1]
    g = np.abs(bf16_to_f64(gamma_bits))[None, :]
    m = np.mean(h * h, axis=1, keepdims=True)
    r = 1.0 / np.sqrt(m + eps)
    dm = np.mean(2 * np.abs(h) * hb + hb * hb, axis=1, keepdims=True) + (N + 2) * U_F32 * m
    dr = r * dm / (2 * (m + eps)) + 8 * U_F32 * r
    y = np.abs(h) * r * g
    return 2 * (g * (hb * r + np.abs(h) * dr) + U_BF16 * y + 4 * U_F32 * y)


def residual_add_f32(partial_bits, peer_bits, R_bits) -> np.ndarray:
    """The reducer's own arithmetic for h on a given bf16 partial: start from
    the local contribution, add the peers in rank order, then the residual,
    each addition rounded to float32, and round to bfloat16.  Returns bf16
    bits; bit-exact by definition."""
    acc = bf16_to_f64(partial_bits).astype(np.float32)
    for pb in peer_bits:
        acc = (acc + bf16_to_f64(pb).astype(np.float32)).astype(np.float32)
    acc = (acc + bf16_to_f64(R_bits).astype(np.float32)).astype(np.float32)
    return f32_to_bf16_rne_bits(acc)
