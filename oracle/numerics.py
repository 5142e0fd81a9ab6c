"""Scalar numerics of the oracle, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

LN_EPS = 1e-5   # LayerNorm epsilon; the paper states none (reading in the design notes)


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    bf16 keeps 8 significant bits (1 implicit + 7 stored) and float32's
    exponent range.  With x = m * 2^e, 0.5 <= |m| < 1 (frexp), the nearest
    value with 8 significant bits is rint(m * 2^8) * 2^(e-8); numpy's rint
    rounds halves to even.  Results at or beyond the bf16 overflow threshold
    become +-inf; NaN stays NaN.  (Values below the normal range do not occur
    in these workloads and are rounded with full 8-bit precision.)
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    r = np.ldexp(np.rint(m * 256.0), e - 8)
    bf16_max = (2.0 - 2.0 ** -7) * 2.0 ** 127
    overflow_at = (2.0 - 2.0 ** -8) * 2.0 ** 127     # halfway to the next binade
    r = np.where(np.abs(x) >= overflow_at, np.copysign(np.inf, x), r)
    r = np.where(np.abs(r) > bf16_max, np.copysign(np.inf, x), r)
    return np.where(np.isnan(x), x, r)


def store(x, dtype: str):
    """Value of x after storage in `dtype` ("f32" is kept in float64: the fp32
    path is compared normwise against the unrounded float64 result)."""
    return round_bf16(x) if dtype == "bf16" else np.asarray(x, dtype=np.float64)


def layernorm(x, gamma, beta, eps: float = LN_EPS):
    """LayerNorm over the last (feature) axis: (x - mean) / sqrt(var + eps) *
    gamma + beta, with the biased variance (Sec. 3.3: normalisation acts on
    each row's static feature tail)."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * np.asarray(gamma, np.float64) + np.asarray(beta, np.float64)


def linear(x, w, b=None):
    """V' = V W^T + b (Sec. 3.3 "Dense work across valid positions"); W is [out, in]."""
    y = np.asarray(x, np.float64) @ np.asarray(w, np.float64).T
    return y if b is None else y + np.asarray(b, np.float64)


def silu(x):
    x = np.asarray(x, np.float64)
    return x / (1.0 + np.exp(-x))


def sigmoid(x):
    """1 / (1 + exp(-x)), evaluated without overflow for large |x|."""
    x = np.asarray(x, np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def gelu(x):
    """Exact (erf) GELU."""
    x = np.asarray(x, np.float64)
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def softmax(s, axis=-1):
    """exp(s_k) / sum_j exp(s_j), evaluated as exp(s_k - max) / sum exp(s_j - max)."""
    s = np.asarray(s, np.float64)
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=axis, keepdims=True)
