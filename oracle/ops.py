"""Building blocks of the decoder, float64, written for clarity rather than speed.

The paper only fixes the residual form x_{l+1} = x_l + f_l(x_l) and the LM head o = g(x_L)
(Sec. "SSD Setup for VLMs"); the blocks below follow the public T5-v1.1 and LLaMA-2
definitions that the evaluated decoders (FlanT5-xl in BLIP-2, LLaMA-2 in LLaVA-1.5) use.

Pins (tests/test_oracle_ops.py): unit RMS / zero-mean-unit-variance outputs, hand-worked
values, GELU-tanh against the erf GELU within the approximation's known error, SiLU against
scipy's logistic, bucket thresholds against an exact integer derivation
(tests/golden/t5_buckets.txt), RoPE against complex multiplication and the relative-position
identity, attention against one-key / equal-score / dominant-key closed forms.
"""
from __future__ import annotations

import math

import numpy as np


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """T5 / LLaMA RMSNorm: gain * x / sqrt(mean(x^2) + eps), over the last axis (no centring)."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return gain * (x / np.sqrt(ms + eps))


def layer_norm(x: np.ndarray, gain: np.ndarray, shift: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm with biased variance: gain * (x - mean) / sqrt(var + eps) + shift."""
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return gain * ((x - mu) / np.sqrt(var + eps)) + shift


def gelu_tanh(u: np.ndarray) -> np.ndarray:
    """The tanh approximation of GELU used by T5-v1.1's gated FFN."""
    return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u ** 3)))


def silu(u: np.ndarray) -> np.ndarray:
    """x * sigmoid(x), LLaMA's FFN activation."""
    return u / (1.0 + np.exp(-u))


def relative_bucket(n: int, num_buckets: int, max_distance: int) -> int:
    """T5 decoder (unidirectional) relative-position bucket for query-minus-key distance n >= 0.

    The first half of the buckets hold the distances 0..num_buckets/2-1 exactly; beyond that the
    distance is binned logarithmically up to max_distance, and everything further shares the last
    bucket.
    """
    if n < 0:
        raise ValueError("decoder self-attention never looks ahead")
    exact = num_buckets // 2
    if n < exact:
        return n
    log_bin = int(math.log(n / exact) / math.log(max_distance / exact) * (num_buckets - exact))
    return min(exact + log_bin, num_buckets - 1)


def rope(v: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotary embedding of one position, half-split pairing (i, i + dh/2), angle pos*theta^(-2i/dh).

    ``v`` has head_dim as its last axis; any leading axes (heads) are rotated alike.
    """
    dh = v.shape[-1]
    half = dh // 2
    i = np.arange(half, dtype=np.float64)
    ang = pos * theta ** (-2.0 * i / dh)
    c, s = np.cos(ang), np.sin(ang)
    a, b = v[..., :half], v[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def softmax(s: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def attend(q: np.ndarray, keys: np.ndarray, values: np.ndarray, bias, scale: float) -> np.ndarray:
    """Multi-head softmax attention of one query position.

    q [H, dh]; keys, values [n, H, dh]; bias [H, n] or None.  Per head h:
    weights = softmax_j(scale * q_h . k_{j,h} + bias[h, j]), output = sum_j weights_j v_{j,h}.
    """
    scores = np.einsum("hd,nhd->hn", q, keys) * scale
    if bias is not None:
        scores = scores + bias
    w = softmax(scores, axis=-1)
    return np.einsum("hn,nhd->hd", w, values)
