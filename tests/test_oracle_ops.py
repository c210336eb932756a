"""Pins of the oracle's building blocks against closed forms, library routines and exact tables."""
import math
import os

import numpy as np
import pytest
import scipy.special

from oracle import ops

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---- RMSNorm / LayerNorm -------------------------------------------------------------------

def test_rms_norm_hand_value():
    # x = (3, 4): mean square 12.5, so x / sqrt(12.5)
    y = ops.rms_norm(np.array([3.0, 4.0]), np.array([1.0, 2.0]), 0.0)
    r = math.sqrt(12.5)
    assert np.allclose(y, [3.0 / r, 8.0 / r], rtol=0, atol=1e-15)


def test_rms_norm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 64)) * 7.0
    y = ops.rms_norm(x, np.ones(64), 0.0)
    assert np.allclose(np.mean(y * y, axis=-1), 1.0, atol=1e-12)
    assert np.allclose(ops.rms_norm(3.5 * x, np.ones(64), 0.0), y, atol=1e-12)
    # no centring: adding a constant changes the output
    assert not np.allclose(ops.rms_norm(x + 1.0, np.ones(64), 0.0), y + 0.0, atol=1e-3)
    # eps enters under the root
    z = ops.rms_norm(np.array([0.0, 0.0]), np.ones(2), 1e-6)
    assert np.all(z == 0.0)
    w = ops.rms_norm(np.array([1e-3, 1e-3]), np.ones(2), 1e-6)
    assert np.allclose(w, 1e-3 / math.sqrt(1e-6 + 1e-6), rtol=1e-12)


def test_layer_norm_hand_value_and_moments():
    y = ops.layer_norm(np.array([1.0, 2.0, 3.0]), np.ones(3), np.zeros(3), 0.0)
    assert np.allclose(y, [-math.sqrt(1.5), 0.0, math.sqrt(1.5)], atol=1e-14)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((4, 100)) * 3 + 5
    y = ops.layer_norm(x, np.ones(100), np.zeros(100), 0.0)
    assert np.allclose(y.mean(-1), 0.0, atol=1e-12)
    assert np.allclose(y.var(-1), 1.0, atol=1e-12)  # biased variance
    g, b = rng.standard_normal(100), rng.standard_normal(100)
    assert np.allclose(ops.layer_norm(x, g, b, 0.0), g * y + b, atol=1e-12)


# ---- activations ---------------------------------------------------------------------------

def test_gelu_tanh_against_erf_gelu():
    u = np.linspace(-8, 8, 20001)
    exact = 0.5 * u * (1 + scipy.special.erf(u / math.sqrt(2)))
    approx = ops.gelu_tanh(u)
    # the tanh form approximates the erf GELU to within about 5e-4 everywhere
    assert np.max(np.abs(approx - exact)) < 1e-3
    assert np.max(np.abs(approx - exact)) > 1e-5  # it is the approximation, not erf itself
    assert ops.gelu_tanh(np.array([0.0]))[0] == 0.0


def test_gelu_tanh_odd_part_identity():
    # 0.5 u (1 + tanh(a)) - 0.5 (-u) (1 + tanh(-a)) == u for any odd inner function a(u)
    u = np.linspace(-5, 5, 101)
    assert np.allclose(ops.gelu_tanh(u) - ops.gelu_tanh(-u), u, atol=1e-13)


def test_silu_against_logistic():
    u = np.linspace(-30, 30, 601)
    assert np.allclose(ops.silu(u), u * scipy.special.expit(u), rtol=1e-13, atol=1e-300)


# ---- relative-position buckets -------------------------------------------------------------

def _golden_buckets():
    rows = []
    with open(os.path.join(GOLDEN, "t5_buckets.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                b, n = line.split()
                rows.append((int(b), int(n)))
    return rows


def test_bucket_thresholds_match_golden_table():
    for b, n in _golden_buckets():
        assert ops.relative_bucket(n, 32, 128) == b, (b, n)
        if n > 0:
            assert ops.relative_bucket(n - 1, 32, 128) == b - 1, (b, n)


def test_bucket_thresholds_exact_integer_derivation():
    # bucket 16 + j is first reached at the least n with n^16 >= 16^16 * 8^j
    first = {}
    for n in range(0, 200):
        first.setdefault(ops.relative_bucket(n, 32, 128), n)
    for j in range(1, 16):
        n = 16
        while n ** 16 < 16 ** 16 * 8 ** j:
            n += 1
        assert first[16 + j] == n, j
    assert all(ops.relative_bucket(n, 32, 128) == 31 for n in range(113, 5000, 7))


def test_bucket_monotone_and_rejects_lookahead():
    prev = 0
    for n in range(0, 3000):
        b = ops.relative_bucket(n, 32, 128)
        assert prev <= b <= 31
        prev = b
    with pytest.raises(ValueError):
        ops.relative_bucket(-1, 32, 128)


# ---- rotary embedding ----------------------------------------------------------------------

def test_rope_against_complex_rotation():
    rng = np.random.default_rng(3)
    dh, theta = 16, 10000.0
    v = rng.standard_normal((3, dh))
    for p in (0, 1, 7, 613):
        half = dh // 2
        zc = v[:, :half] + 1j * v[:, half:]
        freqs = np.array([theta ** (-(2 * i) / dh) for i in range(half)])
        rot = zc * np.exp(1j * p * freqs)
        want = np.concatenate([rot.real, rot.imag], axis=-1)
        assert np.allclose(ops.rope(v, p, theta), want, atol=1e-12)


def test_rope_hand_values():
    # dh = 4: frequencies 1 and theta^(-1/2) = 0.01
    p = 3
    y = ops.rope(np.array([1.0, 0.0, 0.0, 0.0]), p, 10000.0)
    assert np.allclose(y, [math.cos(3), 0, math.sin(3), 0], atol=1e-14)
    y = ops.rope(np.array([0.0, 1.0, 0.0, 0.0]), p, 10000.0)
    assert np.allclose(y, [0, math.cos(0.03), 0, math.sin(0.03)], atol=1e-14)


def test_rope_relative_identity_and_norm():
    rng = np.random.default_rng(4)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    for p, pp in ((5, 2), (700, 11), (9, 9)):
        lhs = ops.rope(q, p, 1e4) @ ops.rope(k, pp, 1e4)
        rhs = ops.rope(q, p - pp, 1e4) @ k
        assert abs(lhs - rhs) < 1e-9
    assert np.allclose(ops.rope(q, 0, 1e4), q, atol=0)
    assert abs(np.linalg.norm(ops.rope(q, 123, 1e4)) - np.linalg.norm(q)) < 1e-12


# ---- attention -----------------------------------------------------------------------------

def test_attend_one_key_returns_value():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((3, 8))
    K, V = rng.standard_normal((1, 3, 8)), rng.standard_normal((1, 3, 8))
    assert np.allclose(ops.attend(q, K, V, rng.standard_normal((3, 1)), 0.7), V[0], atol=1e-14)


def test_attend_equal_scores_mean_and_shift_invariance():
    rng = np.random.default_rng(6)
    K, V = rng.standard_normal((5, 2, 4)), rng.standard_normal((5, 2, 4))
    out = ops.attend(np.zeros((2, 4)), K, V, None, 1.0)
    assert np.allclose(out, V.mean(axis=0), atol=1e-14)
    q = rng.standard_normal((2, 4))
    b = rng.standard_normal((2, 5))
    assert np.allclose(ops.attend(q, K, V, b, 1.0), ops.attend(q, K, V, b + 40.0, 1.0), atol=1e-12)


def test_attend_scale_and_bias_closed_form():
    # two keys, head 0 scores 0 and ln 3 after scaling -> weights 1/4, 3/4
    scale = 0.125
    q = np.array([[1.0, 0.0]])
    K = np.array([[[0.0, 5.0]], [[math.log(3.0) / scale, 0.0]]])
    V = np.array([[[1.0, 2.0]], [[5.0, -2.0]]])
    assert np.allclose(ops.attend(q, K, V, None, scale)[0], [4.0, -1.0], atol=1e-13)
    # a dominant bias on one key selects it, per head
    bias = np.array([[0.0, -1e4]])
    assert np.allclose(ops.attend(q, K, V, bias, scale)[0], V[0, 0], atol=1e-12)


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(7)
    s = rng.standard_normal((4, 33)) * 50
    p = ops.softmax(s)
    assert np.allclose(p.sum(-1), 1.0, atol=1e-14) and np.all(p >= 0)
