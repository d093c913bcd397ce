"""Pins of the oracle's primitives against closed forms, special cases and
independent library routines (no GPU)."""
import math

import numpy as np
import pytest
import scipy.special

from oracle import model as M
from oracle import select as SEL


def test_rmsnorm_closed_form():
    c, d, eps = 3.0, 16, 1e-6
    x = np.full(d, c)
    g = np.linspace(0.5, 2.0, d)
    out = M.rmsnorm(x, g, eps)
    np.testing.assert_allclose(out, c / math.sqrt(c * c + eps) * g, rtol=1e-15)
    # unit-RMS output for unit gains, independent of the input scale
    rng = np.random.default_rng(0)
    y = rng.standard_normal(64) * 7.0
    o = M.rmsnorm(y, np.ones(64), 0.0)
    assert abs(np.sqrt(np.mean(o ** 2)) - 1.0) < 1e-14
    np.testing.assert_allclose(M.rmsnorm(5 * y, np.ones(64), 0.0), o, rtol=1e-14)


def test_rope_two_dims_is_plane_rotation():
    # hd = 2: the single pair rotates by angle pos * theta^0 = pos.
    x = np.array([[0.3, -1.2]])
    for p in (0, 1, 5, 1000):
        r = M.rope(x[None], np.array([p]), 1e4)[0, 0]
        c, s = math.cos(p), math.sin(p)
        np.testing.assert_allclose(r, [0.3 * c + 1.2 * s, -1.2 * c + 0.3 * s], atol=1e-12)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(1)
    hd = 64
    q = rng.standard_normal((1, 1, hd))
    k = rng.standard_normal((1, 1, hd))
    np.testing.assert_allclose(M.rope(q, np.array([0]), 1e4), q, rtol=0, atol=0)
    for p in (1, 17, 8191):
        r = M.rope(q, np.array([p]), 5e5)
        np.testing.assert_allclose(np.linalg.norm(r), np.linalg.norm(q), rtol=1e-13)
    # q.k depends only on the position difference
    dots = []
    for base in (0, 10, 333):
        rq = M.rope(q, np.array([base + 7]), 1e4)
        rk = M.rope(k, np.array([base]), 1e4)
        dots.append(float(np.sum(rq * rk)))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-11)
    # the pair is (f, f + hd/2): a vector with only coordinate 0 set stays in span{0, hd/2}
    e0 = np.zeros((1, 1, hd))
    e0[..., 0] = 1.0
    r = M.rope(e0, np.array([3]), 1e4)[0, 0]
    assert np.count_nonzero(np.abs(r) > 1e-15) == 2 and abs(r[hd // 2]) > 0


def test_silu():
    x = np.linspace(-20, 20, 101)
    np.testing.assert_allclose(M.silu(x), x * scipy.special.expit(x), rtol=1e-13, atol=1e-300)
    assert M.silu(np.array([0.0]))[0] == 0.0


def test_attention_special_cases():
    rng = np.random.default_rng(2)
    hd = 16
    q = rng.standard_normal(hd)
    K = rng.standard_normal((1, hd))
    V = rng.standard_normal((1, hd))
    np.testing.assert_allclose(M.softmax_attention(q, K, V), V[0], rtol=1e-15)
    # equal keys -> mean of values
    K = np.tile(rng.standard_normal(hd), (9, 1))
    V = rng.standard_normal((9, hd))
    np.testing.assert_allclose(M.softmax_attention(q, K, V), V.mean(0), rtol=1e-13)
    # general case against scipy's softmax
    K = rng.standard_normal((50, hd))
    V = rng.standard_normal((50, hd))
    w = scipy.special.softmax(K @ q / math.sqrt(hd))
    np.testing.assert_allclose(M.softmax_attention(q, K, V), w @ V, rtol=1e-12)


def test_bf16_rounding():
    # exactly representable values are unchanged; halfway cases go to even
    vals = np.array([1.0, -2.5, 2.0 ** -15, 65280.0])
    np.testing.assert_array_equal(M.to_bf16(vals), vals)
    one_ulp = 2.0 ** -7  # bf16 spacing in [1, 2)
    assert M.to_bf16(np.array([1.0 + one_ulp / 2]))[0] == 1.0          # tie -> even
    assert M.to_bf16(np.array([1.0 + 1.5 * one_ulp]))[0] == 1.0 + 2 * one_ulp
    assert M.to_bf16(np.array([1.0 + 0.6 * one_ulp]))[0] == 1.0 + one_ulp


def test_cos_closed_forms():
    x = np.array([[1.0, 0.0], [3.0, 4.0], [1.0, 1.0], [0.0, 0.0]])
    y = np.array([[1.0, 1.0], [-3.0, -4.0], [2.0, 2.0], [1.0, 2.0]])
    c = SEL.cos_rows(x, y)
    np.testing.assert_allclose(c, [1 / math.sqrt(2), -1.0, 1.0, 0.0], rtol=1e-15)
    assert SEL.cos_matrix(x, y) == pytest.approx((1 / math.sqrt(2) - 1 + 1 + 0) / 4, rel=1e-15)
    assert SEL.cos_rows(np.array([[0.0, 1.0]]), np.array([[5.0, 0.0]]))[0] == 0.0


def test_expected_tokens_closed_form():
    for a in (0.0, 0.3, 0.9, 0.999):
        for g in range(0, 11):
            want = (1 - a ** (g + 1)) / (1 - a)
            assert SEL.expected_tokens(a, g) == pytest.approx(want, rel=1e-12)
    for g in range(0, 11):
        assert SEL.expected_tokens(1.0, g) == g + 1


def test_lemma1_cosine_bound_keeps_argmax():
    """Lemma 1: if |x'| = |x| and cos(x, x') >= 1 - xi^2 / (2|x|^2 max|w_i* - w_j|^2)
    the greedy token is unchanged."""
    rng = np.random.default_rng(3)
    for trial in range(200):
        V, d = 50, 12
        W = rng.standard_normal((V, d))
        x = rng.standard_normal(d)
        z = W @ x
        i = int(np.argmax(z))
        xi = z[i] - np.max(np.delete(z, i))
        dmax = np.max(np.linalg.norm(W[i] - np.delete(W, i, axis=0), axis=1))
        bound = 1 - xi ** 2 / (2 * np.dot(x, x) * dmax ** 2)
        # random x' on the sphere |x'| = |x| with cos(x, x') exactly at the bound
        u = rng.standard_normal(d)
        u -= u.dot(x) / x.dot(x) * x
        u /= np.linalg.norm(u)
        c = max(bound, -1.0)
        xp = np.linalg.norm(x) * (c * x / np.linalg.norm(x) + math.sqrt(1 - c * c) * u)
        assert abs(np.linalg.norm(xp) - np.linalg.norm(x)) < 1e-9
        assert int(np.argmax(W @ xp)) == i
