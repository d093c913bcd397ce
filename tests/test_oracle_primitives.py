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


def test_rope_pair_frequencies_worked_example():
    # theta = 64, hd = 6: pair f turns by p * 64^(-2f/6) = p / 4^f, so the unit
    # vector on coordinate f goes to cos(p / 4^f) e_f + sin(p / 4^f) e_(f+3)
    hd, p = 6, 3
    for f in range(3):
        e = np.zeros((1, 1, hd))
        e[..., f] = 1.0
        r = M.rope(e, np.array([p]), 64.0)[0, 0]
        want = np.zeros(hd)
        want[f], want[f + 3] = math.cos(p / 4 ** f), math.sin(p / 4 ** f)
        np.testing.assert_allclose(r, want, atol=1e-14)


def _one_layer(**dims):
    """A one-layer oracle model of the given dimensions with zero weights
    (tests set the matrices they use) and unit norm gains."""
    import dataclasses
    import workloads as W
    cfg = dataclasses.replace(W.config("tiny"), L=1, eps=0.0, qk_norm=False, dtype="f32",
                              **dims)
    w = {("embed", -1): np.zeros((cfg.vocab, cfg.d)), ("lm_head", -1): np.zeros((cfg.vocab, cfg.d))}
    shapes = {"wq": (cfg.hq * cfg.hd, cfg.d), "wk": (cfg.hkv * cfg.hd, cfg.d),
              "wv": (cfg.hkv * cfg.hd, cfg.d), "wo": (cfg.d, cfg.hq * cfg.hd),
              "w_gate": (cfg.ffn, cfg.d), "w_up": (cfg.ffn, cfg.d), "w_down": (cfg.d, cfg.ffn)}
    for k, sh in shapes.items():
        w[(k, 0)] = np.zeros(sh)
    return M.Model(cfg, w)


def test_swiglu_mlp_sublayer_worked_example():
    # x = (3, 4), rms = sqrt(12.5); the gate row reads h0, the up row h1, the
    # down column is (1, 2): out = x + (1, 2) * silu(h0) * h1 (hand-computed;
    # gate and up exchanged would give 3.72585 in the first entry)
    m = _one_layer(d=2, ffn=1, hq=1, hkv=1, hd=2, vocab=4)
    W0 = m.layers[0]
    W0["w_gate"][:] = [[1.0, 0.0]]
    W0["w_up"][:] = [[0.0, 1.0]]
    W0["w_down"][:] = [[1.0], [2.0]]
    out = M.mlp_sublayer(m, 0, np.array([[3.0, 4.0]]))
    np.testing.assert_allclose(out[0], [3.6722479628067237, 5.344495925613447], rtol=1e-13)


def test_attention_sublayer_first_position_worked_example():
    # one cached position: every head's softmax is 1, so the output is
    # x + Wo (v, v) with v = Wv rmsnorm(x) (no rotation of values).  x = (1, 2, 3, 4),
    # rms = sqrt(7.5); Wv picks h0 and h3; Wo is not symmetric (its transpose
    # would give 4.92119 in the second entry)
    m = _one_layer(d=4, hq=2, hkv=1, hd=2, ffn=2, vocab=4)
    W0 = m.layers[0]
    W0["wq"][:] = np.arange(16.0).reshape(4, 4) / 7.0
    W0["wk"][:] = np.arange(8.0).reshape(2, 4) / 5.0
    W0["wv"][:] = [[1.0, 0, 0, 0], [0, 0, 0, 1.0]]
    W0["wo"][:] = [[1.0, 0, 0, 0], [0, 0, 1.0, 0], [0, 0, 0, 3.0], [0, 2.0, 0, 0]]
    cache = M.KVCache(m.cfg, 4)
    out = M.attn_sublayer(m, 0, np.array([[1.0, 2.0, 3.0, 4.0]]), np.array([0]), cache, "write")
    np.testing.assert_allclose(out[0], [1.3651483716701107, 2.3651483716701107,
                                        7.381780460041329, 6.921186973360886], rtol=1e-13)


def test_head_worked_example():
    # final RMSNorm then the head rows e0, e1, -e0: logits (3, 4, -3) / sqrt(12.5),
    # argmax 1, top-1 probability 1 / sum exp(l - l_max) = 0.52862
    m = _one_layer(d=2, ffn=1, hq=1, hkv=1, hd=2, vocab=3)
    m.lm_head = np.array([[1.0, 0.0], [0.0, 1.0], [-1.0, 0.0]])
    logits, am, top1 = M.head(m, np.array([[3.0, 4.0]]))
    np.testing.assert_allclose(logits[0], [0.848528137423857, 1.131370849898476,
                                           -0.848528137423857], rtol=1e-14)
    assert am[0] == 1
    assert top1[0] == pytest.approx(0.5286190379315163, rel=1e-13)


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
