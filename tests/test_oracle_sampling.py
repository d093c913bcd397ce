"""Pins of the oracle's speculative sampling (no GPU): the Philox4x32-10
generator against its published known-answer vectors, the filter's special
cases, the inverse-CDF draw, the distribution identity of the acceptance rule
(exact integration over u and a Monte Carlo check of the chain over Philox
streams), and reductions to greedy decoding."""
import os

import numpy as np
import pytest
from scipy import special, stats

import workloads as W
from oracle import model as M
from oracle import sampling as S

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_philox_known_answers():
    rows = [l.split() for l in open(os.path.join(GOLD, "philox4x32_10_kat.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        w = [int(x, 16) for x in r]
        ctr = np.array(w[0:4], dtype=np.uint64)
        key = np.array(w[4:6], dtype=np.uint64)
        assert S.philox4x32_10(ctr, key).tolist() == w[6:10]


def test_uniform_grid_range_and_streams():
    pos = np.arange(200000)
    u = S.uniform(12345, pos, 1)
    assert u.min() >= 0.0 and u.max() < 1.0
    assert np.all(u * 2.0 ** 24 == np.floor(u * 2.0 ** 24))
    assert abs(u.mean() - 0.5) < 3e-3 and abs(u.var() - 1 / 12) < 2e-3
    # the top 24 bits of the first output word of counter (pos, purpose, 0, 0)
    k = np.array([12345, 0], dtype=np.uint64)
    w = S.philox4x32_10(np.array([77, 1, 0, 0], dtype=np.uint64), k)[0]
    assert S.uniform(12345, 77, 1) == (int(w) >> 8) / 2.0 ** 24
    # purposes and seeds give different streams
    assert not np.array_equal(u[:64], S.uniform(12345, pos[:64], 2))
    assert not np.array_equal(u[:64], S.uniform(12346, pos[:64], 1))
    # the seed's high word is the key's second word
    hi = (5 << 32) | 9
    kk = np.array([9, 5], dtype=np.uint64)
    w = S.philox4x32_10(np.array([3, 0, 0, 0], dtype=np.uint64), kk)[0]
    assert S.uniform(hi, 3, 0) == (int(w) >> 8) / 2.0 ** 24


def test_filter_top_k_one_is_argmax():
    rng = np.random.default_rng(0)
    for _ in range(20):
        z = rng.normal(size=300)
        ids, pr = S.filtered(z, S.SamplingParams(0.7, 1, 0.95))
        assert ids.tolist() == [int(np.argmax(z))] and pr.tolist() == [1.0]
    z = np.zeros(10)
    z[[7, 3]] = 2.0
    assert S.filtered(z, S.SamplingParams(1.0, 1, 1.0))[0].tolist() == [3]


def test_filter_without_cuts_is_softmax():
    rng = np.random.default_rng(1)
    z = rng.normal(size=500) * 3
    for T in (0.7, 1.0, 2.5):
        ids, pr = S.filtered(z, S.SamplingParams(T, 0, 1.0))
        ref = special.softmax(z / T)
        assert sorted(ids.tolist()) == list(range(500))
        np.testing.assert_allclose(pr, ref[ids], rtol=1e-12, atol=0)
        assert np.all(np.diff(pr) <= 0)


def test_filter_top_k_renormalises_the_k_largest():
    rng = np.random.default_rng(2)
    z = rng.normal(size=400)
    ids, pr = S.filtered(z, S.SamplingParams(0.7, 50, 1.0))
    top = np.argsort(-z)[:50]
    assert ids.tolist() == top.tolist()
    ref = special.softmax(z[top] / 0.7)
    np.testing.assert_allclose(pr, ref, rtol=1e-12)


def test_filter_top_p_keeps_shortest_sufficient_prefix():
    p = np.array([0.05, 0.5, 0.15, 0.3])  # ids sorted by p: 1, 3, 2, 0
    z = np.log(p)
    for top_p, keep in ((0.49, [1]), (0.79, [1, 3]), (0.81, [1, 3, 2]), (0.96, [1, 3, 2, 0]),
                        (1.0, [1, 3, 2, 0])):
        ids, pr = S.filtered(z, S.SamplingParams(1.0, 0, top_p))
        assert ids.tolist() == keep, top_p
        np.testing.assert_allclose(pr, p[keep] / p[keep].sum(), rtol=1e-12)
    ids, pr = S.filtered(z, S.SamplingParams(1.0, 3, 0.96))  # top-k applies first
    assert ids.tolist() == [1, 3, 2]
    np.testing.assert_allclose(pr, p[[1, 3, 2]] / 0.95, rtol=1e-12)


def test_filter_ties_and_temperature():
    z = np.array([0.0, 1.0, 3.0, 1.0, 3.0, -2.0])
    ids, pr = S.filtered(z, S.SamplingParams(1.0, 4, 1.0))
    assert ids.tolist() == [2, 4, 1, 3]
    assert pr[0] == pr[1] and pr[2] == pr[3]
    rng = np.random.default_rng(3)
    z = rng.normal(size=200)
    a = S.filtered(z, S.SamplingParams(0.5, 30, 0.9))
    b = S.filtered(2.0 * z, S.SamplingParams(1.0, 30, 0.9))
    assert a[0].tolist() == b[0].tolist()
    np.testing.assert_allclose(a[1], b[1], rtol=1e-12)
    # temperature <= 0: greedy point mass
    assert S.filtered(z, S.SamplingParams(0.0, 30, 0.9))[0].tolist() == [int(np.argmax(z))]


def test_draw_is_inverse_cdf_in_table_order():
    ids, pr = np.array([7, 3, 9]), np.array([0.25, 0.5, 0.25])
    for u, t in ((0.0, 7), (0.2499, 7), (0.25, 3), (0.7499, 3), (0.75, 9), (1 - 2 ** -24, 9)):
        assert S.draw(ids, pr, u) == t, u


def _tab(d):
    ids = np.array(list(d.keys()))
    pr = np.array(list(d.values()), dtype=np.float64)
    return ids, pr / pr.sum()


def test_acceptance_rule_preserves_target_exactly():
    """Marginalising the accept/resample step over x ~ q and u gives p: the
    speculative sampling identity, computed by integrating the oracle's decisions
    over a midpoint grid of u (error below 1/N per term)."""
    p = _tab({4: 0.4, 1: 0.25, 9: 0.2, 6: 0.15})      # target
    q = _tab({4: 0.1, 1: 0.5, 9: 0.05, 2: 0.35})      # draft (2 is outside p's support)
    N = 4096
    grid = (np.arange(N) + 0.5) / N
    out = {}
    for x, qx in zip(*q):
        acc = sum(S.accept_or_resample(p, q, int(x), u, 0.5)[0] for u in grid) / N
        out[int(x)] = out.get(int(x), 0.0) + qx * acc
        rej = {}
        for u in grid:
            ok, y = S.accept_or_resample(p, q, int(x), 1.0 - 2 ** -24, u)
            assert not ok or S.prob_of(*p, int(x)) >= S.prob_of(*q, int(x))
            rej[y] = rej.get(y, 0) + 1.0 / N
        if acc < 1.0:
            for y, f in rej.items():
                out[y] = out.get(y, 0.0) + qx * (1 - acc) * f
    for y, py in zip(*p):
        assert out.get(int(y), 0.0) == pytest.approx(py, abs=3.0 / N)
    assert out.get(2, 0.0) == 0.0


def test_verify_chain_monte_carlo():
    """Chain of three drafts with context-free p and q over Philox streams: the
    first emitted token, and the second one given a first acceptance, follow p
    (chi-square, p-value above 1e-4)."""
    p = _tab({0: 0.35, 1: 0.3, 2: 0.2, 3: 0.1, 4: 0.05})
    q = _tab({0: 0.1, 1: 0.4, 2: 0.3, 3: 0.1, 5: 0.1})
    P = 100
    first, second = np.zeros(6), np.zeros(6)
    for seed in range(6000):
        drafts = [S.draw(*q, S.uniform(seed, P + i + 1, 0)) for i in range(3)]
        a, fin = S.verify_chain([p] * 4, [q] * 3, drafts, seed, P)
        em = drafts[:a] + [fin]
        first[em[0]] += 1
        if len(em) >= 2:
            second[em[1]] += 1
    for h in (first, second):
        assert h[5] == 0
        exp = p[1] * h.sum()
        chi = ((h[:5] - exp) ** 2 / exp).sum()
        assert chi < stats.chi2.ppf(1 - 1e-4, 4), (h, exp)


@pytest.fixture(scope="module")
def tiny():
    cfg = W.config("tiny")
    return M.Model(cfg, W.generate_weights(cfg, seed=0)), W.prompt_ids(cfg.vocab, 48, 1)


def test_top_k_one_reduces_to_greedy(tiny):
    model, prompt = tiny
    prm = S.SamplingParams(0.7, 1, 0.95, seed=5)
    assert S.ar_sample(model, prompt, 12, 100, prm) == M.generate_ar(model, prompt, 12, 100)
    mask = [True, False, True, True, False, True, True, True]
    sg = M.prefill(model, prompt, 100, 25)
    ss = S.prefill(model, prompt, 100, 25, prm)
    assert ss.s == sg.s
    for _ in range(4):
        rg = M.ssd_round(model, sg, mask, 4)
        rs = S.spec_round(model, ss, mask, 4, prm)
        assert (rs.drafts, rs.n_accepted, rs.emitted) == (rg.drafts, rg.n_accepted, rg.emitted)
    for bg, bs in zip(sg.blocks, ss.blocks):
        assert np.array_equal(bg[0], bs[0])


def test_empty_skip_set_accepts_every_draft(tiny):
    model, prompt = tiny
    st = S.prefill(model, prompt, 100, 25, S.SamplingParams(seed=3))
    for _ in range(3):
        rd = S.spec_round(model, st, [True] * 8, 4, S.SamplingParams(seed=3))
        assert rd.n_accepted == 4 and len(rd.emitted) == 5


def test_sampled_generation_stays_in_target_support(tiny):
    """Every emitted token has nonzero probability under the filtered target
    distribution of its prefix; the first token is the prefill's draw; output is
    a function of the seed."""
    model, prompt = tiny
    prm = S.SamplingParams(0.7, 50, 0.95, seed=11)
    out, log = S.generate(model, prompt, 24, 4, 8, W.TINY_LATENCY, prm, quant_mode="bins",
                          bins=64)
    assert len(log.selections) >= 2 and sum(log.accepted) >= 1
    cache = M.KVCache(model.cfg, 128)
    fw = M.forward(model, cache, list(prompt) + out, 0)
    n = len(prompt)
    ids0, pr0 = S.filtered(fw.logits[n - 1], prm)
    assert out[0] == S.draw(ids0, pr0, S.uniform(11, n, 2))
    for t, tok in enumerate(out):
        ids, _ = S.filtered(fw.logits[n - 1 + t], prm)
        assert tok in ids.tolist(), t
    again, _ = S.generate(model, prompt, 24, 4, 8, W.TINY_LATENCY, prm, quant_mode="bins",
                          bins=64)
    assert again == out
    other, _ = S.generate(model, prompt, 24, 4, 8, W.TINY_LATENCY,
                          S.SamplingParams(0.7, 50, 0.95, seed=12), quant_mode="bins", bins=64)
    assert other != out


def test_margins_are_recorded(tiny):
    model, prompt = tiny
    mg = []
    S.ar_sample(model, prompt, 6, 100, S.SamplingParams(0.7, 50, 0.95, seed=2), mg)
    assert len(mg) >= 6 and all(m >= 0 for m in mg)
