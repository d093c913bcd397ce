"""GPU parity of speculative sampling: the Philox uniforms (bit-exact), the
T / top-k / top-p filter and its draws on the same logits as the oracle
(order and ids exact; probabilities 2e-5 relative; decisions compared where
the oracle's margin exceeds 1e-5), the acceptance chain, the distribution of
the emitted token, and sampled generation on the fp32 decoder against the
oracle.  Every call goes through the C ABI."""
import numpy as np
import pytest

import workloads as W
from oracle import model as M
from oracle import sampling as S
from tests.gpu_helpers import build

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

MARGIN = 1e-5


@pytest.fixture(scope="module")
def E():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_20217_amd import engine
    return engine


def test_uniforms_bit_exact(E):
    pos = np.concatenate([np.arange(4096), [2 ** 31 - 1, 123456789, 70000]]).astype(np.int32)
    pt = torch.from_numpy(pos).cuda()
    for seed in (0, 7, (5 << 32) | 9, 2 ** 64 - 1):
        for purpose in (0, 1, 2):
            got = E.sample_uniforms(seed, pt, purpose).cpu().numpy().astype(np.float64)
            ref = S.uniform(seed, pos.astype(np.uint64), purpose)
            assert np.array_equal(got, ref), (seed, purpose)


def _check_rows(logits, ids, probs, cnt, top1, tok, prm, pos0):
    """GPU tables of each row against the oracle's filter of the same logits."""
    for r in range(logits.shape[0]):
        z = logits[r].astype(np.float64)
        rid, rpr = S.filtered(z, prm)
        full_id, full_pr = S.filtered(z, S.SamplingParams(prm.temperature, prm.top_k, 1.0))
        m = int(cnt[r])
        assert 1 <= m <= prm.top_k
        common = min(m, len(rid))
        assert ids[r, :common].tolist() == rid[:common].tolist(), r
        if m != len(rid):  # top-p cut within rounding of the cumulative mass
            assert abs(m - len(rid)) == 1
            cut = np.cumsum(full_pr)[min(m, len(rid)) - 1]
            assert abs(cut - prm.top_p) < MARGIN, (r, m, len(rid), cut)
            continue
        np.testing.assert_allclose(probs[r, :m], rpr, rtol=2e-5, atol=1e-7)
        ref_top1 = 1.0 / np.sum(np.exp(z - z.max()))
        assert top1[r] == pytest.approx(ref_top1, rel=1e-4)
        if tok is not None:
            mg = []
            t_ref = S.draw(rid, rpr, S.uniform(prm.seed, pos0 + r, 2), mg)
            if min(mg, default=1.0) > MARGIN:
                assert int(tok[r]) == t_ref, r


CASES = [  # vocab (ragged chunks), top_k, top_p, temperature
    (64, 64, 1.0, 0.7), (100, 50, 0.95, 0.7), (1024, 50, 0.95, 0.7), (5003, 50, 0.95, 0.7),
    (5003, 128, 1.0, 1.3), (5003, 1, 0.95, 0.7), (5003, 50, 0.01, 0.7), (5003, 50, 0.95, 0.05),
    (128256, 50, 0.95, 0.7), (128256, 128, 0.9, 1.0), (151936, 50, 0.95, 0.7),
    (151936, 7, 0.5, 0.7), (262144, 128, 0.95, 0.7)]


@pytest.mark.parametrize("V,k,top_p,T", CASES)
@pytest.mark.parametrize("ties", [False, True])
def test_filter_and_draw_parity(E, V, k, top_p, T, ties):
    R = 3
    logits = W.synthetic_logits(R, V, seed=6, ties=ties, index=V + k)
    prm = S.SamplingParams(T, k, top_p, seed=11)
    out = E.sample_filter(torch.from_numpy(logits).cuda(), T, k, top_p, seed=11, pos0=1000)
    ids, probs, cnt, top1, tok = [x.cpu().numpy() for x in out]
    _check_rows(logits, ids, probs, cnt, top1, tok, prm, 1000)


def test_filter_on_strided_rows_and_errors(E):
    V = 4000
    big = W.synthetic_logits(3, V + 96, seed=7)
    lt = torch.from_numpy(big).cuda()[:, 16:16 + V]  # rows V + 96 apart
    out = E.sample_filter(lt, 0.7, 50, 0.95, seed=2, pos0=5)
    ids, probs, cnt, top1, tok = [x.cpu().numpy() for x in out]
    _check_rows(big[:, 16:16 + V], ids, probs, cnt, top1, tok, S.SamplingParams(0.7, 50, 0.95, 2), 5)
    from paper_2602_20217_amd import _lib as K
    for T, k, p in ((0.0, 50, 0.95), (0.7, 0, 0.95), (0.7, 129, 0.95), (0.7, 50, 0.0),
                    (0.7, 50, 1.5), (float("nan"), 50, 0.95)):
        with pytest.raises(K.KsError):
            E.sample_filter(lt.contiguous(), T, k, p)
    assert K.ks_sample_workspace_bytes(1, 40, 50) == 0  # top_k above the vocabulary
    assert K.ks_sample_workspace_bytes(1, 600000, 128) == 0


def _tables(E, rows, prm, pos0=None, purpose=0):
    out = E.sample_filter(torch.from_numpy(rows).cuda(), prm.temperature, prm.top_k, prm.top_p,
                          seed=prm.seed, pos0=pos0, purpose=purpose)
    return out


@pytest.mark.parametrize("mode", ["close", "far"])
def test_accept_chain_parity(E, mode):
    """Drafts drawn on the device from q, target tables p, acceptance chain:
    equal to the oracle's drafts and (a, token) on the same logits."""
    V, g = 5003, 4
    compared, a_seen = 0, set()
    for seed in range(40):  # fresh logits per seed: the tables' cuts vary too
        Lp = W.synthetic_logits(g + 1, V, seed=8, index=2 * seed)
        noise = W.synthetic_logits(g, V, seed=8, index=2 * seed + 1,
                                   std=0.3 if mode == "close" else 3.0)
        Lq = (Lp[:g] + noise) if mode == "close" else noise
        P = 500 + 7 * seed
        prm = S.SamplingParams(0.7, 50, 0.95, seed)
        qi, qp, qc, _, dr = _tables(E, Lq, prm, pos0=P + 1, purpose=0)
        pi, pp, pc, _, _ = _tables(E, Lp, prm)
        a, tok = E.spec_accept(pi, pp, pc, qi, qp, qc, dr, seed, P)
        mg = []
        qt = [S.filtered(Lq[i].astype(np.float64), prm, mg) for i in range(g)]
        drafts = [S.draw(*qt[i], S.uniform(seed, P + i + 1, 0), mg) for i in range(g)]
        pt = [S.filtered(Lp[i].astype(np.float64), prm, mg) for i in range(g + 1)]
        a_ref, t_ref = S.verify_chain(pt, qt, drafts, seed, P, mg)
        if min(mg) <= MARGIN:
            continue
        compared += 1
        assert dr.cpu().tolist() == drafts, seed
        assert (a, tok) == (a_ref, t_ref), seed
        a_seen.add(a)
    print(f"[accept] {mode}: compared {compared}/40, accepted counts {sorted(a_seen)}", flush=True)
    assert compared >= 30
    assert len(a_seen) >= 2 if mode == "close" else 0 in a_seen


def test_emitted_token_follows_target(E):
    """Context-free p and q: over 3000 Philox streams the first token a round
    emits follows p's filtered distribution (chi-square, p-value above 1e-4)."""
    from scipy import stats
    V, g = 1000, 3
    lp = W.synthetic_logits(1, V, seed=9, std=1.5, index=1)
    lq = lp + W.synthetic_logits(1, V, seed=9, std=1.0, index=2)
    prm = S.SamplingParams(1.0, 12, 1.0, 0)
    pi, pp, pc, _, _ = _tables(E, np.repeat(lp, g + 1, 0), prm)
    pid, ppr = S.filtered(lp[0].astype(np.float64), prm)
    col = {int(t): c for c, t in enumerate(pid)}
    hist = np.zeros(len(pid) + 1)
    for seed in range(3000):
        s = S.SamplingParams(1.0, 12, 1.0, seed)
        qi, qp, qc, _, dr = _tables(E, np.repeat(lq, g, 0), s, pos0=101, purpose=0)
        a, tok = E.spec_accept(pi, pp, pc, qi, qp, qc, dr, seed, 100)
        first = int(dr[0]) if a >= 1 else tok
        hist[col.get(first, len(pid))] += 1
    assert hist[-1] == 0  # never outside p's support
    exp = ppr * hist.sum()
    chi = float(((hist[:-1] - exp) ** 2 / exp).sum())
    assert chi < stats.chi2.ppf(1 - 1e-4, len(pid) - 1), (hist, exp)


@pytest.fixture(scope="module")
def tiny(E):
    cfg, dm, model = build("tiny", n_max=320, gamma_max=4, m_rounds=5, cap_max=128,
                           prefill_chunk=64)
    yield cfg, dm, model
    dm.close()


def test_sampled_generation_matches_oracle(tiny):
    """Speculative sampling on the fp32 decoder (T 0.7, top-k 50, top-p 0.95,
    gamma 4, re-selection every 8 tokens): the tokens, acceptances and
    selections of the oracle, for every seed whose decisions all clear the
    margin; autoregressive sampling likewise."""
    from paper_2602_20217_amd.engine import select_params
    cfg, dm, model = tiny
    prompt = W.prompt_ids(cfg.vocab, 128, 1)
    compared = 0
    for seed in range(1, 9):
        prm = S.SamplingParams(0.7, 50, 0.95, seed)
        mg = []
        ref, log = S.generate(model, prompt, 32, 4, 8, W.TINY_LATENCY, prm, quant_mode="bins",
                              bins=64, n_max=320, margins=mg)
        dm.set_sampling(0.7, 50, 0.95, seed)
        try:
            out, st, sels = dm.generate(prompt, 32, gamma=4, reselect_every=8,
                                        params=select_params(W.TINY_LATENCY, "bins", 64))
        finally:
            dm.set_sampling(0.0)
        print(f"[gen] seed {seed}: min margin {min(mg):.2e}, accepted {st.n_accepted}", flush=True)
        if min(mg) <= MARGIN:
            continue
        compared += 1
        assert out.tolist() == ref, seed
        assert st.n_accepted == sum(log.accepted) and st.n_rounds == len(log.accepted)
        assert len(sels) == len(log.selections)
        for (_, P, wts, sref), sg in zip(log.selections, sels):
            np.testing.assert_array_equal(np.array(sg.exec[:2 * cfg.L], dtype=bool),
                                          sref.exec_mask)
    assert compared >= 3
    compared = 0
    for seed in range(1, 5):
        prm = S.SamplingParams(0.7, 50, 0.95, seed)
        mg = []
        ref = S.ar_sample(model, prompt, 24, 320, prm, mg)
        dm.set_sampling(0.7, 50, 0.95, seed)
        try:
            out, _, _ = dm.generate(prompt, 24, gamma=0)
        finally:
            dm.set_sampling(0.0)
        if min(mg) <= MARGIN:
            continue
        compared += 1
        assert out.tolist() == ref, seed
    assert compared >= 2


def test_sampling_step_calls_and_top_k_one(tiny):
    """Draft steps and verify through the step ABI in sampling mode: with top-k 1
    they reproduce the greedy round; verify without the drafts is refused; the
    emitted-token array holds the accepted drafts, the token, then -1."""
    cfg, dm, model = tiny
    prompt = W.prompt_ids(cfg.vocab, 96, 2)
    mask = np.array([True, False, True, True, False, True, True, True])
    s0 = dm.prefill(prompt)
    g_drafts = [dm.draft_step(mask)[0] for _ in range(4)]
    g_pred, g_a = dm.verify([s0] + g_drafts)
    dm.set_sampling(0.7, 1, 0.95, 3)
    try:
        assert dm.prefill(prompt) == s0
        drafts = [dm.draft_step(mask)[0] for _ in range(4)]
        pred, a = dm.verify([s0] + drafts)
        assert drafts == g_drafts and a == g_a
        assert list(pred[:a + 1]) == list(g_pred[:a + 1]) and all(p == -1 for p in pred[a + 1:])
        from paper_2602_20217_amd import _lib as K
        s1 = int(pred[a])
        with pytest.raises(K.KsError) as e:
            dm.verify([s1, 5, 6])
        assert e.value.status == K.KS_ESTATE
        d1 = dm.draft_step(mask)[0]
        with pytest.raises(K.KsError) as e:
            dm.set_sampling(0.0)  # a draft is pending
        assert e.value.status == K.KS_ESTATE
        with pytest.raises(K.KsError) as e:
            dm.verify([s1, (d1 + 1) % cfg.vocab])  # not the drafted token
        assert e.value.status == K.KS_EINVAL
        dm.verify([s1, d1])
    finally:
        dm.set_sampling(0.0)


def test_sampling_with_dynamic_exit_matches_oracle(tiny):
    """Sampling mode under the draft policy: with tau_conf above 1 every round
    drafts one token; with the selection's gamma* cap rounds stay below it; the
    tokens, acceptances and round lengths equal the oracle's for seeds whose
    decisions clear the margin."""
    from paper_2602_20217_amd.engine import select_params
    cfg, dm, model = tiny
    prompt = W.prompt_ids(cfg.vocab, 128, 3)
    compared = 0
    for tau, source in ((1.01, "fixed"), (0.0, "selected")):
        for seed in range(1, 6):
            prm = S.SamplingParams(0.7, 50, 0.95, seed)
            mg = []
            ref, log = S.generate(model, prompt, 24, 4, 8, W.TINY_LATENCY, prm,
                                  quant_mode="bins", bins=64, n_max=320, tau_conf=tau,
                                  gamma_source=source, margins=mg)
            dm.set_sampling(0.7, 50, 0.95, seed)
            dm.set_draft_policy(tau, source)
            try:
                out, st, _ = dm.generate(prompt, 24, gamma=4, reselect_every=8,
                                         params=select_params(W.TINY_LATENCY, "bins", 64))
            finally:
                dm.set_sampling(0.0)
                dm.set_draft_policy(0.0, "fixed")
            if tau > 1.0:
                assert st.n_drafted == st.n_rounds  # one draft per round
            if min(mg) <= MARGIN:
                continue
            compared += 1
            assert out.tolist() == ref, (tau, source, seed)
            assert st.n_drafted == sum(log.drafted) and st.n_accepted == sum(log.accepted)
    assert compared >= 3


def test_sampling_edge_cases(tiny):
    """One-token prompt, a single generated token (the prefill's draw), draft
    length gamma_max, and a re-selection after every round: tokens equal the
    oracle's where every decision clears the margin; the first token always
    equals the prefill draw."""
    from paper_2602_20217_amd.engine import select_params
    cfg, dm, model = tiny
    params = select_params(W.TINY_LATENCY, "bins", 64)
    for prompt_len, n_new, gamma, every in ((1, 1, 4, 8), (1, 12, 4, 1), (40, 16, 4, 1),
                                            (40, 1, 0, 8)):
        prompt = W.prompt_ids(cfg.vocab, prompt_len, 7)
        prm = S.SamplingParams(0.7, 50, 0.95, 21)
        mg = []
        if gamma == 0:
            ref = S.ar_sample(model, prompt, n_new, 320, prm, mg)
        else:
            ref, _ = S.generate(model, prompt, n_new, gamma, every, W.TINY_LATENCY, prm,
                                quant_mode="bins", bins=64, n_max=320, margins=mg)
        dm.set_sampling(0.7, 50, 0.95, 21)
        try:
            out, st, _ = dm.generate(prompt, n_new, gamma=gamma, reselect_every=every,
                                     params=params if gamma else None)
        finally:
            dm.set_sampling(0.0)
        assert len(out) == n_new
        print(f"[edge] prompt {prompt_len}, {n_new} tokens, gamma {gamma}: "
              f"min margin {min(mg, default=1.0):.1e}", flush=True)
        if min(mg, default=1.0) > MARGIN:
            assert out.tolist() == ref, (prompt_len, n_new, gamma, every)
