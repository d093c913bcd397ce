"""Model-level invariants of the oracle decoder and greedy speculative decoding
(no GPU).  The random-init model has no published outputs; these invariants are
what pins it (Section 2 and 2.1 of the paper)."""
import dataclasses

import numpy as np
import pytest

import workloads as W
from oracle import model as M


@pytest.fixture(scope="module")
def tiny():
    cfg = W.config("tiny")
    return M.Model(cfg, W.generate_weights(cfg, seed=0))


def _prompt(n, vocab=1024, seed=1):
    return W.prompt_ids(vocab, n, seed)


def test_prefill_rows_equal_incremental_decode(tiny):
    prompt = _prompt(24)
    c1 = M.KVCache(tiny.cfg, 64)
    full = M.forward(tiny, c1, prompt, 0)
    c2 = M.KVCache(tiny.cfg, 64)
    for t in range(len(prompt)):
        one = M.forward(tiny, c2, prompt[t:t + 1], t)
        np.testing.assert_allclose(one.logits[0], full.logits[t], rtol=1e-11, atol=1e-12)
        for i in range(2 * tiny.cfg.L + 1):
            np.testing.assert_allclose(one.snaps[i][0], full.snaps[i][t], rtol=1e-11, atol=1e-13)


def test_gqa_mapping_matches_duplicated_heads(tiny):
    """hq=4 / hkv=2 equals the MHA model whose k/v heads are the GQA heads repeated
    per group (head h reads kv head h // 2)."""
    cfg = tiny.cfg
    mha_cfg = dataclasses.replace(cfg, hkv=cfg.hq)
    mha = M.Model.__new__(M.Model)
    mha.cfg = mha_cfg
    mha.embed, mha.lm_head, mha.final_norm = tiny.embed, tiny.lm_head, tiny.final_norm
    mha.layers = []
    g = cfg.hq // cfg.hkv
    for Lw in tiny.layers:
        nl = dict(Lw)
        for k in ("wk", "wv"):
            w = Lw[k].reshape(cfg.hkv, cfg.hd, cfg.d)
            nl[k] = np.repeat(w, g, axis=0).reshape(cfg.hq * cfg.hd, cfg.d)
        mha.layers.append(nl)
    prompt = _prompt(12)
    a = M.forward(tiny, M.KVCache(cfg, 16), prompt, 0)
    b = M.forward(mha, M.KVCache(mha_cfg, 16), prompt, 0)
    np.testing.assert_allclose(a.logits, b.logits, rtol=1e-12, atol=1e-13)


def test_skip_all_is_identity(tiny):
    prompt = _prompt(5)
    fw = M.forward(tiny, M.KVCache(tiny.cfg, 8), prompt, 0, exec_mask=[False] * 8)
    np.testing.assert_array_equal(fw.x, tiny.embed[prompt])
    logits, _, _ = M.head(tiny, tiny.embed[prompt])
    np.testing.assert_array_equal(fw.logits, logits)


def test_verify_rows_equal_ar_rows(tiny):
    prompt = _prompt(20)
    st = M.prefill(tiny, prompt, 64, 5)
    st2 = M.prefill(tiny, prompt, 64, 5)
    ar_logits = []
    for _ in range(5):
        fw = M.forward(tiny, st.cache, [st.s], st.P)
        ar_logits.append(fw.logits[0])
        st.P += 1
        st.s = int(fw.argmax[0])
        st.out.append(st.s)
    toks = st.out[:5]
    fv = M.forward(tiny, st2.cache, toks, st2.P)
    np.testing.assert_allclose(fv.logits, np.array(ar_logits), rtol=1e-11, atol=1e-12)


def test_all_executed_draft_accepts_everything(tiny):
    st = M.prefill(tiny, _prompt(30), 128, 25)
    for _ in range(4):
        rd = M.ssd_round(tiny, st, [True] * 8, gamma=4)
        assert rd.n_accepted == 4
        assert rd.emitted == rd.drafts + [int(rd.verify_argmax[4])]


@pytest.mark.parametrize("mask_seed", [0, 1, 2])
def test_greedy_ssd_equals_greedy_ar(tiny, mask_seed):
    prompt = _prompt(40)
    n_new = 14
    ref = M.generate_ar(tiny, prompt, n_new, 128)
    rng = np.random.default_rng(mask_seed)
    mask = rng.random(8) < 0.6
    st = M.prefill(tiny, prompt, 128, 25)
    while len(st.out) < n_new:
        M.ssd_round(tiny, st, mask, gamma=3)
    assert st.out[:n_new] == ref


def test_history_blocks_are_contiguous_recent_positions(tiny):
    st = M.prefill(tiny, _prompt(30), 128, 10)
    for _ in range(7):
        M.ssd_round(tiny, st, [True, False] * 4, gamma=2, m_rounds=5)
    pos, snaps = M.history(st)
    assert len(st.blocks) == 5
    np.testing.assert_array_equal(pos, np.arange(st.P - len(pos), st.P))
    assert all(s.shape == (len(pos), tiny.cfg.d) for s in snaps)
    # X^(2L) rows are the target's verify rows: their argmax is the next committed token
    _, am, _ = M.head(tiny, snaps[-1])
    full = [int(t) for t in _prompt(30)] + st.out
    np.testing.assert_array_equal(am, [full[p + 1] for p in pos])
