"""Oracle speculative sampling (TEST INFRASTRUCTURE ONLY).

Sampling-mode verification of speculative decoding (Section 2.1): a draft token
x drawn from the draft distribution q is accepted iff u < min(1, p(x) / q(x))
for u ~ U[0, 1); at the first rejection the round emits a token drawn from the
residual max(0, p - q), normalised; when every draft is accepted it emits a
bonus token drawn from p after the last draft.  This is the speculative
sampling construction the paper builds on, which leaves the target's
distribution unchanged.  Distributions are nucleus sampling with temperature T,
top-k and top-p (the paper's sampling experiments use T = 0.7, k = 50,
p = 0.95); T <= 0 means greedy (a point mass on the argmax).

Filter of one logits row (float64): z = logits / T; keep the top_k largest z
(ties: lower id first); softmax over them; keep the shortest prefix, in that
order, whose cumulative probability reaches top_p; renormalise.

Random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw 2011, "Parallel
random numbers: as easy as 1, 2, 3"), counter (position, purpose, 0, 0), key
(seed low 32 bits, seed high 32 bits); u = (first output word >> 8) * 2^-24.
Purposes: 0 draft sampling, 1 acceptance test, 2 target sampling (residual,
bonus token and autoregressive sampling).  The position is that of the token
being produced.

Pins (``tests/test_oracle_sampling.py``): Philox known-answer vectors of the
Random123 distribution; the filter's special cases (top_k = 1 is the argmax,
no filtering is the softmax, top_p keeps the shortest sufficient prefix); the
output distribution of a speculative step equals p (Monte Carlo over Philox
streams, chi-square); top_k = 1 reduces speculative sampling to greedy
self-speculative decoding.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import model as M

_M0, _M1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
_W0, _W1 = np.uint64(0x9E3779B9), np.uint64(0xBB67AE85)
_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds.  ctr: array [..., 4] of uint32 words, key:
    array [..., 2]; returns [..., 4] uint32."""
    c = [np.asarray(ctr[..., i], dtype=np.uint64) for i in range(4)]
    k0 = np.asarray(key[..., 0], dtype=np.uint64)
    k1 = np.asarray(key[..., 1], dtype=np.uint64)
    for r in range(10):
        p0 = _M0 * c[0]
        p1 = _M1 * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c = [(hi1 ^ c[1] ^ k0) & _MASK, lo1, (hi0 ^ c[3] ^ k1) & _MASK, lo0]
        if r < 9:
            k0 = (k0 + _W0) & _MASK
            k1 = (k1 + _W1) & _MASK
    return np.stack(c, axis=-1).astype(np.uint32)


def uniform(seed: int, pos, purpose: int):
    """U[0, 1) on a 2^-24 grid from Philox4x32-10 (scalar or array pos)."""
    pos = np.asarray(pos, dtype=np.uint64)
    ctr = np.zeros(pos.shape + (4,), dtype=np.uint64)
    ctr[..., 0] = pos & _MASK
    ctr[..., 1] = purpose
    key = np.zeros(pos.shape + (2,), dtype=np.uint64)
    key[..., 0] = seed & 0xFFFFFFFF
    key[..., 1] = (seed >> 32) & 0xFFFFFFFF
    w = philox4x32_10(ctr, key)[..., 0].astype(np.float64)
    u = np.floor(w / 256.0) / 16777216.0
    return float(u) if u.shape == () else u


@dataclass
class SamplingParams:
    temperature: float = 0.7
    top_k: int = 50
    top_p: float = 0.95
    seed: int = 0


def filtered(logits, prm: SamplingParams, margins: list | None = None):
    """(ids, probs) of the filtered distribution of one logits row, ids in the
    filter's order (decreasing z, ties by lower id).

    margins, when given, receives the relative gaps of the two cuts (top-k: the
    k-th and (k+1)-th logits; top-p: the cumulative mass against top_p on both
    sides of the cut), which say how far the table is from changing."""
    z = np.asarray(logits, dtype=np.float64)
    V = z.shape[0]
    if prm.temperature <= 0:
        return np.array([int(np.argmax(z))]), np.array([1.0])
    z = z / prm.temperature
    k = V if prm.top_k <= 0 else min(prm.top_k, V)
    order = np.lexsort((np.arange(V), -z))
    if margins is not None and k < V:
        zk, zn = z[order[k - 1]], z[order[k]]
        margins.append((zk - zn) / max(1.0, abs(zk)))
    order = order[:k]
    zk = z[order]
    e = np.exp(zk - zk[0])
    pk = e / e.sum()
    m = k
    if prm.top_p < 1.0:
        cum = np.cumsum(pk)
        m = min(k, int(np.searchsorted(cum, prm.top_p, side="left")) + 1)
        if margins is not None:
            if m < k or cum[m - 1] >= prm.top_p:
                margins.append(cum[m - 1] - prm.top_p)
            if m >= 2:
                margins.append(prm.top_p - cum[m - 2])
    probs = pk[:m] / pk[:m].sum()
    return order[:m].astype(np.int64), probs


def draw(ids, probs, u: float, margins: list | None = None) -> int:
    """Inverse-CDF draw in table order: the first entry whose cumulative
    probability exceeds u (the last entry if rounding leaves u above the total).
    margins receives the distance of u to the chosen entry's interval ends."""
    cum = np.cumsum(probs)
    i = min(int(np.searchsorted(cum, u, side="right")), len(ids) - 1)
    if margins is not None:
        if i > 0:
            margins.append(u - cum[i - 1])
        if i < len(ids) - 1:
            margins.append(cum[i] - u)
    return int(ids[i])


def prob_of(ids, probs, x: int) -> float:
    hit = np.flatnonzero(ids == x)
    return float(probs[hit[0]]) if hit.size else 0.0


def accept_or_resample(p, q, x: int, u_acc: float, u_res: float,
                       margins: list | None = None):
    """One verified position: (accepted, token).  p, q: (ids, probs) tables of
    the target and the draft; x drawn from q."""
    px, qx = prob_of(*p, x), prob_of(*q, x)
    ratio = px / qx
    if margins is not None and ratio < 1.0:
        margins.append(abs(u_acc - ratio))
    if u_acc < min(1.0, ratio):
        return True, x
    pid, ppr = p
    r = np.maximum(0.0, ppr - np.array([prob_of(*q, int(y)) for y in pid]))
    if r.sum() <= 0.0:  # p = q on p's support: the target itself
        return False, draw(pid, ppr, u_res, margins)
    return False, draw(pid, r / r.sum(), u_res, margins)


def verify_chain(p_tabs, q_tabs, drafts, seed: int, P: int, margins: list | None = None):
    """Acceptance chain of one round: drafts d_1..d_g (drafts[i] at position
    P+i+1, drawn from q_tabs[i]) against the target tables p_tabs[0..g] of the
    verify rows.  Returns (a, final): a accepted drafts, then the residual token
    at the first rejection, or the bonus token drawn from p_tabs[g]."""
    g = len(drafts)
    for i in range(g):
        pos = P + i + 1
        ok, tok = accept_or_resample(p_tabs[i], q_tabs[i], drafts[i], uniform(seed, pos, 1),
                                     uniform(seed, pos, 2), margins)
        if not ok:
            return i, tok
    return g, draw(*p_tabs[g], uniform(seed, P + g + 1, 2), margins)


@dataclass
class SampleRound:
    drafts: list
    draft_top1: list
    n_accepted: int
    emitted: list


def spec_round(model: M.Model, st: M.State, exec_mask, gamma: int, prm: SamplingParams,
               m_rounds: int = 5, tau_conf: float = 0.0,
               margins: list | None = None) -> SampleRound:
    """One speculative sampling round from state st: the greedy round's draft,
    verify and history semantics (including the dynamic drafting exit on the
    draft's unfiltered top-1 probability), with drafts drawn from the filtered
    draft distribution (purpose 0) and the acceptance chain above."""
    drafts, qs, tops = [], [], []
    t = st.s
    for k in range(gamma):
        fw = M.forward(model, st.cache, [t], st.P + k, exec_mask)
        q = filtered(fw.logits[0], prm, margins)
        t = draw(*q, uniform(prm.seed, st.P + k + 1, 0), margins)
        drafts.append(t)
        qs.append(q)
        tops.append(float(fw.top1[0]))
        if tau_conf > 0 and not tops[-1] >= tau_conf:
            break
    g = len(drafts)
    fv = M.forward(model, st.cache, [st.s] + drafts, st.P)
    ps = [filtered(fv.logits[i], prm, margins) for i in range(g + 1)]
    a, final = verify_chain(ps, qs, drafts, prm.seed, st.P, margins)
    emitted = drafts[:a] + [final]
    st.blocks.append((st.P + np.arange(a + 1), [sn[:a + 1] for sn in fv.snaps]))
    st.blocks = st.blocks[-m_rounds:]
    st.P += a + 1
    st.s = final
    st.out.extend(emitted)
    return SampleRound(drafts, tops, a, emitted)


def prefill(model: M.Model, prompt, n_max: int, hist_rows: int, prm: SamplingParams,
            margins: list | None = None) -> M.State:
    """Prefill whose first generated token (position len(prompt)) is drawn from
    the filtered target distribution (purpose 2); the last hist_rows prompt rows
    form the first history block, as in the greedy prefill."""
    cache = M.KVCache(model.cfg, n_max)
    n = len(prompt)
    fw = M.forward(model, cache, prompt, 0)
    s = draw(*filtered(fw.logits[-1], prm, margins), uniform(prm.seed, n, 2), margins)
    st = M.State(cache=cache, P=n, s=s, out=[s])
    r0 = min(n, hist_rows)
    st.blocks.append((np.arange(n - r0, n), [sn[n - r0:] for sn in fw.snaps]))
    return st


def ar_sample(model: M.Model, prompt, n_new: int, n_max: int, prm: SamplingParams,
              margins: list | None = None):
    """Autoregressive sampling: the token at position t is drawn from the
    filtered target distribution with the purpose-2 uniform of t."""
    st = prefill(model, prompt, n_max, 1, prm, margins)
    while len(st.out) < n_new:
        fw = M.forward(model, st.cache, [st.s], st.P)
        st.P += 1
        st.s = draw(*filtered(fw.logits[0], prm, margins), uniform(prm.seed, st.P, 2), margins)
        st.out.append(st.s)
    return st.out[:n_new]


def generate(model: M.Model, prompt, n_new: int, gamma: int, T: int, lat, prm: SamplingParams,
             quant_mode: str = "paper_min", bins: int = 0, tau: float = 0.5, D: int = 10,
             m_rounds: int = 5, n_max: int | None = None, tau_conf: float = 0.0,
             gamma_source: str = "fixed", margins: list | None = None):
    """Speculative sampling generation with periodic re-selection of the skip set
    (the greedy loop's schedule, with sampled rounds)."""
    from . import latency as LAT
    from . import select as SEL
    from .generate import GenLog
    assert gamma_source in ("fixed", "selected")
    L = model.cfg.L
    n_max = n_max or (len(prompt) + n_new + gamma + 2)
    st = prefill(model, prompt, n_max, m_rounds * (gamma + 1), prm, margins)
    log = GenLog()

    def choose():
        wts = LAT.quantize(lat, st.P, L, quant_mode, bins)
        sel, _ = SEL.select(model, st, wts.w_attn, wts.w_mlp, wts.C, tau, True, D)
        log.selections.append((len(st.out), st.P, wts, sel))
        return sel

    sel = choose()
    while len(st.out) < n_new:
        before = len(st.out)
        cap = gamma if gamma_source == "fixed" else max(1, min(gamma, sel.gamma_star))
        rd = spec_round(model, st, sel.exec_mask, cap, prm, m_rounds, tau_conf, margins)
        log.accepted.append(rd.n_accepted)
        log.drafted.append(len(rd.drafts))
        log.draft_top1.append(rd.draft_top1)
        if len(st.out) < n_new and len(st.out) // T > before // T:
            sel = choose()
    return st.out[:n_new], log
