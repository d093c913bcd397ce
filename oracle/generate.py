"""Oracle generation loop: greedy self-speculative decoding with periodic
re-selection of the skip set (TEST INFRASTRUCTURE ONLY).

The loop follows Section 3 and Appendix B.1 (t_head, in the latency model's
time unit, adds the LM head to the TPT cost; 0 keeps the paper's cost): the skip set is chosen from the
hidden states of the most recent m = 5 speculation rounds (the last prompt rows
before the first round) and re-chosen every T generated tokens, at the first
round boundary after the count of generated tokens crosses a multiple of T.  The
latency weights use the committed context length at selection time.  The draft
length is the configured gamma (the gamma* of stage 2 is recorded only), or,
with gamma_source "selected", min(gamma*, gamma) of the latest selection; with
tau_conf > 0 a round stops drafting after its first token whose top-1
probability is below tau_conf (the dynamic drafting exit of Section 3, TPT
maximization).

Parity pins: greedy output equals greedy AR output (Section 2.1 guarantees it
for greedy verification); an all-executed skip set accepts every draft.
"""
from __future__ import annotations

from dataclasses import dataclass, field

from . import model as M
from . import latency as LAT
from . import select as SEL


@dataclass
class GenLog:
    selections: list = field(default_factory=list)   # (produced, P, weights, Selection)
    accepted: list = field(default_factory=list)     # n_accepted per round
    drafted: list = field(default_factory=list)      # draft tokens per round
    draft_top1: list = field(default_factory=list)   # top-1 probabilities of each round's drafts


def generate(model: M.Model, prompt, n_new: int, gamma: int, T: int, lat,
             quant_mode: str = "paper_min", bins: int = 0, tau: float = 0.5,
             D: int = 10, m_rounds: int = 5, n_max: int | None = None,
             tau_conf: float = 0.0, gamma_source: str = "fixed", t_head: float = 0.0):
    assert gamma_source in ("fixed", "selected")
    L = model.cfg.L
    n_max = n_max or (len(prompt) + n_new + gamma + 2)
    st = M.prefill(model, prompt, n_max, m_rounds * (gamma + 1))
    log = GenLog()

    def choose():
        wts = LAT.quantize(lat, st.P, L, quant_mode, bins)
        sel, _ = SEL.select(model, st, wts.w_attn, wts.w_mlp, wts.C, tau, True, D,
                            t_head / wts.delta)
        log.selections.append((len(st.out), st.P, wts, sel))
        return sel

    sel = choose()
    while len(st.out) < n_new:
        before = len(st.out)
        cap = gamma if gamma_source == "fixed" else max(1, min(gamma, sel.gamma_star))
        rd = M.ssd_round(model, st, sel.exec_mask, cap, m_rounds, tau_conf)
        log.accepted.append(rd.n_accepted)
        log.drafted.append(len(rd.drafts))
        log.draft_top1.append(rd.draft_top1)
        if len(st.out) < n_new and len(st.out) // T > before // T:
            sel = choose()
    return st.out[:n_new], log
