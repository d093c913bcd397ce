"""Planted mistakes in the oracle, on the CPU: each mutant below is a plausible
slip in one oracle function (a dropped term, a wrong sign, exponent or index,
a transposed operand, a swapped role, an off-by-one).  With the mutant patched
in, at least one of the pins listed for that function must fail; a mutant that
every pin accepts would mean the pins do not fix that part of the oracle."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import additive as A
from oracle import generate as GENM
from oracle import latency as LAT
from oracle import model as M
from oracle import sampling as S
from oracle import select as SEL
from tests import test_oracle_additive as TA
from tests import test_oracle_model as TM
from tests import test_oracle_primitives as TP
from tests import test_oracle_sampling as TS
from tests import test_oracle_select as TSEL

_orig = {name: getattr(mod, name) for mod, name in [
    (M, "attn_sublayer"), (M, "attn_qkv"), (S, "philox4x32_10"), (S, "filtered"),
    (LAT, "fit_latency")]}


# ------------------------------------------------------------------ mutants
def rmsnorm_sum(x, g, eps):  # sum of squares instead of their mean
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps) * g


def rmsnorm_eps_outside(x, g, eps):  # eps added after the square root
    return x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps) * g


def _rope(x, pos, theta, *, sign=1.0, fexp=2.0, interleaved=False, shift=0):
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-fexp * np.arange(half, dtype=np.float64) / hd)
    ang = (np.asarray(pos, dtype=np.float64) + shift)[..., None, None] * inv
    c, s = np.cos(ang), np.sin(ang)
    if interleaved:
        a, b = x[..., 0::2], x[..., 1::2]
        out = np.empty_like(x)
        out[..., 0::2] = a * c - b * s
        out[..., 1::2] = b * c + a * s
        return out
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - sign * b * s, b * c + sign * a * s], axis=-1)


def attention_unscaled(q, K, V):
    s = K @ q
    p = np.exp(s - np.max(s))
    return (p / p.sum()) @ V


def attention_keys_as_values(q, K, V):
    s = K @ q / np.sqrt(q.shape[-1])
    p = np.exp(s - np.max(s))
    return (p / p.sum()) @ K


def silu_negated(x):
    return x / (1.0 + np.exp(x))


def bf16_truncate(x):
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = (f.view(np.uint32) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def mlp_gate_up_swapped(model, layer, x):
    c, Wl = model.cfg, model.layers[layer]
    h = M.rmsnorm(x, Wl["mlp_norm"], c.eps)
    return x + (M.silu(h @ Wl["w_up"].T) * (h @ Wl["w_gate"].T)) @ Wl["w_down"].T


def mlp_without_norm(model, layer, x):
    Wl = model.layers[layer]
    return x + (M.silu(x @ Wl["w_gate"].T) * (x @ Wl["w_up"].T)) @ Wl["w_down"].T


def qkv_values_unnormalised(model, layer, x, pos):
    q, k, v = _orig["attn_qkv"](model, layer, x, pos)
    c = model.cfg
    return q, k, (x @ model.layers[layer]["wv"].T).reshape(-1, c.hkv, c.hd)


def attn_wo_transposed(model, layer, x, pos, cache, mode):
    Wl = model.layers[layer]
    wo = Wl["wo"]
    Wl["wo"] = wo.T.copy()
    try:
        return _orig["attn_sublayer"](model, layer, x, pos, cache, mode)
    finally:
        Wl["wo"] = wo


def _attn(model, layer, x, pos, cache, mode, head_map, self_included=True):
    c, Wl = model.cfg, model.layers[layer]
    q, k, v = M.attn_qkv(model, layer, x, pos)
    k, v = model.store(k), model.store(v)
    for r in range(x.shape[0]):
        cache.K[layer][:, pos[r]] = k[r]
        cache.V[layer][:, pos[r]] = v[r]
    o = np.zeros((x.shape[0], c.hq, c.hd))
    for r in range(x.shape[0]):
        end = int(pos[r]) + (1 if self_included else 0)
        for h in range(c.hq):
            kh = head_map(h, c)
            o[r, h] = M.softmax_attention(q[r, h], cache.K[layer][kh, :end], cache.V[layer][kh, :end])
    return x + o.reshape(x.shape[0], -1) @ Wl["wo"].T


def attn_gqa_modulo(model, layer, x, pos, cache, mode):  # query head h -> kv head h % hkv
    return _attn(model, layer, x, pos, cache, mode, lambda h, c: h % c.hkv)


def attn_excludes_self(model, layer, x, pos, cache, mode):  # causal range one short
    return _attn(model, layer, x, pos, cache, mode, lambda h, c: h // (c.hq // c.hkv), False)


def head_without_final_norm(model, x):
    logits = x @ model.lm_head.T
    am = np.argmax(logits, axis=-1)
    mx = logits[np.arange(len(am)), am]
    return logits, am.astype(np.int64), 1.0 / np.sum(np.exp(logits - mx[:, None]), axis=-1)


def expected_tokens_from_one(alpha, gamma):  # sum over i = 1..gamma
    return sum(alpha ** i for i in range(1, gamma + 1))


def tpt_head_once(alpha, gamma, executed_weight, C, head=0.0):  # head paid once per round
    return SEL.expected_tokens(alpha, gamma) / (gamma * executed_weight + C + head)


def tpt_skipped_weight(alpha, gamma, executed_weight, C, head=0.0):  # cost from the skipped weight
    return SEL.expected_tokens(alpha, gamma) / (gamma * (C - executed_weight) + C)


def cos_without_y_norm(X, Y):
    X, Y = np.asarray(X, dtype=np.float64), np.asarray(Y, dtype=np.float64)
    nx = np.sqrt(np.sum(X * X, axis=-1))
    return np.where(nx > 0, np.sum(X * Y, axis=-1) / np.where(nx > 0, nx, 1.0), 0.0)


def fit_latency_swapped(n_attn, t_attn, t_mlp):  # slope and intercept exchanged
    c1, c2, c3 = _orig["fit_latency"](n_attn, t_attn, t_mlp)
    return c1, c3, c2


def round_floor(x):
    return int(math.floor(x))


def round_half_even(x):
    return int(round(x))


def dp_ties_to_skip(w, q, C, max_skip):
    """knapsack_dp with <= in place of < (ties take the skip)."""
    w = np.asarray(w, dtype=np.int64)
    q = np.asarray(q, dtype=np.int64)
    B, n = w.shape
    best = np.full((B, C + 1), A.INF, dtype=np.int64)
    best[:, 0] = 0
    bits = np.zeros((B, n, C // 64 + 1), dtype=np.uint64)
    jj = np.arange(C + 1)
    for i in range(n):
        src = jj[None, :] - w[:, i][:, None]
        ok = src >= 0
        prev = np.where(ok, best[np.arange(B)[:, None], np.clip(src, 0, C)], A.INF)
        cand = np.where(prev < A.INF, prev + q[:, i][:, None], A.INF)
        take = (cand <= best) & (cand < A.INF) & ok & (jj <= max_skip)[None, :]
        best = np.where(take, cand, best)
        for b in range(B):
            for j in np.nonzero(take[b])[0]:
                bits[b, i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return best.astype(np.int32), bits


def philox_key_words_swapped(ctr, key):
    return _orig["philox4x32_10"](ctr, np.asarray(key)[..., ::-1])


def resample_from_target(p, q, x, u_acc, u_res, margins=None):
    """Rejection draws from p itself instead of the residual max(0, p - q)."""
    ratio = S.prob_of(*p, x) / S.prob_of(*q, x)
    if u_acc < min(1.0, ratio):
        return True, x
    return False, S.draw(p[0], p[1], u_res)


def accept_with_inverted_ratio(p, q, x, u_acc, u_res, margins=None):
    """Acceptance test against q/p instead of p/q."""
    ratio = S.prob_of(*q, x) / max(S.prob_of(*p, x), 1e-300)
    if u_acc < min(1.0, ratio):
        return True, x
    pid, ppr = p
    r = np.maximum(0.0, ppr - np.array([S.prob_of(*q, int(y)) for y in pid]))
    if r.sum() <= 0.0:
        return False, S.draw(pid, ppr, u_res)
    return False, S.draw(pid, r / r.sum(), u_res)


def top_p_one_short(logits, prm, margins=None):
    ids, probs = _orig["filtered"](logits, prm, margins)
    if len(ids) > 1 and prm.top_p < 1.0:
        ids, probs = ids[:-1], probs[:-1] / probs[:-1].sum()
    return ids, probs


def _dp(model, cache, pos, X, w_attn, w_mlp, C, tau=0.5, prune_half=True, *,
        ties_execute=True, strict_tau=True, reset_zero=True, keep_higher=True):
    """Stage 1 with one rule changed by the flags."""
    n_sub = model.n_sub
    J = C // 2 if prune_half else C
    reach = np.zeros(J + 1, dtype=bool)
    reach[0] = True
    g = [None] * (J + 1)
    g[0] = X[0].copy()
    bits = np.zeros((n_sub + 1, J + 1), dtype=np.uint8)
    reach_rows = np.zeros((n_sub + 1, J + 1), dtype=bool)
    reach_rows[0] = reach
    sig_e = np.full((n_sub + 1, J + 1), np.nan)
    sig_s = np.full((n_sub + 1, J + 1), np.nan)
    valid = (lambda v: v > tau) if strict_tau else (lambda v: v >= tau)
    for i in range(1, n_sub + 1):
        w = SEL.item_weight(i, w_attn, w_mlp)
        E = [None] * (J + 1)
        for j in range(J + 1):
            if reach[j]:
                E[j] = M.sublayer(model, i, g[j], pos, cache, mode="own")
                sig_e[i, j] = SEL.cos_matrix(E[j], X[i])
            if j >= w and reach[j - w]:
                sig_s[i, j] = SEL.cos_matrix(g[j - w], X[i])
        ng, nr = [None] * (J + 1), np.zeros(J + 1, dtype=bool)
        for j in range(J + 1):
            e_ok = reach[j] and valid(sig_e[i, j])
            s_ok = j >= w and reach[j - w] and valid(sig_s[i, j])
            if not keep_higher:
                prefer_e = sig_e[i, j] <= sig_s[i, j]
            elif ties_execute:
                prefer_e = sig_e[i, j] >= sig_s[i, j]
            else:
                prefer_e = sig_e[i, j] > sig_s[i, j]
            if e_ok and (not s_ok or prefer_e):
                ng[j], nr[j] = E[j], True
            elif s_ok:
                ng[j], nr[j], bits[i, j] = g[j - w], True, 1
        if reset_zero:
            ng[0], nr[0], bits[i, 0] = X[i].copy(), True, 0
        g, reach = ng, nr
        reach_rows[i] = reach
    return SEL.DPResult(J, reach, g, bits, reach_rows, sig_e, sig_s)


def stage2_last_maximum(model, dp, X_last, w_attn, w_mlp, C, D=10, head=0.0):
    """Stage 2 keeping the last of equal TPT values (>= in place of >)."""
    _, y_ref, _ = M.head(model, X_last)
    best = (0.0, None, 0, 0, 0.0)
    alphas, nm = {}, {}
    for j in range(dp.J + 1):
        if not dp.reach[j]:
            continue
        ex = SEL.backtrack(dp.bits, j, w_attn, w_mlp)
        _, y_j, _ = M.head(model, dp.states[j])
        n_match = int(np.sum(y_j == y_ref))
        a = n_match / X_last.shape[0]
        alphas[j], nm[j] = a, n_match
        for gam in range(1, D + 1):
            v = SEL.tpt(a, gam, C - j, C, head)
            if v >= best[0]:
                best = (v, ex, j, gam, a)
    v, ex, j, gam, a = best
    return SEL.Selection(ex, j, gam, v, a, alphas, nm)


def _ssd_round(model, st, exec_mask, gamma, m_rounds=5, tau_conf=0.0, *, extra_accept=False,
               keep_all_rows=False):
    """One greedy round with one rule changed by the flags."""
    drafts, tops = [], []
    t = st.s
    for k in range(gamma):
        fw = M.forward(model, st.cache, [t], st.P + k, exec_mask)
        t = int(fw.argmax[0])
        drafts.append(t)
        tops.append(float(fw.top1[0]))
        if tau_conf > 0 and not tops[-1] >= tau_conf:
            break
    g = len(drafts)
    fv = M.forward(model, st.cache, [st.s] + drafts, st.P)
    y = fv.argmax
    a = 0
    while a < g and drafts[a] == y[a]:
        a += 1
    if extra_accept and a < g:
        a += 1
    emitted = drafts[:a] + [int(y[a])]
    rows = g + 1 if keep_all_rows else a + 1
    st.blocks.append((st.P + np.arange(rows), [sn[:rows] for sn in fv.snaps]))
    st.blocks = st.blocks[-m_rounds:]
    st.P += a + 1
    st.s = int(y[a])
    st.out.extend(emitted)
    return M.Round(drafts, tops, y, a, emitted)


def generate_reselect_on_multiples(model, prompt, n_new, gamma, T, lat, quant_mode="paper_min",
                                   bins=0, tau=0.5, D=10, m_rounds=5, n_max=None, tau_conf=0.0,
                                   gamma_source="fixed"):
    """The generation loop re-selecting only when the produced count is a
    multiple of T (instead of when a multiple has been passed)."""
    from oracle import generate as GEN
    n_max = n_max or (len(prompt) + n_new + gamma + 2)
    st = M.prefill(model, prompt, n_max, m_rounds * (gamma + 1))
    log = GEN.GenLog()

    def choose():
        wts = LAT.quantize(lat, st.P, model.cfg.L, quant_mode, bins)
        sel, _ = SEL.select(model, st, wts.w_attn, wts.w_mlp, wts.C, tau, True, D)
        log.selections.append((len(st.out), st.P, wts, sel))
        return sel

    sel = choose()
    while len(st.out) < n_new:
        rd = M.ssd_round(model, st, sel.exec_mask, gamma, m_rounds, tau_conf)
        log.accepted.append(rd.n_accepted)
        log.drafted.append(len(rd.drafts))
        log.draft_top1.append(rd.draft_top1)
        if len(st.out) < n_new and len(st.out) % T == 0:
            sel = choose()
    return st.out[:n_new], log


def _additive_stage2(best_b, bits_b, w_b, s_b, D=10, *, alpha_executed=False,
                     cost_skipped=False, keep_last=False):
    """Stage 2 of the isolated knapsack with one rule changed by the flags."""
    Wt = int(np.sum(w_b))
    top = (0.0, -1, 0, None)
    for j in range(len(best_b)):
        if best_b[j] >= A.INF:
            continue
        skip = A.backtrack(bits_b, w_b, j)
        a = 1.0
        for i in range(len(w_b)):
            if bool(skip[i]) != alpha_executed:
                a *= float(s_b[i])
        for g in range(1, D + 1):
            e = sum(a ** t for t in range(g + 1))
            v = e / float(g * (j if cost_skipped else Wt - j) + Wt)
            if v > top[0] or (keep_last and v == top[0]):
                top = (v, j, g, skip)
    return top[1], top[2], top[0], top[3]


# ------------------------------------------------------------------ pins
@pytest.fixture(scope="module")
def tiny():
    cfg = W.config("tiny")
    return M.Model(cfg, W.generate_weights(cfg, seed=0))


@pytest.fixture(scope="module")
def tiny_hist(tiny):
    st = M.prefill(tiny, W.prompt_ids(tiny.cfg.vocab, 48, 1), 128, 10)
    pos, X = M.history(st)
    return tiny, st, pos, X


def _mutants(tiny, tiny_hist):
    rope_pins = [TP.test_rope_two_dims_is_plane_rotation,
                 TP.test_rope_identity_norm_and_relative_position,
                 TP.test_rope_pair_frequencies_worked_example]
    attn_pins = [TP.test_attention_sublayer_first_position_worked_example,
                 lambda: TM.test_gqa_mapping_matches_duplicated_heads(tiny),
                 lambda: TM.test_prefill_rows_equal_incremental_decode(tiny)]
    sampling_pins = [TS.test_acceptance_rule_preserves_target_exactly,
                     TS.test_verify_chain_monte_carlo]
    additive_pins = [TA.test_stage2_no_skip_when_values_tiny, TA.test_stage2_prefers_free_skips]
    round_pins = [lambda: TM.test_greedy_ssd_equals_greedy_ar(tiny, 0),
                  lambda: TM.test_history_blocks_are_contiguous_recent_positions(tiny)]
    dp_pins = [TSEL.test_dp_ties_go_to_execute_and_tau_is_strict,
               TSEL.test_dp_keeps_the_higher_cosine,
               lambda: TSEL.test_dp_reachable_cells_are_subset_sums(tiny_hist),
               lambda: TSEL.test_dp_terminal_states_match_backtracked_masks(tiny_hist),
               lambda: TSEL.test_stage2_fallback_and_alpha(tiny_hist)]
    return [
        ("rmsnorm: sum of squares", M, "rmsnorm", rmsnorm_sum, [TP.test_rmsnorm_closed_form]),
        ("rmsnorm: eps after the root", M, "rmsnorm", rmsnorm_eps_outside,
         [TP.test_rmsnorm_closed_form]),
        ("rope: rotation sign", M, "rope", lambda x, p, t: _rope(x, p, t, sign=-1.0), rope_pins),
        ("rope: theta^(-f/hd)", M, "rope", lambda x, p, t: _rope(x, p, t, fexp=1.0), rope_pins),
        ("rope: interleaved pairs", M, "rope", lambda x, p, t: _rope(x, p, t, interleaved=True),
         rope_pins),
        ("rope: 1-based positions", M, "rope", lambda x, p, t: _rope(x, p, t, shift=1), rope_pins),
        ("attention: no 1/sqrt(hd)", M, "softmax_attention", attention_unscaled,
         [TP.test_attention_special_cases]),
        ("attention: keys as values", M, "softmax_attention", attention_keys_as_values,
         [TP.test_attention_special_cases]),
        ("silu: sigmoid(-x)", M, "silu", silu_negated, [TP.test_silu]),
        ("bf16: truncation", M, "to_bf16", bf16_truncate, [TP.test_bf16_rounding]),
        ("mlp: gate and up swapped", M, "mlp_sublayer", mlp_gate_up_swapped,
         [TP.test_swiglu_mlp_sublayer_worked_example]),
        ("mlp: no RMSNorm", M, "mlp_sublayer", mlp_without_norm,
         [TP.test_swiglu_mlp_sublayer_worked_example]),
        ("attention sublayer: values from the unnormalised input", M, "attn_qkv",
         qkv_values_unnormalised, attn_pins),
        ("attention sublayer: Wo transposed", M, "attn_sublayer", attn_wo_transposed, attn_pins),
        ("attention sublayer: head h -> kv head h % hkv", M, "attn_sublayer", attn_gqa_modulo,
         attn_pins),
        ("attention sublayer: own position excluded", M, "attn_sublayer", attn_excludes_self,
         attn_pins),
        ("head: no final RMSNorm", M, "head", head_without_final_norm, [TP.test_head_worked_example]),
        ("expected tokens: sum from i = 1", SEL, "expected_tokens", expected_tokens_from_one,
         [TP.test_expected_tokens_closed_form]),
        ("cos: |y| dropped", SEL, "cos_rows", cos_without_y_norm, [TP.test_cos_closed_forms]),
        ("TPT: cost from the skipped weight", SEL, "tpt", tpt_skipped_weight,
         [TSEL.test_tpt_full_model_is_one_over_capacity,
          TSEL.test_tpt_reduces_to_tpl_when_latencies_equal, TSEL.test_stage2_grid_toy]),
        ("TPT: head cost paid once per round", SEL, "tpt", tpt_head_once,
         [TSEL.test_tpt_head_cost_closed_forms, TSEL.test_stage2_grid_toy]),
        ("latency fit: slope and intercept exchanged", LAT, "fit_latency", fit_latency_swapped,
         [TSEL.test_latency_fit_recovers_coefficients]),
        ("weights: floor instead of rounding", LAT, "round_half_up", round_floor,
         [TSEL.test_quantize_appendix_c_worked_example, TSEL.test_quantize_bins_tiny,
          TSEL.test_quantize_rounds_halves_up]),
        ("weights: halves to even", LAT, "round_half_up", round_half_even,
         [TSEL.test_quantize_appendix_c_worked_example, TSEL.test_quantize_bins_tiny,
          TSEL.test_quantize_rounds_halves_up]),
        ("additive DP: ties take the skip", A, "knapsack_dp", dp_ties_to_skip,
         [lambda: TA.test_dp_equals_brute_force_with_tie_break(1, 3),
          lambda: TA.test_dp_equals_brute_force_with_tie_break(2, 0)]),
        ("philox: key words exchanged", S, "philox4x32_10", philox_key_words_swapped,
         [TS.test_philox_known_answers]),
        ("sampling: rejection draws from p", S, "accept_or_resample", resample_from_target,
         sampling_pins),
        ("sampling: acceptance ratio q/p", S, "accept_or_resample", accept_with_inverted_ratio,
         sampling_pins),
        ("sampling: top-p cut one entry short", S, "filtered", top_p_one_short,
         [TS.test_filter_top_p_keeps_shortest_sufficient_prefix]),
        ("model-mode DP: ties take the skip", SEL, "dp_select",
         lambda *a, **k: _dp(*a, ties_execute=False, **k), dp_pins),
        ("model-mode DP: the lower cosine kept", SEL, "dp_select",
         lambda *a, **k: _dp(*a, keep_higher=False, **k), dp_pins),
        ("model-mode DP: sigma >= tau", SEL, "dp_select",
         lambda *a, **k: _dp(*a, strict_tau=False, **k), dp_pins),
        ("model-mode DP: cell 0 not reset to X^(i)", SEL, "dp_select",
         lambda *a, **k: _dp(*a, reset_zero=False, **k), dp_pins),
        ("stage 2: last of equal TPT values", SEL, "stage2", stage2_last_maximum,
         [lambda: TSEL.test_stage2_fallback_and_alpha(tiny_hist), TSEL.test_stage2_grid_toy]),
        ("greedy round: one draft past the first mismatch accepted", M, "ssd_round",
         lambda *a, **k: _ssd_round(*a, extra_accept=True, **k), round_pins),
        ("greedy round: history keeps every verify row", M, "ssd_round",
         lambda *a, **k: _ssd_round(*a, keep_all_rows=True, **k), round_pins),
        ("knapsack stage 2: alpha over the executed items", A, "stage2",
         lambda *a, **k: _additive_stage2(*a, alpha_executed=True, **k), additive_pins),
        ("knapsack stage 2: cost from the skipped weight", A, "stage2",
         lambda *a, **k: _additive_stage2(*a, cost_skipped=True, **k), additive_pins),
        ("knapsack stage 2: last of equal TPT values", A, "stage2",
         lambda *a, **k: _additive_stage2(*a, keep_last=True, **k), additive_pins),
        ("generation: re-select only on multiples of T", GENM, "generate",
         generate_reselect_on_multiples,
         [TSEL.test_reselection_at_first_round_end_past_each_multiple]),
    ]


N_MUTANTS = 40


def test_mutant_table_size(tiny, tiny_hist):
    assert len(_mutants(tiny, tiny_hist)) == N_MUTANTS


@pytest.mark.parametrize("idx", range(N_MUTANTS))
def test_pins_reject_mutant(tiny, tiny_hist, monkeypatch, idx):
    name, mod, attr, mutant, pins = _mutants(tiny, tiny_hist)[idx]
    # the pins pass on the oracle as it is
    for pin in pins:
        pin()
    monkeypatch.setattr(mod, attr, mutant)
    rejected = []
    for pin in pins:
        try:
            pin()
        # an assertion, or arithmetic that breaks down (a mutant that raises
        # anything else is itself broken, and the test errors)
        except (AssertionError, ValueError, ZeroDivisionError, FloatingPointError) as e:
            rejected.append((getattr(pin, "__name__", "pin"), type(e).__name__))
    assert rejected, f"no pin rejects the mutant: {name}"
    print(f"[mutant] {name}: rejected by {rejected}")
