"""Oracle of KnapSpec's layer selection (TEST INFRASTRUCTURE ONLY).

* ``cos_rows`` / ``cos_matrix``: Section 2, cos(x, y) = <x, y>/(|x||y|), and for
  matrices the mean of the row cosines.  A zero-norm row scores 0.
* ``expected_tokens``: Eq. expected_tokens, sum_{i=0}^{gamma} alpha^i (the sum
  form, so alpha = 1 gives gamma + 1).
* ``tpt``: Eq. TPT with the quantised latencies of Section 3.4, in units of Delta:
  cost = gamma * (executed weight) + C.  The paper's t_Draft and t_Target leave
  out the LM head; ``head`` (in units of Delta, default 0 = the paper's cost)
  adds it to every draft step and to the verify pass:
  cost = gamma * (executed weight + head) + (C + head).
* ``dp_select``: stage 1, Eq. h_candidates and Eq. dp_main with the pruning of
  Section 3.4 (cos threshold tau and skipped weight at most C/2), in the "pull"
  form: cell j of row i takes the execute candidate f^(i)(g[i-1, j]) or the skip
  candidate g[i-1, j - w_i]; ties go to execute (the >= of Eq. dp_main); a
  candidate survives only if its cosine with X^(i) exceeds tau; g[i, 0] is then
  set to X^(i) as in Algorithm 1 of Appendix D.
* ``stage2``: Algorithm 2, with the backtrack run down to the first sublayer
  using the recorded decisions, Eq. acceptance for alpha-hat, and the grid over
  gamma in 1..D keeping the first strict maximum.

Attention inside a candidate row at position p reads the target cache for
positions < p and the candidate's own key/value at p (the paper does not say
which context a candidate row sees).

Parity pins: cos against closed forms; Eq. expected_tokens; TPT of the full
model equal to 1/C for every gamma; TPT ordering equal to TPL's (Eq. TPL) when
attention and MLP weigh the same; Algorithm 2 on a hand-built stage-1 result
(alpha-hat, the first strict maximum, the backtracked mask); the DP's reachable
cells equal the subset-sum-reachable budgets; each terminal state equals f^(S)
recomputed from its backtracked mask; the DP never beats brute force at any
budget; the j = 0 cell is the full model; ties go to execute and tau is strict
(identity decoder, equal targets); the higher of the two cosines is kept, on an
identity decoder whose targets are unit vectors of one plane so that every
decision and mask is fixed by hand.  The paper calls the model-mode DP
near-optimal, not optimal; on the tiny decoder's seeded history it reaches the
brute-force maximum at all 13 reachable budgets, which the pins assert.
"""
from __future__ import annotations

from dataclasses import dataclass
from itertools import product

import numpy as np

from . import model as M


def cos_rows(X: np.ndarray, Y: np.ndarray) -> np.ndarray:
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    num = np.sum(X * Y, axis=-1)
    nx = np.sqrt(np.sum(X * X, axis=-1))
    ny = np.sqrt(np.sum(Y * Y, axis=-1))
    den = nx * ny
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), 0.0)


def cos_matrix(X: np.ndarray, Y: np.ndarray) -> float:
    return float(np.mean(cos_rows(X, Y)))


def expected_tokens(alpha: float, gamma: int) -> float:
    e, p = 0.0, 1.0
    for _ in range(gamma + 1):
        e += p
        p *= alpha
    return e


def tpt(alpha: float, gamma: int, executed_weight: int, C: int, head: float = 0.0) -> float:
    return expected_tokens(alpha, gamma) / (gamma * (executed_weight + head) + (C + head))


def item_weight(i: int, w_attn: int, w_mlp: int) -> int:
    return w_attn if i % 2 == 1 else w_mlp


@dataclass
class DPResult:
    J: int
    reach: np.ndarray      # [J+1] bool, terminal row
    states: list           # [J+1] terminal states (or None)
    bits: np.ndarray       # [2L+1, J+1] uint8, 1 = skip chosen at (i, j)
    reach_rows: np.ndarray # [2L+1, J+1] bool
    sig_e: np.ndarray      # [2L+1, J+1] cos of execute candidates (nan if absent)
    sig_s: np.ndarray      # [2L+1, J+1] cos of skip candidates (nan if absent)


def dp_select(model: M.Model, cache: M.KVCache, pos: np.ndarray, X: list,
              w_attn: int, w_mlp: int, C: int, tau: float = 0.5,
              prune_half: bool = True) -> DPResult:
    """Stage 1 over history rows X^(0..2L) (each [r, d]) at positions pos [r]."""
    n_sub = model.n_sub
    J = C // 2 if prune_half else C
    reach = np.zeros(J + 1, dtype=bool)
    g = [None] * (J + 1)
    reach[0] = True
    g[0] = X[0].copy()
    bits = np.zeros((n_sub + 1, J + 1), dtype=np.uint8)
    reach_rows = np.zeros((n_sub + 1, J + 1), dtype=bool)
    reach_rows[0] = reach
    sig_e = np.full((n_sub + 1, J + 1), np.nan)
    sig_s = np.full((n_sub + 1, J + 1), np.nan)
    for i in range(1, n_sub + 1):
        w = item_weight(i, w_attn, w_mlp)
        E = [None] * (J + 1)
        for j in range(J + 1):
            if reach[j]:
                E[j] = M.sublayer(model, i, g[j], pos, cache, mode="own")
                sig_e[i, j] = cos_matrix(E[j], X[i])
            if j >= w and reach[j - w]:
                sig_s[i, j] = cos_matrix(g[j - w], X[i])
        ng = [None] * (J + 1)
        nr = np.zeros(J + 1, dtype=bool)
        for j in range(J + 1):
            e_ok = reach[j] and sig_e[i, j] > tau
            s_ok = j >= w and reach[j - w] and sig_s[i, j] > tau
            if e_ok and (not s_ok or sig_e[i, j] >= sig_s[i, j]):
                ng[j], nr[j] = E[j], True
            elif s_ok:
                ng[j], nr[j], bits[i, j] = g[j - w], True, 1
        ng[0], nr[0], bits[i, 0] = X[i].copy(), True, 0
        g, reach = ng, nr
        reach_rows[i] = reach
    return DPResult(J, reach, g, bits, reach_rows, sig_e, sig_s)


def backtrack(bits: np.ndarray, j: int, w_attn: int, w_mlp: int) -> np.ndarray:
    """Exec mask (True = executed) of the terminal cell j, following decisions from
    sublayer 2L down to sublayer 1."""
    n_sub = bits.shape[0] - 1
    ex = np.ones(n_sub, dtype=bool)
    for i in range(n_sub, 0, -1):
        if bits[i, j]:
            ex[i - 1] = False
            j -= item_weight(i, w_attn, w_mlp)
    if j != 0:
        raise AssertionError("backtrack did not end at budget 0")
    return ex


@dataclass
class Selection:
    exec_mask: np.ndarray
    j_star: int
    gamma_star: int
    tpt_star: float
    alpha_hat: float
    alphas: dict          # j -> alpha-hat
    n_match: dict         # j -> matches


def stage2(model: M.Model, dp: DPResult, X_last: np.ndarray, w_attn: int, w_mlp: int,
           C: int, D: int = 10, head: float = 0.0) -> Selection:
    """Algorithm 2: backtrack, alpha-hat by argmax agreement, TPT grid (head:
    the LM head's latency in units of Delta, 0 for the paper's cost)."""
    _, y_ref, _ = M.head(model, X_last)
    r = X_last.shape[0]
    best = (0.0, None, 0, 0, 0.0)
    alphas, nm = {}, {}
    for j in range(dp.J + 1):
        if not dp.reach[j]:
            continue
        ex = backtrack(dp.bits, j, w_attn, w_mlp)
        _, y_j, _ = M.head(model, dp.states[j])
        n_match = int(np.sum(y_j == y_ref))
        a = n_match / r
        alphas[j], nm[j] = a, n_match
        for gam in range(1, D + 1):
            v = tpt(a, gam, C - j, C, head)
            if v > best[0]:
                best = (v, ex, j, gam, a)
    v, ex, j, gam, a = best
    return Selection(ex, j, gam, v, a, alphas, nm)


def select(model: M.Model, st: M.State, w_attn: int, w_mlp: int, C: int,
           tau: float = 0.5, prune_half: bool = True, D: int = 10, head: float = 0.0):
    """Both stages on the session's history."""
    pos, X = M.history(st)
    dp = dp_select(model, st.cache, pos, X, w_attn, w_mlp, C, tau, prune_half)
    return stage2(model, dp, X[-1], w_attn, w_mlp, C, D, head), dp


def brute_force_cos(model: M.Model, cache: M.KVCache, pos: np.ndarray, X: list,
                    w_attn: int, w_mlp: int, J: int):
    """Best cos(f^(S)(X^(0)), X^(2L)) at every exact skipped budget j <= J over all
    2^(2L) skip sets (candidate rows use the same attention context as the DP).
    Returns dict j -> (best cos, exec mask)."""
    n_sub = model.n_sub
    best = {}
    for skip in product([False, True], repeat=n_sub):
        j = sum(item_weight(i + 1, w_attn, w_mlp) for i in range(n_sub) if skip[i])
        if j > J:
            continue
        x = X[0]
        for i in range(1, n_sub + 1):
            if not skip[i - 1]:
                x = M.sublayer(model, i, x, pos, cache, mode="own")
        c = cos_matrix(x, X[-1])
        if j not in best or c > best[j][0]:
            best[j] = (c, ~np.array(skip))
    return best


def apply_mask(model: M.Model, cache: M.KVCache, pos: np.ndarray, X0: np.ndarray,
               exec_mask) -> np.ndarray:
    x = X0
    for i in range(1, model.n_sub + 1):
        if exec_mask[i - 1]:
            x = M.sublayer(model, i, x, pos, cache, mode="own")
    return x
