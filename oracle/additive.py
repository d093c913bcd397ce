"""Oracle of the isolated integer knapsack (TEST INFRASTRUCTURE ONLY).

The per-budget problem of Eq. objective_knapsack picks, for every exact skipped
weight k, the skip set with the best similarity.  In isolation each item i has
an integer weight w_i (its quantised latency, Section 3.4 in BINS mode:
Delta = sum_i t_i / bins, w_i = max(1, floor(t_i/Delta + 1/2))) and a similarity
score s_i in (0, 1] that is lost when it is skipped; the value of a skip set is
prod_{i skipped} s_i.  As an exact integer problem the DP minimises the loss
sum_{i skipped} q_i with q_i = floor(-ln(s_i) * 2^24 + 1/2), over budgets
j = 0..C (Single-pass Efficiency, Section 3.4), with the skipped weight capped at
max_skip (the C/2 prune of Section 3.4).

Recurrence (pull form of Eq. h_candidates): best_i[j] = best_{i-1}[j] (execute)
unless j >= w_i and best_{i-1}[j - w_i] + q_i < best_{i-1}[j] strictly (skip,
decision bit 1).  Ties go to execute, as in Eq. dp_main.

Stage 2 (Algorithm 2 with alpha-hat replaced by the surrogate value):
alpha_j = prod_{i skipped} s_i multiplied in ascending i in float64;
TPT(j, gamma) = (sum_{k=0}^{gamma} alpha_j^k) / (gamma*(W - j) + W) with
W = sum_i w_i; j ascending then gamma = 1..D, first strict maximum wins.

Parity pins: brute force over all 2^n skip sets for n <= 20 (optimum and the
tie-break: the smallest mask integer with the last item as most significant
bit); with all weights 1 the optimum at budget j is the j smallest losses.
"""
from __future__ import annotations

import math

import numpy as np

INF = np.int64(2 ** 31 - 1)


def quantize_items(t: np.ndarray, s: np.ndarray, bins: int):
    """t, s float64 [B, n] -> w int32 [B, n], q int32 [B, n]."""
    t = np.asarray(t, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    B, n = t.shape
    w = np.zeros((B, n), dtype=np.int32)
    q = np.zeros((B, n), dtype=np.int32)
    for b in range(B):
        delta = 0.0
        for i in range(n):
            delta += t[b, i]
        delta /= bins
        for i in range(n):
            w[b, i] = max(1, int(math.floor(t[b, i] / delta + 0.5)))
            q[b, i] = int(math.floor(-math.log(s[b, i]) * 16777216.0 + 0.5))
    return w, q


def knapsack_dp(w: np.ndarray, q: np.ndarray, C: int, max_skip: int):
    """Batched DP, vectorised over instances and budgets.

    Returns best int32 [B, C+1] (INF where unreachable) and bits uint64
    [B, n, C//64 + 1] (bit j%64 of word j//64 is the decision at budget j).
    """
    w = np.asarray(w, dtype=np.int64)
    q = np.asarray(q, dtype=np.int64)
    B, n = w.shape
    words = C // 64 + 1
    best = np.full((B, C + 1), INF, dtype=np.int64)
    best[:, 0] = 0
    bits = np.zeros((B, n, words), dtype=np.uint64)
    jj = np.arange(C + 1)
    valid_j = jj <= max_skip
    for i in range(n):
        wi = w[:, i][:, None]
        src = jj[None, :] - wi
        ok = src >= 0
        prev = np.where(ok, best[np.arange(B)[:, None], np.clip(src, 0, C)], INF)
        cand = np.where(prev < INF, prev + q[:, i][:, None], INF)
        take = (cand < best) & ok & valid_j[None, :]
        best = np.where(take, cand, best)
        for b in range(B):
            idx = np.nonzero(take[b])[0]
            if idx.size:
                np.bitwise_or.at(bits[b, i], idx // 64,
                                 np.left_shift(np.uint64(1), (idx % 64).astype(np.uint64)))
    return best.astype(np.int32), bits


def get_bit(bits_bi: np.ndarray, j: int) -> int:
    return int((int(bits_bi[j // 64]) >> (j % 64)) & 1)


def backtrack(bits_b: np.ndarray, w_b: np.ndarray, j: int) -> np.ndarray:
    """Skip mask uint8 [n] (1 = skipped) of budget j for one instance."""
    n = len(w_b)
    skip = np.zeros(n, dtype=np.uint8)
    for i in range(n - 1, -1, -1):
        if get_bit(bits_b[i], j):
            skip[i] = 1
            j -= int(w_b[i])
    if j != 0:
        raise AssertionError("backtrack did not end at budget 0")
    return skip


def stage2(best_b: np.ndarray, bits_b: np.ndarray, w_b: np.ndarray, s_b: np.ndarray,
           D: int = 10):
    """Returns (j*, gamma*, tpt*, skip mask) for one instance."""
    W = int(np.sum(w_b))
    top = (0.0, -1, 0, None)
    for j in range(len(best_b)):
        if best_b[j] >= INF:
            continue
        skip = backtrack(bits_b, w_b, j)
        a = 1.0
        for i in range(len(w_b)):
            if skip[i]:
                a *= float(s_b[i])
        for g in range(1, D + 1):
            e, p = 0.0, 1.0
            for _ in range(g + 1):
                e += p
                p *= a
            v = e / float(g * (W - j) + W)
            if v > top[0]:
                top = (v, j, g, skip)
    return top[1], top[2], top[0], top[3]


def brute_force(w_b: np.ndarray, q_b: np.ndarray, C: int, max_skip: int):
    """For every budget j <= min(C, max_skip): (min loss, smallest mask integer with the
    last item as most significant bit) over all 2^n skip sets; n <= 20."""
    n = len(w_b)
    if n > 20:
        raise ValueError("brute force limited to 20 items")
    res = {}
    for m in range(1 << n):
        j = 0
        loss = 0
        for i in range(n):
            if (m >> i) & 1:
                j += int(w_b[i])
                loss += int(q_b[i])
        if j > C or j > max_skip:
            continue
        if j not in res or loss < res[j][0] or (loss == res[j][0] and m < res[j][1]):
            res[j] = (loss, m)
    return res
