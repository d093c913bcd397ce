"""Pins of the isolated integer knapsack oracle (no GPU)."""
import numpy as np
import pytest

import workloads as W
from oracle import additive as A


def _rand_instances(B, n, wmax, qmax, seed):
    rng = np.random.default_rng(seed)
    w = rng.integers(1, wmax + 1, size=(B, n)).astype(np.int32)
    q = rng.integers(0, qmax + 1, size=(B, n)).astype(np.int32)
    return w, q


@pytest.mark.parametrize("seed,qmax", [(0, 1000), (1, 3), (2, 0)])
def test_dp_equals_brute_force_with_tie_break(seed, qmax):
    # qmax = 3 and 0 force many equal losses, exercising the tie-break
    B, n, C = 4, 12, 40
    w, q = _rand_instances(B, n, 6, qmax, seed)
    for max_skip in (C, C // 2):
        best, bits = A.knapsack_dp(w, q, C, max_skip)
        for b in range(B):
            bf = A.brute_force(w[b], q[b], C, max_skip)
            for j in range(C + 1):
                if j in bf:
                    assert best[b, j] == bf[j][0]
                    skip = A.backtrack(bits[b], w[b], j)
                    m = int(sum(int(skip[i]) << i for i in range(n)))
                    assert m == bf[j][1], (b, j)
                else:
                    assert best[b, j] == A.INF


def test_unit_weights_pick_smallest_losses():
    rng = np.random.default_rng(7)
    n = 30
    w = np.ones((1, n), dtype=np.int32)
    q = rng.permutation(np.arange(100, 100 + 7 * n, 7)).astype(np.int32)[None]
    best, bits = A.knapsack_dp(w, q, n, n)
    srt = np.sort(q[0])
    for j in range(n + 1):
        assert best[0, j] == int(np.sum(srt[:j]))
        skip = A.backtrack(bits[0], w[0], j)
        assert sorted(q[0][skip == 1].tolist()) == srt[:j].tolist()


def test_quantize_items_generator_instances():
    inst = W.knapsack_instances(B=8, n_items=72, seed=2)
    w, q = A.quantize_items(inst["t"], inst["s"], 4096)
    # total weight lands within rounding of the bin count; losses follow -ln(s)*2^24
    tot = w.sum(1)
    assert np.all(np.abs(tot - 4096) <= 72)
    assert np.all(q >= 0) and np.all(q <= int(-np.log(0.9) * 2 ** 24) + 1)
    np.testing.assert_allclose(q, np.floor(-np.log(inst["s"]) * 2 ** 24 + 0.5), atol=0)
    # attention items get heavier with context length, MLP items do not
    order = np.argsort(inst["ctx"])
    assert w[order[-1], 0::2].mean() > w[order[0], 0::2].mean()


def test_stage2_no_skip_when_values_tiny():
    # with every skip losing most of the value, the full model (j = 0) wins
    w = np.array([[1, 1, 1, 1]], dtype=np.int32)
    s = np.full((1, 4), 0.01)
    q = np.floor(-np.log(s) * 2 ** 24 + 0.5).astype(np.int32)
    best, bits = A.knapsack_dp(w, q, 4, 2)
    j, g, v, skip = A.stage2(best[0], bits[0], w[0], s[0], D=10)
    assert j == 0 and g == 1 and v == pytest.approx(2.0 / 8)
    assert skip.sum() == 0


def test_stage2_prefers_free_skips():
    # items with s = 1 cost nothing to skip: the largest budget of free skips wins
    w = np.array([[2, 3, 2, 3]], dtype=np.int32)
    s = np.array([[1.0, 0.5, 1.0, 0.5]])
    q = np.floor(-np.log(s) * 2 ** 24 + 0.5).astype(np.int32)
    best, bits = A.knapsack_dp(w, q, 10, 5)
    j, g, v, skip = A.stage2(best[0], bits[0], w[0], s[0], D=10)
    assert j == 4 and skip.tolist() == [1, 0, 1, 0] and g == 10
