"""GPU vs oracle: the batched integer knapsack (1024 instances x 72 items x 4097
budgets of Llama-8B-shaped latencies) must match bit for bit."""
import numpy as np
import pytest

import workloads as W
from oracle import additive as A

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def E():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_20217_amd import engine
    return engine


def _run(E, w, q, C, max_skip):
    wd = torch.from_numpy(np.ascontiguousarray(w)).cuda()
    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    best, bits = E.knapsack_batch(wd, qd, C, max_skip)
    torch.cuda.synchronize()
    return wd, best, bits


def test_full_batch_bit_exact(E):
    inst = W.knapsack_instances(B=1024, n_items=72, seed=2)
    w, q = E.knapsack_quantize(inst["t"], inst["s"], 4096)
    w0, q0 = A.quantize_items(inst["t"], inst["s"], 4096)
    np.testing.assert_array_equal(w, w0)
    np.testing.assert_array_equal(q, q0)
    C, max_skip = 4096, 2048
    wd, best, bits = _run(E, w, q, C, max_skip)
    best0, bits0 = A.knapsack_dp(w, q, C, max_skip)
    np.testing.assert_array_equal(best.cpu().numpy(), best0)
    np.testing.assert_array_equal(bits.cpu().numpy().view(np.uint64), bits0)
    # stage 2 on every instance on the GPU; the oracle checks a sample of 24
    s = torch.from_numpy(np.ascontiguousarray(inst["s"])).cuda()
    js, gs, tpt, skip = E.knapsack_batch_select(best, bits, wd, s, C, D=10)
    js, gs, tpt, skip = js.cpu().numpy(), gs.cpu().numpy(), tpt.cpu().numpy(), skip.cpu().numpy()
    rng = np.random.default_rng(0)
    for b in rng.choice(1024, size=24, replace=False):
        j0, g0, v0, sk0 = A.stage2(best0[b], bits0[b], w[b], inst["s"][b], D=10)
        assert v0 == tpt[b], b  # identical float64 operation order
        assert (js[b], gs[b]) == (j0, g0)
        np.testing.assert_array_equal(skip[b], sk0)
    # backtrack of every reachable budget of a few instances
    for b in (0, 511, 1023):
        reach = np.flatnonzero(best0[b] < A.INF)
        jj = torch.from_numpy(reach.astype(np.int32)).cuda()
        bb = bits[b:b + 1].expand(len(reach), -1, -1).contiguous()
        ww = wd[b:b + 1].expand(len(reach), -1).contiguous()
        sk, err = E.knapsack_backtrack(bb, ww, C, jj)
        sk, err = sk.cpu().numpy(), err.cpu().numpy()
        assert not err.any()
        for k, j in enumerate(reach):
            np.testing.assert_array_equal(sk[k], A.backtrack(bits0[b], w[b], int(j)))


@pytest.mark.parametrize("C,max_skip,n", [(40, 40, 12), (40, 20, 12), (100, 57, 9), (0, 0, 5),
                                          (63, 63, 1), (64, 64, 14)])
def test_small_against_brute_force(E, C, max_skip, n):
    rng = np.random.default_rng(C + n)
    B = 6
    w = rng.integers(1, 7, size=(B, n)).astype(np.int32)
    q = rng.integers(0, 4, size=(B, n)).astype(np.int32)  # many ties
    wd, best, bits = _run(E, w, q, C, max_skip)
    best, bits = best.cpu().numpy(), bits.cpu().numpy().view(np.uint64)
    best0, bits0 = A.knapsack_dp(w, q, C, max_skip)
    np.testing.assert_array_equal(best, best0)
    np.testing.assert_array_equal(bits, bits0)
    for b in range(B):
        bf = A.brute_force(w[b], q[b], C, max_skip)
        for j in range(C + 1):
            if j in bf:
                sk = A.backtrack(bits[b], w[b], j)
                assert int(sum(int(sk[i]) << i for i in range(n))) == bf[j][1]
                assert best[b, j] == bf[j][0]
            else:
                assert best[b, j] == A.INF


def test_backtrack_flags_bad_budget(E):
    w = np.ones((2, 4), dtype=np.int32)
    q = np.ones((2, 4), dtype=np.int32)
    wd, best, bits = _run(E, w, q, 8, 2)
    j = torch.tensor([2, 7], dtype=torch.int32, device="cuda")
    sk, err = E.knapsack_backtrack(bits, wd, 8, j)
    assert err.cpu().tolist() == [0, 1]


@pytest.mark.parametrize("C,max_skip", [(4096, 2048), (4096, 4096), (4096, 0), (1000, 255),
                                        (1000, 256), (300, 2000), (8191, 6000)])
def test_dead_budgets_and_slot_sizes(E, C, max_skip):
    """The DP sweeps only the budgets a skip set can reach (0..min(C, max_skip));
    every other cell must still read INF and every decision word above them 0,
    for slot counts from one to 32 per thread.  Stage 2 sweeps up to the largest
    reachable budget (one to 24 slots here): its selection, TPT and mask must
    equal the oracle's on the same instances."""
    rng = np.random.default_rng(C + max_skip)
    B, n = 8, 40
    w = rng.integers(1, max(2, C // 12), size=(B, n)).astype(np.int32)
    q = rng.integers(0, 1 << 20, size=(B, n)).astype(np.int32)
    wd, best, bits = _run(E, w, q, C, max_skip)
    best0, bits0 = A.knapsack_dp(w, q, C, max_skip)
    np.testing.assert_array_equal(best.cpu().numpy(), best0)
    np.testing.assert_array_equal(bits.cpu().numpy().view(np.uint64), bits0)
    s = rng.uniform(0.9, 1.0, size=(B, n))
    js, gs, tpt, skip = E.knapsack_batch_select(best, bits, wd, torch.from_numpy(s).cuda(), C,
                                                D=10)
    js, gs, tpt, skip = js.cpu().numpy(), gs.cpu().numpy(), tpt.cpu().numpy(), skip.cpu().numpy()
    for b in (0, B - 1):
        j0, g0, v0, sk0 = A.stage2(best0[b], bits0[b], w[b], s[b], D=10)
        assert (js[b], gs[b]) == (j0, g0) and v0 == tpt[b], b
        np.testing.assert_array_equal(skip[b], sk0)


def test_negative_weights_and_losses_read_as_zero(E):
    """Every knapsack call reads a negative weight or loss as 0: the DP, the
    backtrack and stage 2 agree with the oracle run on the clamped inputs."""
    rng = np.random.default_rng(11)
    B, n, C, max_skip = 16, 24, 600, 300
    w = rng.integers(1, 40, size=(B, n)).astype(np.int32)
    q = rng.integers(0, 1 << 20, size=(B, n)).astype(np.int32)
    w[rng.random((B, n)) < 0.15] *= -1
    q[rng.random((B, n)) < 0.15] *= -1
    s = rng.uniform(0.9, 1.0, size=(B, n))
    wc, qc = np.maximum(w, 0), np.maximum(q, 0)
    wd, best, bits = _run(E, w, q, C, max_skip)
    best0, bits0 = A.knapsack_dp(wc, qc, C, max_skip)
    np.testing.assert_array_equal(best.cpu().numpy(), best0)
    np.testing.assert_array_equal(bits.cpu().numpy().view(np.uint64), bits0)
    sd = torch.from_numpy(s).cuda()
    js, gs, tpt, skip = E.knapsack_batch_select(best, bits, wd, sd, C, D=10)
    js, gs, tpt, skip = js.cpu().numpy(), gs.cpu().numpy(), tpt.cpu().numpy(), skip.cpu().numpy()
    for b in range(B):
        j0, g0, v0, sk0 = A.stage2(best0[b], bits0[b], wc[b], s[b], D=10)
        assert (js[b], gs[b]) == (j0, g0) and v0 == tpt[b], b
        np.testing.assert_array_equal(skip[b], sk0)
        reach = np.flatnonzero(best0[b] < A.INF)
        jj = torch.from_numpy(reach.astype(np.int32)).cuda()
        sk, err = E.knapsack_backtrack(bits[b:b + 1].expand(len(reach), -1, -1).contiguous(),
                                       wd[b:b + 1].expand(len(reach), -1).contiguous(), C, jj)
        assert not err.cpu().numpy().any()
        for k, j in enumerate(reach):
            np.testing.assert_array_equal(sk.cpu().numpy()[k], A.backtrack(bits0[b], wc[b], int(j)))
