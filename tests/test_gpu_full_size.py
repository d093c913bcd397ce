"""Parity at the full Llama-3-8B shape (bf16), in the launch configurations the
benchmark times: the 8K workload (skinny products, 5-tile attention splits) and
a 128K-position context (streaming attention splits, as in the context sweep).

Sampled outputs the oracle computes one by one: single sublayers (first and last
layer) on decode (1 row) and verify (5 rows) inputs over seeded caches of
8189 and 131067 positions, the last layer on 400, 600, 800 and 1225 candidate
rows of the selection (tiled MFMA products with 1 to 8 K splits, batched
attention;
sampled rows at tile edges and in the ragged tail), the LM head on two rows
(tolerance 2e-2 relative),
and the sampling filter of head logits against the oracle's filter of the same
logits.  Properties that hold at any size: full-model drafts are accepted by
the verify pass at the same positions, and speculative generation (with
knapsack selections) emits exactly the autoregressive tokens after a real 8K
prefill, greedy and as sampling with top-k 1.  Every call goes through the C
ABI."""
import dataclasses

import numpy as np
import pytest

import workloads as W
from oracle import model as M
from tests.gpu_helpers import (rel_err, margin, one_layer_model, fill_layer, check_sublayers,
                               check_rows, update_err)

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOL = 2e-2
CTX = 8192
LAYERS = (0, 31)


@pytest.fixture(scope="module")
def full():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_20217_amd.engine import DeviceModel
    cfg = W.config("llama8b")
    print("\n[setup] llama8b weights", flush=True)
    dm = DeviceModel(cfg, n_max=CTX + 320, gamma_max=8, m_rounds=5, cap_max=256,
                     prefill_chunk=512)
    W.generate_weights(cfg, seed=0, consume=dm.upload)
    dm.finalize()
    yield cfg, dm
    dm.close()


def _one_layer(cfg, layer):
    return one_layer_model(cfg, layer)


def _fill(cfg, dm, layer, n):
    return fill_layer(cfg, dm, layer, n, CTX + 320)


@pytest.mark.parametrize("layer", LAYERS)
@pytest.mark.parametrize("R", [1, 5, 12])
def test_full_size_sublayers(full, layer, R):
    cfg, dm = full
    n = CTX - 3  # ragged against the 320-position splits
    check_sublayers(cfg, dm, _one_layer(cfg, layer), _fill(cfg, dm, layer, n), layer, n, R, TOL,
                    "full")


@pytest.mark.parametrize("R", [5, 12])
def test_full_size_one_row_bits_equal_verify_rows(full, R):
    """A decode row (one row: activation staged in LDS) gives the same bits as
    the same row inside an R-row verify batch (per-step activation loads; at
    12 rows two groups of 8 rows per matrix instruction and two 16-column
    attention blocks), for both sublayers of layer 0 at row lengths on both
    sides of a split boundary (7999..8003 with 320-position splits)."""
    cfg, dm = full
    n = 8000 - 2
    _fill(cfg, dm, 0, n)
    dm.set_context(n, 0)
    x = torch.from_numpy(W.synthetic_rows(R, cfg.d, seed=4, std=1.0, index=77)).cuda()
    pos = np.arange(R) + n
    for i in (1, 2):
        out5 = torch.empty(R, cfg.d, device="cuda")
        dm.sublayer_apply(i, x, pos, mode=0, out=out5)
        for r in range(R):
            out1 = torch.empty(1, cfg.d, device="cuda")
            dm.sublayer_apply(i, x[r:r + 1].contiguous(), pos[r:r + 1], mode=0, out=out1)
            diff = int((out1[0] != out5[r]).sum().item())
            print(f"[bits] sublayer {i} row {r} (length {pos[r] + 1}): {diff} differing elements",
                  flush=True)
            assert diff == 0, (i, r)
        x = out5


# Row counts of the selection's candidate batches at 8K (up to 49 budgets x 25
# history rows): the split-K factor of the tiled products follows the row
# count, and these take 1, 2, 3, 4, 5 and 8 splits among the QKV, O and down
# products (600 rows: a fifth 128-row tile with 88 rows).
@pytest.mark.parametrize("R", [400, 600, 800, 1225])
def test_full_size_batched_sublayers(full, R):
    """Attention with each row's own key/value (the selection's candidate rows)
    and then the MLP of the last layer on R rows.  Rows do not see each other in
    this mode, so the oracle evaluates a sample of rows one by one: the first
    and last rows of 128-row tiles and the ragged last tile."""
    cfg, dm = full
    layer = LAYERS[-1]
    n = CTX - 3
    cache = _fill(cfg, dm, layer, n)
    model = _one_layer(cfg, layer)
    pos = (n - R + np.arange(R)).astype(np.int32)
    x = W.synthetic_rows(R, cfg.d, seed=4, std=1.0, index=700 + R)
    sample = sorted({0, 127, 128, 255, R // 2, (R // 128) * 128, R - 1})
    xin = torch.from_numpy(x).cuda()
    for sub in (1, 2):
        out = torch.empty(R, cfg.d, device="cuda")
        dm.sublayer_apply(2 * layer + sub, xin, pos, mode=1, out=out)
        got = out.cpu().numpy()
        ref = M.sublayer(model, sub, x[sample].astype(np.float64), pos[sample], cache, mode="own")
        e, eu = rel_err(got[sample], ref), update_err(got[sample], x[sample], ref)
        print(f"[batched] layer {layer} sublayer {sub} R {R}: rel err {e:.2e}, update {eu:.2e}"
              f" on rows {sample}", flush=True)
        check_rows(got[sample], x[sample], ref, TOL, (sub, R))
        x, xin = got, out


LONG = 131072


@pytest.fixture(scope="module")
def long_ctx(full):
    """A 128K-position context over the same weights (the streaming decode
    attention's launch configuration at that cache size)."""
    cfg, dm = full
    dl = dm.resized(LONG + 320)
    yield cfg, dl
    dl.close()


@pytest.mark.parametrize("layer", LAYERS)
@pytest.mark.parametrize("R", [1, 5])
def test_full_size_long_context_sublayers(long_ctx, layer, R):
    cfg, dl = long_ctx
    n = LONG - 5  # ragged against the streaming splits
    cache = fill_layer(cfg, dl, layer, n, LONG + 320)
    check_sublayers(cfg, dl, one_layer_model(cfg, layer), cache, layer, n, R, TOL, "long")


def test_full_size_head(full):
    cfg, dm = full
    x = W.synthetic_rows(2, cfg.d, seed=4, std=1.0, index=500)
    logits, am, top1 = dm.head_rows(torch.from_numpy(x).cuda())
    lm = W.weight_tensor(cfg, 0, "lm_head").astype(np.float64)
    h = M.rmsnorm(x.astype(np.float64), np.ones(cfg.d), cfg.eps)
    ref = h @ lm.T
    assert rel_err(logits.cpu().numpy(), ref) < TOL
    am = am.cpu().numpy()
    for r in range(2):
        if margin(ref[r]) > TOL * np.max(np.abs(ref[r])):
            assert am[r] == int(np.argmax(ref[r]))


def test_full_size_decode_equals_verify(full):
    cfg, dm = full
    n = CTX - 100
    for l in LAYERS:
        _fill(cfg, dm, l, n)
    dm.set_context(n, 7)
    all_on = np.ones(2 * cfg.L, dtype=bool)
    drafts = [7]
    for _ in range(4):
        t, _ = dm.draft_step(all_on)
        drafts.append(t)
    pred, a = dm.verify(drafts)
    assert a == 4 and list(pred[:4]) == drafts[1:]


def test_full_size_speculative_equals_ar(full):
    from paper_2602_20217_amd.engine import select_params
    cfg, dm = full
    prompt = W.prompt_ids(cfg.vocab, CTX, 1)
    dm.prefill(prompt)
    ar, _, _ = dm.decode(40, 0)
    dm.prefill(prompt)
    params = select_params((0.074, 1.2e-6, 0.035), "paper_min", 0, tau=0.5, prune_half=True,
                           D=10)
    sd, st, sels = dm.decode(40, 4, 32, params)
    assert np.array_equal(ar, sd)
    assert st.n_selections >= 1
    for s in sels:
        skipped_w = sum(s.w_attn if i % 2 == 0 else s.w_mlp
                        for i in range(2 * cfg.L) if not s.exec[i])
        assert skipped_w == s.j_star and 0 <= s.j_star <= s.C // 2
        assert 1 <= s.gamma_star <= 10 and 0.0 <= s.alpha_hat <= 1.0


def test_full_size_sampling_filter(full):
    """T 0.7 / top-k 50 / top-p 0.95 tables and draws of two rows of 128256
    head logits, against the oracle's filter of the same logits."""
    from oracle import sampling as S
    from paper_2602_20217_amd.engine import sample_filter
    cfg, dm = full
    x = W.synthetic_rows(2, cfg.d, seed=4, std=1.0, index=501)
    logits, _, _ = dm.head_rows(torch.from_numpy(x).cuda())
    ids, probs, cnt, top1, tok = [t.cpu().numpy() for t in
                                  sample_filter(logits, 0.7, 50, 0.95, seed=9, pos0=CTX)]
    lg = logits.cpu().numpy().astype(np.float64)
    for r in range(2):
        prm = S.SamplingParams(0.7, 50, 0.95, 9)
        mg = []
        rid, rpr = S.filtered(lg[r], prm, mg)
        if min(mg) <= 1e-5:
            continue
        assert cnt[r] == len(rid) and ids[r, :cnt[r]].tolist() == rid.tolist()
        np.testing.assert_allclose(probs[r, :cnt[r]], rpr, rtol=2e-5, atol=1e-7)
        assert top1[r] == pytest.approx(1.0 / np.sum(np.exp(lg[r] - lg[r].max())), rel=1e-4)
        dmg = []
        t_ref = S.draw(rid, rpr, S.uniform(9, CTX + r, 2), dmg)
        if min(dmg, default=1.0) > 1e-5:
            assert tok[r] == t_ref


def test_full_size_top_k_one_sampling_is_greedy(full):
    """Speculative sampling with top-k 1 accepts exactly as greedy verification
    does: after the 8K prefill it emits the autoregressive tokens."""
    from paper_2602_20217_amd.engine import select_params
    cfg, dm = full
    prompt = W.prompt_ids(cfg.vocab, CTX, 1)
    dm.prefill(prompt)
    ar, _, _ = dm.decode(40, 0)
    params = select_params((0.074, 1.2e-6, 0.035), "paper_min", 0, tau=0.5, prune_half=True,
                           D=10)
    dm.set_sampling(0.7, 1, 0.95, 4)
    try:
        dm.prefill(prompt)
        sd, st, _ = dm.decode(40, 4, 32, params)
    finally:
        dm.set_sampling(0.0)
    assert np.array_equal(ar, sd)
    assert st.n_rounds >= 1
