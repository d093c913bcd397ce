"""GPU vs oracle parity of decode and verify rows over long caches, where the
decode attention splits hold two, three and five 64-position tiles (cache
sizes up to 2048, up to 5120 and up to 12288), and beyond that the streaming
kernel walks two or three tiles per wave (14000 and 70000 positions with the
two kv heads of the small model).  The cache holds seeded synthetic
keys/values up to a ragged length and NaN beyond it, so any read of a position
past a row's length shows up in the result.  Every call goes through the C
ABI; tolerance 2e-2 (bf16)."""
import numpy as np
import pytest

import workloads as W
from oracle import model as M
from tests.gpu_helpers import build, rel_err, check_rows

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOL = 2e-2


@pytest.fixture(scope="module", params=[1500, 3000, 6000, 14000, 70000])
def setup(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    n_max = request.param
    print(f"\n[setup] small_bf16, n_max {n_max}", flush=True)
    cfg, dm, model = build("small_bf16", n_max=n_max, gamma_max=4, m_rounds=5, cap_max=128,
                           prefill_chunk=64)
    yield n_max, cfg, dm, model
    dm.close()


def _fill(cfg, dm, n_max, n):
    """Seeded keys/values at positions < n, NaN at and beyond n (device), and the
    same values in an oracle cache."""
    cache = M.KVCache(cfg, n_max)
    for l in range(cfg.L):
        K, V = W.synthetic_kv(cfg, n, seed=3, layer=l)
        kk, vv = dm.kv_layer(l)
        kk[:, :n] = torch.from_numpy(K).to(torch.bfloat16).cuda()
        vv[:, :n] = torch.from_numpy(V).to(torch.bfloat16).cuda()
        kk[:, n:] = float("nan")
        vv[:, n:] = float("nan")
        cache.K[l][:, :n] = K
        cache.V[l][:, :n] = V
    torch.cuda.synchronize()
    return cache


@pytest.mark.parametrize("R", [1, 5])
@pytest.mark.parametrize("back", [70, 300])
def test_long_cache_rows(setup, R, back):
    """Rows at positions n..n+R-1 (keys/values written there, attending to all
    earlier positions) for every sublayer, then the head."""
    n_max, cfg, dm, model = setup
    n = n_max - back  # ragged against 64- and 256-position splits
    cache = _fill(cfg, dm, n_max, n)
    dm.set_context(n, 0)
    pos = np.arange(R) + n
    x = W.synthetic_rows(R, cfg.d, seed=4, std=0.5, index=R + back)
    xd = torch.from_numpy(x).cuda()
    xo = x.astype(np.float64)
    for i in range(1, 2 * cfg.L + 1):
        out = torch.empty_like(xd)
        dm.sublayer_apply(i, xd, pos, mode=0, out=out)
        x_in = xd.cpu().numpy()
        xo = M.sublayer(model, i, xo, pos, cache, mode="write")
        got = out.cpu().numpy()
        assert np.all(np.isfinite(got)), i
        check_rows(got, x_in, xo, TOL, (n_max, back, R, i))
        xd = out
        xo = got.astype(np.float64)
    logits, am, top1 = dm.head_rows(xd)
    lg0, _, _ = M.head(model, xo)
    assert rel_err(logits.cpu().numpy(), lg0) < TOL


def test_long_cache_decode_equals_verify(setup):
    """A verify row and the decode step at the same position give identical bits."""
    n_max, cfg, dm, model = setup
    n = n_max - 150
    _fill(cfg, dm, n_max, n)
    dm.set_context(n, 3)
    full = np.ones(2 * cfg.L, dtype=bool)
    drafts = [3]
    for _ in range(4):
        t, _ = dm.draft_step(full)
        drafts.append(t)
    pred, a = dm.verify(drafts)
    # full-model drafts are the target's own greedy tokens
    assert a == 4
    assert list(pred[:4]) == drafts[1:]
