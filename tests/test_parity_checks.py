"""The GPU sublayer checks can fail (no GPU): on the seeded inputs of the GPU
parity tests, an attention sublayer that returned its input unchanged (a zero
attention output) or 0.9x the oracle's update must be rejected by
``check_rows``, while the oracle's own rows pass.  At these cache lengths the
attention's update is about 1% of the residual row, which is why the check
also compares the update and not only the row."""
import dataclasses

import numpy as np
import pytest

import workloads as W
from oracle import model as M
from tests.gpu_helpers import check_rows, rel_err, update_err

TOL = 2e-2


def _attn_case(name, n, R, index, std):
    """Layer-0 attention of a one-layer oracle model over a seeded cache of n
    positions, on R rows at positions n.. (keys/values written there, as in the
    GPU decode and verify tests)."""
    cfg = W.config(name)
    c1 = dataclasses.replace(cfg, L=1)
    w = {("embed", -1): np.zeros((16, cfg.d), np.float32),
         ("lm_head", -1): np.zeros((16, cfg.d), np.float32)}
    for k in ("wq", "wk", "wv", "wo"):
        w[(k, 0)] = W.weight_tensor(cfg, 0, k, 0)
    for k in ("w_gate", "w_up", "w_down"):
        w[(k, 0)] = np.zeros(W.weight_shape(cfg, k), np.float32)
    model = M.Model(c1, w)
    cache = M.KVCache(c1, n + R)
    K, V = W.synthetic_kv(cfg, n, seed=3, layer=0)
    cache.K[0][:, :n], cache.V[0][:, :n] = K, V
    x = W.synthetic_rows(R, cfg.d, seed=4, std=std, index=index)
    ref = M.sublayer(model, 1, x.astype(np.float64), np.arange(R) + n, cache, mode="write")
    return x.astype(np.float64), ref


@pytest.mark.parametrize("case", [
    # the full Llama-3-8B shape at the 8K workload (first layer, 1 and 5 rows)
    ("llama8b", 8189, 1, 100 + 1 + 0, 1.0),
    ("llama8b", 8189, 5, 100 + 5 + 0, 1.0),
    # the small bf16 decoder over the streaming kernel's shortest cache
    ("small_bf16", 13930, 5, 5 + 70, 0.5),
])
def test_update_check_rejects_planted_attention(case):
    name, n, R, index, std = case
    x, ref = _attn_case(name, n, R, index, std)
    share = float(np.max(np.linalg.norm(ref - x, axis=1) / np.linalg.norm(ref, axis=1)))
    print(f"[{name} n={n} R={R}] attention update / row = {share:.4f}")
    check_rows(ref.astype(np.float32), x, ref, TOL, "oracle")
    # a zero attention output leaves the row within tolerance of the oracle's
    # row, so only the update check catches it
    assert rel_err(x, ref) < TOL
    with pytest.raises(AssertionError):
        check_rows(x, x, ref, TOL, "zero attention")
    with pytest.raises(AssertionError):
        check_rows(x + 0.9 * (ref - x), x, ref, TOL, "0.9x attention")
    assert update_err(x + 0.9 * (ref - x), x, ref) == pytest.approx(0.1, rel=1e-9)
