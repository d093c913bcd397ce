"""Shared set-up of the GPU parity tests: seeded weights from ``workloads`` are
uploaded through the C ABI and also handed to the oracle."""
import numpy as np

import workloads as W
from oracle import model as M


def rel_err(a, b):
    """Row-wise ||a - b|| / ||b|| (max over rows)."""
    a = np.asarray(a, dtype=np.float64).reshape(-1, np.shape(b)[-1])
    b = np.asarray(b, dtype=np.float64).reshape(-1, np.shape(b)[-1])
    num = np.linalg.norm(a - b, axis=1)
    den = np.maximum(np.linalg.norm(b, axis=1), 1e-300)
    return float(np.max(num / den))


def update_err(got, x_in, ref):
    """Row-wise relative error of a sublayer's own update: (got - x_in) against
    (ref - x_in), max over rows.  A sublayer adds its output to the residual
    row; at long contexts the attention's update is about 1% of that row, so a
    tolerance on the whole row cannot tell a right attention from a zero one,
    while a tolerance on the update can."""
    x = np.asarray(x_in, dtype=np.float64).reshape(-1, np.shape(ref)[-1])
    g = np.asarray(got, dtype=np.float64).reshape(x.shape)
    r = np.asarray(ref, dtype=np.float64).reshape(x.shape)
    return rel_err(g - x, r - x)


def check_rows(got, x_in, ref, tol, what):
    """A sublayer's output rows against the oracle's: the whole residual row and
    the sublayer's own update, each within tol (row-wise relative)."""
    e_row, e_upd = rel_err(got, ref), update_err(got, x_in, ref)
    assert e_row < tol, (what, "row", e_row)
    assert e_upd < tol, (what, "update", e_upd)
    return e_row, e_upd


def build(name, n_max, gamma_max=6, m_rounds=5, cap_max=128, prefill_chunk=64, seed=0):
    from paper_2602_20217_amd.engine import DeviceModel
    cfg = W.config(name)
    weights = W.generate_weights(cfg, seed=seed)
    dm = DeviceModel(cfg, n_max=n_max, gamma_max=gamma_max, m_rounds=m_rounds,
                     cap_max=cap_max, prefill_chunk=prefill_chunk).upload_all(weights)
    return cfg, dm, M.Model(cfg, weights)


def margin(logits_row):
    """Top-1 minus top-2 logit."""
    s = np.sort(np.asarray(logits_row))
    return float(s[-1] - s[-2])


def one_layer_model(cfg, layer, seed=0):
    """Oracle model holding layer `layer` of the seeded weights as its only
    layer (embedding and head zero: only sublayers 1 and 2 are evaluated)."""
    import dataclasses
    c1 = dataclasses.replace(cfg, L=1)
    w = {("embed", -1): np.zeros((16, cfg.d), np.float32),
         ("lm_head", -1): np.zeros((16, cfg.d), np.float32)}
    for k in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"):
        w[(k, 0)] = W.weight_tensor(cfg, seed, k, layer)
    return M.Model(c1, w)


def fill_layer(cfg, dm, layer, n, n_max, seed=3):
    """Seeded keys/values of one layer at positions < n, written to the device
    cache and to a one-layer oracle cache of n_max positions."""
    import dataclasses
    import torch
    K, V = W.synthetic_kv(cfg, n, seed=seed, layer=layer)
    kk, vv = dm.kv_layer(layer)
    kk[:, :n] = torch.from_numpy(K).to(kk.dtype).cuda()
    vv[:, :n] = torch.from_numpy(V).to(vv.dtype).cuda()
    torch.cuda.synchronize()
    cache = M.KVCache(dataclasses.replace(cfg, L=1), n_max)
    cache.K[0][:, :n] = K
    cache.V[0][:, :n] = V
    return cache


def check_sublayers(cfg, dm, model, cache, layer, n, R, tol, tag, seed_index=0):
    """Attention then MLP of `layer` on R rows at positions n.. through the C
    ABI (mode 0: rows store their keys/values, then attend) against the
    one-layer oracle; returns the relative errors."""
    import torch
    dm.set_context(n, 0)
    pos = np.arange(R) + n
    x = W.synthetic_rows(R, cfg.d, seed=4, std=1.0, index=seed_index + 100 + R + layer)
    errs = []
    for sub in (1, 2):
        i = 2 * layer + sub
        out = torch.empty(R, cfg.d, device="cuda")
        dm.sublayer_apply(i, torch.from_numpy(x).cuda(), pos, mode=0, out=out)
        ref = M.sublayer(model, sub, x.astype(np.float64), pos, cache, mode="write")
        got = out.cpu().numpy()
        e, eu = rel_err(got, ref), update_err(got, x, ref)
        print(f"[{tag}] layer {layer} sublayer {sub} R {R}: rel err {e:.2e}, update {eu:.2e}",
              flush=True)
        check_rows(got, x, ref, tol, (tag, layer, sub, R))
        errs.append(eu)
        x = got
    return errs
