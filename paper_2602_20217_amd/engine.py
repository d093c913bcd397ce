"""Device-side model and call helpers over the C ABI.

PyTorch supplies device memory and the stream; every computation runs in
libknapspec's HIP kernels.  ``DeviceModel`` uploads row-major weights, packs
them into the kernels' layout with ``ks_pack_matrix`` / ``ks_pack_gate_up``,
allocates the KV cache and workspace, and exposes the decode-step calls.
"""
from __future__ import annotations

import ctypes as C
import math

import numpy as np
import torch

from . import _lib as K

_PER_LAYER = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def _ptr(t: torch.Tensor) -> int:
    return t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _bf16_bits(a: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("bf16 model weights must hold exactly representable bf16 values")
    return (u >> 16).astype(np.uint16)


def select_params(c, quant_mode="paper_min", bins=0, tau=0.5, prune_half=True, D=10,
                  t_head=0.0):
    return K.SelectParams(float(c[0]), float(c[1]), float(c[2]),
                          K.KS_QUANT_BINS if quant_mode == "bins" else K.KS_QUANT_PAPER_MIN,
                          int(bins), float(tau), 1 if prune_half else 0, int(D), float(t_head))


class DeviceModel:
    """One decoder on one GPU behind a ks_ctx.

    cfg needs attributes L, d, hq, hkv, hd, ffn, vocab, eps, rope_theta, qk_norm,
    dtype ("f32" or "bf16").  Call ``upload(kind, layer, array)`` for every weight
    (kinds embed, lm_head, wq, wk, wv, wo, w_gate, w_up, w_down; row-major [out, in]
    float32 arrays, bf16-valued for bf16 models), then ``finalize()``.
    """

    def __init__(self, cfg, n_max: int, gamma_max: int = 8, m_rounds: int = 5,
                 cap_max: int = 256, prefill_chunk: int = 256, device: str = "cuda:0"):
        self.cfg = cfg
        self.dev = torch.device(device)
        self.bf = cfg.dtype == "bf16"
        self.desc = K.ModelDesc(cfg.L, cfg.d, cfg.hq, cfg.hkv, cfg.hd, cfg.ffn, cfg.vocab,
                                n_max, 1 if cfg.qk_norm else 0,
                                K.KS_BF16 if self.bf else K.KS_F32, float(cfg.eps),
                                float(cfg.rope_theta))
        self.lim = K.Limits(gamma_max, m_rounds, cap_max, prefill_chunk)
        kvb = K.ks_kv_cache_bytes(C.byref(self.desc))
        wsb = K.ks_workspace_bytes(C.byref(self.desc), C.byref(self.lim))
        if kvb == 0 or wsb == 0:
            raise K.KsError(K.KS_EINVAL, K.last_error())
        self.kv = torch.zeros(kvb, dtype=torch.uint8, device=self.dev)
        self.ws = torch.zeros(wsb, dtype=torch.uint8, device=self.dev)
        wdt = torch.int16 if self.bf else torch.float32
        L, d = cfg.L, cfg.d
        nq = (cfg.hq + 2 * cfg.hkv) * cfg.hd
        e = lambda *s: torch.empty(*s, dtype=wdt, device=self.dev)
        self.w = {
            "embed": e(cfg.vocab, d), "lm_head": e(cfg.vocab, d),
            "wqkv": [e(nq, d) for _ in range(L)], "wo": [e(d, cfg.hq * cfg.hd) for _ in range(L)],
            "w_gate_up": [e(2 * cfg.ffn, d) for _ in range(L)],
            "w_down": [e(d, cfg.ffn) for _ in range(L)],
        }
        ones = lambda n: torch.ones(n, dtype=torch.float32, device=self.dev)
        self.gains = {"final_norm": ones(d), "attn_norm": [ones(d) for _ in range(L)],
                      "mlp_norm": [ones(d) for _ in range(L)],
                      "q_norm": [ones(cfg.hd) for _ in range(L)],
                      "k_norm": [ones(cfg.hd) for _ in range(L)]}
        self._pending = {}
        self._done = set()
        self.ctx = None

    # ------------------------------------------------------------ weights
    def _to_dev(self, a: np.ndarray) -> torch.Tensor:
        if self.bf:
            return torch.from_numpy(_bf16_bits(a).view(np.int16)).to(self.dev)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.dev)

    def _pack(self, src: torch.Tensor, dst: torch.Tensor):
        N, Kd = src.shape
        K.ks_pack_matrix(_ptr(src), _ptr(dst), N, Kd, self.desc.dtype, _stream())

    def upload(self, kind: str, layer: int, a: np.ndarray):
        if kind == "embed":
            self.w["embed"].copy_(self._to_dev(a))
        elif kind == "lm_head":
            self._pack(self._to_dev(a), self.w["lm_head"])
        elif kind in ("wq", "wk", "wv"):
            p = self._pending.setdefault(("qkv", layer), {})
            p[kind] = a
            if len(p) == 3:
                cat = self._to_dev(np.concatenate([p["wq"], p["wk"], p["wv"]], axis=0))
                c = self.cfg
                K.ks_pack_qkv(_ptr(cat), _ptr(self.w["wqkv"][layer]), c.hq, c.hkv, c.hd, c.d,
                              self.desc.dtype, _stream())
                torch.cuda.current_stream().synchronize()
                del self._pending[("qkv", layer)]
        elif kind == "wo":
            self._pack(self._to_dev(a), self.w["wo"][layer])
        elif kind in ("w_gate", "w_up"):
            p = self._pending.setdefault(("gu", layer), {})
            p[kind] = self._to_dev(a)
            if len(p) == 2:
                K.ks_pack_gate_up(_ptr(p["w_gate"]), _ptr(p["w_up"]),
                                  _ptr(self.w["w_gate_up"][layer]), self.cfg.ffn, self.cfg.d,
                                  self.desc.dtype, _stream())
                torch.cuda.current_stream().synchronize()
                del self._pending[("gu", layer)]
        elif kind == "w_down":
            self._pack(self._to_dev(a), self.w["w_down"][layer])
        else:
            raise KeyError(kind)
        self._done.add((kind, layer))

    def upload_all(self, weights: dict):
        for (kind, layer), a in weights.items():
            self.upload(kind, layer, a)
        return self.finalize()

    def finalize(self):
        need = 2 + 7 * self.cfg.L
        if len(self._done) != need or self._pending:
            raise RuntimeError(f"uploaded {len(self._done)} of {need} weight tensors")
        torch.cuda.current_stream().synchronize()
        L = self.cfg.L
        arr = lambda ts: (C.c_void_p * L)(*[_ptr(t) for t in ts])
        self._arrays = {k: arr(self.w[k]) for k in ("wqkv", "wo", "w_gate_up", "w_down")}
        self._arrays.update({k: arr(self.gains[k]) for k in
                             ("attn_norm", "mlp_norm", "q_norm", "k_norm")})
        A = self._arrays
        cast = lambda x: C.cast(x, C.POINTER(C.c_void_p))
        self.weights = K.Weights(_ptr(self.w["embed"]), _ptr(self.w["lm_head"]),
                                 _ptr(self.gains["final_norm"]), cast(A["attn_norm"]),
                                 cast(A["wqkv"]), cast(A["wo"]), cast(A["q_norm"]),
                                 cast(A["k_norm"]), cast(A["mlp_norm"]), cast(A["w_gate_up"]),
                                 cast(A["w_down"]))
        ctx = C.c_void_p()
        K.ks_create(C.byref(self.desc), C.byref(self.lim), C.byref(self.weights),
                    _ptr(self.kv), self.kv.numel(), _ptr(self.ws), self.ws.numel(), _stream(),
                    C.byref(ctx))
        self.ctx = ctx
        torch.cuda.current_stream().synchronize()
        return self

    def resized(self, n_max: int) -> "DeviceModel":
        """A second context over the same uploaded weights, with its own KV cache
        of n_max positions and workspace (the decode attention splits follow the
        cache size, so a deployment sizes the cache to its context)."""
        if self.ctx is None:
            raise RuntimeError("finalize() the weights first")
        other = DeviceModel.__new__(DeviceModel)
        other.cfg, other.dev, other.bf = self.cfg, self.dev, self.bf
        d = self.desc
        other.desc = K.ModelDesc(d.L, d.d, d.hq, d.hkv, d.hd, d.ffn, d.vocab, n_max, d.qk_norm,
                                 d.dtype, d.eps, d.rope_theta)
        other.lim = self.lim
        kvb = K.ks_kv_cache_bytes(C.byref(other.desc))
        wsb = K.ks_workspace_bytes(C.byref(other.desc), C.byref(other.lim))
        if kvb == 0 or wsb == 0:
            raise K.KsError(K.KS_EINVAL, K.last_error())
        other.kv = torch.zeros(kvb, dtype=torch.uint8, device=self.dev)
        other.ws = torch.zeros(wsb, dtype=torch.uint8, device=self.dev)
        other.w, other.gains = self.w, self.gains
        other._pending, other._done = {}, set(self._done)
        other.ctx = None
        return other.finalize()

    def close(self):
        if self.ctx is not None:
            K.ks_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------ cache views
    def kv_layer(self, layer: int):
        """(K, V) views [hkv, n_max, hd] of one layer's cache (bf16 or float32)."""
        c = self.cfg
        es = 2 if self.bf else 4
        n = c.hkv * self.desc.n_max * c.hd * es
        base = 2 * layer * n
        dt = torch.bfloat16 if self.bf else torch.float32
        kk = self.kv[base:base + n].view(dt).view(c.hkv, self.desc.n_max, c.hd)
        vv = self.kv[base + n:base + 2 * n].view(dt).view(c.hkv, self.desc.n_max, c.hd)
        return kk, vv

    # ------------------------------------------------------------ decode calls
    def prefill(self, tokens) -> int:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        out = C.c_int32()
        K.ks_prefill(self.ctx, t.ctypes.data, len(t), C.byref(out))
        return out.value

    def set_context(self, n_cached: int, last_token: int):
        K.ks_set_context(self.ctx, int(n_cached), int(last_token))

    def draft_step(self, exec_mask):
        m = np.ascontiguousarray(np.asarray(exec_mask, dtype=bool).astype(np.uint8))
        tok, p = C.c_int32(), C.c_float()
        K.ks_draft_step(self.ctx, m.ctypes.data, C.byref(tok), C.byref(p))
        return tok.value, p.value

    def verify(self, tokens):
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        pred = np.zeros(len(t), dtype=np.int32)
        a = C.c_int()
        K.ks_verify(self.ctx, t.ctypes.data, len(t) - 1, pred.ctypes.data, C.byref(a))
        return pred, a.value

    def select(self, params: K.SelectParams, debug_cells: int = 0):
        out = K.Selection()
        dbg = None
        if debug_cells:
            n = 2 * self.cfg.L + 1
            self._dbg = {
                "bits": np.zeros((n, debug_cells), dtype=np.uint8),
                "reach": np.zeros((n, debug_cells), dtype=np.uint8),
                "sig_e": np.zeros((n, debug_cells), dtype=np.float64),
                "sig_s": np.zeros((n, debug_cells), dtype=np.float64),
                "n_match": np.zeros(debug_cells, dtype=np.int32),
            }
            g = self._dbg
            dbg = K.SelectionDebug(debug_cells,
                                   g["bits"].ctypes.data_as(C.POINTER(C.c_uint8)),
                                   g["reach"].ctypes.data_as(C.POINTER(C.c_uint8)),
                                   g["sig_e"].ctypes.data_as(C.POINTER(C.c_double)),
                                   g["sig_s"].ctypes.data_as(C.POINTER(C.c_double)),
                                   g["n_match"].ctypes.data_as(C.POINTER(C.c_int)))
        K.ks_knapsack_select(self.ctx, C.byref(params), C.byref(out),
                             C.byref(dbg) if dbg is not None else None)
        return (out, self._dbg) if debug_cells else out

    def set_draft_policy(self, tau_conf: float = 0.0, gamma_source: str = "fixed"):
        """Dynamic drafting exit below tau_conf (0 disables) and the draft cap of
        each round: the call's gamma ("fixed") or min(gamma*, gamma) ("selected")."""
        src = {"fixed": K.KS_GAMMA_FIXED, "selected": K.KS_GAMMA_SELECTED}[gamma_source]
        K.ks_set_draft_policy(self.ctx, C.byref(K.DraftPolicy(tau_conf, src)))

    def set_sampling(self, temperature: float = 0.0, top_k: int = 50, top_p: float = 0.95,
                     seed: int = 0):
        """Speculative sampling with the T / top-k / top-p filter and Philox
        stream `seed`; temperature <= 0 returns to greedy decoding."""
        K.ks_set_sampling(self.ctx, C.byref(K.Sampling(temperature, top_k, top_p, seed)))

    def generate(self, prompt, n_new: int, gamma: int, reselect_every: int = 32,
                 params: K.SelectParams | None = None, max_sel_log: int = 256):
        p = np.ascontiguousarray(prompt, dtype=np.int32)
        out = np.zeros(n_new, dtype=np.int32)
        st = K.GenStats()
        log = (K.Selection * max_sel_log)()
        K.ks_generate(self.ctx, p.ctypes.data, len(p), n_new, gamma, reselect_every,
                      C.byref(params) if params is not None else None, out.ctypes.data,
                      C.byref(st), log, max_sel_log)
        sels = [log[i] for i in range(min(st.n_selections, max_sel_log))]
        return out, st, sels

    def decode(self, n_new: int, gamma: int, reselect_every: int = 32,
               params: K.SelectParams | None = None, max_sel_log: int = 256):
        """Generation loop from the current state (no prefill)."""
        out = np.zeros(n_new, dtype=np.int32)
        st = K.GenStats()
        log = (K.Selection * max_sel_log)()
        K.ks_decode(self.ctx, n_new, gamma, reselect_every,
                    C.byref(params) if params is not None else None, out.ctypes.data,
                    C.byref(st), log, max_sel_log)
        sels = [log[i] for i in range(min(st.n_selections, max_sel_log))]
        return out, st, sels

    def profile_decode(self, exec_mask=None, steps: int = 8, per_kernel: bool = True) -> dict:
        """Mean per-launch duration (ms) of every kernel class of a decode step."""
        m = None
        if exec_mask is not None:
            m = np.ascontiguousarray(np.asarray(exec_mask, dtype=bool).astype(np.uint8))
        pr = K.KernelProfile()
        K.ks_profile_decode(self.ctx, m.ctypes.data if m is not None else None, steps,
                            1 if per_kernel else 0, C.byref(pr))
        return {"ms": {n: pr.ms[i] for i, n in enumerate(K.KS_KC_NAMES)},
                "launches": {n: pr.launches[i] for i, n in enumerate(K.KS_KC_NAMES)},
                "ms_step": pr.ms_step, "steps": pr.steps}

    def sublayer_apply(self, i: int, x: torch.Tensor, pos, mode: int = 0, out=None):
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        out = x if out is None else out
        K.ks_sublayer_apply(self.ctx, i, _ptr(x), _ptr(out), pos.ctypes.data, len(pos), mode)
        return out

    def head_rows(self, x: torch.Tensor, want_logits: bool = True):
        R = x.shape[0]
        logits = (torch.empty(R, self.cfg.vocab, dtype=torch.float32, device=self.dev)
                  if want_logits else None)
        am = torch.empty(R, dtype=torch.int32, device=self.dev)
        top1 = torch.empty(R, dtype=torch.float32, device=self.dev)
        K.ks_head_rows(self.ctx, _ptr(x), R, _ptr(logits) if want_logits else None, _ptr(am),
                       _ptr(top1))
        return logits, am, top1


# ------------------------------------------------------- raw-pointer calls
def hidden_cos(X: torch.Tensor, Y: torch.Tensor) -> torch.Tensor:
    """mean row cosine of every [r, d] group of X [G, r, d] against Y [r, d]."""
    G, r, d = X.shape
    out = torch.empty(G, dtype=torch.float32, device=X.device)
    K.ks_hidden_cos(_ptr(X), _ptr(Y), G, r, d, _ptr(out), _stream())
    return out


def sample_filter(logits: torch.Tensor, temperature: float, top_k: int, top_p: float,
                  seed: int = 0, pos0: int | None = None, purpose: int = 2):
    """Filter tables (ids, probs, counts), unfiltered top-1 probability and, when
    pos0 is given, the draw of row r at position pos0 + r."""
    R, V = logits.shape
    dev = logits.device
    s = K.Sampling(temperature, top_k, top_p, seed)
    ws_b = K.ks_sample_workspace_bytes(R, V, top_k)  # 0: the call reports the bad argument
    ws = torch.empty(max(ws_b, 256), dtype=torch.uint8, device=dev)
    ids = torch.empty(R, K.KS_SAMPLE_KMAX, dtype=torch.int32, device=dev)
    probs = torch.empty(R, K.KS_SAMPLE_KMAX, dtype=torch.float32, device=dev)
    cnt = torch.empty(R, dtype=torch.int32, device=dev)
    top1 = torch.empty(R, dtype=torch.float32, device=dev)
    tok = torch.empty(R, dtype=torch.int32, device=dev) if pos0 is not None else None
    K.ks_sample_filter(_ptr(logits), R, V, logits.stride(0), C.byref(s), pos0 or 0, purpose,
                       _ptr(ids), _ptr(probs), _ptr(cnt), _ptr(top1),
                       _ptr(tok) if tok is not None else None, _ptr(ws), ws_b, _stream())
    return ids, probs, cnt, top1, tok


def spec_accept(p_ids, p_probs, p_cnt, q_ids, q_probs, q_cnt, drafts: torch.Tensor, seed: int,
                pos0: int):
    """Acceptance chain of one round on device tables: (accepted drafts, token)."""
    g = drafts.numel()
    out = torch.empty(2, dtype=torch.int32, device=p_ids.device)
    K.ks_spec_accept(_ptr(p_ids), _ptr(p_probs), _ptr(p_cnt), _ptr(q_ids), _ptr(q_probs),
                     _ptr(q_cnt), _ptr(drafts), g, seed, pos0, _ptr(out), _stream())
    a, t = out.cpu().tolist()
    return a, t


def sample_uniforms(seed: int, pos: torch.Tensor, purpose: int) -> torch.Tensor:
    out = torch.empty(pos.numel(), dtype=torch.float32, device=pos.device)
    K.ks_sample_uniforms(seed, _ptr(pos), pos.numel(), purpose, _ptr(out), _stream())
    return out


def knapsack_quantize(t: np.ndarray, s: np.ndarray, bins: int):
    t = np.ascontiguousarray(t, dtype=np.float64)
    s = np.ascontiguousarray(s, dtype=np.float64)
    B, n = t.shape
    w = np.zeros((B, n), dtype=np.int32)
    q = np.zeros((B, n), dtype=np.int32)
    K.ks_knapsack_quantize(t.ctypes.data, s.ctypes.data, B, n, bins, w.ctypes.data, q.ctypes.data)
    return w, q


def knapsack_batch(w: torch.Tensor, q: torch.Tensor, C_cap: int, max_skip: int):
    B, n = w.shape
    best = torch.empty(B, C_cap + 1, dtype=torch.int32, device=w.device)
    bits = torch.empty(B, n, C_cap // 64 + 1, dtype=torch.int64, device=w.device)
    K.ks_knapsack_batch(_ptr(w), _ptr(q), B, n, C_cap, max_skip, _ptr(best), _ptr(bits), _stream())
    return best, bits


def knapsack_backtrack(bits: torch.Tensor, w: torch.Tensor, C_cap: int, j: torch.Tensor):
    B, n = w.shape
    skip = torch.empty(B, n, dtype=torch.uint8, device=w.device)
    err = torch.empty(B, dtype=torch.int32, device=w.device)
    K.ks_knapsack_backtrack(_ptr(bits), _ptr(w), B, n, C_cap, _ptr(j), _ptr(skip), _ptr(err),
                            _stream())
    return skip, err


def knapsack_batch_select(best, bits, w, s, C_cap: int, D: int = 10):
    B, n = w.shape
    dev = w.device
    js = torch.empty(B, dtype=torch.int32, device=dev)
    gs = torch.empty(B, dtype=torch.int32, device=dev)
    tpt = torch.empty(B, dtype=torch.float64, device=dev)
    skip = torch.empty(B, n, dtype=torch.uint8, device=dev)
    K.ks_knapsack_batch_select(_ptr(best), _ptr(bits), _ptr(w), _ptr(s), B, n, C_cap, D, _ptr(js),
                               _ptr(gs), _ptr(tpt), _ptr(skip), _stream())
    return js, gs, tpt, skip
