"""Oracle decoder and greedy self-speculative decoding (TEST INFRASTRUCTURE ONLY).

Follows Section 2 of the paper: the target model is the composition of 2L
sublayers, f^(2i-1) = Attn_i and f^(2i) = MLP_i, each including its own
normalisation (footnote of Section 2); a skip set leaves the residual stream
unchanged where a sublayer is skipped (f^(S) composes the kept sublayers in
order).  Greedy acceptance follows Section 2.1: a draft token is accepted iff
it equals the target's argmax.

The per-architecture details the paper leaves open (RMSNorm, rotate-half RoPE
with 0-based positions, GQA head mapping, SwiGLU, optional per-head q/k RMSNorm)
follow the standard Llama/Qwen decoder definitions.

Parity pins: closed forms and special cases of every primitive (tests
``test_oracle_model``); prefill rows equal incremental decode rows; verify rows
equal AR rows; an empty skip set gives 100% acceptance; greedy speculative
output equals greedy AR output.  The full random-init model itself has no
published output, so model-level values are pinned only by these invariants.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


# ----------------------------------------------------------------------------
# Primitives
# ----------------------------------------------------------------------------

def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (through float32, ties to even), returned as float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding.  x [..., H, hd], pos broadcastable to x[..., 0, 0].

    Pair (f, f + hd/2) is rotated by angle pos * theta^(-2f/hd); angles in float64.
    """
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None, None] * inv  # [..., 1, half]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Naive attention of one query vector over keys K [n, hd] and values V [n, hd]."""
    s = K @ q / np.sqrt(q.shape[-1])
    s = s - np.max(s)
    p = np.exp(s)
    p = p / np.sum(p)
    return p @ V


# ----------------------------------------------------------------------------
# Model
# ----------------------------------------------------------------------------

class Model:
    """fp64 copy of the generator's weights plus the architecture description."""

    def __init__(self, cfg, weights: dict):
        self.cfg = cfg
        f = lambda a: np.asarray(a, dtype=np.float64)
        self.embed = f(weights[("embed", -1)])
        self.lm_head = f(weights[("lm_head", -1)])
        self.final_norm = np.ones(cfg.d)
        self.layers = []
        for l in range(cfg.L):
            self.layers.append({k: f(weights[(k, l)]) for k in
                                ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")})
            self.layers[-1]["attn_norm"] = np.ones(cfg.d)
            self.layers[-1]["mlp_norm"] = np.ones(cfg.d)
            self.layers[-1]["q_norm"] = np.ones(cfg.hd)
            self.layers[-1]["k_norm"] = np.ones(cfg.hd)

    @property
    def n_sub(self) -> int:
        return 2 * self.cfg.L

    def store(self, a: np.ndarray) -> np.ndarray:
        """Storage rounding of cached keys/values."""
        return to_bf16(a) if self.cfg.dtype == "bf16" else a


class KVCache:
    """Per-layer keys/values [hkv, n_max, hd] in float64 (bf16-valued for bf16 models)."""

    def __init__(self, cfg, n_max: int):
        self.K = [np.zeros((cfg.hkv, n_max, cfg.hd)) for _ in range(cfg.L)]
        self.V = [np.zeros((cfg.hkv, n_max, cfg.hd)) for _ in range(cfg.L)]
        self.n_max = n_max


def attn_qkv(model: Model, layer: int, x: np.ndarray, pos: np.ndarray):
    """Normalised input -> rotated q [R,hq,hd], rotated k [R,hkv,hd], v [R,hkv,hd]."""
    c, W = model.cfg, model.layers[layer]
    h = rmsnorm(x, W["attn_norm"], c.eps)
    q = (h @ W["wq"].T).reshape(-1, c.hq, c.hd)
    k = (h @ W["wk"].T).reshape(-1, c.hkv, c.hd)
    v = (h @ W["wv"].T).reshape(-1, c.hkv, c.hd)
    if c.qk_norm:
        q = rmsnorm(q, W["q_norm"], c.eps)
        k = rmsnorm(k, W["k_norm"], c.eps)
    q = rope(q, pos, c.rope_theta)
    k = rope(k, pos, c.rope_theta)
    return q, k, v


def attn_sublayer(model: Model, layer: int, x: np.ndarray, pos: np.ndarray,
                  cache: KVCache, mode: str) -> np.ndarray:
    """Attn_l applied to rows x [R, d] at positions pos [R]; returns the new residual.

    mode "write": every row's key/value is first stored at its position, then row r
      attends to cache positions 0..pos[r] (causal prefill / decode / verify).
    mode "own":   nothing is stored; row r attends to cache positions 0..pos[r]-1
      plus its own key/value at pos[r] (candidate rows of the selection DP).
    """
    c, W = model.cfg, model.layers[layer]
    q, k, v = attn_qkv(model, layer, x, pos)
    k, v = model.store(k), model.store(v)
    g = c.hq // c.hkv
    if mode == "write":
        for r in range(x.shape[0]):
            cache.K[layer][:, pos[r]] = k[r]
            cache.V[layer][:, pos[r]] = v[r]
    o = np.zeros((x.shape[0], c.hq, c.hd))
    for r in range(x.shape[0]):
        p = int(pos[r])
        for h in range(c.hq):
            kh = h // g
            if mode == "write":
                Kr, Vr = cache.K[layer][kh, :p + 1], cache.V[layer][kh, :p + 1]
            else:
                Kr = np.concatenate([cache.K[layer][kh, :p], k[r, kh][None]], axis=0)
                Vr = np.concatenate([cache.V[layer][kh, :p], v[r, kh][None]], axis=0)
            o[r, h] = softmax_attention(q[r, h], Kr, Vr)
    return x + o.reshape(x.shape[0], -1) @ W["wo"].T


def mlp_sublayer(model: Model, layer: int, x: np.ndarray) -> np.ndarray:
    c, W = model.cfg, model.layers[layer]
    h = rmsnorm(x, W["mlp_norm"], c.eps)
    a = silu(h @ W["w_gate"].T) * (h @ W["w_up"].T)
    return x + a @ W["w_down"].T


def sublayer(model: Model, i: int, x: np.ndarray, pos: np.ndarray, cache: KVCache,
             mode: str = "write") -> np.ndarray:
    """f^(i) for the flattened index i in 1..2L (odd: Attention, even: MLP)."""
    layer = (i - 1) // 2
    if i % 2 == 1:
        return attn_sublayer(model, layer, x, pos, cache, mode)
    return mlp_sublayer(model, layer, x)


def head(model: Model, x: np.ndarray):
    """Final RMSNorm + LM head.  Returns logits [R, V], argmax [R] (lowest index on
    ties), top-1 probability [R]."""
    h = rmsnorm(x, model.final_norm, model.cfg.eps)
    logits = h @ model.lm_head.T
    am = np.argmax(logits, axis=-1)
    mx = logits[np.arange(len(am)), am]
    top1 = 1.0 / np.sum(np.exp(logits - mx[:, None]), axis=-1)
    return logits, am.astype(np.int64), top1


@dataclass
class Forward:
    x: np.ndarray              # final residual rows [R, d]
    snaps: list                # X^(0..2L), each [R, d]
    logits: np.ndarray
    argmax: np.ndarray
    top1: np.ndarray


def forward(model: Model, cache: KVCache, tokens, start: int, exec_mask=None,
            mode: str = "write") -> Forward:
    """Run consecutive tokens at positions start.. through f^(S).

    exec_mask: sequence of 2L booleans (True = sublayer executed); None = all.
    Skipped sublayers are the identity and write no keys/values.
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    pos = start + np.arange(len(tokens))
    x = model.embed[tokens].copy()
    snaps = [x.copy()]
    for i in range(1, model.n_sub + 1):
        if exec_mask is None or exec_mask[i - 1]:
            x = sublayer(model, i, x, pos, cache, mode)
        snaps.append(x.copy())
    logits, am, top1 = head(model, x)
    return Forward(x, snaps, logits, am, top1)


# ----------------------------------------------------------------------------
# Greedy decoding
# ----------------------------------------------------------------------------

@dataclass
class State:
    """Decode state: keys/values exist for positions < P; s is the newest committed
    token (position P, no keys/values yet)."""
    cache: KVCache
    P: int
    s: int
    out: list = field(default_factory=list)
    # history blocks: list of (positions [r_b], snaps list of 2L+1 arrays [r_b, d])
    blocks: list = field(default_factory=list)


def prefill(model: Model, prompt, n_max: int, hist_rows: int) -> State:
    """Run the prompt, commit the first generated token, keep the last hist_rows rows
    of every X^(i) as the first history block."""
    cache = KVCache(model.cfg, n_max)
    n = len(prompt)
    fw = forward(model, cache, prompt, 0)
    st = State(cache=cache, P=n, s=int(fw.argmax[-1]))
    st.out.append(st.s)
    r0 = min(n, hist_rows)
    st.blocks.append((np.arange(n - r0, n), [sn[n - r0:] for sn in fw.snaps]))
    return st


def ar_step(model: Model, st: State) -> int:
    """One greedy autoregressive step: process s at position P, commit the argmax."""
    fw = forward(model, st.cache, [st.s], st.P)
    st.P += 1
    st.s = int(fw.argmax[0])
    st.out.append(st.s)
    return st.s


@dataclass
class Round:
    drafts: list
    draft_top1: list
    verify_argmax: np.ndarray
    n_accepted: int
    emitted: list


def ssd_round(model: Model, st: State, exec_mask, gamma: int, m_rounds: int = 5,
              tau_conf: float = 0.0) -> Round:
    """One greedy self-speculative round (Section 2.1).

    Draft: up to gamma steps of f^(S) starting from s at position P; executed
    attention sublayers store their keys/values at P+k.  With tau_conf > 0 the
    drafting stops after the first draft token whose top-1 probability is below
    tau_conf (the dynamic drafting exit of Section 3, TPT maximization; that token
    is still verified).  Verify: the full model on [s, d_1..d_g] at positions
    P..P+g (g drafts), overwriting those keys/values.  Accept the longest prefix
    with d_i = y_{i-1}; emit d_1..d_a and y_a.
    """
    drafts, tops = [], []
    t = st.s
    for k in range(gamma):
        fw = forward(model, st.cache, [t], st.P + k, exec_mask)
        t = int(fw.argmax[0])
        drafts.append(t)
        tops.append(float(fw.top1[0]))
        if tau_conf > 0 and not tops[-1] >= tau_conf:
            break
    g = len(drafts)
    fv = forward(model, st.cache, [st.s] + drafts, st.P)
    y = fv.argmax
    a = 0
    while a < g and drafts[a] == y[a]:
        a += 1
    emitted = drafts[:a] + [int(y[a])]
    pos = st.P + np.arange(a + 1)
    st.blocks.append((pos, [sn[:a + 1] for sn in fv.snaps]))
    st.blocks = st.blocks[-m_rounds:]
    st.P += a + 1
    st.s = int(y[a])
    st.out.extend(emitted)
    return Round(drafts, tops, y, a, emitted)


def history(st: State):
    """History matrix rows X^(0..2L) and their positions from the kept blocks."""
    pos = np.concatenate([b[0] for b in st.blocks])
    snaps = [np.concatenate([b[1][i] for b in st.blocks], axis=0)
             for i in range(len(st.blocks[0][1]))]
    return pos, snaps


def generate_ar(model: Model, prompt, n_new: int, n_max: int):
    st = prefill(model, prompt, n_max, 1)
    while len(st.out) < n_new:
        ar_step(model, st)
    return st.out[:n_new]
