"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module generates *inputs only*: model weights, prompts, knapsack-instance
latencies and similarity scores, and synthetic KV-cache contents.  It contains
none of the method's arithmetic (no normalisation, attention, quantisation,
dynamic programming or selection), so that the oracle and the HIP path, which
both read its outputs, share no computation.

Every tensor is drawn from its own ``numpy.random.PCG64([seed, index])`` stream,
so a single tensor (one layer's weight, say) can be regenerated on its own.
Index order (fixed, part of the data format):

* 0: token embedding ``[vocab, d]``
* 1: LM head ``[vocab, d]``
* 16 + 8*l + k for layer ``l`` and kind ``k``:
  0 ``wq [hq*hd, d]``, 1 ``wk [hkv*hd, d]``, 2 ``wv [hkv*hd, d]``,
  3 ``wo [d, hq*hd]``, 4 ``w_gate [ffn, d]``, 5 ``w_up [ffn, d]``,
  6 ``w_down [d, ffn]``.

Weights are N(0, 0.02^2); the two output projections ``wo`` and ``w_down`` use
std 0.02/sqrt(2L).  Norm gains are all ones.  For bf16 models every weight is
rounded to the nearest bf16 value (round-to-nearest-even) at generation time, so
the float32 arrays returned here hold exactly representable bf16 values and
``bf16_bits`` recovers their bit patterns losslessly.
"""
from __future__ import annotations

import concurrent.futures as _cf
import math
import os
from dataclasses import dataclass, asdict

import numpy as np

__all__ = [
    "ModelConfig", "CONFIGS", "config", "weight_names", "weight_shape",
    "weight_tensor", "generate_weights", "bf16_bits", "round_to_bf16",
    "prompt_ids", "knapsack_instances", "synthetic_kv", "synthetic_rows",
    "TINY_LATENCY",
]


@dataclass(frozen=True)
class ModelConfig:
    name: str
    L: int
    d: int
    hq: int
    hkv: int
    hd: int
    ffn: int
    vocab: int
    eps: float
    rope_theta: float
    qk_norm: bool
    dtype: str  # "f32" or "bf16"

    def asdict(self):
        return asdict(self)


CONFIGS = {
    # Tiny Llama-style decoder, fp32 (small enough for brute force over 2^8 masks).
    "tiny": ModelConfig("tiny", L=4, d=256, hq=4, hkv=2, hd=64, ffn=1024, vocab=1024,
                        eps=1e-6, rope_theta=1e4, qk_norm=False, dtype="f32"),
    # Llama-3-8B shape, bf16.
    "llama8b": ModelConfig("llama8b", L=32, d=4096, hq=32, hkv=8, hd=128, ffn=14336,
                           vocab=128256, eps=1e-6, rope_theta=5e5, qk_norm=False,
                           dtype="bf16"),
    # Qwen3-8B shape, bf16, per-head q/k RMSNorm.
    "qwen8b": ModelConfig("qwen8b", L=36, d=4096, hq=32, hkv=8, hd=128, ffn=12288,
                          vocab=151936, eps=1e-6, rope_theta=1e6, qk_norm=True,
                          dtype="bf16"),
    # Small bf16 decoders with the 8B head geometry (hd=128, 4 q heads per kv head),
    # used for oracle-checkable parity of the bf16 kernels.
    "small_bf16": ModelConfig("small_bf16", L=2, d=1024, hq=8, hkv=2, hd=128, ffn=2816,
                              vocab=4096, eps=1e-6, rope_theta=5e5, qk_norm=False,
                              dtype="bf16"),
    "small_qwen_bf16": ModelConfig("small_qwen_bf16", L=2, d=1024, hq=8, hkv=2, hd=128,
                                   ffn=2048, vocab=4096, eps=1e-6, rope_theta=1e6,
                                   qk_norm=True, dtype="bf16"),
    # The same geometry with eight layers (16 sublayers): enough DP stages and
    # reachable budgets for the selection parity of the bf16 kernels.
    "deep_bf16": ModelConfig("deep_bf16", L=8, d=1024, hq=8, hkv=2, hd=128, ffn=2816,
                             vocab=4096, eps=1e-6, rope_theta=5e5, qk_norm=False,
                             dtype="bf16"),
}

# Explicit latency coefficients (c1, c2, c3) for the tiny model: t_MLP = c1,
# t_Attn(n) = c2 * n + c3 (arbitrary time unit).
TINY_LATENCY = (1.0, 0.01, 0.2)


def config(name: str) -> ModelConfig:
    return CONFIGS[name]


_KINDS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def weight_names(cfg: ModelConfig):
    names = [("embed", -1), ("lm_head", -1)]
    for l in range(cfg.L):
        names += [(k, l) for k in _KINDS]
    return names


def weight_shape(cfg: ModelConfig, kind: str):
    q, kv = cfg.hq * cfg.hd, cfg.hkv * cfg.hd
    return {
        "embed": (cfg.vocab, cfg.d), "lm_head": (cfg.vocab, cfg.d),
        "wq": (q, cfg.d), "wk": (kv, cfg.d), "wv": (kv, cfg.d), "wo": (cfg.d, q),
        "w_gate": (cfg.ffn, cfg.d), "w_up": (cfg.ffn, cfg.d), "w_down": (cfg.d, cfg.ffn),
    }[kind]


def _tensor_index(kind: str, layer: int) -> int:
    if kind == "embed":
        return 0
    if kind == "lm_head":
        return 1
    return 16 + 8 * layer + _KINDS.index(kind)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round a float32 array of finite values to the nearest bf16 value (ties to
    even).  Works in place on float32 input and returns it."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    t = u >> 16
    t &= 1
    t += 0x7FFF
    u += t  # finite values cannot wrap: |x| < 2^128 keeps u + 0xFFFF below 2^32
    u &= 0xFFFF0000
    return a


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Bit patterns (uint16) of a float32 array whose values are bf16-representable."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("array holds values that are not exactly bf16")
    return (u >> 16).astype(np.uint16)


def weight_tensor(cfg: ModelConfig, seed: int, kind: str, layer: int = -1) -> np.ndarray:
    """One weight tensor, float32, row-major [out, in] (bf16-rounded for bf16 models)."""
    shape = weight_shape(cfg, kind)
    std = 0.02
    if kind in ("wo", "w_down"):
        std = 0.02 / math.sqrt(2 * cfg.L)
    g = np.random.Generator(np.random.PCG64([seed, _tensor_index(kind, layer)]))
    a = g.standard_normal(shape, dtype=np.float32)
    a *= np.float32(std)
    if cfg.dtype == "bf16":
        a = round_to_bf16(a)
    return a


def generate_weights(cfg: ModelConfig, seed: int = 0, threads: int | None = None,
                     consume=None):
    """Generate every weight tensor.

    Without ``consume`` returns ``{(kind, layer): array}``.  With ``consume`` (a
    callable ``consume(kind, layer, array)``), each tensor is handed over as soon
    as it exists and not kept, which bounds host memory for 8B-parameter shapes.
    """
    names = weight_names(cfg)
    threads = threads or min(16, os.cpu_count() or 1)
    out = {}
    window = []  # futures in flight, consumed in submission order
    with _cf.ThreadPoolExecutor(max_workers=threads) as ex:
        it = iter(names)
        while True:
            while len(window) < 2 * threads:
                nxt = next(it, None)
                if nxt is None:
                    break
                window.append((nxt, ex.submit(weight_tensor, cfg, seed, nxt[0], nxt[1])))
            if not window:
                break
            (k, l), f = window.pop(0)
            a = f.result()
            if consume is None:
                out[(k, l)] = a
            else:
                consume(k, l, a)
            del a, f
    return out if consume is None else None


def prompt_ids(vocab: int, n: int, seed: int = 1) -> np.ndarray:
    """Uniform random token ids in [0, vocab), int32."""
    g = np.random.Generator(np.random.PCG64([seed, 0]))
    return g.integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def knapsack_instances(B: int = 1024, n_items: int = 72, seed: int = 2):
    """Isolated knapsack instances with the latencies of a Llama-8B-shaped decoder.

    Items alternate Attention (even index) and MLP (odd index) sublayers.  For
    instance b with context length n_b, log-uniform in [1024, 131072]:

    * Attention item latency  t = a_i + b_i * n_b, a_i = 10.49us*U[0.9,1.1],
      b_i = 0.512ns*U[0.9,1.1] (HBM-roofline figures of that shape on MI355X);
    * MLP item latency        t = 44.04us*U[0.9,1.1];
    * per-item similarity     s ~ U[0.9, 1.0].

    Returns dict with ``ctx`` int64[B], ``t`` float64[B, n] (seconds) and
    ``s`` float64[B, n].
    """
    g = np.random.Generator(np.random.PCG64([seed, 0]))
    ctx = np.rint(np.exp(g.uniform(math.log(1024), math.log(131072), size=B))).astype(np.int64)
    a = 10.49e-6 * g.uniform(0.9, 1.1, size=(B, n_items))
    b = 0.512e-9 * g.uniform(0.9, 1.1, size=(B, n_items))
    m = 44.04e-6 * g.uniform(0.9, 1.1, size=(B, n_items))
    s = g.uniform(0.9, 1.0, size=(B, n_items))
    is_attn = (np.arange(n_items) % 2) == 0
    t = np.where(is_attn[None, :], a + b * ctx[:, None].astype(np.float64), m)
    return {"ctx": ctx, "t": t, "s": s}


def synthetic_kv(cfg: ModelConfig, n: int, seed: int = 3, layer: int = 0):
    """Random cache contents K, V of shape [hkv, n, hd], float32 (bf16 values for bf16
    models), scaled like the keys/values of the random-init model (std ~1.28)."""
    g = np.random.Generator(np.random.PCG64([seed, 1000 + layer]))
    K = g.standard_normal((cfg.hkv, n, cfg.hd), dtype=np.float32) * np.float32(1.28)
    V = g.standard_normal((cfg.hkv, n, cfg.hd), dtype=np.float32) * np.float32(1.28)
    if cfg.dtype == "bf16":
        K, V = round_to_bf16(K), round_to_bf16(V)
    return K, V


def synthetic_rows(rows: int, d: int, seed: int = 4, std: float = 1.0, index: int = 0):
    """Random residual-stream rows [rows, d], float32."""
    g = np.random.Generator(np.random.PCG64([seed, 2000 + index]))
    return g.standard_normal((rows, d), dtype=np.float32) * np.float32(std)


def synthetic_logits(rows: int, vocab: int, seed: int = 5, std: float = 3.0, ties: bool = False,
                     index: int = 0):
    """Random LM-head outputs [rows, vocab], float32: normal with the given std;
    ties=True rounds them to multiples of 1/4, so equal logits occur at the top
    and across the top-k boundary."""
    g = np.random.Generator(np.random.PCG64([seed, 3000 + index]))
    z = g.standard_normal((rows, vocab), dtype=np.float32) * np.float32(std)
    if ties:
        z = np.round(z * 4.0).astype(np.float32) / np.float32(4.0)
    return z
