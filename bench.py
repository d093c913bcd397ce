#!/usr/bin/env python
"""Decode throughput of the self-speculative decode step on one MI355X.

Workload (default): Llama-3-8B-shaped decoder (32 layers, d 4096, 32 query / 8
kv heads of 128, SwiGLU 14336, vocab 128256), random init, bf16 weights and KV
cache; 8192-token random-id prompt; 256 generated tokens; draft length 4; the
skip mask is re-selected every 32 generated tokens by the knapsack DP.

One step = prefill (untimed, restores the state) + the timed generation of
256 tokens, selections included.  The AR baseline runs the same kernels with
no drafting.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


# HBM bytes per launch of the decode gate/up product counted by two rocprofv3
# counter passes (FETCH_SIZE, WRITE_SIZE) scaled by a 256 MiB reference kernel
# (profiles/decode_kernels_llama8b_ctx8k_counters.txt); valid only while the
# product's source has the recorded digest
GATE_UP_TRAFFIC = (235195374, "b43cae1e77f45e6f25cf18667f5525a46a813a985c3fd72cf5e22a880a324183")


def gate_up_traffic(cfg):
    """Counted traffic of the Llama-8B-shaped gate/up launch, if this is that
    workload and the kernel source is unchanged; else None."""
    import hashlib
    if (cfg.name, cfg.d, cfg.ffn) != ("llama8b", 4096, 14336):
        return None
    src = os.path.join(ROOT, "paper_2602_20217_amd", "csrc", "gemm.hip")
    with open(src, "rb") as f:
        digest = hashlib.sha256(f.read()).hexdigest()
    return GATE_UP_TRAFFIC[0] if digest == GATE_UP_TRAFFIC[1] else None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def launch_timer(n):
    """n pairs of timing-enabled HIP events, each recorded once so its handle
    exists, and a call that times what `fn` launches with one pair: the
    library's kernels carry the pair in their own dispatches (ks_time_launches),
    so the elapsed time is the kernels' execution, as a kernel trace reports it."""
    import torch
    from paper_2602_20217_amd import _lib as K
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n)]
    for a, b in ev:
        a.record()
        b.record()

    def timed(k, fn):
        K.ks_time_launches(ev[k][0].cuda_event, ev[k][1].cuda_event)
        try:
            fn()
        finally:
            K.ks_time_launches(None, None)

    def median_ms():
        torch.cuda.synchronize()
        return sorted(a.elapsed_time(b) for a, b in ev)[n // 2]

    return timed, median_ms


def fit_line(n, t):
    """least-squares t = a n + b"""
    import numpy as np
    A = np.stack([np.asarray(n, float), np.ones(len(n))], 1)
    (a, b), *_ = np.linalg.lstsq(A, np.asarray(t, float), rcond=None)
    return float(a), float(b)


def latency_sweep(dm, cfg, ctxs, first_tok, steps=6):
    """Per-sublayer latencies by masked decode steps at several context lengths
    (Appendix C profiling): t_MLP from MLP-only steps, t_Attn(n) from
    attention-only steps, both relative to a step that runs no sublayer."""
    import numpy as np
    L2 = 2 * cfg.L
    none = np.zeros(L2, bool)
    mlp = np.array([i % 2 == 1 for i in range(L2)])
    attn = ~mlp
    rows = []
    for n in ctxs:
        dm.set_context(n, first_tok)
        dm.profile_decode(None, 2, per_kernel=False)  # warm
        t0 = dm.profile_decode(none, steps, per_kernel=False)["ms_step"]
        tm = dm.profile_decode(mlp, steps, per_kernel=False)["ms_step"]
        ta = dm.profile_decode(attn, steps, per_kernel=False)["ms_step"]
        tf = dm.profile_decode(None, steps, per_kernel=False)["ms_step"]
        rows.append({"n": n, "t_attn_ms": (ta - t0) / cfg.L, "t_mlp_ms": (tm - t0) / cfg.L,
                     "t_head_ms": t0, "t_step_ms": tf})
    c2, c3 = fit_line([r["n"] for r in rows], [r["t_attn_ms"] for r in rows])
    c1 = float(np.mean([r["t_mlp_ms"] for r in rows]))
    return (c1, c2, c3), rows


def cpu_baseline(cfg, ctx, budget_s):
    """The oracle (float64 NumPy) timed on the host on a bounded sample: decode
    tokens through 2 of the model's layers at the full context (keys/values
    from the seeded generator) plus the LM head, scaled to all layers."""
    import numpy as np
    import workloads as W
    from oracle import model as M
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    small = dataclasses.replace(cfg, L=2)
    model = M.Model(small, W.generate_weights(small, seed=0))
    cache = M.KVCache(small, ctx + 4160)
    for l in range(2):
        K, V = W.synthetic_kv(small, ctx, seed=3, layer=l)
        cache.K[l][:, :ctx] = K
        cache.V[l][:, :ctx] = V
    tok = int(W.prompt_ids(cfg.vocab, 1, 9)[0])
    x = model.embed[[tok]]
    th = time.perf_counter()
    M.head(model, x)
    t_head = time.perf_counter() - th
    t0 = time.perf_counter()
    n = 0
    while True:
        M.forward(model, cache, [tok], ctx + n)
        n += 1
        if time.perf_counter() - t0 > budget_s or n >= 4096:
            break
    per_tok = (time.perf_counter() - t0) / n
    est = (per_tok - t_head) * cfg.L / 2 + t_head
    return {"value": 1.0 / est, "unit": "tok/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n} float64 oracle decode tokens through 2 of {cfg.L} layers + LM head "
                      f"at {ctx} context (seeded synthetic KV), per-layer time scaled to "
                      f"{cfg.L} layers; {per_tok:.2f} s per sampled token"}


# int32 vector ALU peak: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz, one op per lane per clock
INT32_VALU_OPS = 256 * 4 * 16 * 2.4e9
KNAP_OPS_PER_CELL = 3  # one add, one compare, one select per cell update


def knapsack_leg(steps, warmup):
    """The isolated knapsack batch (1024 instances x 72 items x 4097 budgets,
    Llama-8B-shaped latencies, 4096 bins, skipped weight <= 2048): DP with
    decision bits, then stage 2 (backtrack + TPT grid, D = 10); the median
    launch of each, timed by HIP events carried in the launches."""
    import torch
    import workloads as W
    from paper_2602_20217_amd.engine import (knapsack_quantize, knapsack_batch,
                                             knapsack_batch_select)
    inst = W.knapsack_instances(B=1024, n_items=72, seed=2)
    w, q = knapsack_quantize(inst["t"], inst["s"], 4096)
    C, max_skip, B, n = 4096, 2048, w.shape[0], w.shape[1]
    wd, qd = torch.from_numpy(w).cuda(), torch.from_numpy(q).cuda()
    sd = torch.from_numpy(inst["s"]).cuda()
    for _ in range(warmup):
        best, bits = knapsack_batch(wd, qd, C, max_skip)
        knapsack_batch_select(best, bits, wd, sd, C, 10)
    torch.cuda.synchronize()
    # median launch of each kernel, timed by events its dispatches carry
    reps = 10 * steps
    out = {}
    timed, median_ms = launch_timer(reps)
    for k in range(reps):
        timed(k, lambda: out.update(r=knapsack_batch(wd, qd, C, max_skip)))
    ms_dp = median_ms()
    best, bits = out["r"]
    timed, median_ms = launch_timer(reps)
    for k in range(reps):
        timed(k, lambda: knapsack_batch_select(best, bits, wd, sd, C, 10))
    ms_sel = median_ms()
    # algorithmic work: the budgets a skip set can reach (0..min(C, max_skip));
    # the cells above max_skip are INF by definition and not swept
    live = min(C, max_skip) + 1
    cells = B * n * live
    ops = KNAP_OPS_PER_CELL * cells / (ms_dp * 1e-3)
    return {"workload": f"{B} instances x {n} items x {C + 1} budgets, skipped weight <= {max_skip}",
            "ms_dp": round(ms_dp, 4), "ms_stage2": round(ms_sel, 4),
            "live_budgets": live,
            "cell_updates_per_s": round(cells / (ms_dp * 1e-3), 1),
            "roofline": {"bound": "alu", "kernel": "k_knap_dp", "achieved": round(ops / 1e12, 3),
                         "peak": round(INT32_VALU_OPS / 1e12, 3), "unit": "Tops/s (int32)",
                         "frac": round(ops / INT32_VALU_OPS, 4),
                         "ops_per_cell": KNAP_OPS_PER_CELL}}, (w, q, C, max_skip)


def knapsack_cpu_baseline(w, q, C, max_skip, rows=256):
    """The oracle's vectorised DP timed on the host over the first `rows`
    instances of the same batch."""
    import numpy as np
    from oracle import additive as A
    t0 = time.perf_counter()
    A.knapsack_dp(np.ascontiguousarray(w[:rows]), np.ascontiguousarray(q[:rows]), C, max_skip)
    dt = time.perf_counter() - t0
    cells = rows * w.shape[1] * (min(C, max_skip) + 1)
    return {"value": round(cells / dt, 1), "unit": "cell updates/s",
            "cores": len(os.sched_getaffinity(0)), "kind": "oracle",
            "sample": f"oracle DP over {rows} of {w.shape[0]} instances ({dt:.2f} s)"}


def describe(cfg):
    shape = {"llama8b": "Llama-3-8B-shaped decoder", "qwen8b": "Qwen3-8B-shaped decoder"}
    return (f"{cfg.name}: {shape.get(cfg.name, 'decoder')} (L {cfg.L}, d {cfg.d}, "
            f"{cfg.hq}/{cfg.hkv} heads of {cfg.hd}, ffn {cfg.ffn}, vocab {cfg.vocab})")


def fill_cache(dm, cfg, n, seed=3):
    """Seeded synthetic keys/values (std 1.28, like the random-init model's) at
    positions < n of every layer, generated on the device."""
    import torch
    gen = torch.Generator(device="cuda")
    for l in range(cfg.L):
        gen.manual_seed(seed * 1000 + l)
        kk, vv = dm.kv_layer(l)
        for t in (kk, vv):
            t[:, :n].copy_(torch.randn(cfg.hkv, n, cfg.hd, generator=gen, device="cuda") * 1.28)
    torch.cuda.synchronize()


def history_rounds(dm, cfg, gamma, tok, rounds=5):
    """Full-model draft/verify rounds from the current state: every draft is the
    target's own greedy token, so each round commits gamma + 1 rows of history.
    Returns the committed token and the mean verify time (ms)."""
    import numpy as np
    import torch
    full = np.ones(2 * cfg.L, dtype=bool)
    s = tok
    tv = []
    for _ in range(rounds):
        toks = [s]
        for _ in range(gamma):
            t, _ = dm.draft_step(full)
            toks.append(t)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pred, a = dm.verify(toks)
        tv.append((time.perf_counter() - t0) * 1e3)
        s = int(pred[a])
    return s, sum(tv[1:]) / max(1, len(tv) - 1)


def run_sweep(args, cfg):
    """Context-length x draft-length grid on synthetic caches.  For each context:
    per-sublayer latencies (masked decode steps); the latency model is fitted over
    the whole grid; then for each draft length a knapsack selection, the draft and
    verify rates of the selected mask, and speculative vs autoregressive decode of
    the same tokens from the same state."""
    import numpy as np
    import torch
    import workloads as W
    from paper_2602_20217_amd.engine import DeviceModel, select_params
    ctxs = [int(x) for x in args.sweep_ctx.split(",")]
    gammas = [int(x) for x in args.sweep_gamma.split(",")]
    n_new = args.sweep_new
    # one context per length over the same weights, each with the cache a
    # deployment at that length would allocate
    spare = n_new + 6 * (max(gammas) + 1) + 64
    t = time.time()
    base = DeviceModel(cfg, n_max=min(ctxs) + spare, gamma_max=max(8, max(gammas)), m_rounds=5,
                       cap_max=256, prefill_chunk=512)
    W.generate_weights(cfg, seed=0, consume=base.upload)
    base.finalize()
    models = {n: base if n + spare == base.desc.n_max else base.resized(n + spare) for n in ctxs}
    log(f"weights generated and packed in {time.time() - t:.1f}s (caches of "
        f"{', '.join(str(n + spare) for n in ctxs)} positions)")
    tok = int(W.prompt_ids(cfg.vocab, 1, 1)[0])
    L2 = 2 * cfg.L
    none = np.zeros(L2, bool)
    mlp = np.array([i % 2 == 1 for i in range(L2)])
    lat = []
    for n in ctxs:
        dm = models[n]
        fill_cache(dm, cfg, n)
        dm.set_context(n, tok)
        dm.profile_decode(None, 2, per_kernel=False)
        t0 = dm.profile_decode(none, 6, per_kernel=False)["ms_step"]
        tm = dm.profile_decode(mlp, 6, per_kernel=False)["ms_step"]
        ta = dm.profile_decode(~mlp, 6, per_kernel=False)["ms_step"]
        tf = dm.profile_decode(None, 6, per_kernel=False)["ms_step"]
        lat.append({"n": n, "t_attn_ms": (ta - t0) / cfg.L, "t_mlp_ms": (tm - t0) / cfg.L,
                    "t_head_ms": t0, "t_step_ms": tf})
        log(f"ctx {n}: t_attn {lat[-1]['t_attn_ms'] * 1e3:.1f} us, t_mlp "
            f"{lat[-1]['t_mlp_ms'] * 1e3:.1f} us, AR step {tf:.3f} ms")
    c2, c3 = fit_line([r["n"] for r in lat], [r["t_attn_ms"] for r in lat])
    c1 = float(np.mean([r["t_mlp_ms"] for r in lat]))
    params = select_params((c1, c2, c3), "paper_min", 0, tau=0.5, prune_half=True, D=10)
    points = []
    for n, lr in zip(ctxs, lat):
        dm = models[n]
        fill_cache(dm, cfg, n)
        for gamma in gammas:
            # AR and speculative decode from the same state (same history rounds)
            dm.set_context(n, tok)
            s, _ = history_rounds(dm, cfg, gamma, tok)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            out_ar, _, _ = dm.decode(n_new, 0)
            torch.cuda.synchronize()
            ar_ms = (time.perf_counter() - t0) * 1e3
            # one selection per point, at the start (its cost grows with the
            # context: reported apart as well)
            dm.set_context(n, tok)
            s, verify_ms = history_rounds(dm, cfg, gamma, tok)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            out_sd, st, sels = dm.decode(n_new, gamma, n_new, params)
            torch.cuda.synchronize()
            sd_ms = (time.perf_counter() - t0) * 1e3
            mask = np.array([bool(sels[0].exec[i]) for i in range(L2)])
            draft_ms = dm.profile_decode(mask, 6, per_kernel=False)["ms_step"]
            pt = {"ctx": n, "gamma": gamma, "t_attn_us": round(lr["t_attn_ms"] * 1e3, 2),
                  "t_mlp_us": round(lr["t_mlp_ms"] * 1e3, 2),
                  "draft_ms": round(draft_ms, 4), "draft_tok_s": round(1e3 / draft_ms, 1),
                  "verify_ms": round(verify_ms, 4),
                  "verify_tok_s": round((gamma + 1) * 1e3 / verify_ms, 1),
                  "skipped_attn": int(sum(1 for i in range(0, L2, 2) if not mask[i])),
                  "skipped_mlp": int(sum(1 for i in range(1, L2, 2) if not mask[i])),
                  "ar_tok_s": round((n_new - 1) * 1e3 / ar_ms, 2),
                  "spec_tok_s": round((n_new - 1) * 1e3 / sd_ms, 2),
                  "speedup": round(ar_ms / sd_ms, 4),
                  "speedup_excl_select": round(ar_ms / max(1e-9, sd_ms - st.ms_select), 4),
                  "select_ms": round(st.ms_select, 1),
                  "selections": st.n_selections,
                  "alpha": round(st.n_accepted / max(1, st.n_drafted), 4),
                  "tokens_equal_ar": bool(np.array_equal(out_ar, out_sd))}
            points.append(pt)
            log(json.dumps(pt))
    res = {"mode": "sweep", "workload": f"{describe(cfg)}, bf16, synthetic caches (seeded, "
                                        f"std 1.28) of each context length, {n_new} new tokens "
                                        f"per point after 5 full-model draft/verify rounds of "
                                        f"history, one knapsack selection per point",
           "latency_model_ms": {"c1": c1, "c2": c2, "c3": c3, "points": lat}, "points": points}
    for m in models.values():
        m.close()
    base.close()
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--model", default="llama8b")
    ap.add_argument("--ctx", type=int, default=8192)
    ap.add_argument("--new", type=int, default=256)
    ap.add_argument("--gamma", type=int, default=4)
    ap.add_argument("--reselect", type=int, default=32)
    ap.add_argument("--tau-conf", type=float, default=0.0,
                    help="dynamic drafting exit below this top-1 probability (paper: 0.7; "
                         "0 keeps the fixed draft length of the workload)")
    ap.add_argument("--gamma-source", default="fixed", choices=("fixed", "selected"),
                    help="draft cap per round: --gamma, or min(gamma*, --gamma)")
    ap.add_argument("--sample", default="",
                    help="T,top_k,top_p[,seed]: speculative sampling (paper's sampling "
                         "setting: 0.7,50,0.95) instead of greedy decoding")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--no-knapsack", action="store_true",
                    help="skip the isolated knapsack batch leg")
    ap.add_argument("--knapsack-only", action="store_true",
                    help="only the isolated knapsack batch leg (for traces of its kernels)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-32k", action="store_true",
                    help="skip the 32K leg (Qwen3-8B shape, 32768-token prompt, gamma 6)")
    ap.add_argument("--include-head", action="store_true",
                    help="add the measured LM head time to the TPT cost of the selection "
                         "(the paper's cost leaves it out; off by default)")
    ap.add_argument("--calibrate-stream", action="store_true",
                    help="only the streaming-read reference at the decode launch sizes")
    ap.add_argument("--profile-kernels", action="store_true",
                    help="short run for hardware counters: prefill, 16 decode steps and a "
                         "256 MiB device copy (the reference for counter scaling)")
    ap.add_argument("--profile-select", action="store_true",
                    help="isolated knapsack selections (model-mode DP) at the workload's "
                         "shape after a prefill, for traces and counters of the DP")
    ap.add_argument("--select-coeffs", default="",
                    help="c1,c2,c3 (ms) for --profile-select instead of the fitted ones "
                         "(a profiler's own overhead distorts the fit)")
    ap.add_argument("--sweep", action="store_true",
                    help="context x draft-length grid (synthetic caches): per-sublayer "
                         "latencies, draft/verify rates and speedup over AR at each point")
    ap.add_argument("--sweep-ctx", default="1024,4096,16384,65536,131072")
    ap.add_argument("--sweep-gamma", default="2,4,8")
    ap.add_argument("--sweep-new", type=int, default=64)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import workloads as W
    from paper_2602_20217_amd.engine import DeviceModel, select_params

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    cfg = W.config(args.model)
    if args.knapsack_only:
        leg, _ = knapsack_leg(args.steps, args.warmup)
        print(json.dumps({"mode": "knapsack-only", **leg}), flush=True)
        return
    if args.calibrate_stream:
        q, kv = cfg.hq * cfg.hd, cfg.hkv * cfg.hd
        sizes = {"gemm_o": cfg.d * q * 2, "attn": args.ctx * kv * 2 * 2,
                 "gemm_qkv": (q + 2 * kv) * cfg.d * 2, "gemm_down": cfg.d * cfg.ffn * 2,
                 "gemm_gate_up": 2 * cfg.ffn * cfg.d * 2, "gemm_head": cfg.vocab * cfg.d * 2}
        print(json.dumps({"mode": "calibrate-stream", "model": cfg.name, "ctx": args.ctx,
                          "bytes": sizes, "GBps": stream_ceiling(sizes)}), flush=True)
        return
    if args.sweep:
        return run_sweep(args, cfg)
    n_max = args.ctx + args.new + 64
    t = time.time()
    # the selection profile keeps exactly the m (gamma + 1) history rows a
    # generation's selections use
    gmax = args.gamma if args.profile_select else max(8, args.gamma)
    dm = DeviceModel(cfg, n_max=n_max, gamma_max=gmax, m_rounds=5, cap_max=256,
                     prefill_chunk=512)
    W.generate_weights(cfg, seed=0, consume=dm.upload)
    dm.finalize()
    dm.set_draft_policy(args.tau_conf, args.gamma_source)
    sampling = None
    if args.sample:
        f = args.sample.split(",")
        sampling = {"temperature": float(f[0]), "top_k": int(f[1]), "top_p": float(f[2]),
                    "seed": int(f[3]) if len(f) > 3 else 0}
        dm.set_sampling(**sampling)
    log(f"weights generated and packed in {time.time() - t:.1f}s")
    prompt = W.prompt_ids(cfg.vocab, args.ctx, 1)

    t = time.time()
    first = dm.prefill(prompt)
    torch.cuda.synchronize()
    log(f"prefill {args.ctx} tokens: {time.time() - t:.2f}s")
    if args.profile_kernels:
        # reference of known size for counter scaling: an elementwise product that
        # reads and writes 256 MiB (its own kernel name in the counter output)
        copy_bytes = 256 << 20
        src = torch.empty(copy_bytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        prof = dm.profile_decode(None, 16, per_kernel=False)
        print(json.dumps({"mode": "profile-kernels", "copy_bytes": copy_bytes,
                          "decode_steps": 16, "ms_step": prof["ms_step"]}), flush=True)
        dm.close()
        return
    sweep_ctx = sorted({max(64, args.ctx // 8), args.ctx // 4, args.ctx // 2, args.ctx})
    coeffs, sweep = latency_sweep(dm, cfg, sweep_ctx, first)
    log(f"latency model c1={coeffs[0]:.4f}ms c2={coeffs[1]:.3e}ms/token c3={coeffs[2]:.4f}ms")
    if args.profile_select:
        # isolated selections on the prompt's history rows (the workload's first
        # selection), for per-kernel traces and counters of the DP
        if args.select_coeffs:
            coeffs = tuple(float(x) for x in args.select_coeffs.split(","))
        params = select_params(coeffs, "paper_min", 0, tau=0.5, prune_half=True, D=10)
        dm.prefill(prompt)
        log("prefill for the selections done")
        times = []
        for k in range(args.warmup + args.steps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            sel = dm.select(params)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3
            log(f"selection {k}: {ms:.1f} ms")
            if k >= args.warmup:
                times.append(round(ms, 2))
        print(json.dumps({"mode": "profile-select", "C": sel.C, "w_attn": sel.w_attn,
                          "w_mlp": sel.w_mlp, "cells": sel.n_cells, "rows": sel.n_rows,
                          "j": sel.j_star, "select_ms": times}), flush=True)
        dm.close()
        return
    t_head = coeffs_head(sweep) if args.include_head else 0.0
    params = select_params(coeffs, "paper_min", 0, tau=0.5, prune_half=True, D=10,
                           t_head=t_head)
    core = measure_decode(dm, cfg, prompt, args.ctx, args.new, args.gamma, args.reselect,
                          args.steps, args.warmup, params, sampling is not None)
    ceiling = stream_ceiling({n: b for n, b in core.pop("_launch_bytes").items()})
    for name, e in core["kernels"].items():
        if "GBps" in e:
            e["frac_peak"] = round(e["GBps"] / HBM_PEAK_GBPS, 4)
            if name in ceiling:
                e["stream_ceiling_GBps"] = ceiling[name]
                e["frac_ceiling"] = round(e["GBps"] / ceiling[name], 4)
    timed_tokens = args.new - 1
    res = {
        "metric": "decode tok/s (bs=1) at 8K ctx, speedup vs AR; achieved HBM GB/s",
        "value": core["value"], "unit": "tok/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": core["ms_per_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, random-id prompt)",
        "config": {"workload": f"{describe(cfg)}, bf16 weights and KV, "
                               f"{args.ctx}-token random prompt, {args.new} new tokens, "
                               f"gamma {args.gamma}, mask re-selected every {args.reselect} tokens",
                   "global_batch": 1, "seq_len": args.ctx, "new_tokens": args.new,
                   "timed_tokens": timed_tokens,
                   "gamma": args.gamma, "reselect_every": args.reselect, "parallelism": "none",
                   "draft_policy": {"tau_conf": args.tau_conf,
                                    "gamma_source": args.gamma_source},
                   "tpt_cost": ({"lm_head_ms": round(t_head, 5)} if t_head > 0
                                else "paper (LM head excluded)"),
                   "decoding": ({"mode": "speculative sampling", **sampling} if sampling
                                else {"mode": "greedy"})},
    }
    res.update({k: v for k, v in core.items() if k not in ("value", "ms_per_step")})
    res["latency_model_ms"] = {"c1": coeffs[0], "c2": coeffs[1], "c3": coeffs[2], "sweep": sweep}
    res["stream_ceiling_GBps"] = ceiling
    gu = core["kernels"]["gemm_gate_up"]
    res["roofline"] = {"bound": "hbm",
                       "kernel": "k_gemm_skinny, SwiGLU epilogue (gate/up product, 1 row)",
                       "achieved": gu["GBps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                       "frac": gu["frac_peak"], "traffic": gate_up_traffic(cfg),
                       "bytes_per_launch": gu["bytes_per_launch"], "ms_per_launch": gu["ms"],
                       "stream_ceiling": ceiling.get("gemm_gate_up"),
                       "frac_of_stream_ceiling": gu.get("frac_ceiling")}
    dm.close()
    del dm
    torch.cuda.empty_cache()
    if not args.no_32k and args.model == "llama8b" and not sampling:
        res["qwen32k"] = leg_32k(args)
    knap_in = None
    if not args.no_knapsack:
        res["knapsack_batch"], knap_in = knapsack_leg(max(args.steps, 5), max(args.warmup, 1))
        log(f"knapsack batch: DP {res['knapsack_batch']['ms_dp']:.3f} ms, "
            f"stage 2 {res['knapsack_batch']['ms_stage2']:.3f} ms")
    if not args.no_cpu_baseline:
        t = time.time()
        res["cpu_baseline"] = cpu_baseline(cfg, args.ctx, args.cpu_budget)
        if knap_in is not None:
            res["knapsack_batch"]["cpu_baseline"] = knapsack_cpu_baseline(*knap_in)
        log(f"cpu baseline {time.time() - t:.1f}s")
    print(json.dumps(res), flush=True)


HBM_PEAK_GBPS = 8000.0


def coeffs_head(sweep):
    """LM head + embedding + argmax time of one decode step (the sweep's step
    that runs no sublayer), averaged over the sweep's contexts (ms)."""
    return float(sum(r["t_head_ms"] for r in sweep) / len(sweep))


def stream_ceiling(sizes, pool_bytes=2 << 30, reps=40):
    """Rate (GB/s) of ks_stream_read, a plain streaming read, over buffers of each
    size, timed like the decode kernels by HIP events carried in each launch
    (median launch); the buffers rotate through a pool larger than the 256 MiB
    last-level cache so no launch finds its bytes cached."""
    import torch
    from paper_2602_20217_amd import _lib as K
    pool = torch.empty(pool_bytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    st = torch.cuda.current_stream()
    # the whole pool streamed a few times first, so the first size timed does
    # not pay for clocks and page tables settling; a size is timed once (equal
    # byte counts share the rate) by the median launch
    for k in range(4):
        K.ks_stream_read(pool.data_ptr(), pool_bytes, sink.data_ptr(), st.cuda_stream)
    out, by_size = {}, {}
    for name, nb in sizes.items():
        nb = (int(nb) + 15) // 16 * 16
        if nb > pool_bytes:
            continue
        if nb not in by_size:
            nrot = max(1, pool_bytes // nb)
            timed, median_ms = launch_timer(reps)
            for k in range(5):
                K.ks_stream_read(pool.data_ptr() + (k % nrot) * nb, nb, sink.data_ptr(),
                                 st.cuda_stream)
            for k in range(reps):
                src = pool.data_ptr() + ((k + 5) % nrot) * nb
                timed(k, lambda: K.ks_stream_read(src, nb, sink.data_ptr(), st.cuda_stream))
            ms = median_ms()
            by_size[nb] = round(nb / (ms * 1e-3) / 1e9, 1)
        out[name] = by_size[nb]
    del pool
    return out


def measure_decode(dm, cfg, prompt, ctx, new, gamma, reselect, steps, warmup, params, sampled):
    """Timed AR and speculative generation of `new` tokens after a prefill of
    the prompt (untimed), `warmup` + `steps` times; then per-kernel HIP-event
    timings of 16 decode steps.  Returns the measured quantities."""
    import numpy as np
    import torch

    def run(g):
        dm.prefill(prompt)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        out, st, sels = dm.decode(new, g, reselect, params if g else None)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3, out, st, sels

    ar_ms, ssd_ms, ssd_last, ar_out = [], [], None, None
    for k in range(warmup + steps):
        a_ms, ar_out, _, _ = run(0)
        s_ms, out, st, sels = run(gamma)
        if k >= warmup:
            ar_ms.append(a_ms)
            ssd_ms.append(s_ms)
        ssd_last = (out, st, sels)
        log(f"{cfg.name} step {k}: AR {a_ms:.1f} ms, speculative {s_ms:.1f} ms "
            f"(select {st.ms_select:.1f} ms, accepted {st.n_accepted}/{st.n_drafted})")
    out, st, sels = ssd_last
    same = None if sampled else bool(np.array_equal(out, ar_out))

    dm.set_context(ctx, int(prompt[-1]))
    prof = dm.profile_decode(None, 16, per_kernel=True)
    q, kv = cfg.hq * cfg.hd, cfg.hkv * cfg.hd
    kv_bytes = ctx * kv * 2 * 2  # per layer, K and V, at the profiled context
    launch_bytes = {
        "gemm_qkv": (q + 2 * kv) * cfg.d * 2, "gemm_o": cfg.d * q * 2,
        "gemm_gate_up": 2 * cfg.ffn * cfg.d * 2 + cfg.d * 2 * 2 + cfg.ffn * 2 * 2,
        "gemm_down": cfg.d * cfg.ffn * 2, "gemm_head": cfg.vocab * cfg.d * 2, "attn": kv_bytes}
    kern = {}
    for name, ms in prof["ms"].items():
        if prof["launches"][name] == 0:
            continue
        e = {"ms": round(ms, 5), "launches_per_token": prof["launches"][name]}
        if name in launch_bytes:
            e["bytes_per_launch"] = launch_bytes[name]
            e["GBps"] = round(launch_bytes[name] / (ms * 1e-3) / 1e9, 1)
        kern[name] = e
    if "combine" in kern:
        kern["attn"]["GBps_with_combine"] = round(
            kv_bytes / ((prof["ms"]["attn"] + prof["ms"]["combine"]) * 1e-3) / 1e9, 1)

    timed = new - 1  # decode(n) returns n tokens; the prefill produced the first
    mean_ssd, mean_ar = sum(ssd_ms) / len(ssd_ms), sum(ar_ms) / len(ar_ms)
    value, ar_tps = timed / (mean_ssd / 1e3), timed / (mean_ar / 1e3)
    token_bytes = (cfg.vocab * cfg.d * 2 + cfg.L * ((q + 2 * kv + q) * cfg.d * 2
                   + 3 * cfg.ffn * cfg.d * 2) + cfg.L * (ctx + new // 2) * kv * 2 * 2)
    pvr = []
    for s in sels:
        e_tok = sum(s.alpha_hat ** i for i in range(gamma + 1))
        hd = params.t_head / s.delta
        cost = gamma * (s.C - s.j_star + hd) + (s.C + hd)  # units of Delta (ms / Delta)
        pvr.append({"j": s.j_star, "alpha_hat": round(s.alpha_hat, 4),
                    "predicted_tok_per_ms": round(e_tok / cost / s.delta, 4),
                    "predicted_tok_per_ms_gamma_star": round(s.tpt_star / s.delta, 4),
                    "realized_tok_per_ms": (round(s.iv_tokens / s.iv_ms, 4) if s.iv_ms > 0
                                            else None),
                    "predicted_tokens_per_round": round(e_tok, 3),
                    "realized_tokens_per_round": (round(s.iv_tokens / s.iv_rounds, 3)
                                                  if s.iv_rounds else None),
                    "realized_accept_rate": (round(s.iv_accepted / s.iv_drafted, 4)
                                             if s.iv_drafted else None),
                    "rounds": s.iv_rounds, "tokens": s.iv_tokens, "ms": round(s.iv_ms, 3)})
    return {
        "value": round(value, 2), "ms_per_step": round(mean_ssd, 2),
        "speedup_vs_ar": round(value / ar_tps, 4), "ar_tok_s": round(ar_tps, 2),
        "ar_ms_per_step": round(mean_ar, 2), "tokens_equal_ar": same,
        "accepted": st.n_accepted, "drafted": st.n_drafted, "rounds": st.n_rounds,
        "alpha": round(st.n_accepted / max(1, st.n_drafted), 4),
        "tokens_per_round": round((st.n_accepted + st.n_rounds) / max(1, st.n_rounds), 3),
        "select_ms": round(st.ms_select, 2), "selections": st.n_selections,
        "select_overhead_pct": round(100.0 * st.ms_select / max(1e-9, ssd_ms[-1]), 2),
        "masks": [{"j": s.j_star, "C": s.C, "w_attn": s.w_attn, "w_mlp": s.w_mlp,
                   "skipped_attn": int(sum(1 for i in range(0, 2 * cfg.L, 2) if not s.exec[i])),
                   "skipped_mlp": int(sum(1 for i in range(1, 2 * cfg.L, 2) if not s.exec[i])),
                   "alpha_hat": round(s.alpha_hat, 3), "gamma_star": s.gamma_star} for s in sels],
        "predicted_vs_realized": pvr,
        "ar_step_GBps": round(token_bytes / (mean_ar / timed * 1e-3) / 1e9, 1),
        "kernels": kern, "_launch_bytes": launch_bytes,
    }


def leg_32k(args):
    """The 32K workload: Qwen3-8B-shaped decoder (36 layers, per-head q/k norms,
    vocab 151936), bf16, 32768-token random prompt, 512 new tokens, gamma 6,
    re-selection every 32; min(steps, 3) timed steps after one warm-up (the
    leg's own count, to keep the run short).  Its attention runs the streaming
    decode kernel; that kernel's roofline is reported."""
    import torch
    import workloads as W
    from paper_2602_20217_amd.engine import DeviceModel, select_params
    cfg = W.config("qwen8b")
    ctx, new, gamma, reselect = 32768, 512, 6, 32
    t = time.time()
    dm = DeviceModel(cfg, n_max=ctx + new + 64, gamma_max=8, m_rounds=5, cap_max=256,
                     prefill_chunk=512)
    W.generate_weights(cfg, seed=0, consume=dm.upload)
    dm.finalize()
    log(f"qwen8b weights generated and packed in {time.time() - t:.1f}s")
    prompt = W.prompt_ids(cfg.vocab, ctx, 1)
    t = time.time()
    first = dm.prefill(prompt)
    torch.cuda.synchronize()
    ms_prefill = (time.time() - t) * 1e3
    coeffs, sweep = latency_sweep(dm, cfg, [4096, 8192, 16384, 32768], first)
    params = select_params(coeffs, "paper_min", 0, tau=0.5, prune_half=True, D=10)
    steps = max(1, min(args.steps, 3))
    core = measure_decode(dm, cfg, prompt, ctx, new, gamma, reselect, steps, 1, params, False)
    launch_bytes = core.pop("_launch_bytes")
    ceiling = stream_ceiling({"attn": launch_bytes["attn"], "gemm_gate_up":
                              launch_bytes["gemm_gate_up"]})
    at = core["kernels"]["attn"]
    at["frac_peak"] = round(at["GBps"] / HBM_PEAK_GBPS, 4)
    at["stream_ceiling_GBps"] = ceiling["attn"]
    at["frac_ceiling"] = round(at["GBps"] / ceiling["attn"], 4)
    dm.close()
    torch.cuda.empty_cache()
    out = {"workload": f"{describe(cfg)}, bf16 weights and KV, {ctx}-token random prompt, "
                       f"{new} new tokens, gamma {gamma}, mask re-selected every {reselect} "
                       f"tokens", "steps": steps, "warmup": 1, "timed_tokens": new - 1,
           "tok_s": core.pop("value"), "ms_per_step": core.pop("ms_per_step"),
           "prefill_ms": round(ms_prefill, 1),
           "latency_model_ms": {"c1": coeffs[0], "c2": coeffs[1], "c3": coeffs[2]}}
    out.update(core)
    out["roofline"] = {"bound": "hbm", "kernel": "k_attn_stream (decode attention, 1 row, "
                       f"{ctx} cached positions x {cfg.hkv} kv heads)",
                       "achieved": at["GBps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                       "frac": at["frac_peak"], "traffic": None,
                       "bytes_per_launch": launch_bytes["attn"], "ms_per_launch": at["ms"],
                       "stream_ceiling": ceiling["attn"],
                       "frac_of_stream_ceiling": at["frac_ceiling"]}
    log(f"qwen8b 32K: {out['tok_s']} tok/s, AR {out['ar_tok_s']} tok/s")
    return out


if __name__ == "__main__":
    main()
