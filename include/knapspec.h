/*
 * knapspec.h - C ABI of the MI355X self-speculative decode step of KnapSpec
 * (Cha, Kim, Han, Yang, Han: "KnapSpec: Self-Speculative Decoding via Adaptive
 * Layer Selection as a Knapsack Problem", arXiv 2602.20217).
 *
 * One library, libknapspec.so, built for gfx950.  Every entry point takes plain
 * host or device pointers and sizes.  The caller owns every buffer (model
 * weights, KV cache, workspace); the library never allocates device memory
 * and never frees caller memory.  The only object the library allocates is the
 * host-side ks_ctx.
 *
 * Conventions
 *  - Errors: every call validates its arguments before it launches anything and
 *    returns a negative ks_status on failure, leaving outputs and the context
 *    state unchanged; ks_last_error() then describes the failure (thread-local
 *    string).  No C++ exception crosses this interface.
 *  - Streams: "stream" arguments are hipStream_t values passed as void*.  Calls
 *    that return host values synchronise that stream; calls on raw device
 *    pointers (ks_hidden_cos, ks_knapsack_*) are asynchronous on the stream.
 *  - A ks_ctx is bound to one stream and is not thread-safe.
 *  - Precision: the residual stream, selection history and DP states are float32;
 *    weights and KV cache are float32 (KS_F32) or bf16 (KS_BF16).
 *  - Sublayer numbering follows Section 2 of the paper: sublayer i in 1..2L,
 *    odd i = attention of layer (i+1)/2, even i = MLP of layer i/2.  Masks are
 *    arrays of 2L bytes, byte i-1 nonzero = sublayer i executed.
 */
#ifndef KNAPSPEC_H
#define KNAPSPEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KS_OK = 0,
  KS_EINVAL = -1,     /* bad argument (null pointer, size out of range, ...) */
  KS_ENOMEM = -2,     /* caller-provided buffer smaller than required */
  KS_ECAPACITY = -3,  /* context length would exceed the KV cache capacity */
  KS_ESTATE = -4,     /* call order violated (e.g. verify before prefill) */
  KS_EHIP = -5        /* a HIP runtime call failed */
} ks_status;

enum { KS_F32 = 0, KS_BF16 = 1 };
enum { KS_QUANT_PAPER_MIN = 0, KS_QUANT_BINS = 1 };
enum { KS_MAX_SUBLAYERS = 256 };

/* Decoder description (Llama / Qwen3 style). */
typedef struct ks_model_desc {
  int L;          /* layers; 2L sublayers */
  int d;          /* model width (multiple of 32) */
  int hq, hkv;    /* query / key-value heads, hq % hkv == 0 */
  int hd;         /* head dim: 64 or 128 */
  int ffn;        /* MLP width (multiple of 32) */
  int vocab;      /* vocabulary (multiple of 16) */
  int n_max;      /* KV cache capacity in positions */
  int qk_norm;    /* 1: per-head RMSNorm of q and k before RoPE (Qwen3) */
  int dtype;      /* KS_F32 or KS_BF16: weights and KV cache */
  float eps;      /* RMSNorm epsilon */
  double rope_theta;
} ks_model_desc;

/* Size limits fixed at creation; they set the workspace size. */
typedef struct ks_limits {
  int gamma_max;      /* longest draft; verify runs gamma+1 rows (<= 15) */
  int m_rounds;       /* history keeps the last m rounds (paper: 5) */
  int cap_max;        /* largest knapsack capacity C accepted by the selection */
  int prefill_chunk;  /* rows per prefill pass (multiple of 16) */
} ks_limits;

/*
 * Model weights: device pointers, caller-owned, valid for the context lifetime.
 * Per-layer entries are host arrays of L device pointers.
 *
 * Matrix layouts.  Every matrix is logically W[N][K] (out x in), y = W x.
 *  - KS_F32: plain row-major float32.
 *  - KS_BF16: the MFMA tile layout written by ks_pack_matrix (see there).
 *  wqkv     [ (hq + 2 hkv) hd ][ d ]  rows: q heads, then k heads, then v heads;
 *           bf16: written by ks_pack_qkv (rotary pairs share a tile)
 *  wo       [ d ][ hq hd ]
 *  w_gate_up: written by ks_pack_gate_up from separate gate and up [ffn][d]
 *  w_down   [ d ][ ffn ]
 *  lm_head  [ vocab ][ d ]
 *  embed    [ vocab ][ d ] plain row-major in the model dtype (not packed)
 *  norm gains: float32 vectors (attn_norm, mlp_norm, final_norm: d; q_norm,
 *  k_norm: hd, only read when qk_norm = 1, may be NULL otherwise).
 */
typedef struct ks_weights {
  const void* embed;
  const void* lm_head;
  const float* final_norm;
  const float* const* attn_norm;
  const void* const* wqkv;
  const void* const* wo;
  const float* const* q_norm;
  const float* const* k_norm;
  const float* const* mlp_norm;
  const void* const* w_gate_up;
  const void* const* w_down;
} ks_weights;

/* Selection parameters (Section 3.4 and Appendix C of the paper). */
typedef struct ks_select_params {
  double c1, c2, c3;  /* latency model: t_MLP = c1, t_Attn(n) = c2 n + c3 */
  int quant_mode;     /* KS_QUANT_PAPER_MIN: Delta = min(t_Attn, t_MLP);
                         KS_QUANT_BINS: Delta = L (t_Attn + t_MLP) / bins */
  int bins;
  float tau;          /* cosine pruning threshold (paper: 0.5); -inf disables */
  int prune_half;     /* 1: skipped weight <= C/2 (paper's second pruning rule) */
  int D;              /* largest draft length in the TPT grid (paper: 10) */
  double t_head;      /* LM head latency in the unit of c1..c3, added to every draft
                         step and to the verify pass in the TPT cost; 0 (the
                         paper's cost, which leaves the head out) or > 0 */
} ks_select_params;

/* Result of one selection. */
typedef struct ks_selection {
  uint8_t exec[KS_MAX_SUBLAYERS]; /* chosen draft mask S* (byte i-1: sublayer i) */
  int j_star;        /* skipped weight of S* */
  int gamma_star;    /* gamma of the best (S, gamma) pair (reported only) */
  int C;             /* capacity L (w_attn + w_mlp) */
  int w_attn, w_mlp; /* integer sublayer weights */
  int n_rows;        /* history rows r used */
  int n_cells;       /* reachable terminal budgets */
  double tpt_star;   /* TPT of (S*, gamma*) in tokens per Delta */
  double alpha_hat;  /* estimated acceptance of S* (Eq. acceptance) */
  double delta;      /* latency unit Delta */
  /* ks_generate / ks_decode: the speculative rounds run with this mask, until
     the next selection or the end of the call (0 elsewhere) */
  int iv_rounds, iv_drafted, iv_accepted;
  int iv_tokens;     /* tokens those rounds emitted */
  double iv_ms;      /* their wall time (selections excluded) */
} ks_selection;

/* Optional per-decision record of a selection (host arrays the caller sizes;
 * J = C/2 with prune_half, else C; rows indexed i = 0..2L). */
typedef struct ks_selection_debug {
  int J_cap;          /* in: entries per row available in the arrays below */
  uint8_t* bits;      /* [(2L+1)][J_cap]  1 = skip candidate chosen */
  uint8_t* reach;     /* [(2L+1)][J_cap]  cell reachable after sublayer i */
  double* sig_e;      /* [(2L+1)][J_cap]  cos of execute candidate (NaN if none) */
  double* sig_s;      /* [(2L+1)][J_cap]  cos of skip candidate (NaN if none) */
  int* n_match;       /* [J_cap]  argmax agreements of terminal cells (-1 if none) */
} ks_selection_debug;

typedef struct ks_gen_stats {
  int n_rounds;        /* speculative rounds (verify passes) */
  int n_selections;    /* knapsack selections run */
  int n_drafted;       /* draft tokens proposed */
  int n_accepted;      /* draft tokens accepted */
  double ms_total;     /* wall time of the generation loop (after prefill) */
  double ms_select;    /* part of ms_total spent in selections */
  double ms_prefill;   /* prefill wall time (outside ms_total) */
} ks_gen_stats;

typedef struct ks_ctx ks_ctx;

/*
 * ks_last_error: the message of the last call on this thread that returned an
 * error (thread-local, library-owned; valid until the next failing call on the
 * same thread).
 */
const char* ks_last_error(void);

/* ---- sizing ------------------------------------------------------------- */
/*
 * ks_kv_cache_bytes: bytes of the KV cache ks_create expects,
 * L * 2 * hkv * n_max * hd elements of the model dtype.  ks_workspace_bytes:
 * bytes of its workspace (activations, split-attention and split-K partials,
 * logits, verify stage, history ring, DP states, sampling tables).  Both
 * return 0 for a description or limits that ks_create would reject.
 */
size_t ks_kv_cache_bytes(const ks_model_desc* desc);
size_t ks_workspace_bytes(const ks_model_desc* desc, const ks_limits* lim);

/* ---- weight layout ------------------------------------------------------ */
/*
 * ks_pack_matrix: converts row-major W[N][K] (src, device) into the layout the
 * kernels read (dst, device, same byte size).  KS_F32: plain copy.  KS_BF16:
 * N % 16 == 0, K % 32 == 0; dst is a sequence of 1 KiB tiles, tile (nt, kt)
 * at element offset (nt * K/32 + kt) * 512, covering rows 16 nt..16 nt+15 and
 * columns 32 kt..32 kt+31; inside a tile, lane l = (n % 16) + 16 ((k % 32) / 8)
 * holds elements k % 8 = 0..7 at offset 8 l.  This is the B-operand register
 * layout of the gfx950 16x16x32 bf16 matrix instruction, so one 64-lane load
 * reads one contiguous KiB.  src and dst must not overlap.
 */
ks_status ks_pack_matrix(const void* src, void* dst, int N, int K, int dtype, void* stream);
/*
 * ks_pack_qkv: the fused q/k/v projection, row-major [(hq + 2 hkv) hd][d]
 * (device): q heads, then k heads, then v heads, hd rows each.  KS_F32: plain
 * copy.  KS_BF16 (hd % 16 == 0, d % 32 == 0): packed like ks_pack_matrix after
 * reordering the rows of every head so that its 16-row tile t holds head rows
 * 8t..8t+7 followed by hd/2 + 8t..hd/2 + 8t + 7, the rotate-half RoPE pairs
 * (f, f + hd/2) of the Llama/Qwen decoders; the product's epilogue then owns
 * both members of each pair.  src and dst must not overlap.
 */
ks_status ks_pack_qkv(const void* src, void* dst, int hq, int hkv, int hd, int d, int dtype,
                      void* stream);
/*
 * ks_pack_gate_up: gate and up projections, each row-major [ffn][d] (device).
 * KS_F32: dst = [gate rows; up rows] row-major [2 ffn][d].  KS_BF16: packed as
 * a [2 ffn][d] matrix whose 16-row tile t holds gate rows 8t..8t+7 followed by
 * up rows 8t..8t+7, so one tile yields 8 SwiGLU outputs.
 */
ks_status ks_pack_gate_up(const void* gate, const void* up, void* dst, int ffn, int d,
                          int dtype, void* stream);

/* ---- context ------------------------------------------------------------ */
/*
 * ks_create: kv_cache is a device buffer of ks_kv_cache_bytes(desc) bytes, laid
 * out [L][2 (K, V)][hkv][n_max][hd] in the model dtype; workspace is a device
 * buffer of ks_workspace_bytes(desc, lim) bytes.  Both stay caller-owned.
 * Fills the rotary table (float64 angles rounded to float32) on the stream.
 */
ks_status ks_create(const ks_model_desc* desc, const ks_limits* lim, const ks_weights* w,
                    void* kv_cache, size_t kv_bytes, void* workspace, size_t ws_bytes,
                    void* stream, ks_ctx** out);
/*
 * ks_destroy: releases what the library allocated for the context (its pinned
 * host staging buffer and timing events); the caller's weights, cache and
 * workspace are untouched.  No work a context call leaves queued uses what it
 * releases (calls that read results back synchronise the stream first;
 * ks_create's rotary-table fill writes the caller's workspace), so it may be
 * called between any two calls; the caller keeps its buffers alive until the
 * stream has finished with them.
 */
ks_status ks_destroy(ks_ctx* ctx);

/*
 * ks_prefill (Section 2; setup step): runs the prompt tokens (host int32[n],
 * 1 <= n < n_max) through the full model, fills the KV cache for positions
 * 0..n-1 and commits the target's greedy (or, after ks_set_sampling, sampled)
 * token s at position n (no keys/values yet).  The last min(n, m_rounds (gamma_max+1)) rows of every sublayer output
 * X^(0..2L) become the first history block.  Resets all decode state.
 */
ks_status ks_prefill(ks_ctx* ctx, const int32_t* tokens, int n, int32_t* out_first_token);

/*
 * ks_set_context: declares that the caller has filled the KV cache for
 * positions 0..n_cached-1 itself and that last_token is the committed token at
 * position n_cached.  Clears the history and the pending draft.
 */
ks_status ks_set_context(ks_ctx* ctx, int n_cached, int32_t last_token);

/*
 * ks_draft_step (Section 2.1, draft model f^(S)): one draft token, the argmax
 * (or, after ks_set_sampling, a draw from the draft's filtered distribution).  The
 * k-th call since the last verify (k = 0, 1, ...) processes, at position P+k,
 * the committed token s (k = 0) or the previous draft token; executed attention
 * sublayers store their keys/values at P+k.  exec: host uint8[2L] mask S.
 * Returns the token and its top-1 probability.  k must stay below gamma_max.
 */
ks_status ks_draft_step(ks_ctx* ctx, const uint8_t* exec, int32_t* out_token,
                        float* out_top1_prob);

/*
 * ks_verify (Section 2.1, greedy verification): runs the full model on tokens
 * (host int32[gamma+1] = s, d_1..d_gamma; tokens[0] must be the committed s) at
 * positions P..P+gamma, overwriting their keys/values, and accepts the longest
 * prefix with d_i equal to the target's argmax y_{i-1}.  Commits d_1..d_a and
 * y_a (a+1 tokens); the new s is y_a at position P+a+1.  The rows 0..a of every
 * sublayer output become a history block (the last m_rounds blocks are kept).
 * out_pred: host int32[gamma+1] target argmaxes; out_n_accepted: a.
 * After ks_set_sampling the pass runs the acceptance chain of speculative
 * sampling instead (see there).
 */
ks_status ks_verify(ks_ctx* ctx, const int32_t* tokens, int gamma, int32_t* out_pred,
                    int* out_n_accepted);

/*
 * ks_hidden_cos (Section 2): out[g] = (1/r) sum_t cos(X[g][t], Y[t]) for
 * g < groups; X device float32 [groups][r][d], Y device float32 [r][d], out
 * device float32 [groups].  A row with zero norm contributes 0.  Row sums are
 * accumulated in float64.  Asynchronous on stream.
 */
ks_status ks_hidden_cos(const float* X, const float* Y, int groups, int r, int d, float* out,
                        void* stream);

/*
 * ks_knapsack_select (Section 3.3-3.5, Algorithms 1 and 2 of Appendix D): on
 * the current history (r rows at positions n-r..n-1) computes integer weights
 * from the latency model at the committed length n, runs the model-mode DP over
 * budgets j = 0..J (J = C/2 with prune_half): cell (i, j) takes the execute
 * candidate f^(i)(g[i-1, j]) unless the skip candidate g[i-1, j - w_i] has a
 * strictly higher cosine with X^(i); candidates with cosine <= tau are dropped;
 * g[i, 0] = X^(i).  Attention of a candidate row at position p reads the target
 * cache below p and the row's own key/value at p.  Stage 2 backtracks every
 * reachable terminal cell, estimates alpha by argmax agreement with X^(2L)
 * (Eq. acceptance) and maximises Eq. TPT over gamma = 1..D (first strict max).
 * dbg may be NULL.
 */
ks_status ks_knapsack_select(ks_ctx* ctx, const ks_select_params* p, ks_selection* out,
                             ks_selection_debug* dbg);

/*
 * ks_generate: greedy self-speculative generation (Sections 2.1 and 3): prefill,
 * a first selection, then rounds of gamma draft steps with the selected mask
 * and one verify, re-selecting at the first round boundary after the number of
 * generated tokens crosses a multiple of reselect_every.  gamma = 0 runs plain
 * greedy autoregressive decoding on the same kernels (p may then be NULL).
 * out_tokens: host int32[n_new] (the first is the prefill's token).
 * sel_log: optional host array of max_sel_log selections (may be NULL).
 */
ks_status ks_generate(ks_ctx* ctx, const int32_t* prompt, int n_prompt, int n_new, int gamma,
                      int reselect_every, const ks_select_params* p, int32_t* out_tokens,
                      ks_gen_stats* stats, ks_selection* sel_log, int max_sel_log);

/*
 * ks_decode: the generation loop of ks_generate without its prefill: continues
 * from the current state (after ks_prefill, or after an earlier ks_decode) and
 * returns n_new tokens, the first being the already committed token s.  With
 * gamma > 0 it selects a mask first (the history must hold at least one block)
 * and re-selects as ks_generate does.  stats->ms_prefill is 0.
 */
ks_status ks_decode(ks_ctx* ctx, int n_new, int gamma, int reselect_every,
                    const ks_select_params* p, int32_t* out_tokens, ks_gen_stats* stats,
                    ks_selection* sel_log, int max_sel_log);

/*
 * Draft policy of the generation loop (ks_generate, ks_decode) of a context
 * (Section 3, TPT maximization, dynamic drafting exit):
 *  tau_conf > 0: a round stops drafting after its first draft token whose
 *    top-1 probability is below tau_conf (paper: 0.7); that token is still
 *    verified.  Each draft step then reads its top-1 probability back (one
 *    stream synchronisation per draft step).  0 keeps every round at its cap.
 *  gamma_source KS_GAMMA_FIXED: rounds draft up to the call's gamma;
 *    KS_GAMMA_SELECTED: up to min(gamma*, gamma) of the selection in force
 *    (gamma* from the stage-2 grid, Section 3).
 * A new context starts with {0, KS_GAMMA_FIXED}: the call's gamma every round.
 * Errors: KS_EINVAL for a null pointer, a negative or non-finite tau_conf or
 * an unknown gamma_source (the policy is then unchanged).
 */
enum { KS_GAMMA_FIXED = 0, KS_GAMMA_SELECTED = 1 };
typedef struct ks_draft_policy {
  float tau_conf;
  int gamma_source;
} ks_draft_policy;
ks_status ks_set_draft_policy(ks_ctx* ctx, const ks_draft_policy* p);

/* ---- speculative sampling ------------------------------------------------ */
/*
 * Sampling mode of verification (Section 2.1 with sampled drafts; the paper's
 * sampling experiments use temperature 0.7, top-k 50, top-p 0.95).
 *
 * Filter of one logits row: keep the top_k largest logits (ties: lower token
 * id first), softmax of logit / temperature over them (float32), keep the
 * shortest prefix in that order whose cumulative probability reaches top_p,
 * renormalise.  A table row holds count entries (ids, probs) in that order;
 * table rows are KS_SAMPLE_KMAX entries apart.  A draw with uniform u takes
 * the first entry whose cumulative probability exceeds u (the last entry if
 * rounding leaves none).  Logits must be finite.
 *
 * Uniforms: u = (w >> 8) * 2^-24, w the first output word of Philox4x32-10
 * (Salmon, Moraes, Dror, Shaw, SC 2011) at counter (pos, purpose, 0, 0) under
 * key (seed & 0xffffffff, seed >> 32).  Purposes: 0 draft draw, 1 acceptance
 * test, 2 target draw (residual, bonus, autoregressive and prefill tokens);
 * pos is the position of the token being produced.
 *
 * Acceptance chain of a round from committed position P with drafts d_1..d_g
 * (d_i at position P+i, drawn from draft table q_i) and target tables
 * p_0..p_g of the verify rows: for i = 1..g, d_i is accepted iff
 * u(P+i, 1) < min(1, p_{i-1}(d_i) / q_i(d_i)); at the first rejection the
 * round emits a token drawn with u(P+i, 2) from max(0, p_{i-1} - q_i) over
 * p_{i-1}'s table, normalised (from p_{i-1} itself if that is zero
 * everywhere); when every draft is accepted it emits a token drawn from p_g
 * with u(P+g+1, 2).  The emitted tokens then follow the target's filtered
 * distribution.
 */
enum { KS_SAMPLE_KMAX = 128 };
typedef struct ks_sampling {
  float temperature;  /* > 0 samples; <= 0 (ks_set_sampling only): greedy */
  int top_k;          /* 1..KS_SAMPLE_KMAX, at most vocab */
  float top_p;        /* (0, 1] */
  uint64_t seed;
} ks_sampling;
/*
 * ks_set_sampling: token choice of the context.  s = NULL or temperature <= 0:
 * greedy (the default of a new context).  Otherwise ks_prefill draws its token
 * from the filter of the last prompt row, ks_draft_step draws draft k from the
 * draft model's filter and keeps its table, ks_verify runs the acceptance chain
 * above (it then needs the gamma drafts of ks_draft_step since the last
 * verify; out_pred holds the accepted drafts, the emitted token and -1 after
 * it), and ks_generate / ks_decode sample every token (gamma = 0: each token
 * from the target's filter).  The knapsack selection is unchanged.  Errors:
 * KS_EINVAL for a non-finite temperature or top_k / top_p out of range.
 */
ks_status ks_set_sampling(ks_ctx* ctx, const ks_sampling* s);
/*
 * ks_sample_workspace_bytes: device workspace of ks_sample_filter for rows rows
 * of vocab logits; 0 if the sizes are unsupported (vocab too large for top_k:
 * about 4096 * min(128, 8192 / top_k) logits at most).
 */
size_t ks_sample_workspace_bytes(int rows, int vocab, int top_k);
/*
 * ks_sample_filter: the filter of rows rows of logits (device float32, row r
 * at logits + r * ld) into tables ids / probs (device [rows][KS_SAMPLE_KMAX])
 * and counts (device int32 [rows]).  top1 (optional, device float32 [rows]):
 * the unfiltered softmax maximum (temperature 1).  tokens (optional, device
 * int32 [rows]): row r drawn with u(pos0 + r, purpose).  Asynchronous.
 */
ks_status ks_sample_filter(const float* logits, int rows, int vocab, int ld, const ks_sampling* s,
                           int pos0, int purpose, int32_t* ids, float* probs, int32_t* counts,
                           float* top1, int32_t* tokens, void* workspace, size_t workspace_bytes,
                           void* stream);
/*
 * ks_sample_filter_noalloc: ks_sample_filter for callers that cannot allocate
 * device memory (code under stream capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments and results, minus the workspace:
 * the chunk statistics and candidates live in a 4 MiB array of the library on
 * each device (calls whose ks_sample_workspace_bytes(rows, vocab, top_k)
 * exceeds 4 MiB fail with KS_ENOMEM and change nothing).  Nothing in the
 * scratch needs to start at any value; every call on a device shares that
 * device's scratch, so calls that overlap in time on one device (other streams,
 * other threads) race and must be serialised by the caller.  Asynchronous.
 */
ks_status ks_sample_filter_noalloc(const float* logits, int rows, int vocab, int ld,
                                   const ks_sampling* s, int pos0, int purpose, int32_t* ids,
                                   float* probs, int32_t* counts, float* top1, int32_t* tokens,
                                   void* stream);
/*
 * ks_spec_accept: the acceptance chain of one round on device tables (p: rows
 * 0..gamma, q: rows 0..gamma-1 for d_1..d_gamma, layout of ks_sample_filter),
 * drafts device int32 [gamma] (d_1..d_gamma), pos0 = P; counts in
 * [1, KS_SAMPLE_KMAX] (others are clamped).  Writes out (device
 * int32 [2]) = {accepted drafts a, emitted token}.  Asynchronous.
 */
ks_status ks_spec_accept(const int32_t* p_ids, const float* p_probs, const int32_t* p_counts,
                         const int32_t* q_ids, const float* q_probs, const int32_t* q_counts,
                         const int32_t* drafts, int gamma, uint64_t seed, int pos0, int32_t* out,
                         void* stream);
/* ks_sample_uniforms: out[i] = u(pos[i], purpose) (device arrays).  Asynchronous. */
ks_status ks_sample_uniforms(uint64_t seed, const int32_t* pos, int n, int purpose, float* out,
                             void* stream);

/* Kernel classes of the decode step, for ks_profile_decode. */
enum {
  KS_KC_EMBED = 0,    /* embedding gather */
  KS_KC_NORM,         /* RMSNorm into matrix activations */
  KS_KC_GEMM_QKV,     /* q/k/v projection */
  KS_KC_QKV_POST,     /* q/k norm, RoPE, key/value store */
  KS_KC_ATTN,         /* split attention over the cache */
  KS_KC_COMBINE,      /* merge of attention splits */
  KS_KC_GEMM_O,       /* output projection + residual */
  KS_KC_GEMM_GATE_UP, /* gate/up projection + SwiGLU */
  KS_KC_GEMM_DOWN,    /* down projection + residual */
  KS_KC_GEMM_HEAD,    /* LM head */
  KS_KC_ARGMAX,       /* vocabulary reduction: argmax + top-1 probability, or the sampling filter */
  KS_KC_OTHER,        /* position fill and small copies */
  KS_KC_COUNT
};
typedef struct ks_kernel_profile {
  double ms[KS_KC_COUNT];   /* mean duration of one launch of the class */
  int launches[KS_KC_COUNT];/* launches of the class per decode step */
  double ms_step;           /* mean wall time of one decode step (events around it) */
  int steps;
} ks_kernel_profile;
/*
 * ks_profile_decode: runs `steps` single-row decode steps with mask exec (NULL =
 * every sublayer) at the committed position P and times them with HIP events
 * on the context stream; with per_kernel = 1 every kernel launch also carries
 * an event pair in its own dispatch, as under ks_time_launches (ms[] and
 * launches[] are filled; otherwise they are 0).  Each
 * step writes the keys/values of position P (as a draft step would) and
 * commits nothing.
 */
ks_status ks_profile_decode(ks_ctx* ctx, const uint8_t* exec, int steps, int per_kernel,
                            ks_kernel_profile* out);
/*
 * ks_time_launches: opens a kernel timing bracket on the calling thread
 * (start_event and stop_event: hipEvent_t handles created by the caller with
 * timing enabled), or closes it (both NULL).  While it is open, every kernel the
 * library launches from this thread carries the events in its own dispatch:
 * the first launch records start_event when that kernel begins, every launch
 * records stop_event when it ends, so the elapsed time between them covers the
 * kernels' execution only (no event packets between launches).  A bracket
 * closed without launches records neither event.  Opening a bracket replaces
 * an open one, and ks_profile_decode with per_kernel = 1 uses the same
 * mechanism and leaves no bracket open.  Both handles must be set or both NULL
 * (KS_EINVAL otherwise).
 */
ks_status ks_time_launches(void* start_event, void* stop_event);

/* ---- lower-level calls (per-sublayer parity and latency profiling) ------- */
/*
 * ks_sublayer_apply: applies sublayer i (1..2L) to R rows of the residual
 * stream x_in (device float32 [R][d]) at positions pos (host int32[R]), writing
 * x_out (device float32 [R][d], may equal x_in).  mode 0: rows store their
 * keys/values at their positions, then row t attends cache positions
 * 0..pos[t] (decode / verify semantics).  mode 1: nothing is stored; row t
 * attends cache positions 0..pos[t]-1 plus its own key/value (selection-DP
 * semantics).  R <= 16 uses the decode kernels, larger R the batched ones.
 */
ks_status ks_sublayer_apply(ks_ctx* ctx, int i, const float* x_in, float* x_out,
                            const int32_t* pos, int R, int mode);
/*
 * ks_head_rows: final RMSNorm + LM head + greedy argmax over R rows of x
 * (device float32 [R][d]).  logits (device float32 [R][vocab]) may be NULL
 * (then a workspace buffer is used); argmax (device int32[R]) and top1 (device
 * float32[R], probability of the argmax token) must be valid.  Lowest index
 * wins ties.
 */
ks_status ks_head_rows(ks_ctx* ctx, const float* x, int R, float* logits, int32_t* argmax,
                       float* top1);

/* ---- isolated integer knapsack (batched) -------------------------------- */
/*
 * ks_knapsack_quantize (host): per instance b, Delta_b = sum_i t[b][i] / bins,
 * w[b][i] = max(1, floor(t[b][i]/Delta_b + 1/2)) (Section 3.4, BINS mode) and the
 * integer loss q[b][i] = floor(-ln(s[b][i]) 2^24 + 1/2) of skipping item i, whose
 * similarity score is s in (0, 1].  All arrays host, [B][n] row-major.
 */
ks_status ks_knapsack_quantize(const double* t, const double* s, int B, int n, int bins,
                               int32_t* w, int32_t* q);
/*
 * ks_knapsack_batch (Eq. objective_knapsack in isolation, parallel over the
 * capacity axis): for every instance b (device arrays w, q int32 [B][n]) and
 * budget j = 0..C, best[b][j] = minimum total loss of a skip set whose weights
 * sum to exactly j (INT32_MAX if none or j > max_skip).  Recurrence over items
 * i = 0..n-1: skip item i at budget j iff j >= w_i and
 * best_{i-1}[j - w_i] + q_i < best_{i-1}[j] (strict; ties keep the item).
 * bits[b][i][j/64] bit j%64 records that decision (uint64 words, C/64 + 1 per
 * item).  Requires C <= 8191, n <= 4096, w and q >= 0 (negative entries are
 * read as 0, by every ks_knapsack_* call) and total loss < 2^31.  Only the
 * budgets 0..min(C, max_skip) are swept; the cells above them read INT32_MAX
 * and their decision words 0.  Asynchronous.
 */
ks_status ks_knapsack_batch(const int32_t* w, const int32_t* q, int B, int n, int C,
                            int max_skip, int32_t* best, uint64_t* bits, void* stream);
/*
 * ks_knapsack_backtrack: skip[b][i] (device uint8 [B][n]) of budget j[b]
 * (device int32 [B]) from the decision bits, following items n-1 down to 0.
 * Writes err[b] = 0, or 1 if the walk does not end at budget 0 or j[b] is out
 * of range (device int32 [B]).  Negative weights are read as 0, as by
 * ks_knapsack_batch.  Asynchronous.
 */
ks_status ks_knapsack_backtrack(const uint64_t* bits, const int32_t* w, int B, int n, int C,
                                const int32_t* j, uint8_t* skip, int32_t* err, void* stream);
/*
 * ks_knapsack_batch_select (stage 2 with the surrogate acceptance
 * alpha_j = prod_{i skipped} s_i, float64, ascending i): for every instance,
 * every reachable budget j and gamma = 1..D, TPT = (sum_{k<=gamma} alpha^k) /
 * (gamma (W - j) + W) with W = sum_i w_i; j ascending, gamma ascending, first
 * strict maximum wins.  Outputs j_star, gamma_star (int32 [B]), tpt (double
 * [B]) and skip (uint8 [B][n]); s is device double [B][n].  Negative weights
 * are read as 0 (also in W), as by ks_knapsack_batch.  Requires 1 <= n <= 128,
 * 0 <= C <= 8191 and 1 <= D <= 64 (KS_EINVAL otherwise).  Asynchronous.
 */
ks_status ks_knapsack_batch_select(const int32_t* best, const uint64_t* bits, const int32_t* w,
                                   const double* s, int B, int n, int C, int D,
                                   int32_t* j_star, int32_t* gamma_star, double* tpt,
                                   uint8_t* skip, void* stream);

/* ---- measurement reference ---------------------------------------------- */
/*
 * ks_stream_read: reads bytes (a multiple of 16; src device memory, 16-byte
 * aligned) once with 16-byte streaming loads and keeps nothing (sink: device
 * float32 [1], written only in a case no timing depends on).  The rate it
 * reaches over a buffer of a decode launch's size is the achievable streaming
 * rate that the HBM-bound kernels are compared against.  Asynchronous.
 */
ks_status ks_stream_read(const void* src, size_t bytes, float* sink, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* KNAPSPEC_H */
