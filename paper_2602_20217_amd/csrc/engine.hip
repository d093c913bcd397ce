// libknapspec engine: context, workspace layout, the forward passes of the
// self-speculative decode step, the knapsack selection and the C ABI.
//
//  decode / draft (1 row) and verify (gamma+1 rows): skinny MFMA products
//      (norm carried in, RoPE + K/V stores, SwiGLU and residual epilogues) and
//      decode attention over context splits whose size depends only on the
//      cache size, so a verify row and the decode step at the same position
//      compute the same bits and greedy speculative output equals greedy AR
//      output.
//  prefill (512-row chunks) and selection DP (budgets x history rows): tiled
//      MFMA products with split-K, batched attention.
//  selection (Sections 3.3-3.5): stage 1 runs on the device one sublayer at a
//      time over the reachable budgets; per-row cosines (float64) of both
//      candidates, the decisions of Eq. dp_main with the tau and C/2 pruning,
//      the decision bits and the compacted list of reachable budgets are all
//      produced by kernels, with no host round trip between stages.  Stage 2
//      (argmax rows of the terminal states on the device; alpha-hat, the TPT
//      grid and the backtrack from the decision bits on the host) follows one
//      synchronisation.
#include "ks_internal.h"

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <limits>

namespace ks {
static thread_local std::string g_err;
void set_error(const std::string& m) { g_err = m; }
thread_local LaunchTiming g_timing;
}  // namespace ks

using namespace ks;

#define REQ(cond, msg)        \
  do {                        \
    if (!(cond)) {            \
      set_error(msg);         \
      return KS_EINVAL;       \
    }                         \
  } while (0)
#define HIPCHK(x)                                                          \
  do {                                                                     \
    hipError_t e_ = (x);                                                   \
    if (e_ != hipSuccess) {                                                \
      set_error(std::string(#x) + ": " + hipGetErrorString(e_));           \
      return KS_EHIP;                                                      \
    }                                                                      \
  } while (0)

namespace {

constexpr int PB = 512;        // rows per batched head pass
// rows per batched attention pass: the selection's whole candidate batch at
// 8K (up to 49 budgets x 25 rows) in one split launch and one merge launch
// (a 1225-row selection 2% faster than passes of 512 rows), fewer when the
// split partials of a pass would exceed PA_PART_BYTES
constexpr int PA_MAX = 1280;
constexpr size_t PA_PART_BYTES = (size_t)1 << 30;
// float32 split-K partials of the batched products (prefill chunks, selection)
constexpr size_t GPART_BYTES = (size_t)128 << 20;
// decode/verify splits: 64-position tiles per split, by the model's cache size
// and kv heads only (never by row count, so a verify row and the decode step
// split alike).  Measured on MI355X (split kernel + merge, 1 and 5 rows): the
// one-tile-per-wave kernel with two tiles for caches up to 2048 positions,
// three up to 5120, five up to 12288 (a 160 KiB workgroup: up to 10240
// positions of 8 kv heads fit the 256 CUs in one round; splits sized to put
// an equal share of the cache on every CU, the last tile partly used, were
// slower); above, the streaming kernel with 4 waves and as many tiles per wave
// (at least 2) as keep the splits of all kv heads to one round of 256
// workgroups.
int dec_tiles(int n_max, int hkv) {
  if (n_max <= 2048) return 2;
  if (n_max <= 5120) return 3;
  if (n_max <= 12288) return 5;
  const int n_tiles = (n_max + 63) / 64;
  const int splits = std::max(1, 256 / hkv);
  const int tpw = (n_tiles + 4 * splits - 1) / (4 * splits);
  return 4 * std::max(2, tpw);
}
int dec_span(const ks_model_desc& d) { return 64 * dec_tiles(d.n_max, d.hkv); }
#ifndef KS_BAT_TILES
#define KS_BAT_TILES 16
#endif
// batched attention (prefill, DP): 64-position tiles per split; 16 (1024
// positions) times the 8K selection as fast as 32 and 6% faster than 64
constexpr int BAT_TILES = KS_BAT_TILES;

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t rope, x, a1hi, a1lo, a2hi, a2lo, qkv, q, kvself, part, logits, am, top1;
  size_t tok, pos, len, stage, hist, xh, g0, g1, ge, dpos, dlen, sig, ptrs, ssq, gpart;
  size_t dpc, dpn, dpmean, dpidx, dpbits, dpreach, dpse, dpss;
  size_t vws, tab_ids, tab_pr, tab_cnt, sres, total;
  int FR, RING, cells, DR, XR, LR, nqkv, a2w, part_rows, PA;
  size_t part_elems;
};

Layout make_layout(const ks_model_desc& d, const ks_limits& lim) {
  Layout y{};
  const int gam1 = lim.gamma_max + 1;
  y.FR = std::max(std::max(lim.prefill_chunk, gam1), 16);
  y.RING = (2 * lim.m_rounds - 1) * gam1;
  y.cells = lim.cap_max + 1;
  y.DR = y.cells * y.RING;
  y.XR = std::max(y.FR, y.DR);
  y.LR = std::max(gam1, PB);
  y.nqkv = (d.hq + 2 * d.hkv) * d.hd;
  y.a2w = std::max(d.hq * d.hd, d.ffn);
  const int ns_dec = (d.n_max + dec_span(d) - 1) / dec_span(d);
  const int ns_bat = attn_nsplit(d.n_max, BAT_TILES);
  const size_t row_part = (size_t)d.hq * ns_bat * (d.hd + 2) * 4;  // bytes per batched row
  y.PA = (int)std::max<size_t>(PB, std::min<size_t>(PA_MAX, PA_PART_BYTES / row_part));
  y.part_rows = y.PA;
  y.part_elems = std::max((size_t)16 * d.hq * ns_dec, (size_t)y.PA * d.hq * ns_bat) * (d.hd + 2);
  const size_t es = d.dtype == KS_BF16 ? 2 : 4;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t r = o;
    o = align_up(o + bytes);
    return r;
  };
  y.rope = take((size_t)d.n_max * (d.hd / 2) * 2 * 4);
  y.x = take((size_t)y.XR * d.d * 4);
  y.a1hi = take((size_t)y.XR * d.d * (es == 4 ? 4 : 2));
  y.a1lo = take((size_t)y.XR * d.d * 2);
  y.a2hi = take((size_t)y.XR * y.a2w * (es == 4 ? 4 : 2));
  y.a2lo = take((size_t)y.XR * y.a2w * 2);
  y.qkv = take((size_t)y.XR * y.nqkv * 4);
  y.q = take((size_t)y.XR * d.hq * d.hd * 4);
  y.kvself = take((size_t)y.XR * 2 * d.hkv * d.hd * 4);
  y.part = take(y.part_elems * 4);
  y.logits = take((size_t)y.LR * d.vocab * 4);
  y.am = take((size_t)(y.XR + y.RING + 64) * 4);
  y.top1 = take((size_t)(y.XR + 64) * 4);
  y.tok = take((size_t)(y.FR + 64) * 4);
  y.pos = take((size_t)y.XR * 4);
  y.len = take((size_t)y.XR * 4);
  y.stage = take((size_t)(2 * d.L + 1) * gam1 * d.d * 4);
  y.hist = take((size_t)(2 * d.L + 1) * y.RING * d.d * 4);
  y.xh = take((size_t)(2 * d.L + 1) * y.RING * d.d * 4);
  y.g0 = take((size_t)y.DR * d.d * 4);
  y.g1 = take((size_t)y.DR * d.d * 4);
  y.ge = take((size_t)y.DR * d.d * 4);
  y.dpos = take((size_t)y.DR * 4);
  y.dlen = take((size_t)y.DR * 4);
  y.sig = take((size_t)2 * y.DR * 8);
  y.ptrs = take((size_t)4 * (y.cells + 2 * d.L + 2) * 8);
  y.ssq = take((size_t)16 * (d.d / 16) * 4);
  y.gpart = take(GPART_BYTES);
  // model-mode DP state on the device: two cell lists + counts, cell means,
  // budget index, and per-(stage, budget) bits / reach / cosines
  y.dpc = take((size_t)2 * y.cells * 4);
  y.dpn = take(64);
  y.dpmean = take((size_t)2 * y.cells * 8);
  y.dpidx = take((size_t)y.cells * 4);
  y.dpbits = take((size_t)(2 * d.L + 1) * y.cells);
  y.dpreach = take((size_t)(2 * d.L + 1) * y.cells);
  y.dpse = take((size_t)(2 * d.L + 1) * y.cells * 8);
  y.dpss = take((size_t)(2 * d.L + 1) * y.cells * 8);
  // vocabulary reductions: chunk partials / candidates, and the sampling tables
  // (rows 0..gamma_max: target rows of a verify; rows gamma_max+1..: drafts)
  y.vws = take(std::max(argmax_ws_bytes(y.LR, d.vocab), sample_ws_bytes_max(gam1)));
  y.tab_ids = take((size_t)2 * gam1 * KS_SAMPLE_KMAX * 4);
  y.tab_pr = take((size_t)2 * gam1 * KS_SAMPLE_KMAX * 4);
  y.tab_cnt = take((size_t)2 * gam1 * 4);
  y.sres = take(64);
  y.total = o;
  return y;
}

}  // namespace

struct ks_ctx {
  ks_model_desc md;
  ks_limits lim;
  hipStream_t st;
  const void* embed;
  const void* lm_head;
  const float* final_norm;
  std::vector<const void*> wqkv, wo, wgu, wdown;
  std::vector<const float*> attn_norm, mlp_norm, q_norm, k_norm;
  char* kv;
  char* ws;
  Layout y;
  int32_t* pin = nullptr;  // pinned host staging: [0,16) draft tokens, [16,32) verify argmax
  // kernel timing (ks_profile_decode): event pairs around launches
  bool prof_on = false;
  std::vector<hipEvent_t> prof_ev;
  std::vector<std::pair<int, int>> prof_rec;  // (kernel class, first event)
  // decode state
  bool ready = false;
  int P = 0;
  int32_t s = 0;
  int k_draft = 0;
  std::deque<std::pair<int, int>> blocks;  // (first position, rows)
  float tau_conf = 0.f;                    // draft policy (ks_set_draft_policy)
  int gamma_source = KS_GAMMA_FIXED;
  ks_sampling samp{};                      // temperature <= 0: greedy

  template <typename T>
  T* at(size_t off) const { return (T*)(ws + off); }
  bool bf() const { return md.dtype == KS_BF16; }
  size_t es() const { return bf() ? 2 : 4; }
  void* kc(int l) const {
    return kv + (size_t)l * 2 * md.hkv * md.n_max * md.hd * es();
  }
  void* vc(int l) const {
    return kv + ((size_t)l * 2 + 1) * md.hkv * md.n_max * md.hd * es();
  }
  Act act1() const { return Act{ws + y.a1hi, ws + y.a1lo, md.d}; }
  Act act2() const { return Act{ws + y.a2hi, ws + y.a2lo, y.a2w}; }
  float* hist_row(int i, int slot) const {
    return at<float>(y.hist) + ((size_t)i * y.RING + slot) * md.d;
  }
  float* stage_row(int i, int k) const {
    return at<float>(y.stage) + ((size_t)i * (lim.gamma_max + 1) + k) * md.d;
  }
  bool sampling() const { return samp.temperature > 0.f; }
  // sampling tables: row t of the target (verify) set, row gamma_max + 1 + t of
  // the draft set
  int32_t* tab_ids(int row) const { return at<int32_t>(y.tab_ids) + (size_t)row * KS_SAMPLE_KMAX; }
  float* tab_pr(int row) const { return at<float>(y.tab_pr) + (size_t)row * KS_SAMPLE_KMAX; }
  int32_t* tab_cnt(int row) const { return at<int32_t>(y.tab_cnt) + row; }
  int qrow(int k) const { return lim.gamma_max + 1 + k; }
  // filter of `row` (tables at table row trow), optional draw at position pos
  SampleSpec spec(int trow, float* top1, int32_t* tok, int pos, int purpose) const {
    return SampleSpec{samp.temperature, samp.top_k, samp.top_p, samp.seed, tab_ids(trow),
                      tab_pr(trow), tab_cnt(trow), top1, tok, pos, purpose};
  }
};

namespace {

// ---------------------------------------------------------- kernel timing
// A class's launches carry their events themselves (a timing bracket around
// the statement); a statement that launched nothing records both events where
// it ends, for a duration of about zero.
int prof_begin(ks_ctx* c, int cls) {
  if (!c->prof_on) return -1;
  const int i = 2 * (int)c->prof_rec.size();
  if (i + 2 > (int)c->prof_ev.size()) return -1;
  g_timing = LaunchTiming{c->prof_ev[i], c->prof_ev[i + 1], 0};
  c->prof_rec.push_back({cls, i});
  return i;
}
void prof_end(ks_ctx* c, int i) {
  if (i < 0) return;
  if (g_timing.launches == 0) {
    (void)hipEventRecord(c->prof_ev[i], c->st);
    (void)hipEventRecord(c->prof_ev[i + 1], c->st);
  }
  g_timing = LaunchTiming{};
}
#define PROF(c, cls, stmt)              \
  do {                                  \
    const int pi_ = prof_begin(c, cls); \
    stmt;                               \
    prof_end(c, pi_);                   \
  } while (0)

// ---------------------------------------------------------- forward pieces
// bf16 row products of at most 16 rows (decode, draft, verify) run the skinny
// kernels.  Their normed inputs arrive as planes x * gain in act1 plus per-tile
// sums of squares in the ssq buffer, written by whichever kernel produced x
// (the embedding, a residual epilogue, or act_prep for rows handed in).
bool skinny(const ks_ctx* c, int M, bool batched) { return c->bf() && !batched && M <= 16; }

void run_gemm(ks_ctx* c, GemmArgs& g, bool batched) {
  if (!c->bf()) {
    gemm_f32(g, c->st);
  } else if (skinny(c, g.M, batched)) {
    gemm_bf16_skinny(g, c->st);
  } else {
    g.part = c->at<float>(c->y.gpart);
    g.part_bytes = GPART_BYTES;
    gemm_bf16_tiled(g, c->st);
  }
}

void gemm(ks_ctx* c, int M, int N, int K, Act A, const void* W, int epi, float* out, int ldo,
          const float* res, int ldres, Act aout, bool batched) {
  GemmArgs g{M, N, K, A, W, epi, out, ldo, res, ldres, aout};
  run_gemm(c, g, batched);
}

// norm gain feeding sublayer i (1..2L); i = 2L + 1 is the final norm
const float* gain_of(const ks_ctx* c, int i) {
  if (i > 2 * c->md.L) return c->final_norm;
  const int l = (i - 1) / 2;
  return i % 2 == 1 ? c->attn_norm[l] : c->mlp_norm[l];
}

// planes and tile sums of rmsnorm input x (R rows) for a skinny normed product
void prep_rows(ks_ctx* c, const float* x, int R, const float* gain) {
  PROF(c, KS_KC_NORM,
       act_prep(x, c->md.d, nullptr, c->md.dtype, nullptr, R, c->md.d, nullptr, gain, c->act1(),
                c->at<float>(c->y.ssq), c->st));
}

// skinny normed product over the planes in act1
GemmArgs normed(ks_ctx* c, int M, int N, const void* W, int epi, float* out, int ldo, Act aout) {
  const ks_model_desc& d = c->md;
  GemmArgs g{M, N, d.d, c->act1(), W, epi, out, ldo, nullptr, 0, aout};
  g.ssq_in = c->at<float>(c->y.ssq);
  g.nssq = d.d / 16;
  g.eps = d.eps;
  return g;
}

// residual product; on the skinny path with next_gain it also writes the
// planes and tile sums of its output for the next normed product
void resid_gemm(ks_ctx* c, int R, int K, Act A, const void* W, float* xout, const float* xin,
                bool batched, const float* next_gain) {
  const ks_model_desc& d = c->md;
  GemmArgs g{R, d.d, K, A, W, EPI_RESID, xout, d.d, xin, d.d, Act{}};
  if (skinny(c, R, batched) && next_gain) {
    g.next_gain = next_gain;
    g.next_act = c->act1();
    g.next_ssq = c->at<float>(c->y.ssq);
  }
  run_gemm(c, g, batched);
}

// Attention sublayer of layer l on R rows: x_out = x_in + Wo attn(...).
// mode 0: keys/values stored at pos; mode 1: own key/value (selection DP).
void attn_rows(ks_ctx* c, int l, const float* xin, float* xout, int R, const int32_t* pos,
               const int32_t* len, int max_len, int mode, bool batched, const float* next_gain) {
  const ks_model_desc& d = c->md;
  const Act a1 = c->act1(), a2 = c->act2();
  float* qkv = c->at<float>(c->y.qkv);
  float* q = c->at<float>(c->y.q);
  float* kvs = c->at<float>(c->y.kvself);
  const float* rope = c->at<float>(c->y.rope);
  if (skinny(c, R, batched)) {
    // without q/k norms and for cache writes, RoPE and the key/value stores
    // are the product's epilogue
    const bool fused = mode == 0 && !d.qk_norm;
    GemmArgs g = normed(c, R, c->y.nqkv, c->wqkv[l], fused ? EPI_QKV : EPI_STORE, qkv,
                        c->y.nqkv, Act{});
    if (fused)
      g.qe = QkvEpi{d.hq, d.hkv, d.hd, d.n_max, rope, pos, q, (bf16_t*)c->kc(l),
                    (bf16_t*)c->vc(l)};
    PROF(c, KS_KC_GEMM_QKV, gemm_bf16_skinny(g, c->st));
    if (!fused) {
      QkvPostArgs qp{R, d.hq, d.hkv, d.hd, d.n_max, d.dtype, d.qk_norm, d.eps, qkv, rope,
                     c->q_norm[l], c->k_norm[l], pos, q, c->kc(l), c->vc(l), kvs, mode, 1};
      PROF(c, KS_KC_QKV_POST, qkv_post(qp, c->st));
    }
  } else {
    PROF(c, KS_KC_NORM,
         norm_act(xin, d.d, c->attn_norm[l], d.eps, R, d.d, d.dtype, a1, c->st));
    PROF(c, KS_KC_GEMM_QKV,
         gemm(c, R, c->y.nqkv, d.d, a1, c->wqkv[l], EPI_STORE, qkv, c->y.nqkv, nullptr, 0,
              Act{}, batched));
    QkvPostArgs qp{R, d.hq, d.hkv, d.hd, d.n_max, d.dtype, d.qk_norm, d.eps, qkv, rope,
                   c->q_norm[l], c->k_norm[l], pos, q, c->kc(l), c->vc(l), kvs, mode,
                   c->bf() ? 1 : 0};
    PROF(c, KS_KC_QKV_POST, qkv_post(qp, c->st));
  }
  const int tiles = batched ? BAT_TILES : dec_tiles(d.n_max, d.hkv);
  const int span = batched ? 64 * BAT_TILES : dec_span(d);
  const int ns = (d.n_max + span - 1) / span;
  const int step = batched ? c->y.PA : 16;
  for (int r0 = 0; r0 < R; r0 += step) {
    const int rr = std::min(step, R - r0);
    AttnArgs aa{rr, d.hq, d.hkv, d.hd, d.n_max, d.dtype,
                q + (size_t)r0 * d.hq * d.hd, c->kc(l), c->vc(l), len + r0, max_len, tiles, span,
                attn_rows_per_block(d.hq / d.hkv, batched), c->at<float>(c->y.part), ns};
    PROF(c, KS_KC_ATTN, attn_split(aa, c->st));
    Act out2 = a2;
    const size_t off = (size_t)r0 * a2.ld * (c->bf() ? 2 : 4);
    out2.hi = (char*)a2.hi + off;
    out2.lo = c->bf() ? (char*)a2.lo + (size_t)r0 * a2.ld * 2 : nullptr;
    PROF(c, KS_KC_COMBINE,
         attn_combine(aa, mode == 1 ? kvs + (size_t)r0 * 2 * d.hkv * d.hd : nullptr, out2,
                      c->st));
  }
  PROF(c, KS_KC_GEMM_O, resid_gemm(c, R, d.hq * d.hd, a2, c->wo[l], xout, xin, batched, next_gain));
}

void mlp_rows(ks_ctx* c, int l, const float* xin, float* xout, int R, bool batched,
              const float* next_gain) {
  const ks_model_desc& d = c->md;
  const Act a1 = c->act1(), a2 = c->act2();
  if (skinny(c, R, batched)) {
    PROF(c, KS_KC_GEMM_GATE_UP,
         gemm_bf16_skinny(normed(c, R, 2 * d.ffn, c->wgu[l], EPI_SWIGLU, nullptr, 0, a2),
                          c->st));
  } else {
    PROF(c, KS_KC_NORM,
         norm_act(xin, d.d, c->mlp_norm[l], d.eps, R, d.d, d.dtype, a1, c->st));
    PROF(c, KS_KC_GEMM_GATE_UP,
         gemm(c, R, 2 * d.ffn, d.d, a1, c->wgu[l], EPI_SWIGLU, nullptr, 0, nullptr, 0, a2,
              batched));
  }
  PROF(c, KS_KC_GEMM_DOWN, resid_gemm(c, R, d.ffn, a2, c->wdown[l], xout, xin, batched, next_gain));
}

// Sublayer i on R rows.  Skinny path: the planes of x_in for sublayer i's norm
// must be in act1 (next_gain: also produce those of x_out for the next normed
// product).
void sublayer_rows(ks_ctx* c, int i, const float* xin, float* xout, int R, const int32_t* pos,
                   const int32_t* len, int max_len, int mode, bool batched,
                   const float* next_gain = nullptr) {
  const int l = (i - 1) / 2;
  if (i % 2 == 1) attn_rows(c, l, xin, xout, R, pos, len, max_len, mode, batched, next_gain);
  else mlp_rows(c, l, xin, xout, R, batched, next_gain);
}

// final norm + LM head + argmax for R rows (chunked by the logits buffer);
// prepped: on the skinny path the final-norm planes of x are already in act1
// (sampling: ss != nullptr, R <= gamma_max + 1, tables / draws as ss says)
void head_rows(ks_ctx* c, const float* x, int R, float* logits_out, int32_t* am, float* top1,
               bool batched, bool prepped = false, const SampleSpec* ss = nullptr) {
  const ks_model_desc& d = c->md;
  const Act a1 = c->act1();
  const int step = logits_out ? R : c->y.LR;
  for (int r0 = 0; r0 < R; r0 += step) {
    const int rr = std::min(step, R - r0);
    float* lg = logits_out ? logits_out : c->at<float>(c->y.logits);
    const float* xr = x + (size_t)r0 * d.d;
    if (skinny(c, rr, batched)) {
      if (!prepped) prep_rows(c, xr, rr, c->final_norm);
      PROF(c, KS_KC_GEMM_HEAD,
           gemm_bf16_skinny(normed(c, rr, d.vocab, c->lm_head, EPI_STORE, lg, d.vocab, Act{}),
                            c->st));
    } else {
      PROF(c, KS_KC_NORM, norm_act(xr, d.d, c->final_norm, d.eps, rr, d.d, d.dtype, a1, c->st));
      PROF(c, KS_KC_GEMM_HEAD,
           gemm(c, rr, d.vocab, d.d, a1, c->lm_head, EPI_STORE, lg, d.vocab, nullptr, 0, Act{},
                true));
    }
    if (ss) {
      PROF(c, KS_KC_ARGMAX, sample_rows(lg, rr, d.vocab, d.vocab, *ss, c->ws + c->y.vws, c->st));
      continue;
    }
    for (int a0 = 0; a0 < rr; a0 += c->y.LR) {
      const int ra = std::min(c->y.LR, rr - a0);
      PROF(c, KS_KC_ARGMAX,
           argmax_rows(lg + (size_t)a0 * d.vocab, ra, d.vocab, d.vocab, am + r0 + a0,
                       top1 ? top1 + r0 + a0 : nullptr, c->ws + c->y.vws, c->st));
    }
  }
}

// one decode row at position p from token tok_dev[0]; writes argmax to am_out
// (ss: sample the token instead, see head_rows)
void decode_row(ks_ctx* c, const int32_t* tok_dev, int p, const uint8_t* exec, int32_t* am_out,
                float* top1_out, const SampleSpec* ss = nullptr) {
  const ks_model_desc& d = c->md;
  const int L2 = 2 * d.L;
  float* x = c->at<float>(c->y.x);
  int32_t* pos = c->at<int32_t>(c->y.pos);
  int32_t* len = c->at<int32_t>(c->y.len);
  auto next_exec = [&](int i) {  // first executed sublayer after i (L2 + 1: the head)
    int j = i + 1;
    while (j <= L2 && exec && !exec[j - 1]) ++j;
    return j;
  };
  if (c->bf()) {
    // the embedding launch also writes the row's position and length
    PROF(c, KS_KC_EMBED,
         act_prep(nullptr, d.d, c->embed, d.dtype, tok_dev, 1, d.d, x,
                  gain_of(c, next_exec(0)), c->act1(), c->at<float>(c->y.ssq), c->st,
                  PosFill{pos, len, p, 1, 1}));
  } else {
    PROF(c, KS_KC_OTHER, fill_pos(pos, len, p, 1, 1, 1, c->st));
    PROF(c, KS_KC_EMBED, embed_rows(c->embed, d.dtype, tok_dev, 1, d.d, x, d.d, c->st));
  }
  for (int i = 1; i <= L2; ++i)
    if (!exec || exec[i - 1])
      sublayer_rows(c, i, x, x, 1, pos, len, p + 1, 0, false, gain_of(c, next_exec(i)));
  head_rows(c, x, 1, nullptr, am_out, top1_out, false, true, ss);
}

// verify rows of tokens tok_dev[0..R) at positions P..P+R-1, snapshots into stage
void verify_rows(ks_ctx* c, const int32_t* tok_dev, int R, int32_t* am_out,
                 const SampleSpec* ss = nullptr) {
  const ks_model_desc& d = c->md;
  int32_t* pos = c->at<int32_t>(c->y.pos);
  int32_t* len = c->at<int32_t>(c->y.len);
  if (skinny(c, R, false)) {
    act_prep(nullptr, d.d, c->embed, d.dtype, tok_dev, R, d.d, c->stage_row(0, 0), gain_of(c, 1),
             c->act1(), c->at<float>(c->y.ssq), c->st, PosFill{pos, len, c->P, R, 1});
  } else {
    fill_pos(pos, len, c->P, R, R, 1, c->st);
    embed_rows(c->embed, d.dtype, tok_dev, R, d.d, c->stage_row(0, 0), d.d, c->st);
  }
  for (int i = 1; i <= 2 * d.L; ++i)
    sublayer_rows(c, i, c->stage_row(i - 1, 0), c->stage_row(i, 0), R, pos, len, c->P + R, 0,
                  false, gain_of(c, i + 1));
  head_rows(c, c->stage_row(2 * d.L, 0), R, nullptr, am_out, nullptr, false, true, ss);
}

// copy rows [0, n) of plane set src (plane stride plane_stride_rows rows) into
// the history ring at positions p0..p0+n-1 for every sublayer output
hipError_t stash_history(ks_ctx* c, const float* src0, size_t plane_stride_rows, int n, int p0) {
  const ks_model_desc& d = c->md;
  ring_copy(src0, c->at<float>(c->y.hist), plane_stride_rows, 2 * d.L + 1, n, c->y.RING, p0, d.d,
            true, c->st);
  return hipGetLastError();
}

int hist_rows(const ks_ctx* c) {
  int r = 0;
  for (auto& b : c->blocks) r += b.second;
  return r;
}

}  // namespace

// =============================================================== C ABI
// Scratch of ks_sample_filter_noalloc: one file-scope device array per GPU
// the library runs on (it lives until the process ends).  Host code never
// passes the array's name to a kernel: its device address on each GPU comes
// from hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t KS_NOALLOC_SCRATCH_BYTES = (size_t)4 << 20;
static __device__ __align__(256) unsigned char scratch[KS_NOALLOC_SCRATCH_BYTES];
constexpr int KS_NOALLOC_MAX_DEVICES = 64;
static std::atomic<void*> g_scratch_ptr[KS_NOALLOC_MAX_DEVICES];

static ks_status scratch_address(void** out) {
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= KS_NOALLOC_MAX_DEVICES) {
    set_error("device index beyond the allocation-free entry point's table");
    return KS_EINVAL;
  }
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return KS_OK;
}

extern "C" {

const char* ks_last_error(void) { return g_err.c_str(); }

static ks_status check_desc(const ks_model_desc* d) {
  REQ(d, "desc is null");
  REQ(d->L >= 1 && 2 * d->L <= KS_MAX_SUBLAYERS, "L out of range");
  REQ(d->hq >= 1 && d->hkv >= 1 && d->hq % d->hkv == 0, "hq must be a multiple of hkv");
  REQ(d->hq / d->hkv <= 32, "query heads per kv head must be <= 32");
  REQ(d->dtype == KS_F32 || d->dtype == KS_BF16, "dtype must be KS_F32 or KS_BF16");
  REQ((d->dtype == KS_BF16 && d->hd == 128) || (d->dtype == KS_F32 && d->hd == 64),
      "supported head dims: 128 for bf16 models, 64 for float32 models");
  REQ(d->d >= 32 && d->d % 32 == 0, "d must be a positive multiple of 32");
  REQ(d->ffn >= 32 && d->ffn % 32 == 0, "ffn must be a positive multiple of 32");
  REQ((d->hq * d->hd) % 32 == 0, "hq*hd must be a multiple of 32");
  REQ(d->vocab >= 16 && d->vocab % 16 == 0, "vocab must be a positive multiple of 16");
  REQ(vocab_fits(d->vocab, 0), "vocab must be at most 524288");
  REQ(d->n_max >= 2, "n_max must be >= 2");
  REQ(d->eps >= 0.f, "eps must be >= 0");
  REQ(d->rope_theta > 0.0, "rope_theta must be > 0");
  return KS_OK;
}

static ks_status check_lim(const ks_limits* l) {
  REQ(l, "limits is null");
  REQ(l->gamma_max >= 0 && l->gamma_max <= 15, "gamma_max must be in [0, 15]");
  REQ(l->m_rounds >= 1 && l->m_rounds <= 64, "m_rounds must be in [1, 64]");
  REQ(l->cap_max >= 1 && l->cap_max <= 8192, "cap_max must be in [1, 8192]");
  REQ(l->prefill_chunk >= 16 && l->prefill_chunk <= 4096 && l->prefill_chunk % 16 == 0,
      "prefill_chunk must be a multiple of 16 in [16, 4096]");
  return KS_OK;
}

size_t ks_kv_cache_bytes(const ks_model_desc* d) {
  if (check_desc(d) != KS_OK) return 0;
  return (size_t)d->L * 2 * d->hkv * d->n_max * d->hd * (d->dtype == KS_BF16 ? 2 : 4);
}

size_t ks_workspace_bytes(const ks_model_desc* d, const ks_limits* l) {
  if (check_desc(d) != KS_OK || check_lim(l) != KS_OK) return 0;
  return make_layout(*d, *l).total;
}

ks_status ks_pack_matrix(const void* src, void* dst, int N, int K, int dtype, void* stream) {
  REQ(src && dst, "null pointer");
  REQ(N > 0 && K > 0, "N and K must be positive");
  REQ(dtype == KS_F32 || dtype == KS_BF16, "bad dtype");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == KS_F32) {
    HIPCHK(hipMemcpyAsync(dst, src, (size_t)N * K * 4, hipMemcpyDeviceToDevice, st));
    return KS_OK;
  }
  REQ(N % 16 == 0 && K % 32 == 0, "bf16 packing needs N % 16 == 0 and K % 32 == 0");
  pack_matrix_bf16((const bf16_t*)src, (bf16_t*)dst, N, K, st);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_pack_qkv(const void* src, void* dst, int hq, int hkv, int hd, int d, int dtype,
                      void* stream) {
  REQ(src && dst, "null pointer");
  REQ(hq > 0 && hkv > 0 && hd > 0 && d > 0, "sizes must be positive");
  REQ(dtype == KS_F32 || dtype == KS_BF16, "bad dtype");
  hipStream_t st = (hipStream_t)stream;
  const int N = (hq + 2 * hkv) * hd;
  if (dtype == KS_F32) {
    HIPCHK(hipMemcpyAsync(dst, src, (size_t)N * d * 4, hipMemcpyDeviceToDevice, st));
    return KS_OK;
  }
  REQ(hd % 16 == 0 && d % 32 == 0, "bf16 packing needs hd % 16 == 0 and d % 32 == 0");
  pack_qkv_bf16((const bf16_t*)src, (bf16_t*)dst, hq + 2 * hkv, hd, d, st);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_pack_gate_up(const void* gate, const void* up, void* dst, int ffn, int d, int dtype,
                          void* stream) {
  REQ(gate && up && dst, "null pointer");
  REQ(ffn > 0 && d > 0, "sizes must be positive");
  REQ(dtype == KS_F32 || dtype == KS_BF16, "bad dtype");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == KS_F32) {
    const size_t b = (size_t)ffn * d * 4;
    HIPCHK(hipMemcpyAsync(dst, gate, b, hipMemcpyDeviceToDevice, st));
    HIPCHK(hipMemcpyAsync((char*)dst + b, up, b, hipMemcpyDeviceToDevice, st));
    return KS_OK;
  }
  REQ(ffn % 16 == 0 && d % 32 == 0, "bf16 packing needs ffn % 16 == 0 and d % 32 == 0");
  pack_gate_up_bf16((const bf16_t*)gate, (const bf16_t*)up, (bf16_t*)dst, ffn, d, st);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_create(const ks_model_desc* desc, const ks_limits* lim, const ks_weights* w,
                    void* kv_cache, size_t kv_bytes, void* workspace, size_t ws_bytes,
                    void* stream, ks_ctx** out) {
  ks_status s = check_desc(desc);
  if (s != KS_OK) return s;
  s = check_lim(lim);
  if (s != KS_OK) return s;
  REQ(w && out && kv_cache && workspace, "null pointer");
  REQ(w->embed && w->lm_head && w->final_norm && w->attn_norm && w->wqkv && w->wo &&
          w->mlp_norm && w->w_gate_up && w->w_down,
      "null weight pointer");
  for (int l = 0; l < desc->L; ++l) {
    REQ(w->attn_norm[l] && w->wqkv[l] && w->wo[l] && w->mlp_norm[l] && w->w_gate_up[l] &&
            w->w_down[l],
        "null per-layer weight pointer");
    if (desc->qk_norm) REQ(w->q_norm && w->k_norm && w->q_norm[l] && w->k_norm[l], "qk_norm gains missing");
  }
  const Layout y = make_layout(*desc, *lim);
  if (kv_bytes < ks_kv_cache_bytes(desc)) {
    set_error("kv cache smaller than ks_kv_cache_bytes");
    return KS_ENOMEM;
  }
  if (ws_bytes < y.total) {
    set_error("workspace smaller than ks_workspace_bytes");
    return KS_ENOMEM;
  }
  ks_ctx* c = new ks_ctx();
  c->md = *desc;
  c->lim = *lim;
  c->st = (hipStream_t)stream;
  c->embed = w->embed;
  c->lm_head = w->lm_head;
  c->final_norm = w->final_norm;
  for (int l = 0; l < desc->L; ++l) {
    c->wqkv.push_back(w->wqkv[l]);
    c->wo.push_back(w->wo[l]);
    c->wgu.push_back(w->w_gate_up[l]);
    c->wdown.push_back(w->w_down[l]);
    c->attn_norm.push_back(w->attn_norm[l]);
    c->mlp_norm.push_back(w->mlp_norm[l]);
    c->q_norm.push_back(desc->qk_norm ? w->q_norm[l] : nullptr);
    c->k_norm.push_back(desc->qk_norm ? w->k_norm[l] : nullptr);
  }
  c->kv = (char*)kv_cache;
  c->ws = (char*)workspace;
  c->y = y;
  hipError_t he = hipHostMalloc((void**)&c->pin, 4096, hipHostMallocDefault);
  if (he != hipSuccess) {
    set_error(std::string("pinned staging: ") + hipGetErrorString(he));
    delete c;
    return KS_EHIP;
  }
  rope_table(c->at<float>(y.rope), desc->n_max, desc->hd, desc->rope_theta, c->st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error(std::string("rope table: ") + hipGetErrorString(e));
    (void)hipHostFree(c->pin);
    delete c;
    return KS_EHIP;
  }
  *out = c;
  return KS_OK;
}

ks_status ks_destroy(ks_ctx* c) {
  REQ(c, "ctx is null");
  if (c->pin) (void)hipHostFree(c->pin);
  for (hipEvent_t e : c->prof_ev) (void)hipEventDestroy(e);
  delete c;
  return KS_OK;
}

ks_status ks_prefill(ks_ctx* c, const int32_t* tokens, int n, int32_t* out_first) {
  REQ(c && tokens, "null pointer");
  const ks_model_desc& d = c->md;
  REQ(n >= 1, "prompt must have at least one token");
  if (n >= d.n_max) {
    set_error("prompt does not fit the KV cache");
    return KS_ECAPACITY;
  }
  for (int t = 0; t < n; ++t) REQ(tokens[t] >= 0 && tokens[t] < d.vocab, "token id out of range");
  const int FR = c->lim.prefill_chunk;
  const int r0 = std::min(n, c->lim.m_rounds * (c->lim.gamma_max + 1));
  float* x = c->at<float>(c->y.x);
  int32_t* tok = c->at<int32_t>(c->y.tok);
  int32_t* pos = c->at<int32_t>(c->y.pos);
  int32_t* len = c->at<int32_t>(c->y.len);
  int32_t* am = c->at<int32_t>(c->y.am);
  for (int c0 = 0; c0 < n; c0 += FR) {
    const int R = std::min(FR, n - c0);
    HIPCHK(hipMemcpyAsync(tok, tokens + c0, R * 4, hipMemcpyHostToDevice, c->st));
    fill_pos(pos, len, c0, R, R, 1, c->st);
    embed_rows(c->embed, d.dtype, tok, R, d.d, x, d.d, c->st);
    const int h0 = std::max(c0, n - r0);  // first history row in this chunk
    for (int i = 0; i <= 2 * d.L; ++i) {
      if (i > 0) sublayer_rows(c, i, x, x, R, pos, len, c0 + R, 0, true);
      for (int p = h0; p < c0 + R;) {
        const int slot = p % c->y.RING;
        const int run = std::min(c0 + R - p, c->y.RING - slot);
        HIPCHK(hipMemcpyAsync(c->hist_row(i, slot), x + (size_t)(p - c0) * d.d,
                              (size_t)run * d.d * 4, hipMemcpyDeviceToDevice, c->st));
        p += run;
      }
    }
    if (c0 + R == n) {
      const SampleSpec ss = c->spec(0, nullptr, am, n, 2);
      head_rows(c, x + (size_t)(R - 1) * d.d, 1, nullptr, am, nullptr, false, false,
                c->sampling() ? &ss : nullptr);
    }
  }
  HIPCHK(hipGetLastError());
  int32_t first = 0;
  HIPCHK(hipMemcpyAsync(&first, am, 4, hipMemcpyDeviceToHost, c->st));
  HIPCHK(hipStreamSynchronize(c->st));
  c->P = n;
  c->s = first;
  c->k_draft = 0;
  c->blocks.clear();
  c->blocks.push_back({n - r0, r0});
  c->ready = true;
  if (out_first) *out_first = first;
  return KS_OK;
}

ks_status ks_set_context(ks_ctx* c, int n_cached, int32_t last_token) {
  REQ(c, "ctx is null");
  REQ(n_cached >= 0, "n_cached must be >= 0");
  if (n_cached >= c->md.n_max) {
    set_error("n_cached exceeds the KV cache");
    return KS_ECAPACITY;
  }
  REQ(last_token >= 0 && last_token < c->md.vocab, "token id out of range");
  c->P = n_cached;
  c->s = last_token;
  c->k_draft = 0;
  c->blocks.clear();
  c->ready = true;
  return KS_OK;
}

static ks_status draft_internal(ks_ctx* c, const uint8_t* exec) {
  int32_t* dt = c->at<int32_t>(c->y.tok);
  if (c->k_draft == 0) set_i32(dt, c->s, c->st);
  float* top1 = c->at<float>(c->y.top1) + c->k_draft;
  const SampleSpec ss =
      c->spec(c->qrow(c->k_draft), top1, dt + c->k_draft + 1, c->P + c->k_draft + 1, 0);
  decode_row(c, dt + c->k_draft, c->P + c->k_draft, exec, dt + c->k_draft + 1, top1,
             c->sampling() ? &ss : nullptr);
  c->k_draft++;
  return KS_OK;
}

ks_status ks_draft_step(ks_ctx* c, const uint8_t* exec, int32_t* out_token, float* out_top1) {
  REQ(c && exec, "null pointer");
  if (!c->ready) {
    set_error("ks_draft_step before ks_prefill / ks_set_context");
    return KS_ESTATE;
  }
  REQ(c->k_draft < c->lim.gamma_max, "draft longer than gamma_max");
  if (c->P + c->k_draft + 1 >= c->md.n_max) {
    set_error("draft position exceeds the KV cache");
    return KS_ECAPACITY;
  }
  draft_internal(c, exec);
  HIPCHK(hipGetLastError());
  int32_t t = 0;
  float p = 0.f;
  HIPCHK(hipMemcpyAsync(&t, c->at<int32_t>(c->y.tok) + c->k_draft, 4, hipMemcpyDeviceToHost, c->st));
  HIPCHK(hipMemcpyAsync(&p, c->at<float>(c->y.top1) + c->k_draft - 1, 4, hipMemcpyDeviceToHost, c->st));
  HIPCHK(hipStreamSynchronize(c->st));
  if (out_token) *out_token = t;
  if (out_top1) *out_top1 = p;
  return KS_OK;
}

// verify the gamma+1 tokens already in the device token buffer; host copies of
// the drafts in toks (toks[0] = s)
static ks_status verify_internal(ks_ctx* c, const int32_t* toks, int gamma, int32_t* out_pred,
                                 int* out_a) {
  const int R = gamma + 1;
  int32_t* am = c->at<int32_t>(c->y.am);
  int32_t* tok = c->at<int32_t>(c->y.tok);
  int32_t* y = c->pin + 16;
  int a = 0;
  if (c->sampling()) {
    // target tables of rows 0..gamma, then the acceptance chain against the
    // draft tables the draft steps left (Section 2.1, speculative sampling)
    const SampleSpec ss = c->spec(0, nullptr, nullptr, 0, 0);
    verify_rows(c, tok, R, am, &ss);
    int32_t* res = c->at<int32_t>(c->y.sres);
    const int q0 = c->qrow(0);
    spec_accept(c->tab_ids(0), c->tab_pr(0), c->tab_cnt(0), c->tab_ids(q0), c->tab_pr(q0),
                c->tab_cnt(q0), tok + 1, gamma, c->samp.seed, c->P, res, c->st);
    HIPCHK(hipGetLastError());
    HIPCHK(hipMemcpyAsync(y, res, 8, hipMemcpyDeviceToHost, c->st));
    HIPCHK(hipStreamSynchronize(c->st));
    a = y[0];
    const int32_t fin = y[1];
    for (int i = 0; i < R; ++i) y[i] = i < a ? toks[i + 1] : (i == a ? fin : -1);
  } else {
    verify_rows(c, tok, R, am);
    HIPCHK(hipGetLastError());
    HIPCHK(hipMemcpyAsync(y, am, R * 4, hipMemcpyDeviceToHost, c->st));
    HIPCHK(hipStreamSynchronize(c->st));
    while (a < gamma && toks[a + 1] == y[a]) ++a;
  }
  HIPCHK(stash_history(c, c->stage_row(0, 0), c->lim.gamma_max + 1, a + 1, c->P));
  c->blocks.push_back({c->P, a + 1});
  while ((int)c->blocks.size() > c->lim.m_rounds) c->blocks.pop_front();
  c->P += a + 1;
  c->s = y[a];
  c->k_draft = 0;
  if (out_pred) std::copy(y, y + R, out_pred);
  if (out_a) *out_a = a;
  return KS_OK;
}

ks_status ks_verify(ks_ctx* c, const int32_t* tokens, int gamma, int32_t* out_pred, int* out_a) {
  REQ(c && tokens, "null pointer");
  if (!c->ready) {
    set_error("ks_verify before ks_prefill / ks_set_context");
    return KS_ESTATE;
  }
  REQ(gamma >= 0 && gamma <= c->lim.gamma_max, "gamma out of range");
  REQ(tokens[0] == c->s, "tokens[0] must be the committed token");
  if (c->sampling() && c->k_draft != gamma) {
    set_error("sampling verify needs the gamma drafts of ks_draft_step since the last verify");
    return KS_ESTATE;
  }
  if (c->sampling() && gamma > 0) {
    // the acceptance chain reads the drafts' tables: the tokens must be those drafts
    int32_t* dh = c->pin + 32;
    HIPCHK(hipMemcpyAsync(dh, c->at<int32_t>(c->y.tok), (gamma + 1) * 4, hipMemcpyDeviceToHost,
                          c->st));
    HIPCHK(hipStreamSynchronize(c->st));
    for (int t = 1; t <= gamma; ++t) REQ(tokens[t] == dh[t], "sampling verify: tokens must be the drafts");
  }
  for (int t = 0; t <= gamma; ++t) REQ(tokens[t] >= 0 && tokens[t] < c->md.vocab, "token id out of range");
  if (c->P + gamma + 1 >= c->md.n_max) {
    set_error("verify positions exceed the KV cache");
    return KS_ECAPACITY;
  }
  HIPCHK(hipMemcpyAsync(c->at<int32_t>(c->y.tok), tokens, (gamma + 1) * 4, hipMemcpyHostToDevice,
                        c->st));
  return verify_internal(c, tokens, gamma, out_pred, out_a);
}

ks_status ks_set_draft_policy(ks_ctx* c, const ks_draft_policy* p) {
  REQ(c && p, "null pointer");
  REQ(std::isfinite(p->tau_conf) && p->tau_conf >= 0.f, "tau_conf must be finite and >= 0");
  REQ(p->gamma_source == KS_GAMMA_FIXED || p->gamma_source == KS_GAMMA_SELECTED,
      "gamma_source must be KS_GAMMA_FIXED or KS_GAMMA_SELECTED");
  c->tau_conf = p->tau_conf;
  c->gamma_source = p->gamma_source;
  return KS_OK;
}

ks_status ks_set_sampling(ks_ctx* c, const ks_sampling* s) {
  REQ(c, "ctx is null");
  if (c->k_draft != 0) {
    set_error("ks_set_sampling with a pending draft (verify it first)");
    return KS_ESTATE;
  }
  if (!s || !(s->temperature > 0.f)) {
    REQ(!s || std::isfinite(s->temperature), "temperature must be finite");
    c->samp = ks_sampling{};
    return KS_OK;
  }
  REQ(std::isfinite(s->temperature), "temperature must be finite");
  REQ(s->top_k >= 1 && s->top_k <= KS_SAMPLE_KMAX && s->top_k <= c->md.vocab,
      "top_k must be in [1, min(KS_SAMPLE_KMAX, vocab)]");
  REQ(s->top_p > 0.f && s->top_p <= 1.f, "top_p must be in (0, 1]");
  REQ(vocab_fits(c->md.vocab, s->top_k), "vocabulary too large for the sampling filter");
  c->samp = *s;
  return KS_OK;
}

static ks_status check_sampling(const ks_sampling* s, int vocab) {
  REQ(s, "null pointer");
  REQ(std::isfinite(s->temperature) && s->temperature > 0.f, "temperature must be finite and > 0");
  REQ(s->top_k >= 1 && s->top_k <= KS_SAMPLE_KMAX && s->top_k <= vocab,
      "top_k must be in [1, min(KS_SAMPLE_KMAX, vocab)]");
  REQ(s->top_p > 0.f && s->top_p <= 1.f, "top_p must be in (0, 1]");
  REQ(vocab_fits(vocab, s->top_k), "vocabulary too large for the sampling filter");
  return KS_OK;
}

size_t ks_sample_workspace_bytes(int rows, int vocab, int top_k) {
  if (rows < 1 || vocab < 1 || top_k < 1 || top_k > KS_SAMPLE_KMAX || top_k > vocab ||
      !vocab_fits(vocab, top_k))
    return 0;
  return sample_ws_bytes(rows, vocab, top_k);
}

ks_status ks_sample_filter(const float* logits, int rows, int vocab, int ld, const ks_sampling* s,
                           int pos0, int purpose, int32_t* ids, float* probs, int32_t* counts,
                           float* top1, int32_t* tokens, void* workspace, size_t ws_bytes,
                           void* stream) {
  REQ(logits && ids && probs && counts && workspace, "null pointer");
  REQ(rows >= 1 && rows <= 65535 && vocab >= 1 && ld >= vocab, "sizes out of range");
  ks_status st = check_sampling(s, vocab);
  if (st != KS_OK) return st;
  REQ(pos0 >= 0 && purpose >= 0, "pos0 and purpose must be >= 0");
  if (ws_bytes < sample_ws_bytes(rows, vocab, s->top_k)) {
    set_error("workspace smaller than ks_sample_workspace_bytes");
    return KS_ENOMEM;
  }
  const SampleSpec ss{s->temperature, s->top_k, s->top_p, s->seed, ids, probs, counts, top1,
                      tokens, pos0, purpose};
  sample_rows(logits, rows, vocab, ld, ss, workspace, (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_sample_filter_noalloc(const float* logits, int rows, int vocab, int ld,
                                   const ks_sampling* s, int pos0, int purpose, int32_t* ids,
                                   float* probs, int32_t* counts, float* top1, int32_t* tokens,
                                   void* stream) {
  REQ(logits && ids && probs && counts, "null pointer");
  REQ(rows >= 1 && rows <= 65535 && vocab >= 1 && ld >= vocab, "sizes out of range");
  ks_status st = check_sampling(s, vocab);
  if (st != KS_OK) return st;
  REQ(pos0 >= 0 && purpose >= 0, "pos0 and purpose must be >= 0");
  if (sample_ws_bytes(rows, vocab, s->top_k) > KS_NOALLOC_SCRATCH_BYTES) {
    set_error("rows x vocabulary need more scratch than the allocation-free filter holds "
              "(4 MiB): use ks_sample_filter with a workspace");
    return KS_ENOMEM;
  }
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != KS_OK) return st;
  const SampleSpec ss{s->temperature, s->top_k, s->top_p, s->seed, ids, probs, counts, top1,
                      tokens, pos0, purpose};
  sample_rows(logits, rows, vocab, ld, ss, ws, (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_spec_accept(const int32_t* p_ids, const float* p_probs, const int32_t* p_counts,
                         const int32_t* q_ids, const float* q_probs, const int32_t* q_counts,
                         const int32_t* drafts, int gamma, uint64_t seed, int pos0, int32_t* out,
                         void* stream) {
  REQ(p_ids && p_probs && p_counts && out, "null pointer");
  REQ(gamma == 0 || (q_ids && q_probs && q_counts && drafts), "null pointer");
  REQ(gamma >= 0 && gamma <= 1024 && pos0 >= 0, "gamma must be in [0, 1024], pos0 >= 0");
  spec_accept(p_ids, p_probs, p_counts, q_ids, q_probs, q_counts, drafts, gamma, seed, pos0, out,
              (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_sample_uniforms(uint64_t seed, const int32_t* pos, int n, int purpose, float* out,
                             void* stream) {
  REQ(n >= 0 && purpose >= 0, "n and purpose must be >= 0");
  REQ(n == 0 || (pos && out), "null pointer");
  if (n == 0) return KS_OK;
  uniforms(seed, pos, n, purpose, out, (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_hidden_cos(const float* X, const float* Y, int groups, int r, int d, float* out,
                        void* stream) {
  REQ(X && Y && out, "null pointer");
  REQ(groups >= 0 && r >= 1 && r <= 8192 && d >= 1, "sizes out of range (1 <= r <= 8192)");
  cos_groups(X, Y, groups, r, d, out, (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

// ------------------------------------------------------------- selection
static ks_status select_internal(ks_ctx* c, const ks_select_params* p, ks_selection* out,
                                 ks_selection_debug* dbg) {
  const ks_model_desc& d = c->md;
  const int L2 = 2 * d.L;
  const int r = hist_rows(c);
  const int n = c->P;
  // latency weights (Section 3.4, Appendix C)
  const double ta = p->c2 * n + p->c3, tm = p->c1;
  REQ(ta > 0 && tm > 0, "latency model gives a non-positive latency");
  double delta;
  if (p->quant_mode == KS_QUANT_PAPER_MIN) {
    delta = std::min(ta, tm);
  } else {
    REQ(p->bins >= 1, "bins must be >= 1");
    delta = d.L * (ta + tm) / p->bins;
  }
  const int wa = std::max(1, (int)std::floor(ta / delta + 0.5));
  const int wm = std::max(1, (int)std::floor(tm / delta + 0.5));
  const int C = d.L * (wa + wm);
  if (C > c->lim.cap_max) {
    set_error("knapsack capacity exceeds cap_max");
    return KS_ENOMEM;
  }
  const int J = p->prune_half ? C / 2 : C;
  if (dbg) REQ(dbg->J_cap >= J + 1, "debug arrays too small");
  const int base = n - r;
  float* Xh = c->at<float>(c->y.xh);  // [2L+1][r][d]
  // gather history rows into contiguous planes
  ring_copy(c->at<float>(c->y.hist), Xh, r, L2 + 1, r, c->y.RING, base, d.d, false, c->st);
  HIPCHK(hipGetLastError());
  auto X = [&](int i) { return Xh + (size_t)i * r * d.d; };
  int32_t* dpos = c->at<int32_t>(c->y.dpos);
  int32_t* dlen = c->at<int32_t>(c->y.dlen);
  fill_pos(dpos, dlen, base, r, c->y.cells * r, 0, c->st);
  float* gprev = c->at<float>(c->y.g0);
  float* gnext = c->at<float>(c->y.g1);
  float* E = c->at<float>(c->y.ge);
  double* sig = c->at<double>(c->y.sig);
  const float** ptr_src = c->at<const float*>(c->y.ptrs);
  float** ptr_dst = (float**)(ptr_src + c->y.cells + 2);
  const size_t cell = (size_t)r * d.d;
  HIPCHK(hipMemcpyAsync(gprev, X(0), cell * 4, hipMemcpyDeviceToDevice, c->st));
  // Stage 1 runs on the device stage after stage (k_dp_step), without host
  // round trips.  Each stage is launched for a bound on the reachable budgets:
  // every budget is at most min(J, sum of the weights so far); rows of
  // budgets outside the current list hold stale states that are never scored.
  const int S_ = c->y.cells;
  int* dcells = c->at<int>(c->y.dpc);
  int* dcnt = c->at<int>(c->y.dpn);
  uint8_t* dbits = c->at<uint8_t>(c->y.dpbits);
  set_i32(dcells, 0, c->st);  // stage 0: the single budget 0
  set_i32(dcnt, 1, c->st);
  int bound = 1, cum = 0;
  for (int i = 1; i <= L2; ++i) {
    const int w = (i % 2 == 1) ? wa : wm;
    const int M = bound * r;
    // execute candidates for every (possibly) reachable budget
    sublayer_rows(c, i, gprev, E, M, dpos, dlen, n, 1, true);
    // per-row cosines of both candidates against X^(i)
    cos_rows2(E, gprev, X(i), M, r, d.d, sig, sig + M, c->st);
    cum += w;
    const int bound_out = std::min(J, cum) + 1;
    DpStepArgs da{i, J, w, (double)p->tau, r, M, S_, sig,
                  dcells + ((i - 1) & 1) * S_, dcnt + ((i - 1) & 1),
                  dcells + (i & 1) * S_, dcnt + (i & 1),
                  c->at<double>(c->y.dpmean), c->at<int>(c->y.dpidx), dbits,
                  c->at<uint8_t>(c->y.dpreach), c->at<double>(c->y.dpse),
                  c->at<double>(c->y.dpss), E, gprev, gnext, X(i), cell, ptr_src, ptr_dst,
                  bound_out};
    dp_step(da, c->st);
    copy_rows(ptr_src, ptr_dst, bound_out, (int)cell, c->st);
    HIPCHK(hipGetLastError());
    std::swap(gprev, gnext);
    bound = bound_out;
  }
  // terminal list, decision bits (and the debug record) back to the host
  int nc_h = 0;
  HIPCHK(hipMemcpyAsync(&nc_h, dcnt + (L2 & 1), 4, hipMemcpyDeviceToHost, c->st));
  std::vector<int> cells(S_);
  HIPCHK(hipMemcpyAsync(cells.data(), dcells + (L2 & 1) * S_, (size_t)S_ * 4,
                        hipMemcpyDeviceToHost, c->st));
  std::vector<uint8_t> bits_s((size_t)(L2 + 1) * S_);
  HIPCHK(hipMemcpyAsync(bits_s.data(), dbits, bits_s.size(), hipMemcpyDeviceToHost, c->st));
  std::vector<uint8_t> reach_s;
  std::vector<double> se_s, ss_s;
  if (dbg) {
    reach_s.resize(bits_s.size());
    se_s.resize(bits_s.size());
    ss_s.resize(bits_s.size());
    HIPCHK(hipMemcpyAsync(reach_s.data(), c->at<uint8_t>(c->y.dpreach), reach_s.size(),
                          hipMemcpyDeviceToHost, c->st));
    HIPCHK(hipMemcpyAsync(se_s.data(), c->at<double>(c->y.dpse), se_s.size() * 8,
                          hipMemcpyDeviceToHost, c->st));
    HIPCHK(hipMemcpyAsync(ss_s.data(), c->at<double>(c->y.dpss), ss_s.size() * 8,
                          hipMemcpyDeviceToHost, c->st));
  }
  HIPCHK(hipStreamSynchronize(c->st));
  cells.resize(nc_h);
  std::vector<uint8_t> bits((size_t)(L2 + 1) * (J + 1), 0);
  for (int i = 1; i <= L2; ++i)
    for (int j = 0; j <= J; ++j) bits[(size_t)i * (J + 1) + j] = bits_s[(size_t)i * S_ + j];
  if (dbg) {
    for (int j = 0; j < dbg->J_cap; ++j) dbg->n_match[j] = -1;
    const double qnan = std::numeric_limits<double>::quiet_NaN();
    for (int i = 0; i <= L2; ++i)
      for (int j = 0; j < dbg->J_cap; ++j) {
        const size_t o = (size_t)i * dbg->J_cap + j;
        const bool in = i >= 1 && j <= J;
        const size_t q = (size_t)i * S_ + j;
        dbg->bits[o] = in ? bits_s[q] : 0;
        dbg->reach[o] = in ? reach_s[q] : (i == 0 && j == 0);
        dbg->sig_e[o] = in ? se_s[q] : qnan;
        dbg->sig_s[o] = in ? ss_s[q] : qnan;
      }
  }
  // stage 2: argmax rows of terminal states and of X^(2L)
  const int nc = (int)cells.size();
  int32_t* am = c->at<int32_t>(c->y.am);
  head_rows(c, gprev, nc * r, nullptr, am, nullptr, true);
  head_rows(c, X(L2), r, nullptr, am + (size_t)nc * r, nullptr, true);
  HIPCHK(hipGetLastError());
  std::vector<int32_t> ham((size_t)(nc + 1) * r);
  HIPCHK(hipMemcpyAsync(ham.data(), am, ham.size() * 4, hipMemcpyDeviceToHost, c->st));
  HIPCHK(hipStreamSynchronize(c->st));
  const int32_t* yref = ham.data() + (size_t)nc * r;
  const double hd = p->t_head / delta;  // the head's cost in units of Delta (0: paper's cost)
  double best = 0.0;
  int bj = 0, bg = 1, bm = r;
  std::vector<uint8_t> bex(L2, 1);
  for (int k = 0; k < nc; ++k) {
    const int j = cells[k];
    int nm = 0;
    for (int t = 0; t < r; ++t) nm += ham[(size_t)k * r + t] == yref[t];
    if (dbg) dbg->n_match[j] = nm;
    const double a = (double)nm / r;
    for (int g = 1; g <= p->D; ++g) {
      double e = 0.0, pw = 1.0;
      for (int q = 0; q <= g; ++q) {
        e += pw;
        pw *= a;
      }
      const double v = e / ((double)g * ((double)(C - j) + hd) + ((double)C + hd));
      if (v > best) {
        best = v;
        bj = j;
        bg = g;
        bm = nm;
      }
    }
  }
  // backtrack the winner from sublayer 2L down to 1
  std::vector<uint8_t> ex(L2, 1);
  int jj = bj;
  for (int i = L2; i >= 1; --i) {
    if (bits[(size_t)i * (J + 1) + jj]) {
      ex[i - 1] = 0;
      jj -= (i % 2 == 1) ? wa : wm;
    }
  }
  if (jj != 0) {
    set_error("internal error: backtrack did not end at budget 0");
    return KS_ESTATE;
  }
  std::memset(out->exec, 0, sizeof(out->exec));
  std::copy(ex.begin(), ex.end(), out->exec);
  out->j_star = bj;
  out->gamma_star = bg;
  out->C = C;
  out->w_attn = wa;
  out->w_mlp = wm;
  out->n_rows = r;
  out->n_cells = nc;
  out->tpt_star = best;
  out->alpha_hat = (double)bm / r;
  out->delta = delta;
  out->iv_rounds = out->iv_drafted = out->iv_accepted = out->iv_tokens = 0;
  out->iv_ms = 0.0;
  return KS_OK;
}

ks_status ks_knapsack_select(ks_ctx* c, const ks_select_params* p, ks_selection* out,
                             ks_selection_debug* dbg) {
  REQ(c && p && out, "null pointer");
  if (!c->ready || c->blocks.empty()) {
    set_error("ks_knapsack_select needs a history (run ks_prefill first)");
    return KS_ESTATE;
  }
  REQ(p->D >= 1 && p->D <= 64, "D must be in [1, 64]");
  REQ(p->quant_mode == KS_QUANT_PAPER_MIN || p->quant_mode == KS_QUANT_BINS, "bad quant_mode");
  REQ(!std::isnan(p->tau), "tau is NaN");
  REQ(std::isfinite(p->t_head) && p->t_head >= 0.0, "t_head must be finite and >= 0");
  if (dbg) REQ(dbg->bits && dbg->reach && dbg->sig_e && dbg->sig_s && dbg->n_match, "null debug array");
  return select_internal(c, p, out, dbg);
}

ks_status ks_sublayer_apply(ks_ctx* c, int i, const float* x_in, float* x_out, const int32_t* pos,
                            int R, int mode) {
  REQ(c && x_in && x_out && pos, "null pointer");
  const ks_model_desc& d = c->md;
  REQ(i >= 1 && i <= 2 * d.L, "sublayer index out of range");
  REQ(R >= 1 && R <= c->y.XR, "R out of range");
  REQ(mode == 0 || mode == 1, "mode must be 0 or 1");
  int mx = 0;
  std::vector<int32_t> hl(R);
  for (int t = 0; t < R; ++t) {
    REQ(pos[t] >= 0, "negative position");
    if (pos[t] + 1 >= d.n_max) {
      set_error("position exceeds the KV cache");
      return KS_ECAPACITY;
    }
    hl[t] = pos[t] + (mode == 0 ? 1 : 0);
    mx = std::max(mx, hl[t]);
  }
  int32_t* dp = c->at<int32_t>(c->y.pos);
  int32_t* dl = c->at<int32_t>(c->y.len);
  HIPCHK(hipMemcpyAsync(dp, pos, R * 4, hipMemcpyHostToDevice, c->st));
  HIPCHK(hipMemcpyAsync(dl, hl.data(), R * 4, hipMemcpyHostToDevice, c->st));
  // x_in may alias x_out: every kernel reads a residual element before writing it
  if (skinny(c, R, R > 16)) prep_rows(c, x_in, R, gain_of(c, i));
  sublayer_rows(c, i, x_in, x_out, R, dp, dl, mx, mode, R > 16);
  HIPCHK(hipGetLastError());
  HIPCHK(hipStreamSynchronize(c->st));
  return KS_OK;
}

ks_status ks_head_rows(ks_ctx* c, const float* x, int R, float* logits, int32_t* am, float* top1) {
  REQ(c && x && am && top1, "null pointer");
  REQ(R >= 1 && R <= c->y.XR, "R out of range");
  head_rows(c, x, R, logits, am, top1, R > 16);
  HIPCHK(hipGetLastError());
  HIPCHK(hipStreamSynchronize(c->st));
  return KS_OK;
}

static ks_status decode_internal(ks_ctx* c, int n_new, int gamma, int reselect_every,
                                 const ks_select_params* p, int32_t* out_tokens,
                                 ks_gen_stats* stats, ks_selection* sel_log, int max_sel_log) {
  ks_gen_stats st{};
  if (stats) st.ms_prefill = stats->ms_prefill;
  auto now = [] { return std::chrono::steady_clock::now(); };
  auto ms = [](auto a, auto b) { return std::chrono::duration<double, std::milli>(b - a).count(); };
  const auto t0 = now();
  const int32_t first = c->s;
  int produced = 1;
  out_tokens[0] = first;
  if (gamma == 0) {
    // greedy AR on the decode kernels; tokens chain through a 64-entry device
    // ring and are copied out every 63 steps
    constexpr int RB = 64;
    int32_t* chain = c->at<int32_t>(c->y.tok);
    set_i32(chain, first, c->st);
    const int steps = n_new - 1;
    std::vector<int32_t> tmp(RB);
    int flushed = 0;  // out_tokens[0..flushed] are final
    for (int k = 0; k < steps; ++k) {
      const SampleSpec ss = c->spec(0, nullptr, chain + ((k + 1) % RB), c->P + k + 1, 2);
      decode_row(c, chain + (k % RB), c->P + k, nullptr, chain + ((k + 1) % RB), nullptr,
                 c->sampling() ? &ss : nullptr);
      if ((k + 1) % (RB - 1) == 0 || k == steps - 1) {
        HIPCHK(hipMemcpyAsync(tmp.data(), chain, RB * 4, hipMemcpyDeviceToHost, c->st));
        HIPCHK(hipStreamSynchronize(c->st));
        for (int t = flushed + 1; t <= k + 1; ++t) out_tokens[t] = tmp[t % RB];
        flushed = k + 1;
      }
    }
    HIPCHK(hipGetLastError());
    HIPCHK(hipStreamSynchronize(c->st));
    c->P += steps;
    c->s = out_tokens[n_new - 1];
    c->k_draft = 0;
    c->blocks.clear();  // AR steps record no history
    st.ms_total = ms(t0, now());
    if (stats) *stats = st;
    return KS_OK;
  }
  // the first selection of a generation uses the last m (gamma + 1) prompt rows
  // (the prefill keeps m (gamma_max + 1), as it does not know gamma yet)
  if (c->blocks.size() == 1) {
    auto& b = c->blocks.front();
    const int cap = c->lim.m_rounds * (gamma + 1);
    if (b.second > cap) {
      b.first += b.second - cap;
      b.second = cap;
    }
  }
  ks_selection sel{};
  // the rounds run with the current mask: recorded in its log entry when the
  // next selection replaces it or the loop ends
  ks_selection iv{};
  auto iv_start = now();
  auto close_interval = [&]() {
    const int k = st.n_selections - 1;
    if (sel_log && k >= 0 && k < max_sel_log) {
      sel_log[k].iv_rounds = iv.iv_rounds;
      sel_log[k].iv_drafted = iv.iv_drafted;
      sel_log[k].iv_accepted = iv.iv_accepted;
      sel_log[k].iv_tokens = iv.iv_tokens;
      sel_log[k].iv_ms = ms(iv_start, now());
    }
    iv = ks_selection{};
  };
  auto do_select = [&]() -> ks_status {
    close_interval();
    const auto a = now();
    ks_status r = select_internal(c, p, &sel, nullptr);
    st.ms_select += ms(a, now());
    if (r == KS_OK) {
      if (sel_log && st.n_selections < max_sel_log) sel_log[st.n_selections] = sel;
      st.n_selections++;
    }
    iv_start = now();
    return r;
  };
  ks_status s = do_select();
  if (s != KS_OK) return s;
  int32_t* toks = c->pin;
  float* top1_h = (float*)(c->pin + 64);
  while (produced < n_new) {
    // draft cap of the round, then the dynamic exit on the draft's top-1
    // probability (Section 3, TPT maximization)
    const int cap = c->gamma_source == KS_GAMMA_SELECTED
                        ? std::max(1, std::min(gamma, sel.gamma_star))
                        : gamma;
    int g = 0;
    while (g < cap) {
      draft_internal(c, sel.exec);
      ++g;
      if (c->tau_conf > 0.f) {
        HIPCHK(hipMemcpyAsync(top1_h, c->at<float>(c->y.top1) + g - 1, 4, hipMemcpyDeviceToHost,
                              c->st));
        HIPCHK(hipStreamSynchronize(c->st));
        if (!(*top1_h >= c->tau_conf)) break;
      }
    }
    HIPCHK(hipGetLastError());
    HIPCHK(hipMemcpyAsync(toks, c->at<int32_t>(c->y.tok), (g + 1) * 4, hipMemcpyDeviceToHost,
                          c->st));
    int a = 0;
    int32_t pred[16];
    s = verify_internal(c, toks, g, pred, &a);
    if (s != KS_OK) return s;
    st.n_rounds++;
    st.n_drafted += g;
    st.n_accepted += a;
    iv.iv_rounds++;
    iv.iv_drafted += g;
    iv.iv_accepted += a;
    iv.iv_tokens += a + 1;
    const int before = produced;
    for (int t = 1; t <= a && produced < n_new; ++t) out_tokens[produced++] = toks[t];
    if (produced < n_new) out_tokens[produced++] = pred[a];
    if (produced < n_new && produced / reselect_every > before / reselect_every) {
      s = do_select();
      if (s != KS_OK) return s;
    }
  }
  HIPCHK(hipStreamSynchronize(c->st));
  close_interval();
  st.ms_total = ms(t0, now());
  if (stats) *stats = st;
  return KS_OK;
}

static ks_status check_decode_args(ks_ctx* c, int n_new, int gamma, int reselect_every,
                                   const ks_select_params* p, int32_t* out_tokens) {
  REQ(c && out_tokens, "null pointer");
  REQ(n_new >= 1, "n_new must be >= 1");
  REQ(gamma >= 0 && gamma <= c->lim.gamma_max, "gamma out of range");
  REQ(gamma == 0 || (p && reselect_every >= 1),
      "speculative decoding needs params and reselect_every >= 1");
  if (p) {
    REQ(p->D >= 1 && p->D <= 64, "D must be in [1, 64]");
    REQ(p->quant_mode == KS_QUANT_PAPER_MIN || p->quant_mode == KS_QUANT_BINS, "bad quant_mode");
    REQ(std::isfinite(p->t_head) && p->t_head >= 0.0, "t_head must be finite and >= 0");
  }
  return KS_OK;
}

ks_status ks_decode(ks_ctx* c, int n_new, int gamma, int reselect_every, const ks_select_params* p,
                    int32_t* out_tokens, ks_gen_stats* stats, ks_selection* sel_log,
                    int max_sel_log) {
  ks_status s = check_decode_args(c, n_new, gamma, reselect_every, p, out_tokens);
  if (s != KS_OK) return s;
  if (!c->ready || c->k_draft != 0) {
    set_error("ks_decode needs a committed state with no pending draft");
    return KS_ESTATE;
  }
  if (gamma > 0 && c->blocks.empty()) {
    set_error("ks_decode with gamma > 0 needs a history (run ks_prefill first)");
    return KS_ESTATE;
  }
  if ((long long)c->P + n_new + gamma + 1 >= c->md.n_max) {
    set_error("generation exceeds the KV cache");
    return KS_ECAPACITY;
  }
  if (stats) stats->ms_prefill = 0.0;
  return decode_internal(c, n_new, gamma, reselect_every, p, out_tokens, stats, sel_log,
                         max_sel_log);
}

ks_status ks_generate(ks_ctx* c, const int32_t* prompt, int n_prompt, int n_new, int gamma,
                      int reselect_every, const ks_select_params* p, int32_t* out_tokens,
                      ks_gen_stats* stats, ks_selection* sel_log, int max_sel_log) {
  ks_status s = check_decode_args(c, n_new, gamma, reselect_every, p, out_tokens);
  if (s != KS_OK) return s;
  REQ(prompt, "null pointer");
  if ((long long)n_prompt + n_new + gamma + 1 >= c->md.n_max) {
    set_error("prompt + generation exceeds the KV cache");
    return KS_ECAPACITY;
  }
  const auto tp0 = std::chrono::steady_clock::now();
  int32_t first = 0;
  s = ks_prefill(c, prompt, n_prompt, &first);
  if (s != KS_OK) return s;
  ks_gen_stats st{};
  st.ms_prefill =
      std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - tp0).count();
  s = decode_internal(c, n_new, gamma, reselect_every, p, out_tokens, &st, sel_log, max_sel_log);
  if (stats) *stats = st;
  return s;
}

ks_status ks_profile_decode(ks_ctx* c, const uint8_t* exec, int steps, int per_kernel,
                            ks_kernel_profile* out) {
  REQ(c && out, "null pointer");
  REQ(steps >= 1, "steps must be >= 1");
  if (!c->ready) {
    set_error("ks_profile_decode before ks_prefill / ks_set_context");
    return KS_ESTATE;
  }
  if (c->P + 1 >= c->md.n_max) {
    set_error("position exceeds the KV cache");
    return KS_ECAPACITY;
  }
  const int need = 2 * (16 * c->md.L + 64);
  while ((int)c->prof_ev.size() < need + 2) {
    hipEvent_t e;
    HIPCHK(hipEventCreate(&e));
    c->prof_ev.push_back(e);
  }
  ks_kernel_profile r{};
  int32_t* dt = c->at<int32_t>(c->y.tok) + 32;  // scratch slots past the draft chain
  hipEvent_t e0 = c->prof_ev[c->prof_ev.size() - 2], e1 = c->prof_ev.back();
  for (int sidx = 0; sidx < steps; ++sidx) {
    c->prof_rec.clear();
    set_i32(dt, c->s, c->st);
    HIPCHK(hipEventRecord(e0, c->st));
    c->prof_on = per_kernel != 0;
    decode_row(c, dt, c->P, exec, dt + 1, c->at<float>(c->y.top1));
    c->prof_on = false;
    HIPCHK(hipEventRecord(e1, c->st));
    HIPCHK(hipEventSynchronize(e1));
    HIPCHK(hipGetLastError());
    float ms_step = 0.f;
    HIPCHK(hipEventElapsedTime(&ms_step, e0, e1));
    r.ms_step += ms_step;
    for (auto& pr : c->prof_rec) {
      float m = 0.f;
      HIPCHK(hipEventElapsedTime(&m, c->prof_ev[pr.second], c->prof_ev[pr.second + 1]));
      r.ms[pr.first] += m;
      if (sidx == 0) r.launches[pr.first]++;
    }
  }
  for (int k = 0; k < KS_KC_COUNT; ++k)
    if (r.launches[k]) r.ms[k] /= (double)steps * r.launches[k];
  r.ms_step /= steps;
  r.steps = steps;
  *out = r;
  return KS_OK;
}

ks_status ks_time_launches(void* start_event, void* stop_event) {
  REQ((start_event == nullptr) == (stop_event == nullptr), "events must be both set or both null");
  g_timing = LaunchTiming{(hipEvent_t)start_event, (hipEvent_t)stop_event, 0};
  return KS_OK;
}

// ----------------------------------------------------- isolated knapsack
ks_status ks_knapsack_quantize(const double* t, const double* s, int B, int n, int bins,
                               int32_t* w, int32_t* q) {
#pragma clang fp contract(off)
  REQ(t && s && w && q, "null pointer");
  REQ(B >= 1 && n >= 1 && bins >= 1, "sizes must be positive");
  for (size_t k = 0; k < (size_t)B * n; ++k) REQ(t[k] > 0.0 && s[k] > 0.0 && s[k] <= 1.0, "t must be > 0 and s in (0, 1]");
  for (int b = 0; b < B; ++b) {
    double delta = 0.0;
    for (int i = 0; i < n; ++i) delta += t[(size_t)b * n + i];
    delta /= bins;
    for (int i = 0; i < n; ++i) {
      const size_t k = (size_t)b * n + i;
      const double wf = std::floor(t[k] / delta + 0.5);
      w[k] = std::max(1, (int)wf);
      const double ql = -std::log(s[k]) * 16777216.0;
      q[k] = (int32_t)std::floor(ql + 0.5);
    }
  }
  return KS_OK;
}

ks_status ks_knapsack_batch(const int32_t* w, const int32_t* q, int B, int n, int C, int max_skip,
                            int32_t* best, uint64_t* bits, void* stream) {
  REQ(w && q && best && bits, "null pointer");
  REQ(B >= 1 && n >= 1 && n <= 4096, "B >= 1 and 1 <= n <= 4096 required");
  REQ(C >= 0 && C <= 8191, "C must be in [0, 8191]");
  REQ(max_skip >= 0, "max_skip must be >= 0");
  knapsack_dp(w, q, B, n, C, max_skip, best, bits, (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_knapsack_backtrack(const uint64_t* bits, const int32_t* w, int B, int n, int C,
                                const int32_t* j, uint8_t* skip, int32_t* err, void* stream) {
  REQ(bits && w && j && skip && err, "null pointer");
  REQ(B >= 1 && n >= 1 && C >= 0 && C <= 8191, "sizes out of range");
  knapsack_backtrack(bits, w, B, n, C, j, skip, err, (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

ks_status ks_knapsack_batch_select(const int32_t* best, const uint64_t* bits, const int32_t* w,
                                   const double* s, int B, int n, int C, int D, int32_t* j_star,
                                   int32_t* gamma_star, double* tpt, uint8_t* skip, void* stream) {
  REQ(best && bits && w && s && j_star && gamma_star && tpt && skip, "null pointer");
  REQ(B >= 1 && n >= 1 && n <= 128, "B >= 1 and 1 <= n <= 128 required");
  REQ(C >= 0 && C <= 8191, "C must be in [0, 8191]");
  REQ(D >= 1 && D <= 64, "D must be in [1, 64]");
  knapsack_select(best, bits, w, s, B, n, C, D, j_star, gamma_star, tpt, skip, (hipStream_t)stream);
  HIPCHK(hipGetLastError());
  return KS_OK;
}

}  // extern "C"
