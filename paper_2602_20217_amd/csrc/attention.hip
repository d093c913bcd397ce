// GQA decode attention over a contiguous KV cache, split over the context.
//
// Grid: (split, kv head, row group).  A workgroup owns `tiles` consecutive
// 64-position tiles of one kv head.  Every thread issues its share of a
// tile's K and V loads at once (16-byte chunks, all in flight together) and
// stores them to LDS after one wait.  K rows are padded by four 32-bit words
// so that 16-byte LDS reads of 64 different rows cover all banks.  Each wave
// owns a fixed set of query vectors (the G = hq/hkv query heads of a row share
// the tile); a lane scores one key, softmax statistics use wave shuffles, and
// the output accumulation broadcasts each probability with a lane read.  The
// partial (o, max, sum) of each (row, query head, split) goes to memory and a
// second kernel merges the splits in ascending order.
//
// A row's arithmetic depends only on its own query, its length and the split
// size, never on the other rows of the launch, so the decode step and a verify
// row at the same position produce the same bits.
#include "ks_internal.h"

#include <cfloat>

namespace ks {

constexpr int TILE = 64;  // positions per LDS tile of the split kernel

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ inline float lo16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float hi16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

int attn_nsplit(int n_positions, int tiles) {
  const int span = TILE * tiles;
  return (n_positions + span - 1) / span;
}

// HD: head dim (128 for bf16 caches, 64 for float32 caches).  QMAX: query
// vectors per wave (rows_per_block * G <= 4 QMAX).
template <int HD, bool BF, int QMAX>
__global__ __launch_bounds__(256) void k_attn_split(int M, int hq, int hkv, int n_max,
                                                    const float* __restrict__ q,
                                                    const void* __restrict__ kc,
                                                    const void* __restrict__ vc,
                                                    const int32_t* __restrict__ len, int tiles,
                                                    int rows_per_block,
                                                    float* __restrict__ part, int nsplit) {
  constexpr int KW = BF ? HD / 2 : HD;  // 32-bit words per key row
  constexpr int KS = KW + 4;            // padded K row stride (words)
  constexpr int DPL = HD / 64;          // output dims per lane (1 or 2)
  constexpr int CPR = KW / 4;           // 16-byte chunks per row
  constexpr int NCH = TILE * CPR / 256; // chunks per thread per matrix
  static_assert((TILE * CPR) % 256 == 0, "tile chunking");
  __shared__ __align__(16) uint32_t Ks[TILE * KS];
  __shared__ __align__(16) uint32_t Vs[TILE * KW];

  const int split = blockIdx.x, kvh = blockIdx.y;
  const int r0 = blockIdx.z * rows_per_block;
  const int r1 = min(M, r0 + rows_per_block);
  const int G = hq / hkv;
  const int nq = (r1 - r0) * G;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int start = split * tiles * TILE;
  const float scale = 1.0f / sqrtf((float)HD);

  int maxlen = 0;
  for (int r = r0; r < r1; ++r) maxlen = max(maxlen, len[r]);
  if (start >= maxlen) return;
  const int ntile = min(tiles, (maxlen - start + TILE - 1) / TILE);

  float o[QMAX][DPL];
  float mrun[QMAX], lrun[QMAX];
#pragma unroll
  for (int j = 0; j < QMAX; ++j) {
    mrun[j] = -FLT_MAX;
    lrun[j] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[j][e] = 0.f;
  }

  const size_t es = BF ? 2 : 4;
  const char* kbase = (const char*)kc + (size_t)kvh * n_max * HD * es;
  const char* vbase = (const char*)vc + (size_t)kvh * n_max * HD * es;
  uint4 kr[NCH], vr[NCH];
  // rows past the end of a partial tile repeat its last row (never scored)
#define KS_FETCH(T0, CNT)                                                  \
  _Pragma("unroll") for (int u = 0; u < NCH; ++u) {                        \
    const int c_ = threadIdx.x + 256 * u;                                  \
    const int row_ = min(c_ / CPR, (CNT) - 1), ch_ = c_ % CPR;             \
    const size_t off_ = (size_t)((T0) + row_) * HD * es + ch_ * 16;        \
    kr[u] = *(const uint4*)(kbase + off_);                                 \
    vr[u] = *(const uint4*)(vbase + off_);                                 \
  }
  for (int tile = 0; tile < ntile; ++tile) {
    const int t0 = start + tile * TILE;
    KS_FETCH(t0, min(TILE, maxlen - t0));
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = threadIdx.x + 256 * u;
      const int row = c / CPR, ch = c % CPR;
      *(uint4*)&Ks[row * KS + ch * 4] = kr[u];
      *(uint4*)&Vs[row * KW + ch * 4] = vr[u];
    }
    __syncthreads();

#pragma unroll
    for (int j = 0; j < QMAX; ++j) {
      const int qi = wave + 4 * j;
      if (qi >= nq) break;
      const int r = r0 + qi / G;
      const int h = kvh * G + qi % G;
      const int vcnt = min(TILE, len[r] - t0);
      if (vcnt <= 0) continue;
      const float* qv = q + ((size_t)r * hq + h) * HD;
      float s0 = 0.f;
      const uint32_t* k0p = &Ks[lane * KS];
#pragma unroll 4
      for (int w4 = 0; w4 < KW / 4; ++w4) {
        const uint4 a = *(const uint4*)(k0p + 4 * w4);
        if (BF) {
          const float* qq = qv + 8 * w4;
          s0 = fmaf(qq[0], lo16(a.x), s0); s0 = fmaf(qq[1], hi16(a.x), s0);
          s0 = fmaf(qq[2], lo16(a.y), s0); s0 = fmaf(qq[3], hi16(a.y), s0);
          s0 = fmaf(qq[4], lo16(a.z), s0); s0 = fmaf(qq[5], hi16(a.z), s0);
          s0 = fmaf(qq[6], lo16(a.w), s0); s0 = fmaf(qq[7], hi16(a.w), s0);
        } else {
          const float* qq = qv + 4 * w4;
          s0 = fmaf(qq[0], __uint_as_float(a.x), s0); s0 = fmaf(qq[1], __uint_as_float(a.y), s0);
          s0 = fmaf(qq[2], __uint_as_float(a.z), s0); s0 = fmaf(qq[3], __uint_as_float(a.w), s0);
        }
      }
      s0 = lane < vcnt ? s0 * scale : -FLT_MAX;
      const float mt = wave_max(s0);
      const float mnew = fmaxf(mrun[j], mt);
      const float alpha = __expf(mrun[j] - mnew);
      const float p0 = lane < vcnt ? __expf(s0 - mnew) : 0.f;
      lrun[j] = lrun[j] * alpha + wave_sum(p0);
      mrun[j] = mnew;
      float acc[DPL];
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
#pragma unroll 8
      for (int t = 0; t < vcnt; ++t) {
        const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p0), t));
        const uint32_t vw = Vs[t * KW + lane];
        if (BF) {
          acc[0] = fmaf(pt, lo16(vw), acc[0]);
          acc[DPL - 1] = fmaf(pt, hi16(vw), acc[DPL - 1]);
        } else {
          acc[0] = fmaf(pt, __uint_as_float(vw), acc[0]);
        }
      }
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] = o[j][e] * alpha + acc[e];
    }
    __syncthreads();
  }

#undef KS_FETCH
#pragma unroll
  for (int j = 0; j < QMAX; ++j) {
    const int qi = wave + 4 * j;
    if (qi >= nq) break;
    const int r = r0 + qi / G;
    const int h = kvh * G + qi % G;
    if (len[r] <= start) continue;
    float* dst = part + (((size_t)r * hq + h) * nsplit + split) * (HD + 2);
    if (BF) {
      // lane owns dims 2 lane, 2 lane + 1 (the packed pair order)
      *(float2*)&dst[2 * lane] = make_float2(o[j][0], o[j][DPL - 1]);
    } else {
      dst[lane] = o[j][0];
    }
    if (lane == 0) {
      dst[HD] = mrun[j];
      dst[HD + 1] = lrun[j];
    }
  }
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ inline uint32_t pack2(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

// Batched-row attention with matrix instructions (bf16 cache, head dim 128),
// used for prefill chunks and the candidate rows of the selection DP.
//
// Query vectors of one kv head are ordered qi = row * G + g; a wave owns 16
// consecutive ones, a workgroup NWAVE waves.  Per 64-key tile of the split, K
// (rows padded to 272 bytes) and V (transposed, rows padded to 136 bytes) are
// staged in LDS.  Scores are computed transposed, S^T = K Q^T, with keys as the
// rows of 16x16x32 MFMAs: a lane then holds 16 scores of a single query vector,
// so the softmax statistics need only two cross-lane steps, and the
// probabilities are already laid out as the A operand of O += P V (the k index
// of that product is permuted identically in P and V).  Queries enter as hi +
// lo bf16 pairs; probabilities as bf16.  Partials use the layout of the split
// kernel above.
template <int NWAVE>
__global__ __launch_bounds__(NWAVE * 64) void k_attn_mfma(
    int M, int hq, int hkv, int n_max, const float* __restrict__ q,
    const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const int32_t* __restrict__ len, int span, float* __restrict__ part, int nsplit) {
  constexpr int HD = 128;
  constexpr int KT = 64;          // keys per tile
  constexpr int KSTR = HD + 8;    // K row stride (bf16)
  constexpr int VSTR = KT + 4;    // transposed V row stride (bf16)
  constexpr int NT = NWAVE * 64;  // threads
  constexpr int NCH = KT * 16 / NT;
  static_assert((KT * 16) % NT == 0, "staging");
  constexpr float NEG = -1.0e30f;
  __shared__ __align__(16) bf16_t Ks[KT * KSTR];
  __shared__ __align__(16) bf16_t Vt[HD * VSTR];
  __shared__ int s_len[NWAVE * 16];

  const int split = blockIdx.x, kvh = blockIdx.y;
  const int G = hq / hkv;
  const int NQ = M * G;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int qb = blockIdx.z * NWAVE * 16;
  const int j = lane & 15, g4 = lane >> 4;
  const int start = split * span;
  const float scale = 1.0f / sqrtf((float)HD);

  for (int t = threadIdx.x; t < NWAVE * 16; t += NT) {
    const int qi = qb + t;
    s_len[t] = qi < NQ ? len[qi / G] : 0;
  }
  __syncthreads();
  int maxlen = 0;
  for (int t = 0; t < NWAVE * 16; ++t) maxlen = max(maxlen, s_len[t]);
  const int end = min(maxlen, start + span);
  if (start >= end) return;

  const int qi = qb + wave * 16 + j;
  const int lim = min(s_len[wave * 16 + j], end);  // keys of column j in this split
  bf16x8_t qh[4], ql[4];
  {
    const bool ok = qi < NQ;
    const int row = ok ? qi / G : 0;
    const int h = kvh * G + (ok ? qi % G : 0);
    const float* qv = q + ((size_t)row * hq + h) * HD + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
      if (ok) {
        x0 = *(const float4*)(qv + 32 * ks);
        x1 = *(const float4*)(qv + 32 * ks + 4);
      }
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
      u32x4_t hv, lv;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float a = xs[2 * k], b = xs[2 * k + 1];
        const bf16_t ha = f2bf(a), hb = f2bf(b);
        hv[k] = (uint32_t)ha | ((uint32_t)hb << 16);
        lv[k] = pack2(a - bf2f(ha), b - bf2f(hb));
      }
      qh[ks] = __builtin_bit_cast(bf16x8_t, hv);
      ql[ks] = __builtin_bit_cast(bf16x8_t, lv);
    }
  }
  f32x4_t o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = NEG, l_run = 0.f;

  const bf16_t* kbase = kc + (size_t)kvh * n_max * HD;
  const bf16_t* vbase = vc + (size_t)kvh * n_max * HD;
  for (int t0 = start; t0 < end; t0 += KT) {
    const int cnt = min(KT, end - t0);
    uint4 kr[NCH], vr[NCH];
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = threadIdx.x + NT * u;
      const int r = min(c >> 4, cnt - 1), ch = c & 15;
      const size_t off = (size_t)(t0 + r) * HD + ch * 8;
      kr[u] = *(const uint4*)(kbase + off);
      vr[u] = *(const uint4*)(vbase + off);
    }
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = threadIdx.x + NT * u;
      const int r = c >> 4, ch = c & 15;
      *(uint4*)&Ks[r * KSTR + ch * 8] = kr[u];
      const uint32_t w[4] = {vr[u].x, vr[u].y, vr[u].z, vr[u].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Vt[(ch * 8 + 2 * e) * VSTR + r] = (bf16_t)(w[e] & 0xFFFF);
        Vt[(ch * 8 + 2 * e + 1) * VSTR + r] = (bf16_t)(w[e] >> 16);
      }
    }
    __syncthreads();

    // S^T = K Q^T: s[kt][v] = score(key t0 + 16 kt + 4 g4 + v, query column j)
    f32x4_t s[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      s[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8_t a = __builtin_bit_cast(
            bf16x8_t, *(const u32x4_t*)&Ks[(16 * kt + j) * KSTR + 32 * ks + 8 * g4]);
        s[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qh[ks], s[kt], 0, 0, 0);
        s[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, ql[ks], s[kt], 0, 0, 0);
      }
    }
    float mt = NEG;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = t0 + 16 * kt + 4 * g4 + v;
        s[kt][v] = key < lim ? s[kt][v] * scale : NEG;
        mt = fmaxf(mt, s[kt][v]);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = __expf(m_run - m_new);
    float ps = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = t0 + 16 * kt + 4 * g4 + v;
        const float p = key < lim ? __expf(s[kt][v] - m_new) : 0.f;
        s[kt][v] = p;
        ps += p;
      }
    ps += __shfl_xor(ps, 16);
    ps += __shfl_xor(ps, 32);
    l_run = l_run * alpha + ps;
    m_run = m_new;
    // rows of O are query vectors 4 g4 + v: rescale by their alpha
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float av = __shfl(alpha, 4 * g4 + v);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt][v] *= av;
    }
    // O += P V over two 32-key steps; element e of a lane group g4 is key
    // 4 g4 + e (e < 4) or 16 + 4 g4 + e - 4 (e >= 4) of the step
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      u32x4_t pv;
      pv[0] = pack2(s[2 * k2][0], s[2 * k2][1]);
      pv[1] = pack2(s[2 * k2][2], s[2 * k2][3]);
      pv[2] = pack2(s[2 * k2 + 1][0], s[2 * k2 + 1][1]);
      pv[3] = pack2(s[2 * k2 + 1][2], s[2 * k2 + 1][3]);
      const bf16x8_t pa = __builtin_bit_cast(bf16x8_t, pv);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const bf16_t* vrow = &Vt[(16 * dt + j) * VSTR + 32 * k2 + 4 * g4];
        const uint2 lo = *(const uint2*)vrow;
        const uint2 hi = *(const uint2*)(vrow + 16);
        const u32x4_t bv = {lo.x, lo.y, hi.x, hi.y};
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, __builtin_bit_cast(bf16x8_t, bv),
                                                        o[dt], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // partials: O rows are query vectors 4 g4 + v, columns dims 16 dt + j
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int t = wave * 16 + 4 * g4 + v;
    const int qv = qb + t;
    if (qv >= NQ || s_len[t] <= start) continue;
    const int row = qv / G, h = kvh * G + qv % G;
    float* dst = part + (((size_t)row * hq + h) * nsplit + split) * (HD + 2);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) dst[16 * dt + j] = o[dt][v];
  }
  if (g4 == 0 && qi < NQ && s_len[wave * 16 + j] > start) {
    const int row = qi / G, h = kvh * G + qi % G;
    float* dst = part + (((size_t)row * hq + h) * nsplit + split) * (HD + 2);
    dst[HD] = m_run;
    dst[HD + 1] = l_run;
  }
}

// One workgroup of 4 waves per (row, query head); output dims lane -> (2 lane,
// 2 lane + 1) for bf16 caches, lane for float32 caches.  The split maxima are
// reduced across the workgroup; wave w then merges splits s = w, w + 4, ...
// (loads of different splits are independent, so they are in flight together)
// and the four wave sums are added in wave order.  The row's own key/value
// (selection rows) joins the max and is added last.
template <int HD, bool BF>
__global__ __launch_bounds__(256) void k_attn_combine(int M, int hq, int hkv, int span,
                                                      const float* __restrict__ q,
                                                      const float* __restrict__ part, int nsplit,
                                                      const int32_t* __restrict__ len,
                                                      const float* __restrict__ kvself,
                                                      bf16_t* ohi, bf16_t* olo, float* of,
                                                      int ldact) {
  constexpr int DPL = HD / 64;
  __shared__ float s_m[4];
  __shared__ float s_acc[4][DPL * 64 + 1];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int gid = blockIdx.x;
  const int r = gid / hq, h = gid % hq;
  const int G = hq / hkv;
  const int kvh = h / G;
  const int L = len[r];
  const int ns = (L + span - 1) / span;
  const float* pr = part + ((size_t)r * hq + h) * nsplit * (HD + 2);
  const int d0 = BF ? 2 * lane : lane;

  float mloc = -FLT_MAX;
  for (int s = threadIdx.x; s < ns; s += 256) mloc = fmaxf(mloc, pr[(size_t)s * (HD + 2) + HD]);
  mloc = wave_max(mloc);
  if (lane == 0) s_m[wave] = mloc;
  __syncthreads();
  float mx = fmaxf(fmaxf(s_m[0], s_m[1]), fmaxf(s_m[2], s_m[3]));
  float sself = 0.f;
  if (kvself) {
    const float* ks = kvself + (((size_t)r * 2 + 0) * hkv + kvh) * HD;
    const float* qv = q + ((size_t)r * hq + h) * HD;
    float dd = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) dd = fmaf(qv[d0 + e], ks[d0 + e], dd);
    sself = wave_sum(dd) * (1.0f / sqrtf((float)HD));
    mx = fmaxf(mx, sself);
  }
  float lsum = 0.f, acc[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
#pragma unroll 4
  for (int s = wave; s < ns; s += 4) {
    const float* ps = pr + (size_t)s * (HD + 2);
    const float w = __expf(ps[HD] - mx);
    lsum = fmaf(ps[HD + 1], w, lsum);
    if (DPL == 2) {
      const float2 v = *(const float2*)&ps[d0];
      acc[0] = fmaf(v.x, w, acc[0]);
      acc[DPL - 1] = fmaf(v.y, w, acc[DPL - 1]);
    } else {
      acc[0] = fmaf(ps[d0], w, acc[0]);
    }
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) s_acc[wave][DPL * lane + e] = acc[e];
  if (lane == 0) s_acc[wave][DPL * 64] = lsum;
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int e = 0; e < DPL; ++e)
    acc[e] = ((s_acc[0][DPL * lane + e] + s_acc[1][DPL * lane + e]) + s_acc[2][DPL * lane + e]) +
             s_acc[3][DPL * lane + e];
  lsum = ((s_acc[0][DPL * 64] + s_acc[1][DPL * 64]) + s_acc[2][DPL * 64]) + s_acc[3][DPL * 64];
  if (kvself) {
    const float* vs = kvself + (((size_t)r * 2 + 1) * hkv + kvh) * HD;
    const float w = __expf(sself - mx);
    lsum += w;
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = fmaf(vs[d0 + e], w, acc[e]);
  }
  const float inv = 1.0f / lsum;
  const size_t off = (size_t)r * ldact + (size_t)h * HD + d0;
  if (of) {
#pragma unroll
    for (int e = 0; e < DPL; ++e) of[off + e] = acc[e] * inv;
  } else {
    uint32_t hp = 0, lp = 0;
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      const float v = acc[e] * inv;
      const bf16_t hi = f2bf(v);
      hp |= (uint32_t)hi << (16 * e);
      lp |= (uint32_t)f2bf(v - bf2f(hi)) << (16 * e);
    }
    if (DPL == 2) {
      *(uint32_t*)&ohi[off] = hp;
      *(uint32_t*)&olo[off] = lp;
    } else {
      ohi[off] = (bf16_t)hp;
      olo[off] = (bf16_t)lp;
    }
  }
}

int attn_rows_per_block(int G, bool batched) {
  // decode / verify: one row per workgroup (one query vector per wave for G <= 4);
  // batched rows: 32 query vectors per workgroup share each K/V tile
  if (!batched) return 1;
  return G >= 32 ? 1 : 32 / G;
}

void attn_split(const AttnArgs& a, hipStream_t st) {
  if (a.max_len <= 0) return;
  const int ns = attn_nsplit(a.max_len, a.tiles);
  const int G = a.hq / a.hkv;
  const int nq = a.rows_per_block * G;
  dim3 grid(ns, a.hkv, (a.M + a.rows_per_block - 1) / a.rows_per_block);
#define KS_ATTN(HDV, BFV, QM)                                                                \
  hipLaunchKernelGGL((k_attn_split<HDV, BFV, QM>), grid, dim3(256), 0, st, a.M, a.hq, a.hkv, \
                     a.n_max, a.q, a.kc, a.vc, a.len, a.tiles, a.rows_per_block, a.part,     \
                     a.nsplit)
  if (a.hd == 128 && a.tiles > 1) {
    // batched rows: matrix-instruction kernel, 64 query vectors per workgroup
    const int span = TILE * a.tiles;
    dim3 g2((a.max_len + span - 1) / span, a.hkv, (a.M * G + 63) / 64);
    hipLaunchKernelGGL(k_attn_mfma<4>, g2, dim3(256), 0, st, a.M, a.hq, a.hkv, a.n_max, a.q,
                       (const bf16_t*)a.kc, (const bf16_t*)a.vc, a.len, span, a.part, a.nsplit);
  } else if (a.hd == 128) {
    if (nq <= 4) KS_ATTN(128, true, 1); else KS_ATTN(128, true, 8);
  } else {
    if (nq <= 4) KS_ATTN(64, false, 1); else KS_ATTN(64, false, 8);
  }
#undef KS_ATTN
}

void attn_combine(const AttnArgs& a, const float* kvself, Act act_out, hipStream_t st) {
  dim3 grid(a.M * a.hq);
  const int span = TILE * a.tiles;
  const bool bf = a.dtype == KS_BF16;
#define KS_COMB(HDV, BFV)                                                                    \
  hipLaunchKernelGGL((k_attn_combine<HDV, BFV>), grid, dim3(256), 0, st, a.M, a.hq, a.hkv,   \
                     span, a.q, a.part, a.nsplit, a.len, kvself,                             \
                     bf ? (bf16_t*)act_out.hi : nullptr, bf ? (bf16_t*)act_out.lo : nullptr, \
                     bf ? nullptr : (float*)act_out.hi, act_out.ld)
  if (a.hd == 128) KS_COMB(128, true);
  else KS_COMB(64, false);
#undef KS_COMB
}

}  // namespace ks
