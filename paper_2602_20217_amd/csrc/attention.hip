// GQA decode attention over a contiguous KV cache, split over the context.
//
// Grid: (split, kv head, row group).  A workgroup owns `tiles` consecutive
// 128-position tiles of one kv head.  Every thread issues its share of a
// tile's K and V loads at once (16-byte chunks, all in flight together) and
// stores them to LDS after one wait.  K rows are padded by four 32-bit words
// so that 16-byte LDS reads of 64 different rows cover all banks.  Each wave
// owns a fixed set of query vectors (the G = hq/hkv query heads of a row share
// the tile); a lane scores two keys, softmax statistics use wave shuffles, and
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

constexpr int TILE = 128;

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
      float s0 = 0.f, s1 = 0.f;
      const uint32_t* k0p = &Ks[lane * KS];
      const uint32_t* k1p = &Ks[(lane + 64) * KS];
#pragma unroll 4
      for (int w4 = 0; w4 < KW / 4; ++w4) {
        const uint4 a = *(const uint4*)(k0p + 4 * w4);
        const uint4 b = *(const uint4*)(k1p + 4 * w4);
        if (BF) {
          const float* qq = qv + 8 * w4;
          s0 = fmaf(qq[0], lo16(a.x), s0); s0 = fmaf(qq[1], hi16(a.x), s0);
          s0 = fmaf(qq[2], lo16(a.y), s0); s0 = fmaf(qq[3], hi16(a.y), s0);
          s0 = fmaf(qq[4], lo16(a.z), s0); s0 = fmaf(qq[5], hi16(a.z), s0);
          s0 = fmaf(qq[6], lo16(a.w), s0); s0 = fmaf(qq[7], hi16(a.w), s0);
          s1 = fmaf(qq[0], lo16(b.x), s1); s1 = fmaf(qq[1], hi16(b.x), s1);
          s1 = fmaf(qq[2], lo16(b.y), s1); s1 = fmaf(qq[3], hi16(b.y), s1);
          s1 = fmaf(qq[4], lo16(b.z), s1); s1 = fmaf(qq[5], hi16(b.z), s1);
          s1 = fmaf(qq[6], lo16(b.w), s1); s1 = fmaf(qq[7], hi16(b.w), s1);
        } else {
          const float* qq = qv + 4 * w4;
          s0 = fmaf(qq[0], __uint_as_float(a.x), s0); s0 = fmaf(qq[1], __uint_as_float(a.y), s0);
          s0 = fmaf(qq[2], __uint_as_float(a.z), s0); s0 = fmaf(qq[3], __uint_as_float(a.w), s0);
          s1 = fmaf(qq[0], __uint_as_float(b.x), s1); s1 = fmaf(qq[1], __uint_as_float(b.y), s1);
          s1 = fmaf(qq[2], __uint_as_float(b.z), s1); s1 = fmaf(qq[3], __uint_as_float(b.w), s1);
        }
      }
      s0 = lane < vcnt ? s0 * scale : -FLT_MAX;
      s1 = lane + 64 < vcnt ? s1 * scale : -FLT_MAX;
      const float mt = wave_max(fmaxf(s0, s1));
      const float mnew = fmaxf(mrun[j], mt);
      const float alpha = __expf(mrun[j] - mnew);
      const float p0 = lane < vcnt ? __expf(s0 - mnew) : 0.f;
      const float p1 = lane + 64 < vcnt ? __expf(s1 - mnew) : 0.f;
      lrun[j] = lrun[j] * alpha + wave_sum(p0 + p1);
      mrun[j] = mnew;
      float acc[DPL];
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
      const int n0 = min(vcnt, 64);
#pragma unroll 8
      for (int t = 0; t < n0; ++t) {
        const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p0), t));
        const uint32_t vw = Vs[t * KW + lane];
        if (BF) {
          acc[0] = fmaf(pt, lo16(vw), acc[0]);
          acc[DPL - 1] = fmaf(pt, hi16(vw), acc[DPL - 1]);
        } else {
          acc[0] = fmaf(pt, __uint_as_float(vw), acc[0]);
        }
      }
#pragma unroll 8
      for (int t = 64; t < vcnt; ++t) {
        const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p1), t - 64));
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

// One wave per (row, query head); output dims lane -> (2 lane, 2 lane + 1) for
// bf16 caches, lane for float32 caches.  The split maxima are reduced across
// lanes, then the splits are merged in ascending order (loads of different
// splits are independent, so they are in flight together).
template <int HD, bool BF>
__global__ __launch_bounds__(256) void k_attn_combine(int M, int hq, int hkv, int span,
                                                      const float* __restrict__ q,
                                                      const float* __restrict__ part, int nsplit,
                                                      const int32_t* __restrict__ len,
                                                      const float* __restrict__ kvself,
                                                      bf16_t* ohi, bf16_t* olo, float* of,
                                                      int ldact) {
  constexpr int DPL = HD / 64;
  const int lane = threadIdx.x & 63;
  const int gid = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  if (gid >= M * hq) return;
  const int r = gid / hq, h = gid % hq;
  const int G = hq / hkv;
  const int kvh = h / G;
  const int L = len[r];
  const int ns = (L + span - 1) / span;
  const float* pr = part + ((size_t)r * hq + h) * nsplit * (HD + 2);
  const int d0 = BF ? 2 * lane : lane;

  float mloc = -FLT_MAX;
  for (int s = lane; s < ns; s += 64) mloc = fmaxf(mloc, pr[(size_t)s * (HD + 2) + HD]);
  float mx = wave_max(mloc);
  float sself = 0.f;
  const float* ks = nullptr;
  const float* vs = nullptr;
  if (kvself) {
    ks = kvself + (((size_t)r * 2 + 0) * hkv + kvh) * HD;
    vs = kvself + (((size_t)r * 2 + 1) * hkv + kvh) * HD;
    const float* qv = q + ((size_t)r * hq + h) * HD;
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) d = fmaf(qv[d0 + e], ks[d0 + e], d);
    sself = wave_sum(d) * (1.0f / sqrtf((float)HD));
    mx = fmaxf(mx, sself);
  }
  float lsum = 0.f, acc[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
#pragma unroll 8
  for (int s = 0; s < ns; ++s) {
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
  if (kvself) {
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
  if (a.hd == 128) {
    if (nq <= 4) KS_ATTN(128, true, 1); else KS_ATTN(128, true, 8);
  } else {
    if (nq <= 4) KS_ATTN(64, false, 1); else KS_ATTN(64, false, 8);
  }
#undef KS_ATTN
}

void attn_combine(const AttnArgs& a, const float* kvself, Act act_out, hipStream_t st) {
  dim3 grid((a.M * a.hq + 3) / 4);
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
