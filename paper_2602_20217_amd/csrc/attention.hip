// GQA decode attention over a contiguous KV cache, split over the context.
//
// Grid: (split, kv head, row group).  A workgroup stages one 128-position tile
// of K and V for its kv head in LDS at a time (bf16 pairs packed in 32-bit
// words, K rows padded by one word so that 64 lanes reading 64 different keys
// hit 64 different banks) and applies it to every query vector of its row
// group: the G = hq/hkv query heads of each row share the tile.  Each wave owns
// a fixed set of query vectors and keeps their running max, running sum and
// unnormalised output in registers (online softmax across the tiles of a
// split); a lane scores two keys, and the output accumulation broadcasts each
// probability with a lane read.  The partial (o, max, sum) of each
// (row, query head, split) goes to memory and a second kernel merges the
// splits in ascending order.
//
// A row's arithmetic depends only on its own query, its length and the split
// size, never on the other rows of the launch, so the decode step and a verify
// row at the same position produce the same bits.
#include "ks_internal.h"

#include <cfloat>

namespace ks {

constexpr int TILE = 128;
constexpr int QMAX = 16;  // query vectors per wave (rows_per_block * G <= 64)

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

int attn_nsplit(int n_positions, int tiles) {
  const int span = TILE * tiles;
  return (n_positions + span - 1) / span;
}

// HD: head dim (64 or 128).  BF: cache holds bf16 (else float32).
template <int HD, bool BF>
__global__ __launch_bounds__(256) void k_attn_split(int M, int hq, int hkv, int n_max,
                                                    const float* __restrict__ q,
                                                    const void* __restrict__ kc,
                                                    const void* __restrict__ vc,
                                                    const int32_t* __restrict__ len, int tiles,
                                                    int rows_per_block,
                                                    float* __restrict__ part, int nsplit) {
  constexpr int KW = BF ? HD / 2 : HD;  // 32-bit words per key row
  constexpr int DPL = HD / 64;          // output dims per lane (1 or 2)
  __shared__ uint32_t Ks[TILE][KW + 1];
  __shared__ uint32_t Vs[TILE][KW];
  __shared__ int s_maxlen;

  const int split = blockIdx.x, kvh = blockIdx.y;
  const int r0 = blockIdx.z * rows_per_block;
  const int r1 = min(M, r0 + rows_per_block);
  const int G = hq / hkv;
  const int nq = (r1 - r0) * G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int start = split * tiles * TILE;
  const float scale = 1.0f / sqrtf((float)HD);

  if (threadIdx.x == 0) {
    int mx = 0;
    for (int r = r0; r < r1; ++r) mx = max(mx, len[r]);
    s_maxlen = mx;
  }
  __syncthreads();
  const int maxlen = s_maxlen;
  if (start >= maxlen) return;

  float o[QMAX][DPL];
  float mrun[QMAX], lrun[QMAX];
#pragma unroll
  for (int j = 0; j < QMAX; ++j) {
    mrun[j] = -FLT_MAX;
    lrun[j] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[j][e] = 0.f;
  }

  const size_t head_off = (size_t)kvh * n_max * HD;
  for (int tile = 0; tile < tiles; ++tile) {
    const int t0 = start + tile * TILE;
    if (t0 >= maxlen) break;
    const int cnt = min(TILE, maxlen - t0);
    // stage K and V rows [t0, t0 + cnt): 16-byte chunks, HD*es/16 per row
    constexpr int CPR = KW / 4;  // 16-byte chunks per row
    for (int c = threadIdx.x; c < cnt * CPR; c += 256) {
      const int row = c / CPR, ch = c % CPR;
      const uint32_t* ksrc;
      const uint32_t* vsrc;
      if (BF) {
        ksrc = (const uint32_t*)((const bf16_t*)kc + head_off + (size_t)(t0 + row) * HD) + ch * 4;
        vsrc = (const uint32_t*)((const bf16_t*)vc + head_off + (size_t)(t0 + row) * HD) + ch * 4;
      } else {
        ksrc = (const uint32_t*)((const float*)kc + head_off + (size_t)(t0 + row) * HD) + ch * 4;
        vsrc = (const uint32_t*)((const float*)vc + head_off + (size_t)(t0 + row) * HD) + ch * 4;
      }
      const uint4 kv4 = *(const uint4*)ksrc;
      const uint4 vv4 = *(const uint4*)vsrc;
      Ks[row][ch * 4 + 0] = kv4.x;
      Ks[row][ch * 4 + 1] = kv4.y;
      Ks[row][ch * 4 + 2] = kv4.z;
      Ks[row][ch * 4 + 3] = kv4.w;
      *(uint4*)&Vs[row][ch * 4] = vv4;
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
      // scores of keys lane and lane + 64
      float s0 = 0.f, s1 = 0.f;
      if (BF) {
#pragma unroll 8
        for (int w = 0; w < KW; ++w) {
          const float qa = qv[2 * w], qb = qv[2 * w + 1];
          const uint32_t k0 = Ks[lane][w], k1 = Ks[lane + 64][w];
          s0 = fmaf(qa, bf2f((bf16_t)(k0 & 0xFFFF)), s0);
          s0 = fmaf(qb, bf2f((bf16_t)(k0 >> 16)), s0);
          s1 = fmaf(qa, bf2f((bf16_t)(k1 & 0xFFFF)), s1);
          s1 = fmaf(qb, bf2f((bf16_t)(k1 >> 16)), s1);
        }
      } else {
#pragma unroll 8
        for (int w = 0; w < KW; ++w) {
          const float qa = qv[w];
          s0 = fmaf(qa, __uint_as_float(Ks[lane][w]), s0);
          s1 = fmaf(qa, __uint_as_float(Ks[lane + 64][w]), s1);
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
      for (int t = 0; t < n0; ++t) {
        const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p0), t));
        if (BF) {
          const uint32_t vw = Vs[t][lane];
          acc[0] = fmaf(pt, bf2f((bf16_t)(vw & 0xFFFF)), acc[0]);
          acc[DPL - 1] = DPL == 2 ? fmaf(pt, bf2f((bf16_t)(vw >> 16)), acc[DPL - 1]) : acc[DPL - 1];
        } else {
          acc[0] = fmaf(pt, __uint_as_float(Vs[t][lane]), acc[0]);
        }
      }
      for (int t = 64; t < vcnt; ++t) {
        const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p1), t - 64));
        if (BF) {
          const uint32_t vw = Vs[t][lane];
          acc[0] = fmaf(pt, bf2f((bf16_t)(vw & 0xFFFF)), acc[0]);
          acc[DPL - 1] = DPL == 2 ? fmaf(pt, bf2f((bf16_t)(vw >> 16)), acc[DPL - 1]) : acc[DPL - 1];
        } else {
          acc[0] = fmaf(pt, __uint_as_float(Vs[t][lane]), acc[0]);
        }
      }
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] = o[j][e] * alpha + acc[e];
    }
    __syncthreads();
  }

  // write partials of rows that have keys in this split
#pragma unroll
  for (int j = 0; j < QMAX; ++j) {
    const int qi = wave + 4 * j;
    if (qi >= nq) break;
    const int r = r0 + qi / G;
    const int h = kvh * G + qi % G;
    if (len[r] <= start) continue;
    float* dst = part + (((size_t)r * hq + h) * nsplit + split) * (HD + 2);
    if (BF) {
      // lane owns dims 2*lane, 2*lane+1 (bf16 pair order within the packed word)
      if (DPL == 2) {
        dst[2 * lane] = o[j][0];
        dst[2 * lane + 1] = o[j][DPL - 1];
      } else {
        // HD = 64 with bf16: lanes 0..31 own pairs; never instantiated by the engine
        if (lane < 32) dst[lane] = o[j][0];
      }
    } else {
      for (int e = 0; e < DPL; ++e) dst[lane + 64 * e] = o[j][e];
    }
    if (lane == 0) {
      dst[HD] = mrun[j];
      dst[HD + 1] = lrun[j];
    }
  }
}

// One wave per (row, query head).  Output dims: bf16 caches use lane -> dims
// (2 lane, 2 lane + 1); float32 caches use lane -> dims (lane, lane + 64).
template <int HD, bool BF>
__global__ __launch_bounds__(256) void k_attn_combine(int M, int hq, int hkv, int span,
                                                      const float* __restrict__ q,
                                                      const float* __restrict__ part, int nsplit,
                                                      const int32_t* __restrict__ len,
                                                      const float* __restrict__ kvself,
                                                      bf16_t* ohi, bf16_t* olo, float* of,
                                                      int ldact) {
  constexpr int DPL = HD / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gid = blockIdx.x * 4 + wave;
  if (gid >= M * hq) return;
  const int r = gid / hq, h = gid % hq;
  const int G = hq / hkv;
  const int kvh = h / G;
  const int L = len[r];
  const int ns = (L + span - 1) / span;
  const float* pr = part + ((size_t)r * hq + h) * nsplit * (HD + 2);
  int dims[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) dims[e] = BF ? 2 * lane + e : lane + 64 * e;

  float mx = -FLT_MAX;
  for (int s = 0; s < ns; ++s) mx = fmaxf(mx, pr[(size_t)s * (HD + 2) + HD]);
  float sself = 0.f;
  const float* ks = nullptr;
  const float* vs = nullptr;
  if (kvself) {
    ks = kvself + (((size_t)r * 2 + 0) * hkv + kvh) * HD;
    vs = kvself + (((size_t)r * 2 + 1) * hkv + kvh) * HD;
    const float* qv = q + ((size_t)r * hq + h) * HD;
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) d = fmaf(qv[dims[e]], ks[dims[e]], d);
    sself = wave_sum(d) * (1.0f / sqrtf((float)HD));
    mx = fmaxf(mx, sself);
  }
  float lsum = 0.f, acc[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float* ps = pr + (size_t)s * (HD + 2);
    const float w = __expf(ps[HD] - mx);
    lsum = fmaf(ps[HD + 1], w, lsum);
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = fmaf(ps[dims[e]], w, acc[e]);
  }
  if (kvself) {
    const float w = __expf(sself - mx);
    lsum += w;
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = fmaf(vs[dims[e]], w, acc[e]);
  }
  const float inv = 1.0f / lsum;
#pragma unroll
  for (int e = 0; e < DPL; ++e) {
    const float v = acc[e] * inv;
    const size_t off = (size_t)r * ldact + (size_t)h * HD + dims[e];
    if (of) {
      of[off] = v;
    } else {
      const bf16_t hi = f2bf(v);
      ohi[off] = hi;
      olo[off] = f2bf(v - bf2f(hi));
    }
  }
}

void attn_split(const AttnArgs& a, hipStream_t st) {
  if (a.max_len <= 0) return;
  const int ns = attn_nsplit(a.max_len, a.tiles);
  dim3 grid(ns, a.hkv, (a.M + a.rows_per_block - 1) / a.rows_per_block);
#define KS_ATTN(HDV, BFV)                                                                   \
  hipLaunchKernelGGL((k_attn_split<HDV, BFV>), grid, dim3(256), 0, st, a.M, a.hq, a.hkv,    \
                     a.n_max, a.q, a.kc, a.vc, a.len, a.tiles, a.rows_per_block, a.part,    \
                     a.nsplit)
  if (a.hd == 128) {
    if (a.dtype == KS_BF16) KS_ATTN(128, true); else KS_ATTN(128, false);
  } else {
    KS_ATTN(64, false);
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
  if (a.hd == 128) {
    if (bf) KS_COMB(128, true); else KS_COMB(128, false);
  } else {
    KS_COMB(64, false);
  }
#undef KS_COMB
}

}  // namespace ks
