// Row-wise kernels of the decode step: embedding gather, RMSNorm into the
// products' bf16 hi/lo activation planes, the per-head q/k normalisation +
// rotary embedding + KV store of q/k-normed models, cosine similarity
// (Section 2 of the paper), copies into the history ring, block copies, the
// rotary table and small fills.  (The greedy argmax lives with the other
// vocabulary reductions.)  All reductions use a fixed order so results are
// reproducible run to run and independent of how many rows a launch holds.
#include "ks_internal.h"

#include <cfloat>

namespace ks {

__device__ inline float wsum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ inline double wsum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// --------------------------------------------------------------- embedding
// 256 threads per row, 4 elements per thread per step (d % 4 == 0).
__global__ __launch_bounds__(256) void k_embed(const void* __restrict__ E, int bf,
                                               const int32_t* __restrict__ tok, int d,
                                               float* __restrict__ x, int ldx) {
  const int m = blockIdx.x;
  const size_t base = (size_t)tok[m] * d;
  float* xr = x + (size_t)m * ldx;
  for (int c = 4 * threadIdx.x; c < d; c += 1024) {
    float4 v;
    if (bf) {
      const uint2 u = *(const uint2*)((const bf16_t*)E + base + c);
      v = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                      __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
    } else {
      v = *(const float4*)((const float*)E + base + c);
    }
    *(float4*)(xr + c) = v;
  }
}

void embed_rows(const void* E, int dtype, const int32_t* tok, int M, int d, float* x, int ldx,
                hipStream_t st) {
  if (M <= 0) return;
  KS_LAUNCH(k_embed, dim3(M), dim3(256), 0, st, E, dtype == KS_BF16 ? 1 : 0, tok, d, x,
            ldx);
}

// Normed-product input (bf16 models): one block per row; thread c4 owns
// columns 4 c4..4 c4 + 3, four consecutive threads one 16-column tile whose
// sum of squares is a 2-step butterfly.  d % 16 == 0.
__global__ __launch_bounds__(256) void k_act_prep(const float* __restrict__ xin, int ldx,
                                                  const void* __restrict__ E, int bf,
                                                  const int32_t* __restrict__ tok, int d,
                                                  float* xout, const float* __restrict__ gain,
                                                  bf16_t* hi, bf16_t* lo, int lda, float* ssq,
                                                  PosFill pf) {
  const int m = blockIdx.x;
  if (pf.pos && threadIdx.x == 0) {
    const int p = pf.base + m % pf.r;
    pf.pos[m] = p;
    pf.len[m] = p + pf.len_add;
  }
  const size_t eb = E ? (size_t)tok[m] * d : 0;
  for (int c4 = threadIdx.x; c4 < (d >> 2); c4 += 256) {
    const int c = 4 * c4;
    float4 v;
    if (E) {
      if (bf) {
        const uint2 u = *(const uint2*)((const bf16_t*)E + eb + c);
        v = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                        __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
      } else {
        v = *(const float4*)((const float*)E + eb + c);
      }
      if (xout) *(float4*)(xout + (size_t)m * ldx + c) = v;
    } else {
      v = *(const float4*)(xin + (size_t)m * ldx + c);
    }
    const float4 g = *(const float4*)(gain + c);
    const float a[4] = {v.x * g.x, v.y * g.y, v.z * g.z, v.w * g.w};
    uint32_t h[2], l[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const bf16_t h0 = f2bf(a[2 * k]), h1 = f2bf(a[2 * k + 1]);
      h[k] = (uint32_t)h0 | ((uint32_t)h1 << 16);
      l[k] = (uint32_t)f2bf(a[2 * k] - bf2f(h0)) | ((uint32_t)f2bf(a[2 * k + 1] - bf2f(h1)) << 16);
    }
    *(uint2*)(hi + (size_t)m * lda + c) = make_uint2(h[0], h[1]);
    *(uint2*)(lo + (size_t)m * lda + c) = make_uint2(l[0], l[1]);
    float sq = v.x * v.x;
    sq = fmaf(v.y, v.y, sq);
    sq = fmaf(v.z, v.z, sq);
    sq = fmaf(v.w, v.w, sq);
    sq += __shfl_xor(sq, 1);
    sq += __shfl_xor(sq, 2);
    if ((threadIdx.x & 3) == 0) ssq[(size_t)m * (d >> 4) + (c >> 4)] = sq;
  }
}

void act_prep(const float* xin, int ldx, const void* E, int dtype, const int32_t* tok, int M,
              int d, float* xout, const float* gain, Act act, float* ssq, hipStream_t st,
              PosFill pf) {
  if (M <= 0) return;
  KS_LAUNCH(k_act_prep, dim3(M), dim3(256), 0, st, xin, ldx, E,
            dtype == KS_BF16 ? 1 : 0, tok, d, xout, gain, (bf16_t*)act.hi,
            (bf16_t*)act.lo, act.ld, ssq, pf);
}

// ---------------------------------------------------------------- RMSNorm
// One 256-thread block per row; a thread holds up to 4 float4 of the row
// (d <= 4096; wider rows take a strided loop).  Sum of squares: per-thread
// partials, wave butterfly, then the 4 wave sums added in order.
__global__ __launch_bounds__(256) void k_norm_act(const float* __restrict__ x, int ldx,
                                                  const float* __restrict__ g, float eps, int d,
                                                  int bf, void* ahi, void* alo, int lda) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const float* xr = x + (size_t)m * ldx;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int U = 4;
  float4 v[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int c = 4 * (threadIdx.x + 256 * u);
    v[u] = c < d ? *(const float4*)(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float scale = 1.0f;
  if (g) {
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u)
      s += v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w;
    for (int c = 4 * (threadIdx.x + 256 * U); c < d; c += 1024) {
      const float4 t = *(const float4*)(xr + c);
      s += t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) red[wave] = s;
    __syncthreads();
    scale = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
  }
  auto emit = [&](int c, float4 t) {
    float a[4] = {t.x, t.y, t.z, t.w};
    if (g) {
      const float4 gg = *(const float4*)(g + c);
      a[0] *= scale * gg.x; a[1] *= scale * gg.y; a[2] *= scale * gg.z; a[3] *= scale * gg.w;
    }
    const size_t off = (size_t)m * lda + c;
    if (bf) {
      uint32_t h[2], l[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const bf16_t h0 = f2bf(a[2 * k]), h1 = f2bf(a[2 * k + 1]);
        h[k] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        l[k] = (uint32_t)f2bf(a[2 * k] - bf2f(h0)) | ((uint32_t)f2bf(a[2 * k + 1] - bf2f(h1)) << 16);
      }
      *(uint2*)((bf16_t*)ahi + off) = make_uint2(h[0], h[1]);
      *(uint2*)((bf16_t*)alo + off) = make_uint2(l[0], l[1]);
    } else {
      *(float4*)((float*)ahi + off) = make_float4(a[0], a[1], a[2], a[3]);
    }
  };
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int c = 4 * (threadIdx.x + 256 * u);
    if (c < d) emit(c, v[u]);
  }
  for (int c = 4 * (threadIdx.x + 256 * U); c < d; c += 1024) emit(c, *(const float4*)(xr + c));
}

void norm_act(const float* x, int ldx, const float* g, float eps, int M, int d, int dtype,
              Act act, hipStream_t st) {
  if (M <= 0) return;
  KS_LAUNCH(k_norm_act, dim3(M), dim3(256), 0, st, x, ldx, g, eps, d,
            dtype == KS_BF16 ? 1 : 0, act.hi, act.lo, act.ld);
}

// ------------------------------------------------------- q/k norm, RoPE, KV
// One block per row; one wave per head at a time; lane f < hd/2 owns the
// rotary pair (f, f + hd/2).
__global__ __launch_bounds__(256) void k_qkv_post(QkvPostArgs a) {
  const int m = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int hd = a.hd, half = hd / 2;
  const int nh = a.hq + 2 * a.hkv;
  const int hh = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (hh >= nh) return;
  const int pos = a.pos[m];
  const bool act = lane < half;
  const float* src_row = a.qkv + (size_t)m * nh * hd;
  float c = 1.f, s = 0.f;
  if (act && hh < a.hq + a.hkv) {
    const float2 cs = *(const float2*)&a.rope_cs[((size_t)pos * half + lane) * 2];
    c = cs.x;
    s = cs.y;
  }
  {
    const float* src = src_row + (size_t)hh * hd;
    const int c0 = a.perm ? qkv_perm(lane, hd) : lane;
    const int c1 = a.perm ? qkv_perm(lane + half, hd) : lane + half;
    float x0 = act ? src[c0] : 0.f;
    float x1 = act ? src[c1] : 0.f;
    float y0 = x0, y1 = x1;
    if (hh < a.hq + a.hkv) {
      if (a.qk_norm) {
        const float ss = wsum(x0 * x0 + x1 * x1);
        const float sc = 1.0f / sqrtf(ss / (float)hd + a.eps);
        const float* gn = hh < a.hq ? a.q_norm : a.k_norm;
        if (act) {
          x0 = x0 * sc * gn[lane];
          x1 = x1 * sc * gn[lane + half];
        }
      }
      y0 = x0 * c - x1 * s;
      y1 = x1 * c + x0 * s;
    }
    if (!act) return;
    if (hh < a.hq) {
      float* q = a.q_out + ((size_t)m * a.hq + hh) * hd;
      q[lane] = y0;
      q[lane + half] = y1;
      return;
    }
    const int kv = hh < a.hq + a.hkv ? 0 : 1;
    const int kvh = hh - a.hq - kv * a.hkv;
    if (a.mode == 0) {
      const size_t off = ((size_t)kvh * a.n_max + pos) * hd;
      void* base = kv ? a.vc : a.kc;
      if (a.dtype == KS_BF16) {
        ((bf16_t*)base)[off + lane] = f2bf(y0);
        ((bf16_t*)base)[off + lane + half] = f2bf(y1);
      } else {
        ((float*)base)[off + lane] = y0;
        ((float*)base)[off + lane + half] = y1;
      }
    } else {
      float* dst = a.kvself + (((size_t)m * 2 + kv) * a.hkv + kvh) * hd;
      if (a.dtype == KS_BF16) {
        y0 = bf2f(f2bf(y0));
        y1 = bf2f(f2bf(y1));
      }
      dst[lane] = y0;
      dst[lane + half] = y1;
    }
  }
}

void qkv_post(const QkvPostArgs& a, hipStream_t st) {
  if (a.M <= 0) return;
  const int nh = a.hq + 2 * a.hkv;
  KS_LAUNCH(k_qkv_post, dim3((nh + 3) / 4, a.M), dim3(256), 0, st, a);
}

// ------------------------------------------------------------------ argmax
// One pass per element: running (max, first index of max, sum of exp(v - max))
// per thread over a fixed strided order, then a fixed tree.  Larger value
// wins; equal values keep the lower index.
// ------------------------------------------------------------------ cosine
// One wave per row: <x, y>, |x|^2, |y|^2 accumulated in float64 (every
// float32 product is exact in float64).  Rows of a multiple of 4 floats at
// 16-byte aligned addresses are read as float4, four loads in flight per lane.
__device__ inline void cos_acc4(const float4 a, const float4 b, double& xy, double& xx,
                                double& yy) {
  const double a0 = a.x, a1 = a.y, a2 = a.z, a3 = a.w;
  const double b0 = b.x, b1 = b.y, b2 = b.z, b3 = b.w;
  xy += a0 * b0 + a1 * b1 + a2 * b2 + a3 * b3;
  xx += a0 * a0 + a1 * a1 + a2 * a2 + a3 * a3;
  yy += b0 * b0 + b1 * b1 + b2 * b2 + b3 * b3;
}

__device__ inline double row_cos(const float* x, const float* y, int d, int lane) {
  double xy = 0.0, xx = 0.0, yy = 0.0;
  if ((d & 3) == 0 && (((uintptr_t)x | (uintptr_t)y) & 15) == 0) {
    const float4* x4 = (const float4*)x;
    const float4* y4 = (const float4*)y;
    const int n4 = d >> 2;
    int c = lane;
    for (; c + 192 < n4; c += 256) {
      const float4 a0 = x4[c], a1 = x4[c + 64], a2 = x4[c + 128], a3 = x4[c + 192];
      const float4 b0 = y4[c], b1 = y4[c + 64], b2 = y4[c + 128], b3 = y4[c + 192];
      cos_acc4(a0, b0, xy, xx, yy);
      cos_acc4(a1, b1, xy, xx, yy);
      cos_acc4(a2, b2, xy, xx, yy);
      cos_acc4(a3, b3, xy, xx, yy);
    }
    for (; c < n4; c += 64) cos_acc4(x4[c], y4[c], xy, xx, yy);
  } else {
    for (int c = lane; c < d; c += 64) {
      const double a = x[c], b = y[c];
      xy += a * b;
      xx += a * a;
      yy += b * b;
    }
  }
  xy = wsum_d(xy);
  xx = wsum_d(xx);
  yy = wsum_d(yy);
  const double den = sqrt(xx) * sqrt(yy);
  return den > 0.0 ? xy / den : 0.0;
}

// One 1024-thread block per group; rows round-robin over the 16 waves; the
// mean is summed by one thread in row order.
template <typename OutT>
__global__ __launch_bounds__(1024) void k_cos_groups(const float* __restrict__ X,
                                                     const float* __restrict__ Y, int r, int d,
                                                     OutT* out) {
  extern __shared__ double cs[];
  const int g = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int t = wave; t < r; t += 16) {
    const double c = row_cos(X + ((size_t)g * r + t) * d, Y + (size_t)t * d, d, lane);
    if (lane == 0) cs[t] = c;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int t = 0; t < r; ++t) s += cs[t];
    out[g] = (OutT)(s / r);
  }
}

void cos_groups(const float* X, const float* Y, int groups, int r, int d, float* out,
                hipStream_t st) {
  if (groups <= 0) return;
  KS_LAUNCH(k_cos_groups<float>, dim3(groups), dim3(1024), r * sizeof(double), st, X,
            Y, r, d, out);
}

void cos_groups_f64(const float* X, const float* Y, int groups, int r, int d, double* out,
                    hipStream_t st) {
  if (groups <= 0) return;
  KS_LAUNCH(k_cos_groups<double>, dim3(groups), dim3(1024), r * sizeof(double), st, X,
            Y, r, d, out);
}

__global__ __launch_bounds__(256) void k_cos_rows(const float* __restrict__ X,
                                                  const float* __restrict__ Y, int rows, int ry,
                                                  int d, double* out) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= rows) return;
  const double c = row_cos(X + (size_t)t * d, Y + (size_t)(t % ry) * d, d, lane);
  if (lane == 0) out[t] = c;
}

void cos_rows(const float* X, const float* Y, int rows, int ry, int d, double* out,
              hipStream_t st) {
  if (rows <= 0) return;
  KS_LAUNCH(k_cos_rows, dim3((rows + 3) / 4), dim3(256), 0, st, X, Y, rows, ry, d, out);
}

// Both candidate sets of a DP stage in one launch: rows t < rows of X1 into
// out1, of X2 into out2, each against Y row t % ry.
__global__ __launch_bounds__(256) void k_cos_rows2(const float* __restrict__ X1,
                                                   const float* __restrict__ X2,
                                                   const float* __restrict__ Y, int rows, int ry,
                                                   int d, double* out1, double* out2) {
  const int lane = threadIdx.x & 63;
  const int t2 = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t2 >= 2 * rows) return;
  const bool second = t2 >= rows;
  const int t = second ? t2 - rows : t2;
  const double c = row_cos((second ? X2 : X1) + (size_t)t * d, Y + (size_t)(t % ry) * d, d, lane);
  if (lane == 0) (second ? out2 : out1)[t] = c;
}

void cos_rows2(const float* X1, const float* X2, const float* Y, int rows, int ry, int d,
               double* out1, double* out2, hipStream_t st) {
  if (rows <= 0) return;
  KS_LAUNCH(k_cos_rows2, dim3((2 * rows + 3) / 4), dim3(256), 0, st, X1, X2, Y, rows,
            ry, d, out1, out2);
}

// ------------------------------------------------------------------- copies
// dst[i][0..n) = src[i][0..n) for pointer tables of length cnt; a null
// source marks an unused entry.
__global__ void k_copy_blocks(const float* const* src, float* const* dst, size_t n) {
  const int i = blockIdx.y;
  const float* s = src[i];
  float* d = dst[i];
  if (s == nullptr) return;
  for (size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c < n;
       c += (size_t)gridDim.x * blockDim.x)
    d[c] = s[c];
}

void copy_rows(const float* const* src, float* const* dst, int cnt, int n, hipStream_t st) {
  if (cnt <= 0 || n <= 0) return;
  const int bx = (n + 255) / 256 < 64 ? (n + 255) / 256 : 64;
  KS_LAUNCH(k_copy_blocks, dim3(bx, cnt), dim3(256), 0, st, src, dst, (size_t)n);
}

// History ring copies, one launch for every plane: row t < n of plane i,
// plane[i][t] at flat + (i * plane_stride + t) * d, pairs with ring row
// ring + (i * RING + (p0 + t) % RING) * d.
__global__ __launch_bounds__(256) void k_ring_copy(const float* __restrict__ src,
                                                   float* __restrict__ dst, size_t plane_stride,
                                                   int RING, int p0, int d, int to_ring) {
  const int t = blockIdx.x, i = blockIdx.y;
  const size_t flat = ((size_t)i * plane_stride + t) * d;
  const size_t ring = ((size_t)i * RING + (p0 + t) % RING) * d;
  const float4* s4 = (const float4*)(src + (to_ring ? flat : ring));
  float4* d4 = (float4*)(dst + (to_ring ? ring : flat));
  for (int c = threadIdx.x; c < d / 4; c += 256) d4[c] = s4[c];
}

void ring_copy(const float* src, float* dst, size_t plane_stride, int planes, int n, int RING,
               int p0, int d, bool to_ring, hipStream_t st) {
  if (n <= 0 || planes <= 0) return;
  KS_LAUNCH(k_ring_copy, dim3(n, planes), dim3(256), 0, st, src, dst, plane_stride,
            RING, p0, d, to_ring ? 1 : 0);
}

// ------------------------------------------------------------ rotary table
__global__ void k_rope_table(float* cs, int n_max, int hd, double theta) {
  const int half = hd / 2;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)n_max * half) return;
  const int p = (int)(i / half), f = (int)(i % half);
  const double inv = pow(theta, -2.0 * f / hd);
  const double ang = (double)p * inv;
  cs[2 * i] = (float)cos(ang);
  cs[2 * i + 1] = (float)sin(ang);
}

void rope_table(float* cs, int n_max, int hd, double theta, hipStream_t st) {
  const size_t n = (size_t)n_max * (hd / 2);
  KS_LAUNCH(k_rope_table, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, cs,
            n_max, hd, theta);
}

// --------------------------------------------------------- small fillers
// pos[c*r + t] = base + t, len[.] = pos + len_add, for c < cells.
__global__ void k_fill_pos(int32_t* pos, int32_t* len, int base, int r, int total, int len_add) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int p = base + (i % r);
  pos[i] = p;
  len[i] = p + len_add;
}

void fill_pos(int32_t* pos, int32_t* len, int base, int r, int total, int len_add,
              hipStream_t st) {
  if (total <= 0) return;
  KS_LAUNCH(k_fill_pos, dim3((total + 255) / 256), dim3(256), 0, st, pos, len, base, r,
            total, len_add);
}

__global__ void k_set_i32(int32_t* p, int v) { *p = v; }

void set_i32(int32_t* p, int v, hipStream_t st) {
  KS_LAUNCH(k_set_i32, dim3(1), dim3(1), 0, st, p, v);
}

}  // namespace ks
