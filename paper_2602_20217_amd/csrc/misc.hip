// Row-wise kernels of the decode step: embedding gather, RMSNorm into matrix
// activations, q/k normalisation + rotary embedding + KV store, greedy argmax
// with top-1 probability, cosine similarity (Section 2 of the paper), row
// copies and the rotary table.  All reductions use a fixed order so results
// are reproducible run to run and independent of how many rows a launch holds.
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
__global__ void k_embed(const void* __restrict__ E, int bf, const int32_t* __restrict__ tok,
                        int d, float* __restrict__ x, int ldx) {
  const int m = blockIdx.x;
  const size_t base = (size_t)tok[m] * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    const float v = bf ? bf2f(((const bf16_t*)E)[base + c]) : ((const float*)E)[base + c];
    x[(size_t)m * ldx + c] = v;
  }
}

void embed_rows(const void* E, int dtype, const int32_t* tok, int M, int d, float* x, int ldx,
                hipStream_t st) {
  if (M <= 0) return;
  hipLaunchKernelGGL(k_embed, dim3(M), dim3(256), 0, st, E, dtype == KS_BF16 ? 1 : 0, tok, d, x,
                     ldx);
}

// ---------------------------------------------------------------- RMSNorm
// One 256-thread block per row.  Sum of squares: per-thread strided partial
// sums, then a fixed tree over the block.
__global__ __launch_bounds__(256) void k_norm_act(const float* __restrict__ x, int ldx,
                                                  const float* __restrict__ g, float eps, int d,
                                                  int bf, void* ahi, void* alo, int lda) {
  __shared__ float red[256];
  const int m = blockIdx.x;
  const float* xr = x + (size_t)m * ldx;
  float scale = 1.0f;
  if (g) {
    float s = 0.f;
    for (int c = threadIdx.x; c < d; c += 256) s = fmaf(xr[c], xr[c], s);
    red[threadIdx.x] = s;
    __syncthreads();
    for (int o = 128; o >= 1; o >>= 1) {
      if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
      __syncthreads();
    }
    scale = 1.0f / sqrtf(red[0] / (float)d + eps);
  }
  for (int c = threadIdx.x; c < d; c += 256) {
    const float a = g ? xr[c] * scale * g[c] : xr[c];
    const size_t off = (size_t)m * lda + c;
    if (bf) {
      const bf16_t h = f2bf(a);
      ((bf16_t*)ahi)[off] = h;
      ((bf16_t*)alo)[off] = f2bf(a - bf2f(h));
    } else {
      ((float*)ahi)[off] = a;
    }
  }
}

void norm_act(const float* x, int ldx, const float* g, float eps, int M, int d, int dtype,
              Act act, hipStream_t st) {
  if (M <= 0) return;
  hipLaunchKernelGGL(k_norm_act, dim3(M), dim3(256), 0, st, x, ldx, g, eps, d,
                     dtype == KS_BF16 ? 1 : 0, act.hi, act.lo, act.ld);
}

// ------------------------------------------------------- q/k norm, RoPE, KV
// One block per row; one wave per head at a time; lane f < hd/2 owns the
// rotary pair (f, f + hd/2).
__global__ __launch_bounds__(256) void k_qkv_post(QkvPostArgs a) {
  const int m = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hd = a.hd, half = hd / 2;
  const int nh = a.hq + 2 * a.hkv;
  const int pos = a.pos[m];
  const bool act = lane < half;
  const float* src_row = a.qkv + (size_t)m * nh * hd;
  float c = 1.f, s = 0.f;
  if (act) {
    c = a.rope_cs[((size_t)pos * half + lane) * 2];
    s = a.rope_cs[((size_t)pos * half + lane) * 2 + 1];
  }
  for (int hh = wave; hh < nh; hh += 4) {
    const float* src = src_row + (size_t)hh * hd;
    float x0 = act ? src[lane] : 0.f;
    float x1 = act ? src[lane + half] : 0.f;
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
    if (!act) continue;
    if (hh < a.hq) {
      float* q = a.q_out + ((size_t)m * a.hq + hh) * hd;
      q[lane] = y0;
      q[lane + half] = y1;
      continue;
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
  hipLaunchKernelGGL(k_qkv_post, dim3(a.M), dim3(256), 0, st, a);
}

// ------------------------------------------------------------------ argmax
// Larger value wins; equal values keep the lower index.
__global__ __launch_bounds__(1024) void k_argmax(const float* __restrict__ logits, int V,
                                                 int32_t* am, float* top1) {
  __shared__ float sv[1024];
  __shared__ int si[1024];
  const int m = blockIdx.x;
  const float* row = logits + (size_t)m * V;
  float bv = -FLT_MAX;
  int bi = 0x7FFFFFFF;
  for (int i = threadIdx.x; i < V; i += 1024) {
    const float v = row[i];
    if (v > bv) {
      bv = v;
      bi = i;
    }
  }
  sv[threadIdx.x] = bv;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int o = 512; o >= 1; o >>= 1) {
    if (threadIdx.x < o) {
      const float v2 = sv[threadIdx.x + o];
      const int i2 = si[threadIdx.x + o];
      if (v2 > sv[threadIdx.x] || (v2 == sv[threadIdx.x] && i2 < si[threadIdx.x])) {
        sv[threadIdx.x] = v2;
        si[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  const float mx = sv[0];
  const int arg = si[0];
  __syncthreads();
  float s = 0.f;
  for (int i = threadIdx.x; i < V; i += 1024) s += __expf(row[i] - mx);
  sv[threadIdx.x] = s;
  __syncthreads();
  for (int o = 512; o >= 1; o >>= 1) {
    if (threadIdx.x < o) sv[threadIdx.x] += sv[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    am[m] = arg;
    if (top1) top1[m] = 1.0f / sv[0];
  }
}

void argmax_rows(const float* logits, int M, int V, int32_t* am, float* top1, hipStream_t st) {
  if (M <= 0) return;
  hipLaunchKernelGGL(k_argmax, dim3(M), dim3(1024), 0, st, logits, V, am, top1);
}

// ------------------------------------------------------------------ cosine
// One wave per row: <x, y>, |x|^2, |y|^2 accumulated in float64.
__device__ inline double row_cos(const float* x, const float* y, int d, int lane) {
  double xy = 0.0, xx = 0.0, yy = 0.0;
  for (int c = lane; c < d; c += 64) {
    const double a = x[c], b = y[c];
    xy += a * b;
    xx += a * a;
    yy += b * b;
  }
  xy = wsum_d(xy);
  xx = wsum_d(xx);
  yy = wsum_d(yy);
  const double den = sqrt(xx) * sqrt(yy);
  return den > 0.0 ? xy / den : 0.0;
}

// One 256-thread block per group; rows round-robin over the 4 waves; the mean
// is summed by one thread in row order.
template <typename OutT>
__global__ __launch_bounds__(256) void k_cos_groups(const float* __restrict__ X,
                                                    const float* __restrict__ Y, int r, int d,
                                                    OutT* out) {
  extern __shared__ double cs[];
  const int g = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int t = wave; t < r; t += 4) {
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
  hipLaunchKernelGGL(k_cos_groups<float>, dim3(groups), dim3(256), r * sizeof(double), st, X, Y,
                     r, d, out);
}

void cos_groups_f64(const float* X, const float* Y, int groups, int r, int d, double* out,
                    hipStream_t st) {
  if (groups <= 0) return;
  hipLaunchKernelGGL(k_cos_groups<double>, dim3(groups), dim3(256), r * sizeof(double), st, X,
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
  hipLaunchKernelGGL(k_cos_rows, dim3((rows + 3) / 4), dim3(256), 0, st, X, Y, rows, ry, d, out);
}

// ------------------------------------------------------------------- copies
// dst[i][0..n) = src[i][0..n) for pointer tables of length cnt.
__global__ void k_copy_blocks(const float* const* src, float* const* dst, size_t n) {
  const int i = blockIdx.y;
  const float* s = src[i];
  float* d = dst[i];
  for (size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c < n;
       c += (size_t)gridDim.x * blockDim.x)
    d[c] = s[c];
}

void copy_rows(const float* const* src, float* const* dst, int cnt, int n, hipStream_t st) {
  if (cnt <= 0 || n <= 0) return;
  const int bx = (n + 255) / 256 < 64 ? (n + 255) / 256 : 64;
  hipLaunchKernelGGL(k_copy_blocks, dim3(bx, cnt), dim3(256), 0, st, src, dst, (size_t)n);
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
  hipLaunchKernelGGL(k_rope_table, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, cs,
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
  hipLaunchKernelGGL(k_fill_pos, dim3((total + 255) / 256), dim3(256), 0, st, pos, len, base, r,
                     total, len_add);
}

__global__ void k_set_i32(int32_t* p, int v) { *p = v; }

void set_i32(int32_t* p, int v, hipStream_t st) {
  hipLaunchKernelGGL(k_set_i32, dim3(1), dim3(1), 0, st, p, v);
}

}  // namespace ks
