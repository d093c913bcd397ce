// Batched integer knapsack over skip budgets (Eq. objective_knapsack in
// isolation; Single-pass Efficiency and the C/2 prune of Section 3.4).
//
// One workgroup per instance.  The row best_{i-1}[0..C] lives in LDS (two
// ping-pong buffers); for item i every budget j is updated in parallel from
// best_{i-1}[j] (keep) and best_{i-1}[j - w_i] + q_i (skip, strict).  A wave
// owns 64 consecutive budgets, so its 64 skip decisions form one 64-bit
// ballot that a single lane stores: the decision bitmap costs one word per
// 64 budgets per item.  Integer arithmetic only, so results are exact.
#include "ks_internal.h"

namespace ks {

constexpr int32_t KINF = 0x7FFFFFFF;

__global__ __launch_bounds__(1024) void k_knap_dp(const int32_t* __restrict__ w,
                                                  const int32_t* __restrict__ q, int n, int C,
                                                  int max_skip, int32_t* __restrict__ best,
                                                  uint64_t* __restrict__ bits) {
  extern __shared__ int32_t buf[];
  const int b = blockIdx.x;
  const int cells = C + 1;
  const int words = C / 64 + 1;
  int32_t* cur = buf;
  int32_t* nxt = buf + cells;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int j = threadIdx.x; j < cells; j += blockDim.x) cur[j] = j == 0 ? 0 : KINF;
  __syncthreads();
  for (int i = 0; i < n; ++i) {
    const int wi = w[(size_t)b * n + i];
    const int64_t qi = q[(size_t)b * n + i];
    uint64_t* brow = bits + ((size_t)b * n + i) * words;
    for (int base = wave * 64; base < words * 64; base += nw * 64) {
      const int j = base + lane;
      bool take = false;
      if (j < cells) {
        const int32_t keep = cur[j];
        int32_t v = keep;
        if (j >= wi && j <= max_skip) {
          const int32_t src = cur[j - wi];
          if (src != KINF) {
            const int64_t cand = (int64_t)src + qi;
            if (cand < (int64_t)keep) {
              v = (int32_t)cand;
              take = true;
            }
          }
        }
        nxt[j] = v;
      }
      const uint64_t ballot = __ballot(take);
      if (lane == 0) brow[base >> 6] = ballot;
    }
    __syncthreads();
    int32_t* t = cur;
    cur = nxt;
    nxt = t;
  }
  for (int j = threadIdx.x; j < cells; j += blockDim.x) best[(size_t)b * cells + j] = cur[j];
}

void knapsack_dp(const int32_t* w, const int32_t* q, int B, int n, int C, int max_skip,
                 int32_t* best, uint64_t* bits, hipStream_t st) {
  const size_t lds = 2 * (size_t)(C + 1) * sizeof(int32_t);
  hipLaunchKernelGGL(k_knap_dp, dim3(B), dim3(1024), lds, st, w, q, n, C, max_skip, best, bits);
}

__device__ inline int get_bit(const uint64_t* row, int j) { return (int)((row[j >> 6] >> (j & 63)) & 1ull); }

__global__ void k_knap_backtrack(const uint64_t* __restrict__ bits, const int32_t* __restrict__ w,
                                 int B, int n, int C, const int32_t* __restrict__ jsel,
                                 uint8_t* __restrict__ skip, int32_t* __restrict__ err) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int words = C / 64 + 1;
  int j = jsel[b];
  int bad = (j < 0 || j > C) ? 1 : 0;
  for (int i = n - 1; i >= 0; --i) {
    uint8_t sk = 0;
    if (!bad && get_bit(bits + ((size_t)b * n + i) * words, j)) {
      sk = 1;
      j -= w[(size_t)b * n + i];
      if (j < 0) bad = 1;
    }
    skip[(size_t)b * n + i] = sk;
  }
  err[b] = (bad || j != 0) ? 1 : 0;
}

void knapsack_backtrack(const uint64_t* bits, const int32_t* w, int B, int n, int C,
                        const int32_t* j, uint8_t* skip, int32_t* err, hipStream_t st) {
  hipLaunchKernelGGL(k_knap_backtrack, dim3((B + 255) / 256), dim3(256), 0, st, bits, w, B, n, C,
                     j, skip, err);
}

// Stage 2 with the surrogate acceptance alpha_j = prod_{i skipped} s_i.
// One workgroup per instance, threads over budgets; each thread keeps the
// first strict maximum over gamma for its budget, then a tree keeps the
// largest value and, on equal values, the smallest budget: the same winner as
// a sequential scan over (j ascending, gamma ascending) with strict ">".
// Items are limited to 128 so a backtracked mask fits two 64-bit words.
__global__ __launch_bounds__(256) void k_knap_select(
    const int32_t* __restrict__ best, const uint64_t* __restrict__ bits,
    const int32_t* __restrict__ w, const double* __restrict__ s, int n, int C, int D,
    int32_t* j_star, int32_t* g_star, double* tpt, uint8_t* skip) {
#pragma clang fp contract(off)
  __shared__ double sv[256];
  __shared__ int sj[256], sg[256];
  const int b = blockIdx.x;
  const int words = C / 64 + 1;
  const int32_t* wb = w + (size_t)b * n;
  const double* sb = s + (size_t)b * n;
  long long W = 0;
  for (int i = 0; i < n; ++i) W += wb[i];
  double bv = 0.0;
  int bj = 0x7FFFFFFF, bg = 0;
  for (int j = threadIdx.x; j <= C; j += blockDim.x) {
    if (best[(size_t)b * (C + 1) + j] == KINF) continue;
    uint64_t m0 = 0, m1 = 0;
    int jj = j;
    for (int i = n - 1; i >= 0 && jj >= 0; --i) {
      if (get_bit(bits + ((size_t)b * n + i) * words, jj)) {
        if (i < 64) m0 |= 1ull << i; else m1 |= 1ull << (i - 64);
        jj -= wb[i];
      }
    }
    if (jj != 0) continue;  // inconsistent decisions: not a candidate
    double a = 1.0;
    for (int i = 0; i < n; ++i) {
      const bool sk = i < 64 ? ((m0 >> i) & 1ull) : ((m1 >> (i - 64)) & 1ull);
      if (sk) a = a * sb[i];
    }
    for (int g = 1; g <= D; ++g) {
      double e = 0.0, p = 1.0;
      for (int k = 0; k <= g; ++k) {
        e = e + p;
        p = p * a;
      }
      const double cost = (double)((long long)g * (W - j) + W);
      const double v = e / cost;
      if (v > bv) {  // threads visit their budgets in ascending order
        bv = v;
        bj = j;
        bg = g;
      }
    }
  }
  sv[threadIdx.x] = bv;
  sj[threadIdx.x] = bj;
  sg[threadIdx.x] = bg;
  __syncthreads();
  for (int o = 128; o >= 1; o >>= 1) {
    if (threadIdx.x < o) {
      const double v2 = sv[threadIdx.x + o];
      const int j2 = sj[threadIdx.x + o];
      if (v2 > sv[threadIdx.x] || (v2 == sv[threadIdx.x] && j2 < sj[threadIdx.x])) {
        sv[threadIdx.x] = v2;
        sj[threadIdx.x] = j2;
        sg[threadIdx.x] = sg[threadIdx.x + o];
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int j = sj[0];
    j_star[b] = j;
    g_star[b] = sg[0];
    tpt[b] = sv[0];
    int jj = j;
    for (int i = n - 1; i >= 0; --i) {
      uint8_t sk = 0;
      if (jj >= 0 && jj <= C && get_bit(bits + ((size_t)b * n + i) * words, jj)) {
        sk = 1;
        jj -= wb[i];
      }
      skip[(size_t)b * n + i] = sk;
    }
  }
}

void knapsack_select(const int32_t* best, const uint64_t* bits, const int32_t* w,
                     const double* s, int B, int n, int C, int D, int32_t* j_star,
                     int32_t* g_star, double* tpt, uint8_t* skip, hipStream_t st) {
  hipLaunchKernelGGL(k_knap_select, dim3(B), dim3(256), 0, st, best, bits, w, s, n, C, D, j_star,
                     g_star, tpt, skip);
}

// ------------------------------------------------------- model-mode step
// One stage i of the model-mode DP (Section 3.4, Eq. dp_main, pull form), on
// the device so the stages run without host round trips.  Inputs: the per-row
// cosines of the executed candidates E (sig[0, M)) and of the skip candidates
// g[i-1, .] (sig[M, 2M)) against X^(i), M = (bound cells) * r rows, for the
// reachable budgets cells_in[0..cnt_in) (ascending).  The matrix cosine of a
// cell is the row mean, summed in row order.  For every budget j <= J: j = 0
// takes X^(i); otherwise the executed candidate if its cosine exceeds tau and
// is at least the skip candidate's (ties execute), else the skip candidate
// g[i-1, j - w] if its cosine exceeds tau (decision bit 1), else j is
// unreachable.  Writes the decision bits, the debug record (cosines, reach) of
// row i, the next reachable list and the row-gather table (null beyond the
// list, up to `bound_out` entries).
__global__ __launch_bounds__(256) void k_dp_step(
    int i, int J, int w, double tau, int r, int M, int stride, const double* __restrict__ sig,
    const int* __restrict__ cells_in, const int* __restrict__ cnt_in, int* cells_out,
    int* cnt_out, double* mean, int* idx, uint8_t* bits, uint8_t* reach, double* sig_e,
    double* sig_s, const float* E, const float* gprev, float* gnext, const float* Xi,
    size_t cell, const float** ptr_src, float** ptr_dst, int bound_out) {
  const int nc = *cnt_in;
  for (int k = threadIdx.x; k < 2 * nc; k += blockDim.x) {
    const double* srow = sig + (k < nc ? 0 : M) + (size_t)(k < nc ? k : k - nc) * r;
    double sum = 0.0;
    for (int t = 0; t < r; ++t) sum += srow[t];
    mean[k] = sum / r;
  }
  for (int j = threadIdx.x; j <= J; j += blockDim.x) idx[j] = -1;
  __syncthreads();
  for (int k = threadIdx.x; k < nc; k += blockDim.x) idx[cells_in[k]] = k;
  __syncthreads();
  // every budget decides in parallel; the reached budgets are compacted in
  // ascending order with a workgroup scan, 256 budgets at a time
  __shared__ int s_wsum[4];
  const double qnan = __longlong_as_double(0x7FF8000000000000ll);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int base = 0;
  for (int j0 = 0; j0 <= J; j0 += 256) {
    const int j = j0 + threadIdx.x;
    const float* src = nullptr;
    if (j <= J) {
      const int ie = idx[j];
      const int is = j >= w ? idx[j - w] : -1;
      const double sge = ie >= 0 ? mean[ie] : qnan;
      const double sgs = is >= 0 ? mean[nc + is] : qnan;
      const bool e_ok = ie >= 0 && sge > tau;
      const bool s_ok = is >= 0 && sgs > tau;
      uint8_t bit = 0;
      if (j == 0) {
        src = Xi;
      } else if (e_ok && (!s_ok || sge >= sgs)) {
        src = E + (size_t)ie * cell;
      } else if (s_ok) {
        src = gprev + (size_t)is * cell;
        bit = 1;
      }
      const size_t o = (size_t)i * stride + j;
      bits[o] = bit;
      reach[o] = src != nullptr;
      sig_e[o] = sge;
      sig_s[o] = sgs;
    }
    const unsigned long long bal = __ballot(src != nullptr);
    if (lane == 0) s_wsum[wv] = __popcll(bal);
    __syncthreads();
    int off = base;
    for (int q = 0; q < wv; ++q) off += s_wsum[q];
    if (src) {
      const int p = off + __popcll(bal & ((1ull << lane) - 1ull));
      ptr_src[p] = src;
      ptr_dst[p] = gnext + (size_t)p * cell;
      cells_out[p] = j;
    }
    base += s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    __syncthreads();
  }
  for (int k = base + threadIdx.x; k < bound_out; k += blockDim.x) ptr_src[k] = nullptr;
  if (threadIdx.x == 0) *cnt_out = base;
}

void dp_step(const DpStepArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_dp_step, dim3(1), dim3(256), 0, st, a.i, a.J, a.w, a.tau, a.r, a.M,
                     a.stride, a.sig, a.cells_in, a.cnt_in, a.cells_out, a.cnt_out, a.mean, a.idx,
                     a.bits, a.reach, a.sig_e, a.sig_s, a.E, a.gprev, a.gnext, a.Xi, a.cell,
                     a.ptr_src, a.ptr_dst, a.bound_out);
}

}  // namespace ks
