// Batched integer knapsack over skip budgets (Eq. objective_knapsack in
// isolation; Single-pass Efficiency and the C/2 prune of Section 3.4).
//
// One 256-thread workgroup per instance.  Thread t keeps budgets t + 256 e
// (e < E) of the current row best_{i-1} in registers and mirrors them into
// one of two LDS rows; E covers only the budgets a skip set can reach
// (0..min(C, max_skip)), the rest of the row stays INF without being swept; for item i every budget j is updated in parallel from
// its own best_{i-1}[j] (keep) and best_{i-1}[j - w_i] + q_i (skip, strict),
// the latter read from LDS, so a cell update costs one LDS read and one LDS
// write.  A wave owns 64 consecutive budgets per slot e, so its 64 skip
// decisions form one 64-bit ballot that a single lane stores: the decision
// bitmap costs one word per 64 budgets per item.  Integer arithmetic only, so
// results are exact.
#include "ks_internal.h"

namespace ks {

constexpr int32_t KINF = 0x7FFFFFFF;

template <int E, int Q>
__device__ inline void knap_slots(const uint32_t (&cand)[E], int32_t (&v)[E], uint32_t& wlo,
                                  uint32_t& whi) {
  if constexpr (Q < E) {
    const bool take = cand[Q] < (uint32_t)v[Q];
    v[Q] = take ? (int32_t)cand[Q] : v[Q];
    const uint64_t ballot = __ballot(take);
    if ((threadIdx.x & 63) == Q) {
      wlo = (uint32_t)ballot;
      whi = (uint32_t)(ballot >> 32);
    }
    knap_slots<E, Q + 1>(cand, v, wlo, whi);
  }
}

template <int E>
__global__ __launch_bounds__(256) void k_knap_dp(const int32_t* __restrict__ w,
                                                 const int32_t* __restrict__ q, int n, int C,
                                                 int max_skip, int32_t* __restrict__ best,
                                                 uint64_t* __restrict__ bits) {
  // two LDS rows of 256 E + 1 entries: slot e of thread t is budget 256 e + t,
  // entry 256 E a sentinel that stays INF (budgets past C stay INF too)
  extern __shared__ int32_t buf[];
  constexpr int ROW = 256 * E + 1;
  const int b = blockIdx.x, t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int words = C / 64 + 1;
  int32_t* row0 = buf;
  int32_t* row1 = buf + ROW;
  int32_t v[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    v[e] = e * 256 + t == 0 ? 0 : KINF;
    row0[e * 256 + t] = v[e];
  }
  if (t == 0) row0[256 * E] = row1[256 * E] = KINF;
  __syncthreads();
  const int32_t* wb = w + (size_t)b * n;
  const int32_t* qb = q + (size_t)b * n;
  // jv[e]: budget of slot e, or -1 where no skip can land (beyond C or max_skip)
  const int jmax = min(C, max_skip);
  int jv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) jv[e] = e * 256 + t <= jmax ? e * 256 + t : -1;
  // decision words past the swept slots (budgets above min(C, max_skip)) are 0
  const int swept_words = 4 * E < words ? 4 * E : words;
  auto item = [&](int i, const int32_t* src_row, int32_t* dst_row) {
    const int wi = max(wb[i], 0);                 // negative weights are read as 0
    const uint32_t qi = (uint32_t)max(qb[i], 0);  // so are negative losses
    // all reads first (one wait), then the updates, then all writes.  Skip
    // candidate of slot e: row entry jv[e] - w_i, or the sentinel (entry 256 E)
    // when that is negative (unsigned min).  An INF candidate never wins:
    // INF + q_i >= INF >= best, all below 2^32.
    uint32_t cand[E];
#pragma unroll
    for (int e = 0; e < E; ++e)
      cand[e] = (uint32_t)src_row[min((uint32_t)(jv[e] - wi), (uint32_t)(256 * E))] + qi;
    uint32_t wlo = 0, whi = 0;  // lane e: the 64 decisions of slot e of this wave
    knap_slots<E, 0>(cand, v, wlo, whi);
#pragma unroll
    for (int e = 0; e < E; ++e) dst_row[e * 256 + t] = v[e];
    const int word = 4 * lane + wave;  // lane e stores word 4 e + wave
    if (lane < E && word < words)
      bits[((size_t)b * n + i) * words + word] = ((uint64_t)whi << 32) | wlo;
    for (int k = swept_words + t; k < words; k += 256) bits[((size_t)b * n + i) * words + k] = 0;
    __syncthreads();
  };
  int i = 0;
  for (; i + 1 < n; i += 2) {  // fixed rows per half step: addresses fold into offsets
    item(i, row0, row1);
    item(i + 1, row1, row0);
  }
  if (i < n) item(i, row0, row1);
  const int cells = C + 1;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int j = e * 256 + t;
    if (j < cells) best[(size_t)b * cells + j] = v[e];
  }
  for (int j = 256 * E + t; j < cells; j += 256) best[(size_t)b * cells + j] = KINF;
}

template <int E>
static void launch_knap_dp(const int32_t* w, const int32_t* q, int B, int n, int C, int max_skip,
                           int32_t* best, uint64_t* bits, hipStream_t st) {
  const size_t lds = 2 * (size_t)(256 * E + 1) * sizeof(int32_t);
  hipLaunchKernelGGL(k_knap_dp<E>, dim3(B), dim3(256), lds, st, w, q, n, C, max_skip, best, bits);
}

static int knapsack_dp_slots(int C, int max_skip) {
  // slots per thread: 256 E budgets cover the reachable budgets 0..min(C, max_skip)
  const int need = (max_skip < C ? max_skip : C) + 1;
  for (int e : {1, 2, 3, 4, 5, 6, 8, 9, 12, 17, 24})
    if (need <= 256 * e) return e;
  return 32;  // C <= 8191
}

void knapsack_dp(const int32_t* w, const int32_t* q, int B, int n, int C, int max_skip,
                 int32_t* best, uint64_t* bits, hipStream_t st) {
  switch (knapsack_dp_slots(C, max_skip)) {
    case 1: launch_knap_dp<1>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 2: launch_knap_dp<2>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 3: launch_knap_dp<3>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 4: launch_knap_dp<4>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 5: launch_knap_dp<5>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 6: launch_knap_dp<6>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 8: launch_knap_dp<8>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 9: launch_knap_dp<9>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 12: launch_knap_dp<12>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 17: launch_knap_dp<17>(w, q, B, n, C, max_skip, best, bits, st); break;
    case 24: launch_knap_dp<24>(w, q, B, n, C, max_skip, best, bits, st); break;
    default: launch_knap_dp<32>(w, q, B, n, C, max_skip, best, bits, st); break;
  }
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
      j -= max(w[(size_t)b * n + i], 0);  // negative weights are read as 0, as in the DP
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
// The instance's decision words (and w, s) are staged in LDS when they fit;
// a thread walks four of its budgets' backtracks side by side so their
// dependent reads overlap.  Items are limited to 128 so a backtracked mask
// fits two 64-bit words.
template <bool BITS_IN_LDS>
__global__ __launch_bounds__(256) void k_knap_select(
    const int32_t* __restrict__ best, const uint64_t* __restrict__ bits,
    const int32_t* __restrict__ w, const double* __restrict__ s, int n, int C, int D,
    int32_t* j_star, int32_t* g_star, double* tpt, uint8_t* skip) {
#pragma clang fp contract(off)
  extern __shared__ uint64_t lbits[];
  __shared__ double sv[256];
  __shared__ int sj[256], sg[256];
  __shared__ int32_t sw[128];
  __shared__ double ss[128];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int words = C / 64 + 1;
  const uint64_t* gb = bits + (size_t)b * n * words;
  if (BITS_IN_LDS)
    for (int k = tid; k < n * words; k += 256) lbits[k] = gb[k];
  for (int i = tid; i < n; i += 256) {
    sw[i] = max(w[(size_t)b * n + i], 0);  // negative weights are read as 0, as in the DP
    ss[i] = s[(size_t)b * n + i];
  }
  __syncthreads();
  const uint64_t* bb = BITS_IN_LDS ? lbits : gb;
  long long W = 0;
  for (int i = 0; i < n; ++i) W += sw[i];
  double bv = 0.0;
  int bj = 0x7FFFFFFF, bg = 0;
  constexpr int G = 4;
  for (int k0 = 0; k0 * 256 <= C; k0 += G) {
    int jj[G], j0[G];
    uint64_t m0[G], m1[G];
    bool live[G];
#pragma unroll
    for (int u = 0; u < G; ++u) {
      j0[u] = (k0 + u) * 256 + tid;
      live[u] = j0[u] <= C && best[(size_t)b * (C + 1) + j0[u]] != KINF;
      jj[u] = j0[u];
      m0[u] = m1[u] = 0;
    }
    if (!(live[0] || live[1] || live[2] || live[3])) continue;
    for (int i = n - 1; i >= 0; --i) {
      const int wi = sw[i];
#pragma unroll
      for (int u = 0; u < G; ++u) {
        if (live[u] && jj[u] >= 0 && jj[u] <= C &&
            ((bb[i * words + (jj[u] >> 6)] >> (jj[u] & 63)) & 1ull)) {
          if (i < 64) m0[u] |= 1ull << i; else m1[u] |= 1ull << (i - 64);
          jj[u] -= wi;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < G; ++u) {  // ascending budgets
      if (!live[u] || jj[u] != 0) continue;  // inconsistent decisions: not a candidate
      double a = 1.0;
      for (int i = 0; i < n; ++i) {
        const bool sk = i < 64 ? ((m0[u] >> i) & 1ull) : ((m1[u] >> (i - 64)) & 1ull);
        if (sk) a = a * ss[i];
      }
      // e_g = 1 + a + ... + a^g, summed in ascending powers; one running sum
      // over g gives the same additions in the same order as summing anew
      double e = 1.0, p = a;
      for (int g = 1; g <= D; ++g) {
        e = e + p;
        p = p * a;
        const double cost = (double)((long long)g * (W - j0[u]) + W);
        const double v = e / cost;
        if (v > bv) {
          bv = v;
          bj = j0[u];
          bg = g;
        }
      }
    }
  }
  sv[tid] = bv;
  sj[tid] = bj;
  sg[tid] = bg;
  __syncthreads();
  for (int o = 128; o >= 1; o >>= 1) {
    if (tid < o) {
      const double v2 = sv[tid + o];
      const int j2 = sj[tid + o];
      if (v2 > sv[tid] || (v2 == sv[tid] && j2 < sj[tid])) {
        sv[tid] = v2;
        sj[tid] = j2;
        sg[tid] = sg[tid + o];
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    const int j = sj[0];
    j_star[b] = j;
    g_star[b] = sg[0];
    tpt[b] = sv[0];
    int jj = j;
    for (int i = n - 1; i >= 0; --i) {
      uint8_t sk = 0;
      if (jj >= 0 && jj <= C && ((bb[i * words + (jj >> 6)] >> (jj & 63)) & 1ull)) {
        sk = 1;
        jj -= sw[i];
      }
      skip[(size_t)b * n + i] = sk;
    }
  }
}

void knapsack_select(const int32_t* best, const uint64_t* bits, const int32_t* w,
                     const double* s, int B, int n, int C, int D, int32_t* j_star,
                     int32_t* g_star, double* tpt, uint8_t* skip, hipStream_t st) {
  const size_t lds = (size_t)n * (C / 64 + 1) * 8;
  if (lds <= 48 * 1024)
    hipLaunchKernelGGL(k_knap_select<true>, dim3(B), dim3(256), lds, st, best, bits, w, s, n, C, D,
                       j_star, g_star, tpt, skip);
  else
    hipLaunchKernelGGL(k_knap_select<false>, dim3(B), dim3(256), 0, st, best, bits, w, s, n, C, D,
                       j_star, g_star, tpt, skip);
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
