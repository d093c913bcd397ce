// Batched integer knapsack over skip budgets (Eq. objective_knapsack in
// isolation; Single-pass Efficiency and the C/2 prune of Section 3.4).
//
// One 256-thread workgroup per instance.  Thread t keeps budgets t + 256 e
// (e < E) of the current row best_{i-1} in registers and mirrors them into
// one of two LDS rows; E covers only the budgets a skip set can reach
// (0..jmax = min(C, max_skip)), the rest of the row stays INF without being
// swept.  For item i every budget j is updated in parallel from its own
// best_{i-1}[j] (keep) and best_{i-1}[j - w_i] + q_i (skip, strict), the
// latter read from LDS: each LDS row starts with jmax + 1 INF entries, so the
// skip candidate of every budget is the entry at one per-item base address
// plus a constant offset per slot (no clamp per cell; a weight above jmax,
// which no budget can take, is read as jmax + 1).  A wave owns 64
// consecutive budgets per slot e, so its 64 skip decisions are the compare's
// own lane mask, written into lane e with one v_writelane per half: the
// decision bitmap costs one word per 64 budgets per item.  Decision words
// past the swept budgets are zeroed once, before the items.  Integer
// arithmetic only, so results are exact.
#include "ks_internal.h"

namespace ks {

constexpr int32_t KINF = 0x7FFFFFFF;

// Lanes Q..Q+3 of wlo / whi receive the decision masks of slots Q..Q+3 (one
// v_writelane per half).  The masks were just written to scalar registers by
// vector compares, and v_writelane reads its scalar source early: without the
// s_nop ahead of each block some words took the mask of the previous slot.
template <int E, int Q>
__device__ inline void knap_put(const uint64_t (&bal)[E], uint32_t& wlo, uint32_t& whi) {
  if constexpr (Q < E) {
    if constexpr (Q + 4 <= E) {
      __asm__(
          "s_nop 4\n\t"
          "v_writelane_b32 %0, %2, %10\n\tv_writelane_b32 %1, %3, %10\n\t"
          "v_writelane_b32 %0, %4, %11\n\tv_writelane_b32 %1, %5, %11\n\t"
          "v_writelane_b32 %0, %6, %12\n\tv_writelane_b32 %1, %7, %12\n\t"
          "v_writelane_b32 %0, %8, %13\n\tv_writelane_b32 %1, %9, %13"
          : "+v"(wlo), "+v"(whi)
          : "s"((uint32_t)bal[Q]), "s"((uint32_t)(bal[Q] >> 32)), "s"((uint32_t)bal[Q + 1]),
            "s"((uint32_t)(bal[Q + 1] >> 32)), "s"((uint32_t)bal[Q + 2]),
            "s"((uint32_t)(bal[Q + 2] >> 32)), "s"((uint32_t)bal[Q + 3]),
            "s"((uint32_t)(bal[Q + 3] >> 32)), "i"(Q), "i"(Q + 1), "i"(Q + 2), "i"(Q + 3));
      knap_put<E, Q + 4>(bal, wlo, whi);
    } else {
      __asm__("s_nop 4\n\tv_writelane_b32 %0, %2, %4\n\tv_writelane_b32 %1, %3, %4"
              : "+v"(wlo), "+v"(whi)
              : "s"((uint32_t)bal[Q]), "s"((uint32_t)(bal[Q] >> 32)), "i"(Q));
      knap_put<E, Q + 1>(bal, wlo, whi);
    }
  }
}

// Skip decisions of every slot (strict: an equal candidate keeps), then the
// masks into their lanes.
template <int E>
__device__ inline void knap_slots(const uint32_t (&cand)[E], int32_t (&v)[E], uint32_t& wlo,
                                  uint32_t& whi) {
  uint64_t bal[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool take = cand[e] < (uint32_t)v[e];
    v[e] = take ? (int32_t)cand[e] : v[e];
    bal[e] = __ballot(take);
  }
  knap_put<E, 0>(bal, wlo, whi);
}

template <int E>
__global__ __launch_bounds__(256) void k_knap_dp(const int32_t* __restrict__ w,
                                                 const int32_t* __restrict__ q, int n, int C,
                                                 int max_skip, int32_t* __restrict__ best,
                                                 uint64_t* __restrict__ bits) {
  // two LDS rows of GU + 256 E entries: GU = jmax + 1 INF entries, then slot
  // e of thread t (budget 256 e + t) at GU + 256 e + t
  extern __shared__ int32_t buf[];
  const int jmax = min(C, max_skip);
  const int GU = jmax + 1;
  const int ROW = GU + 256 * E;
  const int b = blockIdx.x, t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int words = C / 64 + 1;
  int32_t* row0 = buf;
  int32_t* row1 = buf + ROW;
  int32_t v[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    v[e] = e * 256 + t == 0 ? 0 : KINF;
    row0[GU + e * 256 + t] = v[e];
  }
  for (int k = t; k < GU; k += 256) row0[k] = row1[k] = KINF;
  const int32_t* wb = w + (size_t)b * n;
  const int32_t* qb = q + (size_t)b * n;
  // decision words past the swept slots (budgets above jmax) are 0 for every item
  const int swept_words = 4 * E < words ? 4 * E : words;
  const int rest = words - swept_words;
  if (rest > 0)
    for (int k = t; k < n * rest; k += 256)
      bits[((size_t)b * n + k / rest) * words + swept_words + k % rest] = 0;
  __syncthreads();
  auto item = [&](int i, const int32_t* src_row, int32_t* dst_row) {
    const int wi = min(max(wb[i], 0), GU);        // negative weights are read as 0
    const uint32_t qi = (uint32_t)max(qb[i], 0);  // so are negative losses
    // all reads first (one wait), then the updates, then all writes.  An INF
    // candidate never wins: INF + q_i >= INF >= best, all below 2^32.
    const int32_t* cb = src_row + GU + t - wi;  // >= src_row: wi <= GU
    uint32_t cand[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      cand[e] = (uint32_t)cb[e * 256] + qi;
      // budgets past jmax never take a skip (unreachable); up to 9 slots the
      // launcher sizes E to the reachable budgets, so only the last slot can
      // reach past jmax
      if (e == E - 1 || E > 9) cand[e] |= e * 256 + t > jmax ? 0xFFFFFFFFu : 0u;
    }
    uint32_t wlo = 0, whi = 0;  // lane e: the 64 decisions of slot e of this wave
    knap_slots<E>(cand, v, wlo, whi);
#pragma unroll
    for (int e = 0; e < E; ++e) dst_row[GU + e * 256 + t] = v[e];
    const int word = 4 * lane + wave;  // lane e stores word 4 e + wave
    if (lane < E && word < words)
      bits[((size_t)b * n + i) * words + word] = ((uint64_t)whi << 32) | wlo;
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
  const int jmax = max_skip < C ? max_skip : C;
  const size_t lds = 2 * (size_t)(jmax + 1 + 256 * E) * sizeof(int32_t);
  KS_LAUNCH(k_knap_dp<E>, dim3(B), dim3(256), lds, st, w, q, n, C, max_skip, best, bits);
}

static int knapsack_dp_slots(int C, int max_skip) {
  // slots per thread: 256 E budgets cover the reachable budgets 0..min(C,
  // max_skip), with no slot wholly past them up to E = 9
  const int need = (max_skip < C ? max_skip : C) + 1;
  for (int e : {1, 2, 3, 4, 5, 6, 7, 8, 9, 12, 17, 24})
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
    case 7: launch_knap_dp<7>(w, q, B, n, C, max_skip, best, bits, st); break;
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
  KS_LAUNCH(k_knap_backtrack, dim3((B + 255) / 256), dim3(256), 0, st, bits, w, B, n, C,
            j, skip, err);
}

// Stage 2 with the surrogate acceptance alpha_j = prod_{i skipped} s_i.
// One workgroup per instance, thread t owning budgets t + 256 e.  Instead of a
// backtrack per budget, one sweep over the items in ascending order carries
// for every budget the product of the path that ends there: P_i[j] =
// P_{i-1}[j - w_i] * s_i where item i's decision bit at budget j is set, else
// P_{i-1}[j], from P_{-1}[0] = 1 (NaN marks a budget no consistent path
// reaches).  Following the decisions back from (n - 1, j) retraces exactly
// the path whose skipped items this product takes, in ascending order, so
// each alpha_j has the bits of the backtrack-then-multiply definition.  The
// sweep keeps the row in LDS (reads of row i - 1, a barrier, then the writes
// of row i) and stops at the largest reachable budget.  Then each thread keeps
// the first strict maximum over gamma for its budgets, and a tree keeps the
// largest value and, on equal values, the smallest budget: the same winner as
// a sequential scan over (j ascending, gamma ascending) with strict ">".
// Items are limited to 128 (the per-item weights and scores live in LDS).
// The sweep and the TPT grid over the first EL slots (EL covers the largest
// reachable budget): branch-free per slot, and a budget below the item's
// weight reads a NaN cell instead of selecting NaN after its load, so no
// lane mask has to live across a load and the item's LDS reads are in flight
// together.
template <int EL>
__device__ __forceinline__ void knap_select_sweep(int n, int C, int D, int tid, int lane,
                                                  int wave, int words,
                                                  const uint64_t* __restrict__ bb, double* row,
                                                  const double* nanp, const int32_t* sw,
                                                  const double* ss,
                                                  uint32_t live, long long W, double& bv, int& bj,
                                                  int& bg) {
#pragma clang fp contract(off)
  const double NaN = __builtin_nan("");
  double pv[EL];
#pragma unroll
  for (int e = 0; e < EL; ++e) pv[e] = 256 * e + tid == 0 ? 1.0 : NaN;
  // The decision words of item i are requested PF items ahead, as vector loads
  // (a zero the compiler cannot see through keeps them off the scalar path,
  // whose waits would also wait for every LDS access), so their memory latency
  // overlaps the sweep of the items before; the ring index of each unrolled
  // copy is a constant.  The barriers wait for this wave's LDS accesses only
  // (a full __syncthreads would also wait for the words in flight).
  // (above 9 slots per thread the ring would cost the occupancy that keeps
  // 1024 instances in one round: those sweeps load each item's words in turn)
  constexpr int PF = EL <= 4 ? 4 : (EL <= 9 ? 3 : 0);
  int vz;
  __asm__ volatile("v_mov_b32 %0, 0" : "=v"(vz));
  uint64_t wr[PF > 0 ? PF : 1][EL];
  auto fetch = [&](int i, uint64_t (&wd_)[EL]) {
    const int ic = i < n ? i : n - 1;
#pragma unroll
    for (int e = 0; e < EL; ++e) {
      const int wd = 4 * e + wave;  // word of budgets 256 e + 64 wave + lane
      wd_[e] = bb[(size_t)ic * words + (wd < words ? wd : 0) + vz];
    }
  };
  auto lds_barrier = [] {
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS accesses are done
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
  };
  if constexpr (PF == 0) {
    for (int i = 0; i < n; ++i) {
      const int wi = sw[i];
      const double si = ss[i];
      double cand[EL];
      uint64_t word[EL];
#pragma unroll
      for (int e = 0; e < EL; ++e) {
        const int j = 256 * e + tid;
        cand[e] = *(j >= wi ? &row[j - wi] : nanp);
        const int wd = 4 * e + wave;
        word[e] = wd < words ? bb[(size_t)i * words + wd] : 0ull;
      }
      __syncthreads();  // row i - 1 read by every thread before it is overwritten
#pragma unroll
      for (int e = 0; e < EL; ++e) {
        const double m = cand[e] * si;
        pv[e] = ((word[e] >> lane) & 1ull) ? m : pv[e];
        row[256 * e + tid] = pv[e];
      }
      __syncthreads();
    }
  } else {
#pragma unroll
    for (int k = 0; k < PF; ++k) fetch(k, wr[k]);
    for (int i0 = 0; i0 < n; i0 += PF) {
#pragma unroll
      for (int k = 0; k < PF; ++k) {
        const int i = i0 + k;
        if (i < n) {
          const int wi = __builtin_amdgcn_readfirstlane(sw[i]);
          const double si = ss[i];
          // rows alternate between the two halves: item i reads row i - 1
          // from one and writes row i to the other, so one barrier per item
          // (after the writes) orders both the reads and the reuse
          const double* src = row + (i & 1) * 256 * EL;
          double* dst = row + ((i & 1) ^ 1) * 256 * EL;
          const double* cb = src + tid - wi;  // skip candidate of budget 256 e + tid at cb[256 e]
          double cand[EL];
#pragma unroll
          for (int e = 0; e < EL; ++e) {
            if (256 * e >= wi) cand[e] = cb[256 * e];  // every budget of the slot covers w_i
            else cand[e] = *(256 * e + tid >= wi ? &cb[256 * e] : nanp);
          }
#pragma unroll
          for (int e = 0; e < EL; ++e) {
            // a word past the instance's last (4 e + wave >= words) holds the
            // bits of other budgets: the budgets of such a slot lie above C,
            // are never live and are never read by a live budget
            const uint64_t word = wr[k][e];
            const double m = cand[e] * si;
            pv[e] = ((word >> lane) & 1ull) ? m : pv[e];
            dst[256 * e + tid] = pv[e];
          }
          fetch(i + PF, wr[k]);
          lds_barrier();
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < EL; ++e) {  // ascending budgets
    const double a = pv[e];
    if (!((live >> e) & 1u) || a != a) continue;  // unreached, or inconsistent decisions
    const int j0 = 256 * e + tid;
    // e_g = 1 + a + ... + a^g, summed in ascending powers; one running sum
    // over g gives the same additions in the same order as summing anew
    double eg = 1.0, p = a;
    for (int g = 1; g <= D; ++g) {
      eg = eg + p;
      p = p * a;
      const double cost = (double)((long long)g * (W - j0) + W);
      const double v = eg / cost;
      if (v > bv) {
        bv = v;
        bj = j0;
        bg = g;
      }
    }
  }
}

template <int E>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void k_knap_select(
    const int32_t* __restrict__ best, const uint64_t* __restrict__ bits,
    const int32_t* __restrict__ w, const double* __restrict__ s, int n, int C, int D,
    int32_t* j_star, int32_t* g_star, double* tpt, uint8_t* skip) {
  // 256 E doubles, budget 256 e + tid at 256 e + tid (sweeps of up to 9 slots
  // use two rows of 256 EL); after the sweep the same space holds the
  // reduction's values, budgets and draft lengths
  extern __shared__ double row[];
  double* sv = row;
  int* sj = (int*)(row + 256);
  int* sg = sj + 256;
  __shared__ int32_t sw[128];
  __shared__ double ss[128];
  __shared__ double s_nan;
  __shared__ int s_jl;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int words = C / 64 + 1;
  // the instance's decision words: one word per wave and slot, read with
  // scalar loads (the address is the same for every lane of the wave)
  const uint64_t* bb = bits + (size_t)b * n * words;
  for (int i = tid; i < n; i += 256) {
    sw[i] = max(w[(size_t)b * n + i], 0);  // negative weights are read as 0, as in the DP
    ss[i] = s[(size_t)b * n + i];
  }
  if (tid == 0) {
    s_jl = 0;
    s_nan = __builtin_nan("");
  }
  uint32_t live = 0;  // bit e: budget 256 e + tid is reachable
  int jl = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int j = 256 * e + tid;
    if (j <= C && best[(size_t)b * (C + 1) + j] != KINF) {
      live |= 1u << e;
      jl = j;
    }
    row[j] = j == 0 ? 1.0 : __builtin_nan("");
  }
  __syncthreads();
  atomicMax(&s_jl, jl);
  __syncthreads();
  const int EL = s_jl / 256 + 1;  // slots up to the largest reachable budget
  long long W = 0;
  for (int i = 0; i < n; ++i) W += sw[i];
  double bv = 0.0;
  int bj = 0x7FFFFFFF, bg = 0;
#define KS_SWEEP(L_)                                                                          \
  knap_select_sweep<(L_ < E ? L_ : E)>(n, C, D, tid, lane, wave, words, bb, row, &s_nan, sw, ss, \
                                       live, W, bv, bj, bg)
  if (EL <= 1) KS_SWEEP(1);
  else if (EL <= 2) KS_SWEEP(2);
  else if (EL <= 3) KS_SWEEP(3);
  else if (EL <= 4) KS_SWEEP(4);
  else if (EL <= 6) KS_SWEEP(6);
  else if (EL <= 9) KS_SWEEP(9);
  else if (EL <= 12) KS_SWEEP(12);
  else if (EL <= 17) KS_SWEEP(17);
  else if (EL <= 24) KS_SWEEP(24);
  else KS_SWEEP(32);
#undef KS_SWEEP
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

template <int E>
static void launch_knap_select(const int32_t* best, const uint64_t* bits, const int32_t* w,
                               const double* s, int B, int n, int C, int D, int32_t* j_star,
                               int32_t* g_star, double* tpt, uint8_t* skip, hipStream_t st) {
  // one row of every budget, or two rows of up to 9 slots; at least the
  // reduction's 512 doubles
  const int two = 2 * (E < 9 ? E : 9);
  const size_t rowb = (size_t)256 * (E > two ? E : (two > 2 ? two : 2)) * sizeof(double);
  KS_LAUNCH(k_knap_select<E>, dim3(B), dim3(256), rowb, st, best, bits, w, s, n, C, D,
            j_star, g_star, tpt, skip);
}

void knapsack_select(const int32_t* best, const uint64_t* bits, const int32_t* w,
                     const double* s, int B, int n, int C, int D, int32_t* j_star,
                     int32_t* g_star, double* tpt, uint8_t* skip, hipStream_t st) {
#define KS_SEL(E_)                                                                           \
  launch_knap_select<E_>(best, bits, w, s, B, n, C, D, j_star, g_star, tpt, skip, st); break
  switch (knapsack_dp_slots(C, C)) {  // slots covering every budget 0..C
    case 1: KS_SEL(1);
    case 2: KS_SEL(2);
    case 3: KS_SEL(3);
    case 4: KS_SEL(4);
    case 5: KS_SEL(5);
    case 6: KS_SEL(6);
    case 7: KS_SEL(7);
    case 8: KS_SEL(8);
    case 9: KS_SEL(9);
    case 12: KS_SEL(12);
    case 17: KS_SEL(17);
    case 24: KS_SEL(24);
    default: KS_SEL(32);
  }
#undef KS_SEL
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
  KS_LAUNCH(k_dp_step, dim3(1), dim3(256), 0, st, a.i, a.J, a.w, a.tau, a.r, a.M,
            a.stride, a.sig, a.cells_in, a.cnt_in, a.cells_out, a.cnt_out, a.mean, a.idx,
            a.bits, a.reach, a.sig_e, a.sig_s, a.E, a.gprev, a.gnext, a.Xi, a.cell,
            a.ptr_src, a.ptr_dst, a.bound_out);
}

}  // namespace ks
