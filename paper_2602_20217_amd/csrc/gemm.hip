// Matrix products of the decoder sublayers.
//
// bf16 weights are stored in a tile layout that matches the B-operand registers
// of v_mfma_f32_16x16x32_bf16: a 16 (rows of W) x 32 (k) tile is 1 KiB and lane
// l holds row l%16, k = 8(l/16)..8(l/16)+7 at byte offset 16 l.  One 64-lane
// load therefore reads one contiguous KiB of HBM.
//
// Skinny path (M <= 16 rows: decode, draft, verify): the batch-1 decode step
// is HBM-bound, so every weight byte is read once.  Activations enter as two
// bf16 planes hi + lo so the product keeps ~16 mantissa bits of the float32
// activations; the 16 rows of the matrix instruction hold the hi planes of
// up to 8 activation rows in rows 0..7 and their lo planes in rows 8..15, so
// one instruction per weight fragment serves 8 rows (two for 9..16 rows, one
// per group of 8), and the two planes' sums are added in the epilogue.  K is
// split over the waves of a workgroup and reduced in LDS in a fixed order, so
// a row's result does not depend on how many rows are in the batch: a verify
// row and the decode step at the same position produce identical bits.
//
// Tiled path (batched rows of the selection DP and of prefill): 128 x 256
// workgroup tiles of eight 64 x 64 wave tiles of 16x16x32 MFMAs over single
// bf16 activations, operands staged through a three-stage LDS ring by direct
// global-to-LDS loads; K is split over workgroups when the row count leaves
// CUs idle (factor from a cost model of resident rounds and partial traffic),
// and the float32 partials are summed in split order.
#include "ks_internal.h"

#include <algorithm>
#include <atomic>

namespace ks {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline bf16x8 ld_frag(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, *(const u32x4*)p);
}
__device__ inline bf16x8 ld_frag_nt(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load((const u32x4*)p));
}
__device__ inline bf16x8 zero_frag() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, z);
}
__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }
__device__ inline void store_split(bf16_t* hi, bf16_t* lo, size_t off, float a) {
  bf16_t h = f2bf(a);
  hi[off] = h;
  if (lo) lo[off] = f2bf(a - bf2f(h));
}

// ------------------------------------------------------------------ skinny
// RMSNorm rides on the producers of the residual stream: the residual
// epilogue (and the embedding) writes x * gain of the next normed product as
// hi + lo bf16 planes together with sums of x^2 per 16-column tile.  AN = 1
// products read those planes like any activation and scale row m by
// 1/sqrt(sum/K + eps) at the end; the 256 tile sums of a row are added by one
// wave in a fixed order, whatever the row count.
template <int NB, int NW, int CH, int MINB, int EPI, int AN, int A1, int MH>
__global__ __launch_bounds__(NW * 64, MINB) void k_gemm_skinny(
    int M, int N, int K, const bf16_t* __restrict__ Ahi, const bf16_t* __restrict__ Alo,
    int lda, const bf16_t* __restrict__ Wp, float* out, int ldo, const float* res, int ldres,
    bf16_t* ohi, bf16_t* olo, int ldact, const float* __restrict__ ssq_in, int nssq, float eps,
    const float* __restrict__ next_gain, bf16_t* nhi, bf16_t* nlo, int ldn, float* next_ssq,
    QkvEpi qe) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int KT = K >> 5;
  const int NT = N >> 4;
  const int nt0 = blockIdx.x * NB;
  const int kb = (wave * KT) / NW;
  const int ke = ((wave + 1) * KT) / NW;
  // matrix row of this lane: plane (0 hi, 1 lo) of activation row 8 h + (slot & 7)
  const int slot = lane & 15;
  const int plane = slot >> 3;
  const int kg = lane >> 4;

  static_assert(NB * 256 <= NW * 64, "one epilogue element per thread");
  static_assert(MH == 1 || (MH == 2 && A1 == 0), "one-row staging serves one group of 8 rows");
  // epilogue element of this thread: tile et, row group eh, hi-plane MFMA lane
  // el (its lo-plane partner is el + 32), accumulator register ev (row em,
  // column en)
  const int et = threadIdx.x >> 8, eh = (threadIdx.x >> 7) & 1, ev = threadIdx.x & 3;
  const int el = (threadIdx.x >> 2) & 31;
  const int em = 8 * eh + 4 * (el >> 4) + ev;
  const int en = (nt0 + et) * 16 + (el & 15);
  const bool eact = threadIdx.x < NB * 256 && eh < MH && em < M && nt0 + et < NT;

  // Epilogue operands that do not depend on the product are requested before
  // the weight stream, so that their memory latency overlaps it instead of
  // trailing every workgroup: the RMSNorm tile sums of this wave's first NPRE
  // rows (UPRE per lane), the residual and next-norm gain of the thread's
  // element, the position of its row.
  // (read unconditionally at clamped, valid indices; entries past M or nssq
  // are dropped when the sums are formed)
  constexpr int NPRE = AN ? (NW >= 16 ? 1 : 2) : 1;
  constexpr int UPRE = 4;
  float pre[NPRE][UPRE];
  if (AN) {
#pragma unroll
    for (int q = 0; q < NPRE; ++q) {
      const int m = min(wave + q * NW, M - 1);
#pragma unroll
      for (int u = 0; u < UPRE; ++u)
        pre[q][u] = ssq_in[(size_t)m * nssq + min(lane + 64 * u, nssq - 1)];
    }
  }
  float e_res = 0.f, e_gain = 0.f;
  int e_pos = 0;
  if (EPI == EPI_RESID && eact) {
    e_res = res[(size_t)em * ldres + en];
    if (next_gain) e_gain = next_gain[en];
  }
  if (EPI == EPI_QKV && eact) e_pos = qe.pos[em];

  // One-row products (A1 > 0, decode and draft steps): the activation row
  // (hi and lo planes) is staged in LDS once per workgroup, so the k loop's
  // only global loads are the weight fragments.  Loaded per k step, the
  // activation fragments are one of every two load instructions (for one row,
  // 8 lanes of each plane fetch the same 16 bytes), and the address unit's
  // time for them delays the weight stream's start.  The
  // matrix instructions see the same operand values either way, so the result
  // bits do not depend on the path.  A1 = 16-byte pieces per thread and plane
  // (the launcher takes the least with 64 NW A1 >= K / 8).
  extern __shared__ __align__(16) uint4 s_act[];  // A1: hi plane [K / 8], then lo plane
  constexpr int A1PT = A1 > 0 ? A1 : 1;
  const int n16 = K >> 3;
  uint4 av[2][A1PT];
  if constexpr (A1 != 0) {
    // unconditional loads at clamped indices, so the wait before the LDS
    // store counts only the weight loads issued after them
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int q = 0; q < A1PT; ++q) {
        const int i = threadIdx.x + q * NW * 64;
        av[pl][q] = ((const uint4*)(pl ? Alo : Ahi))[i < n16 ? i : n16 - 1];
      }
  }

  f32x4 acc[MH][NB];
#pragma unroll
  for (int h = 0; h < MH; ++h)
#pragma unroll
    for (int t = 0; t < NB; ++t) acc[h][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Lanes of rows past M read row 0: their products land in result rows that
  // are never stored (an MFMA result row depends only on its own A row).
  const bf16_t* ap[MH];
#pragma unroll
  for (int h = 0; h < MH; ++h) {
    const int r = 8 * h + (slot & 7);
    ap[h] = (plane ? Alo : Ahi) + (size_t)(r < M ? r : 0) * lda + kg * 8;
  }
  const bf16_t* wb[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    int nt = nt0 + t < NT ? nt0 + t : NT - 1;
    wb[t] = Wp + (size_t)nt * KT * 512 + lane * 8;
  }
  // The wave's k steps [kb, ke) run in full chunks of CH through two register
  // stages: the weight and activation fragments of chunk c + 1 are requested
  // before the matrix instructions of chunk c, so every wave keeps a chunk in
  // flight while it computes (branch-free chunk code, so the compiler counts
  // the loads in flight exactly); the last (ke - kb) % CH steps follow one by
  // one.  The order of the matrix instructions (k ascending, row groups in
  // order) is that of a plain loop.
  bf16x8 w0[NB][CH], x0[MH][CH];
  bf16x8 w1[NB][CH], x1[MH][CH];
  auto fetch = [&](int kc, bf16x8 (&w)[NB][CH], bf16x8 (&x)[MH][CH]) {
#pragma unroll
    for (int u = 0; u < CH; ++u) {
#pragma unroll
      for (int t = 0; t < NB; ++t) w[t][u] = ld_frag_nt(wb[t] + (size_t)(kc + u) * 512);
      if constexpr (A1 == 0) {
#pragma unroll
        for (int h = 0; h < MH; ++h) x[h][u] = ld_frag(ap[h] + (kc + u) * 32);
      }
    }
  };
  // A1: lane (slot, kg) takes k = 32 step + 8 kg .. + 7 of its plane of row 0
  // from LDS
  auto act_lds = [&](int k) {
    return __builtin_bit_cast(bf16x8, s_act[plane * n16 + 4 * k + kg]);
  };
  auto compute = [&](int kc, bf16x8 (&w)[NB][CH], bf16x8 (&x)[MH][CH]) {
#pragma unroll
    for (int u = 0; u < CH; ++u) {
#pragma unroll
      for (int h = 0; h < MH; ++h) {
        const bf16x8 a = A1 ? act_lds(kc + u) : x[h][u];
#pragma unroll
        for (int t = 0; t < NB; ++t)
          acc[h][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w[t][u], acc[h][t], 0, 0, 0);
      }
    }
  };
  const int nfull = (ke - kb) / CH;  // wave-uniform
  auto ck = [&](int c) { return kb + c * CH; };  // the wave's c-th full chunk
  if constexpr (A1 != 0) {
    // Two chunks in flight from the start (the launcher gives every wave at
    // least two): both are requested before the wait for the row, so the
    // stream does not pause while the row lands in LDS; then chunk c + 2 is
    // requested after chunk c's matrix instructions.
    fetch(ck(0), w0, x0);
    fetch(ck(1), w1, x1);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int q = 0; q < A1PT; ++q) {
        const int i = threadIdx.x + q * NW * 64;
        if (i < n16) s_act[pl * n16 + i] = av[pl][q];
      }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
    int c = 0;
    for (; c + 3 < nfull; c += 2) {  // chunks c and c + 1 are in flight
      compute(ck(c), w0, x0);
      fetch(ck(c + 2), w0, x0);
      compute(ck(c + 1), w1, x1);
      fetch(ck(c + 3), w1, x1);
    }
    compute(ck(c), w0, x0);
    if (c + 2 < nfull) {
      fetch(ck(c + 2), w0, x0);
      compute(ck(c + 1), w1, x1);
      compute(ck(c + 2), w0, x0);
    } else {
      compute(ck(c + 1), w1, x1);
    }
  } else {
    if (nfull > 0) fetch(ck(0), w0, x0);
    int c = 0;
    for (; c + 2 < nfull; c += 2) {  // chunk c is in stage 0 and in flight
      fetch(ck(c + 1), w1, x1);
      compute(ck(c), w0, x0);
      fetch(ck(c + 2), w0, x0);
      compute(ck(c + 1), w1, x1);
    }
    if (c + 1 < nfull) {
      fetch(ck(c + 1), w1, x1);
      compute(ck(c), w0, x0);
      compute(ck(c + 1), w1, x1);
    } else if (c < nfull) {
      compute(ck(c), w0, x0);
    }
  }
  for (int k = kb + nfull * CH; k < ke; ++k) {
    bf16x8 b[NB];
#pragma unroll
    for (int t = 0; t < NB; ++t) b[t] = ld_frag_nt(wb[t] + (size_t)k * 512);
#pragma unroll
    for (int h = 0; h < MH; ++h) {
      const bf16x8 a = A1 ? act_lds(k) : ld_frag(ap[h] + k * 32);
#pragma unroll
      for (int t = 0; t < NB; ++t)
        acc[h][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[t], acc[h][t], 0, 0, 0);
    }
  }

  __shared__ f32x4 red[NW][NB][MH][64];
  __shared__ float s_rs[AN ? 16 : 1];
#pragma unroll
  for (int h = 0; h < MH; ++h)
#pragma unroll
    for (int t = 0; t < NB; ++t) red[wave][t][h][lane] = acc[h][t];
  // the product at (tile t, row group h, hi-plane lane l, register v): the
  // waves' hi-plane partials in wave order, plus their lo-plane partials in
  // wave order
  auto rsum = [&](int t, int h, int l, int v) {
    float a = 0.f, b = 0.f;
    for (int w = 0; w < NW; ++w) {
      a += red[w][t][h][l][v];
      b += red[w][t][h][l + 32][v];
    }
    return a + b;
  };
  if (AN) {
    // row sums in the order of a sequential sum over j = lane, lane + 64, ...,
    // then a butterfly
    auto finish = [&](int m, float t) {
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o);
      if (lane == 0) s_rs[m] = 1.0f / sqrtf(t / (float)K + eps);
    };
#pragma unroll
    for (int q = 0; q < NPRE; ++q) {
      const int m = wave + q * NW;
      if (m < M) {
        float t = 0.f;
#pragma unroll
        for (int u = 0; u < UPRE; ++u)
          if (lane + 64 * u < nssq) t += pre[q][u];
        for (int j = lane + 64 * UPRE; j < nssq; j += 64) t += ssq_in[(size_t)m * nssq + j];
        finish(m, t);
      }
    }
    for (int m = wave + NPRE * NW; m < M; m += NW) {
      float t = 0.f;
      for (int j = lane; j < nssq; j += 64) t += ssq_in[(size_t)m * nssq + j];
      finish(m, t);
    }
  }
  __syncthreads();

  if (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
    // tile rows 0..7 pair with rows 8..15 (gate/up, or rotary pairs)
    if (eact && (el & 15) < 8) {
      float g = rsum(et, eh, el, ev), u = rsum(et, eh, el + 8, ev);
      if (AN) {
        g *= s_rs[em];
        u *= s_rs[em];
      }
      if (EPI == EPI_SWIGLU) {
        const int c = (nt0 + et) * 8 + (el & 15);
        store_split(ohi, olo, (size_t)em * ldact + c, silu_mul(g, u));
      } else {
        const int tph = qe.hd >> 4, half = qe.hd >> 1;
        const int hh = (nt0 + et) / tph;
        const int f = 8 * ((nt0 + et) % tph) + (el & 15);
        const int p = e_pos;
        if (hh < qe.hq + qe.hkv) {
          const float2 cs = *(const float2*)&qe.rope_cs[((size_t)p * half + f) * 2];
          const float y0 = g * cs.x - u * cs.y;
          const float y1 = u * cs.x + g * cs.y;
          if (hh < qe.hq) {
            float* q = qe.q_out + ((size_t)em * qe.hq + hh) * qe.hd;
            q[f] = y0;
            q[f + half] = y1;
          } else {
            bf16_t* k = qe.kc + ((size_t)(hh - qe.hq) * qe.n_max + p) * qe.hd;
            k[f] = f2bf(y0);
            k[f + half] = f2bf(y1);
          }
        } else {
          bf16_t* vv = qe.vc + ((size_t)(hh - qe.hq - qe.hkv) * qe.n_max + p) * qe.hd;
          vv[f] = f2bf(g);
          vv[f + half] = f2bf(u);
        }
      }
    }
  } else {
    // thread < 256 owns (row em, column el % 16): in a wave the 16 columns of
    // a row sit on lane bits 2..5, so the tile's sum of squares for the next
    // norm is a 4-step butterfly
    static_assert(EPI != EPI_RESID || NB == 1, "next-norm sums assume one tile per block");
    const bool nn = EPI == EPI_RESID && next_gain != nullptr;
    if (threadIdx.x < NB * 256) {
      float s = 0.f;
      if (eact) {
        s = rsum(et, eh, el, ev);
        if (AN) s *= s_rs[em];
        if (EPI == EPI_RESID) s += e_res;
        out[(size_t)em * ldo + en] = s;
      }
      if (nn) {
        float sq = s * s;
        if (eact) store_split(nhi, nlo, (size_t)em * ldn + en, s * e_gain);
        sq += __shfl_xor(sq, 4);
        sq += __shfl_xor(sq, 8);
        sq += __shfl_xor(sq, 16);
        sq += __shfl_xor(sq, 32);
        if (eact && (el & 15) == 0) next_ssq[(size_t)em * NT + nt0 + et] = sq;
      }
    }
  }
}

template <int NB, int NW, int CH, int MINB, int AN, int A1, int MH>
static void launch_skinny_a1(const GemmArgs& g, hipStream_t st) {
  const int NT = g.N / 16;
  const bf16_t* Ahi = (const bf16_t*)g.A.hi;
  const bf16_t* Alo = (const bf16_t*)g.A.lo;
  const bf16_t* W = (const bf16_t*)g.W;
  dim3 grid((NT + NB - 1) / NB), block(NW * 64);
  const size_t lds = A1 ? (size_t)g.K * 4 : 0;  // hi and lo planes of the row
#define KS_SKINNY(E, OH, OL, OLD)                                                               \
  KS_LAUNCH((k_gemm_skinny<NB, NW, CH, MINB, E, AN, A1, MH>), grid, block, lds, st, g.M, g.N,   \
            g.K, Ahi, Alo, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, OH, OL, OLD,                \
            g.ssq_in, g.nssq, g.eps, g.next_gain, (bf16_t*)g.next_act.hi,                       \
            (bf16_t*)g.next_act.lo, g.next_act.ld, g.next_ssq, g.qe)
  if (g.epi == EPI_SWIGLU)
    KS_SKINNY(EPI_SWIGLU, (bf16_t*)g.act_out.hi, (bf16_t*)g.act_out.lo, g.act_out.ld);
  else if (g.epi == EPI_QKV)
    KS_SKINNY(EPI_QKV, nullptr, nullptr, 0);
  else if (g.epi == EPI_RESID) {
    if constexpr (NB == 1) KS_SKINNY(EPI_RESID, nullptr, nullptr, 0);
  }
  else
    KS_SKINNY(EPI_STORE, nullptr, nullptr, 0);
#undef KS_SKINNY
}

template <int NB, int NW, int CH, int MINB, int AN, int STAGE>
static void launch_skinny_an(const GemmArgs& g, hipStream_t st) {
  // one row and a shape that gains from it (STAGE): the activation row from
  // LDS (hi + lo planes, 4 K bytes; 16-byte aligned planes, at most four
  // pieces per thread and plane, every wave at least two full chunks)
  const int pieces = g.K / 8, per = 64 * NW;
  const bool a1 = STAGE && g.M == 1 && g.K % 8 == 0 && (size_t)g.K * 4 <= 64 * 1024 &&
                  4 * per >= pieces && (g.K / 32) / NW >= 2 * CH &&
                  (((uintptr_t)g.A.hi | (uintptr_t)g.A.lo) & 15) == 0;
  if (!a1 && g.M > 8) launch_skinny_a1<NB, NW, CH, MINB, AN, 0, 2>(g, st);
  else if (!a1) launch_skinny_a1<NB, NW, CH, MINB, AN, 0, 1>(g, st);
  else if (per >= pieces) launch_skinny_a1<NB, NW, CH, MINB, AN, 1, 1>(g, st);
  else if (2 * per >= pieces) launch_skinny_a1<NB, NW, CH, MINB, AN, 2, 1>(g, st);
  else launch_skinny_a1<NB, NW, CH, MINB, AN, 4, 1>(g, st);
}

template <int NB, int NW, int CH, int MINB, int STAGE>
static void launch_skinny(const GemmArgs& g, hipStream_t st) {
  if (g.ssq_in) launch_skinny_an<NB, NW, CH, MINB, 1, STAGE>(g, st);
  else launch_skinny_an<NB, NW, CH, MINB, 0, STAGE>(g, st);
}

// Launch shape by matrix shape only (never by row count; the one-row staging
// changes where the operands come from, not the arithmetic), measured on
// MI355X with the Llama-8B shapes (cold weights; 4/8/16 waves, 1/2/4-deep
// pipelined chunks, workgroups per CU forced by the register budget, staging
// on or off): gate/up one tile per 4-wave workgroup, 2-deep chunks; the long-K
// down projection and the square O projection 16 waves, 4-deep; the vocabulary
// head and the q/k/v projection 8 waves, 4-deep; every shape with the one-row
// activation staged in LDS and two chunks per wave in flight from the start
// (8K decode step 3.22 -> 3.09 ms against per-step activation loads).
// (output tiles per workgroup, waves, k steps per chunk, workgroups per CU
// the register budget must allow, one-row activation staged in LDS)
#ifndef KS_SK_GU
#define KS_SK_GU 1, 4, 2, 1, 1
#endif
#ifndef KS_SK_DOWN
#define KS_SK_DOWN 1, 16, 4, 1, 1
#endif
#ifndef KS_SK_HEAD
#define KS_SK_HEAD 1, 8, 4, 1, 1
#endif
#ifndef KS_SK_SQ
#define KS_SK_SQ 1, 16, 4, 1, 1
#endif
#ifndef KS_SK_WIDE
#define KS_SK_WIDE 1, 8, 4, 1, 1
#endif
void gemm_bf16_skinny(const GemmArgs& g, hipStream_t st) {
  if (g.epi == EPI_SWIGLU) launch_skinny<KS_SK_GU>(g, st);
  else if (g.K >= 8192) launch_skinny<KS_SK_DOWN>(g, st);
  else if (g.N >= 65536) launch_skinny<KS_SK_HEAD>(g, st);
  else if (g.N <= 4096) launch_skinny<KS_SK_SQ>(g, st);
  else launch_skinny<KS_SK_WIDE>(g, st);
}

// ------------------------------------------------------------------- tiled
// Batched rows (prefill chunks, selection DP).  Workgroup tile 16 WM NWM rows x
// 16 NWN WN columns, NWM x NWN waves with 16 WM x 16 WN wave tiles (WM x WN
// MFMAs per k step).
// A 32-wide k step of the workgroup is WM NWM + NWN WN operand tiles of 1 KiB, each
// laid out in LDS in MFMA register order (lane l at byte 16 l: row l % 16,
// k 8 (l / 16)..), so every fragment read is one conflict-free 16-byte read.
// The tiles travel with direct global-to-LDS loads (one 1 KiB load per tile:
// lane l fetches row l % 16, k chunk l / 16 of A, or 16 bytes of the packed W
// tile, which is already in that order), ST - 1 steps ahead of the arithmetic
// in a ring of ST stages: one barrier per step and no staging registers.
// Rows past M and tiles past N read clamped (valid) addresses; their results
// are never stored.  Workgroups that share a weight tile get consecutive
// logical ids on the same XCD.  Split-K (SK > 1): workgroup (.., ks) adds up
// k steps [ks KT / SK, (ks + 1) KT / SK) and stores float32 partials
// part[ks][M][N]; gemm_splitk_reduce adds them in split order.
#ifndef KS_TILED_WPE
#define KS_TILED_WPE 1  // waves per SIMD the register budget must allow
#endif
__device__ constexpr int vmcnt_imm(int n) {
  // s_waitcnt immediate: vmcnt = n, expcnt and lgkmcnt not waited for
  return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14);
}

template <int EPI, int ST, int WM, int WN, int NWM, int NWN>
__global__ __launch_bounds__(64 * NWM * NWN) __attribute__((amdgpu_waves_per_eu(KS_TILED_WPE)))
void k_gemm_tiled(int M, int N, int K,
                                                    const bf16_t* __restrict__ A, int lda,
                                                    const bf16_t* __restrict__ Wp, float* out,
                                                    int ldo, const float* res, int ldres,
                                                    bf16_t* ohi, bf16_t* olo, int ldact, int MB,
                                                    int NB, int SK, float* __restrict__ part) {
  constexpr int NWV = NWM * NWN;  // waves: NWM along M, NWN along N
  constexpr int PA = NWM * WM;    // A pieces per step: 16 WM NWM rows
  constexpr int PB = NWN * WN;   // W pieces per step: 16 NWN WN columns
  constexpr int PPW = (PA + PB) / NWV;
  static_assert((PA + PB) % NWV == 0, "pieces split evenly over the waves");
  __shared__ __align__(16) bf16_t Sg[ST][(PA + PB) * 512];
  const int KT = K >> 5;
  const int NT = N >> 4;
  // XCD-aware logical block id (blocks are dealt round-robin over 8 XCDs)
  const int nblk = gridDim.x;
  const int bid = blockIdx.x;
  int lb = bid;
  if ((nblk & 7) == 0) lb = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int mb = lb % MB, nb = (lb / MB) % NB, ks = lb / (MB * NB);
  const int m0 = mb * 16 * WM * NWM, nt0 = nb * PB;
  const int kb = (ks * KT) / SK, nk = ((ks + 1) * KT) / SK - kb;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % NWM, wn = wave / NWM;

  // wave w moves pieces PPW w .. + PPW - 1 of every step: pieces 0..PA-1 are A
  // tiles (rows m0 + 16 p ..), the rest W tiles nt0 + p - PA
  const bf16_t* src[PPW];
  int adv[PPW];  // elements per k step
#pragma unroll
  for (int q = 0; q < PPW; ++q) {
    const int pc = PPW * wave + q;
    if (pc < PA) {
      const int row = min(m0 + 16 * pc + (lane & 15), M - 1);
      src[q] = A + (size_t)row * lda + (size_t)kb * 32 + (lane >> 4) * 8;
      adv[q] = 32;
    } else {
      const int nt = min(nt0 + pc - PA, NT - 1);
      src[q] = Wp + ((size_t)nt * KT + kb) * 512 + lane * 8;
      adv[q] = 512;
    }
  }
  auto issue = [&](int step, int buf) {
#pragma unroll
    for (int q = 0; q < PPW; ++q) {
      const bf16_t* s_ = src[q] + (size_t)step * adv[q];
      __builtin_amdgcn_global_load_lds(
          (const void*)s_,
          (__attribute__((address_space(3))) void*)&Sg[buf][(PPW * wave + q) * 512], 16, 0, 0);
    }
  };
#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < nk) issue(s, s);

  f32x4 acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int t = 0; t < WN; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int it = 0; it < nk; ++it) {
    // step it has landed once at most the ST - 2 later steps are in flight.
    // The barrier then needs no memory fence (a fence would wait for every
    // step in flight): this wave's tile loads for step it are counted down
    // above, and its LDS reads of the stage refilled next were consumed by
    // the previous step's matrix instructions.
    if (it + ST - 2 < nk) __builtin_amdgcn_s_waitcnt(vmcnt_imm(PPW * (ST - 2)));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
    if (it + ST - 1 < nk) issue(it + ST - 1, (it + ST - 1) % ST);
    const bf16_t* Sb = Sg[it % ST];
    bf16x8 a[WM], b[WN];
#pragma unroll
    for (int i = 0; i < WM; ++i) a[i] = ld_frag(&Sb[(WM * wm + i) * 512 + lane * 8]);
#pragma unroll
    for (int t = 0; t < WN; ++t) b[t] = ld_frag(&Sb[(PA + WN * wn + t) * 512 + lane * 8]);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int t = 0; t < WN; ++t)
        acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[t], acc[i][t], 0, 0, 0);
  }

  const int mw = m0 + wm * 16 * WM;
  const int nw = nt0 + wn * WN;
  float* pk = part + (size_t)ks * M * N;
#pragma unroll
  for (int i = 0; i < WM; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = mw + i * 16 + 4 * (lane >> 4) + v;
      if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int t = 0; t < WN; ++t) {
          const float up = __shfl(acc[i][t][v], (lane & 48) | ((lane + 8) & 15));
          if (m >= M || nw + t >= NT || (lane & 15) >= 8) continue;
          const int c = (nw + t) * 8 + (lane & 15);
          store_split(ohi, olo, (size_t)m * ldact + c, silu_mul(acc[i][t][v], up));
        }
      } else {
        if (m >= M) continue;
#pragma unroll
        for (int t = 0; t < WN; ++t) {
          if (nw + t >= NT) continue;
          const int n = (nw + t) * 16 + (lane & 15);
          float sv = acc[i][t][v];
          if (SK > 1) {
            pk[(size_t)m * N + n] = sv;
          } else {
            if (EPI == EPI_RESID) sv += res[(size_t)m * ldres + n];
            out[(size_t)m * ldo + n] = sv;
          }
        }
      }
    }
  }
}

// out[m][n] = (res[m][n] +) sum over ks in order of part[ks][m][n]; N % 4 == 0
template <int EPI>
__global__ __launch_bounds__(256) void k_splitk_reduce(int M, int N, int SK,
                                                       const float* __restrict__ part,
                                                       float* out, int ldo, const float* res,
                                                       int ldres) {
  const size_t i4 = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int n4 = N >> 2;
  if (i4 >= (size_t)M * n4) return;
  const int m = (int)(i4 / n4), n = (int)(i4 % n4) * 4;
  float4 s = *(const float4*)&part[(size_t)m * N + n];
  for (int k = 1; k < SK; ++k) {
    const float4 t = *(const float4*)&part[((size_t)k * M + m) * N + n];
    s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
  }
  if (EPI == EPI_RESID) {
    const float4 r = *(const float4*)&res[(size_t)m * ldres + n];
    s.x = r.x + s.x; s.y = r.y + s.y; s.z = r.z + s.z; s.w = r.w + s.w;
  }
  *(float4*)&out[(size_t)m * ldo + n] = s;
}

static int compute_units() {
  static std::atomic<int> cached[16];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Split-K factor (1..8) of a tiled product, by a cost model fitted on MI355X
// to the 128 x 256 tile at the Llama-8B product shapes (400..1225 rows, every
// factor 1..6 timed): one k step takes about 0.57 us while a workgroup has its
// CU to itself and 0.97 us while two share it (the CU's matrix and LDS
// throughput is then split, so the pair gains only ~15%); workgroups beyond
// the resident set run in further rounds; SK > 1 adds a launch and SK + 2
// float32 M x N planes of traffic (partials written and read, output) at
// about 4.5 TB/s.  The model picks the measured best factor, or one within
// 1 us of it, at every timed shape; split count 1 is kept when the partials
// would not fit the caller's buffer.
static int splitk_factor(const GemmArgs& g, int tiles, int KT, int lds_kib) {
  constexpr double T_ALONE = 0.57, T_SHARED = 0.97, T_LAUNCH = 3.0, BYTES_PER_US = 4.5e6;
  if (g.epi == EPI_SWIGLU || !g.part) return 1;
  const int cus = compute_units();
  const int resident = cus * std::max(1, 160 / lds_kib);
  double best = 0.0;
  int best_sk = 1;
  for (int sk = 1; sk <= 8; ++sk) {
    if (sk > 1 && ((size_t)sk * g.M * g.N * 4 > g.part_bytes || KT / sk < 8)) break;
    const int steps = (KT + sk - 1) / sk;
    double t = 0.0;
    for (long left = (long)tiles * sk; left > 0; left -= resident)
      t += steps * (std::min<long>(left, resident) > cus ? T_SHARED : T_ALONE);
    if (sk > 1) t += T_LAUNCH + (sk + 2.0) * g.M * (double)g.N * 4.0 / BYTES_PER_US;
    if (sk == 1 || t < best) {
      best = t;
      best_sk = sk;
    }
  }
  return best_sk;
}

template <int ST, int WM, int WN, int NWM, int NWN>
static void launch_tiled(const GemmArgs& g, hipStream_t st) {
  const int NT = g.N / 16;
  const int KT = g.K / 32;
  const int MB = (g.M + 16 * WM * NWM - 1) / (16 * WM * NWM);
  const int NB = (NT + NWN * WN - 1) / (NWN * WN);
  const int SK = splitk_factor(g, MB * NB, KT, ST * (WM * NWM + NWN * WN));
  dim3 grid(MB * NB * SK);
  const bf16_t* A = (const bf16_t*)g.A.hi;
  const bf16_t* W = (const bf16_t*)g.W;
  if (g.epi == EPI_SWIGLU)
    KS_LAUNCH((k_gemm_tiled<EPI_SWIGLU, ST, WM, WN, NWM, NWN>), grid, dim3(64 * NWM * NWN), 0, st, g.M, g.N,
              g.K, A, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, (bf16_t*)g.act_out.hi,
              (bf16_t*)g.act_out.lo, g.act_out.ld, MB, NB, 1, g.part);
  else if (g.epi == EPI_RESID)
    KS_LAUNCH((k_gemm_tiled<EPI_RESID, ST, WM, WN, NWM, NWN>), grid, dim3(64 * NWM * NWN), 0, st, g.M, g.N, g.K,
              A, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0, MB, NB,
              SK, g.part);
  else
    KS_LAUNCH((k_gemm_tiled<EPI_STORE, ST, WM, WN, NWM, NWN>), grid, dim3(64 * NWM * NWN), 0, st, g.M, g.N, g.K,
              A, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0, MB, NB,
              SK, g.part);
  if (SK > 1) {
    const size_t n4 = (size_t)g.M * (g.N / 4);
    dim3 rg((unsigned)((n4 + 255) / 256));
    if (g.epi == EPI_RESID)
      KS_LAUNCH(k_splitk_reduce<EPI_RESID>, rg, dim3(256), 0, st, g.M, g.N, SK, g.part,
                g.out, g.ldo, g.res, g.ldres);
    else
      KS_LAUNCH(k_splitk_reduce<EPI_STORE>, rg, dim3(256), 0, st, g.M, g.N, SK, g.part,
                g.out, g.ldo, g.res, g.ldres);
  }
}

// Workgroup tile 128 x 256 (8 waves of 64 x 64), 3 stages: measured on MI355X
// at the selection shapes (400..1225 rows of the Llama-8B products) against
// 128 x 128 / 4 waves (up to 1.3x slower: it moves 33% more operand bytes per
// flop through the CU's load path), 256 x 128, 256 x 256, 64 x 128 wave tiles
// and 2..5 stages.
#ifndef KS_TILED_WM
#define KS_TILED_WM 4
#endif
#ifndef KS_TILED_WN
#define KS_TILED_WN 4
#endif
#ifndef KS_TILED_ST
#define KS_TILED_ST 3
#endif
#ifndef KS_TILED_NWN
#define KS_TILED_NWN 4
#endif
#ifndef KS_TILED_NWM
#define KS_TILED_NWM 2
#endif
void gemm_bf16_tiled(const GemmArgs& g, hipStream_t st) {
  launch_tiled<KS_TILED_ST, KS_TILED_WM, KS_TILED_WN, KS_TILED_NWM, KS_TILED_NWN>(g, st);
}

// --------------------------------------------------------------------- f32
// Plain 16x16 LDS tiles, k ascending; used only by float32 models.
// EPI_SWIGLU: W is [gate rows; up rows], Nout = N/2 outputs.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(int M, int Nout, int K,
                                                  const float* __restrict__ A, int lda,
                                                  const float* __restrict__ W, float* out,
                                                  int ldo, const float* res, int ldres,
                                                  float* aout, int ldact) {
  __shared__ float As[16][17], Ws[16][17], Us[16][17];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int mb = blockIdx.y * 16, nb = blockIdx.x * 16;
  float acc = 0.f, accu = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
    As[ty][tx] = (mb + ty < M) ? A[(size_t)(mb + ty) * lda + k0 + tx] : 0.f;
    Ws[ty][tx] = (nb + ty < Nout) ? W[(size_t)(nb + ty) * K + k0 + tx] : 0.f;
    if (EPI == EPI_SWIGLU)
      Us[ty][tx] = (nb + ty < Nout) ? W[(size_t)(Nout + nb + ty) * K + k0 + tx] : 0.f;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      acc = fmaf(As[ty][kk], Ws[tx][kk], acc);
      if (EPI == EPI_SWIGLU) accu = fmaf(As[ty][kk], Us[tx][kk], accu);
    }
    __syncthreads();
  }
  const int m = mb + ty, n = nb + tx;
  if (m >= M || n >= Nout) return;
  if (EPI == EPI_SWIGLU) {
    aout[(size_t)m * ldact + n] = silu_mul(acc, accu);
  } else {
    if (EPI == EPI_RESID) acc += res[(size_t)m * ldres + n];
    out[(size_t)m * ldo + n] = acc;
  }
}

void gemm_f32(const GemmArgs& g, hipStream_t st) {
  const int Nout = g.epi == EPI_SWIGLU ? g.N / 2 : g.N;
  dim3 grid((Nout + 15) / 16, (g.M + 15) / 16);
  const float* A = (const float*)g.A.hi;
  const float* W = (const float*)g.W;
  if (g.epi == EPI_SWIGLU)
    KS_LAUNCH(k_gemm_f32<EPI_SWIGLU>, grid, dim3(256), 0, st, g.M, Nout, g.K, A,
              g.A.ld, W, g.out, g.ldo, g.res, g.ldres, (float*)g.act_out.hi,
              g.act_out.ld);
  else if (g.epi == EPI_RESID)
    KS_LAUNCH(k_gemm_f32<EPI_RESID>, grid, dim3(256), 0, st, g.M, Nout, g.K, A, g.A.ld,
              W, g.out, g.ldo, g.res, g.ldres, nullptr, 0);
  else
    KS_LAUNCH(k_gemm_f32<EPI_STORE>, grid, dim3(256), 0, st, g.M, Nout, g.K, A, g.A.ld,
              W, g.out, g.ldo, g.res, g.ldres, nullptr, 0);
}

// ----------------------------------------------------------------- packing
// One thread per 8-element (16-byte) fragment of the destination.
// mode 0: plain; 1: gate/up 8 + 8 interleave; 2: q/k/v heads of hd rows with
// tile t of a head holding rows 8t..8t+7 and hd/2 + 8t..hd/2 + 8t + 7
__global__ void k_pack(const bf16_t* __restrict__ src0, const bf16_t* __restrict__ src1,
                       bf16_t* __restrict__ dst, int N, int K, int mode, int hd) {
  const size_t f = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int KT = K >> 5;
  const size_t nfrag = (size_t)N * K / 8;
  if (f >= nfrag) return;
  const int l = (int)(f & 63);
  const size_t tile = f >> 6;
  const int kt = (int)(tile % KT);
  const int nt = (int)(tile / KT);
  const bf16_t* src = src0;
  int row = nt * 16 + (l & 15);
  if (mode == 1) {  // tile t: gate rows 8t..8t+7, then up rows 8t..8t+7
    src = (l & 8) ? src1 : src0;
    row = nt * 8 + (l & 7);
  } else if (mode == 2) {
    const int tph = hd / 16, h = nt / tph, t = nt % tph;
    row = h * hd + 8 * t + (l & 7) + (hd / 2) * ((l >> 3) & 1);
  }
  const u32x4 v = *(const u32x4*)(src + (size_t)row * K + kt * 32 + (l >> 4) * 8);
  *(u32x4*)(dst + f * 8) = v;
}

void pack_matrix_bf16(const bf16_t* src, bf16_t* dst, int N, int K, hipStream_t st) {
  const size_t nfrag = (size_t)N * K / 8;
  KS_LAUNCH(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, src,
            nullptr, dst, N, K, 0, 0);
}

void pack_qkv_bf16(const bf16_t* src, bf16_t* dst, int heads, int hd, int d, hipStream_t st) {
  const size_t nfrag = (size_t)heads * hd * d / 8;
  KS_LAUNCH(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, src,
            nullptr, dst, heads * hd, d, 2, hd);
}

void pack_gate_up_bf16(const bf16_t* gate, const bf16_t* up, bf16_t* dst, int ffn, int d,
                       hipStream_t st) {
  const size_t nfrag = (size_t)2 * ffn * d / 8;
  KS_LAUNCH(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, gate, up,
            dst, 2 * ffn, d, 1, 0);
}

}  // namespace ks
