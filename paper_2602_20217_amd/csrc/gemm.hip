// Matrix products of the decoder sublayers.
//
// bf16 weights are stored in a tile layout that matches the B-operand registers
// of v_mfma_f32_16x16x32_bf16: a 16 (rows of W) x 32 (k) tile is 1 KiB and lane
// l holds row l%16, k = 8(l/16)..8(l/16)+7 at byte offset 16 l.  One 64-lane
// load therefore reads one contiguous KiB of HBM.
//
// Skinny path (M <= 16 rows: decode, draft, verify): the batch-1 decode step
// is HBM-bound, so every weight byte is read once.  Rows are padded to the 16
// of the matrix instruction; activations enter as two bf16 planes hi + lo
// (two MFMAs per weight fragment, free in the HBM-bound regime) so the product
// keeps ~16 mantissa bits of the float32 activations.  K is split over the
// 16 waves of a workgroup and reduced in LDS in a fixed order, so a row's
// result does not depend on how many rows are in the batch: a verify row and
// the decode step at the same position produce identical bits.
//
// Tiled path (batched rows of the selection DP and of prefill): 128 x 128
// workgroup tiles staged through LDS, 64 x 64 wave tiles of 16x16x32 MFMAs over
// single bf16 activations.
#include "ks_internal.h"

namespace ks {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline bf16x8 ld_frag(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, *(const u32x4*)p);
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
template <int NB, int NW, int CH, int EPI, int AN>
__global__ __launch_bounds__(NW * 64) void k_gemm_skinny(
    int M, int N, int K, const bf16_t* __restrict__ Ahi, const bf16_t* __restrict__ Alo,
    int lda, const bf16_t* __restrict__ Wp, float* out, int ldo, const float* res, int ldres,
    bf16_t* ohi, bf16_t* olo, int ldact, const float* __restrict__ ssq_in, int nssq, float eps,
    const float* __restrict__ next_gain, bf16_t* nhi, bf16_t* nlo, int ldn, float* next_ssq,
    QkvEpi qe) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int KT = K >> 5;
  const int NT = N >> 4;
  const int nt0 = blockIdx.x * NB;
  const int kb = (wave * KT) / NW;
  const int ke = ((wave + 1) * KT) / NW;
  const int row = lane & 15;
  const int kg = lane >> 4;
  const bool rok = row < M;

  f32x4 acc[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bf16_t* ah = Ahi + (size_t)(rok ? row : 0) * lda + kg * 8;
  const bf16_t* al = Alo + (size_t)(rok ? row : 0) * lda + kg * 8;
  const bf16_t* wb[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    int nt = nt0 + t < NT ? nt0 + t : NT - 1;
    wb[t] = Wp + (size_t)nt * KT * 512 + lane * 8;
  }
  // chunks of CH k-steps: every weight fragment of a chunk is requested before
  // the first matrix instruction of the chunk
  for (int kc = kb; kc < ke; kc += CH) {
    const int n = ke - kc < CH ? ke - kc : CH;
    bf16x8 b[NB][CH];
#pragma unroll
    for (int u = 0; u < CH; ++u)
#pragma unroll
      for (int t = 0; t < NB; ++t)
        if (u < n) b[t][u] = ld_frag(wb[t] + (size_t)(kc + u) * 512);
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      if (u < n) {
        bf16x8 a0 = zero_frag(), a1 = zero_frag();
        if (rok) {
          a0 = ld_frag(ah + (kc + u) * 32);
          a1 = ld_frag(al + (kc + u) * 32);
        }
#pragma unroll
        for (int t = 0; t < NB; ++t) {
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b[t][u], acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b[t][u], acc[t], 0, 0, 0);
        }
      }
    }
  }

  __shared__ f32x4 red[NW][NB][64];
  __shared__ float s_rs[AN ? 16 : 1];
#pragma unroll
  for (int t = 0; t < NB; ++t) red[wave][t][lane] = acc[t];
  if (AN) {
    for (int m = wave; m < M; m += NW) {
      float t = 0.f;
      for (int j = lane; j < nssq; j += 64) t += ssq_in[(size_t)m * nssq + j];
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o);
      if (lane == 0) s_rs[m] = 1.0f / sqrtf(t / (float)K + eps);
    }
  }
  __syncthreads();

  if (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
    // tile rows 0..7 pair with rows 8..15 (gate/up, or rotary pairs)
    for (int idx = threadIdx.x; idx < NB * 256; idx += NW * 64) {
      const int t = idx >> 8, l = (idx >> 2) & 63, v = idx & 3;
      const int m = 4 * (l >> 4) + v;
      if (m >= M || nt0 + t >= NT || (l & 15) >= 8) continue;
      float g = 0.f, u = 0.f;
      for (int w = 0; w < NW; ++w) {
        g += red[w][t][l][v];
        u += red[w][t][l + 8][v];
      }
      if (AN) {
        g *= s_rs[m];
        u *= s_rs[m];
      }
      if (EPI == EPI_SWIGLU) {
        const int c = (nt0 + t) * 8 + (l & 15);
        store_split(ohi, olo, (size_t)m * ldact + c, silu_mul(g, u));
      } else {
        const int tph = qe.hd >> 4, half = qe.hd >> 1;
        const int hh = (nt0 + t) / tph;
        const int f = 8 * ((nt0 + t) % tph) + (l & 15);
        const int p = qe.pos[m];
        if (hh < qe.hq + qe.hkv) {
          const float2 cs = *(const float2*)&qe.rope_cs[((size_t)p * half + f) * 2];
          const float y0 = g * cs.x - u * cs.y;
          const float y1 = u * cs.x + g * cs.y;
          if (hh < qe.hq) {
            float* q = qe.q_out + ((size_t)m * qe.hq + hh) * qe.hd;
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
    // thread idx < 256 owns (row 4 (l / 16) + v, column l % 16): in a wave the
    // 16 columns of a row sit on lane bits 2..5, so the tile's sum of squares
    // for the next norm is a 4-step butterfly
    static_assert(EPI != EPI_RESID || NB == 1, "next-norm sums assume one tile per block");
    const bool nn = EPI == EPI_RESID && next_gain != nullptr;
    for (int idx = threadIdx.x; idx < NB * 256; idx += NW * 64) {
      const int t = idx >> 8, l = (idx >> 2) & 63, v = idx & 3;
      const int m = 4 * (l >> 4) + v;
      const bool ok = m < M && nt0 + t < NT;
      const int n = (nt0 + t) * 16 + (l & 15);
      float s = 0.f;
      if (ok) {
        for (int w = 0; w < NW; ++w) s += red[w][t][l][v];
        if (AN) s *= s_rs[m];
        if (EPI == EPI_RESID) s += res[(size_t)m * ldres + n];
        out[(size_t)m * ldo + n] = s;
      }
      if (nn) {
        float sq = s * s;
        if (ok) store_split(nhi, nlo, (size_t)m * ldn + n, s * next_gain[n]);
        sq += __shfl_xor(sq, 4);
        sq += __shfl_xor(sq, 8);
        sq += __shfl_xor(sq, 16);
        sq += __shfl_xor(sq, 32);
        if (ok && (l & 15) == 0) next_ssq[(size_t)m * NT + nt0 + t] = sq;
      }
    }
  }
}

template <int NB, int NW, int CH, int AN>
static void launch_skinny_an(const GemmArgs& g, hipStream_t st) {
  const int NT = g.N / 16;
  const bf16_t* Ahi = (const bf16_t*)g.A.hi;
  const bf16_t* Alo = (const bf16_t*)g.A.lo;
  const bf16_t* W = (const bf16_t*)g.W;
  dim3 grid((NT + NB - 1) / NB), block(NW * 64);
#define KS_SKINNY(E, OH, OL, OLD)                                                            \
  hipLaunchKernelGGL((k_gemm_skinny<NB, NW, CH, E, AN>), grid, block, 0, st, g.M, g.N, g.K,  \
                     Ahi, Alo, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, OH, OL, OLD,         \
                     g.ssq_in, g.nssq, g.eps, g.next_gain, (bf16_t*)g.next_act.hi,           \
                     (bf16_t*)g.next_act.lo, g.next_act.ld, g.next_ssq, g.qe)
  if (g.epi == EPI_SWIGLU)
    KS_SKINNY(EPI_SWIGLU, (bf16_t*)g.act_out.hi, (bf16_t*)g.act_out.lo, g.act_out.ld);
  else if (g.epi == EPI_QKV)
    KS_SKINNY(EPI_QKV, nullptr, nullptr, 0);
  else if (g.epi == EPI_RESID)
    KS_SKINNY(EPI_RESID, nullptr, nullptr, 0);
  else
    KS_SKINNY(EPI_STORE, nullptr, nullptr, 0);
#undef KS_SKINNY
}

template <int NB, int NW, int CH>
static void launch_skinny(const GemmArgs& g, hipStream_t st) {
  if (g.ssq_in) launch_skinny_an<NB, NW, CH, 1>(g, st);
  else launch_skinny_an<NB, NW, CH, 0>(g, st);
}

// Launch shape by matrix shape only (never by row count), measured on MI355X
// with the Llama-8B shapes: the wide products (gate/up, vocabulary head) one
// tile per 8-wave workgroup, the long-K down projection a 16-way K split, the
// remaining square-ish products 16 (N <= 4096) or 8 waves.
void gemm_bf16_skinny(const GemmArgs& g, hipStream_t st) {
  if (g.epi == EPI_SWIGLU) launch_skinny<1, 8, 8>(g, st);
  else if (g.K >= 8192) launch_skinny<1, 16, 8>(g, st);
  else if (g.N >= 65536) launch_skinny<1, 8, 8>(g, st);
  else if (g.N <= 4096) launch_skinny<1, 16, 8>(g, st);
  else launch_skinny<1, 8, 8>(g, st);
}

// ------------------------------------------------------------------- tiled
// Batched rows (prefill chunks, selection DP).  Workgroup tile 128 rows x 128
// columns, 4 waves as 2 x 2 with 64 x 64 wave tiles (4 x 4 MFMAs).  Each
// 32-wide k step of A and W is staged in LDS in the MFMA operand order (A:
// row l%16, k 8(l/16).. of each 16-row tile at byte 16 l; W already arrives in
// that order), so every fragment read is one conflict-free 16-byte LDS read.
// The next step's global loads are in flight while the current step's MFMAs
// run (double-buffered LDS, one barrier per step).  Workgroups that share a
// weight tile get consecutive logical ids on the same XCD, so the XCD's L2
// serves the reuse across row blocks.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_tiled(int M, int N, int K,
                                                    const bf16_t* __restrict__ A, int lda,
                                                    const bf16_t* __restrict__ Wp, float* out,
                                                    int ldo, const float* res, int ldres,
                                                    bf16_t* ohi, bf16_t* olo, int ldact, int MB) {
  __shared__ __align__(16) bf16_t As[2][8 * 512];
  __shared__ __align__(16) bf16_t Bs[2][8 * 512];
  const int KT = K >> 5;
  const int NT = N >> 4;
  // XCD-aware logical block id (blocks are dealt round-robin over 8 XCDs)
  const int nblk = gridDim.x;
  const int bid = blockIdx.x;
  int lb = bid;
  if ((nblk & 7) == 0) lb = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int mb = lb % MB, nb = lb / MB;
  const int m0 = mb * 128, nt0 = nb * 8;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;

  // staging map: chunk c in [0, 512) of 16 bytes, two per thread per operand
  //   A: row c/4, k chunk c%4  -> tile row/16, lane (row%16) + 16 (c%4)
  //   W: tile c/64, lane c%64
  const int c0 = tid, c1 = tid + 256;
  const int ar0 = m0 + (c0 >> 2), ar1 = m0 + (c1 >> 2);
  const bool ak0 = ar0 < M, ak1 = ar1 < M;
  const bf16_t* as0 = A + (size_t)(ak0 ? ar0 : 0) * lda + (c0 & 3) * 8;
  const bf16_t* as1 = A + (size_t)(ak1 ? ar1 : 0) * lda + (c1 & 3) * 8;
  const int ad0 = ((c0 >> 2) >> 4) * 512 + (((c0 >> 2) & 15) + 16 * (c0 & 3)) * 8;
  const int ad1 = ((c1 >> 2) >> 4) * 512 + (((c1 >> 2) & 15) + 16 * (c1 & 3)) * 8;
  const bool bk0 = nt0 + (c0 >> 6) < NT, bk1 = nt0 + (c1 >> 6) < NT;
  const bf16_t* bs0 = Wp + (size_t)(bk0 ? nt0 + (c0 >> 6) : 0) * KT * 512 + (c0 & 63) * 8;
  const bf16_t* bs1 = Wp + (size_t)(bk1 ? nt0 + (c1 >> 6) : 0) * KT * 512 + (c1 & 63) * 8;
  const int bd0 = (c0 >> 6) * 512 + (c0 & 63) * 8;
  const int bd1 = (c1 >> 6) * 512 + (c1 & 63) * 8;
  // sources are clamped to valid rows/tiles; out-of-range chunks are zeroed
  // after the load (a load is never skipped, so no pointer select is formed)
  const uint32_t am0 = ak0 ? ~0u : 0u, am1 = ak1 ? ~0u : 0u;
  const uint32_t bm0 = bk0 ? ~0u : 0u, bm1 = bk1 ? ~0u : 0u;
#define KS_MASK4(v, m) make_uint4((v).x & (m), (v).y & (m), (v).z & (m), (v).w & (m))
  uint4 ra0 = *(const uint4*)as0, ra1 = *(const uint4*)as1;
  uint4 rb0 = *(const uint4*)bs0, rb1 = *(const uint4*)bs1;
  ra0 = KS_MASK4(ra0, am0);
  ra1 = KS_MASK4(ra1, am1);
  rb0 = KS_MASK4(rb0, bm0);
  rb1 = KS_MASK4(rb1, bm1);
  *(uint4*)&As[0][ad0] = ra0;
  *(uint4*)&As[0][ad1] = ra1;
  *(uint4*)&Bs[0][bd0] = rb0;
  *(uint4*)&Bs[0][bd1] = rb1;
  __syncthreads();

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < KT;
    if (more) {
      ra0 = *(const uint4*)(as0 + (kt + 1) * 32);
      ra1 = *(const uint4*)(as1 + (kt + 1) * 32);
      rb0 = *(const uint4*)(bs0 + (size_t)(kt + 1) * 512);
      rb1 = *(const uint4*)(bs1 + (size_t)(kt + 1) * 512);
      ra0 = KS_MASK4(ra0, am0);
      ra1 = KS_MASK4(ra1, am1);
      rb0 = KS_MASK4(rb0, bm0);
      rb1 = KS_MASK4(rb1, bm1);
    }
    bf16x8 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = ld_frag(&As[cur][(4 * wm + i) * 512 + lane * 8]);
#pragma unroll
    for (int t = 0; t < 4; ++t) b[t] = ld_frag(&Bs[cur][(4 * wn + t) * 512 + lane * 8]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[t], acc[i][t], 0, 0, 0);
    if (more) {
      *(uint4*)&As[cur ^ 1][ad0] = ra0;
      *(uint4*)&As[cur ^ 1][ad1] = ra1;
      *(uint4*)&Bs[cur ^ 1][bd0] = rb0;
      *(uint4*)&Bs[cur ^ 1][bd1] = rb1;
    }
    __syncthreads();
  }

#undef KS_MASK4
  const int mw = m0 + wm * 64;
  const int nw = nt0 + wn * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = mw + i * 16 + 4 * (lane >> 4) + v;
      if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const float up = __shfl(acc[i][t][v], (lane & 48) | ((lane + 8) & 15));
          if (m >= M || nw + t >= NT || (lane & 15) >= 8) continue;
          const int c = (nw + t) * 8 + (lane & 15);
          store_split(ohi, olo, (size_t)m * ldact + c, silu_mul(acc[i][t][v], up));
        }
      } else {
        if (m >= M) continue;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (nw + t >= NT) continue;
          const int n = (nw + t) * 16 + (lane & 15);
          float sv = acc[i][t][v];
          if (EPI == EPI_RESID) sv += res[(size_t)m * ldres + n];
          out[(size_t)m * ldo + n] = sv;
        }
      }
    }
  }
}

void gemm_bf16_tiled(const GemmArgs& g, hipStream_t st) {
  const int NT = g.N / 16;
  const int MB = (g.M + 127) / 128;
  const int NBk = (NT + 7) / 8;
  dim3 grid(MB * NBk);
  const bf16_t* A = (const bf16_t*)g.A.hi;
  const bf16_t* W = (const bf16_t*)g.W;
  if (g.epi == EPI_SWIGLU)
    hipLaunchKernelGGL(k_gemm_tiled<EPI_SWIGLU>, grid, dim3(256), 0, st, g.M, g.N, g.K, A,
                       g.A.ld, W, g.out, g.ldo, g.res, g.ldres, (bf16_t*)g.act_out.hi,
                       (bf16_t*)g.act_out.lo, g.act_out.ld, MB);
  else if (g.epi == EPI_RESID)
    hipLaunchKernelGGL(k_gemm_tiled<EPI_RESID>, grid, dim3(256), 0, st, g.M, g.N, g.K, A,
                       g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0, MB);
  else
    hipLaunchKernelGGL(k_gemm_tiled<EPI_STORE>, grid, dim3(256), 0, st, g.M, g.N, g.K, A,
                       g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0, MB);
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
    hipLaunchKernelGGL(k_gemm_f32<EPI_SWIGLU>, grid, dim3(256), 0, st, g.M, Nout, g.K, A,
                       g.A.ld, W, g.out, g.ldo, g.res, g.ldres, (float*)g.act_out.hi,
                       g.act_out.ld);
  else if (g.epi == EPI_RESID)
    hipLaunchKernelGGL(k_gemm_f32<EPI_RESID>, grid, dim3(256), 0, st, g.M, Nout, g.K, A, g.A.ld,
                       W, g.out, g.ldo, g.res, g.ldres, nullptr, 0);
  else
    hipLaunchKernelGGL(k_gemm_f32<EPI_STORE>, grid, dim3(256), 0, st, g.M, Nout, g.K, A, g.A.ld,
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
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, src,
                     nullptr, dst, N, K, 0, 0);
}

void pack_qkv_bf16(const bf16_t* src, bf16_t* dst, int heads, int hd, int d, hipStream_t st) {
  const size_t nfrag = (size_t)heads * hd * d / 8;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, src,
                     nullptr, dst, heads * hd, d, 2, hd);
}

void pack_gate_up_bf16(const bf16_t* gate, const bf16_t* up, bf16_t* dst, int ffn, int d,
                       hipStream_t st) {
  const size_t nfrag = (size_t)2 * ffn * d / 8;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, gate, up,
                     dst, 2 * ffn, d, 1, 0);
}

}  // namespace ks
