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
// Tiled path (batched rows of the selection DP and of prefill): a 64x64 wave
// tile of 16x16x32 MFMAs over single bf16 activations.
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
template <int NB, int NW, int CH, int EPI>
__global__ __launch_bounds__(NW * 64) void k_gemm_skinny(
    int M, int N, int K, const bf16_t* __restrict__ Ahi, const bf16_t* __restrict__ Alo,
    int lda, const bf16_t* __restrict__ Wp, float* out, int ldo, const float* res, int ldres,
    bf16_t* ohi, bf16_t* olo, int ldact) {
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
#pragma unroll
  for (int t = 0; t < NB; ++t) red[wave][t][lane] = acc[t];
  __syncthreads();

  if (EPI == EPI_SWIGLU) {
    // tile rows 0..7 are gate rows, 8..15 the matching up rows
    for (int idx = threadIdx.x; idx < NB * 256; idx += NW * 64) {
      const int t = idx >> 8, l = (idx >> 2) & 63, v = idx & 3;
      const int m = 4 * (l >> 4) + v;
      if (m >= M || nt0 + t >= NT || (l & 15) >= 8) continue;
      float g = 0.f, u = 0.f;
      for (int w = 0; w < NW; ++w) {
        g += red[w][t][l][v];
        u += red[w][t][l + 8][v];
      }
      const int c = (nt0 + t) * 8 + (l & 15);
      store_split(ohi, olo, (size_t)m * ldact + c, silu_mul(g, u));
    }
  } else {
    for (int idx = threadIdx.x; idx < NB * 256; idx += NW * 64) {
      const int t = idx >> 8, l = (idx >> 2) & 63, v = idx & 3;
      const int m = 4 * (l >> 4) + v;
      if (m >= M || nt0 + t >= NT) continue;
      float s = 0.f;
      for (int w = 0; w < NW; ++w) s += red[w][t][l][v];
      const int n = (nt0 + t) * 16 + (l & 15);
      if (EPI == EPI_RESID) s += res[(size_t)m * ldres + n];
      out[(size_t)m * ldo + n] = s;
    }
  }
}

template <int NB, int NW, int CH>
static void launch_skinny(const GemmArgs& g, hipStream_t st) {
  const int NT = g.N / 16;
  const bf16_t* Ahi = (const bf16_t*)g.A.hi;
  const bf16_t* Alo = (const bf16_t*)g.A.lo;
  const bf16_t* W = (const bf16_t*)g.W;
  dim3 grid((NT + NB - 1) / NB), block(NW * 64);
  if (g.epi == EPI_SWIGLU)
    hipLaunchKernelGGL((k_gemm_skinny<NB, NW, CH, EPI_SWIGLU>), grid, block, 0, st, g.M, g.N, g.K,
                       Ahi, Alo, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, (bf16_t*)g.act_out.hi,
                       (bf16_t*)g.act_out.lo, g.act_out.ld);
  else if (g.epi == EPI_RESID)
    hipLaunchKernelGGL((k_gemm_skinny<NB, NW, CH, EPI_RESID>), grid, block, 0, st, g.M, g.N, g.K,
                       Ahi, Alo, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0);
  else
    hipLaunchKernelGGL((k_gemm_skinny<NB, NW, CH, EPI_STORE>), grid, block, 0, st, g.M, g.N, g.K,
                       Ahi, Alo, g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0);
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
// Block: 4 waves as 2 (rows) x 2 (cols); wave tile 64 rows x 64 cols.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_tiled(int M, int N, int K,
                                                    const bf16_t* __restrict__ A, int lda,
                                                    const bf16_t* __restrict__ Wp, float* out,
                                                    int ldo, const float* res, int ldres,
                                                    bf16_t* ohi, bf16_t* olo, int ldact) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int KT = K >> 5;
  const int NT = N >> 4;
  const int m0 = blockIdx.y * 128 + (wave & 1) * 64;
  const int nt0 = blockIdx.x * 8 + (wave >> 1) * 4;
  const int kg = lane >> 4;

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  const bf16_t* ap[4];
  bool aok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = m0 + i * 16 + (lane & 15);
    aok[i] = r < M;
    ap[i] = A + (size_t)(aok[i] ? r : 0) * lda + kg * 8;
  }
  const bf16_t* wp[4];
  bool bok[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    bok[t] = nt0 + t < NT;
    wp[t] = Wp + (size_t)(bok[t] ? nt0 + t : 0) * KT * 512 + lane * 8;
  }
  for (int kt = 0; kt < KT; ++kt) {
    bf16x8 a[4], b[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) b[t] = bok[t] ? ld_frag(wp[t] + (size_t)kt * 512) : zero_frag();
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = aok[i] ? ld_frag(ap[i] + kt * 32) : zero_frag();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[i][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[t], acc[i][t], 0, 0, 0);
  }

#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = m0 + i * 16 + 4 * (lane >> 4) + v;
      if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const float up = __shfl(acc[i][t][v], (lane & 48) | ((lane + 8) & 15));
          if (m >= M || !bok[t] || (lane & 15) >= 8) continue;
          const int c = (nt0 + t) * 8 + (lane & 15);
          store_split(ohi, olo, (size_t)m * ldact + c, silu_mul(acc[i][t][v], up));
        }
      } else {
        if (m >= M) continue;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (!bok[t]) continue;
          const int n = (nt0 + t) * 16 + (lane & 15);
          float s = acc[i][t][v];
          if (EPI == EPI_RESID) s += res[(size_t)m * ldres + n];
          out[(size_t)m * ldo + n] = s;
        }
      }
    }
  }
}

void gemm_bf16_tiled(const GemmArgs& g, hipStream_t st) {
  const int NT = g.N / 16;
  dim3 grid((NT + 7) / 8, (g.M + 127) / 128);
  const bf16_t* A = (const bf16_t*)g.A.hi;
  const bf16_t* W = (const bf16_t*)g.W;
  if (g.epi == EPI_SWIGLU)
    hipLaunchKernelGGL(k_gemm_tiled<EPI_SWIGLU>, grid, dim3(256), 0, st, g.M, g.N, g.K, A,
                       g.A.ld, W, g.out, g.ldo, g.res, g.ldres, (bf16_t*)g.act_out.hi,
                       (bf16_t*)g.act_out.lo, g.act_out.ld);
  else if (g.epi == EPI_RESID)
    hipLaunchKernelGGL(k_gemm_tiled<EPI_RESID>, grid, dim3(256), 0, st, g.M, g.N, g.K, A,
                       g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0);
  else
    hipLaunchKernelGGL(k_gemm_tiled<EPI_STORE>, grid, dim3(256), 0, st, g.M, g.N, g.K, A,
                       g.A.ld, W, g.out, g.ldo, g.res, g.ldres, nullptr, nullptr, 0);
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
__global__ void k_pack(const bf16_t* __restrict__ src0, const bf16_t* __restrict__ src1,
                       bf16_t* __restrict__ dst, int N, int K, int interleave) {
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
  if (interleave) {  // tile t: gate rows 8t..8t+7, then up rows 8t..8t+7
    src = (l & 8) ? src1 : src0;
    row = nt * 8 + (l & 7);
  }
  const u32x4 v = *(const u32x4*)(src + (size_t)row * K + kt * 32 + (l >> 4) * 8);
  *(u32x4*)(dst + f * 8) = v;
}

void pack_matrix_bf16(const bf16_t* src, bf16_t* dst, int N, int K, hipStream_t st) {
  const size_t nfrag = (size_t)N * K / 8;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, src,
                     nullptr, dst, N, K, 0);
}

void pack_gate_up_bf16(const bf16_t* gate, const bf16_t* up, bf16_t* dst, int ffn, int d,
                       hipStream_t st) {
  const size_t nfrag = (size_t)2 * ffn * d / 8;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((nfrag + 255) / 256)), dim3(256), 0, st, gate, up,
                     dst, 2 * ffn, d, 1);
}

}  // namespace ks
