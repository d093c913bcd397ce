// GQA attention of the decoder's attention sublayers (Section 2, the
// attention sublayer of each block) over a contiguous KV cache
// [layer][K | V][kv head][position][dim], split over the context.  Each split
// kernel writes a partial (o, max, sum) per (row, query head, split) and
// k_attn_combine merges the splits of a row in ascending order.
//
//  k_attn_dec      decode and verify rows, bf16 caches of up to 12288
//                  positions: splits of 2, 3 or 5 tiles of 64 keys (by cache
//                  size), one tile per wave, scores and P V on matrix
//                  instructions.
//  k_attn_stream   decode and verify rows, bf16 caches above 12288 positions:
//                  each wave walks several tiles of its split with the next
//                  tile's loads in flight.
//  k_attn_bat      batched rows (prefill chunks, the selection's candidate
//                  rows), bf16 caches: query blocks of several rows against a
//                  ring of key/value tiles.
//  k_attn_split    every other case, on the vector ALU: the float32 caches
//                  (head dim 64) of the float32 models and head shapes the
//                  matrix kernels do not take.
//  k_attn_combine  the split merge (plus, for selection rows, the row's own
//                  key and value).
//
// A row's arithmetic depends only on its own query, its length and the split
// size, never on the other rows of the launch, so the decode step and a verify
// row at the same position produce the same bits.
#include "ks_internal.h"

#include <cfloat>

namespace ks {

constexpr int TILE = 64;  // positions per LDS tile of the split kernel

// Workgroups are dealt to the 8 XCDs round-robin by linear id (id mod 8), and
// each XCD has its own L2.  With 8 kv heads, k_attn_dec runs on a
// one-dimensional grid of 8 ns workgroups that keeps every split of kv head h
// on XCD h, and the merge launch places the query heads of kv head h there
// too, so the split partials it reads were written through its own L2.
// (Decode step at 8K: 3.07 -> 3.03 ms against the two-dimensional grid.)
struct SplitId {
  int split, kvh;
};
__device__ inline SplitId split_id(int xmap) {
  if (xmap) return SplitId{(int)(blockIdx.x >> 3), (int)(blockIdx.x & 7)};
  return SplitId{(int)blockIdx.x, (int)blockIdx.y};
}
#ifndef KS_BAT_NW
#define KS_BAT_NW 8  // waves (16 query vectors each) per batched workgroup
#endif
#ifndef KS_BAT_ST
#define KS_BAT_ST 2  // LDS ring stages of the batched kernel
#endif
#ifndef KS_BAT_CB
#define KS_BAT_CB 1  // 16-vector query blocks per wave of the batched kernel
#endif

// s_waitcnt immediate: vmcnt = n, expcnt and lgkmcnt not waited for
__device__ constexpr int vmcnt_imm_a(int n) {
  return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14);
}

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

// Vector-ALU split kernel.  Grid: (split, kv head, row group); a workgroup
// owns `tiles` consecutive 64-position tiles of one kv head.  K rows are
// padded by four 32-bit words in LDS so that 16-byte reads of 64 different
// rows cover all banks.  Each wave owns a fixed set of query vectors (the G =
// hq / hkv query heads of a row share the tile); a lane scores one key,
// softmax statistics use wave shuffles, and the output accumulation
// broadcasts each probability with a lane read.
// HD: head dim (128 for bf16 caches, 64 for float32 caches).  QMAX: query
// vectors per wave (rows_per_block * G <= 4 QMAX).
//
// The first tile's keys/values, the queries and the row lengths are requested
// together at the start, so a workgroup waits for one memory round trip before
// its arithmetic.  The workgroup's query vectors are staged in LDS once (read
// back as broadcasts).  Tiles are double-buffered through registers: the loads
// of tile k + 1 are issued before the arithmetic of tile k.  A lane loads its
// key row from LDS once per tile and scores it against each of its wave's
// queries; the value pass always runs over the 64 rows of a tile (rows past the
// end are zero and carry probability 0), so its loop is unrolled and its LDS
// reads are in flight together.
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
  __shared__ __align__(16) float Qs[4 * QMAX * HD];

  const int split = blockIdx.x, kvh = blockIdx.y;
  const int r0 = blockIdx.z * rows_per_block;
  const int r1 = min(M, r0 + rows_per_block);
  const int G = hq / hkv;
  const int nq = (r1 - r0) * G;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int start = split * tiles * TILE;
  const float scale = 1.0f / sqrtf((float)HD);

  const size_t es = BF ? 2 : 4;
  const char* kbase = (const char*)kc + (size_t)kvh * n_max * HD * es;
  const char* vbase = (const char*)vc + (size_t)kvh * n_max * HD * es;
  static_assert(NCH == 4, "four 16-byte chunks per thread per matrix");
  // named registers (an array carried around the tile loop lands in scratch)
  uint4 k0, k1, k2, k3, v0, v1, v2, v3;
  // Tile loads clamp rows to the cache only, so the first tile is requested
  // before the row lengths arrive; rows at or past the end are zeroed when the
  // tile is stored to LDS (their scores are masked, their values weigh 0).
#define KS_LD(U, KD, VD, T0)                                               \
  {                                                                        \
    const int c_ = threadIdx.x + 256 * (U);                                \
    const int row_ = min((T0) + c_ / CPR, n_max - 1), ch_ = c_ % CPR;      \
    const size_t off_ = (size_t)row_ * HD * es + ch_ * 16;                 \
    KD = *(const uint4*)(kbase + off_);                                    \
    VD = *(const uint4*)(vbase + off_);                                    \
  }
#define KS_FETCH(T0)                                                       \
  KS_LD(0, k0, v0, T0) KS_LD(1, k1, v1, T0) KS_LD(2, k2, v2, T0) KS_LD(3, k3, v3, T0)
#define KS_ST(U, KD, VD, CNT)                                              \
  {                                                                        \
    const int c_ = threadIdx.x + 256 * (U);                                \
    const int row_ = c_ / CPR, ch_ = c_ % CPR;                             \
    const uint32_t m_ = row_ < (CNT) ? ~0u : 0u; /* mask, not a select */ \
    *(uint4*)&Ks[row_ * KS + ch_ * 4] =                                    \
        make_uint4(KD.x & m_, KD.y & m_, KD.z & m_, KD.w & m_);            \
    *(uint4*)&Vs[row_ * KW + ch_ * 4] =                                    \
        make_uint4(VD.x & m_, VD.y & m_, VD.z & m_, VD.w & m_);            \
  }
  KS_FETCH(start);
  // query vector j of the workgroup: row r0 + j / G, head kvh * G + j % G
  for (int e = threadIdx.x; e < nq * HD; e += 256) {
    const int j = e / HD, c = e % HD;
    Qs[e] = q[((size_t)(r0 + j / G) * hq + kvh * G + j % G) * HD + c];
  }

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

  for (int tile = 0; tile < ntile; ++tile) {
    const int t0 = start + tile * TILE;
    const int cnt = min(TILE, maxlen - t0);
    KS_ST(0, k0, v0, cnt) KS_ST(1, k1, v1, cnt) KS_ST(2, k2, v2, cnt) KS_ST(3, k3, v3, cnt)
    __syncthreads();
    if (tile + 1 < ntile) KS_FETCH(t0 + TILE);

    // scores: lane = key t0 + lane
    uint4 krow[KW / 4];
#pragma unroll
    for (int w4 = 0; w4 < KW / 4; ++w4) krow[w4] = *(const uint4*)&Ks[lane * KS + 4 * w4];
    float p[QMAX];
#pragma unroll
    for (int j = 0; j < QMAX; ++j) {
      p[j] = 0.f;
      const int qi = wave + 4 * j;
      if (qi >= nq) continue;
      const int vcnt = min(TILE, len[r0 + qi / G] - t0);
      if (vcnt <= 0) continue;
      const float* qv = &Qs[qi * HD];
      // four interleaved partial sums (shorter dependency chains), added in a
      // fixed order
      float sp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w4 = 0; w4 < KW / 4; ++w4) {
        const uint4 a = krow[w4];
        float& acc = sp[w4 & 3];
        if (BF) {
          const float4 qa = *(const float4*)(qv + 8 * w4);
          const float4 qb = *(const float4*)(qv + 8 * w4 + 4);
          acc = fmaf(qa.x, lo16(a.x), acc); acc = fmaf(qa.y, hi16(a.x), acc);
          acc = fmaf(qa.z, lo16(a.y), acc); acc = fmaf(qa.w, hi16(a.y), acc);
          acc = fmaf(qb.x, lo16(a.z), acc); acc = fmaf(qb.y, hi16(a.z), acc);
          acc = fmaf(qb.z, lo16(a.w), acc); acc = fmaf(qb.w, hi16(a.w), acc);
        } else {
          const float4 qa = *(const float4*)(qv + 4 * w4);
          acc = fmaf(qa.x, __uint_as_float(a.x), acc); acc = fmaf(qa.y, __uint_as_float(a.y), acc);
          acc = fmaf(qa.z, __uint_as_float(a.z), acc); acc = fmaf(qa.w, __uint_as_float(a.w), acc);
        }
      }
      float s0 = (sp[0] + sp[1]) + (sp[2] + sp[3]);
      s0 = lane < vcnt ? s0 * scale : -FLT_MAX;
      const float mt = wave_max(s0);
      const float mnew = fmaxf(mrun[j], mt);
      const float alpha = __expf(mrun[j] - mnew);
      p[j] = lane < vcnt ? __expf(s0 - mnew) : 0.f;
      lrun[j] = lrun[j] * alpha + wave_sum(p[j]);
      mrun[j] = mnew;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] *= alpha;
    }
    // values: every row of the tile, each value word read once per wave
#pragma unroll 16
    for (int t = 0; t < TILE; ++t) {
      const uint32_t vw = Vs[t * KW + lane];
#pragma unroll
      for (int j = 0; j < QMAX; ++j) {
        if (wave + 4 * j >= nq) continue;
        const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p[j]), t));
        if (BF) {
          o[j][0] = fmaf(pt, lo16(vw), o[j][0]);
          o[j][DPL - 1] = fmaf(pt, hi16(vw), o[j][DPL - 1]);
        } else {
          o[j][0] = fmaf(pt, __uint_as_float(vw), o[j][0]);
        }
      }
    }
    __syncthreads();
  }

#undef KS_FETCH
#undef KS_LD
#undef KS_ST
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

typedef __bf16 bf16x8_d __attribute__((ext_vector_type(8)));
typedef float f32x4_d __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_d __attribute__((ext_vector_type(4)));

typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_d;

// Decode / verify rows of bf16 caches with head dim 128, all products on
// matrix instructions.  A workgroup of S waves owns S consecutive 64-key tiles
// of one kv head and RB = 16 CB / G consecutive rows: its 16 CB query columns
// are c = row * G + g (row < RB, G query heads per kv head) in CB blocks of 16,
// so the rows of a verify pass share every key/value load.  Wave w owns tile w:
// it requests its queries, then 16 KiB of keys, then 16 KiB of values, the
// tiles with direct global-to-LDS loads (no staging registers), and scores the
// keys while the values are still arriving.  Rows are stored unpadded with
// 16-byte chunk c of row r at slot c ^ (r % 16).
//  scores  S^T = K Q^T per column block, keys as rows of 16x16x32 products
//          (queries as hi + lo bf16 columns): lane (j, g) holds keys
//          16 kt + 4 g + v of column j of the block, so the tile max and sum
//          need two cross-lane steps; a column only counts keys below its
//          row's length;
//  values  O = P V with the probabilities (bf16) taken from the score registers
//          as the A operand: k slot e of lane group g is key 4 g + e (e < 4) or
//          16 + 4 g + e - 4 (e >= 4) of a 32-key step.  The V operand in that
//          key order comes from transposing LDS reads (a 16-lane group turns
//          16 8-byte row pieces into 4 keys x 16 dims), shared by the column
//          blocks.  Rows at or past the longest length of the workgroup are
//          zeroed in LDS first (probability 0 must not meet a non-finite stale
//          value).
// The S tile results meet in LDS and the whole workgroup merges them in tile
// order into the split's partial (o, max, sum) per query column, the layout
// k_attn_combine reads.  (Merging the splits inside this launch instead, in
// the workgroup that draws the last of a per-kv-head ticket, costs more than
// the second launch, with a release fence per workgroup and also without one:
// partials stored at device scope, the wait for their acknowledgement, the
// ticket and the device-scope loads of all partials trail the split
// workgroups by more than the merge kernel takes.)
// A column's arithmetic depends only on its own query, its length and the
// split size, never on the other columns or on CB, so a verify row and the
// decode step at the same position give the same bits.
template <int S, int CB>
__global__ __launch_bounds__(64 * S) void k_attn_dec(
    int M, int hq, int hkv, int n_max, const float* __restrict__ q,
    const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const int32_t* __restrict__ len, float* __restrict__ part, int nsplit, int span, int xmap) {
  constexpr int HD = 128;
  constexpr int RS = HD + 4;  // LDS merge record per column: o, max, sum (bank-shifted)
  constexpr int NCOL = 16 * CB;
  static_assert(CB == 1 || CB == 2, "one or two column blocks");
  static_assert(16 * RS + NCOL * (S + 3) <= TILE * 64, "records and scratch fit a tile");
  __shared__ __align__(16) uint4 Ks[S][TILE * 16];
  __shared__ __align__(16) uint4 Vs[S][TILE * 16];
  // once every wave is past its tiles: wave w's key tile holds the records of
  // column block 0, its value tile those of block 1; wave 0's key tile also
  // holds the row length of every column after its records
  int* s_len = (int*)((float*)&Ks[0][0] + 16 * RS);  // [NCOL] row length per column
  const SplitId sid = split_id(xmap);
  const int split = sid.split, kvh = sid.kvh;
  const int G = hq / hkv;
  const int RB = NCOL / G;
  const int r0 = blockIdx.z * RB;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the split covers [start, send), span = S TILE positions
  const int start = split * span;
  const int send = start + span;
  const int t0 = start + w * TILE;
  const int nc = min(NCOL, (M - r0) * G);  // query columns with a row

  // column 16 b + j of the workgroup (j = lane % 16): row r0 + (16 b + j) / G,
  // head kvh G + j % G, dims 32 ks + 8 g .. + 7 (g = lane / 16)
  const int j = lane & 15, g = lane >> 4;
  float4 xq[CB][8];
  int Lj[CB];
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    const int rj = r0 + (16 * b + j) / G;
    const bool qok = rj < M;
    const float* qv = q + ((size_t)(qok ? rj : r0) * hq + kvh * G + j % G) * HD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      xq[b][2 * ks] = *(const float4*)(qv + 32 * ks);
      xq[b][2 * ks + 1] = *(const float4*)(qv + 32 * ks + 4);
    }
    // this column's row length (0: no row); loaded unconditionally at a valid
    // row, so the compiler's wait for it counts only the loads issued before it
    const int lv = len[qok ? rj : r0];
    Lj[b] = qok ? lv : 0;
  }
  // piece i (1 KiB): rows 4 i .. + 3 of the tile; lane l writes chunk slot
  // l % 16 of row 4 i + l / 16
  // (cache-policy operand 2 = nt: the cache is streamed once per step, so its
  // lines are not kept in L2 ahead of the query, sums and partials)
  {
    const bf16_t* kb = kc + (size_t)kvh * n_max * HD;
    const bf16_t* vb = vc + (size_t)kvh * n_max * HD;
    const int rr0 = lane >> 4, slot = lane & 15;
    const int rlast = min(send, n_max) - 1;  // rows past the split re-read its last row
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int rr = 4 * i + rr0;
      const int row = min(t0 + rr, rlast);
      __builtin_amdgcn_global_load_lds(
          (const void*)(kb + (size_t)row * HD + ((slot ^ (rr & 15)) << 3)),
          (__attribute__((address_space(3))) void*)&Ks[w][i * 64], 16, 0, 2);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int rr = 4 * i + rr0;
      const int row = min(t0 + rr, rlast);
      __builtin_amdgcn_global_load_lds(
          (const void*)(vb + (size_t)row * HD + ((slot ^ (rr & 15)) << 3)),
          (__attribute__((address_space(3))) void*)&Vs[w][i * 64], 16, 0, 2);
    }
  }
  int Lmax = 0;  // longest row of the workgroup
  for (int r = r0; r < min(M, r0 + RB); ++r) Lmax = max(Lmax, len[r]);
  // keys of this tile any column uses (may be <= 0)
  const int cnt = min(TILE, min(Lmax, send) - t0);
  // queries as hi + lo bf16 (waits for the query loads only), scaled by
  // log2(e) / sqrt(HD): scores in base-2 units, probabilities powers of two
  const float qscale = 1.4426950408889634f / sqrtf((float)HD);
  bf16x8_d qh[CB][4], ql[CB][4];
#pragma unroll
  for (int b = 0; b < CB; ++b)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const float4 x0 = xq[b][2 * ks], x1 = xq[b][2 * ks + 1];
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = Lj[b] > 0 ? xs[e] * qscale : 0.f;
        const __bf16 h = (__bf16)x;
        qh[b][ks][e] = h;
        ql[b][ks][e] = (__bf16)(x - (float)h);
      }
    }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm_a(16));  // keys have landed

  float m[CB], l[CB];
  f32x4_d o[CB][8], sc[CB][4];
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    m[b] = -FLT_MAX;
    l[b] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[b][dt] = f32x4_d{0.f, 0.f, 0.f, 0.f};
  }
  if (cnt > 0) {
    // S^T: sc[b][kt][v] = score(key 16 kt + 4 g + v, column 16 b + j)
    const uint4* Kt = &Ks[w][0];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int b = 0; b < CB; ++b) sc[b][kt] = f32x4_d{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int c = 4 * ks + g;  // 16-byte chunk of the key row
        const bf16x8_d kf = __builtin_bit_cast(bf16x8_d, Kt[(16 * kt + j) * 16 + (c ^ j)]);
#pragma unroll
        for (int b = 0; b < CB; ++b) {
          sc[b][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qh[b][ks], sc[b][kt], 0, 0, 0);
          sc[b][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, ql[b][ks], sc[b][kt], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      const int cj = min(TILE, min(Lj[b], send) - t0);  // keys of this tile the column uses
      float mt = -FLT_MAX;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          sc[b][kt][v] = 16 * kt + 4 * g + v < cj ? sc[b][kt][v] : -FLT_MAX;
          mt = fmaxf(mt, sc[b][kt][v]);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float p = 16 * kt + 4 * g + v < cj ? __builtin_amdgcn_exp2f(sc[b][kt][v] - mt) : 0.f;
          sc[b][kt][v] = p;
          ps += p;
        }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      m[b] = mt;
      l[b] = ps;
    }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm_a(0));  // values have landed
  if (cnt > 0) {
    uint4* Vt = &Vs[w][0];
    if (cnt < TILE) {
      for (int c = cnt * 16 + lane; c < TILE * 16; c += 64) Vt[c] = make_uint4(0u, 0u, 0u, 0u);
    }
    // transposing reads: lane 16 g + 4 s + u points at the 8-byte piece of V row
    // 32 k2 + 16 h + 4 g + s, dims 16 dt + 4 u .. + 3
    const int s4 = (lane & 15) >> 2, u4 = lane & 3;
    const char* Vb = (const char*)Vt;
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      bf16x8_d pa[CB];
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          pa[b][v] = (__bf16)sc[b][2 * k2][v];
          pa[b][4 + v] = (__bf16)sc[b][2 * k2 + 1][v];
        }
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        bf16x4_d h2[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int row = 32 * k2 + 16 * h + 4 * g + s4;
          const int c = 2 * dt + (u4 >> 1);
          const char* pp = Vb + row * 256 + ((c ^ (row & 15)) << 4) + ((u4 & 1) << 3);
          h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (__attribute__((address_space(3))) bf16x4_d*)pp);
        }
        bf16x8_d vb;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vb[e] = h2[0][e];
          vb[4 + e] = h2[1][e];
        }
#pragma unroll
        for (int b = 0; b < CB; ++b)
          o[b][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[b], vb, o[b][dt], 0, 0, 0);
      }
    }
  }
  // tile results to LDS: o[b][dt][v] is column 16 b + 4 g + v, dim 16 dt + j;
  // the max and sum of column 16 b + c live in lane c.  A wave overwrites only
  // its own tiles (LDS accesses of a wave stay in order).
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    float* rec = b == 0 ? (float*)&Ks[w][0] : (float*)&Vs[w][0];
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) rec[(4 * g + v) * RS + 16 * dt + j] = o[b][dt][v];
    if (lane < 16) {
      rec[lane * RS + HD] = m[b];
      rec[lane * RS + HD + 1] = l[b];
    }
  }
  if (threadIdx.x < nc) s_len[threadIdx.x] = CB == 1 || threadIdx.x < 16 ? Lj[0] : Lj[CB - 1];
  __syncthreads();
  auto record = [&](int s, int c) -> const float* {
    return (c < 16 ? (const float*)&Ks[s][0] : (const float*)&Vs[s][0]) + (c & 15) * RS;
  };
  // the split's partial of every column whose row reaches this split: the
  // threads are dealt out over the columns (tpc per column); each forms its
  // column's common max and tile weights once, then its dims d = k, k + tpc, ..
  // (one barrier; the arithmetic per dim is the same for any thread count)
  const int tpc = (64 * S) / nc;
  const int c = threadIdx.x / tpc, k = threadIdx.x - c * tpc;
  if (c < nc && s_len[c] > start) {
    float ms[S], wt[S];
    float mx = -FLT_MAX;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      ms[s] = record(s, c)[HD];
      mx = fmaxf(mx, ms[s]);
    }
#pragma unroll
    for (int s = 0; s < S; ++s) wt[s] = ms[s] == -FLT_MAX ? 0.f : __builtin_amdgcn_exp2f(ms[s] - mx);
    float* dst = part + (((size_t)(r0 + c / G) * hq + kvh * G + c % G) * nsplit + split) * (HD + 2);
    for (int d = k; d < HD; d += tpc) {
      float acc = 0.f;
#pragma unroll
      for (int s = 0; s < S; ++s) acc = fmaf(record(s, c)[d], wt[s], acc);
      dst[d] = acc;
    }
    if (k == 0) {
      float lx = 0.f;
#pragma unroll
      for (int s = 0; s < S; ++s) lx = fmaf(record(s, c)[HD + 1], wt[s], lx);
      dst[HD] = mx * 0.6931471805599453f;  // back to natural-log units
      dst[HD + 1] = lx;
    }
  }
}

// Decode / verify rows over long bf16 caches (head dim 128): a streaming
// variant of k_attn_dec.  A workgroup of NW waves owns NW * tpw consecutive
// 64-key tiles of one kv head (the split) and the same 16 CB query columns as
// k_attn_dec.  Wave w walks tiles i NW + w (i < tpw, stopping at the longest
// row of the workgroup); the key fragment of a 16x16x32 product is 16
// contiguous bytes per lane, so keys go straight from memory into registers,
// and values through the wave's own two-stage LDS ring (direct global-to-LDS
// loads, rows at slot c ^ (r % 16)).  Tile i + 1's keys and values are
// requested before tile i is computed, so every wave keeps two tiles in
// flight and no barrier is needed until the end.  Per tile: S^T = K Q^T on
// matrix instructions, an online base-2 softmax per column (queries
// pre-scaled by log2(e) / sqrt(HD); keys masked only in tiles that reach past
// the shortest column of the wave; the running output rescaled only when some
// column's max moved, as the factor is otherwise exactly 1), then O += P V with
// the value operand from transposing LDS reads.  The NW wave results are merged
// in wave order into the split's partial, exactly as in k_attn_dec.  A column's
// arithmetic depends only on its own query, its length and the split size, so
// a verify row and the decode step at the same position give the same bits.
template <int NW, int CB>
__global__ __launch_bounds__(64 * NW) void k_attn_stream(
    int M, int hq, int hkv, int n_max, const float* __restrict__ q,
    const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const int32_t* __restrict__ len, float* __restrict__ part, int nsplit, int tpw, int xmap) {
  constexpr int HD = 128;
  constexpr int RS = HD + 4;  // LDS merge record per column: o, max, sum (bank-shifted)
  constexpr int NCOL = 16 * CB;
  static_assert(CB == 1 || CB == 2, "one or two column blocks");
  static_assert(16 * RS + NCOL * (NW + 3) <= TILE * 64, "records and scratch fit a stage");
  // the two ring stages are separate arrays, so the compiler can tell that the
  // loads into one stage never alias reads of the other
  __shared__ __align__(16) uint4 Vr0[NW][TILE * 16];
  __shared__ __align__(16) uint4 Vr1[NW][TILE * 16];
  const SplitId sid = split_id(xmap);
  const int split = sid.split, kvh = sid.kvh;
  const int G = hq / hkv;
  const int RB = NCOL / G;
  const int r0 = blockIdx.z * RB;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int start = split * NW * tpw * TILE;
  const int nc = min(NCOL, (M - r0) * G);  // query columns with a row
  const int j = lane & 15, g = lane >> 4;

  // queries (column 16 b + j: row r0 + (16 b + j) / G, head kvh G + j % G, dims
  // 32 ks + 8 g .. + 7) as hi + lo bf16, scaled to base-2 units
  const float qscale = 1.4426950408889634f / sqrtf((float)HD);
  int Lj[CB];
  int lim_min = INT_MAX;  // shortest column of the workgroup with a row
  bf16x8_d qh[CB][4], ql[CB][4];
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    const int rj = r0 + (16 * b + j) / G;
    const bool qok = rj < M;
    const int lv = len[qok ? rj : r0];  // unconditional load at a valid row (see k_attn_dec)
    Lj[b] = qok ? lv : 0;
    if (qok) lim_min = min(lim_min, Lj[b]);
    const float* qv = q + ((size_t)(qok ? rj : r0) * hq + kvh * G + j % G) * HD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const float4 x0 = *(const float4*)(qv + 32 * ks), x1 = *(const float4*)(qv + 32 * ks + 4);
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = qok ? xs[e] * qscale : 0.f;
        const __bf16 h = (__bf16)x;
        qh[b][ks][e] = h;
        ql[b][ks][e] = (__bf16)(x - (float)h);
      }
    }
  }
#pragma unroll
  for (int o_ = 32; o_ >= 1; o_ >>= 1) lim_min = min(lim_min, __shfl_xor(lim_min, o_));
  int Lmax = 0;  // longest row of the workgroup
  for (int r = r0; r < min(M, r0 + RB); ++r) Lmax = max(Lmax, len[r]);
  // tiles of this wave holding a key below Lmax
  const int first = start + w * TILE;
  const int ntl = Lmax > first ? min(tpw, (Lmax - first + NW * TILE - 1) / (NW * TILE)) : 0;

  const bf16_t* kb = kc + (size_t)kvh * n_max * HD;
  const bf16_t* vb = vc + (size_t)kvh * n_max * HD;
  bf16x8_d kr[2][16];  // key fragments of two tiles: [kt * 4 + ks]
  auto issue = [&](int i, int buf) {
    const int t0 = first + i * NW * TILE;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const int row = min(t0 + 16 * kt + j, n_max - 1);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        kr[buf][kt * 4 + ks] =
            __builtin_bit_cast(bf16x8_d, *(const uint4*)(kb + (size_t)row * HD + 32 * ks + 8 * g));
    }
    const int rr0 = lane >> 4, slot = lane & 15;
#pragma unroll
    for (int p = 0; p < 16; ++p) {
      const int rr = 4 * p + rr0;
      const int row = min(t0 + rr, n_max - 1);
      __builtin_amdgcn_global_load_lds(
          (const void*)(vb + (size_t)row * HD + ((slot ^ (rr & 15)) << 3)),
          (__attribute__((address_space(3))) void*)&(buf ? Vr1 : Vr0)[w][p * 64], 16, 0, 0);
    }
  };

  float m_run[CB], l_run[CB];
  f32x4_d o[CB][8];
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    m_run[b] = -FLT_MAX;
    l_run[b] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[b][dt] = f32x4_d{0.f, 0.f, 0.f, 0.f};
  }
  const int s4 = (lane & 15) >> 2, u4 = lane & 3;
  auto step = [&](int i, int buf) {
    const bool more = i + 1 < ntl;
    if (more) issue(i + 1, buf ^ 1);
    const int t0 = first + i * NW * TILE;
    const bool edge = t0 + TILE > lim_min;
    f32x4_d sc[CB][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int b = 0; b < CB; ++b) sc[b][kt] = f32x4_d{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int b = 0; b < CB; ++b) {
          sc[b][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[buf][kt * 4 + ks], qh[b][ks],
                                                              sc[b][kt], 0, 0, 0);
          sc[b][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[buf][kt * 4 + ks], ql[b][ks],
                                                              sc[b][kt], 0, 0, 0);
        }
    }
    bf16x8_d pa[CB][2];
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      if (edge) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (t0 + 16 * kt + 4 * g + v >= Lj[b]) sc[b][kt][v] = -FLT_MAX;
      }
      float mt = -FLT_MAX;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) mt = fmaxf(mt, sc[b][kt][v]);
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float m_new = fmaxf(m_run[b], mt);
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float p = __builtin_amdgcn_exp2f(sc[b][kt][v] - m_new);
          sc[b][kt][v] = p;
          ps += p;
        }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      if (__ballot(m_new != m_run[b])) {
        const float alpha = m_run[b] == -FLT_MAX ? 0.f : __builtin_amdgcn_exp2f(m_run[b] - m_new);
        l_run[b] *= alpha;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float av = __shfl(alpha, 4 * g + v);
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) o[b][dt][v] *= av;
        }
      }
      l_run[b] += ps;
      m_run[b] = m_new;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          pa[b][k2][v] = (__bf16)sc[b][2 * k2][v];
          pa[b][k2][4 + v] = (__bf16)sc[b][2 * k2 + 1][v];
        }
    }
    // this tile's values have landed once at most the next tile's loads are in flight
    if (more) __builtin_amdgcn_s_waitcnt(vmcnt_imm_a(32));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm_a(0));
    uint4* Vt = &(buf ? Vr1 : Vr0)[w][0];
    const int cnt = min(TILE, Lmax - t0);
    if (cnt < TILE) {
      for (int c = cnt * 16 + lane; c < TILE * 16; c += 64) Vt[c] = make_uint4(0u, 0u, 0u, 0u);
    }
    const char* Vb = (const char*)Vt;
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        bf16x4_d h2[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int row = 32 * k2 + 16 * h + 4 * g + s4;
          const int c = 2 * dt + (u4 >> 1);
          const char* pp = Vb + row * 256 + ((c ^ (row & 15)) << 4) + ((u4 & 1) << 3);
          h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (__attribute__((address_space(3))) bf16x4_d*)pp);
        }
        bf16x8_d vbv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vbv[e] = h2[0][e];
          vbv[4 + e] = h2[1][e];
        }
#pragma unroll
        for (int b = 0; b < CB; ++b)
          o[b][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[b][k2], vbv, o[b][dt], 0, 0, 0);
      }
    }
  };
  if (ntl > 0) issue(0, 0);
  // the ring position is a constant of each unrolled copy
  for (int i0 = 0; i0 < ntl; i0 += 2) {
    step(i0, 0);
    if (i0 + 1 < ntl) step(i0 + 1, 1);
  }

  // wave results to LDS (the wave's own stages: block b in stage b): o[b][dt][v]
  // is column 16 b + 4 g + v, dim 16 dt + j; the max and sum of column
  // 16 b + c live in lane c.  Wave 0's first stage also holds the merge scratch.
  float* s_w = (float*)&Vr0[0][0] + 16 * RS;
  float* s_mx = s_w + NCOL * NW;
  float* s_lx = s_mx + NCOL;
  int* s_len = (int*)(s_lx + NCOL);
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    float* rec = b == 0 ? (float*)&Vr0[w][0] : (float*)&Vr1[w][0];
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) rec[(4 * g + v) * RS + 16 * dt + j] = o[b][dt][v];
    if (lane < 16) {
      rec[lane * RS + HD] = m_run[b];
      rec[lane * RS + HD + 1] = l_run[b];
    }
  }
  __syncthreads();
  auto record = [&](int s, int c) -> const float* {
    return (c < 16 ? (const float*)&Vr0[s][0] : (const float*)&Vr1[s][0]) + (c & 15) * RS;
  };
  if (threadIdx.x < nc) {  // wave 0, lane c: column c (its Lj[c / 16] is the column's length)
    const int c = threadIdx.x;
    float mx = -FLT_MAX;
#pragma unroll
    for (int s = 0; s < NW; ++s) mx = fmaxf(mx, record(s, c)[HD]);
    float lx = 0.f;
#pragma unroll
    for (int s = 0; s < NW; ++s) {
      const float* rs = record(s, c);
      const float wt = rs[HD] == -FLT_MAX ? 0.f : __builtin_amdgcn_exp2f(rs[HD] - mx);
      s_w[c * NW + s] = wt;
      lx = fmaf(rs[HD + 1], wt, lx);
    }
    s_mx[c] = mx;
    s_lx[c] = lx;
    s_len[c] = CB == 1 || c < 16 ? Lj[0] : Lj[CB - 1];
  }
  __syncthreads();
  // the split's partial of every column whose row reaches this split
  for (int i = threadIdx.x; i < nc * HD; i += 64 * NW) {
    const int c = i >> 7, d = i & (HD - 1);
    if (s_len[c] <= start) continue;
    float acc = 0.f;
#pragma unroll
    for (int s = 0; s < NW; ++s) acc = fmaf(record(s, c)[d], s_w[c * NW + s], acc);
    float* dst = part + (((size_t)(r0 + c / G) * hq + kvh * G + c % G) * nsplit + split) * (HD + 2);
    dst[d] = acc;
    if (d == 0) {
      dst[HD] = s_mx[c] * 0.6931471805599453f;  // back to natural-log units
      dst[HD + 1] = s_lx[c];
    }
  }
}

// Batched rows (prefill chunks, selection candidates), bf16 caches, head dim
// 128.  Query vectors of one kv head are ordered qi = row * G + g; wave w of a
// workgroup owns 16 CB consecutive ones in CB column blocks (each key fragment
// and each transposed value read from LDS feeds CB matrix instructions; one
// block measured fastest, as two need 240 VGPRs).  The workgroup walks the
// 64-key tiles of
// its split through a ring of ST LDS stages filled by direct global-to-LDS
// loads ST - 1 tiles ahead (one barrier per tile, no staging registers); rows
// are stored with 16-byte chunk c of row r at slot c ^ (r % 16).  Per tile and
// wave: S^T = K Q^T (keys as rows, queries as hi + lo bf16 columns), an online
// softmax per query column (two cross-lane steps per statistic), then O += P V
// with the probabilities (bf16) taken from the score registers and the value
// operand from transposing LDS reads in the same key order.  The softmax is
// kept light, as the vector ALU and not the matrix unit bounds this kernel:
// scores arrive in base-2 units (queries pre-scaled), keys are masked only in
// tiles that reach past the shortest column of the wave, and the rescale of
// the running output is skipped when no column's max moved (its factor would
// be exactly 1).  Tile rows at or past max_len repeat row max_len - 1 (finite;
// their probability is 0).  Partials use the layout of the split kernels
// (max in natural-log units).
template <int NW, int ST, int CB>
__global__ __launch_bounds__(NW * 64) void k_attn_bat(int M, int hq, int hkv, int n_max,
                                                      const float* __restrict__ q,
                                                      const bf16_t* __restrict__ kc,
                                                      const bf16_t* __restrict__ vc,
                                                      const int32_t* __restrict__ len,
                                                      int max_len, int span,
                                                      float* __restrict__ part, int nsplit) {
  constexpr int HD = 128;
  constexpr int PPW = 32 / NW;  // 1 KiB pieces per wave per tile
  constexpr int QW = 16 * CB;   // query vectors per wave
  __shared__ __align__(16) uint4 KV[ST][2 * TILE * 16];
  const int split = blockIdx.x, kvh = blockIdx.y;
  const int G = hq / hkv;
  const int NQ = M * G;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int j = lane & 15, g = lane >> 4;
  const int start = split * span;
  const int end = min(max_len, start + span);
  const int ntile = (end - start + TILE - 1) / TILE;  // >= 1: the grid covers max_len

  // piece i (1 KiB) of a tile: rows 4 (i % 16) .. + 3 of K (i < 16) or V
  const bf16_t* kb = kc + (size_t)kvh * n_max * HD;
  const bf16_t* vb = vc + (size_t)kvh * n_max * HD;
  auto issue = [&](int tile, int buf) {
    const int t0 = start + tile * TILE;
#pragma unroll
    for (int u = 0; u < PPW; ++u) {
      const int i = w * PPW + u;
      const int rr = 4 * (i & 15) + (lane >> 4);
      const int row = min(t0 + rr, max_len - 1);
      const bf16_t* src =
          (i < 16 ? kb : vb) + (size_t)row * HD + (((lane & 15) ^ (rr & 15)) << 3);
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)&KV[buf][i * 64],
                                       16, 0, 0);
    }
  };
#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < ntile) issue(s, s);

  // query column j of block b of this wave: vector qb + 16 b + j.  Queries are
  // scaled by log2(e) / sqrt(HD), so scores are in base-2 units and the
  // probabilities are plain powers of two.
  const float qscale = 1.4426950408889634f / sqrtf((float)HD);
  const int qb = (blockIdx.z * NW + w) * QW;
  int lim[CB];      // keys of the column in this split
  int lim_min = end;  // fewest keys over the wave's columns with a query
  bf16x8_d qh[CB][4], ql[CB][4];
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    const int qi = qb + 16 * b + j;
    const bool qok = qi < NQ;
    lim[b] = qok ? min(len[qi / G], end) : 0;
    lim_min = min(lim_min, qok ? lim[b] : end);
    const int row = qok ? qi / G : 0;
    const int h = kvh * G + (qok ? qi % G : 0);
    const float* qv = q + ((size_t)row * hq + h) * HD + 8 * g;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      float4 x0 = *(const float4*)(qv + 32 * ks), x1 = *(const float4*)(qv + 32 * ks + 4);
      if (!qok) x0 = x1 = make_float4(0.f, 0.f, 0.f, 0.f);
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = xs[e] * qscale;
        const __bf16 hh = (__bf16)x;
        qh[b][ks][e] = hh;
        ql[b][ks][e] = (__bf16)(x - (float)hh);
      }
    }
  }
#pragma unroll
  for (int o_ = 32; o_ >= 1; o_ >>= 1) lim_min = min(lim_min, __shfl_xor(lim_min, o_));
  f32x4_d o[CB][8];
  float m_run[CB], l_run[CB];
#pragma unroll
  for (int b = 0; b < CB; ++b) {
    m_run[b] = -FLT_MAX;
    l_run[b] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[b][dt] = f32x4_d{0.f, 0.f, 0.f, 0.f};
  }
  const int s4 = (lane & 15) >> 2, u4 = lane & 3;

  auto step = [&](int it, int buf) {
    // tile it has landed once at most ST - 2 later tiles are in flight; the
    // barrier needs no fence (see k_gemm_tiled)
    if (it + ST - 2 < ntile) __builtin_amdgcn_s_waitcnt(vmcnt_imm_a(PPW * (ST - 2)));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm_a(0));
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
    if (it + ST - 1 < ntile) issue(it + ST - 1, (buf + ST - 1) % ST);
    const uint4* Kt = &KV[buf][0];
    const char* Vb = (const char*)&KV[buf][TILE * 16];
    const int t0 = start + it * TILE;
    // keys past a column's length only in tiles that reach past the shortest
    // column of the wave (wave-uniform)
    const bool edge = t0 + TILE > lim_min;
    // S^T per column block; each key fragment feeds every block
    f32x4_d sc[CB][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int b = 0; b < CB; ++b) sc[b][kt] = f32x4_d{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int c = 4 * ks + g;
        const bf16x8_d kf = __builtin_bit_cast(bf16x8_d, Kt[(16 * kt + j) * 16 + (c ^ j)]);
#pragma unroll
        for (int b = 0; b < CB; ++b) {
          sc[b][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qh[b][ks], sc[b][kt], 0, 0, 0);
          sc[b][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, ql[b][ks], sc[b][kt], 0, 0, 0);
        }
      }
    }
    bf16x8_d pa[CB][2];
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      if (edge) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (t0 + 16 * kt + 4 * g + v >= lim[b]) sc[b][kt][v] = -FLT_MAX;
      }
      float mt = -FLT_MAX;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) mt = fmaxf(mt, sc[b][kt][v]);
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float m_new = fmaxf(m_run[b], mt);
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          // masked scores give 2^(-huge) = 0
          const float p = __builtin_amdgcn_exp2f(sc[b][kt][v] - m_new);
          sc[b][kt][v] = p;
          ps += p;
        }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      // a column whose max moved rescales its sum and output rows; when no
      // column of the wave moved the factor is exactly 1 and is skipped
      if (__ballot(m_new != m_run[b])) {
        const float alpha = m_run[b] == -FLT_MAX ? 0.f : __builtin_amdgcn_exp2f(m_run[b] - m_new);
        l_run[b] *= alpha;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float av = __shfl(alpha, 4 * g + v);
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) o[b][dt][v] *= av;
        }
      }
      l_run[b] += ps;
      m_run[b] = m_new;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          pa[b][k2][v] = (__bf16)sc[b][2 * k2][v];
          pa[b][k2][4 + v] = (__bf16)sc[b][2 * k2 + 1][v];
        }
    }
    // O += P V; each transposed value operand feeds every block
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        bf16x4_d h2[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int row = 32 * k2 + 16 * h + 4 * g + s4;
          const int c = 2 * dt + (u4 >> 1);
          const char* pp = Vb + row * 256 + ((c ^ (row & 15)) << 4) + ((u4 & 1) << 3);
          h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (__attribute__((address_space(3))) bf16x4_d*)pp);
        }
        bf16x8_d vbv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vbv[e] = h2[0][e];
          vbv[4 + e] = h2[1][e];
        }
#pragma unroll
        for (int b = 0; b < CB; ++b)
          o[b][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[b][k2], vbv, o[b][dt], 0, 0, 0);
      }
    }
  };
  // the ring position is a constant of each unrolled copy
  for (int it0 = 0; it0 < ntile; it0 += ST) {
#pragma unroll
    for (int u = 0; u < ST; ++u)
      if (it0 + u < ntile) step(it0 + u, u);
  }

  // partials: O rows of block b are query columns 16 b + 4 g + v, dims 16 dt + j;
  // the max goes back to natural-log units
#pragma unroll
  for (int b = 0; b < CB; ++b) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int qv = qb + 16 * b + 4 * g + v;
      const int lv = __shfl(lim[b], 4 * g + v);
      if (qv >= NQ || lv <= start) continue;
      const int row = qv / G, h = kvh * G + qv % G;
      float* dst = part + (((size_t)row * hq + h) * nsplit + split) * (HD + 2);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) dst[16 * dt + j] = o[b][dt][v];
    }
    const int qi = qb + 16 * b + j;
    if (g == 0 && qi < NQ && lim[b] > start) {
      const int row = qi / G, h = kvh * G + qi % G;
      float* dst = part + (((size_t)row * hq + h) * nsplit + split) * (HD + 2);
      dst[HD] = m_run[b] * 0.6931471805599453f;
      dst[HD + 1] = l_run[b];
    }
  }
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ inline uint32_t pack2(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

// One workgroup of 4 waves per (row, query head); output dims lane -> (2 lane,
// 2 lane + 1) for bf16 caches, lane for float32 caches.  Wave w takes the
// splits s = w, w + 4, ... of the launch; the maxima, sums and output dims of
// up to CB of them are requested together with the row length, so a wave
// waits for one memory round trip per CB splits.  Splits at or past the row's
// own split count are skipped, the others enter a running max and sum in
// order.  The four wave results are rescaled to the common max and added in
// wave order, the row's own key/value (selection rows) last.
template <int HD, bool BF>
__global__ __launch_bounds__(256) void k_attn_combine(int M, int hq, int hkv, int span,
                                                      int ngrid, const float* __restrict__ q,
                                                      const float* __restrict__ part, int nsplit,
                                                      const int32_t* __restrict__ len,
                                                      const float* __restrict__ kvself,
                                                      bf16_t* ohi, bf16_t* olo, float* of,
                                                      int ldact, int xmap) {
  constexpr int DPL = HD / 64;
  constexpr int CB = 8;
  __shared__ float s_m[4], s_l[4];
  __shared__ float s_acc[4][DPL * 64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int G = hq / hkv;
  // xmap: query head h of kv head h / G on XCD h / G (see split_id)
  const int rest = blockIdx.x >> 3;
  const int r = xmap ? rest / G : blockIdx.x / hq;
  const int h = xmap ? (blockIdx.x & 7) * G + rest % G : blockIdx.x % hq;
  const int kvh = h / G;
  const float* pr = part + ((size_t)r * hq + h) * nsplit * (HD + 2);
  const int d0 = BF ? 2 * lane : lane;
  const int L = len[r];
  // the row's own key (selection rows): its score joins the max
  float sself = -FLT_MAX;
  if (kvself && wave == 0) {
    const float* ks = kvself + (((size_t)r * 2 + 0) * hkv + kvh) * HD;
    const float* qv = q + ((size_t)r * hq + h) * HD;
    float dd = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) dd = fmaf(qv[d0 + e], ks[d0 + e], dd);
    sself = wave_sum(dd) * (1.0f / sqrtf((float)HD));
  }
  float mr = -FLT_MAX, lr = 0.f, acc[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
  for (int s0 = wave; s0 < ngrid; s0 += 4 * CB) {
    float ms[CB], ls[CB], ov[CB][DPL];
#pragma unroll
    for (int k = 0; k < CB; ++k) {
      ms[k] = -FLT_MAX;
      ls[k] = 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) ov[k][e] = 0.f;
      if (s0 + 4 * k < ngrid) {  // wave-uniform: only splits the launch ran
        const float* ps = pr + (size_t)(s0 + 4 * k) * (HD + 2);
        ms[k] = ps[HD];
        ls[k] = ps[HD + 1];
        if (DPL == 2) {
          const float2 v = *(const float2*)&ps[d0];
          ov[k][0] = v.x;
          ov[k][DPL - 1] = v.y;
        } else {
          ov[k][0] = ps[d0];
        }
      }
    }
    const int ns = (L + span - 1) / span;  // splits holding keys of this row
#pragma unroll
    for (int k = 0; k < CB; ++k) {
      if (s0 + 4 * k < ns) {
        const float mn = fmaxf(mr, ms[k]);
        const float ea = __expf(mr - mn), eb = __expf(ms[k] - mn);
        lr = fmaf(ls[k], eb, lr * ea);
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[e] = fmaf(ov[k][e], eb, acc[e] * ea);
        mr = mn;
      }
    }
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) s_acc[wave][DPL * lane + e] = acc[e];
  if (lane == 0) {
    s_m[wave] = mr;
    s_l[wave] = lr;
  }
  __syncthreads();
  if (wave != 0) return;
  const float mx = fmaxf(fmaxf(fmaxf(s_m[0], s_m[1]), fmaxf(s_m[2], s_m[3])), sself);
  float lsum = 0.f;
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float ew = s_m[w] == -FLT_MAX ? 0.f : __expf(s_m[w] - mx);
    lsum = fmaf(s_l[w], ew, lsum);
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = fmaf(s_acc[w][DPL * lane + e], ew, acc[e]);
  }
  if (kvself) {
    const float* vs = kvself + (((size_t)r * 2 + 1) * hkv + kvh) * HD;
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

// Decode / verify rows of bf16 caches with head dim 128 take k_attn_dec (1..5
// tiles per split) or k_attn_stream (splits of a multiple of STREAM_NW tiles
// above that).
constexpr int STREAM_NW = 4;
bool attn_dec_path(const AttnArgs& a) {
  const int G = a.hq / a.hkv;
  return a.dtype == KS_BF16 && a.hd == 128 && G <= 16 && 16 % G == 0 &&
         a.rows_per_block == 1 && a.tiles >= 1 && (a.tiles <= 5 || a.tiles % STREAM_NW == 0);
}

void attn_split(const AttnArgs& a, hipStream_t st) {
  if (a.max_len <= 0) return;
  const int ns = (a.max_len + a.span - 1) / a.span;
  const int G = a.hq / a.hkv;
  const int nq = a.rows_per_block * G;
  dim3 grid(ns, a.hkv, (a.M + a.rows_per_block - 1) / a.rows_per_block);
#define KS_ATTN(HDV, BFV, QM)                                                                \
  KS_LAUNCH((k_attn_split<HDV, BFV, QM>), grid, dim3(256), 0, st, a.M, a.hq, a.hkv,          \
            a.n_max, a.q, a.kc, a.vc, a.len, a.tiles, a.rows_per_block, a.part,              \
            a.nsplit)
  if (attn_dec_path(a)) {
    // decode / verify rows: 16 query columns per workgroup when one block holds
    // all rows, else 32 (16 CB / G rows per workgroup)
    const int CB = a.M * G <= 16 ? 1 : 2;
    const int RB = 16 * CB / G;
    // the XCD placement pays for the one-round split kernel (k_attn_dec), not
    // for the streaming one (32K: 27.9 -> 28.3 us and the merge 4.2 -> 4.4 us)
    const int xmap = a.hkv == 8 && a.tiles <= 5;
    const dim3 g3 = xmap ? dim3(8 * ns, 1, (a.M + RB - 1) / RB) : dim3(ns, a.hkv, (a.M + RB - 1) / RB);
    const bf16_t* kc = (const bf16_t*)a.kc;
    const bf16_t* vc = (const bf16_t*)a.vc;
#define KS_DEC(S_, CB_)                                                                      \
  KS_LAUNCH((k_attn_dec<S_, CB_>), g3, dim3(64 * S_), 0, st, a.M, a.hq, a.hkv,               \
            a.n_max, a.q, kc, vc, a.len, a.part, a.nsplit, a.span, xmap)
#define KS_DEC_S(CB_)            \
  switch (a.tiles) {             \
    case 1: KS_DEC(1, CB_); break; \
    case 2: KS_DEC(2, CB_); break; \
    case 3: KS_DEC(3, CB_); break; \
    case 4: KS_DEC(4, CB_); break; \
    default: KS_DEC(5, CB_); break; \
  }
    if (a.tiles > 5) {
      const int tpw = a.tiles / STREAM_NW;
      if (CB == 1)
        KS_LAUNCH((k_attn_stream<STREAM_NW, 1>), g3, dim3(64 * STREAM_NW), 0, st, a.M,
                  a.hq, a.hkv, a.n_max, a.q, kc, vc, a.len, a.part, a.nsplit, tpw, xmap);
      else
        KS_LAUNCH((k_attn_stream<STREAM_NW, 2>), g3, dim3(64 * STREAM_NW), 0, st, a.M,
                  a.hq, a.hkv, a.n_max, a.q, kc, vc, a.len, a.part, a.nsplit, tpw, xmap);
    } else if (CB == 1) {
      KS_DEC_S(1);
    } else {
      KS_DEC_S(2);
    }
#undef KS_DEC_S
#undef KS_DEC
  } else if (a.hd == 128 && a.tiles > 1) {
    // batched rows: matrix-instruction kernel, 64 query vectors per workgroup
    const int span = TILE * a.tiles;
    constexpr int QWG = 16 * KS_BAT_NW * KS_BAT_CB;  // query vectors per workgroup
    dim3 g2((a.max_len + span - 1) / span, a.hkv, (a.M * G + QWG - 1) / QWG);
    KS_LAUNCH((k_attn_bat<KS_BAT_NW, KS_BAT_ST, KS_BAT_CB>), g2, dim3(64 * KS_BAT_NW), 0,
              st, a.M, a.hq, a.hkv, a.n_max, a.q, (const bf16_t*)a.kc,
              (const bf16_t*)a.vc, a.len, a.max_len, span, a.part, a.nsplit);
  } else if (a.hd == 128) {
    if (nq <= 4) KS_ATTN(128, true, 1); else KS_ATTN(128, true, 8);
  } else {
    if (nq <= 4) KS_ATTN(64, false, 1); else KS_ATTN(64, false, 8);
  }
#undef KS_ATTN
}

void attn_combine(const AttnArgs& a, const float* kvself, Act act_out, hipStream_t st) {
  dim3 grid(a.M * a.hq);
  const int xmap = attn_dec_path(a) && a.hkv == 8 && a.tiles <= 5;  // placed like the split kernel
  const int span = a.span;
  const int ngrid = (a.max_len + span - 1) / span;  // splits the split kernel ran
  const bool bf = a.dtype == KS_BF16;
#define KS_COMB(HDV, BFV)                                                                    \
  KS_LAUNCH((k_attn_combine<HDV, BFV>), grid, dim3(256), 0, st, a.M, a.hq, a.hkv,            \
            span, ngrid, a.q, a.part, a.nsplit, a.len, kvself,                               \
            bf ? (bf16_t*)act_out.hi : nullptr, bf ? (bf16_t*)act_out.lo : nullptr,          \
            bf ? nullptr : (float*)act_out.hi, act_out.ld, xmap)
  if (a.hd == 128) KS_COMB(128, true);
  else KS_COMB(64, false);
#undef KS_COMB
}

}  // namespace ks
