// Internal declarations of libknapspec: device helpers, kernel launchers and the
// context structure.  Not part of the public interface (see include/knapspec.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>
#include <deque>

#include "../../include/knapspec.h"

namespace ks {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // raw bf16 storage

// ---------------------------------------------------------------- bf16 helpers
__host__ __device__ inline float bf2f(bf16_t b) {
  union { uint32_t u; float f; } c;
  c.u = (uint32_t)b << 16;
  return c.f;
}
// round to nearest even (finite inputs)
__host__ __device__ inline bf16_t f2bf(float f) {
  union { uint32_t u; float f; } c;
  c.f = f;
  uint32_t u = c.u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// ------------------------------------------------------------------ epilogues
enum Epi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };

// Activations feeding a matrix product.  bf16 models: two bf16 planes with
// a = hi + lo (lo = bf16(a - hi)); float32 models: one float plane in hi.
struct Act {
  void* hi;
  void* lo;
  int ld;  // elements per row
};

// ----------------------------------------------------------- kernel launchers
// GEMM: y[m][n] = sum_k A[m][k] W[n][k] for m < M, n < N (N = rows of W).
//  EPI_STORE : out[m][n] = y
//  EPI_RESID : out[m][n] = res[m][n] + y          (out may alias res)
//  EPI_SWIGLU: W holds gate/up rows interleaved by 8 inside each 16-row tile
//              (see ks_pack_gate_up); writes act_out[m][u] = silu(gate_u) * up_u
//              for u < N/2.
struct GemmArgs {
  int M, N, K;
  Act A;
  const void* W;
  int epi;
  float* out;
  int ldo;
  const float* res;
  int ldres;
  Act act_out;
};
void gemm_bf16_skinny(const GemmArgs& g, hipStream_t st);  // M <= 16
void gemm_bf16_tiled(const GemmArgs& g, hipStream_t st);   // any M, A.hi only
void gemm_f32(const GemmArgs& g, hipStream_t st);          // any M

void pack_matrix_bf16(const bf16_t* src, bf16_t* dst, int N, int K, hipStream_t st);
void pack_gate_up_bf16(const bf16_t* gate, const bf16_t* up, bf16_t* dst, int ffn, int d,
                       hipStream_t st);

// x[m][:] = embed[tok[m]][:]
void embed_rows(const void* E, int dtype, const int32_t* tok, int M, int d, float* x,
                int ldx, hipStream_t st);
// act = bf16 split (or f32 copy) of rmsnorm(x) * g ; g == nullptr means no norm (plain
// conversion).
void norm_act(const float* x, int ldx, const float* g, float eps, int M, int d, int dtype,
              Act act, hipStream_t st);
// q/k normalisation (optional), RoPE, store of k/v.
//  mode 0: k, v stored to the cache at pos[m]; mode 1: to kvself[m][2][hkv][hd].
struct QkvPostArgs {
  int M, hq, hkv, hd, n_max, dtype, qk_norm;
  float eps;
  const float* qkv;      // [M][(hq+2hkv)hd]
  const float* rope_cs;  // [n_max][hd/2][2]
  const float* q_norm;
  const float* k_norm;
  const int32_t* pos;    // device [M]
  float* q_out;          // [M][hq][hd]
  void* kc;              // layer K cache [hkv][n_max][hd]
  void* vc;
  float* kvself;         // [M][2][hkv][hd] (mode 1)
  int mode;
};
void qkv_post(const QkvPostArgs& a, hipStream_t st);

// Split attention over the cache.  Row m attends cache positions [0, len[m]);
// splits of 64 * tiles positions; partial (o[hd], max, sum)
// per (row, q head, split).
struct AttnArgs {
  int M, hq, hkv, hd, n_max, dtype;
  const float* q;        // [M][hq][hd]
  const void* kc;
  const void* vc;
  const int32_t* len;    // device [M]
  int max_len;           // host upper bound of len[]
  int tiles;             // 64-position tiles per split
  int rows_per_block;
  float* part;           // [M][hq][nsplit][hd+2]
  int nsplit;            // stride: splits per (row, head)
};
void attn_split(const AttnArgs& a, hipStream_t st);
// Merge splits (and, when kvself != nullptr, the row's own key/value) and write
// the attention output as O-projection input activations.
void attn_combine(const AttnArgs& a, const float* kvself, Act act_out, hipStream_t st);
int attn_nsplit(int n_positions, int tiles);
int attn_rows_per_block(int G, bool batched);

// argmax (lowest index on ties) and top-1 probability of each row of logits
void argmax_rows(const float* logits, int M, int V, int32_t* am, float* top1, hipStream_t st);
// out[g] = mean_t cos(X[g][t], Y[t])
void cos_groups(const float* X, const float* Y, int groups, int r, int d, float* out,
                hipStream_t st);
// per-row cosine with float64 accumulation: out[t] = cos(X[t], Y[t % ry])
void cos_rows(const float* X, const float* Y, int rows, int ry, int d, double* out,
              hipStream_t st);
void cos_groups_f64(const float* X, const float* Y, int groups, int r, int d, double* out,
                    hipStream_t st);
// block copies: dst[i][0..n) = src[i][0..n) via device pointer tables of length cnt
void copy_rows(const float* const* src, float* const* dst, int cnt, int n, hipStream_t st);
// pos[c*r + t] = base + t and len[] = pos[] + len_add for c*r + t < total
void fill_pos(int32_t* pos, int32_t* len, int base, int r, int total, int len_add,
              hipStream_t st);
void set_i32(int32_t* p, int v, hipStream_t st);
// rotary table: cs[p][f] = (cos, sin)(p * theta^(-2f/hd)) computed in float64
void rope_table(float* cs, int n_max, int hd, double theta, hipStream_t st);

// isolated knapsack
void knapsack_dp(const int32_t* w, const int32_t* q, int B, int n, int C, int max_skip,
                 int32_t* best, uint64_t* bits, hipStream_t st);
void knapsack_backtrack(const uint64_t* bits, const int32_t* w, int B, int n, int C,
                        const int32_t* j, uint8_t* skip, int32_t* err, hipStream_t st);
void knapsack_select(const int32_t* best, const uint64_t* bits, const int32_t* w,
                     const double* s, int B, int n, int C, int D, int32_t* j_star,
                     int32_t* g_star, double* tpt, uint8_t* skip, hipStream_t st);

// ------------------------------------------------------------------ errors
void set_error(const std::string& msg);

}  // namespace ks
