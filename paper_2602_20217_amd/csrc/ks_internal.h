// Internal declarations of libknapspec: device helpers, kernel launchers and the
// context structure.  Not part of the public interface (see include/knapspec.h).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

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

// ------------------------------------------------------------ kernel timing
// While a timing bracket is open on a thread (stop != nullptr), every kernel
// the library launches from that thread carries the bracket's events in its
// own dispatch: the first launch takes `start` when it begins, each launch
// takes `stop` when it ends.  Elapsed time then covers the kernels' execution
// only, without the separate event packets that would sit between launches.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
  int launches = 0;
};
extern thread_local LaunchTiming g_timing;

#define KS_LAUNCH(kern, grid, block, lds, st, ...)                                  \
  do {                                                                             \
    if (::ks::g_timing.stop) {                                                     \
      hipExtLaunchKernelGGL(kern, grid, block, lds, st, ::ks::g_timing.start,      \
                            ::ks::g_timing.stop, 0, __VA_ARGS__);                  \
      ::ks::g_timing.start = nullptr;                                              \
      ++::ks::g_timing.launches;                                                   \
    } else {                                                                       \
      hipLaunchKernelGGL(kern, grid, block, lds, st, __VA_ARGS__);                 \
    }                                                                              \
  } while (0)

// ---------------------------------------------------------------- bf16 helpers
__host__ __device__ inline float bf2f(bf16_t b) {
  union { uint32_t u; float f; } c;
  c.u = (uint32_t)b << 16;
  return c.f;
}
// round to nearest even (finite inputs); on the device the gfx950 conversion
// instruction, which gives the same bits as the integer form (checked over
// denormals, ties and random finite values)
__host__ __device__ inline bf16_t f2bf(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_bit_cast(bf16_t, (__bf16)f);
#else
  union { uint32_t u; float f; } c;
  c.f = f;
  uint32_t u = c.u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
#endif
}

// ------------------------------------------------------------------ epilogues
enum Epi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3 };

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
//  EPI_QKV   : W is the fused q/k/v projection packed by ks_pack_qkv (rotary
//              pairs f, f + hd/2 of a head in rows 8 apart of one tile); applies
//              rotate-half RoPE at pos[m] to q and k, writes q (float32) to
//              q_out[m][hq][hd] and k, v (bf16) to the cache at position pos[m].
struct QkvEpi {
  int hq, hkv, hd, n_max;
  const float* rope_cs;  // [n_max][hd/2][2]
  const int32_t* pos;    // device [M]
  float* q_out;
  bf16_t* kc;            // layer K cache [hkv][n_max][hd]
  bf16_t* vc;
};
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
  // Skinny bf16 path, RMSNorm carried by the producers (see act_prep):
  //  ssq_in != nullptr: A holds x * gain (not yet divided by rms(x)) and
  //    ssq_in[m][0..nssq) the partial sums of x^2 of row m; the product scales
  //    row m by 1/sqrt(sum/K + eps).
  //  next_gain != nullptr (EPI_RESID): besides out, writes next_act = bf16
  //    split of out * next_gain and next_ssq[m][n/16] = sum of out^2 over the
  //    16 columns of each tile (ld d/16), the input of the next normed product.
  const float* ssq_in = nullptr;
  int nssq = 0;
  float eps = 0.f;
  const float* next_gain = nullptr;
  Act next_act{};
  float* next_ssq = nullptr;
  QkvEpi qe{};
  // tiled path: float32 split-K partial buffer (optional)
  float* part = nullptr;
  size_t part_bytes = 0;
};
void gemm_bf16_skinny(const GemmArgs& g, hipStream_t st);  // M <= 16
void gemm_bf16_tiled(const GemmArgs& g, hipStream_t st);   // any M, A.hi only
void gemm_f32(const GemmArgs& g, hipStream_t st);          // any M

void pack_matrix_bf16(const bf16_t* src, bf16_t* dst, int N, int K, hipStream_t st);
void pack_gate_up_bf16(const bf16_t* gate, const bf16_t* up, bf16_t* dst, int ffn, int d,
                       hipStream_t st);
// rows of a head reordered so each 16-row tile holds the rotary pairs
void pack_qkv_bf16(const bf16_t* src, bf16_t* dst, int heads, int hd, int d, hipStream_t st);
// packed column of head dimension i (rotate-half pairs 8 apart in a 16-row tile)
__host__ __device__ inline int qkv_perm(int i, int hd) {
  const int half = hd / 2, f = i % half;
  return 16 * (f / 8) + (f % 8) + 8 * (i / half);
}

// x[m][:] = embed[tok[m]][:]
void embed_rows(const void* E, int dtype, const int32_t* tok, int M, int d, float* x,
                int ldx, hipStream_t st);
// Positions of R rows starting at base (row m: base + m % r) and their
// lengths (position + len_add), written by the launch that prepares the rows.
struct PosFill {
  int32_t* pos = nullptr;
  int32_t* len = nullptr;
  int base = 0, r = 1, len_add = 0;
};
// RMSNorm input of a skinny product: for row m, x = (E ? embedding row tok[m] :
// xin row m) is written to xout (when not null and not xin), act = bf16 split of
// x * gain and ssq[m][j] = sum of x^2 over columns 16 j..16 j + 15 (ld d/16);
// with pf.pos also pos[m] and len[m] (as fill_pos).
void act_prep(const float* xin, int ldx, const void* E, int dtype, const int32_t* tok, int M,
              int d, float* xout, const float* gain, Act act, float* ssq, hipStream_t st,
              PosFill pf = PosFill{});
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
  int perm;              // qkv columns in the ks_pack_qkv order (bf16 models)
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
  int tiles;             // 64-position tiles per split (waves of the decode kernel)
  int span;              // positions per split (TILE * tiles)
  int rows_per_block;
  float* part;           // [M][hq][nsplit][hd+2]
  int nsplit;            // stride: splits per (row, head)
};
bool attn_dec_path(const AttnArgs& a);
void attn_split(const AttnArgs& a, hipStream_t st);
// Merge splits (and, when kvself != nullptr, the row's own key/value) and write
// the attention output as O-projection input activations.
void attn_combine(const AttnArgs& a, const float* kvself, Act act_out, hipStream_t st);
int attn_nsplit(int n_positions, int tiles);
int attn_rows_per_block(int G, bool batched);

// ---------------------------------------------------- vocabulary reductions
// argmax (lowest index on ties) and top-1 probability of each of M rows of V
// logits (rows ld floats apart); ws: argmax_ws_bytes(M, V) device bytes
size_t argmax_ws_bytes(int M, int V);
void argmax_rows(const float* logits, int M, int V, int ld, int32_t* am, float* top1, void* ws,
                 hipStream_t st);
// Sampling filter of R rows: tables of the top_k largest logits (ties by lower
// id), softmax at the temperature, shortest prefix reaching top_p, ids / probs
// rows KS_SAMPLE_KMAX apart, count[r] entries; top1 (optional) = unfiltered
// softmax maximum; tok (optional) = draw of row r with the Philox uniform of
// (seed, pos0 + r, purpose).  ws: sample_ws_bytes(R, V, top_k) device bytes.
struct SampleSpec {
  float temperature;
  int top_k;
  float top_p;
  uint64_t seed;
  int32_t* ids;
  float* probs;
  int32_t* count;
  float* top1;
  int32_t* tok;
  int pos0;
  int purpose;
};
bool vocab_fits(int V, int top_k);  // top_k = 0: the argmax reduction
size_t sample_ws_bytes(int R, int V, int top_k);
size_t sample_ws_bytes_max(int R);  // any top_k <= KS_SAMPLE_KMAX
void sample_rows(const float* logits, int R, int V, int ld, const SampleSpec& s, void* ws,
                 hipStream_t st);
// acceptance chain of one speculative sampling round; out = {a, token}
void spec_accept(const int32_t* pid, const float* ppr, const int32_t* pcnt, const int32_t* qid,
                 const float* qpr, const int32_t* qcnt, const int32_t* drafts, int g,
                 uint64_t seed, int pos0, int32_t* out, hipStream_t st);
void uniforms(uint64_t seed, const int32_t* pos, int n, int purpose, float* out, hipStream_t st);
// out[g] = mean_t cos(X[g][t], Y[t])
void cos_groups(const float* X, const float* Y, int groups, int r, int d, float* out,
                hipStream_t st);
// per-row cosine with float64 accumulation: out[t] = cos(X[t], Y[t % ry])
void cos_rows(const float* X, const float* Y, int rows, int ry, int d, double* out,
              hipStream_t st);
void cos_rows2(const float* X1, const float* X2, const float* Y, int rows, int ry, int d,
               double* out1, double* out2, hipStream_t st);
void cos_groups_f64(const float* X, const float* Y, int groups, int r, int d, double* out,
                    hipStream_t st);
// history ring <-> contiguous planes for `planes` planes of n rows of d floats
// (d % 4 == 0): flat row (i, t) at (i * plane_stride + t) * d, ring row (i, t) at
// (i * RING + (p0 + t) % RING) * d; to_ring copies flat -> ring, else ring -> flat
void ring_copy(const float* src, float* dst, size_t plane_stride, int planes, int n, int RING,
               int p0, int d, bool to_ring, hipStream_t st);
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

// one stage of the model-mode DP on the device (see k_dp_step)
struct DpStepArgs {
  int i, J, w;
  double tau;
  int r, M, stride;
  const double* sig;
  const int* cells_in;
  const int* cnt_in;
  int* cells_out;
  int* cnt_out;
  double* mean;    // [2 cells]
  int* idx;        // [J + 1]
  uint8_t* bits;   // [2L+1][stride]
  uint8_t* reach;  // [2L+1][stride]
  double* sig_e;   // [2L+1][stride]
  double* sig_s;   // [2L+1][stride]
  const float* E;
  const float* gprev;
  float* gnext;
  const float* Xi;
  size_t cell;     // floats per cell (r d)
  const float** ptr_src;
  float** ptr_dst;
  int bound_out;
};
void dp_step(const DpStepArgs& a, hipStream_t st);

// ------------------------------------------------------------------ errors
void set_error(const std::string& msg);

}  // namespace ks
