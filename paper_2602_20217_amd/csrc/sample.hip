// Vocabulary reductions of the LM head output: the greedy argmax / top-1
// probability, the temperature / top-k / top-p filter and token draw of
// sampling, and the speculative sampling acceptance chain (Section 2.1: a draft
// x ~ q is accepted iff u < min(1, p(x) / q(x)); the first rejection emits a
// token drawn from max(0, p - q), normalised; a round whose drafts are all
// accepted emits a token drawn from p after the last draft).
//
// Every reduction over a logits row runs in two launches.  k_vocab_scan splits
// the row into NB chunks of at most 4096 logits (one 256-thread workgroup per
// (chunk, row), so a single row still spreads over ~128 CUs) and writes, per
// chunk, the running (max, lowest argmax, sum of exp(l - max)) and, when
// sampling, the chunk's top-k candidates: radix selection of the k-th largest
// key in four 8-bit digits over LDS histograms, then an index-ordered
// compaction that keeps ties at the threshold by lower id.  The second launch
// reduces the NB partials of a row (argmax) or selects the row's top-k from
// the NB * k candidates the same way, sorts them by rank, and applies the
// softmax, the top-p cut and the draw.
//
// Order of the filter: decreasing logit, ties by lower token id.  Keys are the
// float bits mapped to an unsigned order (-0 is taken as +0).
#include "ks_internal.h"

#include <cfloat>

namespace ks {

namespace {

constexpr int SCAN_NT = 256;   // threads of a chunk workgroup
constexpr int SCAN_E = 16;     // logits per thread (chunk <= 4096)
constexpr int ROW_NT = 512;    // threads of a row-selection workgroup
constexpr int ROW_E = 16;      // candidates per thread (NB * k <= 8192)
constexpr int CAND_MAX = ROW_NT * ROW_E;
constexpr int NB_MAX = 128;
static_assert(ROW_NT == 4 * KS_SAMPLE_KMAX, "the rank count splits each entry over 4 threads");

struct VStat {
  float m;  // chunk max
  float s;  // sum of exp(l - m) over the chunk
  int i;    // lowest id attaining m
  int pad;
};

// Cross-lane steps on DPP lane moves (no LDS round trip).  dpp(x, ctrl, rows):
// the value of the lane the control names, 0 where the source lane lies
// outside the row or the destination row is masked off.
template <int CTRL, int ROWS = 0xF, bool BOUND = true>
__device__ inline int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROWS, 0xF, BOUND);
}
template <int CTRL, int ROWS = 0xF, bool BOUND = true>
__device__ inline float dpp_f(float x) {
  return __int_as_float(dpp_i<CTRL, ROWS, BOUND>(__float_as_int(x)));
}
constexpr int ROW_SHR1 = 0x111, ROW_SHR2 = 0x112, ROW_SHR4 = 0x114, ROW_SHR8 = 0x118;
constexpr int ROW_ROR1 = 0x121, ROW_ROR2 = 0x122, ROW_ROR4 = 0x124, ROW_ROR8 = 0x128;
constexpr int ROW_BCAST15 = 0x142, ROW_BCAST31 = 0x143;

__device__ inline uint32_t fkey(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline float key_f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

__device__ inline void st_push(VStat& a, float v, int i) {
  if (v > a.m) {
    a.s = a.s * __expf(a.m - v) + 1.0f;
    a.m = v;
    a.i = i;
  } else {
    a.s += __expf(v - a.m);
  }
}
__device__ inline VStat st_merge(VStat a, VStat b) {
  VStat r;
  if (b.m > a.m || (b.m == a.m && b.i < a.i)) {
    r.m = b.m;
    r.i = b.i;
  } else {
    r.m = a.m;
    r.i = a.i;
  }
  r.s = a.s * __expf(a.m - r.m) + b.s * __expf(b.m - r.m);
  r.pad = 0;
  return r;
}
template <int CTRL>
__device__ inline VStat st_rot(VStat a) {  // row rotations: every source lane is valid
  return VStat{dpp_f<CTRL, 0xF, false>(a.m), dpp_f<CTRL, 0xF, false>(a.s),
               dpp_i<CTRL, 0xF, false>(a.i), 0};
}
__device__ inline VStat st_lane(VStat a, int l) {
  return VStat{__int_as_float(__builtin_amdgcn_readlane(__float_as_int(a.m), l)),
               __int_as_float(__builtin_amdgcn_readlane(__float_as_int(a.s), l)),
               __builtin_amdgcn_readlane(a.i, l), 0};
}
// wave reduction (every lane gets the result): row rotations (DPP), then the
// four row results (merge is commutative and associative up to rounding)
__device__ inline VStat st_wave(VStat a) {
  a = st_merge(a, st_rot<ROW_ROR8>(a));
  a = st_merge(a, st_rot<ROW_ROR4>(a));
  a = st_merge(a, st_rot<ROW_ROR2>(a));
  a = st_merge(a, st_rot<ROW_ROR1>(a));
  return st_merge(st_merge(st_lane(a, 0), st_lane(a, 16)), st_merge(st_lane(a, 32), st_lane(a, 48)));
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): first output word of
// counter (pos, purpose, 0, 0) under key (seed_lo, seed_hi), as a uniform on
// the 2^-24 grid of [0, 1).
__device__ inline float philox_uniform(uint32_t k0, uint32_t k1, uint32_t pos, uint32_t purpose) {
  uint32_t c0 = pos, c1 = purpose, c2 = 0u, c3 = 0u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return (float)(c0 >> 8) * (1.0f / 16777216.0f);
}

// inclusive prefix sum over the 64 lanes: scans of the four 16-lane rows, then
// lane 15 added into row 1 and 3, lane 31 into rows 2 and 3
__device__ inline int wave_scan(int x) {
  x += dpp_i<ROW_SHR1>(x);
  x += dpp_i<ROW_SHR2>(x);
  x += dpp_i<ROW_SHR4>(x);
  x += dpp_i<ROW_SHR8>(x);
  x += dpp_i<ROW_BCAST15, 0xA, false>(x);
  x += dpp_i<ROW_BCAST31, 0xC, false>(x);
  return x;
}
__device__ inline float wave_scan(float x) {
  x += dpp_f<ROW_SHR1>(x);
  x += dpp_f<ROW_SHR2>(x);
  x += dpp_f<ROW_SHR4>(x);
  x += dpp_f<ROW_SHR8>(x);
  x += dpp_f<ROW_BCAST15, 0xA, false>(x);
  x += dpp_f<ROW_BCAST31, 0xC, false>(x);
  return x;
}
__device__ inline float lane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}
// wave-uniform sum / max: row rotations, then the four row results
__device__ inline float wave_sum(float x) {
  x += dpp_f<ROW_ROR8>(x);
  x += dpp_f<ROW_ROR4>(x);
  x += dpp_f<ROW_ROR2>(x);
  x += dpp_f<ROW_ROR1>(x);
  return (lane_f(x, 0) + lane_f(x, 16)) + (lane_f(x, 32) + lane_f(x, 48));
}
__device__ inline float wave_max(float x) {
  x = fmaxf(x, dpp_f<ROW_ROR8>(x));
  x = fmaxf(x, dpp_f<ROW_ROR4>(x));
  x = fmaxf(x, dpp_f<ROW_ROR2>(x));
  x = fmaxf(x, dpp_f<ROW_ROR1>(x));
  return fmaxf(fmaxf(lane_f(x, 0), lane_f(x, 16)), fmaxf(lane_f(x, 32), lane_f(x, 48)));
}

// Exclusive prefix over the block of v (thread order) and the block total.
template <int NT>
__device__ inline int block_excl_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int x = wave_scan(v);
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const int t = sh[w];
    base += w < wave ? t : 0;
    tot += t;
  }
  __syncthreads();
  total = tot;
  return base + x - v;
}

// Histogram update of the wave's lanes with pred set.  agg (the top digit,
// where a selection's keys mostly agree and same-address LDS atomics would
// serialise): the lanes sharing the first two distinct digits of the wave add
// their count through one lane each, the rest one by one; otherwise every lane
// adds its own.
__device__ inline void hist_add(int* hist, bool pred, uint32_t d, bool agg) {
  if (!agg) {
    if (pred) atomicAdd(&hist[d], 1);
    return;
  }
  const int lane = threadIdx.x & 63;
  uint64_t act = __ballot(pred);
#pragma unroll
  for (int round = 0; round < 2; ++round) {
    if (!act) return;  // wave-uniform
    const int leader = __ffsll((unsigned long long)act) - 1;
    const uint32_t dl = (uint32_t)__builtin_amdgcn_readlane((int)d, leader);
    const uint64_t same = __ballot(pred && d == dl);
    if (lane == leader) atomicAdd(&hist[dl], (int)__popcll(same));
    act &= ~same;
    pred = pred && d != dl;
  }
  if (pred) atomicAdd(&hist[d], 1);
}

// k-th largest key (k = want on entry, 1 <= want <= number of valid keys) of
// the block's valid keys: on return thr is that key and want the number of
// keys equal to thr that belong to the top k (keys above thr number k - want).
// Key e of a thread is valid iff e < nv (nv <= E).
template <int NT, int E>
__device__ inline void radix_kth(const uint32_t (&key)[E], int nv, int* hist, int* sh,
                                 uint32_t& thr, int& want) {
  uint32_t prefix = 0u, himask = 0u;
  const int lane = threadIdx.x & 63;
#pragma unroll 1
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += NT) hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e)
      hist_add(hist, e < nv && (key[e] & himask) == prefix, (key[e] >> shift) & 255u,
               shift == 24);
    __syncthreads();
    if (threadIdx.x < 64) {
      // lane l holds digits 255 - 4l down to 252 - 4l; the prefix sum over the
      // lanes counts the keys from the top digit down
      const int4 q = *(const int4*)&hist[252 - 4 * lane];
      const int h[4] = {q.w, q.z, q.y, q.x};  // digits 255 - 4l - j
      const int tot = h[0] + h[1] + h[2] + h[3];
      const int s = wave_scan(tot);
      int above = s - tot;  // keys in digits above 255 - 4l
      if (above < want && want <= s) {
        int d = 252 - 4 * lane;
        for (int j = 0; j < 4; ++j) {
          if (above + h[j] >= want) {
            d = 255 - 4 * lane - j;
            break;
          }
          above += h[j];
        }
        sh[0] = d;
        sh[1] = want - above;
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sh[0] << shift;
    himask |= 255u << shift;
    want = sh[1];
    __syncthreads();
  }
  thr = prefix;
}

// Index-ordered compaction of the top k.  Thread t holds the consecutive
// elements t * c .. t * c + nv - 1 (c per thread, nv <= c valid) in key[0..nv);
// selected are all keys above thr and the first `want` keys equal to thr
// (all: every valid element).  One block scan; calls put(slot, e), slot < k.
template <int NT, int E, typename F>
__device__ inline void compact_top(const uint32_t (&key)[E], int nv, bool all, uint32_t thr,
                                   int want, int* sh, F put) {
  int cg = 0, ce = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if (e < nv) {
      cg += (all || key[e] > thr) ? 1 : 0;
      ce += (!all && key[e] == thr) ? 1 : 0;
    }
  }
  int total = 0;
  const int ex = block_excl_scan<NT>(cg | (ce << 16), sh, total);
  int gtb = ex & 0xFFFF, eqb = ex >> 16;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if (e < nv) {
      if (all || key[e] > thr) {
        put(gtb + min(eqb, want), e);
        ++gtb;
      } else if (key[e] == thr) {
        if (eqb < want) put(gtb + eqb, e);
        ++eqb;
      }
    }
  }
}

// candidates of a row: NB * k (key, id) pairs, rows an even number of pairs
// apart so that every row starts 16-byte aligned
__host__ __device__ inline int cand_stride(int NB, int k) { return (NB * k + 1) & ~1; }

// grid (NB, rows), SCAN_NT threads.  Row r of logits (ld floats apart), chunk
// b = ids [b * chunk, min(V, (b + 1) * chunk)); thread t reads the c = chunk /
// SCAN_NT consecutive logits from t * c.  k > 0: also the chunk's top-k
// candidates, (key, id) pairs in id order at cand[r * stride + b * k ..],
// padded with (0, INT_MAX) when the chunk is shorter than k.
__global__ __launch_bounds__(SCAN_NT) void k_vocab_scan(const float* __restrict__ logits, int ld,
                                                        int V, int chunk, int k, VStat* stat,
                                                        uint2* cand) {
  __shared__ __align__(16) int hist[256];
  __shared__ int sh[8];
  __shared__ VStat sred[SCAN_NT / 64];
  const int b = blockIdx.x, NB = gridDim.x, r = blockIdx.y, t = threadIdx.x;
  const int j0 = b * chunk;
  const int n = min(chunk, V - j0);
  const int c = chunk / SCAN_NT;  // chunk is a multiple of SCAN_NT
  const int i0 = t * c;           // first element of this thread within the chunk
  const int nv = max(0, min(c, n - i0));
  const float* row = logits + (size_t)r * ld + j0 + i0;
  float v[SCAN_E];
  const bool vec = ((((uintptr_t)row) & 15) == 0) && (c & 3) == 0;
#pragma unroll
  for (int e = 0; e < SCAN_E; e += 4) {
    if (vec && e + 4 <= nv) {
      const float4 q = *(const float4*)(row + e);
      v[e] = q.x;
      v[e + 1] = q.y;
      v[e + 2] = q.z;
      v[e + 3] = q.w;
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) v[e + u] = e + u < nv ? row[e + u] : -FLT_MAX;
    }
  }
  VStat a{-FLT_MAX, 0.f, 0x7FFFFFFF, 0};
#pragma unroll
  for (int e = 0; e < SCAN_E; ++e)
    if (e < nv) st_push(a, v[e], j0 + i0 + e);
  a = st_wave(a);
  if ((t & 63) == 0) sred[t >> 6] = a;
  __syncthreads();
  if (t == 0) {
    VStat s = sred[0];
#pragma unroll
    for (int w = 1; w < SCAN_NT / 64; ++w) s = st_merge(s, sred[w]);
    stat[(size_t)r * NB + b] = s;
  }
  if (k <= 0) return;
  uint32_t key[SCAN_E];
#pragma unroll
  for (int e = 0; e < SCAN_E; ++e) key[e] = fkey(v[e]);
  const bool all = n <= k;
  uint32_t thr = 0u;
  int want = k;
  if (!all) radix_kth<SCAN_NT, SCAN_E>(key, nv, hist, sh, thr, want);
  uint2* out = cand + (size_t)r * cand_stride(NB, k) + (size_t)b * k;
  compact_top<SCAN_NT, SCAN_E>(key, nv, all, thr, want, sh, [&](int slot, int e) {
    if (slot < k) out[slot] = make_uint2(key[e], (uint32_t)(j0 + i0 + e));
  });
  for (int s = min(n, k) + t; s < k; s += SCAN_NT) out[s] = make_uint2(0u, 0x7FFFFFFFu);
}

// grid rows, 128 threads: argmax (lowest id on ties) and top-1 probability of
// each row from its NB chunk partials.
__global__ __launch_bounds__(128) void k_argmax_merge(const VStat* stat, int NB, int32_t* am,
                                                     float* top1) {
  __shared__ VStat sred[2];
  const int r = blockIdx.x, t = threadIdx.x;
  VStat a{-FLT_MAX, 0.f, 0x7FFFFFFF, 0};
  for (int b = t; b < NB; b += 128) a = st_merge(a, stat[(size_t)r * NB + b]);
  a = st_wave(a);
  if ((t & 63) == 0) sred[t >> 6] = a;
  __syncthreads();
  if (t == 0) {
    const VStat s = st_merge(sred[0], sred[1]);
    am[r] = s.i;
    if (top1) top1[r] = 1.0f / s.s;
  }
}

struct RowArgs {
  const VStat* stat;
  int NB;
  const uint2* cand;
  int k;
  float temperature, top_p;
  uint32_t seed_lo, seed_hi;
  int32_t* ids;    // [rows][KS_SAMPLE_KMAX]
  float* probs;    // [rows][KS_SAMPLE_KMAX]
  int32_t* count;  // [rows]
  float* top1;     // optional [rows]
  int32_t* tok;    // optional [rows]: draw of row r at position pos0 + r
  int pos0, purpose;
};

// Inverse-CDF draw over the first n entries of a table held two per lane
// (entry l in w0, entry l + 64 in w1): the first entry whose cumulative weight
// exceeds u, else the last one.  Returns the entry index.
__device__ inline int wave_draw(float w0, float w1, int n, float u, int lane) {
  const float c0 = wave_scan(lane < n ? w0 : 0.f);
  const float t0 = lane_f(c0, 63);
  const float c1 = t0 + wave_scan(lane + 64 < n ? w1 : 0.f);
  const uint64_t b0 = __ballot(lane < n && c0 > u);
  if (b0) return __ffsll((unsigned long long)b0) - 1;
  const uint64_t b1 = __ballot(lane + 64 < n && c1 > u);
  if (b1) return 64 + __ffsll((unsigned long long)b1) - 1;
  return n - 1;
}

// grid rows, ROW_NT threads: top-k of the row's NB * k candidates, sorted by
// (logit desc, id asc); softmax at temperature T; top-p cut; table write and
// optional draw.
__global__ __launch_bounds__(ROW_NT) void k_sample_row(RowArgs A) {
  __shared__ __align__(16) int hist[256];
  __shared__ int sh[16];
  __shared__ __align__(16) uint32_t sk[KS_SAMPLE_KMAX];
  __shared__ __align__(16) int32_t si[KS_SAMPLE_KMAX];
  __shared__ uint32_t ok[KS_SAMPLE_KMAX];
  __shared__ int32_t oi[KS_SAMPLE_KMAX];
  __shared__ int srank[KS_SAMPLE_KMAX];
  __shared__ VStat sred[ROW_NT / 64];
  const int r = blockIdx.x, t = threadIdx.x, lane = t & 63;
  const int k = A.k, n = A.NB * k;
  // candidates first (their loads overlap the partials' merge): thread t holds
  // the c consecutive pairs from t * c, c even, two pairs per 16-byte load
  const uint2* cr = A.cand + (size_t)r * cand_stride(A.NB, k);
  const int c = 2 * ((n + 2 * ROW_NT - 1) / (2 * ROW_NT));
  const int i0 = t * c;
  const int nv = max(0, min(c, n - i0));
  uint32_t key[ROW_E];
  int32_t cand_id[ROW_E];
#pragma unroll
  for (int e = 0; e < ROW_E; e += 2) {
    uint4 q = make_uint4(0u, 0x7FFFFFFFu, 0u, 0x7FFFFFFFu);
    if (e < nv) q = *(const uint4*)(cr + i0 + e);  // pair e + 1 is inside the padded row
    key[e] = q.x;
    cand_id[e] = (int32_t)q.y;
    key[e + 1] = q.z;
    cand_id[e + 1] = (int32_t)q.w;
  }
  if (t < KS_SAMPLE_KMAX) srank[t] = 0;
  if (A.top1) {
    VStat a{-FLT_MAX, 0.f, 0x7FFFFFFF, 0};
    for (int b = t; b < A.NB; b += ROW_NT) a = st_merge(a, A.stat[(size_t)r * A.NB + b]);
    a = st_wave(a);
    if (lane == 0) sred[t >> 6] = a;
    __syncthreads();
    if (t == 0) {
      VStat s = sred[0];
#pragma unroll
      for (int w = 1; w < ROW_NT / 64; ++w) s = st_merge(s, sred[w]);
      A.top1[r] = 1.0f / s.s;
    }
  }
  const bool all = n <= k;
  uint32_t thr = 0u;
  int want = k;
  if (!all) radix_kth<ROW_NT, ROW_E>(key, nv, hist, sh, thr, want);
  compact_top<ROW_NT, ROW_E>(key, nv, all, thr, want, sh, [&](int slot, int e) {
    if (slot < k) {
      sk[slot] = key[e];
      si[slot] = cand_id[e];
    }
  });
  __syncthreads();
  {  // rank of entry i in (key desc, id asc), counted by 4 threads of 32 entries each
    const int i = t & (KS_SAMPLE_KMAX - 1), part = t / KS_SAMPLE_KMAX;
    if (i < k) {
      const uint32_t mk = sk[i];
      const int32_t mi = si[i];
      int cnt = 0;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int j = part * 32 + 4 * q;
        if (j < k) {
          const uint4 kk = *(const uint4*)&sk[j];
          const int4 ii = *(const int4*)&si[j];
          cnt += (kk.x > mk || (kk.x == mk && ii.x < mi)) ? 1 : 0;
          cnt += (j + 1 < k && (kk.y > mk || (kk.y == mk && ii.y < mi))) ? 1 : 0;
          cnt += (j + 2 < k && (kk.z > mk || (kk.z == mk && ii.z < mi))) ? 1 : 0;
          cnt += (j + 3 < k && (kk.w > mk || (kk.w == mk && ii.w < mi))) ? 1 : 0;
        }
      }
      if (cnt) atomicAdd(&srank[i], cnt);
    }
  }
  __syncthreads();
  if (t < k) {
    ok[srank[t]] = sk[t];
    oi[srank[t]] = si[t];
  }
  __syncthreads();
  if (t >= 64) return;
  // wave 0: entries lane and lane + 64 of the sorted table
  const float l0 = key_f(ok[0]);
  const float inv_t = 1.0f / A.temperature;
  const float e0 = lane < k ? expf((key_f(ok[lane]) - l0) * inv_t) : 0.f;
  const float e1 = lane + 64 < k ? expf((key_f(ok[lane + 64]) - l0) * inv_t) : 0.f;
  const float c0 = wave_scan(e0);
  const float t0 = lane_f(c0, 63);
  const float c1 = t0 + wave_scan(e1);
  const float sk_all = k > 64 ? lane_f(c1, k - 65) : lane_f(c0, k - 1);
  int m = k;
  if (A.top_p < 1.0f) {
    const float cut = A.top_p * sk_all;
    const uint64_t b0 = __ballot(lane < k && c0 >= cut);
    const uint64_t b1 = __ballot(lane + 64 < k && c1 >= cut);
    const int first = b0 ? __ffsll((unsigned long long)b0) - 1
                         : (b1 ? 64 + __ffsll((unsigned long long)b1) - 1 : k - 1);
    m = first + 1;
  }
  const float sm = m > 64 ? lane_f(c1, m - 65) : lane_f(c0, m - 1);
  const float p0 = lane < m ? e0 / sm : 0.f;
  const float p1 = lane + 64 < m ? e1 / sm : 0.f;
  int32_t* ids = A.ids + (size_t)r * KS_SAMPLE_KMAX;
  float* probs = A.probs + (size_t)r * KS_SAMPLE_KMAX;
  if (lane < m) {
    ids[lane] = oi[lane];
    probs[lane] = p0;
  }
  if (lane + 64 < m) {
    ids[lane + 64] = oi[lane + 64];
    probs[lane + 64] = p1;
  }
  if (lane == 0) A.count[r] = m;
  if (A.tok) {
    const float u = philox_uniform(A.seed_lo, A.seed_hi, (uint32_t)(A.pos0 + r),
                                   (uint32_t)A.purpose);
    const int j = wave_draw(p0, p1, m, u, lane);
    if (lane == 0) A.tok[r] = oi[j];
  }
}

// One wave.  Acceptance chain of a round: drafts[i] (position pos0 + i + 1)
// against target table p row i and draft table q row i; out = {a, token}.
__global__ __launch_bounds__(64) void k_spec_accept(const int32_t* pid, const float* ppr,
                                                    const int32_t* pcnt, const int32_t* qid,
                                                    const float* qpr, const int32_t* qcnt,
                                                    const int32_t* drafts, int g, uint32_t s_lo,
                                                    uint32_t s_hi, int pos0, int32_t* out) {
  __shared__ int32_t sq_id[KS_SAMPLE_KMAX];
  __shared__ float sq_pr[KS_SAMPLE_KMAX];
  const int lane = threadIdx.x;
  constexpr int LD = KS_SAMPLE_KMAX;
  for (int i = 0; i < g; ++i) {
    const int x = drafts[i];
    const int np = min(max(pcnt[i], 1), LD), nq = min(max(qcnt[i], 1), LD);
    const int32_t* pi = pid + (size_t)i * LD;
    const float* pp = ppr + (size_t)i * LD;
    const int32_t* qi = qid + (size_t)i * LD;
    const float* qp = qpr + (size_t)i * LD;
    float px = 0.f, qx = 0.f;
    if (lane < np && pi[lane] == x) px = pp[lane];
    if (lane + 64 < np && pi[lane + 64] == x) px = pp[lane + 64];
    if (lane < nq && qi[lane] == x) qx = qp[lane];
    if (lane + 64 < nq && qi[lane + 64] == x) qx = qp[lane + 64];
    px = wave_max(px);
    qx = wave_max(qx);
    const float ratio = qx > 0.f ? px / qx : 0.f;
    const uint32_t pos = (uint32_t)(pos0 + i + 1);
    const float u = philox_uniform(s_lo, s_hi, pos, 1u);
    if (u < fminf(1.0f, ratio)) continue;
    // rejected: residual max(0, p - q) over p's table
    sq_id[lane] = lane < nq ? qi[lane] : -1;
    sq_pr[lane] = lane < nq ? qp[lane] : 0.f;
    sq_id[lane + 64] = lane + 64 < nq ? qi[lane + 64] : -1;
    sq_pr[lane + 64] = lane + 64 < nq ? qp[lane + 64] : 0.f;
    __syncthreads();
    const int y0 = lane < np ? pi[lane] : -2, y1 = lane + 64 < np ? pi[lane + 64] : -2;
    float q0 = 0.f, q1 = 0.f;
    for (int j = 0; j < nq; ++j) {
      const int32_t id = sq_id[j];
      if (id == y0) q0 = sq_pr[j];
      if (id == y1) q1 = sq_pr[j];
    }
    const float p0 = lane < np ? pp[lane] : 0.f, p1 = lane + 64 < np ? pp[lane + 64] : 0.f;
    float r0 = fmaxf(0.f, p0 - q0), r1 = fmaxf(0.f, p1 - q1);
    const float sr = wave_sum(r0 + r1);
    if (sr > 0.f) {
      r0 /= sr;
      r1 /= sr;
    } else {  // p = q on p's support: draw from p
      r0 = p0;
      r1 = p1;
    }
    const float ur = philox_uniform(s_lo, s_hi, pos, 2u);
    const int j = wave_draw(r0, r1, np, ur, lane);
    if (lane == 0) {
      out[0] = i;
      out[1] = pi[j];
    }
    return;
  }
  const int np = min(max(pcnt[g], 1), LD);
  const int32_t* pi = pid + (size_t)g * LD;
  const float* pp = ppr + (size_t)g * LD;
  const float p0 = lane < np ? pp[lane] : 0.f, p1 = lane + 64 < np ? pp[lane + 64] : 0.f;
  const float u = philox_uniform(s_lo, s_hi, (uint32_t)(pos0 + g + 1), 2u);
  const int j = wave_draw(p0, p1, np, u, lane);
  if (lane == 0) {
    out[0] = g;
    out[1] = pi[j];
  }
}

__global__ void k_uniforms(uint32_t s_lo, uint32_t s_hi, const int32_t* pos, int n, int purpose,
                           float* out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = philox_uniform(s_lo, s_hi, (uint32_t)pos[i], (uint32_t)purpose);
}

// chunking of a row of V logits for k candidates per chunk
struct Chunking {
  int NB, chunk;
};
Chunking chunking(int V, int k) {
  const int nb_max = k > 0 ? std::min(NB_MAX, CAND_MAX / k) : NB_MAX;
  int nb = std::min(nb_max, std::max(1, (V + 1023) / 1024));
  int chunk = (V + nb - 1) / nb;
  chunk = (chunk + SCAN_NT - 1) / SCAN_NT * SCAN_NT;  // whole logits per thread
  nb = (V + chunk - 1) / chunk;
  return {nb, chunk};
}

// argmax of M rows: ~1024-logit chunks spread one row over ~128 CUs; from 16
// rows on, 4096-logit chunks keep the workgroup count (and its per-workgroup
// overhead) down while still filling the GPU
Chunking argmax_chunking(int M, int V) {
  if (M < 16) return chunking(V, 0);
  const int chunk = SCAN_NT * SCAN_E;
  return {(V + chunk - 1) / chunk, chunk};
}

}  // namespace

bool vocab_fits(int V, int k) {
  const Chunking ch = chunking(V, k);
  return V >= 1 && ch.chunk <= SCAN_NT * SCAN_E && k <= KS_SAMPLE_KMAX && k <= V;
}

size_t argmax_ws_bytes(int M, int V) {
  return (size_t)M * std::max(chunking(V, 0).NB, argmax_chunking(M, V).NB) * sizeof(VStat);
}

size_t sample_ws_bytes(int R, int V, int k) {
  const Chunking ch = chunking(V, k);
  return (size_t)R * ch.NB * sizeof(VStat) + (size_t)R * cand_stride(ch.NB, k) * 8;
}

size_t sample_ws_bytes_max(int R) {
  return (size_t)R * NB_MAX * sizeof(VStat) + (size_t)R * (CAND_MAX + 2) * 8;
}

void argmax_rows(const float* logits, int M, int V, int ld, int32_t* am, float* top1, void* ws,
                 hipStream_t st) {
  if (M <= 0) return;
  const Chunking ch = argmax_chunking(M, V);
  VStat* stat = (VStat*)ws;
  for (int m0 = 0; m0 < M; m0 += 65535) {
    const int mm = std::min(65535, M - m0);
    KS_LAUNCH(k_vocab_scan, dim3(ch.NB, mm), dim3(SCAN_NT), 0, st,
              logits + (size_t)m0 * ld, ld, V, ch.chunk, 0, stat + (size_t)m0 * ch.NB,
              nullptr);
  }
  KS_LAUNCH(k_argmax_merge, dim3(M), dim3(128), 0, st, stat, ch.NB, am, top1);
}

void sample_rows(const float* logits, int R, int V, int ld, const SampleSpec& s, void* ws,
                 hipStream_t st) {
  if (R <= 0) return;
  const int k = s.top_k;
  const Chunking ch = chunking(V, k);
  VStat* stat = (VStat*)ws;
  uint2* cand = (uint2*)((char*)ws + (size_t)R * ch.NB * sizeof(VStat));  // 16-byte aligned
  KS_LAUNCH(k_vocab_scan, dim3(ch.NB, R), dim3(SCAN_NT), 0, st, logits, ld, V, ch.chunk,
            k, stat, cand);
  RowArgs A{stat, ch.NB, cand, k, s.temperature, s.top_p, (uint32_t)s.seed,
            (uint32_t)(s.seed >> 32), s.ids, s.probs, s.count, s.top1, s.tok, s.pos0, s.purpose};
  KS_LAUNCH(k_sample_row, dim3(R), dim3(ROW_NT), 0, st, A);
}

void spec_accept(const int32_t* pid, const float* ppr, const int32_t* pcnt, const int32_t* qid,
                 const float* qpr, const int32_t* qcnt, const int32_t* drafts, int g,
                 uint64_t seed, int pos0, int32_t* out, hipStream_t st) {
  KS_LAUNCH(k_spec_accept, dim3(1), dim3(64), 0, st, pid, ppr, pcnt, qid, qpr, qcnt,
            drafts, g, (uint32_t)seed, (uint32_t)(seed >> 32), pos0, out);
}

void uniforms(uint64_t seed, const int32_t* pos, int n, int purpose, float* out, hipStream_t st) {
  if (n <= 0) return;
  KS_LAUNCH(k_uniforms, dim3((n + 255) / 256), dim3(256), 0, st, (uint32_t)seed,
            (uint32_t)(seed >> 32), pos, n, purpose, out);
}

}  // namespace ks
