// Coarse quantizer of the index: a lower bound on a row's distance that lets
// the Rank stage (Section 2, stage 2) skip rows which cannot enter a query's
// top k, without changing any result.
//
// The scan's distance of row x is ||q - x^||_w^2, the weighted squared
// distance from q to the row reconstructed from the query's conditioned
// codebook C_iFVS = C_PQ + Delta (Section 2, first display).  A coarse
// centroid is itself a vector of PQ codes, so its distance D_c = ||q - c^||_w^2
// is a sum of the same table entries.  By the triangle inequality
//     ||q - x^||_w >= ||q - c^||_w - ||c^ - x^||_w
//     ||c^ - x^||_w <= sqrt(max_j w_j) * (||c0 - x0|| + delta)
// where c0, x0 are the reconstructions from C_PQ alone, r = ||c0 - x0|| is
// stored per row (at build), and delta bounds ||Delta(c) - Delta(x)|| for any
// two code vectors: sqrt(sum over subspaces of (2 max_c ||Delta[m][c]||)^2)
// (per query).  A row is skipped when the square of the bound exceeds the
// query's current k-th distance.
//
// Rounding: every quantity is widened by a relative margin that covers the
// fp32 (or binary16) rounding of the tables and of the bound itself, so the
// computed bound never exceeds the computed distance:
//   grow = 1 + 2 (d + M + 8) 2^-24 + 2^-20 on delta,
//   keep = 1 - eps on both squared distances (eps from the table precision),
//   an absolute term for binary16 tables (subnormal entries).
//
// Build (once per index): k-means with a fixed iteration count on the
// reconstructions of evenly spaced rows, every sum in a fixed order (the
// build is deterministic); the centroids are encoded with C_PQ; every row
// gets its nearest encoded centroid and the distance to it, rounded up.
#include <algorithm>
#include <cfloat>
#include <cmath>

#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

constexpr int kMaxD = kCoarseMaxDim;
constexpr int kCentChunk = 32;     // centroids staged in LDS at a time

__device__ __forceinline__ int code_at(const uint32_t* codes_t, int mw, int64_t r, int m) {
  const uint32_t w = codes_t[((r >> 6) * mw + (m >> 2)) * 64 + (r & 63)];
  return static_cast<int>((w >> (8 * (m & 3))) & 0xFFu);
}

__device__ __forceinline__ float widen(float v) { return v; }
__device__ __forceinline__ float widen(__half v) { return __half2float(v); }

// X[i][j] = reconstruction of physical row i * stride, dimension j.
__global__ __launch_bounds__(256) void coarse_sample_kernel(const uint32_t* __restrict__ codes_t, int mw, int dsub,
                                                            int D, const float* __restrict__ cpq, int64_t S,
                                                            int64_t stride, float* __restrict__ X) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= S * D) return;
  const int64_t i = e / D;
  const int j = static_cast<int>(e % D);
  const int m = j / dsub;
  const int code = code_at(codes_t, mw, i * stride, m);
  X[e] = cpq[(static_cast<size_t>(m) * kKsub + code) * dsub + j % dsub];
}

// Nearest of the C centroids `cent` [C][D] to x (squared L2 summed in j
// order, ties to the lower index); the centroids pass through LDS
// kCentChunk at a time.  Every thread of the block must call it.
__device__ __forceinline__ void nearest(const float (&x)[kMaxD], int D, const float* __restrict__ cent, int C,
                                        float* s_c, int* best_out, float* best_d_out, bool active) {
  float best_d = __builtin_inff();
  int best = 0;
  for (int c0 = 0; c0 < C; c0 += kCentChunk) {
    const int nc = min(kCentChunk, C - c0);
    __syncthreads();
    for (int e = threadIdx.x; e < nc * D; e += blockDim.x) s_c[e] = cent[static_cast<size_t>(c0) * D + e];
    __syncthreads();
    if (active) {
      for (int c = 0; c < nc; ++c) {
        const float* cc = s_c + c * D;
        float d = 0.0f;
#pragma unroll
        for (int j = 0; j < kMaxD; ++j)
          if (j < D) {
            const float t = __fsub_rn(x[j], cc[j]);
            d = __fadd_rn(d, __fmul_rn(t, t));
          }
        if (d < best_d) {
          best_d = d;
          best = c0 + c;
        }
      }
    }
  }
  *best_out = best;
  *best_d_out = best_d;
}

__global__ __launch_bounds__(256) void coarse_assign_kernel(const float* __restrict__ X, int64_t S, int D,
                                                            const float* __restrict__ cent, int C,
                                                            int32_t* __restrict__ assign) {
  __shared__ float s_c[kCentChunk * kMaxD];
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const bool active = i < S;
  float x[kMaxD];
#pragma unroll
  for (int j = 0; j < kMaxD; ++j) x[j] = active && j < D ? X[i * D + j] : 0.0f;
  int best;
  float best_d;
  nearest(x, D, cent, C, s_c, &best, &best_d, active);
  if (active) assign[i] = best;
}

// Centroid c = mean of its members, summed in sample order (one workgroup per
// centroid, thread j sums dimension j); an empty cluster keeps its centroid.
__global__ __launch_bounds__(kMaxD) void coarse_update_kernel(const float* __restrict__ X, int64_t S, int D,
                                                              const int32_t* __restrict__ assign,
                                                              float* __restrict__ cent) {
  const int c = blockIdx.x;
  const int j = threadIdx.x;
  float acc = 0.0f;
  int64_t cnt = 0;
  for (int64_t i = 0; i < S; ++i) {
    if (assign[i] != c) continue;
    if (j < D) acc = __fadd_rn(acc, X[i * D + j]);
    ++cnt;
  }
  if (cnt > 0 && j < D) cent[static_cast<size_t>(c) * D + j] = __fdiv_rn(acc, static_cast<float>(cnt));
}

// Centroid c encoded with C_PQ (nearest codeword per subspace, ties to the
// lower code) as code words like a row's (cc [C][mw], word w holding
// subspaces 4w..4w+3, least significant byte first), and its
// reconstruction chat [C][D].
__global__ __launch_bounds__(256) void coarse_encode_kernel(const float* __restrict__ cent, int C, int M, int mw,
                                                            int dsub, const float* __restrict__ cpq,
                                                            uint32_t* __restrict__ cc, float* __restrict__ chat) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<int64_t>(C) * mw) return;
  const int c = static_cast<int>(e / mw), w = static_cast<int>(e % mw);
  const int D = M * dsub;
  uint32_t word = 0;
  for (int b = 0; b < 4; ++b) {
    const int m = 4 * w + b;
    if (m >= M) break;
    const float* x = cent + static_cast<size_t>(c) * D + m * dsub;
    float best_d = __builtin_inff();
    int best = 0;
    for (int k = 0; k < kKsub; ++k) {
      const float* cw = cpq + (static_cast<size_t>(m) * kKsub + k) * dsub;
      float d = 0.0f;
      for (int j = 0; j < dsub; ++j) {
        const float t = __fsub_rn(x[j], cw[j]);
        d = __fadd_rn(d, __fmul_rn(t, t));
      }
      if (d < best_d) {
        best_d = d;
        best = k;
      }
    }
    word |= static_cast<uint32_t>(best) << (8 * b);
    const float* cw = cpq + (static_cast<size_t>(m) * kKsub + best) * dsub;
    for (int j = 0; j < dsub; ++j) chat[static_cast<size_t>(c) * D + m * dsub + j] = cw[j];
  }
  cc[e] = word;
}

// Every physical row r < n_pad: word[r] = centroid id (low 16 bits) | the
// radius as the upper half of an fp32 (a bfloat16), rounded up.  The radius
// ||c0 - x0|| is summed in fp32 (relative error below 2^-17 for D <= 128)
// and multiplied by 1 + 2^-14 first, so the stored value bounds the exact
// one.  Rows past n get word 0 (never selected).
__global__ __launch_bounds__(256) void coarse_rows_kernel(const uint32_t* __restrict__ codes_t, int64_t n,
                                                          int64_t n_pad, int M, int mw, int dsub,
                                                          const float* __restrict__ cpq,
                                                          const float* __restrict__ chat, int C,
                                                          uint32_t* __restrict__ words) {
  __shared__ float s_c[kCentChunk * kMaxD];
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const bool active = r < n;
  const int D = M * dsub;
  float x[kMaxD];
#pragma unroll
  for (int j = 0; j < kMaxD; ++j) {
    float v = 0.0f;
    if (active && j < D) {
      const int m = j / dsub;
      v = cpq[(static_cast<size_t>(m) * kKsub + code_at(codes_t, mw, r, m)) * dsub + j % dsub];
    }
    x[j] = v;
  }
  int best;
  float best_d;
  nearest(x, D, chat, C, s_c, &best, &best_d, active);
  if (r < n_pad) {
    uint32_t w = 0;
    if (active) {
      uint32_t bits = __float_as_uint(__fmul_rn(sqrtf(best_d), 1.0f + 0x1p-14f));
      if (bits & 0xFFFFu) bits = (bits + 0x10000u) & 0xFFFF0000u;   // up to the next bfloat16
      w = bits | static_cast<uint32_t>(best);
    }
    words[r] = w;
  }
}

// Bounds of the coarse bound, two kernels.  Partial (one workgroup per
// subspace m and chunk of kBoundQueries queries, one thread per codeword c,
// the operands of the table build in registers): per query,
//   parts[q][0][m] = max_c ||C_iFVS[m][c] - C_PQ[m][c]||^2, the conditioned
//                    codeword recomputed with exactly the table kernel's
//                    operations (so this is the shift the tables saw);
//   parts[q][1][m] = max_j w_f[m*d + j] (NaN when a weight of the subspace is
//                    negative or not finite; 1 without weights).
// Final (one thread per query): bounds[q] = {sqrt(max_m parts[q][1][m])
// widened by 2^-19, sqrt(sum_m 4 parts[q][0][m]) * grow}.
constexpr int kBoundQueries = 16;

__device__ __forceinline__ float nan_max(float a, float b) {
  return (a != a || b != b) ? __builtin_nanf("") : fmaxf(a, b);
}

template <int DSUB, int R>
__global__ __launch_bounds__(256) void bound_parts_kernel(const float* __restrict__ alpha, const float* __restrict__ wf,
                                                          const float* __restrict__ cpq, const float* __restrict__ W,
                                                          int M, int dsub_rt, int r_rt, int nq,
                                                          float* __restrict__ parts) {
  constexpr bool kFixed = DSUB > 0;
  const int dsub = kFixed ? DSUB : dsub_rt;
  const int r = kFixed ? R : r_rt;
  const int m = blockIdx.x;
  const int c = threadIdx.x;
  const int lane = c & 63, wave = c >> 6;
  __shared__ float s_red[4];
  float creg[kFixed ? DSUB : 1];
  float wreg[kFixed ? R : 1][kFixed ? DSUB : 1];
  if constexpr (kFixed) {
#pragma unroll
    for (int j = 0; j < DSUB; ++j) creg[j] = cpq[(static_cast<size_t>(m) * kKsub + c) * DSUB + j];
    if (alpha) {
#pragma unroll
      for (int t = 0; t < R; ++t)
#pragma unroll
        for (int j = 0; j < DSUB; ++j) wreg[t][j] = W[((static_cast<size_t>(m) * R + t) * kKsub + c) * DSUB + j];
    }
  }
  const int q_begin = blockIdx.y * kBoundQueries;
  const int q_end = min(nq, q_begin + kBoundQueries);
  for (int q = q_begin; q < q_end; ++q) {
    float n2 = 0.0f;
    if (alpha) {
      const float* aq = alpha + (static_cast<size_t>(q) * M + m) * r;
      for (int j = 0; j < dsub; ++j) {
        float delta = 0.0f;
        float base;
        if constexpr (kFixed) {
#pragma unroll
          for (int t = 0; t < R; ++t) delta = __fadd_rn(delta, __fmul_rn(aq[t], wreg[t][j]));
          base = creg[j];
        } else {
          for (int t = 0; t < r; ++t)
            delta = __fadd_rn(delta, __fmul_rn(aq[t], W[((static_cast<size_t>(m) * r + t) * kKsub + c) * dsub + j]));
          base = cpq[(static_cast<size_t>(m) * kKsub + c) * dsub + j];
        }
        const float e = __fsub_rn(__fadd_rn(base, delta), base);
        n2 = __fadd_rn(n2, __fmul_rn(e, e));
      }
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) n2 = nan_max(n2, __shfl_xor(n2, o, 64));
    if (lane == 0) s_red[wave] = n2;
    __syncthreads();
    if (c == 0) {
      float mx = nan_max(nan_max(s_red[0], s_red[1]), nan_max(s_red[2], s_red[3]));
      float wm = 1.0f;
      if (wf) {
        wm = 0.0f;
        for (int j = 0; j < dsub; ++j) {
          const float v = wf[static_cast<size_t>(q) * M * dsub + m * dsub + j];
          wm = (v >= 0.0f && v <= FLT_MAX && wm == wm) ? fmaxf(wm, v) : __builtin_nanf("");
        }
      }
      parts[(static_cast<size_t>(q) * 2) * M + m] = mx;
      parts[(static_cast<size_t>(q) * 2 + 1) * M + m] = wm;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void bound_final_kernel(const float* __restrict__ parts, int M, int nq, float grow,
                                                          float* __restrict__ bounds) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= nq) return;
  const float* pd = parts + static_cast<size_t>(q) * 2 * M;
  const float* pw = pd + M;
  float d2 = 0.0f, wm = 0.0f;
  for (int m = 0; m < M; ++m) {
    d2 = __fadd_rn(d2, __fmul_rn(4.0f, pd[m]));
    wm = nan_max(wm, pw[m]);
  }
  bounds[2 * q] = __fmul_rn(sqrtf(wm), 1.0f + 0x1p-19f);
  bounds[2 * q + 1] = __fmul_rn(sqrtf(d2), grow);
}

// List order (rows grouped by coarse centroid, each list in layout order):
// code tiles gathered from the layout's tiles, src_rows[p] = layout row of
// list position p; positions past n get zero words.
__global__ __launch_bounds__(256) void gather_code_tiles_kernel(const uint32_t* __restrict__ src_t, int mw,
                                                                const int32_t* __restrict__ src_rows, int64_t n,
                                                                int64_t n_tiles, uint32_t* __restrict__ dst_t) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= n_tiles * mw * 64) return;
  const int64_t tile = e / (static_cast<int64_t>(mw) * 64);
  const int w = static_cast<int>((e / 64) % mw);
  const int64_t p = tile * 64 + (e & 63);
  uint32_t v = 0;
  if (p < n) {
    const int64_t r = src_rows[p];
    v = src_t[((r >> 6) * mw + w) * 64 + (r & 63)];
  }
  dst_t[e] = v;
}

// Per list position p < n_pad: the row's original id (perm null: the layout
// row is the id); 0 past n.
__global__ __launch_bounds__(256) void gather_list_rows_kernel(const int32_t* __restrict__ perm,
                                                               const int32_t* __restrict__ src_rows, int64_t n,
                                                               int64_t n_pad, int32_t* __restrict__ ids) {
  const int64_t p = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (p >= n_pad) return;
  int32_t id = 0;
  if (p < n) {
    const int64_t r = src_rows[p];
    id = perm ? perm[r] : static_cast<int32_t>(r);
  }
  ids[p] = id;
}

// Per query q (original index): the sub-lists holding rows of its
// interval, in increasing order of their lower bound.  Sub-list s = (list c,
// band b) holds the rows of centroid c whose radius falls in band b of the
// list (radius quantiles), in layout order, so the rows of the query's layout
// interval [x0, x1) are positions [off[s] + rank_s(x0), off[s] + rank_s(x1)),
// rank_s(x) = rows of s among layout rows [0, x): the table entry at the last
// multiple of 2^f_shift below x plus a count over the rest.  Per sub-list
// with selected rows:
//   sdc = a lower bound of ||q - c^||_w: sqrt((sum_m LUT[m][cc_m] - abs) keep)
//         widened down by 2^-20 (0 when not a positive finite number),
//   lb  = sdc - (rmax_s + delta) sqrt(max w), rmax_s the sub-list's largest
//         radius: a lower bound of the distance of each of its rows,
// sorted ascending by lb rounded down to 18 bits of its order-preserving
// code (the item index fills the other 14); the items carry that rounded
// lb, so a scan may stop at the first item it can prune: every later item
// has a bound at least as large.  Before them come, with no bound (NaN), the
// sub-lists of the query's nearest centroid that has selected rows (its
// rows hold the query's nearest rows as a rule, so the scan's k-th distance
// is tight from its first tiles) and any sub-list whose bound is NaN.
// Header: the item count; T, the 64-row tiles of the items before the first
// one the seed's k-th distance prunes (of all items when there is no seed or
// a table entry is negative or NaN); sqrt(max w); delta.
//
// Seed: the distances (summed exactly as the scan sums them) of the
// selected rows among the first kSeedRows positions of the list of the
// centroid with the smallest sdc; when there are k of them, the k-th
// smallest bounds the query's k-th distance (k distinct selected rows lie
// at or below it) and goes to the query's shared threshold, with the
// largest id so rows at that distance stay eligible.
template <typename LutT>
__global__ __launch_bounds__(1024) void list_plan_kernel(const ListPlanArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int C = a.C, S = a.n_sub, Sp = a.Sp;
  float* s_sdc = reinterpret_cast<float*>(smem);                          // [C]
  unsigned char* scratch = smem + ((static_cast<size_t>(C) * 4 + 15) & ~size_t{15});
  LutT* s_lut = reinterpret_cast<LutT*>(scratch);                         // phase 1
  uint32_t* s_seed = reinterpret_cast<uint32_t*>(scratch + static_cast<size_t>(a.m) * kKsub * sizeof(LutT));
  int32_t* s_cnt = reinterpret_cast<int32_t*>(scratch);                   // phase 2: [S]
  uint32_t* s_key = reinterpret_cast<uint32_t*>(s_cnt + S);               // phase 2: [Sp]
  __shared__ int s_count;
  __shared__ unsigned long long s_near;   // (sdc bits, centroid) of the nearest selected centroid
  __shared__ unsigned long long s_first;  // (sdc bits, centroid) of the nearest centroid
  __shared__ int s_lut_bad;               // a table entry is negative or NaN: no pruning
  __shared__ int s_stop;                  // the first item the seed's bound prunes
  __shared__ uint32_t s_seed_kth;         // the seed's k-th distance (order-preserving bits)
  const int q = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t x0 = a.iv[2 * q], x1 = a.iv[2 * q + 1];
  const float sw = a.bounds[2 * q], delta = a.bounds[2 * q + 1];
  float* hdr = a.hdr + 4 * static_cast<size_t>(q);
  for (int i = tid; i < kListSlots; i += 1024) a.slots[static_cast<size_t>(q) * kListSlots + i] = ~0u;
  if (x1 <= x0) {
    if (tid == 0) {
      hdr[0] = __int_as_float(0);
      hdr[1] = __int_as_float(0);
      hdr[2] = sw;
      hdr[3] = delta;
    }
    return;
  }
  // Phase 1: the table, then each centroid's bound.
  const LutT* lut = static_cast<const LutT*>(a.lut) + static_cast<size_t>(q) * a.m * kKsub;
  const int lut_vecs = a.m * kKsub * static_cast<int>(sizeof(LutT)) / 16;
  if (tid == 0) {
    s_count = 0;
    s_near = ~0ull;
    s_first = ~0ull;
    s_lut_bad = 0;
    s_stop = 0x7FFFFFFF;
  }
  __syncthreads();
  {
    bool bad = false;
    for (int v = tid; v < lut_vecs; v += 1024) {
      const uint4 x = reinterpret_cast<const uint4*>(lut)[v];
      reinterpret_cast<uint4*>(s_lut)[v] = x;
      const LutT* xe = reinterpret_cast<const LutT*>(&x);
      for (int e = 0; e < 16 / static_cast<int>(sizeof(LutT)); ++e) bad = bad || !(widen(xe[e]) >= 0.0f);
    }
    if (bad) s_lut_bad = 1;
  }
  __syncthreads();
  for (int c = tid; c < C; c += 1024) {
    float d = 0.0f;
    for (int w = 0; w < a.mw; ++w) {
      const uint32_t word = a.cc_t[static_cast<size_t>(w) * C + c];
      for (int b = 0; b < 4; ++b) {
        const int m = 4 * w + b;
        if (m < a.m) d = __fadd_rn(d, widen(s_lut[m * kKsub + static_cast<int>((word >> (8 * b)) & 0xFFu)]));
      }
    }
    const float lo = __fmul_rn(__fsub_rn(d, a.abs_m), a.keep);
    s_sdc[c] = lo > 0.0f && lo <= FLT_MAX ? __fmul_rn(sqrtf(lo), 1.0f - 0x1p-20f) : 0.0f;
    atomicMin(&s_first, (static_cast<unsigned long long>(ordered_bits(s_sdc[c])) << 32) | static_cast<uint32_t>(c));
  }
  __syncthreads();
  {
    // The seed (see above), from the nearest centroid's list.
    const int c0 = static_cast<int>(s_first & 0xFFFFFFFFu);
    const int32_t p0 = a.sub_off[c0 * kBands], p1 = min(a.sub_off[c0 * kBands + kBands], p0 + kSeedRows);
    for (int i = tid; i < kSeedRows; i += 1024) {
      uint32_t key = ~0u;
      const int32_t p = p0 + i;
      if (p < p1) {
        const int64_t r = a.lrow[p];
        if (r >= x0 && r < x1) {
          const uint32_t* tile = a.codes_t + static_cast<size_t>(p >> 6) * a.mw * 64 + (p & 63);
          float d = 0.0f;
          for (int w = 0; w < a.mw; ++w) {
            const uint32_t word = tile[w * 64];
            for (int b = 0; b < 4; ++b) {
              const int m = 4 * w + b;
              if (m < a.m) d = __fadd_rn(d, widen(s_lut[m * kKsub + static_cast<int>((word >> (8 * b)) & 0xFFu)]));
            }
          }
          key = ordered_bits(d);
        }
      }
      s_seed[i] = key;
    }
    __syncthreads();
    for (int size = 2; size <= kSeedRows; size <<= 1) {
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int p = tid; p < kSeedRows / 2; p += 1024) {
          const int i = ((p & ~(stride - 1)) << 1) | (p & (stride - 1));
          const int j = i | stride;
          const uint32_t x = s_seed[i], y = s_seed[j];
          const bool up = (i & size) == 0;
          if (up ? (x > y) : (x < y)) {
            s_seed[i] = y;
            s_seed[j] = x;
          }
        }
        __syncthreads();
      }
    }
    if (tid == 0) s_seed_kth = a.k <= kSeedRows ? s_seed[a.k - 1] : ~0u;
    if (tid == 0 && a.k <= kSeedRows && s_seed[a.k - 1] != ~0u)
      atomicMin(reinterpret_cast<unsigned long long*>(a.gthr + q),
                (static_cast<unsigned long long>(s_seed[a.k - 1]) << 32) | 0xFFFFFFFFull);
  }
  __syncthreads();
  // Phase 2: ranks at x0 (kept in tmp_r0), then at x1 with the items'
  // rows, bounds and sort keys.
  const size_t base = static_cast<size_t>(q) * S;
  const int64_t b0 = x0 >> a.f_shift, b1 = x1 >> a.f_shift;
  for (int pass = 0; pass < 2; ++pass) {
    const int64_t x = pass == 0 ? x0 : x1, bx = pass == 0 ? b0 : b1;
    for (int s = tid; s < S; s += 1024) s_cnt[s] = a.cnt_f[bx * S + s];
    __syncthreads();
    for (int64_t r = (bx << a.f_shift) + tid; r < x; r += 1024)
      atomicAdd(&s_cnt[static_cast<int>(a.words[r] & 0xFFFFu) * kBands + a.band[r]], 1);
    __syncthreads();
    if (pass == 0) {
      for (int s = tid; s < S; s += 1024) a.tmp_r0[base + s] = a.sub_off[s] + s_cnt[s];
    } else {
      for (int s = tid; s < S; s += 1024) {
        const int32_t r0 = a.tmp_r0[base + s];
        const int32_t r1 = a.sub_off[s] + s_cnt[s];
        a.tmp_r1[base + s] = r1;
        if (r1 > r0) {
          const int c = s / kBands;
          atomicMin(&s_near, (static_cast<unsigned long long>(ordered_bits(s_sdc[c])) << 32) |
                                 static_cast<uint32_t>(c));
        }
      }
    }
    __syncthreads();
  }
  {
    const int near = s_near == ~0ull ? -1 : static_cast<int>(s_near & 0xFFFFFFFFu);
    int mine = 0;
    for (int s = tid; s < Sp; s += 1024) {
      uint32_t key = ~0u;
      if (s < S) {
        const int32_t r0 = a.tmp_r0[base + s];
        const int32_t r1 = a.tmp_r1[base + s];
        if (r1 > r0) {
          const float lb = __fsub_rn(s_sdc[s / kBands], __fmul_rn(__fadd_rn(a.rmax[s], delta), sw));
          // the nearest centroid's sub-lists and NaN bounds sort first with
          // the top bits 0, carried as NaN (never pruned)
          const uint32_t ob = lb == lb && s / kBands != near ? ordered_bits(lb) : 0u;
          key = (ob & ~uint32_t{kItemMask}) | static_cast<uint32_t>(s);
          ++mine;
        }
      }
      s_key[s] = key;
    }
    atomicAdd(&s_count, mine);
  }
  __syncthreads();
  // ascending bitonic sort of the Sp keys
  for (int size = 2; size <= Sp; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = tid; p < Sp / 2; p += 1024) {
        const int i = ((p & ~(stride - 1)) << 1) | (p & (stride - 1));
        const int j = i | stride;
        const uint32_t x = s_key[i], y = s_key[j];
        const bool up = (i & size) == 0;
        if (up ? (x > y) : (x < y)) {
          s_key[i] = y;
          s_key[j] = x;
        }
      }
      __syncthreads();
    }
  }
  const int n_items = s_count;
  int32_t* s_nt = s_cnt;   // the counts are no longer needed: tile counts in sorted order
  for (int i = tid; i < n_items; i += 1024) {
    const uint32_t key = s_key[i];
    const int s = static_cast<int>(key & kItemMask);
    const int32_t r0 = a.tmp_r0[base + s], r1 = a.tmp_r1[base + s];
    s_nt[i] = ((r1 - 1) >> 6) - (r0 >> 6) + 1;
    a.it_r0[base + i] = r0;
    a.it_r1[base + i] = r1;
    const uint32_t ob = key & ~uint32_t{kItemMask};
    a.it_lb[base + i] = ob == 0u ? __builtin_nanf("") : from_ordered_bits(ob);
  }
  __syncthreads();
  // inclusive scan of the tile counts (Hillis-Steele), then exclusive
  for (int off = 1; off < n_items; off <<= 1) {
    int v[kMaxItems / 1024] = {};
#pragma unroll
    for (int u = 0; u < kMaxItems / 1024; ++u) {
      const int i = tid + u * 1024;
      if (i < n_items && i >= off) v[u] = s_nt[i - off];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kMaxItems / 1024; ++u) {
      const int i = tid + u * 1024;
      if (i < n_items) s_nt[i] += v[u];
    }
    __syncthreads();
  }
  for (int i = tid; i < n_items; i += 1024) a.it_t[base + i] = i == 0 ? 0 : s_nt[i - 1];
  // T: the items' bounds rise in order, so the first item the seed's k-th
  // distance prunes (the test the scan makes, whose bound is never looser)
  // ends what any scan of the query visits.
  if (s_lut_bad == 0 && s_seed_kth != ~0u) {
    const float cut = from_ordered_bits(s_seed_kth);
    for (int i = tid; i < n_items; i += 1024) {
      const uint32_t ob = s_key[i] & ~uint32_t{kItemMask};
      const float lb = ob == 0u ? __builtin_nanf("") : from_ordered_bits(ob);
      if (lb > 0.0f && __fsub_rn(__fmul_rn(__fmul_rn(lb, lb), a.keep), a.abs_m) > cut) atomicMin(&s_stop, i);
    }
  }
  __syncthreads();
  if (tid == 0) {
    const int stop = min(s_stop, n_items);
    hdr[0] = __int_as_float(n_items);
    hdr[1] = __int_as_float(stop > 0 ? s_nt[stop - 1] : 0);
    hdr[2] = sw;
    hdr[3] = delta;
  }
}

}  // namespace

int64_t coarse_samples(int64_t n, int C) {
  return std::min<int64_t>(n, std::max<int64_t>(static_cast<int64_t>(C) * 64, 65536));
}

float coarse_keep(int m, int dsub, int lut_dtype) {
  const float eps =
      2.0f * static_cast<float>(dsub + m + 8) * 0x1p-24f + 0x1p-18f + (lut_dtype == 1 ? 0x1p-10f : 0.0f);
  return 1.0f - eps;
}

float coarse_abs(int m, int lut_dtype) {
  // binary16 entries below 2^-14 are subnormal (absolute error up to 2^-25
  // each); fp32 subnormal rounding stays far below 2^-120 over any table
  return lut_dtype == 1 ? static_cast<float>(m) * 0x1p-24f : 0x1p-120f;
}

hipError_t launch_coarse_sample(const uint32_t* codes_t, int mw, int m, int dsub, const float* cpq, int64_t S,
                                int64_t stride, float* X, hipStream_t s) {
  const int64_t total = S * m * dsub;
  coarse_sample_kernel<<<static_cast<unsigned>((total + 255) / 256), 256, 0, s>>>(codes_t, mw, dsub, m * dsub, cpq,
                                                                               S, stride, X);
  return hipGetLastError();
}

hipError_t launch_coarse_kmeans_step(const float* X, int64_t S, int D, float* cent, int C, int32_t* assign,
                                     hipStream_t s) {
  coarse_assign_kernel<<<static_cast<unsigned>((S + 255) / 256), 256, 0, s>>>(X, S, D, cent, C, assign);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  coarse_update_kernel<<<static_cast<unsigned>(C), kMaxD, 0, s>>>(X, S, D, assign, cent);
  return hipGetLastError();
}

hipError_t launch_coarse_encode(const float* cent, int C, int m, int mw, int dsub, const float* cpq, uint32_t* cc,
                                float* chat, hipStream_t s) {
  const int64_t total = static_cast<int64_t>(C) * mw;
  coarse_encode_kernel<<<static_cast<unsigned>((total + 255) / 256), 256, 0, s>>>(cent, C, m, mw, dsub, cpq, cc, chat);
  return hipGetLastError();
}

hipError_t launch_coarse_rows(const uint32_t* codes_t, int64_t n, int64_t n_pad, int m, int mw, int dsub,
                              const float* cpq, const float* chat, int C, uint32_t* words, hipStream_t s) {
  coarse_rows_kernel<<<static_cast<unsigned>((n_pad + 255) / 256), 256, 0, s>>>(codes_t, n, n_pad, m, mw, dsub, cpq,
                                                                             chat, C, words);
  return hipGetLastError();
}

hipError_t launch_lut_bounds(const float* alpha, const float* wf, const float* cpq, const float* W, int nq, int m,
                             int r, int dsub, float* parts, float* bounds, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const dim3 g(static_cast<unsigned>(m), static_cast<unsigned>((nq + kBoundQueries - 1) / kBoundQueries));
  if (dsub == 2 && r == 8)
    bound_parts_kernel<2, 8><<<g, 256, 0, s>>>(alpha, wf, cpq, W, m, dsub, r, nq, parts);
  else if (dsub == 8 && r == 8)
    bound_parts_kernel<8, 8><<<g, 256, 0, s>>>(alpha, wf, cpq, W, m, dsub, r, nq, parts);
  else
    bound_parts_kernel<0, 0><<<g, 256, 0, s>>>(alpha, wf, cpq, W, m, dsub, r, nq, parts);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const float grow = 1.0f + 2.0f * static_cast<float>(dsub + m + 8) * 0x1p-24f + 0x1p-20f;
  bound_final_kernel<<<static_cast<unsigned>((nq + 255) / 256), 256, 0, s>>>(parts, m, nq, grow, bounds);
  return hipGetLastError();
}

size_t list_plan_lds_bytes(int m, int lut_dtype, int C) {
  const size_t lut = static_cast<size_t>(m) * kKsub * (lut_dtype == 1 ? 2 : 4) + kSeedRows * 4;
  const size_t items = static_cast<size_t>(C) * kBands * 4 + static_cast<size_t>(list_plan_width(C)) * 4;
  return ((static_cast<size_t>(C) * 4 + 15) & ~size_t{15}) + std::max(lut, items);
}

int list_plan_width(int C) {
  int p = 2;
  while (p < C * kBands) p <<= 1;
  return p;
}

hipError_t launch_list_plan(const ListPlanArgs& a, int lut_dtype, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  const void* fn = lut_dtype == 1 ? reinterpret_cast<const void*>(&list_plan_kernel<__half>)
                                  : reinterpret_cast<const void*>(&list_plan_kernel<float>);
  const size_t lds = list_plan_lds_bytes(a.m, lut_dtype, a.C);
  if (a.n_sub != a.C * kBands || a.Sp != list_plan_width(a.C) || a.Sp > kMaxItems) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  ListPlanArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchKernel(fn, dim3(static_cast<unsigned>(a.nq)), dim3(1024), kargs, lds, s);
}

hipError_t launch_gather_list(const uint32_t* src_t, int mw, const int32_t* perm, const int32_t* src_rows, int64_t n,
                              int64_t n_tiles, uint32_t* dst_t, int32_t* ids, hipStream_t s) {
  const int64_t total = n_tiles * mw * 64;
  gather_code_tiles_kernel<<<static_cast<unsigned>((total + 255) / 256), 256, 0, s>>>(src_t, mw, src_rows, n, n_tiles,
                                                                                    dst_t);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n_pad = n_tiles * 64;
  gather_list_rows_kernel<<<static_cast<unsigned>((n_pad + 255) / 256), 256, 0, s>>>(perm, src_rows, n, n_pad, ids);
  return hipGetLastError();
}

}  // namespace ifvs
