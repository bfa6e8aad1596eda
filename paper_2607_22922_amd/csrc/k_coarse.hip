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
  __shared__ float s_red[kBoundQueries][4];
  // every query's shift first (independent loads together), then one
  // reduction round
  float n2[kBoundQueries];
#pragma unroll
  for (int qi = 0; qi < kBoundQueries; ++qi) {
    const int q = q_begin + qi;
    n2[qi] = 0.0f;
    if (alpha && q < q_end) {
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
        n2[qi] = __fadd_rn(n2[qi], __fmul_rn(e, e));
      }
    }
  }
#pragma unroll
  for (int qi = 0; qi < kBoundQueries; ++qi) {
    float v = n2[qi];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) v = nan_max(v, __shfl_xor(v, o, 64));
    if (lane == 0) s_red[qi][wave] = v;
  }
  __syncthreads();
  const int q = q_begin + c;
  if (c < kBoundQueries && q < q_end) {
    const float mx = nan_max(nan_max(s_red[c][0], s_red[c][1]), nan_max(s_red[c][2], s_red[c][3]));
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
}

// sqrt(max_m parts[1][m]) widened by 2^-19 and sqrt(sum_m 4 parts[0][m]) *
// grow, from one query's parts (pd = parts[q]).
__device__ void reduce_bound_parts(const float* __restrict__ pd, int M, float grow, float& sw, float& delta) {
  const float* pw = pd + M;
  float d2 = 0.0f, wm = 0.0f;
  for (int m0 = 0; m0 < M; m0 += 16) {
    // sixteen subspaces' loads at a time, summed in subspace order
    float vd[16], vw[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      vd[u] = m0 + u < M ? pd[m0 + u] : 0.0f;
      vw[u] = m0 + u < M ? pw[m0 + u] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      if (m0 + u < M) {
        d2 = __fadd_rn(d2, __fmul_rn(4.0f, vd[u]));
        wm = nan_max(wm, vw[u]);
      }
    }
  }
  sw = __fmul_rn(sqrtf(wm), 1.0f + 0x1p-19f);
  delta = __fmul_rn(sqrtf(d2), grow);
}

__global__ __launch_bounds__(256) void bound_final_kernel(const float* __restrict__ parts, int M, int nq, float grow,
                                                          float* __restrict__ bounds) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= nq) return;
  reduce_bound_parts(parts + static_cast<size_t>(q) * 2 * M, M, grow, bounds[2 * q], bounds[2 * q + 1]);
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

// The job table (one 1024-thread workgroup): per query position, jobs =
// min(max_jobs, ceil(T / kJobTiles)) chunks of about equal size (multiples of
// kScanWaves positions) of its T tiles (the tiles of the items the plan
// kept), the queries with the most tiles first; the keys each position's
// jobs write are counted for the merge; the job counter is reset.  LDS:
// list_jobs_lds_bytes(nq) at smem.
__device__ void build_job_table(const ListJobArgs& a, unsigned char* smem) {
  uint64_t* s_key = reinterpret_cast<uint64_t*>(smem);   // [np2]
  int32_t* s_base = reinterpret_cast<int32_t*>(s_key + a.np2);   // [np2 + 1]
  const int tid = threadIdx.x;
  for (int i = tid; i < a.np2; i += 1024) {
    uint64_t key = ~0ull;
    if (i < a.nq) {
      const int q = a.qorder[i];
      const int w = __float_as_int(a.hdr[4 * static_cast<size_t>(q) + 1]);
      key = (static_cast<uint64_t>(0x7FFFFFFF - w) << 32) | static_cast<uint32_t>(i);
    }
    s_key[i] = key;
  }
  __syncthreads();
  for (int size = 2; size <= a.np2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = tid; p < a.np2 / 2; p += 1024) {
        const int i = ((p & ~(stride - 1)) << 1) | (p & (stride - 1));
        const int j = i | stride;
        const uint64_t x = s_key[i], y = s_key[j];
        const bool up = (i & size) == 0;
        if (up ? (x > y) : (x < y)) {
          s_key[i] = y;
          s_key[j] = x;
        }
      }
      __syncthreads();
    }
  }
  // jobs per position in sorted order, then their exclusive prefix (serial
  // per thread block of positions, then across blocks)
  auto jobs_of = [&](int i) -> int {
    if (i >= a.nq) return 0;
    const int w = 0x7FFFFFFF - static_cast<int>(s_key[i] >> 32);
    return w <= 0 ? 0 : min(a.max_jobs, (w + kJobTiles - 1) / kJobTiles);
  };
  const int per = (a.np2 + 1023) / 1024;
  int mine = 0;
  for (int u = 0; u < per; ++u) mine += jobs_of(tid * per + u);
  s_base[tid] = mine;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int v = tid >= off ? s_base[tid - off] : 0;
    __syncthreads();
    s_base[tid] += v;
    __syncthreads();
  }
  int base = tid == 0 ? 0 : s_base[tid - 1];
  for (int u = 0; u < per; ++u) {
    const int i = tid * per + u;
    if (i >= a.nq) break;
    const int pos = static_cast<int>(s_key[i] & 0xFFFFFFFFu);
    const int w = 0x7FFFFFFF - static_cast<int>(s_key[i] >> 32);
    const int nj = jobs_of(i);
    const int chunk = nj > 0 ? ((w + nj - 1) / nj + kScanWaves - 1) / kScanWaves * kScanWaves : 0;
    for (int c = 0; c < nj; ++c)
      a.jobs[base + c] = make_int4(pos, c, c * chunk, min(w, (c + 1) * chunk));
    base += nj;
    a.n_keys[pos] = nj * kScanWaves * a.k;   // the merge reads the written chunks only
  }
  if (tid == 1023) {
    *a.job_total = s_base[1023];
    *a.job_next = 0;
  }
}

// Wavefront minimum / maximum (one LDS atomic per wavefront then, not one
// per lane on a single address).
__device__ __forceinline__ unsigned long long wave_min_u64(unsigned long long v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long y = __shfl_xor(v, o, 64);
    v = y < v ? y : v;
  }
  return v;
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), o, 64));
    v = y < v ? y : v;
  }
  return v;
}
__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), o, 64));
    v = y > v ? y : v;
  }
  return v;
}

// Exclusive prefix sum of one value per thread over a 1024-thread
// workgroup; the total goes to every thread.  s_w: 16 ints of LDS.
__device__ int block_exclusive_sum(int v, int* s_w, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_w[wave] = x;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < 16; ++w) {
    const int t = s_w[w];
    off += w < wave ? t : 0;
    tot += t;
  }
  __syncthreads();
  total = tot;
  return off + x - v;
}

// Per query q (original index): the sub-lists holding rows of its
// interval, in increasing order of a lower bound of their rows' distances.
// Sub-list s = (list c, band b) holds the rows of centroid c whose radius
// falls in band b of the list (radius quantiles), in layout order, so the
// rows of the query's layout interval [x0, x1) are positions
// [off[s] + rank_s(x0), off[s] + rank_s(x1)), rank_s(x) = rows of s among
// layout rows [0, x): the table entry at the last multiple of 2^f_shift
// below x plus a count over the rest.  Per sub-list with selected rows:
//   sdc = a lower bound of ||q - c^||_w: sqrt((sum_m LUT[m][cc_m] - abs) keep)
//         widened down by 2^-20 (0 when not a positive finite number),
//   lb  = sdc - (rmax_s + delta) sqrt(max w), rmax_s the sub-list's largest
//         radius: a lower bound of the distance of each of its rows.
// Order: a counting sort into kPlanBuckets buckets: bucket 0 for the
// sub-lists of the query's nearest centroid that has selected rows (its rows
// hold the query's nearest rows as a rule, so the scan's k-th distance is
// tight from its first tiles) and those whose lb is NaN, bucket 1 for lb <= 0
// (never pruned), then buckets of 2^shift consecutive order-preserving codes
// of positive lb (a monotone function of lb, so every lb of a bucket is at
// most every lb of the next; shift the least that fits the query's range).
// Each item carries its bucket's smallest lb (NaN in bucket 0): the carried
// bounds never decrease along the order, so a scan may stop at the first
// item it can prune, and the items from the first bucket that the seed's
// k-th distance prunes on are left out.  The order inside a bucket is the
// order the threads reach it.  Header: the items kept; T, their 64-row
// tiles; sqrt(max w); delta.
//
// Seed: the distances (summed exactly as the scan sums them) of the
// selected rows among the first kSeedRows positions of the list of the
// centroid with the smallest sdc; when there are k of them, the k-th
// smallest (a radix select, 8 bits a pass) bounds the query's k-th distance
// (k distinct selected rows lie at or below it) and goes to the query's
// shared threshold, with the largest id so rows at that distance stay
// eligible.
template <int MT, typename LutT>
__device__ __forceinline__ void plan_one_query(const ListPlanArgs& a, const float sw, const float delta) {
  constexpr int kMW = (MT + 3) / 4;
  constexpr int kSPer = kMaxItems / 1024;   // sub-lists a thread holds (in registers)
  static_assert(kSeedRows % 1024 == 0 && kPlanBuckets % 1024 == 0 && kMaxItems % 1024 == 0,
                "a 1024-thread plan takes whole shares");
  extern __shared__ __align__(16) unsigned char smem[];
  const int C = a.C, S = a.n_sub;
  float* s_sdc = reinterpret_cast<float*>(smem);                          // [C]
  int32_t* s_off = reinterpret_cast<int32_t*>(s_sdc + C);                 // [C + 1] first list position of centroid c
  unsigned char* scratch = smem + ((static_cast<size_t>(2 * C + 1) * 4 + 15) & ~size_t{15});
  LutT* s_lut = reinterpret_cast<LutT*>(scratch);                         // phase 1
  int32_t* s_cnt = reinterpret_cast<int32_t*>(scratch);                   // phase 2: [S] ranks, then items
  int32_t* s_hist = s_cnt + S;                                            // phase 2: [kPlanBuckets]
  uint32_t* s_bmin = reinterpret_cast<uint32_t*>(s_hist + kPlanBuckets);  // phase 2: [kPlanBuckets]
  __shared__ int s_count;
  __shared__ unsigned long long s_near;   // (sdc bits, centroid) of the nearest selected centroid
  __shared__ unsigned long long s_first;  // (sdc bits, centroid) of the nearest centroid
  __shared__ int s_lut_bad;               // a table entry is negative or NaN: no pruning
  __shared__ int s_stop;                  // the first bucket the seed's bound prunes
  __shared__ uint32_t s_lo, s_hi;         // smallest and largest positive bounded lb (order-preserving bits)
  __shared__ int s_rh[256];               // radix select histogram
  __shared__ int s_pick[2];
  __shared__ int s_w[16];
  const int q = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t x0 = a.iv[2 * q], x1 = a.iv[2 * q + 1];
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
  // A row's distance from its code words, summed as the scan sums it.
  auto code_distance = [&](const uint32_t (&wd)[kMW]) -> float {
    float d = 0.0f;
#pragma unroll
    for (int m = 0; m < MT; ++m)
      d = __fadd_rn(d, widen(s_lut[m * kKsub + static_cast<int>((wd[m >> 2] >> (8 * (m & 3))) & 0xFFu)]));
    return d;
  };
  // Phase 1: the table, then each centroid's bound.
  const LutT* lut = static_cast<const LutT*>(a.lut) + static_cast<size_t>(q) * MT * kKsub;
  constexpr int kLutVecs = MT * kKsub * static_cast<int>(sizeof(LutT)) / 16;
  if (tid == 0) {
    s_count = 0;
    s_near = ~0ull;
    s_first = ~0ull;
    s_lut_bad = 0;
    s_stop = 0x7FFFFFFF;
    s_lo = ~0u;
    s_hi = 0u;
  }
  __syncthreads();
  {
    bool bad = false;
    for (int v = tid; v < kLutVecs; v += 1024) {
      const uint4 x = reinterpret_cast<const uint4*>(lut)[v];
      reinterpret_cast<uint4*>(s_lut)[v] = x;
      const LutT* xe = reinterpret_cast<const LutT*>(&x);
#pragma unroll
      for (int e = 0; e < 16 / static_cast<int>(sizeof(LutT)); ++e) bad = bad || !(widen(xe[e]) >= 0.0f);
    }
    if (bad) s_lut_bad = 1;
  }
  __syncthreads();
  {
    unsigned long long first = ~0ull;
    for (int c = tid; c <= C; c += 1024) {
      // (its list's first position too, for the seed: sub_off[C * kBands] ends the last list)
      s_off[c] = a.sub_off[c * kBands];
      if (c == C) break;
      uint32_t wd[kMW];
#pragma unroll
      for (int w = 0; w < kMW; ++w) wd[w] = a.cc_t[static_cast<size_t>(w) * C + c];
      const float lo = __fmul_rn(__fsub_rn(code_distance(wd), a.abs_m), a.keep);
      const float sdc = lo > 0.0f && lo <= FLT_MAX ? __fmul_rn(sqrtf(lo), 1.0f - 0x1p-20f) : 0.0f;
      s_sdc[c] = sdc;
      const unsigned long long key = (static_cast<unsigned long long>(ordered_bits(sdc)) << 32) | static_cast<uint32_t>(c);
      first = key < first ? key : first;
    }
    first = wave_min_u64(first);
    if ((tid & 63) == 0 && first != ~0ull) atomicMin(&s_first, first);
  }
  __syncthreads();
  uint32_t seed_kth = ~0u;   // the seed's k-th distance (order-preserving bits; all ones: none)
  if (a.k <= kSeedRows) {
    // The seed (see above), from the nearest centroid's list.
    constexpr int kPer = kSeedRows / 1024;
    const int c0 = static_cast<int>(s_first & 0xFFFFFFFFu);
    const int32_t p0 = s_off[c0], p1 = min(s_off[c0 + 1], p0 + kSeedRows);
    int64_t row[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int32_t p = p0 + tid + u * 1024;
      row[u] = p < p1 ? a.lrow[p] : -1;
    }
    uint32_t key[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      key[u] = ~0u;
      if (row[u] >= x0 && row[u] < x1) {
        const int32_t p = p0 + tid + u * 1024;
        const uint32_t* tile = a.codes_t + static_cast<size_t>(p >> 6) * kMW * 64 + (p & 63);
        uint32_t wd[kMW];
#pragma unroll
        for (int w = 0; w < kMW; ++w) wd[w] = tile[w * 64];
        key[u] = ordered_bits(code_distance(wd));
      }
    }
    // k-th smallest of the kSeedRows keys (all ones for rows not selected):
    // per pass the digit whose bin holds it among the keys with the digits
    // found so far.  Three passes fix its top 24 bits; the seed is the top of
    // that bin (at most 255 ulps above the k-th value, and still a bound:
    // k selected rows lie at or below it; all ones stays all ones).
    uint32_t prefix = 0, pmask = 0;
    int kk = a.k;
    for (int shift = 24; shift >= 8; shift -= 8) {
      if (tid < 256) s_rh[tid] = 0;
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kPer; ++u)
        if ((key[u] & pmask) == prefix) atomicAdd(&s_rh[(key[u] >> shift) & 0xFFu], 1);
      __syncthreads();
      if (tid < 64) {
        int c[4], sum = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          c[j] = s_rh[4 * tid + j];
          sum += c[j];
        }
        int x = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(x, o, 64);
          if (tid >= o) x += y;
        }
        int acc = x - sum;
        if (acc < kk && kk <= x) {
          int j = 0;
          while (acc + c[j] < kk) acc += c[j++];
          s_pick[0] = 4 * tid + j;
          s_pick[1] = kk - acc;
        }
      }
      __syncthreads();
      prefix |= static_cast<uint32_t>(s_pick[0]) << shift;
      pmask |= 0xFFu << shift;
      kk = s_pick[1];
    }
    seed_kth = prefix | 0xFFu;
    if (tid == 0 && seed_kth != ~0u)
      atomicMin(reinterpret_cast<unsigned long long*>(a.gthr + q),
                (static_cast<unsigned long long>(seed_kth) << 32) | 0xFFFFFFFFull);
  }
  __syncthreads();
  // Phase 2: each sub-list's positions of rows x0 and x1 (ranks), held by
  // the thread of sub-list s = tid + 1024 j in slot j: the rank table's rows
  // at x0 and x1 plus counts over the rows after them (fewer than
  // 2^f_shift).  The table rows and the first 4096 rows after each table
  // entry (four a thread) go out in one round; longer stretches (f_shift
  // above 12) take more rounds.
  auto count_rest = [&](int64_t from, int64_t x) {
    for (int64_t r = from + tid; r < x; r += 4 * 1024) {
      uint32_t wv[4];
      int bv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t rr = r + u * 1024;
        wv[u] = rr < x ? a.words[rr] : 0u;
        bv[u] = rr < x ? a.band[rr] : 0;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (r + u * 1024 < x) atomicAdd(&s_cnt[static_cast<int>(wv[u] & 0xFFFFu) * kBands + bv[u]], 1);
    }
  };
  int32_t r0[kSPer], r1[kSPer];
  float rm[kSPer];   // each selected sub-list's largest radius
  {
    const int64_t bx0 = x0 >> a.f_shift, bx1 = x1 >> a.f_shift;
    int32_t c0[kSPer], c1[kSPer], so[kSPer];
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      const int s = tid + j * 1024;
      c0[j] = s < S ? a.cnt_f[bx0 * S + s] : 0;
      c1[j] = s < S ? a.cnt_f[bx1 * S + s] : 0;
    }
    uint32_t w0[4], w1[4];
    int b0[4], b1[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t ra = (bx0 << a.f_shift) + tid + u * 1024, rb = (bx1 << a.f_shift) + tid + u * 1024;
      w0[u] = ra < x0 ? a.words[ra] : 0u;
      b0[u] = ra < x0 ? a.band[ra] : 0;
      w1[u] = rb < x1 ? a.words[rb] : 0u;
      b1[u] = rb < x1 ? a.band[rb] : 0;
    }
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      const int s = tid + j * 1024;
      if (s < S) s_cnt[s] = c0[j];
    }
    __syncthreads();
    // (the offsets in c0's registers, on their way during the counting)
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      const int s = tid + j * 1024;
      so[j] = s < S ? a.sub_off[s] : 0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t ra = (bx0 << a.f_shift) + tid + u * 1024;
      if (ra < x0) atomicAdd(&s_cnt[static_cast<int>(w0[u] & 0xFFFFu) * kBands + b0[u]], 1);
    }
    count_rest((bx0 << a.f_shift) + 4 * 1024, x0);
    __syncthreads();
    // (entry s is this thread's until the next barrier: x0's rank out, x1's
    // table row in)
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      const int s = tid + j * 1024;
      r0[j] = s < S ? so[j] + s_cnt[s] : 0;
      if (s < S) s_cnt[s] = c1[j];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rb = (bx1 << a.f_shift) + tid + u * 1024;
      if (rb < x1) atomicAdd(&s_cnt[static_cast<int>(w1[u] & 0xFFFFu) * kBands + b1[u]], 1);
    }
    count_rest((bx1 << a.f_shift) + 4 * 1024, x1);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      const int s = tid + j * 1024;
      r1[j] = s < S ? so[j] + s_cnt[s] : 0;
    }
  }
  // Items: the nearest selected centroid, the bounds' range, then the
  // buckets' counts and smallest bounds.
  {
    unsigned long long nearest = ~0ull;
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      const int s = tid + j * 1024;
      if (s < S && r1[j] > r0[j]) {
        const int c = s / kBands;
        const unsigned long long key = (static_cast<unsigned long long>(ordered_bits(s_sdc[c])) << 32) |
                                       static_cast<uint32_t>(c);
        nearest = key < nearest ? key : nearest;
      }
    }
    nearest = wave_min_u64(nearest);
    if ((tid & 63) == 0 && nearest != ~0ull) atomicMin(&s_near, nearest);
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {   // (on their way across the barrier)
      const int s = tid + j * 1024;
      rm[j] = s < S && r1[j] > r0[j] ? a.rmax[s] : 0.0f;
    }
    for (int b = tid; b < kPlanBuckets; b += 1024) {
      s_hist[b] = 0;
      s_bmin[b] = ~0u;
    }
  }
  __syncthreads();
  const int near = s_near == ~0ull ? -1 : static_cast<int>(s_near & 0xFFFFFFFFu);
  float lb[kSPer];
  {
    int mine = 0;
    uint32_t lo_b = ~0u, hi_b = 0u;
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      const int s = tid + j * 1024;
      lb[j] = 0.0f;
      if (s < S && r1[j] > r0[j]) {
        ++mine;
        lb[j] = __fsub_rn(s_sdc[s / kBands], __fmul_rn(__fadd_rn(rm[j], delta), sw));
        if (lb[j] > 0.0f && s / kBands != near) {
          lo_b = min(lo_b, ordered_bits(lb[j]));
          hi_b = max(hi_b, ordered_bits(lb[j]));
        }
      }
    }
    lo_b = wave_min_u32(lo_b);
    hi_b = wave_max_u32(hi_b);
    if ((tid & 63) == 0 && lo_b != ~0u) {
      atomicMin(&s_lo, lo_b);
      atomicMax(&s_hi, hi_b);
    }
    mine = wave_sum_i32(mine);
    if ((tid & 63) == 0 && mine) atomicAdd(&s_count, mine);
  }
  __syncthreads();
  // positive bounds: buckets of 2^shift order-preserving codes from the
  // smallest, shift the least that fits the range in the buckets
  const uint32_t lo_bits = s_lo, span = s_lo == ~0u ? 0u : s_hi - s_lo;
  int shift = 0;
  while ((span >> shift) > static_cast<uint32_t>(kPlanBuckets - 3)) ++shift;
  auto bucket = [&](int s, float v) -> int {
    if (!(v == v) || s / kBands == near) return 0;
    if (!(v > 0.0f)) return 1;
    return 2 + static_cast<int>((ordered_bits(v) - lo_bits) >> shift);
  };
#pragma unroll
  for (int j = 0; j < kSPer; ++j) {
    const int s = tid + j * 1024;
    if (s < S && r1[j] > r0[j]) {
      const int b = bucket(s, lb[j]);
      atomicAdd(&s_hist[b], 1);
      if (b != 0) atomicMin(&s_bmin[b], ordered_bits(lb[j]));
    }
  }
  __syncthreads();
  {
    // bucket offsets: exclusive prefix of the counts, kPlanBuckets / 1024 a thread
    constexpr int kPer = kPlanBuckets / 1024;
    int c[kPer], sum = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      c[j] = s_hist[kPer * tid + j];
      sum += c[j];
    }
    int total = 0;
    int off = block_exclusive_sum(sum, s_w, total);
    // The first bucket whose smallest bound the seed's k-th distance prunes
    // (the scan's test, whose bound is never looser): the carried bounds
    // never decrease, so it and every later bucket are never visited and
    // are left out.
    const bool can_prune = s_lut_bad == 0 && seed_kth != ~0u;
    const float cut = can_prune ? from_ordered_bits(seed_kth) : 0.0f;
    uint32_t stop = kPlanBuckets;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int b = kPer * tid + j;
      s_hist[b] = off;
      off += c[j];
      if (can_prune && c[j] > 0 && b >= 2) {
        const float blb = from_ordered_bits(s_bmin[b]);
        if (__fsub_rn(__fmul_rn(__fmul_rn(blb, blb), a.keep), a.abs_m) > cut) stop = min(stop, static_cast<uint32_t>(b));
      }
    }
    stop = wave_min_u32(stop);
    if ((tid & 63) == 0 && stop != static_cast<uint32_t>(kPlanBuckets)) atomicMin(&s_stop, static_cast<int>(stop));
  }
  __syncthreads();
  // Each item before the first pruned bucket gets its place; then its
  // fields go out field by field through LDS (s_cnt, free now), so that the
  // stores are coalesced: rows, carried bound, and the tile counts, which
  // stay in s_nt for the offsets.
  int32_t* s_nt = s_cnt;
  const int stop_b = min(s_stop, kPlanBuckets);
  const int n_items = stop_b < kPlanBuckets ? s_hist[stop_b] : s_count;
  const size_t base = static_cast<size_t>(q) * S;
  __syncthreads();   // s_hist[stop_b] read before the cursors move
  static_assert(kMaxItems <= (1 << kItemBits) && kPlanBuckets <= (1 << (31 - kItemBits)),
                "a place and a bucket in one non-negative word");
  int32_t place[kSPer];   // (bucket << kItemBits) | position, or -1
#pragma unroll
  for (int j = 0; j < kSPer; ++j) {
    const int s = tid + j * 1024;
    place[j] = -1;
    if (s < S && r1[j] > r0[j]) {
      const int b = bucket(s, lb[j]);
      if (b < stop_b) place[j] = (b << kItemBits) | atomicAdd(&s_hist[b], 1);
    }
  }
  int32_t* const outs[3] = {a.it_r0, a.it_r1, reinterpret_cast<int32_t*>(a.it_lb)};
#pragma unroll
  for (int field = 0; field < 4; ++field) {
    __syncthreads();   // the previous field is out (the ranks are read, for the first)
#pragma unroll
    for (int j = 0; j < kSPer; ++j) {
      if (place[j] < 0) continue;
      const int b = place[j] >> kItemBits;
      int32_t v;
      if (field == 0) v = r0[j];
      else if (field == 1) v = r1[j];
      else if (field == 2) v = __float_as_int(b == 0 ? __builtin_nanf("") : from_ordered_bits(s_bmin[b]));
      else v = ((r1[j] - 1) >> 6) - (r0[j] >> 6) + 1;
      s_cnt[place[j] & kItemMask] = v;
    }
    __syncthreads();
    if (field < 3)
      for (int i = tid; i < n_items; i += 1024) outs[field][base + i] = s_cnt[i];
  }
  {
    // tile offsets: exclusive prefix, a contiguous run of items a thread
    const int per = (n_items + 1023) / 1024;
    int sum = 0;
    for (int u = 0; u < per; ++u) {
      const int i = tid * per + u;
      if (i < n_items) sum += s_nt[i];
    }
    int total = 0;
    int off = block_exclusive_sum(sum, s_w, total);
    for (int u = 0; u < per; ++u) {
      const int i = tid * per + u;
      if (i < n_items) {
        const int nt = s_nt[i];
        s_nt[i] = off;
        off += nt;
      }
    }
    if (tid == 0) {
      hdr[0] = __int_as_float(n_items);
      hdr[1] = __int_as_float(total);
      hdr[2] = sw;
      hdr[3] = delta;
    }
  }
  __syncthreads();
  for (int i = tid; i < n_items; i += 1024) a.it_t[base + i] = s_nt[i];
}

// The plan of query blockIdx.x, its bound factors reduced from the parts
// first.  (Building the job table in the workgroup that finishes last, behind
// a device-wide counter, cost more than its own launch: every workgroup's
// release fence writes back its L2.)
template <int MT, typename LutT>
__global__ __launch_bounds__(1024) void list_plan_kernel(const ListPlanArgs a) {
  __shared__ float s_bounds[2];
  if (threadIdx.x == 0) {
    float sw, delta;
    reduce_bound_parts(a.parts + static_cast<size_t>(blockIdx.x) * 2 * a.m, a.m, a.grow, sw, delta);
    s_bounds[0] = sw;
    s_bounds[1] = delta;
  }
  __syncthreads();
  plan_one_query<MT, LutT>(a, s_bounds[0], s_bounds[1]);
}

__global__ __launch_bounds__(1024) void list_jobs_kernel(const ListJobArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  build_job_table(a, smem);
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

float bound_grow(int m, int dsub) { return 1.0f + 2.0f * static_cast<float>(dsub + m + 8) * 0x1p-24f + 0x1p-20f; }

hipError_t launch_bound_parts(const float* alpha, const float* wf, const float* cpq, const float* W, int nq, int m,
                              int r, int dsub, float* parts, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const dim3 g(static_cast<unsigned>(m), static_cast<unsigned>((nq + kBoundQueries - 1) / kBoundQueries));
  if (dsub == 2 && r == 8)
    bound_parts_kernel<2, 8><<<g, 256, 0, s>>>(alpha, wf, cpq, W, m, dsub, r, nq, parts);
  else if (dsub == 8 && r == 8)
    bound_parts_kernel<8, 8><<<g, 256, 0, s>>>(alpha, wf, cpq, W, m, dsub, r, nq, parts);
  else
    bound_parts_kernel<0, 0><<<g, 256, 0, s>>>(alpha, wf, cpq, W, m, dsub, r, nq, parts);
  return hipGetLastError();
}

hipError_t launch_lut_bounds(const float* alpha, const float* wf, const float* cpq, const float* W, int nq, int m,
                             int r, int dsub, float* parts, float* bounds, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const hipError_t e = launch_bound_parts(alpha, wf, cpq, W, nq, m, r, dsub, parts, s);
  if (e != hipSuccess) return e;
  bound_final_kernel<<<static_cast<unsigned>((nq + 255) / 256), 256, 0, s>>>(parts, m, nq, bound_grow(m, dsub),
                                                                             bounds);
  return hipGetLastError();
}

size_t list_plan_lds_bytes(int m, int lut_dtype, int C) {
  const size_t lut = static_cast<size_t>(m) * kKsub * (lut_dtype == 1 ? 2 : 4);
  const size_t items = static_cast<size_t>(C) * kBands * 4 + static_cast<size_t>(kPlanBuckets) * 8;
  return ((static_cast<size_t>(2 * C + 1) * 4 + 15) & ~size_t{15}) + std::max(lut, items);
}

size_t list_jobs_lds_bytes(int nq) {
  size_t np2 = 1;
  while (np2 < static_cast<size_t>(nq)) np2 *= 2;
  return np2 * 8 + 1025 * 4;
}

hipError_t launch_list_plan(const ListPlanArgs& a, int lut_dtype, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  const bool h = lut_dtype == 1;
  const void* fn = nullptr;
  switch (a.m) {
    case 16: fn = h ? reinterpret_cast<const void*>(&list_plan_kernel<16, __half>)
                    : reinterpret_cast<const void*>(&list_plan_kernel<16, float>); break;
    case 48: fn = h ? reinterpret_cast<const void*>(&list_plan_kernel<48, __half>)
                    : reinterpret_cast<const void*>(&list_plan_kernel<48, float>); break;
    case 120: fn = h ? reinterpret_cast<const void*>(&list_plan_kernel<120, __half>)
                     : reinterpret_cast<const void*>(&list_plan_kernel<120, float>); break;
    default: return hipErrorInvalidValue;
  }
  const size_t lds = list_plan_lds_bytes(a.m, lut_dtype, a.C);
  if (a.n_sub != a.C * kBands || a.n_sub > kMaxItems) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  ListPlanArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchKernel(fn, dim3(static_cast<unsigned>(a.nq)), dim3(1024), kargs, lds, s);
}

hipError_t launch_list_jobs(const ListJobArgs& a, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  const size_t lds = list_jobs_lds_bytes(a.nq);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&list_jobs_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  ListJobArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchKernel(reinterpret_cast<const void*>(&list_jobs_kernel), dim3(1), dim3(1024), kargs, lds, s);
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
