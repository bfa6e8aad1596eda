// Exact filtered kNN over the full-precision vectors: the exact top-k over
// the predicate-passing rows that Section 3.1 takes as ground truth, and the
// pre-filtering baseline (i) of Section 3.2.  A row's distance is
//   d = sum_{j<D} (x_j - q_j)^2,
// summed in j order from +0 in fp32 with the difference, its square and each
// addition rounded separately; rows rank by (d, original id).
//
// Two plans, chosen per batch by the host:
//  * direct: every selected row of a query is scored exactly
//    (exact_rerank_kernel over the query's row interval, its selection
//    bitmap masking residual clauses);
//  * screened, for batches whose queries share rows (wide intervals, or an
//    unclustered index where every query spans all rows): a bf16 matrix-core
//    pass computes dd = |x|^2 + |q|^2 - 2 x.q for 32 queries x 32 rows per
//    tile.  eps(q) bounds |dd - d| for every row (bf16 rounding of x and q,
//    fp32 accumulation, and the fp32 rounding of d itself).  Pass 1 keeps,
//    per (query, wavefront, chunk, group of R lanes), the smallest dd of the
//    rows it saw (R is chosen so that a query's interval spans several times
//    k such bins); these come from distinct rows, so the k-th smallest of
//    them, v_k, has k rows with d <= v_k + eps, and every row of the exact
//    top k has dd <= v_k + 2 eps.  Pass 2 lists the rows under that bound, and only
//    those are scored exactly.  Both plans end in the same exact scoring and
//    merge, so results are identical.
#include <hip/hip_runtime.h>
#include <cfloat>
#include <climits>
#include <cmath>

#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr int kExWaves = 8;        // wavefronts per screening workgroup
constexpr int kExKC = 8;           // K steps (16 dims each) loaded per round

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Eight consecutive values of a row (zero past `dim`) as one MFMA fragment.
__device__ __forceinline__ uint4 pack_fragment(const float* __restrict__ row, int dim, int k0) {
  uint32_t w[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const int k = k0 + 2 * h;
    const uint32_t lo = k < dim ? bf16_bits(row[k]) : 0u;
    const uint32_t hi = k + 1 < dim ? bf16_bits(row[k + 1]) : 0u;
    w[h] = lo | (hi << 16);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// ---------------------------------------------------------------- staging
// One thread per physical row: the fp32 copies (64-row tiles,
// xt[(r / 64 * dim + j) * 64 + r % 64], for scans of consecutive rows, and
// row-major, xr[r * dim + j], for scattered rows), |x|^2 (fp32, summed in j
// order) and the
// bf16 fragments of its 32-row tile (xb[(tile32 * ks + s) * 64 + lane]: lane
// l holds row l % 32, dims s * 16 + (l / 32) * 8 .. + 8).  Also the largest
// norm (as fp32 bits; norms are non-negative) and a count of non-finite
// values.
__global__ __launch_bounds__(256) void exact_stage_kernel(const float* __restrict__ x, int64_t n, int dim,
                                                          int ks, const int32_t* __restrict__ perm,
                                                          float* __restrict__ xt, float* __restrict__ xr,
                                                          uint4* __restrict__ xb,
                                                          float* __restrict__ xn, unsigned* __restrict__ max_norm_bits,
                                                          unsigned long long* __restrict__ bad) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t n32 = (n + 31) / 32 * 32;
  if (r >= n32) return;
  const bool real = r < n;
  const float* src = real ? x + static_cast<size_t>(perm ? perm[r] : r) * dim : nullptr;
  float acc = 0.0f;
  unsigned nonfinite = 0;
  if (real) {
    for (int j = 0; j < dim; ++j) {
      const float v = src[j];
      xt[(static_cast<size_t>(r >> 6) * dim + j) * 64 + (r & 63)] = v;
      xr[static_cast<size_t>(r) * dim + j] = v;
      acc = __fadd_rn(acc, __fmul_rn(v, v));
      nonfinite += isfinite(v) ? 0u : 1u;
    }
  }
  xn[r] = acc;
  const int64_t t32 = r >> 5;
  const int lane_lo = static_cast<int>(r & 31);
  for (int s = 0; s < ks; ++s)
    for (int h = 0; h < 2; ++h) {
      const uint4 f = real ? pack_fragment(src, dim, s * 16 + h * 8) : make_uint4(0, 0, 0, 0);
      xb[(static_cast<size_t>(t32) * ks + s) * 64 + h * 32 + lane_lo] = f;
    }
  if (real) {
    atomicMax(max_norm_bits, __float_as_uint(sqrtf(acc)));
    if (nonfinite) atomicAdd(bad, static_cast<unsigned long long>(nonfinite));
  }
}

// ------------------------------------------------------------ query prep
// One wavefront per query position p (original query qorder[p]): its bf16
// fragments in 32-query tiles, |q|^2, and eps(p) (see the header), computed
// in fp64 from the largest row norm X and |q| and rounded up.  Also clears
// the position's candidate count.
__global__ __launch_bounds__(64) void exact_query_kernel(const float* __restrict__ q, int dim, int ks, int nq,
                                                         const int32_t* __restrict__ qorder,
                                                         const unsigned* __restrict__ max_norm_bits,
                                                         uint4* __restrict__ qb, float* __restrict__ qn,
                                                         float* __restrict__ eps, int32_t* __restrict__ cand_n) {
  const int p = blockIdx.x;
  const int lane = threadIdx.x;
  const int t = p / 32, lane_lo = p % 32;
  const bool real = p < nq;
  const float* row = real ? q + static_cast<size_t>(qorder[p]) * dim : nullptr;
  for (int s = lane; s < 2 * ks; s += 64) {
    const int step = s >> 1, h = s & 1;
    const uint4 f = real ? pack_fragment(row, dim, step * 16 + h * 8) : make_uint4(0, 0, 0, 0);
    qb[(static_cast<size_t>(t) * ks + step) * 64 + h * 32 + lane_lo] = f;
  }
  if (!real) return;
  double s2 = 0.0;
  float acc = 0.0f;
  if (lane == 0) {
    for (int j = 0; j < dim; ++j) {
      acc = __fadd_rn(acc, __fmul_rn(row[j], row[j]));
      s2 += static_cast<double>(row[j]) * row[j];
    }
    const double qnorm = sqrt(s2);
    const double X = static_cast<double>(__uint_as_float(*max_norm_bits));
    const double u_b = 0x1p-8;                        // bf16 rounding, relative
    const double g = (4.0 * dim + 16.0) * 0x1p-23;    // fp32 sums of dim terms, generously
    const double e = 2.0 * ((4.1 * u_b + g) * X * qnorm + g * (X + qnorm) * (X + qnorm)) + 1e-30;
    qn[p] = acc;
    eps[p] = static_cast<float>(e * (1.0 + 0x1p-20));
    cand_n[p] = 0;
  }
}

// --------------------------------------------------------------- screening
struct ScreenArgs {
  const uint4* xb;            // row fragments
  const float* xn;            // [n32] |x|^2
  const uint4* qb;            // query fragments
  const float* qn;            // [positions] |q|^2
  const float* thr;           // [positions] pass 2: keep rows with dd <= thr
  const int32_t* qorder;
  const int64_t* iv;          // [nq original][2]
  const DevPred* preds;       // residual_mask per original query
  const uint64_t* bitmap;     // [nq original][stride64] physical order
  int64_t stride64;
  int nq, ks;
  int64_t chunk_rows;         // rows per workgroup chunk (multiple of 32 * kExWaves)
  int splits;                 // chunks per query tile
  int bin_lanes;              // R: lanes whose minima share one bin (1, 2, ..., 32)
  float* bins;                // pass 1: [positions][splits * kExWaves * 32 / R]
  int32_t* cand;              // pass 2: [positions][cand_cap]
  int32_t* cand_n;
  int64_t cand_cap;
};

struct QueryInfo {
  int64_t iv0, iv1;
  float qn, thr;
  int32_t orig, resid;
};

// grid.x = splits * query tiles.  Each workgroup scores the rows of one
// chunk of its 32-query tile's hull (the smallest row range holding all 32
// intervals); wavefront w takes the chunk's 32-row tiles w, w + 8, ...
template <int PASS, int KS>
__global__ __launch_bounds__(kExWaves * 64) void exact_screen_kernel(const ScreenArgs a) {
  __shared__ QueryInfo s_q[32];
  __shared__ int64_t s_hull[2];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int qt = blockIdx.x / a.splits, chunk = blockIdx.x % a.splits;
  const int ks = KS > 0 ? KS : a.ks;
  if (threadIdx.x < 32) {
    const int p = qt * 32 + threadIdx.x;
    QueryInfo qi{0, 0, 0.0f, -1.0f, -1, 0};
    if (p < a.nq) {
      const int o = a.qorder[p];
      qi.iv0 = a.iv[2 * o];
      qi.iv1 = a.iv[2 * o + 1];
      qi.qn = a.qn[p];
      qi.thr = PASS == 2 ? a.thr[p] : 0.0f;
      qi.orig = o;
      qi.resid = a.preds[o].residual_mask != 0;
      if (qi.iv1 <= qi.iv0) qi.iv0 = qi.iv1 = 0;
    }
    s_q[threadIdx.x] = qi;
    // hull of the tile's non-empty intervals
    int64_t lo = qi.iv1 > qi.iv0 ? qi.iv0 : INT64_MAX, hi = qi.iv1 > qi.iv0 ? qi.iv1 : 0;
    bool res = qi.resid != 0;
#pragma unroll
    for (int o = 16; o > 0; o >>= 1) {
      lo = min(lo, static_cast<int64_t>(__shfl_xor(lo, o, 32)));
      hi = max(hi, static_cast<int64_t>(__shfl_xor(hi, o, 32)));
      const int other = __shfl_xor(static_cast<int>(res), o, 32);   // every lane shuffles
      res = res || other != 0;
    }
    if (threadIdx.x == 0) {
      s_hull[0] = lo;
      s_hull[1] = hi;
    }
    if (threadIdx.x == 0) s_q[0].resid |= res ? 2 : 0;   // bit 1: some query of the tile has residual clauses
  }
  __syncthreads();
  const bool any_resid = (s_q[0].resid & 2) != 0;
  const int64_t hull_lo = s_hull[0], hull_hi = s_hull[1];
  int64_t r_begin = hull_lo + static_cast<int64_t>(chunk) * a.chunk_rows;
  int64_t r_end = min(hull_hi, r_begin + a.chunk_rows);
  if (hull_hi <= hull_lo) r_begin = r_end = 0;
  // 32-row tiles of the chunk (rows outside [r_begin, r_end) are masked)
  const int64_t t_begin = r_begin >> 5, t_end = (r_end + 31) >> 5;

  // This lane's 16 output cells: query m(i) = 8 (i / 4) + 4 (lane / 32) + i % 4,
  // row lane % 32 of the tile.
  const int half = lane >> 5;
  float run_min[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) run_min[i] = __builtin_inff();
  const uint4* a_frag = a.qb + static_cast<size_t>(qt) * ks * 64;

  for (int64_t t = t_begin + wave; t < t_end; t += kExWaves) {
    f32x16 acc = {};
    const uint4* b_frag = a.xb + static_cast<size_t>(t) * ks * 64;
    for (int s0 = 0; s0 < ks; s0 += kExKC) {
      uint4 bv[kExKC], av[kExKC];
#pragma unroll
      for (int u = 0; u < kExKC; ++u)
        if (KS > 0 ? (s0 + u < KS) : (s0 + u < ks)) {
          bv[u] = b_frag[(s0 + u) * 64 + lane];
          av[u] = a_frag[(s0 + u) * 64 + lane];
        }
#pragma unroll
      for (int u = 0; u < kExKC; ++u)
        if (KS > 0 ? (s0 + u < KS) : (s0 + u < ks))
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(&av[u]),
                                                          *reinterpret_cast<const bf16x8*>(&bv[u]), acc, 0, 0, 0);
    }
    const int64_t row = t * 32 + (lane & 31);
    const bool in_chunk = row >= r_begin && row < r_end;
    const float xr = a.xn[row];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int m = 8 * (i >> 2) + 4 * half + (i & 3);
      const QueryInfo& qi = s_q[m];
      bool sel = in_chunk && row >= qi.iv0 && row < qi.iv1;
      if (any_resid && sel && (qi.resid & 1))
        sel = (a.bitmap[static_cast<size_t>(qi.orig) * a.stride64 + (row >> 6)] >> (row & 63)) & 1ull;
      const float dd = __fsub_rn(__fadd_rn(xr, qi.qn), __fmul_rn(2.0f, acc[i]));
      if (PASS == 1) {
        if (sel) run_min[i] = fminf(run_min[i], dd);
      } else if (sel && dd <= qi.thr) {
        const int p = qt * 32 + m;
        const int pos = atomicAdd(&a.cand_n[p], 1);
        if (pos < a.cand_cap) a.cand[static_cast<size_t>(p) * a.cand_cap + pos] = static_cast<int32_t>(row);
      }
    }
  }
  if (PASS == 1) {
    // One value per (query, wavefront, chunk, group of R lanes): the smallest
    // over the R lanes' rows.
    const int R = a.bin_lanes, per = 32 / R;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float v = run_min[i];
      for (int o = 1; o < R; o <<= 1) v = fminf(v, __shfl_xor(v, o, 32));
      run_min[i] = v;
    }
    if ((lane & (R - 1)) == 0) {
      const size_t n_bins = static_cast<size_t>(a.splits) * kExWaves * per;
      const size_t slot = static_cast<size_t>(chunk * kExWaves + wave) * per + (lane & 31) / R;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int p = qt * 32 + 8 * (i >> 2) + 4 * half + (i & 3);
        if (p < a.nq) a.bins[static_cast<size_t>(p) * n_bins + slot] = run_min[i];
      }
    }
  }
}

// ---------------------------------------------------------------- threshold
// One wavefront per query position: v_k = k-th smallest bin value, and the
// candidate bound thr = v_k + 2 eps (+inf while fewer than k bins hold a
// row).
__global__ __launch_bounds__(64) void exact_threshold_kernel(const float* __restrict__ bins, int64_t n_bins, int k,
                                                             int kpl, const float* __restrict__ eps,
                                                             float* __restrict__ thr) {
  extern __shared__ uint64_t pool[];
  const int p = blockIdx.x;
  const int lane = threadIdx.x;
  const float* src = bins + static_cast<size_t>(p) * n_bins;
  int cnt = 0;
  uint64_t kth = kNoKey;
  for (int64_t b = 0; b < n_bins; b += 64) {
    const int64_t i = b + lane;
    const float v = i < n_bins ? src[i] : __builtin_inff();
    const bool ok = v < __builtin_inff();
    const uint64_t key = (static_cast<uint64_t>(ordered_bits(v)) << 32) | static_cast<uint32_t>(i);
    pool_push(pool, cnt, kth, key, ok && key < kth, k, kpl);
  }
  pool_compact(pool, cnt, kth, k, kpl);
  if (lane == 0) {
    float t = __builtin_inff();
    if (kth != kNoKey) {
      const double bound = static_cast<double>(from_ordered_bits(static_cast<uint32_t>(kth >> 32))) +
                           2.0 * static_cast<double>(eps[p]);
      t = static_cast<float>(bound * (1.0 + 0x1p-20) + 1e-30);
    }
    thr[p] = t;
  }
}

// ------------------------------------------------------------------ rerank
constexpr int kStageDims = 64;     // dimensions of 64 rows staged in LDS per step

struct RerankArgs {
  const float* xt;            // fp32 rows in 64-row tiles, physical order
  const float* xr;            // fp32 rows, row-major, physical order
  int dim;
  const float* q;             // [nq original][dim]
  const int32_t* qorder;
  const int64_t* iv;
  const DevPred* preds;
  const uint64_t* bitmap;
  int64_t stride64;
  const int32_t* perm;
  const int32_t* cand;        // screened: [positions][cand_cap]
  const int32_t* cand_n;      // null: direct plan
  int64_t cand_cap;
  int k, kpl, chunks;
  uint64_t* partials;         // [positions][chunks][k]
};

// grid = (chunks, positions), one wavefront each: chunk c of the query's
// work -- its candidate list (LISTED: screened plan, list not overflowed) or
// its row interval (direct plan, or a list that overflowed) -- scored
// exactly, the k best keys written to partials.
//  * Consecutive rows (an interval): each lane reads its own row from the
//    64-row tiles, one coalesced 256-byte load per dimension for the wave.
//  * Scattered rows (a candidate list): the 64 lanes' rows are staged in
//    LDS 64 dimensions at a time from the row-major copy, one coalesced
//    256-byte load per row, then each lane reads its own row.
// Either way each lane adds its row's terms in j order.
template <bool LISTED>
__global__ __launch_bounds__(64) void exact_rerank_kernel(const RerankArgs a) {
  extern __shared__ uint64_t smem_r[];
  uint64_t* pool = smem_r;
  const int dim_pad = (a.dim + kStageDims - 1) / kStageDims * kStageDims;
  float* s_q = reinterpret_cast<float*>(smem_r + 64 * a.kpl);
  float* s_x = s_q + dim_pad;                     // LISTED: [64 rows][kStageDims + 1]
  const int c = blockIdx.x, p = blockIdx.y;
  const int lane = threadIdx.x;
  const int o = a.qorder[p];
  for (int j = lane; j < dim_pad; j += 64) s_q[j] = j < a.dim ? a.q[static_cast<size_t>(o) * a.dim + j] : 0.0f;
  __syncthreads();
  const int64_t iv0 = a.iv[2 * o], iv1 = a.iv[2 * o + 1];
  const bool resid = a.preds[o].residual_mask != 0;
  const bool listed = LISTED && a.cand_n[p] <= a.cand_cap;
  int cnt = 0;
  uint64_t thr = kNoKey;
  auto offer = [&](int64_t row, bool ok, float d) {
    uint64_t key = kNoKey;
    if (ok) {
      const uint32_t id = a.perm ? static_cast<uint32_t>(a.perm[row]) : static_cast<uint32_t>(row);
      key = (static_cast<uint64_t>(ordered_bits(d)) << 32) | id;
    }
    pool_push(pool, cnt, thr, key, ok && key < thr, a.k, a.kpl);
  };
  if (listed) {
    const int64_t n_items = a.cand_n[p];
    const int64_t per = (n_items + a.chunks - 1) / a.chunks;
    const int64_t i0 = static_cast<int64_t>(c) * per, i1 = min(n_items, i0 + per);
    const int32_t* list = a.cand + static_cast<size_t>(p) * a.cand_cap;
    for (int64_t b = i0; b < i1; b += 64) {
      const int64_t i = b + lane;
      const bool ok = i < i1;
      const int32_t row = ok ? list[i] : 0;
      const uint64_t okm = __ballot(ok);
      float d = 0.0f;
      for (int j0 = 0; j0 < a.dim; j0 += kStageDims) {
        const int nj = min(kStageDims, a.dim - j0);
#pragma unroll
        for (int r0 = 0; r0 < 64; r0 += 16) {
          float v[16];
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const int ri = __builtin_amdgcn_readlane(row, r0 + u);
            const bool live = ((okm >> (r0 + u)) & 1) && lane < nj;
            v[u] = live ? a.xr[static_cast<size_t>(ri) * a.dim + j0 + lane] : 0.0f;
          }
#pragma unroll
          for (int u = 0; u < 16; ++u) s_x[(r0 + u) * (kStageDims + 1) + lane] = v[u];
        }
        wave_lds_fence();
        if (ok) {
          const float* xrow = s_x + lane * (kStageDims + 1);
          for (int j = 0; j < nj; ++j) {
            const float e = __fsub_rn(xrow[j], s_q[j0 + j]);
            d = __fadd_rn(d, __fmul_rn(e, e));
          }
        }
        wave_lds_fence();
      }
      offer(row, ok, d);
    }
  } else if (iv1 > iv0) {
    // 64-row tiles of the interval, dealt out in contiguous runs
    const int64_t t0 = iv0 >> 6, t1 = (iv1 + 63) >> 6;
    const int64_t per = (t1 - t0 + a.chunks - 1) / a.chunks;
    const int64_t ta = t0 + static_cast<int64_t>(c) * per, tb = min(t1, ta + per);
    for (int64_t t = ta; t < tb; ++t) {
      const int64_t row = t * 64 + lane;
      bool ok = row >= iv0 && row < iv1;
      if (ok && resid) ok = (a.bitmap[static_cast<size_t>(o) * a.stride64 + t] >> lane) & 1ull;
      float d = 0.0f;
      if (ok) {
        const float* xr = a.xt + static_cast<size_t>(t) * a.dim * 64 + lane;
        // 16 values in flight, then added in j order
        int j = 0;
        for (; j + 16 <= a.dim; j += 16) {
          float v[16];
#pragma unroll
          for (int u = 0; u < 16; ++u) v[u] = xr[static_cast<size_t>(j + u) * 64];
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const float e = __fsub_rn(v[u], s_q[j + u]);
            d = __fadd_rn(d, __fmul_rn(e, e));
          }
        }
        for (; j < a.dim; ++j) {
          const float e = __fsub_rn(xr[static_cast<size_t>(j) * 64], s_q[j]);
          d = __fadd_rn(d, __fmul_rn(e, e));
        }
      }
      offer(row, ok, d);
    }
  }
  pool_compact(pool, cnt, thr, a.k, a.kpl);
  uint64_t* dst = a.partials + (static_cast<size_t>(p) * a.chunks + c) * a.k;
  for (int e = lane; e < a.k; e += 64) dst[e] = pool[e];
}

template <int KS>
const void* screen_symbol(int pass) {
  return pass == 1 ? reinterpret_cast<const void*>(&exact_screen_kernel<1, KS>)
                   : reinterpret_cast<const void*>(&exact_screen_kernel<2, KS>);
}

// Reconstruction from the codes (the reconstruct-then-exact baseline (ii) of
// Section 3.2): physical row r, dimension m * dsub + j, is codeword
// C_PQ[m][code_r[m]][j]; one thread per (row, subspace).
__global__ __launch_bounds__(256) void decode_kernel(const uint32_t* __restrict__ codes_t, int64_t n, int M, int mw,
                                                     int dsub, const float* __restrict__ cpq, float* __restrict__ x) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n * M) return;
  const int64_t r = i / M;
  const int m = static_cast<int>(i % M);
  const uint32_t word = codes_t[((r >> 6) * mw + (m >> 2)) * 64 + (r & 63)];
  const int code = static_cast<int>((word >> (8 * (m & 3))) & 0xFFu);
  const float* c = cpq + (static_cast<size_t>(m) * kKsub + code) * dsub;
  float* dst = x + static_cast<size_t>(r) * M * dsub + static_cast<size_t>(m) * dsub;
  for (int j = 0; j < dsub; ++j) dst[j] = c[j];
}

}  // namespace

hipError_t launch_decode(const uint32_t* codes_t, int64_t n, int m, int mw, int dsub, const float* cpq, float* x,
                         hipStream_t s) {
  const int64_t total = n * m;
  decode_kernel<<<static_cast<unsigned>((total + 255) / 256), 256, 0, s>>>(codes_t, n, m, mw, dsub, cpq, x);
  return hipGetLastError();
}

int exact_ksteps(int dim) { return (dim + 15) / 16; }

hipError_t launch_exact_stage(const float* x, int64_t n, int dim, const int32_t* perm, float* xt, float* xr,
                              uint4* xb, float* xn, unsigned* max_norm_bits, unsigned long long* bad, hipStream_t s) {
  const int64_t n32 = (n + 31) / 32 * 32;
  const unsigned blocks = static_cast<unsigned>((n32 + 255) / 256);
  exact_stage_kernel<<<blocks, 256, 0, s>>>(x, n, dim, exact_ksteps(dim), perm, xt, xr, xb, xn, max_norm_bits,
                                            bad);
  return hipGetLastError();
}

hipError_t launch_exact_queries(const float* q, int dim, int nq, const int32_t* qorder, const unsigned* max_norm_bits,
                                uint4* qb, float* qn, float* eps, int32_t* cand_n, hipStream_t s) {
  const int padded = (nq + 31) / 32 * 32;
  exact_query_kernel<<<padded, 64, 0, s>>>(q, dim, exact_ksteps(dim), nq, qorder, max_norm_bits, qb, qn, eps,
                                          cand_n);
  return hipGetLastError();
}

hipError_t launch_exact_screen(const ExactScreen& e, int pass, hipStream_t s) {
  ScreenArgs a{};
  a.xb = e.xb;
  a.xn = e.xn;
  a.qb = e.qb;
  a.qn = e.qn;
  a.thr = e.thr;
  a.qorder = e.qorder;
  a.iv = e.iv;
  a.preds = e.preds;
  a.bitmap = e.bitmap;
  a.stride64 = e.stride64;
  a.nq = e.nq;
  a.ks = exact_ksteps(e.dim);
  a.chunk_rows = e.chunk_rows;
  a.splits = e.splits;
  a.bin_lanes = e.bin_lanes;
  a.bins = e.bins;
  a.cand = e.cand;
  a.cand_n = e.cand_n;
  a.cand_cap = e.cand_cap;
  const void* fn = nullptr;
  switch (a.ks) {
    case 6: fn = screen_symbol<6>(pass); break;      // 96 dims
    case 8: fn = screen_symbol<8>(pass); break;      // 128 dims
    default: fn = screen_symbol<0>(pass); break;
  }
  const int n_qtiles = (e.nq + 31) / 32;
  void* args[] = {&a};
  return hipLaunchKernel(fn, dim3(static_cast<unsigned>(n_qtiles * e.splits)), dim3(kExWaves * 64), args, 0, s);
}

hipError_t launch_exact_threshold(const float* bins, int64_t n_bins, int nq, int k, const float* eps, float* thr,
                                  hipStream_t s) {
  const int kpl = pool_kpl(k);
  exact_threshold_kernel<<<nq, 64, static_cast<size_t>(64 * kpl) * sizeof(uint64_t), s>>>(bins, n_bins, k, kpl, eps,
                                                                                         thr);
  return hipGetLastError();
}

int64_t exact_bins_per_query(int splits, int bin_lanes) {
  return static_cast<int64_t>(splits) * kExWaves * (32 / bin_lanes);
}
int64_t exact_chunk_quantum() { return 32 * kExWaves; }

hipError_t launch_exact_rerank(const ExactRerank& e, hipStream_t s) {
  RerankArgs a{};
  a.xt = e.xt;
  a.xr = e.xr;
  a.dim = e.dim;
  a.q = e.q;
  a.qorder = e.qorder;
  a.iv = e.iv;
  a.preds = e.preds;
  a.bitmap = e.bitmap;
  a.stride64 = e.stride64;
  a.perm = e.perm;
  a.cand = e.cand;
  a.cand_n = e.cand_n;
  a.cand_cap = e.cand_cap;
  a.k = e.k;
  a.kpl = pool_kpl(e.k);
  a.chunks = e.chunks;
  a.partials = e.partials;
  const bool listed = e.cand_n != nullptr;
  const int dim_pad = (e.dim + kStageDims - 1) / kStageDims * kStageDims;
  const size_t lds = static_cast<size_t>(64 * a.kpl) * sizeof(uint64_t) +
                     (static_cast<size_t>(dim_pad) + (listed ? 64 * (kStageDims + 1) : 0)) * sizeof(float);
  if (lds > static_cast<size_t>(kLdsBudget)) return hipErrorInvalidValue;
  const void* fn = listed ? reinterpret_cast<const void*>(&exact_rerank_kernel<true>)
                          : reinterpret_cast<const void*>(&exact_rerank_kernel<false>);
  hipError_t err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (err != hipSuccess) return err;
  void* args[] = {&a};
  return hipLaunchKernel(fn, dim3(static_cast<unsigned>(e.chunks), static_cast<unsigned>(e.nq)), dim3(64), args, lds, s);
}

}  // namespace ifvs
