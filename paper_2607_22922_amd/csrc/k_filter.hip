// Filter stage (Section 2, stage 1): evaluate each query's conjunctive
// predicate over the attribute columns and emit the candidate pool P as a
// selection bitmap, plus the pool size.
//
// One wavefront covers 4096 consecutive vectors: in step `it` (0..63) lane L
// loads the attributes of vector base + 64*it + L once and tests them against
// the predicates of all kFilterQueries queries of its workgroup; the compare
// result of the wavefront is itself the 64-bit ballot word of those 64
// vectors, which lane `it` keeps (one word per query).  After 64 steps every
// lane holds one word per query and the wavefront stores 512 contiguous bytes
// per query.  Clause lists live in LDS; each attribute value is read once per
// group of kFilterQueries queries.
#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr int kFilterWaves = 4;
constexpr int kRowsPerWave = 64 * 64;

// A predicate's clause list for one pass, as the kernel reads it from LDS.
struct PassClauses {
  int32_t nc;                 // clauses to test; -1: nothing passes
  int32_t col[kMaxClauses];
  uint32_t lo[kMaxClauses];
  uint32_t width[kMaxClauses];
};

__device__ __forceinline__ int32_t column_value(const int32_t* __restrict__ attrs, int64_t n, int col,
                                                int64_t i, int32_t a0, int32_t a1) {
  return col == 0 ? a0 : (col == 1 ? a1 : attrs[static_cast<int64_t>(col) * n + i]);
}

__global__ __launch_bounds__(kFilterWaves * 64) void filter_kernel(
    const int32_t* __restrict__ attrs, int64_t n, int n_attr,
    const DevPred* __restrict__ preds, int nq, int residual_only, uint64_t* __restrict__ bitmap,
    int64_t stride64, unsigned long long* __restrict__ counts) {
  __shared__ PassClauses sc[kFilterQueries];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int q0 = blockIdx.y * kFilterQueries;
  const int qn = min(kFilterQueries, nq - q0);
  // The clause list of each query of the group for this pass: all effective
  // clauses, or only the residual ones.
  if (threadIdx.x < qn) {
    const DevPred& p = preds[q0 + threadIdx.x];
    PassClauses c{};
    if (p.n_eff < 0) {
      c.nc = -1;
    } else {
      c.nc = residual_only ? p.n_res : p.n_eff;
      for (int j = 0; j < c.nc; ++j) {
        c.col[j] = residual_only ? p.res_col[j] : p.col[j];
        c.lo[j] = static_cast<uint32_t>(residual_only ? p.res_lo[j] : p.lo[j]);
        c.width[j] = residual_only ? p.res_width[j] : p.width[j];
      }
    }
    sc[threadIdx.x] = c;
  }
  __syncthreads();
  const int64_t base = (static_cast<int64_t>(blockIdx.x) * kFilterWaves + wave) * kRowsPerWave;
  if (base >= n) return;
  // Common case: every query of the group tests one clause on the same
  // column.  Then each step is one load and, per query, a subtract, a
  // compare whose lane mask is the ballot word, and two selects.
  int single_col = qn > 0 && sc[0].nc == 1 ? sc[0].col[0] : -1;
  for (int qi = 1; qi < qn; ++qi)
    if (sc[qi].nc != 1 || sc[qi].col[0] != single_col) single_col = -1;

  // held_{lo,hi}[qi] of lane L: the ballot word of step L for query qi.
  uint32_t held_lo[kFilterQueries], held_hi[kFilterQueries];
#pragma unroll
  for (int qi = 0; qi < kFilterQueries; ++qi) held_lo[qi] = held_hi[qi] = 0;

  if (single_col >= 0) {
    const int32_t* __restrict__ col = attrs + static_cast<int64_t>(single_col) * n;
    uint32_t lo[kFilterQueries], width[kFilterQueries];
#pragma unroll
    for (int qi = 0; qi < kFilterQueries; ++qi) {
      lo[qi] = qi < qn ? sc[qi].lo[0] : 0;
      width[qi] = qi < qn ? sc[qi].width[0] : 0;   // width 0: nothing passes
    }
#pragma unroll 4
    for (int it = 0; it < 64; ++it) {
      const int64_t i = base + static_cast<int64_t>(it) * 64 + lane;
      const bool in = i < n;
      const uint32_t v = static_cast<uint32_t>(col[in ? i : n - 1]);
      const bool mine = lane == it;
#pragma unroll
      for (int qi = 0; qi < kFilterQueries; ++qi) {
        const uint64_t word = __ballot(in && v - lo[qi] < width[qi]);
        held_lo[qi] = mine ? static_cast<uint32_t>(word) : held_lo[qi];
        held_hi[qi] = mine ? static_cast<uint32_t>(word >> 32) : held_hi[qi];
      }
    }
  } else {
  for (int it = 0; it < 64; ++it) {
    const int64_t i = base + static_cast<int64_t>(it) * 64 + lane;
    const bool in = i < n;
    const int64_t ii = in ? i : n - 1;
    const int32_t a0 = n_attr > 0 ? attrs[ii] : 0;
    const int32_t a1 = n_attr > 1 ? attrs[n + ii] : 0;
    const bool mine = lane == it;
#pragma unroll
    for (int qi = 0; qi < kFilterQueries; ++qi) {
      if (qi < qn) {
        const int nc = sc[qi].nc;
        bool pass = in && nc >= 0;
        for (int c = 0; c < nc; ++c) {
          const int32_t v = column_value(attrs, n, sc[qi].col[c], ii, a0, a1);
          pass &= static_cast<uint32_t>(v) - sc[qi].lo[c] < sc[qi].width[c];
        }
        const uint64_t word = __ballot(pass);
        held_lo[qi] = mine ? static_cast<uint32_t>(word) : held_lo[qi];
        held_hi[qi] = mine ? static_cast<uint32_t>(word >> 32) : held_hi[qi];
      }
    }
  }
  }

  const int64_t w64 = base / 64 + lane;           // this lane's 64-bit word
#pragma unroll
  for (int qi = 0; qi < kFilterQueries; ++qi) {
    if (qi < qn) {
      const uint64_t word = (static_cast<uint64_t>(held_hi[qi]) << 32) | held_lo[qi];
      if (w64 < stride64) bitmap[static_cast<int64_t>(q0 + qi) * stride64 + w64] = word;
      if (counts) {
        unsigned long long c = __popcll(word);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) c += __shfl_down(c, off, 64);
        if (lane == 0) atomicAdd(&counts[q0 + qi], c);
      }
    }
  }
}

// codes [n][m] bytes -> tiles of 64 rows: word j of physical row (64t + L) is
// stored at codes_t[(t*mw + j)*64 + L] and holds bytes 4j..4j+3 of original
// row perm[64t + L] (zero past m and past n), so a wavefront reading word j of
// a tile reads 256 contiguous bytes.
__global__ void relayout_kernel(const uint8_t* __restrict__ codes, int64_t n, int m, int mw,
                                const int32_t* __restrict__ perm, uint32_t* __restrict__ codes_t,
                                int64_t n_tiles) {
  const int64_t total = n_tiles * mw * 64;
  for (int64_t o = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; o < total;
       o += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t lane = o & 63;
    const int64_t j = (o >> 6) % mw;
    const int64_t t = (o >> 6) / mw;
    const int64_t row = t * 64 + lane;
    uint32_t w = 0;
    if (row < n) {
      const int64_t src = perm ? perm[row] : row;
      for (int b = 0; b < 4; ++b) {
        const int64_t col = j * 4 + b;
        if (col < m) w |= static_cast<uint32_t>(codes[src * m + col]) << (8 * b);
      }
    }
    codes_t[o] = w;
  }
}

__global__ void zero_counts_kernel(unsigned long long* __restrict__ counts, int nq) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nq) counts[i] = 0;
}

}  // namespace

hipError_t launch_relayout_codes(const uint8_t* codes, int64_t n, int m, int mw, const int32_t* perm,
                                 uint32_t* codes_t, int64_t n_tiles, hipStream_t s) {
  const int64_t total = n_tiles * mw * 64;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
  relayout_kernel<<<dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s>>>(codes, n, m, mw, perm,
                                                                          codes_t, n_tiles);
  return hipGetLastError();
}

hipError_t launch_filter(const int32_t* attrs, int64_t n, int n_attr, const DevPred* preds,
                         int nq, bool residual_only, uint64_t* bitmap, int64_t stride64,
                         unsigned long long* counts, hipStream_t s) {
  const int64_t rows_per_block = static_cast<int64_t>(kFilterWaves) * kRowsPerWave;
  const int64_t gx = (n + rows_per_block - 1) / rows_per_block;
  const int gy = (nq + kFilterQueries - 1) / kFilterQueries;
  if (counts) {
    zero_counts_kernel<<<dim3((nq + 255) / 256), dim3(256), 0, s>>>(counts, nq);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  filter_kernel<<<dim3(static_cast<unsigned>(gx), gy), dim3(kFilterWaves * 64), 0, s>>>(
      attrs, n, n_attr, preds, nq, residual_only ? 1 : 0, bitmap, stride64, counts);
  return hipGetLastError();
}

}  // namespace ifvs
