// Filter stage (Section 2, stage 1): evaluate each query's conjunctive
// predicate over the attribute columns and emit the candidate pool P as a
// selection bitmap, plus the pool size.
//
// One wavefront covers 4096 consecutive vectors and tests each attribute
// value it reads against the predicates of all kFilterQueries queries of its
// workgroup.  Clause lists live in LDS.
//  * Single-column groups (every query one range clause on the same column,
//    the common case): the wavefront stages 2048 values at a time in LDS with
//    coalesced loads, then lane L walks rows 32L + 31 .. 32L of the block
//    (padded LDS layout, no bank conflicts) and shifts each query's compare
//    bit into its own 32-bit word: word = 2 * word + (v - lo < width).  Each
//    lane then holds bitmap word L of the block per query (bit r = row
//    32L + r), so the stores are coalesced and no cross-lane move is needed:
//    three VALU operations per 64 (row, query) pairs.
//  * Other groups: in step `it` (0..63) lane L loads the attributes of vector
//    base + 64*it + L; the compare result of the wavefront is the 64-bit
//    ballot word of those 64 vectors, which lane `it` keeps (one word per
//    query), and the wavefront stores 512 contiguous bytes per query.
// Pool sizes: each workgroup sums its waves' popcounts in LDS and writes one
// partial count per query (no atomics: device-wide atomics on the same few
// counters serialised the whole kernel); a small kernel adds the partials
// and leaves their exclusive prefix sums for the row-list compaction.
#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr int kFilterWaves = 4;
constexpr int kRowsPerWave = 64 * 64;
static_assert(kFilterWaves * kRowsPerWave == kFilterPartRows, "one count partial per workgroup");
constexpr int kBlockRows = 2048;                        // rows staged per wavefront at a time
constexpr int kBlockPad = kBlockRows + kBlockRows / 32; // one pad word per 32 rows

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
    int64_t stride64, uint32_t* __restrict__ count_parts) {
  __shared__ PassClauses sc[kFilterQueries];
  __shared__ uint32_t s_vals[kFilterWaves * kBlockPad];
  __shared__ uint32_t s_cnt[kFilterWaves][kFilterQueries];
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
  // A wavefront past the last row does nothing but still joins the count
  // reduction's barrier.
  const bool active = base < n;
  // Common case: every query of the group tests one clause on the same
  // column (the transposed path below).
  int single_col = qn > 0 && sc[0].nc == 1 ? sc[0].col[0] : -1;
  for (int qi = 1; qi < qn; ++qi)
    if (sc[qi].nc != 1 || sc[qi].col[0] != single_col) single_col = -1;

  uint32_t cnt[kFilterQueries];   // this lane's selected rows per query
#pragma unroll
  for (int qi = 0; qi < kFilterQueries; ++qi) cnt[qi] = 0;

  if (active && single_col >= 0) {
    const int32_t* __restrict__ col = attrs + static_cast<int64_t>(single_col) * n;
    uint32_t lo[kFilterQueries], width[kFilterQueries];
#pragma unroll
    for (int qi = 0; qi < kFilterQueries; ++qi) {
      lo[qi] = qi < qn ? sc[qi].lo[0] : 0;
      width[qi] = qi < qn ? sc[qi].width[0] : 0;   // width 0: nothing passes
    }
    uint32_t* vals = s_vals + wave * kBlockPad;
    uint32_t* bitmap32 = reinterpret_cast<uint32_t*>(bitmap);
    for (int blk = 0; blk < kRowsPerWave / kBlockRows; ++blk) {
      const int64_t bb = base + static_cast<int64_t>(blk) * kBlockRows;
      // Stage the block: local row r at vals[r + r / 32] (rows past n repeat
      // the last row and are masked below).
#pragma unroll 8
      for (int j = 0; j < kBlockRows / 64; ++j) {
        const int r = 64 * j + lane;
        const int64_t i = bb + r;
        vals[r + (r >> 5)] = static_cast<uint32_t>(col[i < n ? i : n - 1]);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // Lane L: rows 32L + 31 down to 32L, so row 32L + r lands in bit r.
      uint32_t word[kFilterQueries];
#pragma unroll
      for (int qi = 0; qi < kFilterQueries; ++qi) word[qi] = 0;
      const uint32_t* mine = vals + 33 * lane;
#pragma unroll 4
      for (int r = 31; r >= 0; --r) {
        const uint32_t v = mine[r];
#pragma unroll
        for (int qi = 0; qi < kFilterQueries; ++qi)
          word[qi] = word[qi] + word[qi] + (v - lo[qi] < width[qi] ? 1u : 0u);
      }
      const int64_t row0 = bb + 32 * lane;
      uint32_t valid = ~0u;
      if (row0 + 32 > n) valid = row0 >= n ? 0u : ((1u << static_cast<int>(n - row0)) - 1u);
      const int64_t w32 = bb / 32 + lane;
#pragma unroll
      for (int qi = 0; qi < kFilterQueries; ++qi) {
        if (qi < qn) {
          const uint32_t wd = word[qi] & valid;
          if (w32 < 2 * stride64) bitmap32[static_cast<int64_t>(q0 + qi) * 2 * stride64 + w32] = wd;
          cnt[qi] += static_cast<uint32_t>(__popc(wd));
        }
      }
      // The next block overwrites vals only after every lane has read it.
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  } else if (active) {
  // held_{lo,hi}[qi] of lane L: the ballot word of step L for query qi.
  uint32_t held_lo[kFilterQueries], held_hi[kFilterQueries];
#pragma unroll
  for (int qi = 0; qi < kFilterQueries; ++qi) held_lo[qi] = held_hi[qi] = 0;

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

  const int64_t w64 = base / 64 + lane;           // this lane's 64-bit word
#pragma unroll
  for (int qi = 0; qi < kFilterQueries; ++qi) {
    if (qi < qn) {
      const uint64_t word = (static_cast<uint64_t>(held_hi[qi]) << 32) | held_lo[qi];
      if (w64 < stride64) bitmap[static_cast<int64_t>(q0 + qi) * stride64 + w64] = word;
      cnt[qi] = static_cast<uint32_t>(__popcll(word));
    }
  }
  }

  // Pool sizes: wavefront sums, then one partial per (workgroup, query).
  if (count_parts) {
#pragma unroll
    for (int qi = 0; qi < kFilterQueries; ++qi) {
      unsigned c = cnt[qi];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) c += __shfl_down(c, off, 64);
      if (lane == 0) s_cnt[wave][qi] = c;
    }
    __syncthreads();
    if (threadIdx.x < qn) {
      uint32_t sum = 0;
#pragma unroll
      for (int w = 0; w < kFilterWaves; ++w) sum += s_cnt[w][threadIdx.x];
      count_parts[static_cast<int64_t>(q0 + threadIdx.x) * gridDim.x + blockIdx.x] = sum;
    }
  }
}

// counts[q] = sum of the q-th row of count_parts ([nq][parts]), and the
// row is turned into its exclusive prefix sums in place (the compaction
// kernel's output offsets; every count is below 2^31).  One wavefront per
// query.
__global__ __launch_bounds__(64) void reduce_counts_kernel(uint32_t* __restrict__ count_parts, int parts,
                                                           int nq, unsigned long long* __restrict__ counts) {
  const int q = blockIdx.x;
  if (q >= nq) return;
  const int lane = threadIdx.x;
  uint32_t* row = count_parts + static_cast<int64_t>(q) * parts;
  uint32_t carry = 0;
  for (int i0 = 0; i0 < parts; i0 += 64) {
    const int i = i0 + lane;
    const uint32_t v = i < parts ? row[i] : 0u;
    uint32_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t y = __shfl_up(incl, off, 64);
      if (lane >= off) incl += y;
    }
    if (i < parts) row[i] = carry + incl - v;
    carry += __shfl(incl, 63, 64);
  }
  if (lane == 0) counts[q] = carry;
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

}  // namespace

hipError_t launch_relayout_codes(const uint8_t* codes, int64_t n, int m, int mw, const int32_t* perm,
                                 uint32_t* codes_t, int64_t n_tiles, hipStream_t s) {
  const int64_t total = n_tiles * mw * 64;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
  relayout_kernel<<<dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s>>>(codes, n, m, mw, perm,
                                                                          codes_t, n_tiles);
  return hipGetLastError();
}

int64_t filter_count_parts(int64_t n) {
  const int64_t rows_per_block = static_cast<int64_t>(kFilterWaves) * kRowsPerWave;
  return (n + rows_per_block - 1) / rows_per_block;
}

hipError_t launch_filter(const int32_t* attrs, int64_t n, int n_attr, const DevPred* preds,
                         int nq, bool residual_only, uint64_t* bitmap, int64_t stride64,
                         unsigned long long* counts, uint32_t* count_parts, hipStream_t s) {
  const int64_t gx = filter_count_parts(n);
  const int gy = (nq + kFilterQueries - 1) / kFilterQueries;
  filter_kernel<<<dim3(static_cast<unsigned>(gx), gy), dim3(kFilterWaves * 64), 0, s>>>(
      attrs, n, n_attr, preds, nq, residual_only ? 1 : 0, bitmap, stride64, counts ? count_parts : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !counts) return e;
  reduce_counts_kernel<<<dim3(nq), dim3(64), 0, s>>>(count_parts, static_cast<int>(gx), nq, counts);
  return hipGetLastError();
}

}  // namespace ifvs
