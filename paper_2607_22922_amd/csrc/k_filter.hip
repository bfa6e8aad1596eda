// Filter stage (Section 2, stage 1): evaluate each query's conjunctive
// predicate over the attribute columns and emit the candidate pool P as a
// selection bitmap, plus the pool size.
//
// One wavefront covers 4096 consecutive vectors: in step `it` (0..63) lane L
// tests vector base + 64*it + L against up to kFilterQueries predicates; the
// compare result of the wavefront is itself the 64-bit ballot word of those
// 64 vectors, which lane `it` keeps.  After 64 steps every lane holds one
// 64-bit word per query and the wavefront stores 512 contiguous bytes per
// query.  Attribute values are read once per group of kFilterQueries queries.
#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr int kFilterWaves = 4;
constexpr int kRowsPerWave = 64 * 64;

__device__ __forceinline__ int32_t attr_value(const int32_t* __restrict__ attrs, int64_t n,
                                              int col, int64_t i, int32_t a0, int32_t a1) {
  if (col == 0) return a0;
  if (col == 1) return a1;
  return attrs[static_cast<int64_t>(col) * n + i];
}

__global__ __launch_bounds__(kFilterWaves * 64) void filter_kernel(
    const int32_t* __restrict__ attrs, int64_t n, int n_attr,
    const DevPred* __restrict__ preds, int nq, uint64_t* __restrict__ bitmap, int64_t stride64,
    unsigned long long* __restrict__ counts) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int q0 = blockIdx.y * kFilterQueries;
  const int qn = min(kFilterQueries, nq - q0);
  const int64_t base = (static_cast<int64_t>(blockIdx.x) * kFilterWaves + wave) * kRowsPerWave;
  if (base >= n) return;

  uint64_t held[kFilterQueries];
#pragma unroll
  for (int qi = 0; qi < kFilterQueries; ++qi) held[qi] = 0;

  for (int it = 0; it < 64; ++it) {
    const int64_t i = base + static_cast<int64_t>(it) * 64 + lane;
    const bool in = i < n;
    const int32_t a0 = (in && n_attr > 0) ? attrs[i] : 0;
    const int32_t a1 = (in && n_attr > 1) ? attrs[n + i] : 0;
#pragma unroll
    for (int qi = 0; qi < kFilterQueries; ++qi) {
      if (qi >= qn) break;
      const DevPred& p = preds[q0 + qi];
      bool pass = in && p.n_eff >= 0;
      for (int c = 0; c < p.n_eff; ++c) {
        const int32_t v = in ? attr_value(attrs, n, p.col[c], i, a0, a1) : 0;
        pass = pass && (static_cast<uint32_t>(v) - static_cast<uint32_t>(p.lo[c]) < p.width[c]);
      }
      const uint64_t word = __ballot(pass);
      if (lane == it) held[qi] = word;
    }
  }

  const int64_t w64 = base / 64 + lane;           // this lane's 64-bit word
#pragma unroll
  for (int qi = 0; qi < kFilterQueries; ++qi) {
    if (qi >= qn) break;
    if (w64 < stride64) bitmap[static_cast<int64_t>(q0 + qi) * stride64 + w64] = held[qi];
    unsigned long long c = __popcll(held[qi]);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) c += __shfl_down(c, off, 64);
    if (lane == 0 && counts) atomicAdd(&counts[q0 + qi], c);
  }
}

// codes [n][m] bytes -> tiles of 64 rows: word j of row (64t + L) is stored at
// codes_t[(t*mw + j)*64 + L] and holds bytes 4j..4j+3 of the row (zero past m
// and past n), so a wavefront reading word j of a tile reads 256 contiguous
// bytes.
__global__ void relayout_kernel(const uint8_t* __restrict__ codes, int64_t n, int m, int mw,
                                uint32_t* __restrict__ codes_t, int64_t n_tiles) {
  const int64_t total = n_tiles * mw * 64;
  for (int64_t o = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; o < total;
       o += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t lane = o & 63;
    const int64_t j = (o >> 6) % mw;
    const int64_t t = (o >> 6) / mw;
    const int64_t row = t * 64 + lane;
    uint32_t w = 0;
    if (row < n) {
      for (int b = 0; b < 4; ++b) {
        const int64_t col = j * 4 + b;
        if (col < m) w |= static_cast<uint32_t>(codes[row * m + col]) << (8 * b);
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

hipError_t launch_relayout_codes(const uint8_t* codes, int64_t n, int m, int mw,
                                 uint32_t* codes_t, int64_t n_tiles, hipStream_t s) {
  const int64_t total = n_tiles * mw * 64;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
  relayout_kernel<<<dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s>>>(codes, n, m, mw, codes_t,
                                                                          n_tiles);
  return hipGetLastError();
}

hipError_t launch_filter(const int32_t* attrs, int64_t n, int n_attr, const DevPred* preds,
                         int nq, uint64_t* bitmap, int64_t stride64,
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
      attrs, n, n_attr, preds, nq, bitmap, stride64, counts);
  return hipGetLastError();
}

}  // namespace ifvs
