// Device pieces of the per-query conditioning (Section 2, opening paragraph
// and first display), shared by the condition kernel and the predicate
// encoder (which conditions the queries it encodes in the same launch):
// the FNV-1a-64 fingerprint of <q, f>, the h SplitMix64-hashed memory-bank
// rows, alpha as their sum, and w_f = softplus(w_z).
//
// A wavefront conditions one query.  FNV-1a is sequential over the bytes by
// definition; the state is the same for every lane, so the fold runs on the
// scalar unit (operands are moved to scalar registers with readlane) while
// the bank-row hashes and sums are spread over the 64 lanes.
#pragma once

#include "ifvs_internal.h"

namespace ifvs {

constexpr uint64_t kFnvOffset = 0xCBF29CE484222325ull;
constexpr uint64_t kFnvPrime = 0x100000001B3ull;
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr int kMaxHashes = 16;   // h limit checked at load
constexpr int kAlphaUnroll = 4;  // alpha elements per lane per pass

// One FNV-1a-64 step (xor the byte, multiply by the prime) on a state held as
// two 32-bit halves.  The prime is 2^40 + 0x1B3, so state * prime =
// (state << 40) + state * 0x1B3 modulo 2^64: the new low word is
// lo * 0x1B3 and the new high word is hi * 0x1B3 + the high half of
// lo * 0x1B3 + (lo << 8).  With uniform operands this is scalar arithmetic.
__device__ __forceinline__ void fnv_byte(uint32_t& lo, uint32_t& hi, uint32_t b) {
  static_assert(kFnvPrime == (1ull << 40) + 0x1B3ull, "prime decomposition");
  lo ^= b;
  hi = hi * 0x1B3u + __umulhi(lo, 0x1B3u) + (lo << 8);
  lo = lo * 0x1B3u;
}

// The four bytes of a 32-bit word, least significant first.
__device__ __forceinline__ void fnv_word(uint32_t& lo, uint32_t& hi, uint32_t w) {
  fnv_byte(lo, hi, w & 0xFFu);
  fnv_byte(lo, hi, (w >> 8) & 0xFFu);
  fnv_byte(lo, hi, (w >> 16) & 0xFFu);
  fnv_byte(lo, hi, w >> 24);
}

// SplitMix64 output for generator state x: add the golden-ratio increment,
// then two xor-shift-multiply rounds and a final xor-shift.
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + kGolden;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint32_t lane_word(uint32_t v, int j) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), j));
}

// The fingerprint's first part: the FNV-1a offset basis folded with q's
// fp32 words (dim of them at qrow, a wave-uniform address), read 8 at a time
// with scalar loads, the next 8 loading while the current 8 are folded.
__device__ __forceinline__ void fingerprint_query(const float* qrow, int dim, uint32_t& lo, uint32_t& hi) {
  lo = static_cast<uint32_t>(kFnvOffset);
  hi = static_cast<uint32_t>(kFnvOffset >> 32);
  const uint32_t* qw = reinterpret_cast<const uint32_t*>(qrow);
  int i = 0;
  if (dim >= 8) {
    uint32_t w[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) w[t] = qw[t];
    for (; i + 8 <= dim; i += 8) {
      const int nx = i + 16 <= dim ? i + 8 : i;  // stays inside the row
      uint32_t nw[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) nw[t] = qw[nx + t];
#pragma unroll
      for (int t = 0; t < 8; ++t) fnv_word(lo, hi, w[t]);
#pragma unroll
      for (int t = 0; t < 8; ++t) w[t] = nw[t];
    }
  }
  for (; i < dim; ++i) fnv_word(lo, hi, qw[i]);
}

// Dword offset of a DevPred field (the predicate is held one dword per lane).
#define IFVS_PRED_WORD(field) static_cast<int>(offsetof(DevPred, field) / 4)

// The rest of the fingerprint, the predicate as given (clause count int32,
// then every clause as col int32, lo int64, hi int64, little-endian; pw is
// dword `lane` of the DevPred), and the 64-bit key.
__device__ __forceinline__ uint64_t fingerprint_key(uint32_t lo, uint32_t hi, uint32_t pw) {
  const int n_raw = static_cast<int>(lane_word(pw, IFVS_PRED_WORD(n_raw)));
  fnv_word(lo, hi, static_cast<uint32_t>(n_raw));
  for (int c = 0; c < n_raw; ++c) {
    fnv_word(lo, hi, lane_word(pw, IFVS_PRED_WORD(raw_col) + c));
    fnv_word(lo, hi, lane_word(pw, IFVS_PRED_WORD(raw_lo) + 2 * c));
    fnv_word(lo, hi, lane_word(pw, IFVS_PRED_WORD(raw_lo) + 2 * c + 1));
    fnv_word(lo, hi, lane_word(pw, IFVS_PRED_WORD(raw_hi) + 2 * c));
    fnv_word(lo, hi, lane_word(pw, IFVS_PRED_WORD(raw_hi) + 2 * c + 1));
  }
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

#undef IFVS_PRED_WORD

// Bank row of hash function j = lane (lanes below h; 0 elsewhere).
__device__ __forceinline__ uint32_t hashed_bank_row(uint64_t key, uint64_t seed, int lane, int h, int bank_rows) {
  if (lane >= h) return 0u;
  return static_cast<uint32_t>(splitmix64(key ^ splitmix64(seed + static_cast<uint64_t>(lane))) %
                               static_cast<uint64_t>(bank_rows));
}

// alpha = bank[row_0] + bank[row_1] + ... in hash-function order from +0
// (row j held by lane j), written to arow [mr].  Each pass covers
// kAlphaUnroll elements per lane; all H * kAlphaUnroll loads are issued
// before the first add.
template <int H>
__device__ __forceinline__ void gather_alpha(const float* __restrict__ bank, uint32_t my_row, int mr, int lane,
                                             float* __restrict__ arow) {
  for (int e0 = lane; e0 < mr; e0 += 64 * kAlphaUnroll) {
    float v[H][kAlphaUnroll];
#pragma unroll
    for (int j = 0; j < H; ++j) {
      const float* brow = bank + static_cast<int64_t>(lane_word(my_row, j)) * mr;
#pragma unroll
      for (int u = 0; u < kAlphaUnroll; ++u) {
        const int e = e0 + 64 * u;
        v[j][u] = brow[e < mr ? e : mr - 1];
      }
    }
#pragma unroll
    for (int u = 0; u < kAlphaUnroll; ++u) {
      float acc = 0.0f;
#pragma unroll
      for (int j = 0; j < H; ++j) acc = __fadd_rn(acc, v[j][u]);
      const int e = e0 + 64 * u;
      if (e < mr) arow[e] = acc;
    }
  }
}

// w_f = softplus(w_z), computed in fp64 and rounded once to fp32.
__device__ __forceinline__ float softplus_weight(float wz) {
  const double x = static_cast<double>(wz);
  return static_cast<float>(x > 20.0 ? x : log1p(exp(x)));
}

}  // namespace ifvs
