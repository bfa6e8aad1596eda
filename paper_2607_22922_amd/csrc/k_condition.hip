// Per-query conditioning (Section 2, opening paragraph and first display):
// fingerprint <q, f>, gather and sum the h hashed memory-bank rows into alpha
// (M*r values), and w_f = softplus(w_z).
//
// One wavefront per query.  FNV-1a is sequential over the bytes by
// definition; the state is the same for every lane, so the fold runs on the
// scalar unit (operands are moved to scalar registers with readlane) while
// the softplus, the h bank-row hashes and the bank-row sums are spread over
// the 64 lanes.
#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr uint64_t kFnvOffset = 0xCBF29CE484222325ull;
constexpr uint64_t kFnvPrime = 0x100000001B3ull;
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

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

// Dword offset of a DevPred field (the predicate is held one dword per lane).
#define PRED_WORD(field) static_cast<int>(offsetof(DevPred, field) / 4)

__device__ __forceinline__ uint32_t lane_word(uint32_t v, int j) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), j));
}

constexpr int kMaxHashes = 16;   // h limit checked at load
constexpr int kAlphaUnroll = 4;  // alpha elements per lane per pass

// H is the number of hash functions h (1..kMaxHashes), or 0 when there is no
// memory bank (w_f only).
template <int H>
__global__ __launch_bounds__(64) void condition_kernel(
    const float* __restrict__ q, int dim, const DevPred* __restrict__ preds,
    const float* __restrict__ bank, int bank_rows, int mr, uint64_t seed,
    const float* __restrict__ w_z, float* __restrict__ alpha_out, float* __restrict__ wf_out,
    int32_t* __restrict__ rows_out) {
  const int qi = blockIdx.x;
  const int lane = threadIdx.x;
  const float* qrow = q + static_cast<int64_t>(qi) * dim;
  const float* wzrow = w_z ? w_z + static_cast<int64_t>(qi) * dim : nullptr;
  float* wfrow = wf_out + static_cast<int64_t>(qi) * dim;
  constexpr bool conditioned = H > 0;

  // The predicate (one dword per lane from the staging slot in pinned host
  // memory, the slowest load) and w_z's first 64 values go out first.
  constexpr int kPredWords = static_cast<int>(sizeof(DevPred) / 4);
  static_assert(sizeof(DevPred) % 4 == 0 && kPredWords <= 64, "one dword per lane");
  const uint32_t pw =
      (conditioned && lane < kPredWords) ? reinterpret_cast<const uint32_t*>(preds + qi)[lane] : 0u;
  const float wz0 = (wzrow && lane < dim) ? wzrow[lane] : 0.0f;

  // Fingerprint: FNV-1a-64 over q's fp32 bytes, the clause count (int32) and
  // every clause as (col int32, lo int64, hi int64), little-endian.  q's
  // words are read 8 at a time with uniform (scalar) loads, the next 8
  // loading while the current 8 are folded.
  uint32_t lo = static_cast<uint32_t>(kFnvOffset);
  uint32_t hi = static_cast<uint32_t>(kFnvOffset >> 32);
  if constexpr (conditioned) {
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

  // w_f = softplus(w_z) in fp64, one rounding to fp32; no w_z means w_f = 1.
  for (int i = lane; i < dim; i += 64) {
    float w = 1.0f;
    if (wzrow) {
      const double x = static_cast<double>(i == lane ? wz0 : wzrow[i]);
      w = static_cast<float>(x > 20.0 ? x : log1p(exp(x)));
    }
    wfrow[i] = w;
  }
  if constexpr (!conditioned) return;

  const int n_raw = static_cast<int>(lane_word(pw, PRED_WORD(n_raw)));
  fnv_word(lo, hi, static_cast<uint32_t>(n_raw));
  for (int c = 0; c < n_raw; ++c) {
    fnv_word(lo, hi, lane_word(pw, PRED_WORD(raw_col) + c));
    fnv_word(lo, hi, lane_word(pw, PRED_WORD(raw_lo) + 2 * c));
    fnv_word(lo, hi, lane_word(pw, PRED_WORD(raw_lo) + 2 * c + 1));
    fnv_word(lo, hi, lane_word(pw, PRED_WORD(raw_hi) + 2 * c));
    fnv_word(lo, hi, lane_word(pw, PRED_WORD(raw_hi) + 2 * c + 1));
  }
  const uint64_t key = (static_cast<uint64_t>(hi) << 32) | lo;

  // Bank row of hash function j, computed once by lane j.
  uint32_t my_row = 0;
  if (lane < H)
    my_row = static_cast<uint32_t>(
        splitmix64(key ^ splitmix64(seed + static_cast<uint64_t>(lane))) %
        static_cast<uint64_t>(bank_rows));

  if (rows_out && lane < H) rows_out[static_cast<int64_t>(qi) * H + lane] = static_cast<int32_t>(my_row);

  // alpha = bank[row_0] + bank[row_1] + ... in hash-function order from +0.
  // Each pass covers kAlphaUnroll elements per lane; all H * kAlphaUnroll
  // loads are issued before the first add.
  float* arow = alpha_out + static_cast<int64_t>(qi) * mr;
  for (int e0 = lane; e0 < mr; e0 += 64 * kAlphaUnroll) {
    float v[H > 0 ? H : 1][kAlphaUnroll];
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

#undef PRED_WORD

}  // namespace

hipError_t launch_condition(const float* q, int dim, const DevPred* preds, int nq,
                            const float* bank, int bank_rows, int mr, int h, uint64_t seed,
                            const float* w_z, float* alpha_out, float* wf_out, hipStream_t s,
                            int32_t* rows_out) {
  const int hh = (bank_rows > 0 && alpha_out != nullptr) ? h : 0;
  if (hh < 0 || hh > kMaxHashes) return hipErrorInvalidValue;
  const dim3 grid(nq), block(64);
#define IFVS_CONDITION_CASE(H)                                                              \
  case H:                                                                                    \
    condition_kernel<H><<<grid, block, 0, s>>>(q, dim, preds, bank, bank_rows, mr, seed, w_z, \
                                               alpha_out, wf_out, rows_out);                 \
    break;
  switch (hh) {
    IFVS_CONDITION_CASE(0) IFVS_CONDITION_CASE(1) IFVS_CONDITION_CASE(2)
    IFVS_CONDITION_CASE(3) IFVS_CONDITION_CASE(4) IFVS_CONDITION_CASE(5)
    IFVS_CONDITION_CASE(6) IFVS_CONDITION_CASE(7) IFVS_CONDITION_CASE(8)
    IFVS_CONDITION_CASE(9) IFVS_CONDITION_CASE(10) IFVS_CONDITION_CASE(11)
    IFVS_CONDITION_CASE(12) IFVS_CONDITION_CASE(13) IFVS_CONDITION_CASE(14)
    IFVS_CONDITION_CASE(15) IFVS_CONDITION_CASE(16)
  }
#undef IFVS_CONDITION_CASE
  return hipGetLastError();
}

}  // namespace ifvs
