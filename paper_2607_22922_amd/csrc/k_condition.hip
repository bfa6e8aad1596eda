// Per-query conditioning (Section 2, opening paragraph and first display):
// fingerprint <q, f>, gather and sum the h hashed memory-bank rows into alpha
// (M*r values), and w_f = softplus(w_z).
//
// One wavefront per query.  FNV-1a is sequential over the bytes by
// definition, so lane 0 folds the fingerprint while the other lanes wait;
// the bank-row sums and the softplus are spread over all 64 lanes.
#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr uint64_t kFnvOffset = 0xCBF29CE484222325ull;
constexpr uint64_t kFnvPrime = 0x100000001B3ull;
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t fnv_bytes(uint64_t h, uint64_t v, int nbytes) {
  for (int b = 0; b < nbytes; ++b) {
    h ^= (v >> (8 * b)) & 0xFFull;
    h *= kFnvPrime;
  }
  return h;
}

// SplitMix64 output for generator state x: add the golden-ratio increment,
// then two xor-shift-multiply rounds and a final xor-shift.
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + kGolden;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

constexpr int kMaxDim = 4096;

__global__ __launch_bounds__(64) void condition_kernel(
    const float* __restrict__ q, int dim, const DevPred* __restrict__ preds,
    const float* __restrict__ bank, int bank_rows, int mr, int h, uint64_t seed,
    const float* __restrict__ w_z, float* __restrict__ alpha_out, float* __restrict__ wf_out) {
  __shared__ uint32_t qbits[kMaxDim];
  const int qi = blockIdx.x;
  const int lane = threadIdx.x;
  const float* qrow = q + static_cast<int64_t>(qi) * dim;

  // w_f = softplus(w_z) in fp64, one rounding to fp32; no w_z means w_f = 1.
  for (int i = lane; i < dim; i += 64) {
    float w = 1.0f;
    if (w_z) {
      const double x = static_cast<double>(w_z[static_cast<int64_t>(qi) * dim + i]);
      w = static_cast<float>(x > 20.0 ? x : log1p(exp(x)));
    }
    wf_out[static_cast<int64_t>(qi) * dim + i] = w;
  }
  if (bank_rows <= 0 || alpha_out == nullptr) return;

  // Fingerprint: FNV-1a-64 over q's fp32 bytes, the clause count (int32) and
  // every clause as (col int32, lo int64, hi int64), little-endian.  The
  // row is staged in LDS by all lanes; the fold itself is serial.
  // The predicate comes from the staging slot (pinned host memory): one
  // wavefront-wide copy into LDS, then the serial fold reads LDS.
  __shared__ DevPred sp;
  for (int i = lane; i < dim; i += 64) qbits[i] = __float_as_uint(qrow[i]);
  copy_pred(preds + qi, &sp, lane);
  __syncthreads();
  uint64_t key = 0;
  if (lane == 0) {
    uint64_t hh = kFnvOffset;
    for (int i = 0; i < dim; ++i) hh = fnv_bytes(hh, qbits[i], 4);
    const DevPred& p = sp;
    hh = fnv_bytes(hh, static_cast<uint32_t>(p.n_raw), 4);
    for (int c = 0; c < p.n_raw; ++c) {
      hh = fnv_bytes(hh, static_cast<uint32_t>(p.raw_col[c]), 4);
      hh = fnv_bytes(hh, static_cast<uint64_t>(p.raw_lo[c]), 8);
      hh = fnv_bytes(hh, static_cast<uint64_t>(p.raw_hi[c]), 8);
    }
    key = hh;
  }
  {
    const int lo = __shfl(static_cast<int>(static_cast<uint32_t>(key)), 0, 64);
    const int hi = __shfl(static_cast<int>(static_cast<uint32_t>(key >> 32)), 0, 64);
    key = (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
  }

  // alpha = bank[row_0] + bank[row_1] + ... in hash-function order from +0.
  for (int e = lane; e < mr; e += 64) {
    float acc = 0.0f;
    for (int j = 0; j < h; ++j) {
      const uint64_t row = splitmix64(key ^ splitmix64(seed + static_cast<uint64_t>(j))) %
                           static_cast<uint64_t>(bank_rows);
      acc = __fadd_rn(acc, bank[static_cast<int64_t>(row) * mr + e]);
    }
    alpha_out[static_cast<int64_t>(qi) * mr + e] = acc;
  }
}

}  // namespace

hipError_t launch_condition(const float* q, int dim, const DevPred* preds, int nq,
                            const float* bank, int bank_rows, int mr, int h, uint64_t seed,
                            const float* w_z, float* alpha_out, float* wf_out, hipStream_t s) {
  condition_kernel<<<dim3(nq), dim3(64), 0, s>>>(q, dim, preds, bank, bank_rows, mr, h, seed, w_z,
                                                 alpha_out, wf_out);
  return hipGetLastError();
}

}  // namespace ifvs
