// Per-query conditioning (Section 2, opening paragraph and first display):
// fingerprint <q, f>, gather and sum the h hashed memory-bank rows into alpha
// (M*r values), and w_f = softplus(w_z).  One wavefront per query; the
// pieces (fingerprint, hashes, gather, softplus) are shared with the
// predicate encoder, which conditions the queries it encodes itself.
#include "condition_device.h"

namespace ifvs {

namespace {

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
  uint32_t lo = 0, hi = 0;
  if constexpr (conditioned) fingerprint_query(qrow, dim, lo, hi);
  // no w_z means w_f = 1
  for (int i = lane; i < dim; i += 64) wfrow[i] = wzrow ? softplus_weight(i == lane ? wz0 : wzrow[i]) : 1.0f;
  if constexpr (!conditioned) return;
  const uint64_t key = fingerprint_key(lo, hi, pw);
  const uint32_t my_row = hashed_bank_row(key, seed, lane, H, bank_rows);
  if (rows_out && lane < H) rows_out[static_cast<int64_t>(qi) * H + lane] = static_cast<int32_t>(my_row);
  if constexpr (conditioned) gather_alpha<H>(bank, my_row, mr, lane, alpha_out + static_cast<int64_t>(qi) * mr);
}

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
