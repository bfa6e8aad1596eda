// Select stage (Section 2, stage 3): reduce the per-wavefront candidate
// lists written by the scan to each query's k best (distance, id) pairs in
// ascending order, ties to the smaller id, padding with (-1, +inf) when the
// candidate pool holds fewer than k vectors.
//
// One wavefront per query streams its partial keys (512 at a time, loaded
// together) through the same threshold-filtered pool used by the scan; the
// partial lists are each sorted, so after the first few lists almost every
// key is rejected by one compare.
// When the scan's chunks are absolute cells of a grid, only the slots of the
// cells the query's row interval touches are read (the scan leaves the others
// unwritten); with per-position key counts, only the first that many.
#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

constexpr int kMergeBatch = 8;

__global__ __launch_bounds__(64) void topk_merge_kernel(const uint64_t* __restrict__ partials,
                                                        int64_t per_query, int k, int kpl,
                                                        const int64_t* __restrict__ iv,
                                                        int64_t cell_tiles, int64_t slot_keys,
                                                        const int32_t* __restrict__ qorder,
                                                        const int32_t* __restrict__ n_keys,
                                                        int32_t* __restrict__ ids_out,
                                                        float* __restrict__ dist_out) {
  extern __shared__ uint64_t pool[];
  const int pos = blockIdx.x;                 // position in the scan's query order
  const int q = qorder ? qorder[pos] : pos;   // original query index
  const int lane = threadIdx.x;
  int cnt = 0;
  uint64_t thr = kNoKey;
  const uint64_t* src = partials + static_cast<size_t>(pos) * per_query;
  int64_t first = 0, end = n_keys ? min(per_query, static_cast<int64_t>(n_keys[pos])) : per_query;
  if (cell_tiles > 0) {
    const int64_t r0 = iv[2 * q], r1 = iv[2 * q + 1];
    first = end = 0;
    if (r1 > r0) {
      first = min(per_query, (r0 / 64) / cell_tiles * slot_keys);
      end = min(per_query, ((r1 + 63) / 64 - 1) / cell_tiles * slot_keys + slot_keys);
    }
  }
  // kMergeBatch chunks of 64 keys are loaded together, then offered in order.
  for (int64_t b = first; b < end; b += 64 * kMergeBatch) {
    uint64_t keys[kMergeBatch];
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) {
      const int64_t i = b + 64 * u + lane;
      keys[u] = i < end ? src[i] : kNoKey;
    }
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) {
      if (b + 64 * u >= end) break;
      pool_push(pool, cnt, thr, keys[u], keys[u] < thr, k, kpl);
    }
  }
  pool_compact(pool, cnt, thr, k, kpl);
  for (int e = lane; e < k; e += 64) {
    const uint64_t key = pool[e];
    const size_t o = static_cast<size_t>(q) * k + e;
    if (key == kNoKey) {
      ids_out[o] = -1;
      dist_out[o] = __builtin_inff();
    } else {
      ids_out[o] = static_cast<int32_t>(static_cast<uint32_t>(key));
      dist_out[o] = from_ordered_bits(static_cast<uint32_t>(key >> 32));
    }
  }
}

}  // namespace

hipError_t launch_topk_merge(const uint64_t* partials, int nq, int64_t per_query, int k,
                             const int64_t* iv, int64_t cell_tiles, int64_t slot_keys,
                             const int32_t* qorder, int32_t* ids_out, float* dist_out,
                             hipStream_t s, const int32_t* n_keys) {
  const int kpl = pool_kpl(k);
  const size_t lds = static_cast<size_t>(64 * kpl) * sizeof(uint64_t);
  topk_merge_kernel<<<dim3(nq), dim3(64), lds, s>>>(partials, per_query, k, kpl, iv, cell_tiles,
                                                    slot_keys, qorder, n_keys, ids_out, dist_out);
  return hipGetLastError();
}

}  // namespace ifvs
