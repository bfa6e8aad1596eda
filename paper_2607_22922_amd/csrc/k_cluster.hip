// Instance-optimized physical layout: rows stored in the order of their
// cluster-key attribute values, so that a range (or equality + range) clause
// on the key selects one contiguous interval of rows (the Filter stage of
// Section 2 over a layout tailored to the workload's predicates; the paper's
// theme is tailoring components to a given dataset and query workload).
//
// The permutation is a stable LSD radix sort of 64-bit keys
// (order-preserving attr[c0] bits << 32 | attr[c1] bits) paired with row ids,
// so rows with equal keys keep id order.  Each query's interval comes from two
// binary searches over the clustered key columns.
#include <hipcub/hipcub.hpp>

#include "ifvs_internal.h"
#include "intervals_device.h"

namespace ifvs {

namespace {

__device__ __forceinline__ uint32_t key_bits(int32_t v) { return static_cast<uint32_t>(v) ^ 0x80000000u; }

__global__ void make_keys_kernel(const int32_t* __restrict__ attrs, int64_t n, int n_cluster, int c0,
                                 int c1, uint64_t* __restrict__ keys, int32_t* __restrict__ ids) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const uint64_t hi = key_bits(attrs[static_cast<int64_t>(c0) * n + i]);
    const uint64_t lo = n_cluster > 1 ? key_bits(attrs[static_cast<int64_t>(c1) * n + i]) : 0u;
    keys[i] = (hi << 32) | lo;
    ids[i] = static_cast<int32_t>(i);
  }
}

__global__ void gather_attrs_kernel(const int32_t* __restrict__ attrs, int64_t n, int n_attr,
                                    const int32_t* __restrict__ perm, int32_t* __restrict__ out) {
  const int64_t total = n * n_attr;
  for (int64_t o = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; o < total;
       o += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t col = o / n, row = o % n;
    out[o] = attrs[col * n + perm[row]];
  }
}

// Two wavefronts per query (lower and upper bound), one per workgroup; the
// dispatch-order copy is spread over all of them.
__global__ __launch_bounds__(64) void intervals_kernel(const IntervalArgs a) {
  copy_slot_order(a, blockIdx.x, gridDim.x, threadIdx.x);
  const int q = blockIdx.x >> 1;
  if (q < a.nq) interval_bound(a, q, blockIdx.x & 1, threadIdx.x);
}

unsigned grid_for(int64_t work) { return static_cast<unsigned>(std::min<int64_t>((work + 255) / 256, 65536)); }

}  // namespace

hipError_t cluster_permutation(const int32_t* attrs, int64_t n, int n_cluster, int c0, int c1,
                               int32_t* perm, hipStream_t s) {
  uint64_t *keys = nullptr, *keys_sorted = nullptr;
  int32_t* ids = nullptr;
  void* temp = nullptr;
  size_t temp_bytes = 0;
  hipError_t e = hipMalloc(&keys, sizeof(uint64_t) * n);
  if (e == hipSuccess) e = hipMalloc(&keys_sorted, sizeof(uint64_t) * n);
  if (e == hipSuccess) e = hipMalloc(&ids, sizeof(int32_t) * n);
  if (e == hipSuccess) {
    make_keys_kernel<<<grid_for(n), 256, 0, s>>>(attrs, n, n_cluster, c0, c1, keys, ids);
    e = hipGetLastError();
  }
  // All 64 key bits, also for one column (low word zero): a sort restricted to
  // bits [32, 64) returned unsorted output for n >= 1e4 on this ROCm's
  // rocPRIM, while the full range is sorted and stable.
  const int begin_bit = 0;
  if (e == hipSuccess)
    e = hipcub::DeviceRadixSort::SortPairs(nullptr, temp_bytes, keys, keys_sorted, ids, perm, n,
                                           begin_bit, 64, s);
  if (e == hipSuccess) e = hipMalloc(&temp, temp_bytes);
  if (e == hipSuccess)
    e = hipcub::DeviceRadixSort::SortPairs(temp, temp_bytes, keys, keys_sorted, ids, perm, n,
                                           begin_bit, 64, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  hipFree(temp);
  hipFree(ids);
  hipFree(keys_sorted);
  hipFree(keys);
  return e;
}

hipError_t launch_gather_attrs(const int32_t* attrs, int64_t n, int n_attr, const int32_t* perm,
                               int32_t* attrs_phys, hipStream_t s) {
  gather_attrs_kernel<<<grid_for(n * n_attr), 256, 0, s>>>(attrs, n, n_attr, perm, attrs_phys);
  return hipGetLastError();
}

hipError_t launch_intervals(const IntervalArgs& a, hipStream_t s) {
  if (a.nq <= 0 && a.n_slots <= 0) return hipSuccess;
  intervals_kernel<<<dim3(2 * a.nq > 0 ? 2 * a.nq : 1), dim3(64), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace ifvs
