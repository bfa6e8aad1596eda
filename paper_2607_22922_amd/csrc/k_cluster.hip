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

// First row whose (c0, c1) key is >= (x0, x1) (x1 ignored when c1 < 0).
__device__ int64_t lower_bound_rows(const int32_t* __restrict__ a0, const int32_t* __restrict__ a1,
                                    int64_t n, int64_t x0, int64_t x1) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    const int64_t v0 = a0[mid];
    bool less = v0 < x0;
    if (a1 && v0 == x0) less = static_cast<int64_t>(a1[mid]) < x1;
    if (less) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__global__ void intervals_kernel(const int32_t* __restrict__ attrs_phys, int64_t n, int c0, int c1,
                                 const DevPred* __restrict__ preds, int nq, int64_t* __restrict__ iv) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= nq) return;
  const DevPred& p = preds[q];
  int64_t r0 = 0, r1 = n;
  if (p.n_eff < 0) {
    r0 = r1 = 0;
  } else if (p.iv_mode == 1) {
    const int32_t* a0 = attrs_phys + static_cast<int64_t>(c0) * n;
    r0 = lower_bound_rows(a0, nullptr, n, p.iv_lo0, 0);
    r1 = lower_bound_rows(a0, nullptr, n, p.iv_hi0, 0);
  } else if (p.iv_mode == 2) {
    const int32_t* a0 = attrs_phys + static_cast<int64_t>(c0) * n;
    const int32_t* a1 = attrs_phys + static_cast<int64_t>(c1) * n;
    r0 = lower_bound_rows(a0, a1, n, p.iv_lo0, p.iv_lo1);
    r1 = lower_bound_rows(a0, a1, n, p.iv_lo0, p.iv_hi1);
  }
  if (r1 < r0) r1 = r0;
  iv[2 * q] = r0;
  iv[2 * q + 1] = r1;
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

hipError_t launch_intervals(const int32_t* attrs_phys, int64_t n, int c0, int c1,
                            const DevPred* preds, int nq, int64_t* iv, hipStream_t s) {
  intervals_kernel<<<dim3((nq + 63) / 64), dim3(64), 0, s>>>(attrs_phys, n, c0, c1, preds, nq, iv);
  return hipGetLastError();
}

}  // namespace ifvs
