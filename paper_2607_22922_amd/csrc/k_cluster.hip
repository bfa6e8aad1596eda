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

// (c0, c1) key of row r is below (x0, x1)?  (x1 ignored when a1 is null.)
__device__ __forceinline__ bool key_below(const int32_t* __restrict__ a0, const int32_t* __restrict__ a1,
                                          int64_t r, int64_t x0, int64_t x1) {
  const int64_t v0 = a0[r];
  if (a1 && v0 == x0) return static_cast<int64_t>(a1[r]) < x1;
  return v0 < x0;
}

// First row of [lo, hi) whose key is >= (x0, x1) (hi when there is none),
// given that the rows before lo are below it: a 64-ary search by one
// wavefront.  Each step every lane probes one of 64 evenly spaced rows of the
// current range; the ballot of "probe below x" narrows the range to the gap
// after the last such probe, so 10^7 rows take four dependent loads.
__device__ int64_t wave_lower_bound(const int32_t* __restrict__ a0, const int32_t* __restrict__ a1,
                                    int64_t lo, int64_t hi, int64_t x0, int64_t x1) {
  const int lane = threadIdx.x & 63;
  while (hi - lo > 64) {
    const int64_t step = (hi - lo + 63) / 64;
    const int64_t r = lo + lane * step; // probes lo, lo+step, ... (< hi or past it)
    const bool below = r < hi && key_below(a0, a1, r, x0, x1);
    const uint64_t mask = __ballot(below);
    if (mask == 0) {
      hi = lo;                           // key(lo) >= x
    } else {
      const int last = 63 - __clzll(mask);
      const int64_t r_last = lo + last * step;
      lo = r_last + 1;
      hi = min(hi, r_last + step);
    }
  }
  // Final <= 64 rows: one probe per lane.
  const int64_t r = lo + lane;
  const bool below = r < hi && key_below(a0, a1, r, x0, x1);
  return lo + __popcll(__ballot(below));
}

// First row whose leading key is >= x, from the value table (vstart[t] =
// first row with leading key >= vmin + t, t < vcount; the last entry is n).
__device__ __forceinline__ int64_t table_lower_bound(const int32_t* __restrict__ vstart, int64_t vmin,
                                                     int64_t vcount, int64_t n, int64_t x) {
  if (x <= vmin) return 0;
  if (x >= vmin + (vcount - 1)) return n;
  return vstart[x - vmin];
}

__global__ __launch_bounds__(64) void intervals_kernel(const int32_t* __restrict__ attrs_phys, int64_t n,
                                                       int c0, int c1, const int32_t* __restrict__ vstart,
                                                       int64_t vmin, int64_t vcount,
                                                       const DevPred* __restrict__ staged_preds,
                                                       const int32_t* __restrict__ staged_order, int nq,
                                                       DevPred* __restrict__ preds_out,
                                                       int32_t* __restrict__ order_out,
                                                       int64_t* __restrict__ iv,
                                                       uint64_t* __restrict__ gthr,
                                                       const int32_t* __restrict__ slots_src,
                                                       int32_t* __restrict__ slots_dst, int64_t n_slots) {
  const int q = blockIdx.x >> 1;        // two wavefronts per query: lower and upper bound
  const bool upper = blockIdx.x & 1;
  // The scan's dispatch order, spread over all workgroups of this launch.
  for (int64_t i = blockIdx.x * 64 + threadIdx.x; i < n_slots; i += static_cast<int64_t>(gridDim.x) * 64)
    slots_dst[i] = slots_src[i];
  if (q >= nq) return;
  __shared__ DevPred sp;
  copy_pred(staged_preds + q, &sp, threadIdx.x);
  __syncthreads();
  if (!upper) {
    copy_pred(&sp, preds_out + q, threadIdx.x);
    if (threadIdx.x == 0) order_out[q] = staged_order[q];
  }
  const DevPred& p = sp;
  int64_t r = upper ? n : 0;
  if (p.n_eff < 0) {
    r = 0;
  } else if (p.iv_mode == 1) {
    const int64_t x = upper ? p.iv_hi0 : p.iv_lo0;
    if (vstart) {
      r = table_lower_bound(vstart, vmin, vcount, n, x);
    } else {
      const int32_t* a0 = attrs_phys + static_cast<int64_t>(c0) * n;
      r = wave_lower_bound(a0, nullptr, 0, n, x, 0);
    }
  } else if (p.iv_mode == 2) {
    // Leading key equal to iv_lo0, second key in [iv_lo1, iv_hi1): the value
    // table (when present) gives the rows of that leading key, the search
    // runs inside them.
    const int32_t* a0 = attrs_phys + static_cast<int64_t>(c0) * n;
    const int32_t* a1 = attrs_phys + static_cast<int64_t>(c1) * n;
    int64_t lo = 0, hi = n;
    if (vstart) {
      lo = table_lower_bound(vstart, vmin, vcount, n, p.iv_lo0);
      hi = table_lower_bound(vstart, vmin, vcount, n, p.iv_lo0 + 1);
    }
    r = wave_lower_bound(a0, a1, lo, hi, p.iv_lo0, upper ? p.iv_hi1 : p.iv_lo1);
  }
  if (threadIdx.x == 0) {
    iv[2 * q + (upper ? 1 : 0)] = r;
    if (!upper) gthr[q] = ~0ull;
  }
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

hipError_t launch_intervals(const int32_t* attrs_phys, int64_t n, int c0, int c1, const int32_t* vstart,
                            int64_t vmin, int64_t vcount, const DevPred* staged_preds,
                            const int32_t* staged_order, int nq, DevPred* preds_out, int32_t* order_out,
                            int64_t* iv, uint64_t* gthr, const int32_t* slots_src, int32_t* slots_dst,
                            int64_t n_slots, hipStream_t s) {
  intervals_kernel<<<dim3(2 * nq), dim3(64), 0, s>>>(attrs_phys, n, c0, c1, vstart, vmin, vcount, staged_preds,
                                                     staged_order, nq, preds_out, order_out, iv, gthr, slots_src,
                                                     slots_dst, n_slots);
  return hipGetLastError();
}

}  // namespace ifvs
