// Device pieces of the per-query row intervals on the clustered layout
// (the Filter stage of Section 2 over rows stored in cluster-key order),
// shared by the interval kernel and the predicate encoder (which computes
// the intervals of the batch it encodes in workgroups of the same launch).
// A wavefront finds one bound of one query; no workgroup barrier is used, so
// the wavefronts of a workgroup may each take a different query.
#pragma once

#include "ifvs_internal.h"

namespace ifvs {

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
__device__ inline int64_t wave_lower_bound(const int32_t* __restrict__ a0, const int32_t* __restrict__ a1,
                                           int64_t lo, int64_t hi, int64_t x0, int64_t x1) {
  const int lane = threadIdx.x & 63;
  while (hi - lo > 64) {
    const int64_t step = (hi - lo + 63) / 64;
    const int64_t r = lo + lane * step;  // probes lo, lo+step, ... (< hi or past it)
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

// Words [worker * 64, ...) of the scan's dispatch order, strided by all
// n_workers wavefronts, from the staging slot to the device.
__device__ __forceinline__ void copy_slot_order(const IntervalArgs& a, int64_t worker, int64_t n_workers, int lane) {
  for (int64_t i = worker * 64 + lane; i < a.n_slots; i += n_workers * 64) a.slots_dst[i] = a.slots_src[i];
}

// Field of the predicate held one dword per lane (pw = dword `lane`).
#define IFVS_IV_WORD(field) static_cast<int>(offsetof(DevPred, field) / 4)
__device__ __forceinline__ int32_t pred_i32(uint32_t pw, int word) {
  return __builtin_amdgcn_readlane(static_cast<int>(pw), word);
}
__device__ __forceinline__ int64_t pred_i64(uint32_t pw, int word) {
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(pw), word));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(pw), word + 1));
  return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// The lower (upper = false) or upper bound of query q's interval; the lower
// bound's wavefront also leaves the device copies of the predicate and the
// scan order and resets the query's threshold.
__device__ inline void interval_bound(const IntervalArgs& a, int q, bool upper, int lane) {
  constexpr int kWords = static_cast<int>(sizeof(DevPred) / 4);
  static_assert(sizeof(DevPred) % 4 == 0 && kWords <= 64 && offsetof(DevPred, iv_lo0) % 4 == 0,
                "one dword per lane");
  const uint32_t pw = lane < kWords ? reinterpret_cast<const uint32_t*>(a.staged_preds + q)[lane] : 0u;
  if (!upper) {
    if (lane < kWords) reinterpret_cast<uint32_t*>(a.preds_out + q)[lane] = pw;
    if (lane == 0) a.order_out[q] = a.staged_order[q];
  }
  const int n_eff = pred_i32(pw, IFVS_IV_WORD(n_eff));
  const int iv_mode = pred_i32(pw, IFVS_IV_WORD(iv_mode));
  int64_t r = upper ? a.n : 0;
  if (n_eff < 0) {
    r = 0;
  } else if (iv_mode == 1) {
    const int64_t x = pred_i64(pw, upper ? IFVS_IV_WORD(iv_hi0) : IFVS_IV_WORD(iv_lo0));
    if (a.vstart) {
      r = table_lower_bound(a.vstart, a.vmin, a.vcount, a.n, x);
    } else {
      const int32_t* a0 = a.attrs_phys + static_cast<int64_t>(a.c0) * a.n;
      r = wave_lower_bound(a0, nullptr, 0, a.n, x, 0);
    }
  } else if (iv_mode == 2) {
    // Leading key equal to iv_lo0, second key in [iv_lo1, iv_hi1): the value
    // table (when present) gives the rows of that leading key, the search
    // runs inside them.
    const int64_t lo0 = pred_i64(pw, IFVS_IV_WORD(iv_lo0));
    const int64_t x1 = pred_i64(pw, upper ? IFVS_IV_WORD(iv_hi1) : IFVS_IV_WORD(iv_lo1));
    const int32_t* a0 = a.attrs_phys + static_cast<int64_t>(a.c0) * a.n;
    const int32_t* a1 = a.attrs_phys + static_cast<int64_t>(a.c1) * a.n;
    int64_t lo = 0, hi = a.n;
    if (a.vstart) {
      lo = table_lower_bound(a.vstart, a.vmin, a.vcount, a.n, lo0);
      hi = table_lower_bound(a.vstart, a.vmin, a.vcount, a.n, lo0 + 1);
    }
    r = wave_lower_bound(a0, a1, lo, hi, lo0, x1);
  }
  if (lane == 0) {
    a.iv[2 * q + (upper ? 1 : 0)] = r;
    if (!upper) a.gthr[q] = ~0ull;
  }
}
#undef IFVS_IV_WORD

}  // namespace ifvs
