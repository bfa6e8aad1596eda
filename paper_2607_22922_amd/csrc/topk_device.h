// Wavefront-level top-k selection on 64-bit keys, shared by the scan and the
// merge kernels.
//
// A key is (order-preserving bits of the fp32 distance) << 32 | vector id, so
// ascending keys are ascending (distance, id): ties go to the smaller id
// (the Select stage of Section 2 returns the k best; equal distances are
// ordered by id so the answer is unique).  The all-ones key is "no result".
//
// Each (wavefront, query) owns a candidate pool in LDS of 64*kpl >= k + 64
// keys (a power of two) and a
// threshold: the k-th smallest key seen so far (all-ones until k keys were
// seen).  Lanes whose key beats the threshold are appended with one ballot
// and a prefix count; when an append would overflow, the pool is sorted with
// a register bitonic sort across the wavefront and cut back to its k
// smallest keys, which also tightens the threshold.
//
// On a clustered index rows are stored in a permuted order and a key must
// carry the original id (ties break by it).  Looking the id up when a row
// becomes a candidate would put a dependent global load on the scan's path,
// so candidates enter the pool as row keys -- the physical row with
// kRowFlag set in the id field -- and the ids are looked up in `perm` when
// the pool is compacted, once for all of them.  A row key only knows its
// distance, so it is offered whenever its distance does not exceed the
// threshold's; compaction then decides ties by the real id.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace ifvs {

constexpr uint64_t kNoKey = ~0ull;

__device__ __forceinline__ uint32_t ordered_bits(float d) {
  const uint32_t u = __float_as_uint(d);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_ordered_bits(uint32_t t) {
  const uint32_t u = (t & 0x80000000u) ? (t & 0x7fffffffu) : ~t;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t make_key(float d, uint32_t id) {
  return (static_cast<uint64_t>(ordered_bits(d)) << 32) | id;
}

// Id field of a row key: a physical row (< 2^31) still to be mapped to its
// original id through perm.
constexpr uint32_t kRowFlag = 0x80000000u;

__device__ __forceinline__ uint64_t row_key(uint32_t dist_bits, uint32_t row) {
  return (static_cast<uint64_t>(dist_bits) << 32) | kRowFlag | row;
}

// The key with its id field resolved (keys that are not row keys unchanged).
__device__ __forceinline__ uint64_t resolve_key(uint64_t key, const int32_t* __restrict__ perm) {
  if (key == ~0ull || !(static_cast<uint32_t>(key) & kRowFlag)) return key;
  const uint32_t row = static_cast<uint32_t>(key) & ~kRowFlag;
  return (key & 0xFFFFFFFF00000000ull) | static_cast<uint32_t>(perm[row]);
}

// May `key` still belong below `thr`?  Exact for resolved keys; a row key
// is compared by distance only.
__device__ __forceinline__ bool may_beat(uint64_t key, uint64_t thr, bool row_keys) {
  return row_keys ? (key >> 32) <= (thr >> 32) : key < thr;
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Number of set bits of `mask` in lanes below this one.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0));
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  const int lo = __shfl_xor(static_cast<int>(static_cast<uint32_t>(v)), mask, 64);
  const int hi = __shfl_xor(static_cast<int>(static_cast<uint32_t>(v >> 32)), mask, 64);
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const int lo = __shfl(static_cast<int>(static_cast<uint32_t>(v)), src, 64);
  const int hi = __shfl(static_cast<int>(static_cast<uint32_t>(v >> 32)), src, 64);
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}

// Ascending bitonic sort of 64*KPL keys held KPL per lane; element e of the
// sequence is slot e % KPL of lane e / KPL.  Pairs closer than KPL are
// exchanged inside a lane, farther pairs across lanes with a shuffle.
template <int KPL>
__device__ __forceinline__ void wave_bitonic_sort(uint64_t (&v)[KPL]) {
  const int lane = lane_id();
#pragma unroll
  for (int size = 2; size <= 64 * KPL; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= KPL) {
        const int lstride = stride / KPL;
#pragma unroll
        for (int s = 0; s < KPL; ++s) {
          const int e = lane * KPL + s;
          const uint64_t o = shfl_xor_u64(v[s], lstride);
          const bool up = (e & size) == 0;
          const bool lower = (e & stride) == 0;
          const uint64_t mn = v[s] < o ? v[s] : o;
          const uint64_t mx = v[s] < o ? o : v[s];
          v[s] = (lower == up) ? mn : mx;
        }
      } else {
#pragma unroll
        for (int s = 0; s < KPL; ++s) {
          if (s & stride) continue;
          const int s2 = s | stride;
          const int e = lane * KPL + s;
          const bool up = (e & size) == 0;
          const uint64_t a = v[s], b = v[s2];
          const bool swap = up ? (a > b) : (a < b);
          v[s] = swap ? b : a;
          v[s2] = swap ? a : b;
        }
      }
    }
  }
}

// Sort the first `cnt` keys of `pool`, keep the k smallest in pool[0..k)
// (padded with kNoKey), and set the threshold once k keys exist.  Pools of
// up to 256 keys are sorted in registers (KPL keys per lane).
template <int KPL>
__device__ __forceinline__ uint64_t pool_compact_regs(uint64_t* pool, int cnt, uint64_t thr, int k,
                                                      const int32_t* perm) {
  const int lane = lane_id();
  uint64_t v[KPL];
#pragma unroll
  for (int s = 0; s < KPL; ++s) {
    const int e = lane * KPL + s;
    v[s] = e < cnt ? pool[e] : kNoKey;
  }
  if (perm) {
#pragma unroll
    for (int s = 0; s < KPL; ++s) v[s] = resolve_key(v[s], perm);
  }
  wave_bitonic_sort<KPL>(v);
#pragma unroll
  for (int s = 0; s < KPL; ++s) {
    const int e = lane * KPL + s;
    if (e < k) pool[e] = v[s];
  }
  if (cnt >= k) {
    const int e = k - 1;
    const int slot = e % KPL;
    uint64_t mine = v[0];
#pragma unroll
    for (int s = 1; s < KPL; ++s)
      if (s == slot) mine = v[s];
    thr = shfl_u64(mine, e / KPL);
  }
  return thr;
}

// Larger pools (64*kpl keys of LDS) are sorted in place: one compare-exchange
// per lane per step, the wavefront's LDS accesses ordered by fences.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ uint64_t pool_compact_lds(uint64_t* pool, int cnt, uint64_t thr, int k, int kpl,
                                                     const int32_t* perm) {
  const int lane = lane_id();
  const int n = 64 * kpl;
  if (perm)
    for (int e = lane; e < cnt; e += 64) pool[e] = resolve_key(pool[e], perm);
  for (int e = cnt + lane; e < n; e += 64) pool[e] = kNoKey;
  wave_lds_fence();
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = lane; p < n / 2; p += 64) {
        // p-th pair: lower index i has bit `stride` clear.
        const int i = ((p & ~(stride - 1)) << 1) | (p & (stride - 1));
        const int j = i | stride;
        const uint64_t a = pool[i], b = pool[j];
        const bool up = (i & size) == 0;
        if (up ? (a > b) : (a < b)) {
          pool[i] = b;
          pool[j] = a;
        }
      }
      wave_lds_fence();
    }
  }
  if (cnt >= k) thr = pool[k - 1];
  wave_lds_fence();
  return thr;
}

// Sort the pool, keep its k smallest keys first; returns the new threshold
// (the pool then holds min(cnt, k) keys).  Not inlined: compaction is rare,
// and one copy per kernel keeps the code small.
// Row keys (perm non-null) are resolved first.
__device__ __noinline__ uint64_t pool_compact_call(uint64_t* pool, int cnt, uint64_t thr, int k, int kpl,
                                                   const int32_t* perm) {
  if (kpl == 2) return pool_compact_regs<2>(pool, cnt, thr, k, perm);
  if (kpl == 4) return pool_compact_regs<4>(pool, cnt, thr, k, perm);
  return pool_compact_lds(pool, cnt, thr, k, kpl, perm);
}

__device__ __forceinline__ void pool_compact(uint64_t* pool, int& cnt, uint64_t& thr, int k, int kpl,
                                             const int32_t* perm = nullptr) {
  thr = pool_compact_call(pool, cnt, thr, k, kpl, perm);
  cnt = cnt < k ? cnt : k;
}

// Offer one key per lane (`cand` false = nothing to offer).  Must be called
// by every lane of the wavefront with the same pool, cnt and thr.  The pool
// holds 64*kpl >= k + 64 keys (a power of two).  perm non-null: the keys
// offered are row keys.
__device__ __forceinline__ void pool_push(uint64_t* pool, int& cnt, uint64_t& thr,
                                          uint64_t key, bool cand, int k, int kpl,
                                          const int32_t* perm = nullptr) {
  uint64_t mask = __ballot(cand);
  if (mask == 0) return;
  int n = __popcll(mask);
  if (cnt + n > k + 64) {
    pool_compact(pool, cnt, thr, k, kpl, perm);
    cand = cand && may_beat(key, thr, perm != nullptr);
    mask = __ballot(cand);
    if (mask == 0) return;
    n = __popcll(mask);
  }
  const int pos = cnt + lanes_below(mask);
  if (cand) pool[pos] = key;
  cnt += n;
}

}  // namespace ifvs
