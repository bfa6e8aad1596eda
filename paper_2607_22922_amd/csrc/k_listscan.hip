// Rank and Select stages (Section 2, stages 2 and 3) in coarse-list order:
// the same distances and the same top k as the interval scan, with rows that
// cannot enter the top k skipped before their codes are read.
//
// The index keeps a second copy of its codes grouped by coarse centroid and
// radius band (sub-lists; each in layout order, so the rows of a query's
// layout interval are one run of positions per sub-list).  The list plan
// gives each query its sub-lists that hold selected rows (items) in
// increasing order of lb, a lower bound on the distance of every row of the
// item.  A query's work is the concatenation of its items' tiles up to the
// first item that the plan's seed bound prunes; the job table splits it into
// up to kListJobs chunks of about kJobTiles tiles or more (the queries with
// the most tiles first) and a persistent grid of workgroups takes the jobs
// from a counter, so a query with many tiles no longer holds the batch up.
// In a job the kScanWaves wavefronts share the chunk by position (wavefront
// w takes the positions congruent to w mod kScanWaves), so each row is scored
// by exactly one wavefront whatever each one skips.  A wavefront stops at the first item
// (or in the middle of one) whose lb^2 * keep - abs exceeds its current k-th
// distance: every later item has a bound at least as large.  lb^2 * keep -
// abs never exceeds the computed distance of a row of the item (the
// rounding allowances of the bound), so a skipped row is one whose distance
// exceeds the cut and the top k is unchanged.  (A bound per row, from each
// row's own radius, prunes about a quarter of the rows the items leave at
// 50% selectivity on 10M x 48-byte codes, but costs more than it saves.)
//
// Per tile the work is the interval scan's: sum of M table entries in
// groups of subspaces with early abandonment, candidates into per-wavefront
// pools of row keys resolved to original ids at compaction, thresholds
// shared through LDS and a per-query global word.
//
// Query-wide union bound (k <= kListSlots): a wavefront's own k-th key is loose
// while it has seen only a tile or two of the nearest lists, so each
// wavefront also keeps its two smallest full distances (two distinct rows)
// in the query's global slots (one per wavefront of each job), both in one
// 8-byte word stored whole (a reader never sees one new and one old value,
// which could show one row twice); the wavefronts scan disjoint rows, so the
// k-th smallest of the kListSlots values is the distance of one of k distinct rows at or below it, a bound
// on the query's k-th distance (published like a threshold, with the
// largest id so rows at that distance stay eligible).
#include <algorithm>
#include <climits>
#include <map>
#include <mutex>
#include <tuple>

#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

__device__ __forceinline__ float widen(float v) { return v; }
__device__ __forceinline__ float widen(__half v) { return __half2float(v); }

// Bits [lo, hi) of a 64-bit word, 0 <= lo < hi <= 64.
__device__ __forceinline__ uint64_t bit_range(int lo, int hi) {
  const uint64_t upto_hi = hi >= 64 ? ~0ull : ((1ull << hi) - 1);
  return upto_hi & ~((1ull << lo) - 1);
}

// Two register sets of ceil(M/4) code words each, and a subspace group's
// addresses and entries: M = 120 needs the register file of two waves per
// SIMD.
template <int MT, typename LutT>
constexpr int list_waves_per_eu() {
  return MT == 120 ? 2 : 4;
}

// kCount: a measurement build that also counts the table reads by active
// lanes (entries 1..64 of a.lookup_hist) and the code tiles summed (entry 0).
// kDepth register sets: the tiles of kDepth - 1 of them are in flight while
// one is summed.
//
// Persistent: as many workgroups as the chip holds at once take jobs from a
// global counter (the job table lists the heaviest queries first).  Job
// (pos, c, p0, p1): chunk c of the query at position pos, the positions
// [p0, p1) of its items' concatenated tiles; wavefront w takes the positions
// congruent to w mod kScanWaves.  Each (job, wavefront) has its own partial
// list ([pos][c][wave][k]) and union-bound word ([q][c * kScanWaves + wave]).
//
// A tile's code words are fetched in two parts: the words of the first
// kPreGroups groups of subspaces ahead of time (the ring below), the rest
// only when a row is still live after those groups (on 10M x 48-byte codes
// at 10% and 50% selectivity, 86% of the tiles lose every row within the
// first two groups of eight subspaces and 97% within three, and fetching
// every tile's 48 bytes a row was most of the kernel's fabric traffic).
template <int MT, typename LutT, bool kCount = false, int kDepth = 2, int kPreGroups = kListPreGroups>
__global__ __launch_bounds__(kScanWaves * 64) __attribute__((amdgpu_waves_per_eu(list_waves_per_eu<MT, LutT>())))
void list_scan_kernel(const ListScanArgs a) {
  constexpr int kMW = (MT + 3) / 4;
  constexpr int kGroup = MT % 8 == 0 && MT > 16 ? 8 : (MT % 4 == 0 ? 4 : MT);
  constexpr int kPre = (kPreGroups * kGroup + 3) / 4 < kMW ? (kPreGroups * kGroup + 3) / 4 : kMW;   // words fetched ahead
  constexpr int kRest = kMW - kPre;
  static_assert(kRest == 0 || (kPre * 4) % kGroup == 0, "the words fetched ahead end on a group");
  constexpr int kThreads = kScanWaves * 64;
  constexpr int kVec = 16 / sizeof(LutT);
  constexpr int kVecQ = MT * kKsub / kVec;
  __shared__ __align__(16) LutT s_lut[MT * kKsub];
  __shared__ int4 s_job;
  extern __shared__ __align__(16) unsigned char smem[];
  int4* s_item = reinterpret_cast<int4*>(smem);                       // [kScanWaves][64] (r0, r1, first, end)
  int2* s_item2 = reinterpret_cast<int2*>(s_item + kScanWaves * 64);  // [kScanWaves][64] (tile base, bound test)
  uint64_t* pools = reinterpret_cast<uint64_t*>(s_item2 + kScanWaves * 64);
  unsigned long long* s_thr = reinterpret_cast<unsigned long long*>(pools + kScanWaves * a.pool_stride);
  uint32_t* s_bad = reinterpret_cast<uint32_t*>(s_thr + 1);
  uint32_t* s_hist = s_bad + kScanWaves;   // [kReadHistEntries], counting build only

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int k = a.k;
  if constexpr (kCount) {
    if (threadIdx.x < kReadHistEntries) s_hist[threadIdx.x] = 0;
  }
  int cur_q = -1;
  bool monotone = true;
  uint64_t* pool = pools + static_cast<size_t>(wave) * a.pool_stride;
  const int total_jobs = *a.job_total;

  for (;;) {
    __syncthreads();   // every wavefront is done with the previous job's table and job record
    if (threadIdx.x == 0) {
      const int j = atomicAdd(a.job_next, 1);
      s_job = j < total_jobs ? a.jobs[j] : make_int4(-1, 0, 0, 0);
    }
    __syncthreads();
    const int4 job = s_job;
    const int pos = __builtin_amdgcn_readfirstlane(job.x);
    if (pos < 0) break;
    const int c = __builtin_amdgcn_readfirstlane(job.y);
    const int p_begin = __builtin_amdgcn_readfirstlane(job.z);
    const int p_end = __builtin_amdgcn_readfirstlane(job.w);
    const int q = __builtin_amdgcn_readfirstlane(a.qorder[pos]);
    if (q != cur_q) {
      // The query's table into LDS, noting negative or NaN entries (then
      // partial sums bound nothing: no abandonment and no skipping).
      const uint4* src =
          reinterpret_cast<const uint4*>(static_cast<const LutT*>(a.lut) + static_cast<size_t>(q) * MT * kKsub);
      bool bad = false;
      for (int v = threadIdx.x; v < kVecQ; v += kThreads) {
        const uint4 x = src[v];
        reinterpret_cast<uint4*>(s_lut)[v] = x;
        const LutT* xe = reinterpret_cast<const LutT*>(&x);
#pragma unroll
        for (int e = 0; e < kVec; ++e) bad = bad || !(widen(xe[e]) >= 0.0f);
      }
      const bool wave_bad = __ballot(bad) != 0;
      if (lane == 0) s_bad[wave] = wave_bad ? 1u : 0u;
      if (threadIdx.x == 0) *s_thr = kNoKey;
      __syncthreads();
      bool mono = true;
#pragma unroll
      for (int w = 0; w < kScanWaves; ++w) mono = mono && s_bad[w] == 0;
      monotone = __builtin_amdgcn_readfirstlane(mono ? 1 : 0) != 0;
      cur_q = q;
    }
    const float* hdr = a.hdr + 4 * static_cast<size_t>(q);
    const int n_items = __float_as_int(hdr[0]);

    int cnt = 0;
    uint64_t thr = kNoKey, published = kNoKey, bound = kNoKey;
    uint64_t gview = __hip_atomic_load(a.gthr + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float cut = __builtin_nanf("");
    // bound = min(own k-th key, workgroup's, query's); cut its distance (NaN
    // while there is none, or when the table is not monotone).
    // (every lane holds the same three values; taking lane 0's tells the
    // compiler so, which keeps the tile walk's state and branches scalar)
    auto refresh = [&]() {
      const uint64_t blk = __hip_atomic_load(s_thr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      uint64_t b = thr < blk ? thr : blk;
      b = b < gview ? b : gview;
      bound = (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32))))
               << 32) |
              static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b)));
      cut = monotone ? from_ordered_bits(static_cast<uint32_t>(bound >> 32)) : __builtin_nanf("");
    };
    refresh();

    // The item holding position p_begin: the last with tile offset <= p_begin
    // (offsets increase), by 64-way search.
    const size_t ib = static_cast<size_t>(q) * a.C;
    int item0 = 0;
    if (n_items > 0) {
      int lo = 0, hi = n_items;
      while (hi - lo > 64) {
        const int step = (hi - lo + 63) / 64;
        const int idx = min(lo + lane * step, hi - 1);
        const bool le = lo + lane * step < hi && a.it_t[ib + idx] <= p_begin;
        const uint64_t m = __ballot(le);
        const int l = 63 - __builtin_clzll(m | 1ull);
        lo = lo + l * step;
        hi = min(hi, lo + step);
      }
      const int idx = min(lo + lane, hi - 1);
      const bool le = lo + lane < hi && a.it_t[ib + idx] <= p_begin;
      item0 = lo + (63 - __builtin_clzll(__ballot(le) | 1ull));
    }

    // Tile generator over the job's items.  A batch of 64 items is read one
    // item a lane; what a wavefront needs of each item is kept in its LDS
    // rows (an item's start reads them back), so no per-lane register is
    // carried along the tile loop.
    int batch = item0 - 64;
    int stop_at = n_items;   // items from here on are prunable or past the job
    uint64_t pend = 0;
    bool in_item = false;
    int i_r0 = 0, i_r1 = 0, i_end = 0, i_tb = 0, p = 0;
    float i_lbv = 0.0f;   // the item's lb^2 * keep - abs (-inf when lb is not positive)
    int4* my_items = s_item + wave * 64;
    int2* my_items2 = s_item2 + wave * 64;
    auto next_tile = [&](int& t, uint64_t& mask) -> bool {
      for (;;) {
        if (in_item) {
          if (i_lbv > cut) {
            // this item and every later one
            stop_at = 0;
            pend = 0;
            in_item = false;
            return false;
          }
          if (p < i_end) {
            t = i_tb + p;
            p += kScanWaves;
            const int row0 = t * 64;
            mask = bit_range(max(i_r0 - row0, 0), min(i_r1 - row0, 64));
            return true;
          }
          in_item = false;
        }
        if (pend == 0) {
          batch += 64;
          if (batch >= stop_at) return false;
          // Every lane loads (lanes past the end reload the batch's first
          // item) and uses what it loaded before the ballot.
          const int it = batch + lane;
          const int itc = it < stop_at ? it : batch;
          const int v_r0 = a.it_r0[ib + itc];
          const int v_r1 = a.it_r1[ib + itc];
          const int v_t = a.it_t[ib + itc];
          const float v_lb = a.it_lb[ib + itc];
          const int nt = ((v_r1 - 1) >> 6) - (v_r0 >> 6) + 1;
          const int from = max(v_t, p_begin);
          const int first = from + ((wave - from) & (kScanWaves - 1));   // this wavefront's first position
          const int end = min(v_t + nt, p_end);
          const float lbv = v_lb > 0.0f ? __fsub_rn(__fmul_rn(__fmul_rn(v_lb, v_lb), a.keep), a.abs_m)
                                        : -__builtin_inff();
          const bool gone = it < stop_at && (lbv > cut || v_t >= p_end);
          bool ok = it < stop_at && first < end && !gone;
          my_items[lane] = make_int4(v_r0, v_r1, first, end);
          my_items2[lane] = make_int2((v_r0 >> 6) - v_t, __float_as_int(lbv));
          const uint64_t gm = __ballot(gone);
          if (gm != 0) {
            // the first prunable item, or the first past the job, ends it
            const int j0 = __builtin_ctzll(gm);
            stop_at = batch + j0;
            ok = ok && lane < j0;
          }
          pend = __ballot(ok);
          continue;
        }
        const int j = __builtin_ctzll(pend);
        pend &= pend - 1;
        const int4 x = my_items[j];
        const int2 y = my_items2[j];
        i_r0 = __builtin_amdgcn_readfirstlane(x.x);
        i_r1 = __builtin_amdgcn_readfirstlane(x.y);
        p = __builtin_amdgcn_readfirstlane(x.z);
        i_end = __builtin_amdgcn_readfirstlane(x.w);
        i_tb = __builtin_amdgcn_readfirstlane(y.x);
        i_lbv = __int_as_float(__builtin_amdgcn_readfirstlane(y.y));
        in_item = true;
      }
    };
    auto load = [&](int t, uint32_t (&w)[kPre]) {
      const uint32_t* __restrict__ tile = a.codes_t + static_cast<size_t>(t) * (kMW * 64);
#pragma unroll
      for (int j = 0; j < kPre; ++j) w[j] = tile[j * 64 + lane];
    };
    const bool union_bound = a.union_bound != 0 && k <= kListSlots;
    unsigned long long* pairs = reinterpret_cast<unsigned long long*>(a.slots + static_cast<size_t>(q) * kListSlots);
    const int my_pair = c * kScanWaves + wave;
    uint32_t best1 = ~0u, best2 = ~0u;   // this wavefront's two smallest full distances in this job
    auto publish = [&](uint64_t key) {
      if (key < published) {
        published = key;
        if (lane == 0) {
          atomicMin(s_thr, static_cast<unsigned long long>(key));
          __hip_atomic_fetch_min(a.gthr + q, key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    };
    auto consider = [&](bool act, float d, int t) {
      uint64_t key = kNoKey;
      bool cand = false;
      if (act) {
        const uint32_t db = ordered_bits(d);
        if (db <= static_cast<uint32_t>(bound >> 32)) {
          key = row_key(db, static_cast<uint32_t>(t * 64 + lane));
          cand = true;
        }
      }
      if (union_bound) {
        // The step's two smallest distances (pairs merged across lanes), then
        // the wavefront's two smallest so far.
        uint32_t x1 = act ? ordered_bits(d) : ~0u, x2 = ~0u;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y1 = static_cast<uint32_t>(__shfl_xor(static_cast<int>(x1), o, 64));
          const uint32_t y2 = static_cast<uint32_t>(__shfl_xor(static_cast<int>(x2), o, 64));
          const uint32_t hi = x1 > y1 ? x1 : y1;
          const uint32_t lo2 = x2 < y2 ? x2 : y2;
          x1 = x1 < y1 ? x1 : y1;
          x2 = hi < lo2 ? hi : lo2;
        }
        const uint32_t hi = best1 > x1 ? best1 : x1;
        const uint32_t lo2 = best2 < x2 ? best2 : x2;
        const uint32_t n1 = best1 < x1 ? best1 : x1;
        const uint32_t n2 = hi < lo2 ? hi : lo2;
        if (n1 < best1 || n2 < best2) {
          // The k-th smallest slot only falls when a slot drops from at or
          // above the published value to below it.
          const uint32_t kth = static_cast<uint32_t>(published >> 32);
          const bool crossed = (n1 < kth && best1 >= kth) || (n2 < kth && best2 >= kth);
          best1 = n1;
          best2 = n2;
          if (lane == 0)
            __hip_atomic_store(&pairs[my_pair], (static_cast<unsigned long long>(n2) << 32) | n1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
          if (crossed) {
            // all kListSlots / 2 words are loaded (the unused ones hold all
            // ones), together, with one wait; each lane reads its own words
            constexpr int kW = kListSlots / 128;
            unsigned long long pw[kW];
#pragma unroll
            for (int u = 0; u < kW; ++u)
              pw[u] = __hip_atomic_load(&pairs[lane * kW + u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            uint64_t v[2 * kW];
#pragma unroll
            for (int u = 0; u < kW; ++u) {
              v[2 * u] = (static_cast<uint64_t>(static_cast<uint32_t>(pw[u])) << 32) | 0xFFFFFFFFull;
              v[2 * u + 1] = (static_cast<uint64_t>(static_cast<uint32_t>(pw[u] >> 32)) << 32) | 0xFFFFFFFFull;
            }
            wave_bitonic_sort<2 * kW>(v);
            const int e = k - 1;
            uint64_t mine = v[0];
#pragma unroll
            for (int u = 1; u < 2 * kW; ++u)
              if (u == e % (2 * kW)) mine = v[u];
            const uint64_t ub = shfl_u64(mine, e / (2 * kW));
            if ((ub >> 32) != 0xFFFFFFFFull) publish(ub);
          }
        }
      }
      pool_push(pool, cnt, thr, key, cand, k, a.kpl, a.ids);
      publish(thr);
    };
    auto sum_tile = [&](int t, uint64_t mask, const uint32_t (&w)[kPre]) {
      if constexpr (kCount) {
        if (lane == 0) atomicAdd(&s_hist[0], 1u);
      }
      uint64_t live = mask;   // live lanes, as a wavefront-wide mask
      float d = 0.0f;
      uint32_t rest[kRest > 0 ? kRest : 1];
      // (most tiles lose every row to the first groups: the loop ends as soon
      // as no lane is live)
#pragma unroll
      for (int gr = 0; gr < MT / kGroup; ++gr) {
        if (live == 0) break;
        if constexpr (kRest > 0) {
          if (gr * kGroup == kPre * 4) {
            // a row is live past the words fetched ahead: the rest of the tile
            if constexpr (kCount) {
              if (lane == 0) atomicAdd(&s_hist[65], 1u);
            }
            const uint32_t* __restrict__ tile = a.codes_t + static_cast<size_t>(t) * (kMW * 64);
#pragma unroll
            for (int j = 0; j < kRest; ++j) rest[j] = tile[(kPre + j) * 64 + lane];
          }
        }
        int addr[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
          const int m = gr * kGroup + u;
          const uint32_t word = (m >> 2) < kPre ? w[m >> 2] : rest[(m >> 2) - kPre];
          addr[u] = m * kKsub + static_cast<int>((word >> (8 * (m & 3))) & 0xFFu);
        }
        if constexpr (kCount) {
          if (lane == 0) atomicAdd(&s_hist[__popcll(live)], static_cast<uint32_t>(kGroup));
        }
        if (__builtin_amdgcn_inverse_ballot_w64(live)) {
          LutT v[kGroup];
#pragma unroll
          for (int u = 0; u < kGroup; ++u) v[u] = s_lut[addr[u]];
#pragma unroll
          for (int u = 0; u < kGroup; ++u) d = __fadd_rn(d, widen(v[u]));
        }
        live &= __ballot(!(d > cut));
      }
      if (live != 0) consider(__builtin_amdgcn_inverse_ballot_w64(live), d, t);
    };

    // Register sets in a ring: step i refills the set summed in the step
    // before with the next tile, then sums set i.  Tiles come in generation
    // order, so the first set without one ends the job.  The loads are
    // issued on every path (tile 0 stands in when there is no next tile, in
    // bounds and unused), so the compiler's wait counts never make a sum wait
    // for the tile loaded after it.  The bound is refreshed once per round
    // of kDepth tiles (a bound a few tiles old is looser, never wrong).
    uint32_t ws[kDepth][kPre];
    int ts[kDepth];
    uint64_t ms[kDepth];
    bool hs[kDepth];
#pragma unroll
    for (int i = 0; i < kDepth; ++i) {
      ts[i] = 0;
      ms[i] = 0;
      hs[i] = false;
    }
#pragma unroll
    for (int i = 0; i < kDepth - 1; ++i) {
      hs[i] = next_tile(ts[i], ms[i]);
      load(hs[i] ? ts[i] : 0, ws[i]);
    }
    for (;;) {
      // The query's shared threshold is loaded at the top of a round and
      // read at its end, when the tile loads issued after it have been waited
      // for anyway (read at the next round's top, its wait also held back
      // the round's first tile loads).
      const uint64_t gload = __hip_atomic_load(a.gthr + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
      for (int i = 0; i < kDepth; ++i) {
        const int j = (i + kDepth - 1) % kDepth;
        hs[j] = next_tile(ts[j], ms[j]);
        load(hs[j] ? ts[j] : 0, ws[j]);
        if (!hs[i]) goto scanned;
        sum_tile(ts[i], ms[i], ws[i]);
      }
      gview = gload;
      refresh();
    }
  scanned:
    pool_compact(pool, cnt, thr, k, a.kpl, a.ids);
    uint64_t* dst = a.partials + ((static_cast<size_t>(pos) * a.max_jobs + c) * kScanWaves + wave) * k;
    for (int e = lane; e < k; e += 64) dst[e] = pool[e];
  }
  if constexpr (kCount) {
    __syncthreads();
    if (threadIdx.x < kReadHistEntries && s_hist[threadIdx.x] != 0)
      atomicAdd(&a.lookup_hist[threadIdx.x], static_cast<unsigned long long>(s_hist[threadIdx.x]));
  }
}


template <int MT>
const void* pick_list_t(int lut_dtype, bool count) {
  if (count)
    return lut_dtype == 1 ? reinterpret_cast<const void*>(&list_scan_kernel<MT, __half, true>)
                          : reinterpret_cast<const void*>(&list_scan_kernel<MT, float, true>);
  return lut_dtype == 1 ? reinterpret_cast<const void*>(&list_scan_kernel<MT, __half>)
                        : reinterpret_cast<const void*>(&list_scan_kernel<MT, float>);
}

const void* pick_list(int m, int lut_dtype, bool count) {
  switch (m) {
    case 16: return pick_list_t<16>(lut_dtype, count);
    case 48: return pick_list_t<48>(lut_dtype, count);
    case 120: return pick_list_t<120>(lut_dtype, count);
    default: return nullptr;
  }
}

size_t list_dyn_bytes(int pool_stride) {
  // item rows, pools, the workgroup threshold, monotonicity flags, the
  // counting build's histogram
  return static_cast<size_t>(kScanWaves) * 64 * (sizeof(int4) + sizeof(int2)) +
         static_cast<size_t>(kScanWaves) * pool_stride * sizeof(uint64_t) + 8 + 4 * kScanWaves + kLookupHistBytes;
}

}  // namespace

bool list_scan_supported(int m, int lut_dtype) { return pick_list(m, lut_dtype, false) != nullptr; }

size_t list_scan_lds_bytes(int m, int lut_dtype, int pool_stride) {
  return static_cast<size_t>(m) * kKsub * (lut_dtype == 1 ? 2 : 4) + list_dyn_bytes(pool_stride);
}

hipError_t launch_list_scan(const ListScanArgs& a, int lut_dtype, hipStream_t s) {
  const void* fn = pick_list(a.m, lut_dtype, a.lookup_hist != nullptr);
  if (!fn) return hipErrorInvalidValue;
  if (a.nq <= 0) return hipSuccess;
  const size_t dyn = list_dyn_bytes(a.pool_stride);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(dyn));
  if (e != hipSuccess) return e;
  // Persistent: the workgroups the chip holds at once (looked up once per
  // device, kernel and LDS size).
  int device = 0;
  if ((e = hipGetDevice(&device)) != hipSuccess) return e;
  int grid = 0;
  {
    static std::mutex mu;
    static std::map<std::tuple<int, const void*, size_t>, int> cache;
    std::lock_guard<std::mutex> lock(mu);
    const auto key = std::make_tuple(device, fn, dyn);
    auto it = cache.find(key);
    if (it == cache.end()) {
      int cus = 0, per_cu = 0;
      if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device)) != hipSuccess) return e;
      if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kScanWaves * 64, dyn)) != hipSuccess)
        return e;
      it = cache.emplace(key, std::max(1, cus * std::max(1, per_cu))).first;
    }
    grid = it->second;
  }
  ListScanArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchKernel(fn, dim3(static_cast<unsigned>(grid)), dim3(kScanWaves * 64), kargs, dyn, s);
}

}  // namespace ifvs
