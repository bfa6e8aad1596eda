// Rank stage (Section 2, stage 2) as an asymmetric-distance scan over the
// 8-bit PQ codes of the selected vectors, feeding the Select stage's
// per-wavefront candidate pools.
//
// For a candidate v of query q: dist(v) = sum_{m<M} LUT_q[m][code_v[m]],
// summed in m order from +0 with separately rounded fp32 additions.
//
// Workgroup = kScanWaves wavefronts; grid = (code chunks, query tiles).
//  * A query tile is QT queries (taken in the planner's order).  Each query
//    selects the rows of its interval [iv0, iv1) -- the whole index, or the
//    rows its cluster-key clauses select on a clustered index -- and, when
//    it has residual clauses, the rows set in its selection bitmap.  The
//    tile's chunk of work is a slice of the union of its intervals.
//  * The tables of the QT queries live in LDS as [m][qi][256] so that, once
//    a lane has turned its vector's M code bytes into M LDS addresses, the
//    same addresses serve every query of the tile (query qi adds a constant
//    qi*256 that folds into the instruction's offset field).
//  * Codes are stored in 64-row tiles ("word j of all 64 rows" contiguous),
//    so each of the ceil(M/4) dword loads of a wavefront reads 256
//    consecutive bytes; the next tile's words are loaded while the current
//    one is being summed.  A tile is loaded once for all QT queries, and a
//    tile no query selects is skipped without touching memory.
//  * Each lane whose row is selected sums its M table entries in groups and
//    drops out as soon as its partial sum exceeds the wavefront's current
//    k-th distance (all entries are squares times non-negative weights, so
//    partial sums only grow; checked per query when its table is staged).
//    Lanes beating the current k-th best key are appended to that query's
//    pool (ballot + prefix count), which is sorted and cut back to k keys
//    when it would overflow.  The "current k-th distance" is the smallest
//    valid bound known: the wavefront's own, the workgroup's and the
//    query's (shared through LDS and global atomics), the k-th smallest of
//    the wavefronts' two best distances (union bound), and a seed computed
//    before the scan from rows ranked by their first subspace group.  Keys carry original vector ids (on a clustered
//    layout looked up when a pool is compacted), so ties break by original id
//    on any layout.  At the end each
//    wavefront writes its k best keys per query; a merge kernel reduces them.
#include <climits>

#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

constexpr int kXcds = 8;   // accelerator complex dies of an MI355X

__device__ __forceinline__ float widen(float v) { return v; }
__device__ __forceinline__ float widen(__half v) { return __half2float(v); }

struct ScanArgs {
  const uint32_t* codes_t;
  int64_t n, n_tiles;
  int m, mw;
  const void* lut;
  int nq;
  int splits, n_qtiles;
  const int32_t* qorder;
  const int64_t* iv;
  const DevPred* preds;
  const uint64_t* bitmap;
  int64_t stride64;
  const int32_t* perm;
  int k, pool_stride, kpl, min_chunk;
  int64_t chunk_tiles;   // > 0: chunks on a grid of this many tiles (see below)
  int abs_cells;         // 1: chunk c is absolute grid cell c (all XCDs walk the same cells)
  uint64_t* partials;
  uint64_t* gthr;   // [nq] per original query: smallest k-th key any wavefront has published
  const int32_t* mode;   // [nq] 1: scored by the gather scan instead (null: none)
  // Dispatch order (null: index order): workgroup b scans item
  // slot_order[(b % kXcds) * per_xcd * splits + b / kXcds] of its XCD, item
  // c * per_xcd + t meaning chunk c of the XCD's t-th query tile.
  const int32_t* slot_order;
  int shared_bound;      // 1: wavefronts publish their best keys (union bound, k <= 16)
  int seed_tiles;        // > 0: seeded bound from up to this many tiles per wavefront (QT = 1, k <= 64)
  // Counting instantiation only: lookup_hist[n] += the table reads (one
  // per subspace and wavefront instruction) issued with n active lanes.
  unsigned long long* lookup_hist;
};

// Bits [lo, hi) of a 64-bit word, 0 <= lo < hi <= 64.
__device__ __forceinline__ uint64_t bit_range(int64_t lo, int64_t hi) {
  const uint64_t upto_hi = hi >= 64 ? ~0ull : ((1ull << hi) - 1);
  return upto_hi & ~((1ull << lo) - 1);
}

// Waves per SIMD that one-query workgroups can reach, set by their LDS
// (tables + pools, two or more workgroups of eight waves per CU): the
// register budget of a wave follows from it (512 / waves VGPRs), and the
// code pipeline takes as many tiles in flight as that budget holds.  The
// code stream is latency-bound otherwise: with one tile in flight per wave a
// CU has 16 x 3 KB outstanding and waits about 1 us for each.
template <int MT, int QT, typename LutT>
constexpr int scan_waves_per_eu() {
  if constexpr (QT != 1) return 1;
  else if constexpr (MT == 120 && sizeof(LutT) == 4) return 2;
  else if constexpr ((MT == 48 && sizeof(LutT) == 4) || MT == 120) return 4;
  else return 6;
}

// Register sets (tiles in flight + the one being summed) of the pipeline,
// chosen so that the kernel fits the register budget above without spills.
template <int MT, int QT, typename LutT>
constexpr int scan_depth() {
  if constexpr (QT != 1 || MT <= 0) return 2;
  else if constexpr (MT <= 16) return 3;
  else if constexpr (sizeof(LutT) == 4 && scan_waves_per_eu<MT, QT, LutT>() <= 4) return 4;
  else return 2;
}

// kCount: the same scan, also counting its table reads by active lanes in
// an LDS histogram flushed to a.lookup_hist, and in entry 0 the code tiles
// it sums (a measurement build: the counting adds LDS atomics, so it is
// never the timed kernel).
template <int MT, int QT, typename LutT, bool kCount = false>
__global__ __launch_bounds__(kScanWaves * 64) __attribute__((amdgpu_waves_per_eu(scan_waves_per_eu<MT, QT, LutT>())))
void scan_kernel(const ScanArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kMW = MT > 0 ? (MT + 3) / 4 : 1;
  // Subspaces summed between two early-abandonment checks (fixed M).
  constexpr int kGroup = MT % 8 == 0 && MT > 16 ? 8 : (MT % 4 == 0 ? 4 : MT);
  const int M = MT > 0 ? MT : a.m;
  // LDS: the tables, then (dynamic) the pools, the workgroup thresholds and
  // the monotonicity flags.  With M fixed at compile time the tables are a
  // static array at a known address: a table address is then the code byte
  // times the entry size (one shift with a byte select) plus a constant that
  // folds into the instruction's offset.
  LutT* slut;
  const size_t lut_bytes = static_cast<size_t>(M) * QT * kKsub * sizeof(LutT);
  uint64_t* pools;
  if constexpr (MT > 0) {
    __shared__ __align__(16) unsigned char s_lut[static_cast<size_t>(MT > 0 ? MT : 1) * QT * kKsub * sizeof(LutT)];
    slut = reinterpret_cast<LutT*>(s_lut);
    pools = reinterpret_cast<uint64_t*>(smem);
  } else {
    slut = reinterpret_cast<LutT*>(smem);
    pools = reinterpret_cast<uint64_t*>(smem + lut_bytes);
  }
  unsigned long long* s_thr = reinterpret_cast<unsigned long long*>(
      pools + static_cast<size_t>(kScanWaves) * QT * a.pool_stride);   // smallest k-th key published in this workgroup
  uint32_t* s_bad = reinterpret_cast<uint32_t*>(s_thr + QT);   // [wave][qi]: the wave saw a negative or NaN entry
  // [qi][wave]: each wavefront's two smallest distances (order-preserving
  // bits, the second in the high half) in one 8-byte word, stored whole so a
  // reader never sees one new and one old value (the area holds kScanPub
  // words per wavefront; the first is used)
  unsigned long long* s_pub = reinterpret_cast<unsigned long long*>(s_bad + kScanWaves * QT);
  // [wave][kScanSeed]: distances (order-preserving bits) of the seed candidates
  uint32_t* s_seed = reinterpret_cast<uint32_t*>(s_pub + QT * kScanWaves * kScanPub);
  // [65]: the counting build's histogram of table reads by active lanes
  uint32_t* s_hist = s_seed + kScanWaves * kScanSeed;
  auto count_reads = [&](uint64_t lanes, int reads) {
    if constexpr (kCount) {
      if (lanes != 0 && (threadIdx.x & 63) == 0) atomicAdd(&s_hist[__popcll(lanes)], static_cast<uint32_t>(reads));
    }
  };

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // XCD-aware grid.  The dispatcher deals workgroups round-robin to the 8
  // XCDs (workgroup b runs on XCD b % 8).  Each XCD gets a contiguous run of
  // query tiles -- the planner orders queries by interval, so neighbours
  // read nearly the same rows and share that XCD's L2 -- and walks it chunk
  // by chunk: chunk c of all its query tiles, then chunk c + 1, so every XCD
  // has work and empty chunks come last.
  const int xcd = blockIdx.x % kXcds;
  const int per_xcd = (a.n_qtiles + kXcds - 1) / kXcds;
  const int slot = a.slot_order ? a.slot_order[static_cast<int64_t>(xcd) * per_xcd * a.splits + blockIdx.x / kXcds]
                                : static_cast<int>(blockIdx.x / kXcds);
  const int chunk = slot / per_xcd;
  const int qtile = xcd * per_xcd + slot % per_xcd;
  if (qtile >= a.n_qtiles || chunk >= a.splits) return;   // grid padding
  const int q0 = qtile * QT;
  const int qn = min(QT, a.nq - q0);
  const int k = a.k;

  // The tile's queries.
  int qid[QT];
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) qid[qi] = qi < qn ? a.qorder[q0 + qi] : 0;

  // Their tables (global [q][m][c]).  With M fixed at compile time every
  // load of the staging is issued here, so the tables, the intervals below
  // and the first code tile are all in flight together; the words land in
  // LDS further down.
  constexpr int kThreads = kScanWaves * 64;
  constexpr int kVec = 16 / sizeof(LutT);
  constexpr int kVecQ = (MT > 0 ? MT : 1) * kKsub / kVec;   // 16-byte vectors per table
  constexpr int kLutPer = MT > 0 ? (kVecQ + kThreads - 1) / kThreads : 1;
  const LutT* lut = static_cast<const LutT*>(a.lut);
  uint4 lx[QT][kLutPer];
  if constexpr (MT > 0) {
#pragma unroll
    for (int qi = 0; qi < QT; ++qi) {
      if (qi >= qn) break;
      const uint4* src = reinterpret_cast<const uint4*>(lut + static_cast<size_t>(qid[qi]) * M * kKsub);
#pragma unroll
      for (int u = 0; u < kLutPer; ++u) {
        const int v = threadIdx.x + u * kThreads;
        if (kVecQ % kThreads == 0 || v < kVecQ) lx[qi][u] = src[v];
      }
    }
  }

  // Their row intervals, and the chunk of this workgroup.
  int64_t r0[QT], r1[QT];
  bool resid[QT];
  int64_t hull_lo = INT64_MAX, hull_hi = 0;
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    r0[qi] = r1[qi] = 0;
    resid[qi] = false;
    if (qi < qn) {
      r0[qi] = a.iv[2 * qid[qi]];
      r1[qi] = a.iv[2 * qid[qi] + 1];
      if (a.mode && a.mode[qid[qi]] == 1) r1[qi] = r0[qi];   // the gather scan scores it
      resid[qi] = a.preds[qid[qi]].residual_mask != 0;
      if (r1[qi] > r0[qi]) {
        hull_lo = min(hull_lo, r0[qi]);
        hull_hi = max(hull_hi, r1[qi]);
      }
    }
  }
  // Chunks: with a chunk grid, chunk c of the tile is grid cell
  // (first cell of its span) + c cut to the span, so query tiles with nearby
  // spans read the same cells and, scheduled together on one XCD, share its
  // L2.  A span that needs more cells than there are chunks (the planner's
  // estimate fell short) is cut into equal chunks instead.
  int64_t t_begin = 0, t_end = 0;
  if (hull_hi > hull_lo) {
    const int64_t t_lo = hull_lo / 64, t_hi = (hull_hi + 63) / 64;
    const int64_t g = a.chunk_tiles;
    if (g > 0 && a.abs_cells) {
      t_begin = max(t_lo, chunk * g);
      t_end = min(t_hi, (chunk + 1) * g);
    } else if (g > 0 && (t_hi - 1) / g - t_lo / g < a.splits) {
      const int64_t cell = t_lo / g + chunk;
      t_begin = max(t_lo, cell * g);
      t_end = min(t_hi, (cell + 1) * g);
    } else {
      const int64_t ch = max(static_cast<int64_t>(a.min_chunk), (t_hi - t_lo + a.splits - 1) / a.splits);
      t_begin = t_lo + chunk * ch;
      t_end = min(t_hi, t_begin + ch);
    }
  }
  bool work = false;
#pragma unroll
  for (int qi = 0; qi < QT; ++qi)
    work = work || (t_begin < t_end && r1[qi] > r0[qi] && r0[qi] < t_end * 64 && r1[qi] > t_begin * 64);
  // Tile indices fit 32 bits (n < 2^31 rows), so the loop's uniform
  // arithmetic stays on the scalar unit.  ft/lt: first and last tile a
  // query's interval touches (ft > lt when it is empty).
  const int tb = static_cast<int>(t_begin), te = static_cast<int>(t_end);
  int ft[QT], lt[QT];
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    const bool any = qi < qn && r1[qi] > r0[qi];
    ft[qi] = any ? static_cast<int>(r0[qi] >> 6) : INT_MAX;
    lt[qi] = any ? static_cast<int>((r1[qi] - 1) >> 6) : -1;
  }
  if (!work) {
    // Nothing selected in this chunk: empty partial lists (with absolute
    // cells the merge reads only the cells a query's interval touches, so
    // there is nothing to write).
    if (a.abs_cells) return;
    for (int qi = 0; qi < qn; ++qi) {
      uint64_t* dst = a.partials + ((static_cast<size_t>(q0 + qi) * a.splits + chunk) * kScanWaves + wave) * k;
      for (int e = lane; e < k; e += 64) dst[e] = kNoKey;
    }
    return;
  }

  // Selection word of query qi for tile t: interval bits (all ones inside
  // the interval, computed only on its first and last tile), and bitmap
  // bits when the query has residual clauses.
  auto tile_masks = [&](int t, uint64_t (&bm)[QT]) -> uint64_t {
    uint64_t any = 0;
#pragma unroll
    for (int qi = 0; qi < QT; ++qi) {
      uint64_t mk = 0;
      if (t > ft[qi] && t < lt[qi]) {
        mk = ~0ull;
      } else if (t == ft[qi] || t == lt[qi]) {
        const int64_t row0 = static_cast<int64_t>(t) * 64;
        mk = bit_range(max(r0[qi] - row0, static_cast<int64_t>(0)), min(r1[qi] - row0, static_cast<int64_t>(64)));
      }
      if (resid[qi] && mk != 0) mk &= a.bitmap[static_cast<size_t>(qid[qi]) * a.stride64 + t];
      bm[qi] = mk;
      any |= mk;
    }
    return any;
  };

  // Software pipeline over kDepth register sets (fixed M): while the tile in
  // one set is summed, the next kDepth - 1 selected tiles' code words are in
  // flight into the others (no register copy, so nothing waits for the loads
  // in flight).
  auto next_selected = [&](int t, uint64_t (&bm)[QT]) -> int {
    while (t < te && tile_masks(t, bm) == 0) t += kScanWaves;
    return t;
  };
  // Past the chunk's end the loads repeat its last tile (in bounds, unused).
  auto load_tile = [&](int t, uint32_t (&w)[kMW]) {
    const int tc = t < te ? t : te - 1;
    const uint32_t* __restrict__ tile = a.codes_t + static_cast<size_t>(tc) * (kMW * 64);
#pragma unroll
    for (int j = 0; j < kMW; ++j) w[j] = tile[j * 64 + lane];
  };
  constexpr int kDepth = scan_depth<MT, QT, LutT>();
  uint64_t bms[kDepth][QT];
  uint32_t ws[kDepth][kMW];
  int ts[kDepth];
  int t_next = tb + wave;
  auto preload = [&]() {
#pragma unroll
    for (int i = 0; i < kDepth - 1; ++i) {
      ts[i] = next_selected(t_next, bms[i]);
      load_tile(ts[i], ws[i]);
      t_next = ts[i] + kScanWaves;
    }
  };

  // Seed tiles (see the seeded bound below).  Slot i of this wavefront is
  // tile tb + wave + 8i of the chunk on a chunk grid; on short intervals the
  // seed is drawn from the query's whole interval, so every chunk of the
  // query gets the same query-wide bound: all its tiles when there are at
  // most 8 * seed_tiles of them, else that many evenly spaced ones.
  constexpr int kSW = (kGroup + 3) / 4;   // code words holding the first group
  constexpr int kSB = 24;                 // seed tiles per wavefront and round of loads
  const bool seeding = MT > 0 && QT == 1 && a.seed_tiles > 0 && k <= kScanWaves * kScanSeed && te > tb;
  const int64_t seed_span = static_cast<int64_t>(lt[0]) - ft[0] + 1;
  const int64_t seed_slots = static_cast<int64_t>(kScanWaves) * a.seed_tiles;
  auto seed_tile = [&](int i) -> int {
    if (i >= a.seed_tiles) return -1;
    if (a.chunk_tiles > 0) {
      const int t = tb + wave + kScanWaves * i;
      return t < te ? t : -1;
    }
    const int64_t sl = wave + static_cast<int64_t>(kScanWaves) * i;
    if (seed_span <= seed_slots) return sl < seed_span ? static_cast<int>(ft[0] + sl) : -1;
    return static_cast<int>(ft[0] + sl * seed_span / seed_slots);
  };
  // Selection word of seed slot i (0: no tile or nothing selected); the
  // tile in *t.
  auto seed_mask = [&](int i, int* t) -> uint64_t {
    *t = seed_tile(i);
    if (*t < 0) return 0;
    uint64_t b1[QT];
    return tile_masks(*t, b1) != 0 ? b1[0] : 0;
  };
  uint32_t sw[kSB][kSW];
  auto seed_load = [&](int round) {
#pragma unroll
    for (int i = 0; i < kSB; ++i) {
      int t;
      if (seed_mask(round * kSB + i, &t) != 0) {
        const uint32_t* __restrict__ tile = a.codes_t + static_cast<size_t>(t) * (kMW * 64);
#pragma unroll
        for (int j = 0; j < kSW; ++j) sw[i][j] = tile[j * 64 + lane];
      }
    }
  };
  if constexpr (MT > 0) {
    if (seeding) seed_load(0);
    else preload();
  }

  // Tables into LDS as [m][qi][c], noting any entry that is negative or NaN
  // (then partial sums are no lower bound).
  bool bad[QT];
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) bad[qi] = false;
  if constexpr (MT > 0) {
#pragma unroll
    for (int qi = 0; qi < QT; ++qi) {
      if (qi >= qn) break;
#pragma unroll
      for (int u = 0; u < kLutPer; ++u) {
        const int v = threadIdx.x + u * kThreads;
        if (kVecQ % kThreads == 0 || v < kVecQ) {
          const int e = v * kVec;
          const int m = e / kKsub, c = e % kKsub;
          *reinterpret_cast<uint4*>(slut + (static_cast<size_t>(m) * QT + qi) * kKsub + c) = lx[qi][u];
          const LutT* xe = reinterpret_cast<const LutT*>(&lx[qi][u]);
#pragma unroll
          for (int w = 0; w < kVec; ++w) bad[qi] = bad[qi] || !(widen(xe[w]) >= 0.0f);
        }
      }
    }
  } else {
    const int vec_per_query = M * kKsub / kVec;
    for (int qi = 0; qi < qn; ++qi) {
      const uint4* src = reinterpret_cast<const uint4*>(lut + static_cast<size_t>(qid[qi]) * M * kKsub);
      for (int v = threadIdx.x; v < vec_per_query; v += kThreads) {
        const int e = v * kVec;
        const int m = e / kKsub, c = e % kKsub;
        const uint4 x = src[v];
        *reinterpret_cast<uint4*>(slut + (static_cast<size_t>(m) * QT + qi) * kKsub + c) = x;
        const LutT* xe = reinterpret_cast<const LutT*>(&x);
#pragma unroll
        for (int w = 0; w < kVec; ++w) bad[qi] = bad[qi] || !(widen(xe[w]) >= 0.0f);
      }
    }
  }
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    const bool wave_bad = __ballot(bad[qi]) != 0;
    if (lane == 0) s_bad[wave * QT + qi] = wave_bad ? 1u : 0u;
  }
  if (threadIdx.x < QT) s_thr[threadIdx.x] = kNoKey;
  if (threadIdx.x < QT * kScanWaves * kScanPub) s_pub[threadIdx.x] = kNoKey;
  if constexpr (kCount) {
    if (threadIdx.x < 65) s_hist[threadIdx.x] = 0;
  }
  __syncthreads();
  // Early abandonment: every entry >= 0 and fp32 addition of non-negative
  // terms never decreases, so a partial sum above the current k-th distance
  // bounds the full sum from below and the row cannot enter the top k.
  bool monotone[QT];
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    bool mono = qi < qn;
#pragma unroll
    for (int w = 0; w < kScanWaves; ++w) mono = mono && s_bad[w * QT + qi] == 0;
    monotone[qi] = mono;
  }

  // Seeded bound (one query per tile).  A wavefront's own k-th key stays
  // far above the query's answer until its pool holds rows near the query,
  // which on a short interval is about when the scan ends, so before the
  // scan proper each wavefront sums the first subspace group of every
  // selected row of its first seed_tiles selected tiles, keeps each lane's
  // smallest such partial sum, and computes the full distance of the
  // kScanSeed rows with the smallest ones (rows close to the query in the
  // first subspaces are likely close overall).  They are selected rows and
  // their distances are summed exactly as below, so the k-th smallest
  // distance among the workgroup's candidates bounds the query's k-th
  // distance: rows above it are dropped from the first tile on.
  uint64_t seed = kNoKey;
  if constexpr (MT > 0 && QT == 1) {
    if (seeding && monotone[0]) {
      float best_p = __builtin_inff();
      int best_t = -1;
      for (int round = 0;; ++round) {
#pragma unroll
        for (int i = 0; i < kSB; ++i) {
          int t;
          const uint64_t mk = seed_mask(round * kSB + i, &t);
          if (mk != 0) {
            count_reads(~0ull, kGroup);
            float p = 0.0f;
#pragma unroll
            for (int u = 0; u < kGroup; ++u)
              p = __fadd_rn(p, widen(slut[u * kKsub + static_cast<int>((sw[i][u >> 2] >> (8 * (u & 3))) & 0xFFu)]));
            if (((mk >> lane) & 1) && p < best_p) {
              best_p = p;
              best_t = t;
            }
          }
        }
        if ((round + 1) * kSB >= a.seed_tiles) break;
        seed_load(round + 1);
      }
      // The kScanSeed lanes with the smallest partial sums (lane breaks ties).
      uint64_t ck = best_t >= 0 ? (static_cast<uint64_t>(ordered_bits(best_p)) << 32) | static_cast<uint32_t>(lane)
                                : kNoKey;
      bool chosen = false;
#pragma unroll
      for (int j = 0; j < kScanSeed; ++j) {
        uint64_t mn = ck;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint64_t x = shfl_xor_u64(mn, o);
          mn = x < mn ? x : mn;
        }
        if (mn == kNoKey) break;
        if (ck == mn) {
          chosen = true;
          ck = kNoKey;
        }
      }
      // The scan's first tiles are loaded while the candidates' rows are.
      preload();
      float dfull = 0.0f;
      count_reads(__ballot(chosen), MT);
      if (chosen) {
        const uint32_t* __restrict__ tile = a.codes_t + static_cast<size_t>(best_t) * (kMW * 64);
        uint32_t w[kMW];
#pragma unroll
        for (int j = 0; j < kMW; ++j) w[j] = tile[j * 64 + lane];
#pragma unroll
        for (int m = 0; m < MT; ++m)
          dfull = __fadd_rn(dfull, widen(slut[m * kKsub + static_cast<int>((w[m >> 2] >> (8 * (m & 3))) & 0xFFu)]));
      }
      const uint64_t cm = __ballot(chosen);
      const int nc = __popcll(cm);
      if (chosen) s_seed[wave * kScanSeed + lanes_below(cm)] = ordered_bits(dfull);
      if (lane >= nc && lane < kScanSeed) s_seed[wave * kScanSeed + lane] = ~0u;
      __syncthreads();
      uint64_t v[1] = {lane < kScanWaves * kScanSeed ? (static_cast<uint64_t>(s_seed[lane]) << 32) | 0xFFFFFFFFull
                                                     : kNoKey};
      wave_bitonic_sort<1>(v);
      seed = shfl_u64(v[0], k - 1);
      if (threadIdx.x == 0 && seed != kNoKey)
        __hip_atomic_fetch_min(a.gthr + qid[0], seed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else if (seeding) {
      preload();
    }
  }

  int cnt[QT];
  uint64_t thr[QT];
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    cnt[qi] = 0;
    thr[qi] = kNoKey;
  }
  uint64_t* my_pools = pools + static_cast<size_t>(wave) * QT * a.pool_stride;

  // Thresholds.  thr[qi] is the k-th smallest key of this wavefront's own
  // pool.  Any wavefront's k-th key also bounds the query's answer (k smaller
  // keys exist), so each wavefront publishes its threshold to the workgroup
  // (LDS) and to the query (global memory) and filters with the smallest
  // one it knows: bound[qi] = min(own, workgroup, query).  A row whose key is
  // not below the bound cannot be among the query's k best.
  //
  // The query's value is read once per two tiles and taken in one loop
  // iteration (two tiles) later, by when the load has long landed.  Every
  // load of a step is issued on every path, so the compiler's wait counts
  // never make the current tile wait for the next one's words.
  uint64_t published[QT], gview[QT], gnext[QT], bound[QT];
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) published[qi] = gview[qi] = gnext[qi] = bound[qi] = kNoKey;
  // Union bound.  A wavefront's own k-th key reflects only the rows it
  // scanned, and the workgroup's smallest such key is about the
  // (waves * k)-th best row the workgroup has seen -- too loose to stop the
  // summation early on short intervals.  So each wavefront keeps the two
  // smallest distances it has summed in full (two distinct rows; a wavefront
  // reduction over the step's surviving lanes, no pool work) and, when they
  // fall, stores them in its slots of s_best.  Wavefronts scan disjoint
  // rows, so the k-th smallest of the workgroup's 16 slots is the distance of
  // one of k distinct rows at or below it: a bound on the query's answer,
  // published like a threshold (with the largest id, so rows at that
  // distance stay eligible).
  const bool union_bound = a.shared_bound && k <= kScanWaves * kScanPub;
  uint32_t best1[QT], best2[QT];   // this wavefront's two smallest full distances
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) best1[qi] = best2[qi] = ~0u;
  auto global_issue = [&]() {
#pragma unroll
    for (int qi = 0; qi < QT; ++qi)
      gnext[qi] = __hip_atomic_load(a.gthr + qid[qi], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };
  auto global_finish = [&]() {
#pragma unroll
    for (int qi = 0; qi < QT; ++qi) gview[qi] = gnext[qi];
  };
  auto refresh_bounds = [&]() {
#pragma unroll
    for (int qi = 0; qi < QT; ++qi) {
      if (qi >= qn) continue;
      const uint64_t blk = s_thr[qi];
      uint64_t b = thr[qi] < blk ? thr[qi] : blk;
      b = b < gview[qi] ? b : gview[qi];
      bound[qi] = QT == 1 && seed < b ? seed : b;
    }
  };

  auto consider = [&](int qi, bool act, float d, int t) {
    uint64_t key = kNoKey;
    bool cand = false;
    if (act) {
      const uint32_t db = ordered_bits(d);
      if (db <= static_cast<uint32_t>(bound[qi] >> 32)) {
        const uint32_t row = static_cast<uint32_t>(t * 64 + lane);
        if (a.perm) {
          key = row_key(db, row);   // original id looked up when the pool is compacted
          cand = true;
        } else {
          key = (static_cast<uint64_t>(db) << 32) | row;
          cand = key < bound[qi];
        }
      }
    }
    if (union_bound) {
      // The step's two smallest full distances (pairs merged across lanes),
      // then the wavefront's two smallest so far.
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
      const uint32_t hi = best1[qi] > x1 ? best1[qi] : x1;
      const uint32_t lo2 = best2[qi] < x2 ? best2[qi] : x2;
      const uint32_t n1 = best1[qi] < x1 ? best1[qi] : x1;
      const uint32_t n2 = hi < lo2 ? hi : lo2;
      if (n1 < best1[qi] || n2 < best2[qi]) {
        // The k-th smallest slot only falls when a slot drops from at or
        // above it to below it; the other improvements are only stored.
        const uint32_t kth = static_cast<uint32_t>(published[qi] >> 32);
        const bool crossed = (n1 < kth && best1[qi] >= kth) || (n2 < kth && best2[qi] >= kth);
        best1[qi] = n1;
        best2[qi] = n2;
        unsigned long long* pairs = s_pub + qi * kScanWaves;
        if (lane == 0)
          __hip_atomic_store(&pairs[wave], (static_cast<unsigned long long>(n2) << 32) | n1, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_WORKGROUP);
        if (crossed) {
          // Rank of each of the 16 slots (ties by slot index); the slot of
          // rank k - 1 is the k-th smallest.  Lanes 2w and 2w + 1 read
          // wavefront w's word in the same instruction, so they see one pair.
          const unsigned long long pw =
              lane < kScanWaves * kScanPub
                  ? __hip_atomic_load(&pairs[lane >> 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)
                  : ~0ull;
          const uint32_t v = static_cast<uint32_t>((lane & 1) ? pw >> 32 : pw);
          int rank = 0;
#pragma unroll
          for (int j = 0; j < kScanWaves * kScanPub; ++j) {
            const uint32_t vj = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), j));
            rank += (vj < v || (vj == v && j < lane)) ? 1 : 0;
          }
          const uint64_t at = __ballot(lane < kScanWaves * kScanPub && rank == k - 1);
          const uint32_t kv = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), __builtin_ctzll(at)));
          const uint64_t ub = (static_cast<uint64_t>(kv) << 32) | 0xFFFFFFFFull;
          if (ub < published[qi]) {
            published[qi] = ub;
            if (lane == 0) {
              atomicMin(&s_thr[qi], static_cast<unsigned long long>(ub));
              __hip_atomic_fetch_min(a.gthr + qid[qi], ub, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
          }
        }
      }
    }
    uint64_t* pool = my_pools + qi * a.pool_stride;
    pool_push(pool, cnt[qi], thr[qi], key, cand, k, a.kpl, a.perm);
    if (thr[qi] < published[qi]) {
      published[qi] = thr[qi];
      if (lane == 0) {
        atomicMin(&s_thr[qi], static_cast<unsigned long long>(thr[qi]));
        __hip_atomic_fetch_min(a.gthr + qid[qi], thr[qi], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  };

  if constexpr (MT > 0) {
    auto sum_tile = [&](int t, const uint64_t (&bm)[QT], const uint32_t (&w)[kMW]) {
      refresh_bounds();
      if constexpr (kCount) {
        if ((threadIdx.x & 63) == 0) atomicAdd(&s_hist[0], 1u);
      }
      // Subspaces are summed in groups, all of the tile's queries side by
      // side: a group's table reads of every query are issued before its
      // additions, so the reads of different queries overlap.  After each
      // group a lane whose partial sum already exceeds its query's k-th
      // distance drops out (NaN cut before k candidates exist: nothing drops).
      float cut[QT], d[QT];
      bool live[QT];
#pragma unroll
      for (int qi = 0; qi < QT; ++qi) {
        cut[qi] = monotone[qi] ? from_ordered_bits(static_cast<uint32_t>(bound[qi] >> 32)) : __builtin_nanf("");
        live[qi] = __builtin_amdgcn_inverse_ballot_w64(bm[qi]);
        d[qi] = 0.0f;
      }
#pragma unroll
      for (int g = 0; g < MT / kGroup; ++g) {
        int addr[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
          const int m = g * kGroup + u;
          addr[u] = m * QT * kKsub + static_cast<int>((w[m >> 2] >> (8 * (m & 3))) & 0xFFu);
        }
        LutT v[QT][kGroup];
#pragma unroll
        for (int qi = 0; qi < QT; ++qi) {
          count_reads(__ballot(live[qi]), kGroup);
          if (live[qi]) {
#pragma unroll
            for (int u = 0; u < kGroup; ++u) v[qi][u] = slut[addr[u] + qi * kKsub];
          }
        }
#pragma unroll
        for (int qi = 0; qi < QT; ++qi) {
          if (live[qi]) {
#pragma unroll
            for (int u = 0; u < kGroup; ++u) d[qi] = __fadd_rn(d[qi], widen(v[qi][u]));
          }
          live[qi] = live[qi] && !(d[qi] > cut[qi]);
        }
      }
#pragma unroll
      for (int qi = 0; qi < QT; ++qi)
        // Usually every lane has dropped out: nothing to offer.
        if (__ballot(live[qi]) != 0) consider(qi, live[qi], d[qi], t);
    };
    // Step i sums set i and refills the set summed in the step before with
    // the tile kDepth - 1 places ahead; tiles are visited in increasing
    // order, so the first one past the chunk ends the loop.
    for (;;) {
      global_finish();
      global_issue();
#pragma unroll
      for (int i = 0; i < kDepth; ++i) {
        constexpr int unused = 0;
        (void)unused;
        const int j = (i + kDepth - 1) % kDepth;
        ts[j] = next_selected(t_next, bms[j]);
        load_tile(ts[j], ws[j]);
        t_next = ts[j] + kScanWaves;
        if (ts[i] >= te) goto scanned;
        sum_tile(ts[i], bms[i], ws[i]);
      }
    }
  scanned:;
  } else {
    for (int t = tb + wave; t < te; t += kScanWaves) {
      uint64_t bm[QT];
      if (tile_masks(t, bm) == 0) continue;
      global_issue();
      global_finish();
      refresh_bounds();
#pragma unroll
      for (int qi = 0; qi < QT; ++qi) {
        if (bm[qi] == 0) continue;
        const bool act = __builtin_amdgcn_inverse_ballot_w64(bm[qi]);
        float d = 0.0f;
        if (act) {
          for (int m = 0; m < M; ++m) {
            const uint32_t wv = a.codes_t[(static_cast<size_t>(t) * a.mw + (m >> 2)) * 64 + lane];
            const int c = static_cast<int>((wv >> (8 * (m & 3))) & 0xFFu);
            d = __fadd_rn(d, widen(slut[(static_cast<size_t>(m) * QT + qi) * kKsub + c]));
          }
        }
        consider(qi, act, d, t);
      }
    }
  }

  // Each wavefront's k best keys per query, ascending, padded with kNoKey.
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    if (qi >= qn) break;
    uint64_t* pool = my_pools + qi * a.pool_stride;
    pool_compact(pool, cnt[qi], thr[qi], k, a.kpl, a.perm);
    uint64_t* dst = a.partials + ((static_cast<size_t>(q0 + qi) * a.splits + chunk) * kScanWaves + wave) * k;
    for (int e = lane; e < k; e += 64) dst[e] = pool[e];
  }
  if constexpr (kCount) {
    __syncthreads();
    if (threadIdx.x < 65 && s_hist[threadIdx.x] != 0)
      atomicAdd(&a.lookup_hist[threadIdx.x], static_cast<unsigned long long>(s_hist[threadIdx.x]));
  }
}

template <int MT, int QT, typename LutT>
const void* scan_symbol() {
  return reinterpret_cast<const void*>(&scan_kernel<MT, QT, LutT>);
}

constexpr int kQtiles[] = {1, 2, 3, 4, 6, 8};

// Instantiated only where the static tables and the smallest pools fit.
template <int MT, int QT, typename LutT>
constexpr bool scan_fits() {
  return static_cast<size_t>(MT) * QT * kKsub * sizeof(LutT) +
             static_cast<size_t>(QT) * (kScanWaves * 65 * sizeof(uint64_t) + 8 + 4 * kScanWaves +
                                        kScanWaves * kScanPub * sizeof(uint64_t)) +
             kScanWaves * kScanSeed * sizeof(uint32_t) <=
         static_cast<size_t>(kLdsBudget);
}

template <int MT, int QT, typename LutT>
const void* scan_symbol_if_fits() {
  if constexpr (scan_fits<MT, QT, LutT>()) return scan_symbol<MT, QT, LutT>();
  else return nullptr;
}

template <typename LutT, int MT>
const void* pick_q(int qt) {
  switch (qt) {
    case 1: return scan_symbol_if_fits<MT, 1, LutT>();
    case 2: return scan_symbol_if_fits<MT, 2, LutT>();
    case 3: return scan_symbol_if_fits<MT, 3, LutT>();
    case 4: return scan_symbol_if_fits<MT, 4, LutT>();
    case 6: return scan_symbol_if_fits<MT, 6, LutT>();
    case 8: return scan_symbol_if_fits<MT, 8, LutT>();
    default: return nullptr;
  }
}

// The counting build exists for one-query tiles of a fixed M.
template <typename LutT, int MT>
const void* count_symbol_if_fits() {
  if constexpr (scan_fits<MT, 1, LutT>()) return reinterpret_cast<const void*>(&scan_kernel<MT, 1, LutT, true>);
  else return nullptr;
}

template <typename LutT>
const void* pick_count(int m, int qt) {
  if (qt != 1) return nullptr;
  switch (m) {
    case 16: return count_symbol_if_fits<LutT, 16>();
    case 48: return count_symbol_if_fits<LutT, 48>();
    case 120: return count_symbol_if_fits<LutT, 120>();
    default: return nullptr;
  }
}

template <typename LutT>
const void* pick(int m, int qt) {
  switch (m) {
    case 16: return pick_q<LutT, 16>(qt);
    case 48: return pick_q<LutT, 48>(qt);
    case 120: return pick_q<LutT, 120>(qt);
    default: return pick_q<LutT, 0>(qt);
  }
}

}  // namespace

int pool_kpl(int k) {
  int kpl = 2;
  while (64 * kpl < k + 64) kpl *= 2;
  return kpl;
}

int pool_stride_for(int k) {
  // Register-sorted pools need only k + 64 slots; pools sorted in LDS use the
  // whole power of two.
  const int kpl = pool_kpl(k);
  return kpl <= 4 ? k + 64 : 64 * kpl;
}

size_t scan_lds_bytes(int m, int qtile, int lut_bytes, int pool_stride) {
  // tables, pools, workgroup thresholds (8 B), per-wave monotonicity flags
  // (4 B each) and published best keys, then the seed candidates
  return static_cast<size_t>(qtile) *
             (static_cast<size_t>(m) * kKsub * lut_bytes +
              static_cast<size_t>(kScanWaves) * pool_stride * sizeof(uint64_t) + 8 + 4 * kScanWaves +
              static_cast<size_t>(kScanWaves) * kScanPub * sizeof(uint64_t)) +
         static_cast<size_t>(kScanWaves) * kScanSeed * sizeof(uint32_t);
}

int scan_max_qtile(int m, int lut_bytes, int k) {
  int q = 0;
  while (scan_lds_bytes(m, q + 1, lut_bytes, pool_stride_for(k)) <= static_cast<size_t>(kLdsBudget)) ++q;
  return q;
}

int scan_supported_qtile(int want) {
  int best = 0;
  for (int q : kQtiles)
    if (q <= want) best = q;
  return best;
}

bool scan_can_count(int m, int qtile, int lut_dtype) {
  return (lut_dtype == 1 ? pick_count<__half>(m, qtile) : pick_count<float>(m, qtile)) != nullptr;
}

hipError_t launch_scan(const ScanBatch& b, const ScanPlan& plan, hipStream_t s) {
  const void* fn = b.lookup_hist ? (b.lut_dtype == 1 ? pick_count<__half>(b.m, plan.qtile)
                                                     : pick_count<float>(b.m, plan.qtile))
                                 : (b.lut_dtype == 1 ? pick<__half>(b.m, plan.qtile) : pick<float>(b.m, plan.qtile));
  if (!fn) return hipErrorInvalidValue;
  // Fixed-M kernels hold their tables in static LDS; the rest is dynamic.
  const bool fixed_m = b.m == 16 || b.m == 48 || b.m == 120;
  const size_t table = static_cast<size_t>(b.m) * plan.qtile * kKsub * (b.lut_dtype == 1 ? 2 : 4);
  const size_t dyn = (fixed_m ? plan.lds_bytes - table : plan.lds_bytes) + (b.lookup_hist ? kLookupHistBytes : 0);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(dyn));
  if (e != hipSuccess) return e;
  ScanArgs a{};
  a.codes_t = b.codes_t;
  a.n = b.n;
  a.n_tiles = b.n_tiles;
  a.m = b.m;
  a.mw = b.mw;
  a.lut = b.lut;
  a.nq = b.nq;
  a.qorder = b.qorder;
  a.iv = b.iv;
  a.preds = b.preds;
  a.bitmap = b.bitmap;
  a.stride64 = b.stride64;
  a.perm = b.perm;
  a.k = b.k;
  a.pool_stride = plan.pool_stride;
  a.kpl = plan.kpl;
  a.min_chunk = plan.min_chunk;
  a.chunk_tiles = plan.chunk_tiles;
  a.abs_cells = plan.abs_cells ? 1 : 0;
  a.mode = b.mode;
  a.slot_order = b.slot_order;
  a.shared_bound = plan.shared_bound ? 1 : 0;
  a.seed_tiles = plan.seed_tiles;
  a.partials = b.partials;
  a.gthr = b.gthr;
  a.lookup_hist = b.lookup_hist;
  a.splits = plan.splits;
  a.n_qtiles = (b.nq + plan.qtile - 1) / plan.qtile;
  const unsigned per_xcd = static_cast<unsigned>((a.n_qtiles + kXcds - 1) / kXcds);
  const dim3 grid(static_cast<unsigned>(kXcds) * per_xcd * static_cast<unsigned>(a.splits));
  void* args[] = {&a};
  return hipLaunchKernel(fn, grid, dim3(kScanWaves * 64), args, dyn, s);
}

}  // namespace ifvs
