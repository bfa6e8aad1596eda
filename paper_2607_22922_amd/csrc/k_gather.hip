// Selectivity-adaptive Rank stage (Section 2, stage 2) for batches scanned
// through selection bitmaps.  A query that selects few rows does not need a
// pass over every code tile: its bitmap is compacted into the ascending list
// of selected physical rows, and a gather scan scores just those rows from a
// row-major copy of the codes (one contiguous code row per lane).  Queries
// selecting more rows than the list holds stay on the tiled scan.
//
// The choice is made on the device, per query, from the Filter stage's pool
// size; the tiled scan skips gather-mode queries and the gather scan writes
// every partial-list slot of its queries, so the merge is the same for both.
// Scoring follows the tiled scan: the M table entries of a row are summed in
// m order from +0 with separately rounded fp32 additions (early abandonment
// in groups when the table is non-negative), candidates beating the
// wavefront's k-th key go to its pool, thresholds are shared through LDS
// and the query's global key.
#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

constexpr int kCompactThreads = 256;
constexpr int kCompactWordsPerThread = 4;
constexpr int64_t kWordsPerPart = kFilterPartRows / 64;   // bitmap words per filter count partial
constexpr int kCompactParts = kCompactThreads * kCompactWordsPerThread / kWordsPerPart;
static_assert(kCompactParts * kWordsPerPart == kCompactThreads * kCompactWordsPerThread, "whole parts");
constexpr int kCompactStage = 8192;   // rows a compaction workgroup stages in LDS (32 KB)
// Rows a gather workgroup scores at most (8 wavefronts x 64 lanes x 16).
constexpr int64_t kGatherRowsPerBlock = static_cast<int64_t>(kScanWaves) * 64 * 16;

__device__ __forceinline__ float widen_g(float v) { return v; }
__device__ __forceinline__ float widen_g(__half v) { return __half2float(v); }

// codes_rm[row][j] = word j of physical row `row` (zero past mw).
__global__ void rowmajor_kernel(const uint32_t* __restrict__ codes_t, int64_t n, int mw, int rw,
                                uint32_t* __restrict__ codes_rm) {
  const int64_t total = n * rw;
  for (int64_t o = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; o < total;
       o += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t row = o / rw;
    const int j = static_cast<int>(o % rw);
    codes_rm[o] = j < mw ? codes_t[((row >> 6) * mw + j) * 64 + (row & 63)] : 0u;
  }
}

// mode[q] = 1 (gather) when the pool holds at most max_rows rows, and then
// the ascending list of its selected physical rows.  Workgroup (g, q) covers
// kCompactParts consecutive filter parts of query q (thread t: 4 consecutive
// bitmap words); its rows start at the Filter stage's prefix count of its
// first part, and a workgroup prefix sum orders them within.
__global__ __launch_bounds__(kCompactThreads) void compact_kernel(
    const uint64_t* __restrict__ bitmap, int64_t stride64, const unsigned long long* __restrict__ counts,
    const uint32_t* __restrict__ count_prefix, int64_t parts, int nq, int64_t max_rows, int64_t list_cap,
    int32_t* __restrict__ lists, int32_t* __restrict__ list_n, int32_t* __restrict__ mode) {
  const int q = blockIdx.y;
  const int64_t part0 = static_cast<int64_t>(blockIdx.x) * kCompactParts;
  if (q >= nq || part0 >= parts) return;
  const unsigned long long cnt = counts[q];
  const bool gather = max_rows >= 0 && cnt <= static_cast<unsigned long long>(max_rows);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    mode[q] = gather ? 1 : 0;
    list_n[q] = gather ? static_cast<int32_t>(cnt) : 0;
  }
  if (!gather) return;
  __shared__ int s_wave_sum[kCompactThreads / 64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint64_t* words = bitmap + static_cast<size_t>(q) * stride64;
  int32_t* out = lists + static_cast<size_t>(q) * list_cap;
  const int64_t first = part0 * kWordsPerPart + static_cast<int64_t>(threadIdx.x) * kCompactWordsPerThread;
  uint64_t wv[kCompactWordsPerThread];
  int c = 0;
#pragma unroll
  for (int u = 0; u < kCompactWordsPerThread; ++u) {
    wv[u] = first + u < stride64 ? words[first + u] : 0ull;
    c += __popcll(wv[u]);
  }
  // Exclusive prefix of c over the workgroup (threads in word order).
  int incl = c;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) s_wave_sum[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int i = 0; i < kCompactThreads / 64; ++i) {
    const int sw = s_wave_sum[i];
    before += i < wave ? sw : 0;
    total += sw;
  }
  const int64_t base = static_cast<int64_t>(count_prefix[static_cast<int64_t>(q) * parts + part0]);
  if (total <= kCompactStage) {
    // Each thread's rows go to LDS at their rank, then the workgroup copies
    // them out with coalesced stores (a thread's own run of rows would make
    // every store instruction touch up to 64 cache lines).
    __shared__ int32_t s_rows[kCompactStage];
    int pos = before + incl - c;
#pragma unroll
    for (int u = 0; u < kCompactWordsPerThread; ++u) {
      uint64_t x = wv[u];
      while (x) {
        const int b = __ffsll(static_cast<long long>(x)) - 1;
        s_rows[pos++] = static_cast<int32_t>((first + u) * 64 + b);
        x &= x - 1;
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < total; i += kCompactThreads)
      if (base + i < list_cap) out[base + i] = s_rows[i];
    return;
  }
  int64_t pos = base + before + incl - c;
#pragma unroll
  for (int u = 0; u < kCompactWordsPerThread; ++u) {
    uint64_t x = wv[u];
    while (x) {
      const int b = __ffsll(static_cast<long long>(x)) - 1;
      if (pos < list_cap) out[pos] = static_cast<int32_t>((first + u) * 64 + b);
      ++pos;
      x &= x - 1;
    }
  }
}

struct GatherArgs {
  const uint32_t* codes_rm;   // [n][rw] words
  int rw;
  const void* lut;            // [nq][M][256] by original query index
  int nq;
  const int32_t* qorder;      // position -> original query index
  const int32_t* mode;        // [nq] 1: gather
  const int32_t* lists;       // [nq][list_cap]
  const int32_t* list_n;      // [nq]
  int64_t list_cap;
  int gblocks;                // workgroups per query position
  int splits;                 // partial-list slots per query position
  const int32_t* perm;        // physical row -> original id (null: identity)
  int k, pool_stride, kpl;
  uint64_t* partials;         // [positions][splits][kScanWaves][k]
  uint64_t* gthr;
};

// Workgroup (position p, c): when its query is in gather mode and c < G (G =
// workgroups its list needs), it scores list entries [c·n/G, (c+1)·n/G) and
// writes its wavefronts' k best keys to slot c; it also owns slots
// c + gblocks, c + 2·gblocks, ... < splits, which it fills with empty lists.
template <int MT, typename LutT>
__global__ __launch_bounds__(kScanWaves * 64) void gather_scan_kernel(const GatherArgs a) {
  constexpr int kMW = (MT + 3) / 4;
  constexpr int kGroup = MT % 8 == 0 && MT > 16 ? 8 : (MT % 4 == 0 ? 4 : MT);
  __shared__ __align__(16) unsigned char s_lut_raw[static_cast<size_t>(MT) * kKsub * sizeof(LutT)];
  extern __shared__ __align__(16) unsigned char smem[];
  LutT* slut = reinterpret_cast<LutT*>(s_lut_raw);
  uint64_t* pools = reinterpret_cast<uint64_t*>(smem);
  unsigned long long* s_thr = reinterpret_cast<unsigned long long*>(pools + static_cast<size_t>(kScanWaves) * a.pool_stride);
  uint32_t* s_not_monotone = reinterpret_cast<uint32_t*>(s_thr + 1);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int p = blockIdx.x / a.gblocks;
  const int c = blockIdx.x % a.gblocks;
  if (p >= a.nq) return;
  const int qid = a.qorder[p];
  if (a.mode[qid] != 1) return;   // the tiled scan handled this query
  const int k = a.k;
  const int64_t cnt = min(static_cast<int64_t>(a.list_n[qid]), a.list_cap);
  const int64_t need = (cnt + kGatherRowsPerBlock - 1) / kGatherRowsPerBlock;
  const int g = static_cast<int>(max(static_cast<int64_t>(1), min(static_cast<int64_t>(a.gblocks), need)));
  auto slot_out = [&](int slot) {
    return a.partials + ((static_cast<size_t>(p) * a.splits + slot) * kScanWaves + wave) * k;
  };
  for (int slot = c + a.gblocks; slot < a.splits; slot += a.gblocks)
    for (int e = lane; e < k; e += 64) slot_out(slot)[e] = kNoKey;
  const int64_t r_begin = c < g ? c * cnt / g : 0;
  const int64_t r_end = c < g ? (c + 1) * cnt / g : 0;
  if (r_begin >= r_end) {
    for (int e = lane; e < k; e += 64) slot_out(c)[e] = kNoKey;
    return;
  }

  // Stage the query's table, noting negative or NaN entries.
  if (threadIdx.x == 0) {
    s_not_monotone[0] = 0;
    s_thr[0] = kNoKey;
  }
  __syncthreads();
  constexpr int kVec = 16 / sizeof(LutT);
  constexpr int vec_per_query = MT * kKsub / kVec;
  {
    const uint4* src = reinterpret_cast<const uint4*>(static_cast<const LutT*>(a.lut) +
                                                      static_cast<size_t>(qid) * MT * kKsub);
    bool bad = false;
    for (int v = threadIdx.x; v < vec_per_query; v += kScanWaves * 64) {
      const uint4 x = src[v];
      reinterpret_cast<uint4*>(slut)[v] = x;
      const LutT* xe = reinterpret_cast<const LutT*>(&x);
#pragma unroll
      for (int u = 0; u < kVec; ++u) bad = bad || !(widen_g(xe[u]) >= 0.0f);
    }
    if (bad) atomicOr(&s_not_monotone[0], 1u);
  }
  __syncthreads();
  const bool monotone = s_not_monotone[0] == 0;

  int cnt_pool = 0;
  uint64_t thr = kNoKey, published = kNoKey, gview = kNoKey, bound = kNoKey;
  uint64_t* pool = pools + static_cast<size_t>(wave) * a.pool_stride;
  const int32_t* list = a.lists + static_cast<size_t>(qid) * a.list_cap;

  // Wavefront step s scores list entries r_begin + (s·8 + wave)·64 + lane.
  constexpr int kUnitRows = kScanWaves * 64;
  auto load_rows = [&](int64_t r0, uint32_t (&w)[kMW], int32_t& row) {
    const int64_t r = r0 + lane;
    row = r < r_end ? list[r] : -1;
    const uint32_t* src = a.codes_rm + static_cast<size_t>(row < 0 ? list[r_begin] : row) * a.rw;
#pragma unroll
    for (int j = 0; j < kMW; j += 4) {
      const uint4 x = *reinterpret_cast<const uint4*>(src + j);
      w[j] = x.x;
      if (j + 1 < kMW) w[j + 1] = x.y;
      if (j + 2 < kMW) w[j + 2] = x.z;
      if (j + 3 < kMW) w[j + 3] = x.w;
    }
  };
  auto score = [&](const uint32_t (&w)[kMW], int32_t row) {
    const uint64_t blk = s_thr[0];
    bound = thr < blk ? thr : blk;
    bound = bound < gview ? bound : gview;
    const float cut = monotone ? from_ordered_bits(static_cast<uint32_t>(bound >> 32)) : __builtin_nanf("");
    bool live = row >= 0;
    float d = 0.0f;
#pragma unroll
    for (int gi = 0; gi < MT / kGroup; ++gi) {
      if (live) {
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
          const int m = gi * kGroup + u;
          const int code = static_cast<int>((w[m >> 2] >> (8 * (m & 3))) & 0xFFu);
          d = __fadd_rn(d, widen_g(slut[m * kKsub + code]));
        }
      }
      live = live && !(d > cut);
    }
    if (__ballot(live) == 0) return;
    uint64_t key = kNoKey;
    bool cand = false;
    if (live) {
      const uint32_t db = ordered_bits(d);
      if (db <= static_cast<uint32_t>(bound >> 32)) {
        if (a.perm) {
          key = row_key(db, static_cast<uint32_t>(row));   // original id looked up when the pool is compacted
          cand = true;
        } else {
          key = (static_cast<uint64_t>(db) << 32) | static_cast<uint32_t>(row);
          cand = key < bound;
        }
      }
    }
    pool_push(pool, cnt_pool, thr, key, cand, k, a.kpl, a.perm);
    if (thr < published) {
      published = thr;
      if (lane == 0) {
        atomicMin(&s_thr[0], static_cast<unsigned long long>(thr));
        __hip_atomic_fetch_min(a.gthr + qid, thr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  };
  // Two register sets alternate (the next rows load while these are scored);
  // the query's global key is read once per pair and taken in a pair later.
  uint32_t wa[kMW], wb[kMW];
  int32_t ra, rb;
  uint64_t gnext = kNoKey;
  int64_t s0 = r_begin + static_cast<int64_t>(wave) * 64;
  load_rows(s0, wa, ra);
  while (s0 < r_end) {
    const int64_t s1 = s0 + kUnitRows;
    gview = gnext;
    gnext = __hip_atomic_load(a.gthr + qid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    load_rows(s1, wb, rb);
    score(wa, ra);
    if (s1 >= r_end) break;
    s0 = s1 + kUnitRows;
    load_rows(s0, wa, ra);
    score(wb, rb);
  }
  pool_compact(pool, cnt_pool, thr, k, a.kpl, a.perm);
  for (int e = lane; e < k; e += 64) slot_out(c)[e] = pool[e];
}

template <typename LutT>
const void* pick_gather(int m) {
  switch (m) {
    case 16: return reinterpret_cast<const void*>(&gather_scan_kernel<16, LutT>);
    case 48: return reinterpret_cast<const void*>(&gather_scan_kernel<48, LutT>);
    case 120: return reinterpret_cast<const void*>(&gather_scan_kernel<120, LutT>);
    default: return nullptr;
  }
}

}  // namespace

bool gather_supported(int m, int lut_dtype) {
  const size_t table = static_cast<size_t>(m) * kKsub * (lut_dtype == 1 ? 2 : 4);
  return (m == 16 || m == 48 || m == 120) && table <= static_cast<size_t>(kLdsBudget);
}

int gather_row_words(int m) { return ((m + 15) / 16) * 4; }

size_t gather_lds_bytes(int pool_stride) {
  return static_cast<size_t>(kScanWaves) * pool_stride * sizeof(uint64_t) + 12;
}

int gather_blocks_per_query(int64_t list_cap, int splits) {
  const int64_t want = (list_cap + kGatherRowsPerBlock - 1) / kGatherRowsPerBlock;
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(want, splits)));
}

hipError_t launch_rowmajor_codes(const uint32_t* codes_t, int64_t n, int mw, int rw, uint32_t* codes_rm,
                                 hipStream_t s) {
  const int64_t total = n * rw;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 65536);
  rowmajor_kernel<<<dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s>>>(codes_t, n, mw, rw, codes_rm);
  return hipGetLastError();
}

hipError_t launch_compact(const uint64_t* bitmap, int64_t stride64, const unsigned long long* counts,
                          const uint32_t* count_prefix, int64_t parts, int nq, int64_t max_rows,
                          int64_t list_cap, int32_t* lists, int32_t* list_n, int32_t* mode, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>((parts + kCompactParts - 1) / kCompactParts), static_cast<unsigned>(nq));
  compact_kernel<<<grid, dim3(kCompactThreads), 0, s>>>(bitmap, stride64, counts, count_prefix, parts, nq,
                                                         max_rows, list_cap, lists, list_n, mode);
  return hipGetLastError();
}

hipError_t launch_gather_scan(const GatherBatch& b, hipStream_t s) {
  const void* fn = b.lut_dtype == 1 ? pick_gather<__half>(b.m) : pick_gather<float>(b.m);
  if (!fn) return hipErrorInvalidValue;
  const size_t dyn = gather_lds_bytes(b.pool_stride);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(dyn));
  if (e != hipSuccess) return e;
  GatherArgs a{};
  a.codes_rm = b.codes_rm;
  a.rw = b.rw;
  a.lut = b.lut;
  a.nq = b.nq;
  a.qorder = b.qorder;
  a.mode = b.mode;
  a.lists = b.lists;
  a.list_n = b.list_n;
  a.list_cap = b.list_cap;
  a.gblocks = b.gblocks;
  a.splits = b.splits;
  a.perm = b.perm;
  a.k = b.k;
  a.pool_stride = b.pool_stride;
  a.kpl = b.kpl;
  a.partials = b.partials;
  a.gthr = b.gthr;
  void* args[] = {&a};
  const dim3 grid(static_cast<unsigned>(b.nq) * static_cast<unsigned>(b.gblocks));
  return hipLaunchKernel(fn, grid, dim3(kScanWaves * 64), args, dyn, s);
}

}  // namespace ifvs
