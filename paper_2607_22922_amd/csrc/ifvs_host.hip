// Host runtime of libifvs: the C ABI declared in include/ifvs.h.
//
// Owns the device-resident index (codes re-laid out into 64-row tiles,
// possibly in cluster-key order, codebook, attribute columns, memory bank,
// direction tensor), a workspace sized once at load (device copies of the
// predicates and the query order, row intervals, selection bitmaps, pool
// sizes, per-wavefront top-k partials, pinned staging), argument validation,
// and the launch plan of each call.  The hot calls allocate nothing.
#include "ifvs.h"
#include "ifvs_internal.h"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <mutex>
#include <numeric>
#include <thread>
#include <string>
#include <vector>

using namespace ifvs;

namespace {

thread_local std::string g_error = "no error";

ifvs_status fail(ifvs_status st, const std::string& msg) {
  g_error = msg;
  return st;
}

ifvs_status hip_fail(hipError_t e, const char* what) {
  return fail(IFVS_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define IFVS_HIP(call, what)                         \
  do {                                               \
    const hipError_t e_ = (call);                    \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

// Test hook: IFVS_FAIL_ALLOC=n makes the n-th allocation of a process fail
// (1-based), so out-of-memory paths can be exercised on purpose.
int g_alloc_counter = 0;

bool forced_alloc_failure() {
  static const int fail_at = [] {
    const char* s = std::getenv("IFVS_FAIL_ALLOC");
    return s ? std::atoi(s) : 0;
  }();
  ++g_alloc_counter;
  return fail_at > 0 && g_alloc_counter == fail_at;
}

constexpr int kStagingSlots = 8;
// Automatic list scan: batches whose widest interval spans at least this
// many 64-row tiles (measured on 10M x 48-byte codes, 256 queries: at 10%
// selectivity, 15.6K tiles, the list scan and its plan take 0.74 ms against
// the interval scan's 1.16; at 1%, 1.6K tiles, 1.2 ms against 0.25), on
// indexes of at least kCoarseAutoM subspaces (on 100M x 16-byte codes, whose
// bounds prune little and whose one-kilobyte tiles leave the list scan's
// per-tile work in front, it ran 1.6x the interval scan's time at 1% and
// 1.26x at 10%).
constexpr int64_t kCoarseAutoTiles = 8192;
constexpr int kCoarseAutoM = 32;
// Radius quantiles that split each coarse list into its kBands bands.
constexpr float kBandQuantiles[kBands - 1] = {0.5f, 0.85f, 0.97f};

// Optional per-stage kernel timing with HIP events (IFVS_OPT_PROFILE).
enum Stage { kStCondition = 0, kStLut, kStFilter, kStScan, kStMerge, kStEncode, kStCoarse, kStages };
// The list scan's launches: reported under kStScan, selectable on their own
// (IFVS_OPT_PROFILE 3) by this bit of the profile mask.
constexpr int kStListScan = kStages;
constexpr int kProfilePairs = 4096;

struct StageTimer {
  hipEvent_t ev[2 * kProfilePairs] = {};
  int used = 0;
  double ms = 0.0;
  int64_t launches = 0;
};

constexpr int kFences = 4096;
constexpr int64_t kMaxValueTable = int64_t{1} << 22;   // entries (16 MB) of the cluster key table

constexpr int64_t kI32Min = std::numeric_limits<int32_t>::min();
constexpr int64_t kI32End = int64_t(std::numeric_limits<int32_t>::max()) + 1;

}  // namespace

// Workspace of ifvs_filtered_search_noalloc: a static array in device memory,
// one copy on every GPU the library runs on, placed with the code object (no
// allocation call at run time) and held until the process ends.  In host code
// `scratch` names a host-side stand-in, never the device copy: kernels and
// copies use the device address that static_scratch_bind() looks up once per
// device (hipGetSymbolAddress with that device current).
constexpr size_t kStaticScratchBytes = size_t{64} << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};   // device address of `scratch` per device (null: not looked up)

// Look up this device's copy of the static scratch array (the current device
// must be `device`); later calls for the same device return at once.
ifvs_status static_scratch_bind(int device) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (device < 0 || device >= kMaxDevices)
    return fail(IFVS_E_UNSUPPORTED, "device ordinal " + std::to_string(device) + " beyond the static scratch table");
  if (g_scratch_dev[device]) return IFVS_OK;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || p == nullptr) {
    (void)hipGetLastError();
    return fail(IFVS_E_HIP, std::string("locating the static scratch array: ") + hipGetErrorString(e));
  }
  g_scratch_dev[device] = p;
  return IFVS_OK;
}

void* static_scratch_ptr(int device) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return device >= 0 && device < kMaxDevices ? g_scratch_dev[device] : nullptr;
}

// The coarse quantizer and the second copy of the codes in list order
// (rows grouped by sub-list: centroid and radius band, each sub-list in
// layout order), with the list plan's workspace.  Null words: none built.
struct CoarseLists {
  int C = 0;
  int f_shift = 12;
  uint32_t* words = nullptr;     // [n_tiles * 64] layout row: centroid id | radius (bfloat16, rounded up)
  uint8_t* band = nullptr;       // [n] layout row: radius band within its list
  uint32_t* cc_t = nullptr;      // [mw][C] centroid code words
  int32_t* sub_off = nullptr;    // [C * kBands + 1] sub-list offsets in list order
  float* rmax = nullptr;         // [C * kBands] largest radius of each sub-list
  int32_t* cnt_f = nullptr;      // [(n >> f_shift) + 1][C * kBands]
  uint32_t* codes_t = nullptr;   // [n_tiles][mw][64] list order
  int32_t* ids = nullptr;        // [n_tiles * 64] list position -> original id
  int32_t* lrow = nullptr;       // [n] list position -> layout row
  int32_t* it_r0 = nullptr;      // [max_batch][C * kBands] list plan items
  int32_t* it_r1 = nullptr;
  int32_t* it_t = nullptr;
  float* it_lb = nullptr;
  float* hdr = nullptr;          // [max_batch][4]
  uint32_t* slots = nullptr;     // [max_batch][kListSlots]
  int4* jobs = nullptr;          // [max_batch * kListJobs] list scan job table
  int32_t* n_keys = nullptr;     // [max_batch] partial keys written per query position
  int32_t* job_ctr = nullptr;    // [2] next job, job count

  void release() {
    for (void* p : {static_cast<void*>(words), static_cast<void*>(band), static_cast<void*>(cc_t),
                    static_cast<void*>(sub_off), static_cast<void*>(rmax), static_cast<void*>(cnt_f),
                    static_cast<void*>(codes_t), static_cast<void*>(ids),
                    static_cast<void*>(lrow),
                    static_cast<void*>(it_r0),
                    static_cast<void*>(it_r1), static_cast<void*>(it_t),
                    static_cast<void*>(it_lb), static_cast<void*>(hdr), static_cast<void*>(slots),
                    static_cast<void*>(jobs), static_cast<void*>(n_keys), static_cast<void*>(job_ctr)})
      if (p) (void)hipFree(p);
    *this = CoarseLists{};
  }
};

}  // namespace

struct ifvs_index {
  int device = 0;
  int64_t n = 0;
  int dim = 0, m = 0, dsub = 0, n_attr = 0;
  int bank_rows = 0, r = 0, h = 0;
  uint64_t hash_seed = 0;
  int mw = 0;
  int64_t n_tiles = 0;
  int max_batch = 0, max_k = 0;
  int n_cluster = 0, c0 = -1, c1 = -1;

  uint32_t* codes_t = nullptr;   // [n_tiles][mw][64] code words, physical row order
  float* cpq = nullptr;          // [m][256][dsub]
  float* sdc = nullptr;          // [m][256][256] codeword-to-codeword squared distances
  int32_t* attrs = nullptr;      // [n_attr][n] original id order
  int32_t* attrs_phys = nullptr; // [n_attr][n] physical order (== attrs when not clustered)
  // Leading cluster key value table: vstart[t] = first physical row whose key
  // is >= vmin + t (t < vcount, last entry n); null when the key's value
  // range is too wide.
  int32_t* vstart = nullptr;
  int64_t vmin = 0, vcount = 0;
  int32_t* perm = nullptr;       // physical row -> original id (null when not clustered)
  float* bank = nullptr;         // [bank_rows][m*r]
  float* W = nullptr;            // [m][r][256][dsub]

  DevPred* preds_dev = nullptr;  // [max_batch]
  int32_t* qorder_dev = nullptr; // [max_batch]
  int64_t* iv_dev = nullptr;     // [max_batch][2]
  uint64_t* gthr_dev = nullptr;  // [max_batch] shared scan thresholds
  float* bound_parts = nullptr;  // [max_batch][2][m] coarse-bound partial maxima
  int32_t* slot_order_dev = nullptr;  // [slot_order_cap] chunk-grid scan dispatch order
  int64_t slot_order_cap = 0;
  DevPred* staging[kStagingSlots] = {};   // pinned: [max_batch] DevPred + [max_batch] int32
  DevPred* staging_dev[kStagingSlots] = {};  // the same slots as the device addresses them
  hipEvent_t staged[kStagingSlots] = {};
  bool slot_busy[kStagingSlots] = {};
  // A slot released through a done word (StageDone) instead of its event:
  // the slot is free once done_host[slot] == slot_seq[slot].
  bool slot_by_word[kStagingSlots] = {};
  uint64_t slot_seq[kStagingSlots] = {};
  uint64_t* done_host = nullptr;   // pinned [kStagingSlots]
  uint64_t* done_dev = nullptr;    // the same words as the device addresses them
  uint64_t release_seq = 0;
  int next_slot = 0;

  uint64_t* bitmap = nullptr;    // [max_batch][stride64]
  int64_t stride64 = 0;
  unsigned long long* counts = nullptr;  // [max_batch]
  uint32_t* count_parts = nullptr;       // [max_batch][filter_count_parts(n)] per-workgroup pool sizes
  uint64_t* partials = nullptr;  // per-wavefront top-k keys
  size_t partial_keys = 0;
  // Gather scan of masked batches (null when M has no gather kernel).
  uint32_t* codes_rm = nullptr;  // [n][rw] row-major code words, physical order
  int rw = 0;
  int32_t* lists = nullptr;      // [max_batch][list_cap] selected physical rows
  int32_t* list_n = nullptr;     // [max_batch]
  int32_t* qmode = nullptr;      // [max_batch] 1: gather scan
  int64_t list_cap = 0;

  // Full-precision vectors (ifvs_load_vectors) and the exact search's
  // workspace.
  float* xt = nullptr;           // [ceil(n/64)][dim][64] fp32, physical order
  float* xr = nullptr;           // [n][dim] fp32, physical order
  uint4* xb = nullptr;           // [ceil(n/32)][ksteps][64] bf16 fragments
  float* xn = nullptr;           // [ceil(n/32)*32] squared norms
  unsigned* xmax = nullptr;      // largest row norm (fp32 bits)
  unsigned long long* xbad = nullptr;
  uint4* qb = nullptr;           // query fragments
  float* qn_x = nullptr;         // [max_batch] |q|^2
  float* eps_x = nullptr;        // [max_batch] screening error bounds
  float* thr_x = nullptr;        // [max_batch] candidate bounds
  float* bins_x = nullptr;       // [max_batch][bins_cap]
  int64_t bins_cap = 0;
  int exact_splits_max = 0;
  int32_t* cand_x = nullptr;     // [max_batch][cand_cap]
  int32_t* cand_n_x = nullptr;   // [max_batch]
  int64_t cand_cap = 0;
  uint64_t* partials_x = nullptr;  // [max_batch][exact_chunks_max][max_k]
  int exact_chunks_max = 0;

  // Training workspace (ifvs_train_step), allocated on its first call.
  float* tr_alpha = nullptr;     // [max_batch][m*r]
  float* tr_wf = nullptr;        // [max_batch][dim]
  float* tr_lut = nullptr;       // [max_batch][m][256]
  float* tr_gdelta = nullptr;    // [max_batch][m][256][dsub]
  float* tr_galpha = nullptr;    // [max_batch][m*r]
  int32_t* tr_rows = nullptr;    // [max_batch][h]
  int32_t* inv_perm = nullptr;   // original id -> physical row (clustered layouts)

  // Every (n / kFences)-th clustered key, copied to the host at load: lets
  // the planner estimate each query's interval length without touching the
  // device.
  std::vector<int32_t> fence0, fence1;

  int opt_qtile = 0, opt_splits = 0, opt_min_chunk = 0;
  int64_t opt_grid_tiles = 0;
  int opt_gather = 0;   // 0 automatic, 1 every query whose list fits, 2 never
  int opt_grid_relative = 0;   // 1: grid chunks relative to each query tile's first cell
  int opt_slot_order = 0;      // 0: chunk-grid slots in estimated-work order, 1: in index order
  int opt_exact_plan = 0;      // ifvs_exact_search: 0 automatic, 1 direct, 2 screened
  int opt_shared_bound = 0;    // workgroup bound from the wavefronts' best distances: 0 auto, 1 off, 2 on
  int opt_seed_tiles = 0;      // seeded bound: 0 auto, 1 off, n > 1 at most n tiles per wavefront
  int opt_gather_auto_pct = 30;   // automatic mode: pools up to this % of the rows
  int profile_mask = 0;          // stages timed with HIP events (IFVS_OPT_PROFILE)
  // IFVS_OPT_COUNT_READS: scans run the read-counting build, which adds its
  // table reads by active lanes into this device histogram ([65]).
  int opt_count_reads = 0;
  unsigned long long* read_hist = nullptr;
  // Predicate encoder (ifvs_load_encoder); null params: none attached.
  float* enc_params = nullptr;
  double* enc_off = nullptr;     // [n_attr]
  double* enc_scale = nullptr;   // [n_attr]
  int enc_H = 0, enc_heads = 0, enc_layers = 0, enc_F = 0;
  // Coarse quantizer and the list order of the codes (ifvs_build_coarse).
  CoarseLists coarse;
  int opt_coarse = 0;                // 0 automatic, 1 never, 2 whenever the batch allows the list scan
  StageTimer* timers = nullptr;  // [kStages] once profiling was enabled
  ScanPlan last_plan{};
  bool last_coarse = false;

  void free_vectors() {
    for (void* p : {static_cast<void*>(xt), static_cast<void*>(xr), static_cast<void*>(xb), static_cast<void*>(xn),
                    static_cast<void*>(xmax), static_cast<void*>(xbad), static_cast<void*>(qb),
                    static_cast<void*>(qn_x), static_cast<void*>(eps_x), static_cast<void*>(thr_x),
                    static_cast<void*>(bins_x), static_cast<void*>(cand_x), static_cast<void*>(cand_n_x),
                    static_cast<void*>(partials_x)})
      if (p) hipFree(p);
    xt = nullptr;
    xr = nullptr;
    xb = nullptr;
    xn = nullptr;
    xmax = nullptr;
    xbad = nullptr;
    qb = nullptr;
    qn_x = eps_x = thr_x = bins_x = nullptr;
    cand_x = cand_n_x = nullptr;
    partials_x = nullptr;
  }

  ~ifvs_index() {
    hipSetDevice(device);
    hipDeviceSynchronize();
    if (timers) {
      for (int st = 0; st < kStages; ++st)
        for (hipEvent_t e : timers[st].ev)
          if (e) hipEventDestroy(e);
      delete[] timers;
    }
    if (attrs_phys && attrs_phys != attrs) hipFree(attrs_phys);
    for (void* p : {static_cast<void*>(codes_t), static_cast<void*>(cpq), static_cast<void*>(sdc),
                    static_cast<void*>(attrs),
                    static_cast<void*>(perm), static_cast<void*>(bank), static_cast<void*>(W),
                    static_cast<void*>(preds_dev), static_cast<void*>(qorder_dev),
                    static_cast<void*>(iv_dev), static_cast<void*>(gthr_dev), static_cast<void*>(bitmap),
                    static_cast<void*>(bound_parts),
                    static_cast<void*>(slot_order_dev),
                    static_cast<void*>(counts), static_cast<void*>(count_parts), static_cast<void*>(vstart),
                    static_cast<void*>(partials), static_cast<void*>(codes_rm),
                    static_cast<void*>(lists), static_cast<void*>(list_n), static_cast<void*>(qmode),
                    static_cast<void*>(read_hist), static_cast<void*>(enc_params),
                    static_cast<void*>(enc_off), static_cast<void*>(enc_scale)})
      if (p) hipFree(p);
    free_vectors();
    coarse.release();
    for (void* p : {static_cast<void*>(tr_alpha), static_cast<void*>(tr_wf), static_cast<void*>(tr_lut),
                    static_cast<void*>(tr_gdelta), static_cast<void*>(tr_galpha), static_cast<void*>(tr_rows),
                    static_cast<void*>(inv_perm)})
      if (p) hipFree(p);
    for (int i = 0; i < kStagingSlots; ++i) {
      if (staging[i]) hipHostFree(staging[i]);
      if (staged[i]) hipEventDestroy(staged[i]);
    }
    if (done_host) hipHostFree(done_host);
  }
};

namespace {

template <typename T>
ifvs_status dev_alloc(T** p, size_t count, const char* what) {
  *p = nullptr;
  if (count == 0) count = 1;
  if (forced_alloc_failure()) return fail(IFVS_E_NOMEM, std::string("forced allocation failure: ") + what);
  const hipError_t e = hipMalloc(reinterpret_cast<void**>(p), count * sizeof(T));
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(IFVS_E_NOMEM, std::string("device allocation failed: ") + what);
  }
  return IFVS_OK;
}

// Device memory one filtered search works in: the index's workspace, or, for
// ifvs_filtered_search_noalloc, pieces of the library's static scratch array.
struct SearchWs {
  DevPred* preds = nullptr;          // [nq] normalized predicates
  int32_t* qorder = nullptr;         // [nq] scan order
  int64_t* iv = nullptr;             // [nq][2] row intervals
  uint64_t* gthr = nullptr;          // [nq] shared scan thresholds
  int32_t* slot_order = nullptr;     // chunk-grid dispatch order
  int64_t slot_order_cap = 0;
  uint64_t* bitmap = nullptr;        // [nq][stride64] selection words (null: batch needs none)
  int64_t stride64 = 0;
  unsigned long long* counts = nullptr;  // pool sizes and their per-part prefix sums (gather scan)
  uint32_t* count_parts = nullptr;
  int32_t* lists = nullptr;          // [nq][list_cap] row lists (null: no gather scan)
  int32_t* list_n = nullptr;
  int32_t* qmode = nullptr;
  int64_t list_cap = 0;
  uint64_t* partials = nullptr;      // per-wavefront top-k keys
  size_t partial_keys = 0;
};

SearchWs index_ws(const ifvs_index* idx) {
  SearchWs w;
  w.preds = idx->preds_dev;
  w.qorder = idx->qorder_dev;
  w.iv = idx->iv_dev;
  w.gthr = idx->gthr_dev;
  w.slot_order = idx->slot_order_dev;
  w.slot_order_cap = idx->slot_order_cap;
  w.bitmap = idx->bitmap;
  w.stride64 = idx->stride64;
  w.counts = idx->counts;
  w.count_parts = idx->count_parts;
  w.lists = idx->lists;
  w.list_n = idx->list_n;
  w.qmode = idx->qmode;
  w.list_cap = idx->list_cap;
  w.partials = idx->partials;
  w.partial_keys = idx->partial_keys;
  return w;
}

// The search's workspace carved from the device's static scratch array, in
// 256-byte aligned pieces: predicates, scan order, intervals, thresholds,
// selection bitmaps when the batch needs them, the dispatch order, and all
// the rest for top-k partials (the planner keeps the chunk count within it).
// Nothing in it needs to start at zero: the interval kernel resets the
// thresholds, and every other piece is written before it is read.
ifvs_status carve_static_ws(const ifvs_index* idx, int32_t nq, int32_t k, bool bitmaps, SearchWs* ws) {
  char* base = static_cast<char*>(static_scratch_ptr(idx->device));
  if (!base) return fail(IFVS_E_STATE, "the static scratch array of this device was not looked up");
  size_t used = 0;
  auto take = [&](size_t bytes) {
    used = (used + 255) & ~size_t{255};
    char* p = base + used;
    used += bytes;
    return p;
  };
  const size_t n = static_cast<size_t>(nq);
  ws->preds = reinterpret_cast<DevPred*>(take(sizeof(DevPred) * n));
  ws->qorder = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * n));
  ws->iv = reinterpret_cast<int64_t*>(take(2 * sizeof(int64_t) * n));
  ws->gthr = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * n));
  ws->stride64 = idx->stride64;
  ws->bitmap = bitmaps ? reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * n * idx->stride64)) : nullptr;
  ws->slot_order_cap = std::min<int64_t>(idx->slot_order_cap, int64_t{1} << 18);
  ws->slot_order = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * ws->slot_order_cap));
  used = (used + 255) & ~size_t{255};
  const size_t min_partials = n * kScanWaves * static_cast<size_t>(k) * sizeof(uint64_t);
  if (used + min_partials > kStaticScratchBytes)
    return fail(IFVS_E_INVALID, "this batch needs " + std::to_string(used + min_partials) +
                                    " bytes of scratch, more than the " + std::to_string(kStaticScratchBytes) +
                                    " bytes of the allocation-free search (fewer queries, or ifvs_filtered_search)");
  ws->partials = reinterpret_cast<uint64_t*>(base + used);
  ws->partial_keys = (kStaticScratchBytes - used) / sizeof(uint64_t);
  return IFVS_OK;
}

ifvs_status check_index(const ifvs_index* idx) {
  if (!idx) return fail(IFVS_E_STATE, "NULL index handle");
  return IFVS_OK;
}

ifvs_status check_nq(const ifvs_index* idx, int32_t nq) {
  if (nq < 0 || nq > idx->max_batch)
    return fail(IFVS_E_INVALID, "nq = " + std::to_string(nq) + " outside 0.." +
                                    std::to_string(idx->max_batch) + " (max_batch)");
  return IFVS_OK;
}

// Validate the caller's predicates and turn them into DevPred records: the
// effective int32 clauses, and on a clustered index the row interval of the
// cluster-key clauses plus the residual clauses still tested per row.
ifvs_status normalize_predicates(const ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                                 DevPred* out) {
  if (nq > 0 && !preds) return fail(IFVS_E_INVALID, "preds is NULL");
  for (int32_t i = 0; i < nq; ++i) {
    const ifvs_predicate& p = preds[i];
    if (p.n_clauses < 0 || p.n_clauses > IFVS_MAX_CLAUSES)
      return fail(IFVS_E_INVALID, "query " + std::to_string(i) + ": n_clauses = " +
                                      std::to_string(p.n_clauses) + " outside 0..4");
    if (p.reserved != 0) return fail(IFVS_E_INVALID, "query " + std::to_string(i) + ": reserved field not 0");
    DevPred d{};
    d.n_raw = p.n_clauses;
    int n_eff = 0;
    bool empty = false;
    int eff_col[kMaxClauses];
    // Intersections of the clauses on the two cluster columns.
    int64_t lo0 = kI32Min, hi0 = kI32End, lo1 = kI32Min, hi1 = kI32End;
    bool has0 = false, has1 = false;
    for (int c = 0; c < p.n_clauses; ++c) {
      const ifvs_clause& cl = p.c[c];
      if (cl.col < 0 || cl.col >= idx->n_attr)
        return fail(IFVS_E_INVALID, "query " + std::to_string(i) + ": clause " + std::to_string(c) +
                                        " column " + std::to_string(cl.col) + " outside 0.." +
                                        std::to_string(idx->n_attr - 1));
      if (cl.reserved != 0)
        return fail(IFVS_E_INVALID, "query " + std::to_string(i) + ": clause reserved field not 0");
      d.raw_col[c] = cl.col;
      d.raw_lo[c] = cl.lo;
      d.raw_hi[c] = cl.hi;
      // Intersect [lo, hi) with the int32 range.
      const int64_t lo = std::max<int64_t>(cl.lo, kI32Min);
      const int64_t hi = std::min<int64_t>(cl.hi, kI32End);
      if (cl.lo >= cl.hi || lo >= hi) {
        empty = true;
        continue;
      }
      if (idx->n_cluster > 0 && cl.col == idx->c0) {
        has0 = true;
        lo0 = std::max(lo0, lo);
        hi0 = std::min(hi0, hi);
      }
      if (idx->n_cluster > 1 && cl.col == idx->c1) {
        has1 = true;
        lo1 = std::max(lo1, lo);
        hi1 = std::min(hi1, hi);
      }
      const uint64_t width = static_cast<uint64_t>(hi - lo);
      if (width >= (1ull << 32)) continue;           // admits every int32 value
      d.col[n_eff] = cl.col;
      d.lo[n_eff] = static_cast<int32_t>(lo);
      d.width[n_eff] = static_cast<uint32_t>(width);
      eff_col[n_eff] = cl.col;
      ++n_eff;
    }
    d.n_eff = empty ? -1 : n_eff;
    // Interval of the cluster-key clauses; everything else stays residual.
    d.iv_mode = 0;
    if (has0 && lo0 < hi0) {
      if (has1 && hi0 - lo0 == 1) {
        d.iv_mode = 2;
        d.iv_lo0 = lo0;
        d.iv_hi0 = hi0;
        d.iv_lo1 = lo1;
        d.iv_hi1 = std::max(lo1, hi1);
      } else {
        d.iv_mode = 1;
        d.iv_lo0 = lo0;
        d.iv_hi0 = hi0;
      }
    } else if (has0) {
      d.n_eff = -1;                                   // contradictory clauses on c0
    }
    int resid = 0;
    for (int c = 0; c < n_eff; ++c) {
      const bool covered = (d.iv_mode >= 1 && eff_col[c] == idx->c0) ||
                           (d.iv_mode == 2 && eff_col[c] == idx->c1);
      if (!covered) resid |= 1 << c;
    }
    d.residual_mask = d.n_eff < 0 ? 0 : resid;
    d.n_res = 0;
    for (int c = 0; c < n_eff; ++c) {
      if (!((d.residual_mask >> c) & 1)) continue;
      d.res_col[d.n_res] = d.col[c];
      d.res_lo[d.n_res] = d.lo[c];
      d.res_width[d.n_res] = d.width[c];
      ++d.n_res;
    }
    out[i] = d;
  }
  return IFVS_OK;
}

// Estimated 64-row tiles [*t_lo, *t_hi) of a query's cluster-key interval,
// from the fences (widened by one fence gap on each side).
void estimate_interval_range(const ifvs_index* idx, const DevPred& d, int64_t* t_lo, int64_t* t_hi) {
  const auto& f0 = idx->fence0;
  const auto& f1 = idx->fence1;
  const int64_t nf = static_cast<int64_t>(f0.size());
  *t_lo = *t_hi = 0;
  if (d.n_eff < 0 || nf == 0) return;
  if (d.iv_mode == 0) {
    *t_hi = idx->n_tiles;
    return;
  }
  auto rank = [&](int64_t x0, int64_t x1) {      // fences below (x0, x1)
    int64_t lo = 0, hi = nf;
    while (lo < hi) {
      const int64_t mid = (lo + hi) / 2;
      const bool below = d.iv_mode == 2 && f0[mid] == x0 ? f1[mid] < x1 : f0[mid] < x0;
      if (below) lo = mid + 1;
      else hi = mid;
    }
    return lo;
  };
  const int64_t r0 = d.iv_mode == 2 ? rank(d.iv_lo0, d.iv_lo1) : rank(d.iv_lo0, 0);
  const int64_t r1 = d.iv_mode == 2 ? rank(d.iv_lo0, d.iv_hi1) : rank(d.iv_hi0, 0);
  const int64_t row_lo = std::max<int64_t>(0, r0 - 1) * idx->n / (nf - 1);
  const int64_t row_hi = std::min<int64_t>(idx->n, r1 * idx->n / (nf - 1));
  *t_lo = std::min<int64_t>(idx->n_tiles, row_lo / 64);
  *t_hi = std::min<int64_t>(idx->n_tiles, std::max<int64_t>(*t_lo, (row_hi + 63) / 64));
}

// Estimated 64-row tiles of a query's cluster-key interval.
int64_t estimate_interval_tiles(const ifvs_index* idx, const DevPred& d) {
  int64_t lo = 0, hi = 0;
  estimate_interval_range(idx, d, &lo, &hi);
  return hi - lo;
}

// Dispatch order of a chunk-grid scan's slots.  Slot (query tile t, cell c)
// of XCD x is item c * per_xcd + (t - x * per_xcd); out[x * per_xcd * splits
// + i] is XCD x's i-th item.  Every item of every XCD appears once.  Items
// whose estimated work is a whole cell come first, in cell order (all XCDs
// walk the same cells together), then the rest by decreasing estimated work
// in steps of 1/16 cell, and the estimated-empty ones last: the workgroups
// dispatched last are short, so fewer CUs idle at the end of the launch.
void order_scan_slots(const ifvs_index* idx, const DevPred* host, const int32_t* qorder, int nq,
                      const ScanPlan& plan, int32_t* out) {
  const int n_qtiles = (nq + plan.qtile - 1) / plan.qtile;
  const int per_xcd = (n_qtiles + 7) / 8;
  const int64_t g = plan.chunk_tiles;
  const int64_t step = std::max<int64_t>(1, g / 16);
  std::vector<int64_t> hull_lo(n_qtiles, 0), hull_hi(n_qtiles, 0);
  for (int t = 0; t < n_qtiles; ++t) {
    int64_t lo = INT64_MAX, hi = 0;
    for (int qi = 0; qi < plan.qtile && t * plan.qtile + qi < nq; ++qi) {
      int64_t a = 0, b = 0;
      estimate_interval_range(idx, host[qorder[t * plan.qtile + qi]], &a, &b);
      if (b > a) {
        lo = std::min(lo, a);
        hi = std::max(hi, b);
      }
    }
    if (hi > lo) {
      hull_lo[t] = lo;
      hull_hi[t] = hi;
    }
  }
  constexpr int kBuckets = 18;   // 0: empty, 1..16: partial in 1/16-cell steps, 17: whole cell
  const int64_t items = static_cast<int64_t>(per_xcd) * plan.splits;
  std::vector<uint8_t> bucket(static_cast<size_t>(items));
  for (int x = 0; x < 8; ++x) {
    int64_t count[kBuckets] = {};
    for (int c = 0; c < plan.splits; ++c) {
      for (int ql = 0; ql < per_xcd; ++ql) {
        const int t = x * per_xcd + ql;
        int64_t work = 0;
        if (t < n_qtiles) work = std::max<int64_t>(0, std::min(hull_hi[t], (c + 1) * g) - std::max(hull_lo[t], c * g));
        const int b = work >= g ? kBuckets - 1 : (work == 0 ? 0 : 1 + static_cast<int>(std::min<int64_t>(15, work / step)));
        bucket[static_cast<size_t>(c) * per_xcd + ql] = static_cast<uint8_t>(b);
        ++count[b];
      }
    }
    int64_t start[kBuckets];
    int64_t pos = 0;
    for (int b = kBuckets - 1; b >= 0; --b) {
      start[b] = pos;
      pos += count[b];
    }
    int32_t* o = out + x * items;
    for (int64_t i = 0; i < items; ++i) o[start[bucket[i]]++] = static_cast<int32_t>(i);
  }
}

// Wait until the kernel carrying slot's StageDone has started (its word
// holds the slot's sequence number).  The word is written from the device
// over the host link; after about a second of polling the device is
// synchronized once, after which it must hold the number.
ifvs_status wait_done_word(ifvs_index* idx, int slot) {
  const uint64_t want = idx->slot_seq[slot];
  const auto t0 = std::chrono::steady_clock::now();
  while (__atomic_load_n(&idx->done_host[slot], __ATOMIC_ACQUIRE) != want) {
    if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(1)) {
      IFVS_HIP(hipDeviceSynchronize(), "waiting for staging slot");
      if (__atomic_load_n(&idx->done_host[slot], __ATOMIC_ACQUIRE) != want)
        return fail(IFVS_E_HIP, "staging slot " + std::to_string(slot) + ": its done word was not written");
      break;
    }
    std::this_thread::yield();
  }
  return IFVS_OK;
}

// Validate and normalize predicates into the next pinned staging slot (and
// the scan's query order, when asked).  With copy_to_device the slot is
// copied to the device workspace and released at once; otherwise the
// caller's kernels read the slot itself (one wavefront-wide load per
// predicate) and the caller releases it after enqueuing the last of them.
ifvs_status stage_predicates(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                             bool with_order, bool copy_to_device, hipStream_t s, int* slot_out,
                             DevPred** host_out = nullptr) {
  const int slot = idx->next_slot;
  if (idx->slot_busy[slot] && idx->slot_by_word[slot]) {
    if (ifvs_status st = wait_done_word(idx, slot); st != IFVS_OK) return st;
  } else if (idx->slot_busy[slot]) {
    IFVS_HIP(hipEventSynchronize(idx->staged[slot]), "waiting for staging slot");
  }
  idx->slot_busy[slot] = false;
  idx->slot_by_word[slot] = false;
  DevPred* host = idx->staging[slot];
  const ifvs_status st = normalize_predicates(idx, nq, preds, host);
  if (st != IFVS_OK) return st;
  idx->next_slot = (slot + 1) % kStagingSlots;
  if (with_order) {
    // Scan order: queries with nearby cluster-key intervals next to each
    // other, so that a query tile's intervals overlap; stable by index.
    int32_t* order = reinterpret_cast<int32_t*>(host + idx->max_batch);
    std::iota(order, order + nq, 0);
    std::stable_sort(order, order + nq, [&](int32_t a, int32_t b) {
      const DevPred& x = host[a];
      const DevPred& y = host[b];
      if (x.iv_mode != y.iv_mode) return x.iv_mode < y.iv_mode;
      if (x.iv_lo0 != y.iv_lo0) return x.iv_lo0 < y.iv_lo0;
      return x.iv_lo1 < y.iv_lo1;
    });
  }
  if (copy_to_device) {
    IFVS_HIP(hipMemcpyAsync(idx->preds_dev, host, sizeof(DevPred) * nq, hipMemcpyHostToDevice, s),
             "copying predicates");
    IFVS_HIP(hipEventRecord(idx->staged[slot], s), "recording staging event");
    idx->slot_busy[slot] = true;
  }
  *slot_out = slot;
  if (host_out) *host_out = host;
  return IFVS_OK;
}

// A slot released through its done word: the word is set by the kernel that
// carries the StageDone, which starts only after the slot's readers ran.
StageDone slot_done_word(ifvs_index* idx, int slot) {
  idx->slot_seq[slot] = ++idx->release_seq;
  return StageDone{idx->done_dev + slot, idx->slot_seq[slot]};
}

void release_slot_by_word(ifvs_index* idx, int slot) {
  idx->slot_busy[slot] = true;
  idx->slot_by_word[slot] = true;
}

// The slot's readers are enqueued on s: it may be reused once they ran.
ifvs_status release_slot(ifvs_index* idx, int slot, hipStream_t s) {
  IFVS_HIP(hipEventRecord(idx->staged[slot], s), "recording staging event");
  idx->slot_busy[slot] = true;
  return IFVS_OK;
}

// Fold recorded event pairs of one stage into its total.
ifvs_status flush_timer(StageTimer& t) {
  if (t.used == 0) return IFVS_OK;
  IFVS_HIP(hipEventSynchronize(t.ev[t.used - 1]), "waiting for profile events");
  for (int i = 0; i + 1 < t.used; i += 2) {
    float ms = 0.0f;
    IFVS_HIP(hipEventElapsedTime(&ms, t.ev[i], t.ev[i + 1]), "reading profile events");
    t.ms += ms;
    ++t.launches;
  }
  t.used = 0;
  return IFVS_OK;
}

// Launch through `fn`, bracketed by events when profiling.
template <typename Fn>
ifvs_status timed(ifvs_index* idx, int stage, hipStream_t s, const char* what, Fn&& fn) {
  StageTimer* t = (idx->profile_mask >> stage) & 1 ? &idx->timers[stage == kStListScan ? kStScan : stage] : nullptr;
  if (t) {
    if (t->used + 2 > 2 * kProfilePairs)
      if (ifvs_status st = flush_timer(*t); st != IFVS_OK) return st;
    IFVS_HIP(hipEventRecord(t->ev[t->used++], s), "recording profile event");
  }
  IFVS_HIP(fn(), what);
  if (t) IFVS_HIP(hipEventRecord(t->ev[t->used++], s), "recording profile event");
  return IFVS_OK;
}

#define IFVS_LAUNCH(idx, stage, s, what, expr)                                                  \
  do {                                                                                          \
    const ifvs_status st_ = timed(idx, stage, s, what, [&]() -> hipError_t { return (expr); }); \
    if (st_ != IFVS_OK) return st_;                                                             \
  } while (0)

// Largest pool (rows) the automatic mode scores from a row list.
int64_t gather_auto_rows(const ifvs_index* idx) { return idx->n * idx->opt_gather_auto_pct / 100; }

// interval_batch: every query has a cluster-key interval; one query per tile
// then keeps all lanes busy and the scan is bound by LDS lookups, so sharing
// code tiles across queries would not help.  Otherwise (masked rows) tiles
// of several queries share each pass over the codes.
ifvs_status plan_scan(const ifvs_index* idx, int32_t nq, int32_t k, int32_t lut_dtype,
                      bool interval_batch, int64_t span_tiles, size_t partial_keys, ScanPlan* plan) {
  const int lut_bytes = lut_dtype == IFVS_LUT_F16 ? 2 : 4;
  const int qmax = scan_max_qtile(idx->m, lut_bytes, k);
  if (qmax < 1)
    return fail(IFVS_E_UNSUPPORTED, "one query's distance table (" + std::to_string(idx->m) +
                                        " x 256 x " + std::to_string(lut_bytes) +
                                        " B) plus its top-k pools exceeds the 160 KB LDS budget; use IFVS_LUT_F16");
  int want = idx->opt_qtile > 0 ? idx->opt_qtile : (interval_batch ? 1 : 8);
  want = std::min(want, std::max(1, nq));
  want = std::min(want, qmax);
  plan->qtile = std::max(1, scan_supported_qtile(want));
  const int64_t gy = (std::max(1, nq) + plan->qtile - 1) / plan->qtile;
  // Interval scans: at least 8 tiles per wavefront per chunk, so the table
  // staged into LDS is amortized over >= 512 rows.
  plan->min_chunk = idx->opt_min_chunk > 0 ? idx->opt_min_chunk : (interval_batch ? 8 * kScanWaves : 16);
  // Masked scans: enough workgroups to fill 256 CUs several times.  Interval
  // scans: chunks of about 8192 tiles (measured best between 2K and 8K
  // tiles per 8-wavefront workgroup), at least ~512 workgroups, at most 16
  // chunks per query tile.
  int64_t splits = (4096 + gy - 1) / gy;
  plan->chunk_tiles = 0;
  plan->abs_cells = false;
  plan->seed_tiles = 0;
  if (interval_batch) {
    // Long spans (>= 8192 tiles) are cut on a chunk grid of cells of about
    // 5K tiles (measured best between 4K and 5K on 10M x 48-byte codes), so
    // queries with nearby spans read the same cells at the same time; a span
    // not aligned to the grid touches one cell more.  Short spans are cut
    // into equal chunks, at least ~512 workgroups per batch.
    if (idx->opt_grid_tiles > 0) {
      plan->chunk_tiles = idx->opt_grid_tiles;
    } else if (span_tiles >= 8192) {
      const int64_t cells = (span_tiles + 5119) / 5120;
      plan->chunk_tiles = (span_tiles + cells - 1) / cells;
    }
    // Seeded bound (one query per tile, tables of a fixed M).  Automatic on
    // chunk-grid cells, each wavefront ranking its first 64 tiles of the
    // cell (6-9% less scan time at 10% and 50% selectivity on 10M x 48-byte
    // codes).  Short intervals end before a wavefront's own k-th key gets
    // close, but the seed must then rank nearly every tile of the query to
    // find its k nearest rows, and every workgroup of the query pays for it:
    // measured 4-45% slower at 0.1% and 1%, so only on request there.
    const bool seedable = plan->qtile == 1 && (idx->m == 16 || idx->m == 48 || idx->m == 120) &&
                          k <= kScanWaves * kScanSeed;
    if (seedable && idx->opt_seed_tiles > 1)
      plan->seed_tiles = idx->opt_seed_tiles;
    else if (seedable && idx->opt_seed_tiles == 0 && plan->chunk_tiles > 0)
      plan->seed_tiles = 64;
    // Chunk c is absolute cell c of the grid: every XCD walks the same cells
    // at the same time, so one HBM read of a cell can serve the other XCDs
    // from the Infinity Cache.  Cells a query's interval misses cost one
    // empty workgroup each.
    plan->abs_cells = plan->chunk_tiles > 0 && idx->opt_grid_relative == 0;
    if (plan->abs_cells)
      splits = (idx->n_tiles + plan->chunk_tiles - 1) / plan->chunk_tiles;
    else if (plan->chunk_tiles > 0)
      splits = (span_tiles + plan->chunk_tiles - 1) / plan->chunk_tiles + 1;
    else
      splits = std::min<int64_t>(16, std::max<int64_t>((span_tiles + 8191) / 8192, (512 + gy - 1) / gy));
  }
  if (idx->opt_splits > 0) splits = idx->opt_splits;
  splits = std::min<int64_t>(splits, std::max<int64_t>(1, (idx->n_tiles + plan->min_chunk - 1) / plan->min_chunk));
  const int64_t cap = static_cast<int64_t>(partial_keys /
                                           (static_cast<size_t>(std::max(1, nq)) * kScanWaves * k));
  splits = std::max<int64_t>(1, std::min<int64_t>(splits, std::min<int64_t>(cap, 65535)));
  if (plan->abs_cells && splits != (idx->n_tiles + plan->chunk_tiles - 1) / plan->chunk_tiles) {
    // Absolute cells need exactly one chunk per cell (a forced chunk count
    // or too little partial-list room): chunks relative to each query tile,
    // which handle any count.
    plan->abs_cells = false;
  }
  plan->splits = static_cast<int>(splits);
  plan->kpl = pool_kpl(k);
  plan->pool_stride = pool_stride_for(k);
  // The workgroup bound pays on the longest intervals (measured: 5% less
  // scan time at 50% selectivity on 10M x 48-byte codes, 7% at 10% on 100M x
  // 16-byte codes, both spans of 78K+ tiles) and costs 3-9% on spans of
  // about 16K tiles (10% of 10M, 1% of 100M rows) and more on short ones:
  // its k-th slot needs many wavefronts' best rows before it is tight.
  plan->shared_bound = idx->opt_shared_bound == 2 ||
                       (idx->opt_shared_bound == 0 && plan->chunk_tiles > 0 && span_tiles >= 32768);
  plan->lds_bytes = scan_lds_bytes(idx->m, plan->qtile, lut_bytes, plan->pool_stride);
  return IFVS_OK;
}

ifvs_status filter_into_workspace(ifvs_index* idx, const SearchWs& ws, int32_t nq, bool residual_only,
                                  bool counts, hipStream_t s) {
  IFVS_LAUNCH(idx, kStFilter, s, "launching filter kernel",
              launch_filter(residual_only ? idx->attrs_phys : idx->attrs, idx->n, idx->n_attr,
                            ws.preds, nq, residual_only, ws.bitmap, ws.stride64,
                            counts ? ws.counts : nullptr, ws.count_parts, s));
  return IFVS_OK;
}

ifvs_status copy_bitmaps_out(ifvs_index* idx, const SearchWs& ws, int32_t nq, uint32_t* bitmap_out,
                             hipStream_t s) {
  const size_t words = static_cast<size_t>((idx->n + 31) / 32);
  IFVS_HIP(hipMemcpy2DAsync(bitmap_out, words * 4, ws.bitmap, ws.stride64 * 8, words * 4, nq,
                            hipMemcpyDeviceToDevice, s),
           "copying bitmaps");
  return IFVS_OK;
}

}  // namespace

extern "C" {

const char* ifvs_last_error(void) { return g_error.c_str(); }

ifvs_status ifvs_load_index(const ifvs_index_desc* desc, ifvs_index** out) {
  if (!desc || !out) return fail(IFVS_E_INVALID, "desc or out is NULL");
  *out = nullptr;
  const ifvs_index_desc& d = *desc;
  if (d.n < 1 || d.n >= (int64_t(1) << 31)) return fail(IFVS_E_INVALID, "n must be in 1..2^31-1");
  if (d.dim < 1 || d.dim > 4096) return fail(IFVS_E_INVALID, "dim must be in 1..4096");
  if (d.m < 1 || d.m > 256 || d.dim % d.m != 0) return fail(IFVS_E_INVALID, "m must divide dim and be in 1..256");
  if (d.ksub != IFVS_KSUB) return fail(IFVS_E_INVALID, "ksub must be 256 (8-bit codes)");
  if (d.n_attr < 0 || d.n_attr > IFVS_MAX_ATTR) return fail(IFVS_E_INVALID, "n_attr must be in 0..16");
  if (d.mem_kind != IFVS_MEM_HOST && d.mem_kind != IFVS_MEM_DEVICE) return fail(IFVS_E_INVALID, "unknown mem_kind");
  if (!d.codes || !d.codebook) return fail(IFVS_E_INVALID, "codes or codebook is NULL");
  if (d.n_attr > 0 && !d.attrs) return fail(IFVS_E_INVALID, "attrs is NULL but n_attr > 0");
  if (d.bank_rows < 0) return fail(IFVS_E_INVALID, "bank_rows must be >= 0");
  if (d.bank_rows > 0) {
    if (d.r < 1 || d.r > 64) return fail(IFVS_E_INVALID, "r must be in 1..64");
    if (d.h < 1 || d.h > 16) return fail(IFVS_E_INVALID, "h must be in 1..16");
    if (!d.bank || !d.W) return fail(IFVS_E_INVALID, "bank or W is NULL but bank_rows > 0");
  }
  if (d.max_batch < 1 || d.max_batch > 65535) return fail(IFVS_E_INVALID, "max_batch must be in 1..65535");
  if (d.max_k < 1 || d.max_k > IFVS_MAX_K) return fail(IFVS_E_INVALID, "max_k must be in 1..1024");
  if (d.n_cluster < 0 || d.n_cluster > 2) return fail(IFVS_E_INVALID, "n_cluster must be 0, 1 or 2");
  for (int i = 0; i < d.n_cluster; ++i)
    if (d.cluster_col[i] < 0 || d.cluster_col[i] >= d.n_attr)
      return fail(IFVS_E_INVALID, "cluster_col outside 0..n_attr-1");
  if (d.n_cluster == 2 && d.cluster_col[0] == d.cluster_col[1])
    return fail(IFVS_E_INVALID, "the two cluster columns must differ");

  ifvs_index* idx = new ifvs_index();
  auto bail = [&](ifvs_status st) {
    delete idx;
    return st;
  };
  if (hipError_t e = hipGetDevice(&idx->device); e != hipSuccess) return bail(hip_fail(e, "hipGetDevice"));
  if (ifvs_status st0 = static_scratch_bind(idx->device); st0 != IFVS_OK) return bail(st0);
  idx->n = d.n;
  idx->dim = d.dim;
  idx->m = d.m;
  idx->dsub = d.dim / d.m;
  idx->n_attr = d.n_attr;
  idx->bank_rows = d.bank_rows;
  idx->r = d.bank_rows > 0 ? d.r : 0;
  idx->h = d.bank_rows > 0 ? d.h : 0;
  idx->hash_seed = d.hash_seed;
  idx->mw = (d.m + 3) / 4;
  idx->n_tiles = (d.n + kTileRows - 1) / kTileRows;
  idx->max_batch = d.max_batch;
  idx->max_k = d.max_k;
  idx->n_cluster = d.n_cluster;
  idx->c0 = d.n_cluster > 0 ? d.cluster_col[0] : -1;
  idx->c1 = d.n_cluster > 1 ? d.cluster_col[1] : -1;
  const hipMemcpyKind kind = d.mem_kind == IFVS_MEM_DEVICE ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;

  ifvs_status st;
  if (d.n_attr > 0) {
    const size_t na = static_cast<size_t>(d.n_attr) * d.n;
    if ((st = dev_alloc(&idx->attrs, na, "attributes")) != IFVS_OK) return bail(st);
    if (hipError_t e = hipMemcpy(idx->attrs, d.attrs, na * sizeof(int32_t), kind); e != hipSuccess)
      return bail(hip_fail(e, "loading attributes"));
  }
  idx->attrs_phys = idx->attrs;
  if (d.n_cluster > 0) {
    if ((st = dev_alloc(&idx->perm, static_cast<size_t>(d.n), "cluster permutation")) != IFVS_OK) return bail(st);
    if (hipError_t e = cluster_permutation(idx->attrs, d.n, d.n_cluster, idx->c0, idx->c1, idx->perm, nullptr);
        e != hipSuccess)
      return bail(hip_fail(e, "clustering rows"));
    int32_t* phys = nullptr;
    if ((st = dev_alloc(&phys, static_cast<size_t>(d.n_attr) * d.n, "clustered attributes")) != IFVS_OK)
      return bail(st);
    idx->attrs_phys = phys;
    if (hipError_t e = launch_gather_attrs(idx->attrs, d.n, d.n_attr, idx->perm, phys, nullptr); e != hipSuccess)
      return bail(hip_fail(e, "gathering clustered attributes"));
    // Host copy of every (n / kFences)-th clustered key (planner statistics).
    std::vector<int32_t> col(static_cast<size_t>(d.n));
    for (int c = 0; c < d.n_cluster; ++c) {
      if (hipError_t e = hipMemcpy(col.data(), phys + static_cast<int64_t>(d.cluster_col[c]) * d.n,
                                   sizeof(int32_t) * d.n, hipMemcpyDeviceToHost);
          e != hipSuccess)
        return bail(hip_fail(e, "reading cluster keys"));
      auto& f = c == 0 ? idx->fence0 : idx->fence1;
      f.resize(kFences + 1);
      for (int i = 0; i <= kFences; ++i) f[i] = col[std::min<int64_t>(d.n - 1, static_cast<int64_t>(i) * d.n / kFences)];
      // The leading key is sorted: where its values span at most kMaxValueTable
      // integers, a value -> first-row table turns each interval bound into
      // one load instead of a 64-ary search.
      if (c == 0 && static_cast<int64_t>(col[d.n - 1]) - col[0] + 2 <= kMaxValueTable) {
        const int64_t vmin = col[0];
        const int64_t vcount = static_cast<int64_t>(col[d.n - 1]) - vmin + 2;
        std::vector<int32_t> table(static_cast<size_t>(vcount));
        int64_t row = 0;
        for (int64_t t = 0; t < vcount; ++t) {
          while (row < d.n && col[row] < vmin + t) ++row;
          table[t] = static_cast<int32_t>(row);
        }
        if ((st = dev_alloc(&idx->vstart, static_cast<size_t>(vcount), "cluster key value table")) != IFVS_OK)
          return bail(st);
        if (hipError_t e = hipMemcpy(idx->vstart, table.data(), sizeof(int32_t) * vcount, hipMemcpyHostToDevice);
            e != hipSuccess)
          return bail(hip_fail(e, "loading cluster key value table"));
        idx->vmin = vmin;
        idx->vcount = vcount;
      }
    }
  }
  // codes -> 64-row tiles (in physical order)
  {
    uint8_t* tmp = nullptr;
    if ((st = dev_alloc(&tmp, static_cast<size_t>(d.n) * d.m, "codes staging")) != IFVS_OK) return bail(st);
    if ((st = dev_alloc(&idx->codes_t, static_cast<size_t>(idx->n_tiles) * idx->mw * 64, "codes")) != IFVS_OK) {
      hipFree(tmp);
      return bail(st);
    }
    hipError_t e = hipMemcpy(tmp, d.codes, static_cast<size_t>(d.n) * d.m, kind);
    if (e == hipSuccess)
      e = launch_relayout_codes(tmp, d.n, d.m, idx->mw, idx->perm, idx->codes_t, idx->n_tiles, nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    hipFree(tmp);
    if (e != hipSuccess) return bail(hip_fail(e, "loading codes"));
  }
  // Row-major copy of the codes and the row lists for the gather scan.
  if (gather_supported(d.m, IFVS_LUT_F16)) {
    idx->rw = gather_row_words(d.m);
    if ((st = dev_alloc(&idx->codes_rm, static_cast<size_t>(d.n) * idx->rw, "row-major codes")) != IFVS_OK)
      return bail(st);
    if (hipError_t e = launch_rowmajor_codes(idx->codes_t, d.n, idx->mw, idx->rw, idx->codes_rm, nullptr);
        e != hipSuccess)
      return bail(hip_fail(e, "building row-major codes"));
    // Lists hold up to 30% of the rows, capped at 2 GiB for the whole batch.
    const int64_t by_rows = (3 * d.n + 9) / 10;
    const int64_t by_bytes = std::max<int64_t>(4096, (int64_t(2) << 30) / (4 * static_cast<int64_t>(d.max_batch)));
    idx->list_cap = std::min<int64_t>(d.n, std::min(by_rows, by_bytes));
    if ((st = dev_alloc(&idx->lists, static_cast<size_t>(d.max_batch) * idx->list_cap, "row lists")) != IFVS_OK)
      return bail(st);
    if ((st = dev_alloc(&idx->list_n, static_cast<size_t>(d.max_batch), "row list sizes")) != IFVS_OK)
      return bail(st);
    if ((st = dev_alloc(&idx->qmode, static_cast<size_t>(d.max_batch), "scan modes")) != IFVS_OK)
      return bail(st);
  }
  const size_t cb = static_cast<size_t>(d.m) * kKsub * idx->dsub;
  if ((st = dev_alloc(&idx->cpq, cb, "codebook")) != IFVS_OK) return bail(st);
  if (hipError_t e = hipMemcpy(idx->cpq, d.codebook, cb * sizeof(float), kind); e != hipSuccess)
    return bail(hip_fail(e, "loading codebook"));
  if ((st = dev_alloc(&idx->sdc, static_cast<size_t>(d.m) * kKsub * kKsub, "codeword distance table")) != IFVS_OK)
    return bail(st);
  if (hipError_t e = launch_sdc_table(idx->cpq, d.m, idx->dsub, idx->sdc, 0); e != hipSuccess)
    return bail(hip_fail(e, "building the codeword distance table"));
  if (d.bank_rows > 0) {
    const size_t nb = static_cast<size_t>(d.bank_rows) * d.m * d.r;
    const size_t nw = static_cast<size_t>(d.m) * d.r * kKsub * idx->dsub;
    if ((st = dev_alloc(&idx->bank, nb, "memory bank")) != IFVS_OK) return bail(st);
    if ((st = dev_alloc(&idx->W, nw, "direction tensor W")) != IFVS_OK) return bail(st);
    if (hipError_t e = hipMemcpy(idx->bank, d.bank, nb * sizeof(float), kind); e != hipSuccess)
      return bail(hip_fail(e, "loading memory bank"));
    if (hipError_t e = hipMemcpy(idx->W, d.W, nw * sizeof(float), kind); e != hipSuccess)
      return bail(hip_fail(e, "loading W"));
  }

  // Workspace.
  if ((st = dev_alloc(&idx->preds_dev, d.max_batch, "predicates")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->qorder_dev, d.max_batch, "query order")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->iv_dev, 2 * static_cast<size_t>(d.max_batch), "row intervals")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->bound_parts, static_cast<size_t>(d.max_batch) * 2 * d.m, "bound workspace")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->gthr_dev, static_cast<size_t>(d.max_batch), "scan thresholds")) != IFVS_OK)
    return bail(st);
  // Room for the dispatch order of a chunk-grid scan: 8 XCD runs of query
  // tiles times cells of at least 2048 tiles (the automatic grid uses
  // larger ones), between 2^16 and 2^20 items.
  idx->slot_order_cap = std::min<int64_t>(
      int64_t{1} << 20,
      std::max<int64_t>(int64_t{1} << 16, 8 * ((d.max_batch + 7) / 8) * ((idx->n_tiles + 2047) / 2048)));
  if ((st = dev_alloc(&idx->slot_order_dev, static_cast<size_t>(idx->slot_order_cap), "scan dispatch order")) != IFVS_OK)
    return bail(st);
  for (int i = 0; i < kStagingSlots; ++i) {
    const size_t bytes = (sizeof(DevPred) + sizeof(int32_t)) * d.max_batch + sizeof(int32_t) * idx->slot_order_cap;
    if (forced_alloc_failure() ||
        hipHostMalloc(reinterpret_cast<void**>(&idx->staging[i]), bytes, hipHostMallocDefault) != hipSuccess) {
      idx->staging[i] = nullptr;
      (void)hipGetLastError();
      return bail(fail(IFVS_E_NOMEM, "pinned staging allocation failed"));
    }
    if (hipError_t e = hipHostGetDevicePointer(reinterpret_cast<void**>(&idx->staging_dev[i]), idx->staging[i], 0);
        e != hipSuccess)
      return bail(hip_fail(e, "mapping the staging slot"));
    // (the event only tells the host that the kernels reading the slot have
    // run: no timing, and no system-scope fence, which would write back and
    // invalidate the caches at each record)
    if (hipError_t e = hipEventCreateWithFlags(&idx->staged[i], hipEventDisableTiming | hipEventDisableSystemFence);
        e != hipSuccess)
      return bail(hip_fail(e, "creating staging event"));
  }
  if (forced_alloc_failure() ||
      // (coherent: the device's store reaches host memory without a cache flush)
      hipHostMalloc(reinterpret_cast<void**>(&idx->done_host), sizeof(uint64_t) * kStagingSlots,
                    hipHostMallocCoherent) != hipSuccess) {
    idx->done_host = nullptr;
    (void)hipGetLastError();
    return bail(fail(IFVS_E_NOMEM, "pinned staging allocation failed"));
  }
  std::fill(idx->done_host, idx->done_host + kStagingSlots, uint64_t{0});
  if (hipError_t e = hipHostGetDevicePointer(reinterpret_cast<void**>(&idx->done_dev), idx->done_host, 0);
      e != hipSuccess)
    return bail(hip_fail(e, "mapping the staging done words"));
  idx->stride64 = idx->n_tiles;
  if ((st = dev_alloc(&idx->bitmap, static_cast<size_t>(d.max_batch) * idx->stride64, "selection bitmaps")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->counts, d.max_batch, "pool sizes")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->count_parts, static_cast<size_t>(d.max_batch) * filter_count_parts(idx->n),
                      "pool size partials")) != IFVS_OK)
    return bail(st);
  // Partials: room for at least 16 chunks per query, capped near 512 MB.
  {
    const size_t per_chunk = static_cast<size_t>(d.max_batch) * kScanWaves * d.max_k;
    const size_t chunks = std::max<size_t>(16, std::min<size_t>(256, (size_t(512) << 20) / 8 / per_chunk));
    idx->partial_keys = per_chunk * chunks;
    if ((st = dev_alloc(&idx->partials, idx->partial_keys, "top-k partials")) != IFVS_OK) return bail(st);
  }
  if (hipError_t e = hipDeviceSynchronize(); e != hipSuccess) return bail(hip_fail(e, "finishing load"));
  *out = idx;
  return IFVS_OK;
}

void ifvs_free_index(ifvs_index* idx) { delete idx; }

ifvs_status ifvs_set_option(ifvs_index* idx, int32_t option, int64_t value) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (value < 0 || value > (1 << 20)) return fail(IFVS_E_INVALID, "option value out of range");
  switch (option) {
    case IFVS_OPT_QTILE: idx->opt_qtile = static_cast<int>(value); return IFVS_OK;
    case IFVS_OPT_SPLITS: idx->opt_splits = static_cast<int>(value); return IFVS_OK;
    case IFVS_OPT_MIN_CHUNK: idx->opt_min_chunk = static_cast<int>(value); return IFVS_OK;
    case IFVS_OPT_GRID_TILES: idx->opt_grid_tiles = value; return IFVS_OK;
    case IFVS_OPT_GRID_RELATIVE:
      if (value > 1) return fail(IFVS_E_INVALID, "IFVS_OPT_GRID_RELATIVE takes 0 or 1");
      idx->opt_grid_relative = static_cast<int>(value);
      return IFVS_OK;
    case IFVS_OPT_GATHER:
      if (value > 2) return fail(IFVS_E_INVALID, "IFVS_OPT_GATHER takes 0, 1 or 2");
      idx->opt_gather = static_cast<int>(value);
      return IFVS_OK;
    case IFVS_OPT_SLOT_ORDER:
      if (value > 1) return fail(IFVS_E_INVALID, "IFVS_OPT_SLOT_ORDER takes 0 or 1");
      idx->opt_slot_order = static_cast<int>(value);
      return IFVS_OK;
    case IFVS_OPT_EXACT_PLAN:
      if (value > 2) return fail(IFVS_E_INVALID, "IFVS_OPT_EXACT_PLAN takes 0, 1 or 2");
      idx->opt_exact_plan = static_cast<int>(value);
      return IFVS_OK;
    case IFVS_OPT_SEED_TILES: idx->opt_seed_tiles = static_cast<int>(value); return IFVS_OK;
    case IFVS_OPT_SHARED_BOUND:
      if (value > 2) return fail(IFVS_E_INVALID, "IFVS_OPT_SHARED_BOUND takes 0, 1 or 2");
      idx->opt_shared_bound = static_cast<int>(value);
      return IFVS_OK;
    case IFVS_OPT_COARSE:
      if (value > 2) return fail(IFVS_E_INVALID, "IFVS_OPT_COARSE takes 0, 1 or 2");
      idx->opt_coarse = static_cast<int>(value);
      return IFVS_OK;
    case IFVS_OPT_COUNT_READS:
      if (value > 1) return fail(IFVS_E_INVALID, "IFVS_OPT_COUNT_READS takes 0 or 1");
      if (value == 1 && !idx->read_hist) {
        IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
        if (ifvs_status st = dev_alloc(&idx->read_hist, kReadHistEntries, "read histogram"); st != IFVS_OK)
          return st;
        IFVS_HIP(hipMemset(idx->read_hist, 0, kReadHistEntries * sizeof(unsigned long long)),
                 "clearing the read histogram");
      }
      idx->opt_count_reads = static_cast<int>(value);
      return IFVS_OK;
    case IFVS_OPT_PROFILE:
      if (value != 0 && !idx->timers) {
        idx->timers = new StageTimer[kStages];
        for (int st = 0; st < kStages; ++st)
          for (hipEvent_t& e : idx->timers[st].ev)   // timing only: no system-scope fence
            IFVS_HIP(hipEventCreateWithFlags(&e, hipEventDisableSystemFence), "creating profile events");
      }
      if (value > 3) return fail(IFVS_E_INVALID, "IFVS_OPT_PROFILE takes 0, 1, 2 or 3");
      idx->profile_mask = value == 0   ? 0
                          : value == 1 ? (1 << (kStListScan + 1)) - 1
                          : value == 2 ? (1 << kStScan) | (1 << kStListScan)
                                       : 1 << kStListScan;
      return IFVS_OK;
    default: return fail(IFVS_E_INVALID, "unknown option " + std::to_string(option));
  }
}

ifvs_status ifvs_select_codebook(ifvs_index* idx, int32_t nq, const float* q,
                                 const ifvs_predicate* preds, const float* w_z, float* alpha_out,
                                 float* wf_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (nq == 0) return IFVS_OK;
  if (!q || !wf_out) return fail(IFVS_E_INVALID, "q or wf_out is NULL");
  if (idx->bank_rows > 0 && !alpha_out) return fail(IFVS_E_INVALID, "alpha_out is NULL but the index has a memory bank");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  int slot = 0;
  if (ifvs_status st = stage_predicates(idx, nq, preds, false, false, s, &slot); st != IFVS_OK) return st;
  IFVS_LAUNCH(idx, kStCondition, s, "launching condition kernel",
              launch_condition(q, idx->dim, idx->staging_dev[slot], nq, idx->bank, idx->bank_rows,
                               idx->m * idx->r, idx->h, idx->hash_seed, w_z,
                               idx->bank_rows > 0 ? alpha_out : nullptr, wf_out, s));
  return release_slot(idx, slot, s);
}

ifvs_status ifvs_build_lut(ifvs_index* idx, int32_t nq, const float* q, const float* alpha,
                           const float* wf, int32_t lut_dtype, void* lut_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (lut_dtype != IFVS_LUT_F32 && lut_dtype != IFVS_LUT_F16) return fail(IFVS_E_INVALID, "unknown lut_dtype");
  if (nq == 0) return IFVS_OK;
  if (!q || !lut_out) return fail(IFVS_E_INVALID, "q or lut_out is NULL");
  if (alpha && idx->bank_rows == 0) return fail(IFVS_E_INVALID, "alpha given but the index has no memory bank");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  IFVS_LAUNCH(idx, kStLut, s, "launching LUT kernel",
              launch_build_lut(q, idx->dim, idx->m, idx->dsub, idx->r, idx->cpq, idx->W, alpha, wf,
                               nq, lut_dtype, lut_out, s));
  return IFVS_OK;
}

ifvs_status ifvs_build_sdc_lut(ifvs_index* idx, int32_t nq, const float* q, int32_t lut_dtype, void* lut_out,
                               void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (lut_dtype != IFVS_LUT_F32 && lut_dtype != IFVS_LUT_F16) return fail(IFVS_E_INVALID, "unknown lut_dtype");
  if (nq == 0) return IFVS_OK;
  if (!q || !lut_out) return fail(IFVS_E_INVALID, "q or lut_out is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  IFVS_LAUNCH(idx, kStLut, s, "launching SDC table kernel",
              launch_sdc_lut(q, idx->dim, idx->m, idx->dsub, idx->cpq, idx->sdc, nq, lut_dtype, lut_out, s));
  return IFVS_OK;
}

ifvs_status ifvs_filter(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                        uint32_t* bitmap_out, int64_t* count_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (nq == 0) return IFVS_OK;
  if (!bitmap_out) return fail(IFVS_E_INVALID, "bitmap_out is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  int slot = 0;
  if (ifvs_status st = stage_predicates(idx, nq, preds, false, true, s, &slot); st != IFVS_OK) return st;
  const SearchWs ws = index_ws(idx);
  if (ifvs_status st = filter_into_workspace(idx, ws, nq, false, true, s); st != IFVS_OK) return st;
  if (ifvs_status st = copy_bitmaps_out(idx, ws, nq, bitmap_out, s); st != IFVS_OK) return st;
  if (count_out)
    IFVS_HIP(hipMemcpyAsync(count_out, idx->counts, sizeof(int64_t) * nq, hipMemcpyDeviceToDevice, s),
             "copying pool sizes");
  return IFVS_OK;
}

}  // extern "C"

namespace {

// Selection shape of a staged batch: a clause tested row by row somewhere,
// every selection a run of rows of the layout, the widest run in 64-row
// tiles.
struct BatchShape {
  bool need_bitmap = false;
  bool interval_batch = true;
  int64_t span = 0;
};

BatchShape batch_shape(const ifvs_index* idx, int32_t nq, const DevPred* host) {
  BatchShape b;
  for (int i = 0; i < nq; ++i) {
    b.need_bitmap = b.need_bitmap || host[i].residual_mask != 0;
    // A predicate no row can satisfy has the empty interval on a clustered
    // index, so it does not take the batch off the interval plan.
    b.interval_batch = b.interval_batch && (host[i].iv_mode != 0 || (idx->n_cluster > 0 && host[i].n_eff < 0));
    if (idx->n_cluster > 0) b.span = std::max(b.span, estimate_interval_tiles(idx, host[i]));
  }
  return b;
}

// The list scan's conditions that depend on the index, the tables' type and
// the batch's selections (the search adds its workspace's): a coarse build,
// no clause tested row by row, a supported M, and IFVS_OPT_COARSE (forced,
// or automatic for batches whose widest interval spans kCoarseAutoTiles or
// more tiles on indexes of kCoarseAutoM or more subspaces).
bool list_scan_wanted(const ifvs_index* idx, int32_t lut_dtype, const BatchShape& b) {
  return idx->coarse.words && idx->opt_coarse != 1 && !b.need_bitmap && list_scan_supported(idx->m, lut_dtype) &&
         (idx->opt_coarse == 2 || (b.span >= kCoarseAutoTiles && idx->m >= kCoarseAutoM));
}

// The host side of a search, before anything is enqueued: validation, the
// staged predicates (or the caller's staging, pre_slot >= 0), the batch's
// shape, the workspace, the scan plan, whether the list scan runs, the
// scan's dispatch order.  With static_scratch the device workspace is carved
// from the static array of the index's device instead of the index's own
// workspace (no gather scan then: every query takes the tiled scan, with the
// same results).  bounded: the caller gave the alpha and w_f its tables were
// built with (either may be null), so the list scan may run with the coarse
// bound.
struct SearchPrep {
  bool empty = false;   // nq == 0: nothing to do
  int slot = 0;
  DevPred* host = nullptr;
  BatchShape shape;
  SearchWs ws;
  ScanPlan plan{};
  int list_jobs = 1;
  bool list_mode = false;
  bool ordered = false;
  int64_t n_order = 0;
};

ifvs_status prepare_search(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds, const void* lut,
                           int32_t lut_dtype, bool bounded, const float* alpha, int32_t k, int32_t* ids_out,
                           float* dist_out, uint32_t* bitmap_out, hipStream_t s, bool static_scratch, int pre_slot,
                           DevPred* pre_host, SearchPrep& p) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (lut_dtype != IFVS_LUT_F32 && lut_dtype != IFVS_LUT_F16) return fail(IFVS_E_INVALID, "unknown lut_dtype");
  if (k < 1 || k > idx->max_k)
    return fail(IFVS_E_INVALID, "k = " + std::to_string(k) + " outside 1.." + std::to_string(idx->max_k) + " (max_k)");
  p.empty = nq == 0;
  if (p.empty) return IFVS_OK;
  if (!lut || !ids_out || !dist_out) return fail(IFVS_E_INVALID, "lut, ids_out or dist_out is NULL");
  if (alpha && idx->bank_rows == 0) return fail(IFVS_E_INVALID, "alpha given but the index has no memory bank");
  if (reinterpret_cast<uintptr_t>(lut) % 16 != 0) return fail(IFVS_E_INVALID, "lut must be 16-byte aligned");
  ScanPlan probe{};
  if (ifvs_status st = plan_scan(idx, nq, k, lut_dtype, false, 0, size_t{1} << 40, &probe); st != IFVS_OK) return st;
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  DevPred*& host = p.host;
  int& slot = p.slot;
  // Predicates are validated before anything is enqueued (or were, with the
  // scan order, by a caller that staged them for earlier kernels too).
  if (pre_slot >= 0) {
    slot = pre_slot;
    host = pre_host;
  } else if (ifvs_status st = stage_predicates(idx, nq, preds, true, false, s, &slot, &host); st != IFVS_OK) {
    return st;
  }
  p.shape = batch_shape(idx, nq, host);
  const BatchShape& shape = p.shape;
  const bool need_bitmap = shape.need_bitmap, interval_batch = shape.interval_batch;
  const int64_t span = shape.span;
  SearchWs& ws = p.ws;
  if (!static_scratch) {
    ws = index_ws(idx);
  } else if (ifvs_status st = carve_static_ws(idx, nq, k, need_bitmap || bitmap_out != nullptr, &ws);
             st != IFVS_OK) {
    return st;
  }
  ScanPlan& plan = p.plan;
  if (ifvs_status st = plan_scan(idx, nq, k, lut_dtype, interval_batch, span, ws.partial_keys, &plan); st != IFVS_OK)
    return st;
  // List scan (coarse bound): when the caller passed the tables' operands, a
  // coarse build exists and every query's selection is its row interval
  // (no residual clauses); automatic for batches whose widest interval spans
  // at least kCoarseAutoTiles 64-row tiles.
  const CoarseLists& cl = idx->coarse;
  // Jobs per query: at most kListJobs (IFVS_OPT_SPLITS lowers the cap), as
  // the partial lists have room.
  int& list_jobs = p.list_jobs;
  list_jobs = std::min(kListJobs, idx->opt_splits > 0 ? idx->opt_splits : kListJobs);
  while (list_jobs > 1 && static_cast<size_t>(nq) * list_jobs * kScanWaves * k > ws.partial_keys) --list_jobs;
  const int list_splits = list_jobs;
  p.list_mode =
      bounded && !static_scratch && list_scan_wanted(idx, lut_dtype, shape) &&
      list_plan_lds_bytes(idx->m, lut_dtype, cl.C) <= size_t{kLdsBudget} &&
      list_scan_lds_bytes(idx->m, lut_dtype, pool_stride_for(k)) <= size_t{kLdsBudget} &&
      list_jobs_lds_bytes(nq) <= size_t{kLdsBudget} &&
      static_cast<size_t>(nq) * list_splits * kScanWaves * k <= ws.partial_keys;
  if (idx->opt_count_reads && !p.list_mode &&
      (!scan_can_count(idx->m, plan.qtile, lut_dtype) || plan.lds_bytes + kLookupHistBytes > size_t{kLdsBudget}))
    return fail(IFVS_E_UNSUPPORTED, "IFVS_OPT_COUNT_READS: no read-counting scan for this plan (it needs one query "
                                    "per tile, M of 16, 48 or 120, and 272 bytes of LDS to spare)");
  // Chunk-grid scans: the slot dispatch order goes into the staging slot and
  // the interval kernel copies it to the device.
  const int32_t* qorder_host = reinterpret_cast<const int32_t*>(host + idx->max_batch);
  int32_t* order_host = reinterpret_cast<int32_t*>(host + idx->max_batch) + idx->max_batch;
  // (the list scan takes its work from its job table: no dispatch order)
  p.n_order = plan.abs_cells && idx->opt_slot_order == 0 && !p.list_mode
                  ? static_cast<int64_t>(8) * ((((nq + plan.qtile - 1) / plan.qtile) + 7) / 8) * plan.splits
                  : 0;
  p.ordered = p.n_order > 0 && p.n_order <= ws.slot_order_cap;
  if (p.ordered) order_scan_slots(idx, host, qorder_host, nq, plan, order_host);
  return IFVS_OK;
}

// The interval kernel's work for a prepared search: the batch's predicates,
// scan order and dispatch order from its staging slot.
IntervalArgs search_intervals(const ifvs_index* idx, int32_t nq, const SearchPrep& p) {
  IntervalArgs a;
  a.attrs_phys = idx->attrs_phys;
  a.n = idx->n;
  a.c0 = idx->c0;
  a.c1 = idx->c1;
  a.vstart = idx->vstart;
  a.vmin = idx->vmin;
  a.vcount = idx->vcount;
  a.staged_preds = idx->staging_dev[p.slot];
  a.staged_order = reinterpret_cast<const int32_t*>(idx->staging_dev[p.slot] + idx->max_batch);
  a.nq = nq;
  a.preds_out = p.ws.preds;
  a.order_out = p.ws.qorder;
  a.iv = p.ws.iv;
  a.gthr = p.ws.gthr;
  a.slots_src = p.ordered ? a.staged_order + idx->max_batch : nullptr;
  a.slots_dst = p.ws.slot_order;
  a.n_slots = p.ordered ? p.n_order : 0;
  return a;
}

// The device side of a prepared search (intervals_done: the caller already
// enqueued search_intervals' work; parts_ready: the table kernel wrote the
// coarse bound's factors; slot_released: the caller released the staging
// slot, whose readers all ran before this search's kernels).
ifvs_status run_search(ifvs_index* idx, int32_t nq, const void* lut, int32_t lut_dtype, const float* alpha,
                       const float* wf, int32_t k, int32_t* ids_out, float* dist_out, uint32_t* bitmap_out,
                       hipStream_t s, const SearchPrep& p, bool intervals_done, bool parts_ready,
                       bool slot_released = false) {
  if (p.empty) return IFVS_OK;
  const SearchWs& ws = p.ws;
  const ScanPlan& plan = p.plan;
  const bool need_bitmap = p.shape.need_bitmap, interval_batch = p.shape.interval_batch;
  const int list_jobs = p.list_jobs, list_splits = p.list_jobs;
  const bool ordered = p.ordered;
  const CoarseLists& cl = idx->coarse;
  if (!intervals_done)
    IFVS_LAUNCH(idx, kStFilter, s, "launching interval kernel", launch_intervals(search_intervals(idx, nq, p), s));
  if (!slot_released)
    if (ifvs_status st = release_slot(idx, p.slot, s); st != IFVS_OK) return st;
  if (p.list_mode) {
    // (the table kernel wrote the bound's factors when the caller says so)
    if (!parts_ready)
      IFVS_LAUNCH(idx, kStCoarse, s, "launching table bound kernel",
                  launch_bound_parts(alpha, wf, idx->cpq, idx->W, nq, idx->m, idx->r, idx->dsub, idx->bound_parts,
                                     s));
    ListPlanArgs pa{};
    pa.lut = lut;
    pa.m = idx->m;
    pa.nq = nq;
    pa.cc_t = cl.cc_t;
    pa.mw = idx->mw;
    pa.C = cl.C;
    pa.n_sub = cl.C * kBands;
    pa.parts = idx->bound_parts;
    pa.grow = bound_grow(idx->m, idx->dsub);
    pa.iv = ws.iv;
    pa.cnt_f = cl.cnt_f;
    pa.f_shift = cl.f_shift;
    pa.words = cl.words;
    pa.band = cl.band;
    pa.sub_off = cl.sub_off;
    pa.rmax = cl.rmax;
    pa.lrow = cl.lrow;
    pa.codes_t = cl.codes_t;
    pa.k = k;
    pa.gthr = ws.gthr;
    pa.keep = coarse_keep(idx->m, idx->dsub, lut_dtype);
    pa.abs_m = coarse_abs(idx->m, lut_dtype);
    pa.it_r0 = cl.it_r0;
    pa.it_r1 = cl.it_r1;
    pa.it_t = cl.it_t;
    pa.it_lb = cl.it_lb;
    pa.hdr = cl.hdr;
    pa.slots = cl.slots;
    ListJobArgs ja{};
    ja.hdr = cl.hdr;
    ja.qorder = ws.qorder;
    ja.nq = nq;
    ja.np2 = 1;
    while (ja.np2 < nq) ja.np2 *= 2;
    ja.k = k;
    ja.max_jobs = list_jobs;
    ja.jobs = cl.jobs;
    ja.n_keys = cl.n_keys;
    ja.job_next = cl.job_ctr;
    ja.job_total = cl.job_ctr + 1;
    IFVS_LAUNCH(idx, kStCoarse, s, "launching list plan kernel", launch_list_plan(pa, lut_dtype, s));
    IFVS_LAUNCH(idx, kStCoarse, s, "launching list job table kernel", launch_list_jobs(ja, s));
    ListScanArgs sa{};
    sa.codes_t = cl.codes_t;
    sa.ids = cl.ids;
    sa.m = idx->m;
    sa.mw = idx->mw;
    sa.lut = lut;
    sa.nq = nq;
    sa.max_jobs = list_jobs;
    sa.qorder = ws.qorder;
    sa.jobs = cl.jobs;
    sa.job_next = cl.job_ctr;
    sa.job_total = cl.job_ctr + 1;
    sa.it_r0 = cl.it_r0;
    sa.it_r1 = cl.it_r1;
    sa.it_t = cl.it_t;
    sa.it_lb = cl.it_lb;
    sa.hdr = cl.hdr;
    sa.C = cl.C * kBands;
    sa.keep = pa.keep;
    sa.abs_m = pa.abs_m;
    sa.k = k;
    sa.pool_stride = pool_stride_for(k);
    sa.kpl = pool_kpl(k);
    sa.partials = ws.partials;
    sa.gthr = ws.gthr;
    sa.slots = cl.slots;
    sa.lookup_hist = idx->opt_count_reads ? idx->read_hist : nullptr;
    sa.union_bound = idx->opt_shared_bound == 1 ? 0 : 1;
    IFVS_LAUNCH(idx, kStListScan, s, "launching list scan kernel", launch_list_scan(sa, lut_dtype, s));
    IFVS_LAUNCH(idx, kStMerge, s, "launching top-k merge kernel",
                launch_topk_merge(ws.partials, nq, static_cast<int64_t>(list_jobs) * kScanWaves * k, k, ws.iv, 0,
                                  static_cast<int64_t>(kScanWaves) * k, ws.qorder, ids_out, dist_out, s,
                                  cl.n_keys));
    if (bitmap_out) {
      if (ifvs_status st = filter_into_workspace(idx, ws, nq, false, false, s); st != IFVS_OK) return st;
      if (ifvs_status st = copy_bitmaps_out(idx, ws, nq, bitmap_out, s); st != IFVS_OK) return st;
    }
    ScanPlan lp{};
    lp.qtile = 1;
    lp.splits = list_splits;
    lp.min_chunk = 0;
    lp.lds_bytes = list_scan_lds_bytes(idx->m, lut_dtype, pool_stride_for(k));
    idx->last_plan = lp;
    idx->last_coarse = true;
    return IFVS_OK;
  }
  // Masked batches: a query whose pool is small is scored from its compacted
  // row list (decided on the device from the pool size); the rest take the
  // tiled scan.  The full selection bitmap (physical order) and the pool
  // sizes come from the Filter stage.
  const int gather_lut = lut_dtype == IFVS_LUT_F16 ? 2 : 4;
  const bool gather = !interval_batch && idx->codes_rm && ws.lists && idx->opt_gather != 2 &&
                      gather_supported(idx->m, lut_dtype) &&
                      static_cast<size_t>(idx->m) * kKsub * gather_lut + gather_lds_bytes(plan.pool_stride) <=
                          static_cast<size_t>(kLdsBudget);
  if (gather) {
    IFVS_LAUNCH(idx, kStFilter, s, "launching filter kernel",
                launch_filter(idx->attrs_phys, idx->n, idx->n_attr, ws.preds, nq, false, ws.bitmap,
                              ws.stride64, ws.counts, ws.count_parts, s));
    const int64_t max_rows = idx->opt_gather == 1 ? ws.list_cap : std::min(ws.list_cap, gather_auto_rows(idx));
    IFVS_LAUNCH(idx, kStFilter, s, "launching compaction kernel",
                launch_compact(ws.bitmap, ws.stride64, ws.counts, ws.count_parts,
                               filter_count_parts(idx->n), nq, max_rows, ws.list_cap, ws.lists,
                               ws.list_n, ws.qmode, s));
  } else if (need_bitmap) {
    if (ifvs_status st = filter_into_workspace(idx, ws, nq, true, false, s); st != IFVS_OK) return st;
  }
  ScanBatch b{};
  b.codes_t = idx->codes_t;
  b.n = idx->n;
  b.n_tiles = idx->n_tiles;
  b.m = idx->m;
  b.mw = idx->mw;
  b.lut = lut;
  b.lut_dtype = lut_dtype;
  b.nq = nq;
  b.qorder = ws.qorder;
  b.iv = ws.iv;
  b.preds = ws.preds;
  b.bitmap = ws.bitmap;
  b.stride64 = ws.stride64;
  b.perm = idx->perm;
  b.k = k;
  b.partials = ws.partials;
  b.gthr = ws.gthr;
  b.mode = gather ? ws.qmode : nullptr;
  b.slot_order = ordered ? ws.slot_order : nullptr;
  b.lookup_hist = idx->opt_count_reads ? idx->read_hist : nullptr;
  IFVS_LAUNCH(idx, kStScan, s, "launching scan kernel", launch_scan(b, plan, s));
  if (gather) {
    GatherBatch g{};
    g.codes_rm = idx->codes_rm;
    g.rw = idx->rw;
    g.m = idx->m;
    g.lut = lut;
    g.lut_dtype = lut_dtype;
    g.nq = nq;
    g.qorder = ws.qorder;
    g.mode = ws.qmode;
    g.lists = ws.lists;
    g.list_n = ws.list_n;
    g.list_cap = ws.list_cap;
    g.splits = plan.splits;
    g.gblocks = gather_blocks_per_query(ws.list_cap, plan.splits);
    g.perm = idx->perm;
    g.k = k;
    g.pool_stride = plan.pool_stride;
    g.kpl = plan.kpl;
    g.partials = ws.partials;
    g.gthr = ws.gthr;
    IFVS_LAUNCH(idx, kStScan, s, "launching gather scan kernel", launch_gather_scan(g, s));
  }
  const int64_t per_query = static_cast<int64_t>(plan.splits) * kScanWaves * k;
  IFVS_LAUNCH(idx, kStMerge, s, "launching top-k merge kernel",
              launch_topk_merge(ws.partials, nq, per_query, k, ws.iv,
                                plan.abs_cells ? plan.chunk_tiles : 0, static_cast<int64_t>(kScanWaves) * k,
                                ws.qorder, ids_out, dist_out, s));
  if (bitmap_out) {
    // The Filter stage's bitmaps in id order (the scan itself reads row
    // intervals and residual bits in the physical order).
    if (ifvs_status st = filter_into_workspace(idx, ws, nq, false, false, s); st != IFVS_OK) return st;
    if (ifvs_status st = copy_bitmaps_out(idx, ws, nq, bitmap_out, s); st != IFVS_OK) return st;
  }
  idx->last_plan = plan;
  idx->last_coarse = false;
  return IFVS_OK;
}

// Filter, Rank and Select for one batch: prepare_search, then run_search.
ifvs_status search_impl(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds, const void* lut,
                        int32_t lut_dtype, bool bounded, const float* alpha, const float* wf, int32_t k,
                        int32_t* ids_out, float* dist_out, uint32_t* bitmap_out, void* stream,
                        bool static_scratch) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  SearchPrep p;
  if (ifvs_status st = prepare_search(idx, nq, preds, lut, lut_dtype, bounded, alpha, k, ids_out, dist_out,
                                      bitmap_out, s, static_scratch, -1, nullptr, p);
      st != IFVS_OK)
    return st;
  return run_search(idx, nq, lut, lut_dtype, alpha, wf, k, ids_out, dist_out, bitmap_out, s, p, false, false);
}

}  // namespace

extern "C" {

ifvs_status ifvs_filtered_search(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                                 const void* lut, int32_t lut_dtype, int32_t k, int32_t* ids_out,
                                 float* dist_out, uint32_t* bitmap_out, void* stream) {
  return search_impl(idx, nq, preds, lut, lut_dtype, false, nullptr, nullptr, k, ids_out, dist_out, bitmap_out,
                     stream, false);
}

ifvs_status ifvs_filtered_search_bounded(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                                         const void* lut, int32_t lut_dtype, const float* alpha, const float* wf,
                                         int32_t k, int32_t* ids_out, float* dist_out, uint32_t* bitmap_out,
                                         void* stream) {
  return search_impl(idx, nq, preds, lut, lut_dtype, true, alpha, wf, k, ids_out, dist_out, bitmap_out, stream,
                     false);
}

ifvs_status ifvs_query_batch(ifvs_index* idx, int32_t nq, const float* q, const ifvs_predicate* preds,
                             const float* w_z, float* wz_out, float* alpha_out, float* wf_out, int32_t lut_dtype,
                             void* lut_out, int32_t k, int32_t* ids_out, float* dist_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (lut_dtype != IFVS_LUT_F32 && lut_dtype != IFVS_LUT_F16) return fail(IFVS_E_INVALID, "unknown lut_dtype");
  if (k < 1 || k > idx->max_k)
    return fail(IFVS_E_INVALID, "k = " + std::to_string(k) + " outside 1.." + std::to_string(idx->max_k) + " (max_k)");
  if (nq == 0) return IFVS_OK;
  if (!q || !wf_out || !lut_out || !ids_out || !dist_out)
    return fail(IFVS_E_INVALID, "q, wf_out, lut_out, ids_out or dist_out is NULL");
  if (idx->bank_rows > 0 && !alpha_out) return fail(IFVS_E_INVALID, "alpha_out is NULL but the index has a memory bank");
  if (!w_z && !idx->enc_params)
    return fail(IFVS_E_STATE, "w_z is NULL and no encoder is attached (ifvs_load_encoder)");
  if (!w_z && !wz_out) return fail(IFVS_E_INVALID, "w_z and wz_out are both NULL");
  if (reinterpret_cast<uintptr_t>(lut_out) % 16 != 0) return fail(IFVS_E_INVALID, "lut must be 16-byte aligned");
  ScanPlan probe{};
  if (ifvs_status st = plan_scan(idx, nq, k, lut_dtype, false, 0, size_t{1} << 40, &probe); st != IFVS_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  // One staging of the predicates (validated, with the scan order) for the
  // encoder, the condition and the search kernels.
  DevPred* host = nullptr;
  int slot = 0;
  if (ifvs_status st = stage_predicates(idx, nq, preds, true, false, s, &slot, &host); st != IFVS_OK) return st;
  // (a failed launch still releases the slot: kernels enqueued before it
  // may read it)
  auto launch = [&](int stage, const char* what, auto&& fn) -> ifvs_status {
    const ifvs_status st = timed(idx, stage, s, what, fn);
    if (st != IFVS_OK) (void)release_slot(idx, slot, s);
    return st;
  };
  float* alpha = idx->bank_rows > 0 ? alpha_out : nullptr;
  // The encoder conditions the queries it encodes in the same launch (alpha
  // and w_f, the condition kernel's bits) where it can.
  const bool fused_condition = !w_z && encoder_conditions(idx->h, alpha != nullptr);
  // The search's host side now (its intervals can then go into the encoder's
  // launch too).
  SearchPrep prep;
  if (ifvs_status st = prepare_search(idx, nq, preds, lut_out, lut_dtype, true, alpha, k, ids_out, dist_out, nullptr,
                                      s, false, slot, host, prep);
      st != IFVS_OK) {
    (void)release_slot(idx, slot, s);
    return st;
  }
  const IntervalArgs iva = search_intervals(idx, nq, prep);
  const float* wz = w_z;
  if (!w_z) {
    EncCondition cond;
    cond.q = q;
    cond.bank = idx->bank;
    cond.bank_rows = idx->bank_rows;
    cond.mr = idx->m * idx->r;
    cond.h = idx->h;
    cond.seed = idx->hash_seed;
    cond.alpha = alpha;
    cond.wf = wf_out;
    if (ifvs_status st = launch(kStEncode, "launching encoder kernel", [&]() -> hipError_t {
          return launch_encoder(idx->enc_params, idx->enc_off, idx->enc_scale, idx->enc_H, idx->enc_heads,
                                idx->enc_layers, idx->enc_F, idx->dim, idx->n_attr, idx->staging_dev[slot], nq, wz_out,
                                s, fused_condition ? &cond : nullptr, &iva);
        });
        st != IFVS_OK)
      return st;
    wz = wz_out;
  }
  // When the list scan runs, the table kernel writes the coarse bound's
  // factors as it forms the conditioned codewords (the search then skips its
  // own bound kernel).
  float* parts =
      prep.list_mode && lut_emits_bound_parts(idx->dsub, idx->r, alpha != nullptr) ? idx->bound_parts : nullptr;
  if (!fused_condition) {
    if (ifvs_status st = launch(kStCondition, "launching condition kernel", [&]() -> hipError_t {
          return launch_condition(q, idx->dim, idx->staging_dev[slot], nq, idx->bank, idx->bank_rows,
                                  idx->m * idx->r, idx->h, idx->hash_seed, wz, alpha, wf_out, s);
        });
        st != IFVS_OK)
      return st;
  }
  // When the encoder ran, every reader of the staging slot (the encoder's
  // launch with the intervals, the condition kernel) runs before the table
  // kernel, which then releases the slot through its done word.
  const StageDone done = !w_z ? slot_done_word(idx, slot) : StageDone{};
  if (ifvs_status st = launch(kStLut, "launching LUT kernel", [&]() -> hipError_t {
        return launch_build_lut(q, idx->dim, idx->m, idx->dsub, idx->r, idx->cpq, idx->W, alpha, wf_out, nq,
                                lut_dtype, lut_out, s, parts, done);
      });
      st != IFVS_OK)
    return st;
  if (!w_z) release_slot_by_word(idx, slot);
  // (the encoder's launch computed the intervals when it ran)
  const ifvs_status st = run_search(idx, nq, lut_out, lut_dtype, alpha, wf_out, k, ids_out, dist_out, nullptr, s,
                                    prep, !w_z, parts != nullptr, !w_z);
  if (st != IFVS_OK && !idx->slot_busy[slot]) (void)release_slot(idx, slot, s);   // the earlier kernels read it
  return st;
}

ifvs_status ifvs_filtered_search_noalloc(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                                         const void* lut, int32_t lut_dtype, int32_t k, int32_t* ids_out,
                                         float* dist_out, uint32_t* bitmap_out, void* stream) {
  return search_impl(idx, nq, preds, lut, lut_dtype, false, nullptr, nullptr, k, ids_out, dist_out, bitmap_out,
                     stream, true);
}

}  // extern "C"

namespace {

// Attach vectors to the index for the exact search: src is device memory
// [n][dim]; src_perm maps physical row r to its row of src (null: src is in
// physical order already).  Allocates the copies and the workspace.
ifvs_status attach_vectors(ifvs_index* idx, const float* src, const int32_t* src_perm) {
  const int64_t n = idx->n, n32 = (n + 31) / 32 * 32;
  const int dim = idx->dim, ks = exact_ksteps(dim);
  auto bail = [&](ifvs_status st) {
    idx->free_vectors();
    return st;
  };
  ifvs_status st;
  if ((st = dev_alloc(&idx->xt, static_cast<size_t>((n + 63) / 64) * dim * 64, "fp32 vector tiles")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->xr, static_cast<size_t>(n) * dim, "fp32 vectors")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->xb, static_cast<size_t>(n32 / 32) * ks * 64, "bf16 vector fragments")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->xn, static_cast<size_t>(n32), "vector norms")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->xmax, 1, "largest norm")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->xbad, 1, "non-finite count")) != IFVS_OK) return bail(st);
  // Workspace of the searches: chunks and bins per query are bounded so the
  // buffers stay small; the planner never exceeds them.
  const int max_batch = idx->max_batch;
  idx->exact_splits_max = 2048;
  idx->exact_chunks_max = 1024;
  idx->cand_cap = 16384;
  const int n_qtiles = (max_batch + 31) / 32;
  if ((st = dev_alloc(&idx->qb, static_cast<size_t>(n_qtiles) * ks * 64, "query fragments")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->qn_x, max_batch, "query norms")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->eps_x, max_batch, "error bounds")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->thr_x, max_batch, "candidate bounds")) != IFVS_OK) return bail(st);
  idx->bins_cap = 65536;
  if ((st = dev_alloc(&idx->bins_x, static_cast<size_t>(max_batch) * idx->bins_cap, "screening minima")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->cand_x, static_cast<size_t>(max_batch) * idx->cand_cap, "candidate lists")) != IFVS_OK)
    return bail(st);
  if ((st = dev_alloc(&idx->cand_n_x, max_batch, "candidate counts")) != IFVS_OK) return bail(st);
  if ((st = dev_alloc(&idx->partials_x, static_cast<size_t>(max_batch) * idx->exact_chunks_max * idx->max_k,
                      "exact top-k partials")) != IFVS_OK)
    return bail(st);
  hipError_t e = hipMemset(idx->xmax, 0, sizeof(unsigned));
  if (e == hipSuccess) e = hipMemset(idx->xbad, 0, sizeof(unsigned long long));
  if (e == hipSuccess)
    e = launch_exact_stage(src, n, dim, src_perm, idx->xt, idx->xr, idx->xb, idx->xn, idx->xmax, idx->xbad, 0);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  unsigned long long bad = 0;
  if (e == hipSuccess) e = hipMemcpy(&bad, idx->xbad, sizeof(bad), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return bail(hip_fail(e, "staging vectors"));
  if (bad) return bail(fail(IFVS_E_INVALID, std::to_string(bad) + " vector values are NaN or infinite"));
  return IFVS_OK;
}

}  // namespace

namespace {

// The interval kernel's work for the exact search (the index's own device
// copies; no dispatch order).
IntervalArgs exact_intervals(const ifvs_index* idx, int slot, int32_t nq) {
  IntervalArgs a;
  a.attrs_phys = idx->attrs_phys;
  a.n = idx->n;
  a.c0 = idx->c0;
  a.c1 = idx->c1;
  a.vstart = idx->vstart;
  a.vmin = idx->vmin;
  a.vcount = idx->vcount;
  a.staged_preds = idx->staging_dev[slot];
  a.staged_order = reinterpret_cast<const int32_t*>(idx->staging_dev[slot] + idx->max_batch);
  a.nq = nq;
  a.preds_out = idx->preds_dev;
  a.order_out = idx->qorder_dev;
  a.iv = idx->iv_dev;
  a.gthr = idx->gthr_dev;
  a.slots_dst = idx->slot_order_dev;
  return a;
}

}  // namespace

extern "C" {

ifvs_status ifvs_load_vectors(ifvs_index* idx, const float* x, int32_t mem_kind) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (idx->xr) return fail(IFVS_E_STATE, "vectors are already attached to this index");
  if (!x) return fail(IFVS_E_INVALID, "x is NULL");
  if (mem_kind != IFVS_MEM_HOST && mem_kind != IFVS_MEM_DEVICE) return fail(IFVS_E_INVALID, "unknown mem_kind");
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  const float* src = x;
  float* staged = nullptr;
  if (mem_kind == IFVS_MEM_HOST) {
    if (ifvs_status st = dev_alloc(&staged, static_cast<size_t>(idx->n) * idx->dim, "vector staging"); st != IFVS_OK)
      return st;
    if (hipError_t e = hipMemcpy(staged, x, sizeof(float) * idx->n * idx->dim, hipMemcpyHostToDevice);
        e != hipSuccess) {
      hipFree(staged);
      return hip_fail(e, "copying vectors");
    }
    src = staged;
  }
  const ifvs_status st = attach_vectors(idx, src, idx->perm);
  if (staged) hipFree(staged);
  return st;
}

ifvs_status ifvs_load_reconstructions(ifvs_index* idx) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (idx->xr) return fail(IFVS_E_STATE, "vectors are already attached to this index");
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  float* rec = nullptr;
  if (ifvs_status st = dev_alloc(&rec, static_cast<size_t>(idx->n) * idx->dim, "reconstructions"); st != IFVS_OK)
    return st;
  if (hipError_t e = launch_decode(idx->codes_t, idx->n, idx->m, idx->mw, idx->dsub, idx->cpq, rec, 0);
      e != hipSuccess) {
    hipFree(rec);
    return hip_fail(e, "decoding codes");
  }
  const ifvs_status st = attach_vectors(idx, rec, nullptr);   // already in physical order
  hipFree(rec);
  return st;
}

ifvs_status ifvs_exact_search(ifvs_index* idx, int32_t nq, const float* q, const ifvs_predicate* preds, int32_t k,
                              int32_t* ids_out, float* dist_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (!idx->xr) return fail(IFVS_E_STATE, "no vectors attached to this index (ifvs_load_vectors)");
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (k < 1 || k > idx->max_k)
    return fail(IFVS_E_INVALID, "k = " + std::to_string(k) + " outside 1.." + std::to_string(idx->max_k) + " (max_k)");
  if (nq == 0) return IFVS_OK;
  if (!q || !ids_out || !dist_out) return fail(IFVS_E_INVALID, "q, ids_out or dist_out is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  DevPred* host = nullptr;
  int slot = 0;
  if (ifvs_status st = stage_predicates(idx, nq, preds, true, false, s, &slot, &host); st != IFVS_OK) return st;
  // Plan.  Screening reads every row of a 32-query tile's hull twice in bf16
  // (2 x 2 bytes per dimension); scoring directly reads each query's own
  // interval once in fp32 (4 bytes per dimension).  Screen when the hulls
  // together are shorter than the intervals together -- queries sharing
  // rows -- unless forced.
  const int32_t* qorder_host = reinterpret_cast<const int32_t*>(host + idx->max_batch);
  bool need_bitmap = false;
  int64_t sum_iv = 0, sum_hull = 0, max_iv = 0, min_iv = INT64_MAX;
  for (int t = 0; t * 32 < nq; ++t) {
    int64_t lo = INT64_MAX, hi = 0;
    for (int i = t * 32; i < std::min(nq, t * 32 + 32); ++i) {
      const DevPred& d = host[qorder_host[i]];
      need_bitmap = need_bitmap || d.residual_mask != 0;
      int64_t a = 0, b = idx->n_tiles;
      if (idx->n_cluster > 0) estimate_interval_range(idx, d, &a, &b);
      if (d.n_eff < 0) a = b = 0;
      if (b > a) {
        sum_iv += b - a;
        max_iv = std::max(max_iv, b - a);
        min_iv = std::min(min_iv, b - a);
        lo = std::min(lo, a);
        hi = std::max(hi, b);
      }
    }
    if (hi > lo) sum_hull += hi - lo;
  }
  const bool screened = idx->opt_exact_plan == 2 || (idx->opt_exact_plan == 0 && sum_hull < sum_iv);
  IFVS_LAUNCH(idx, kStFilter, s, "launching interval kernel",
              launch_intervals(exact_intervals(idx, slot, nq), s));
  if (ifvs_status st = release_slot(idx, slot, s); st != IFVS_OK) return st;
  if (need_bitmap)
    if (ifvs_status st = filter_into_workspace(idx, index_ws(idx), nq, true, false, s); st != IFVS_OK) return st;
  IFVS_LAUNCH(idx, kStCondition, s, "launching exact query kernel",
              launch_exact_queries(q, idx->dim, nq, idx->qorder_dev, idx->xmax, idx->qb, idx->qn_x, idx->eps_x,
                                   idx->cand_n_x, s));
  ExactRerank r{};
  r.xt = idx->xt;
  r.xr = idx->xr;
  r.dim = idx->dim;
  r.q = q;
  r.qorder = idx->qorder_dev;
  r.iv = idx->iv_dev;
  r.preds = idx->preds_dev;
  r.bitmap = idx->bitmap;
  r.stride64 = idx->stride64;
  r.perm = idx->perm;
  r.nq = nq;
  r.k = k;
  r.partials = idx->partials_x;
  if (screened) {
    // Chunks of the hull: enough workgroups to fill the GPU, every row of
    // the largest possible hull (the whole index) covered.
    const int64_t quantum = exact_chunk_quantum();
    const int64_t n_qtiles = (nq + 31) / 32;
    int64_t chunk_rows = (idx->n * n_qtiles + 2047) / 2048;
    chunk_rows = std::min<int64_t>(65536, std::max<int64_t>(4 * quantum, (chunk_rows + quantum - 1) / quantum * quantum));
    int64_t splits = (idx->n + chunk_rows - 1) / chunk_rows;
    if (splits > idx->exact_splits_max) {
      splits = idx->exact_splits_max;
      chunk_rows = ((idx->n + splits - 1) / splits + quantum - 1) / quantum * quantum;
    }
    // Bins: R lanes share one; R as large as leaves the shortest interval
    // (estimated, in rows) at least 4k bins, within the bin budget.
    const int64_t lane_rows = std::max<int64_t>(1, chunk_rows / (32 * 8));
    const int64_t short_rows = min_iv == INT64_MAX ? 0 : min_iv * 64;
    int bin_lanes = 32;
    while (bin_lanes > 1 && short_rows / (lane_rows * bin_lanes) < 4 * static_cast<int64_t>(k)) bin_lanes /= 2;
    while (exact_bins_per_query(static_cast<int>(splits), bin_lanes) > idx->bins_cap) bin_lanes *= 2;
    ExactScreen e{};
    e.bin_lanes = bin_lanes;
    e.xb = idx->xb;
    e.xn = idx->xn;
    e.dim = idx->dim;
    e.qb = idx->qb;
    e.qn = idx->qn_x;
    e.thr = idx->thr_x;
    e.qorder = idx->qorder_dev;
    e.iv = idx->iv_dev;
    e.preds = idx->preds_dev;
    e.bitmap = idx->bitmap;
    e.stride64 = idx->stride64;
    e.nq = nq;
    e.chunk_rows = chunk_rows;
    e.splits = static_cast<int>(splits);
    e.bins = idx->bins_x;
    e.cand = idx->cand_x;
    e.cand_n = idx->cand_n_x;
    e.cand_cap = idx->cand_cap;
    IFVS_LAUNCH(idx, kStScan, s, "launching exact screening (pass 1)", launch_exact_screen(e, 1, s));
    IFVS_LAUNCH(idx, kStScan, s, "launching exact threshold kernel",
                launch_exact_threshold(idx->bins_x, exact_bins_per_query(e.splits, e.bin_lanes), nq, k, idx->eps_x,
                                       idx->thr_x, s));
    IFVS_LAUNCH(idx, kStScan, s, "launching exact screening (pass 2)", launch_exact_screen(e, 2, s));
    r.cand = idx->cand_x;
    r.cand_n = idx->cand_n_x;
    r.cand_cap = idx->cand_cap;
    r.chunks = 16;
  } else {
    // About 4096 rows per wavefront (the planner's interval estimates only
    // size the grid; every chunk covers its share of the true interval).
    r.chunks = static_cast<int>(std::min<int64_t>(idx->exact_chunks_max, std::max<int64_t>(1, (max_iv + 63) / 64)));
  }
  IFVS_LAUNCH(idx, kStScan, s, "launching exact scoring kernel", launch_exact_rerank(r, s));
  IFVS_LAUNCH(idx, kStMerge, s, "launching top-k merge kernel",
              launch_topk_merge(idx->partials_x, nq, static_cast<int64_t>(r.chunks) * k, k, idx->iv_dev, 0, k,
                                idx->qorder_dev, ids_out, dist_out, s));
  return IFVS_OK;
}

ifvs_status ifvs_read_profile(ifvs_index* idx, double* ms_out, int64_t* launches_out) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (!ms_out || !launches_out) return fail(IFVS_E_INVALID, "ms_out or launches_out is NULL");
  for (int st = 0; st < kStages; ++st) {
    ms_out[st] = 0.0;
    launches_out[st] = 0;
    if (!idx->timers) continue;
    StageTimer& t = idx->timers[st];
    if (ifvs_status e = flush_timer(t); e != IFVS_OK) return e;
    ms_out[st] = t.ms;
    launches_out[st] = t.launches;
    t.ms = 0.0;
    t.launches = 0;
  }
  return IFVS_OK;
}

int64_t ifvs_encoder_params(int32_t hidden, int32_t heads, int32_t layers, int32_t ffn, int32_t n_attr,
                            int32_t dim) {
  if (hidden < 16 || hidden > 128 || hidden % 16 != 0) return -1;
  if (heads < 1 || heads > 16 || hidden % heads != 0) return -1;
  if (layers < 1 || layers > 8) return -1;
  if (ffn < 16 || ffn > 256 || ffn % 16 != 0) return -1;
  if (n_attr < 1 || dim < 1) return -1;
  const int64_t H = hidden, F = ffn;
  const int64_t per_layer = 2 * H + H * 3 * H + 3 * H + H * H + H + 2 * H + H * F + F + F * H + H;
  return int64_t{n_attr} * H + 2 * H + H + H + layers * per_layer + 2 * H + H * dim + dim;
}

ifvs_status ifvs_load_encoder(ifvs_index* idx, const ifvs_encoder_desc* desc) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (!desc) return fail(IFVS_E_INVALID, "desc is NULL");
  const ifvs_encoder_desc& d = *desc;
  if (d.reserved != 0) return fail(IFVS_E_INVALID, "encoder desc: reserved field not 0");
  if (idx->n_attr < 1) return fail(IFVS_E_INVALID, "the index has no attribute columns to encode");
  const int64_t want = ifvs_encoder_params(d.hidden, d.heads, d.layers, d.ffn, idx->n_attr, idx->dim);
  if (want < 0)
    return fail(IFVS_E_INVALID, "encoder sizes out of range (hidden 16..128 and ffn 16..256, multiples of 16; "
                                "heads 1..16 dividing hidden; layers 1..8)");
  if (d.n_params != want)
    return fail(IFVS_E_INVALID, "encoder n_params = " + std::to_string(d.n_params) + ", the sizes need " +
                                    std::to_string(want));
  if (!d.params || !d.col_offset || !d.col_scale) return fail(IFVS_E_INVALID, "encoder arrays must not be NULL");
  if (d.mem_kind != IFVS_MEM_HOST && d.mem_kind != IFVS_MEM_DEVICE) return fail(IFVS_E_INVALID, "unknown mem_kind");
  const hipMemcpyKind kind = d.mem_kind == IFVS_MEM_HOST ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice;
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  std::vector<double> off(idx->n_attr), sc(idx->n_attr);
  IFVS_HIP(hipMemcpy(off.data(), d.col_offset, off.size() * sizeof(double),
                     d.mem_kind == IFVS_MEM_HOST ? hipMemcpyHostToHost : hipMemcpyDeviceToHost),
           "reading encoder offsets");
  IFVS_HIP(hipMemcpy(sc.data(), d.col_scale, sc.size() * sizeof(double),
                     d.mem_kind == IFVS_MEM_HOST ? hipMemcpyHostToHost : hipMemcpyDeviceToHost),
           "reading encoder scales");
  for (int c = 0; c < idx->n_attr; ++c)
    if (!std::isfinite(off[c]) || !std::isfinite(sc[c]))
      return fail(IFVS_E_INVALID, "encoder offset or scale of column " + std::to_string(c) + " is not finite");
  float* p = nullptr;
  double* o = nullptr;
  double* k = nullptr;
  auto undo = [&](ifvs_status st) {
    for (void* x : {static_cast<void*>(p), static_cast<void*>(o), static_cast<void*>(k)})
      if (x) (void)hipFree(x);
    return st;
  };
  if (ifvs_status st = dev_alloc(&p, static_cast<size_t>(want), "encoder parameters"); st != IFVS_OK) return undo(st);
  if (ifvs_status st = dev_alloc(&o, static_cast<size_t>(idx->n_attr), "encoder offsets"); st != IFVS_OK)
    return undo(st);
  if (ifvs_status st = dev_alloc(&k, static_cast<size_t>(idx->n_attr), "encoder scales"); st != IFVS_OK)
    return undo(st);
  if (hipError_t e = hipMemcpy(p, d.params, static_cast<size_t>(want) * sizeof(float), kind); e != hipSuccess)
    return undo(hip_fail(e, "loading encoder parameters"));
  if (hipError_t e = hipMemcpy(o, off.data(), off.size() * sizeof(double), hipMemcpyHostToDevice); e != hipSuccess)
    return undo(hip_fail(e, "loading encoder offsets"));
  if (hipError_t e = hipMemcpy(k, sc.data(), sc.size() * sizeof(double), hipMemcpyHostToDevice); e != hipSuccess)
    return undo(hip_fail(e, "loading encoder scales"));
  if (hipError_t e = hipDeviceSynchronize(); e != hipSuccess) return undo(hip_fail(e, "loading the encoder"));
  for (void* x : {static_cast<void*>(idx->enc_params), static_cast<void*>(idx->enc_off),
                  static_cast<void*>(idx->enc_scale)})
    if (x) (void)hipFree(x);
  idx->enc_params = p;
  idx->enc_off = o;
  idx->enc_scale = k;
  idx->enc_H = d.hidden;
  idx->enc_heads = d.heads;
  idx->enc_layers = d.layers;
  idx->enc_F = d.ffn;
  return IFVS_OK;
}

ifvs_status ifvs_encode_predicates(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds, float* wz_out,
                                   void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (!idx->enc_params) return fail(IFVS_E_STATE, "no encoder attached (ifvs_load_encoder)");
  if (nq == 0) return IFVS_OK;
  if (!wz_out) return fail(IFVS_E_INVALID, "wz_out is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  int slot = 0;
  if (ifvs_status st = stage_predicates(idx, nq, preds, false, false, s, &slot); st != IFVS_OK) return st;
  IFVS_LAUNCH(idx, kStEncode, s, "launching encoder kernel",
              launch_encoder(idx->enc_params, idx->enc_off, idx->enc_scale, idx->enc_H, idx->enc_heads,
                             idx->enc_layers, idx->enc_F, idx->dim, idx->n_attr, idx->staging_dev[slot], nq,
                             wz_out, s));
  return release_slot(idx, slot, s);
}

ifvs_status ifvs_read_scan_reads(ifvs_index* idx, int64_t* hist_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (!hist_out) return fail(IFVS_E_INVALID, "hist_out is NULL");
  for (int i = 0; i < kReadHistEntries; ++i) hist_out[i] = 0;
  if (!idx->read_hist) return IFVS_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  unsigned long long h[kReadHistEntries];
  IFVS_HIP(hipMemcpyAsync(h, idx->read_hist, sizeof(h), hipMemcpyDeviceToHost, s), "reading the read histogram");
  IFVS_HIP(hipStreamSynchronize(s), "reading the read histogram");
  IFVS_HIP(hipMemsetAsync(idx->read_hist, 0, sizeof(h), s), "clearing the read histogram");
  IFVS_HIP(hipStreamSynchronize(s), "clearing the read histogram");
  for (int i = 0; i < kReadHistEntries; ++i) hist_out[i] = static_cast<int64_t>(h[i]);
  return IFVS_OK;
}

ifvs_status ifvs_probe_lds_gather(int32_t active_lanes, double* wave_reads_per_s, void* stream) {
  if (active_lanes < 1 || active_lanes > 64) return fail(IFVS_E_INVALID, "active_lanes outside 1..64");
  if (!wave_reads_per_s) return fail(IFVS_E_INVALID, "wave_reads_per_s is NULL");
  // Three eight-wavefront workgroups per CU (24 waves: as many 48 KB tables
  // as the LDS holds), 1024 iterations of 32 reads each, 4 timed launches.
  IFVS_HIP(lds_gather_probe(active_lanes, 1024, 3, 4, static_cast<hipStream_t>(stream), wave_reads_per_s),
           "LDS gather probe");
  return IFVS_OK;
}

ifvs_status ifvs_train_step(ifvs_index* idx, int32_t nq, const float* q, const ifvs_predicate* preds,
                            const float* w_z, const int32_t* cand, int32_t n_cand, int32_t n_pos, float tau,
                            float lambda, float lr, float* loss_out, float* dwz_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (idx->bank_rows == 0) return fail(IFVS_E_STATE, "the index has no memory bank and W to train");
  if (n_cand < 1 || n_cand > 4096) return fail(IFVS_E_INVALID, "n_cand must be in 1..4096");
  if (n_pos < 0 || n_pos > n_cand) return fail(IFVS_E_INVALID, "n_pos must be in 0..n_cand");
  if (!(tau > 0.0f) || !std::isfinite(tau)) return fail(IFVS_E_INVALID, "tau must be positive and finite");
  if (!(lambda >= 0.0f) || !std::isfinite(lambda)) return fail(IFVS_E_INVALID, "lambda must be >= 0 and finite");
  if (!std::isfinite(lr)) return fail(IFVS_E_INVALID, "lr must be finite");
  if (nq == 0) return IFVS_OK;
  if (!q || !cand || !loss_out) return fail(IFVS_E_INVALID, "q, cand or loss_out is NULL");
  if (dwz_out && !w_z) return fail(IFVS_E_INVALID, "dwz_out needs w_z");
  const int mr = idx->m * idx->r;
  if (train_query_lds_bytes(idx->m, idx->dim, n_cand, mr) > static_cast<size_t>(kLdsBudget))
    return fail(IFVS_E_UNSUPPORTED, "one query's table, candidates and gradients exceed the 160 KB LDS budget");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  if (!idx->tr_alpha) {
    const size_t b = static_cast<size_t>(idx->max_batch);
    ifvs_status st = IFVS_OK;
    if ((st = dev_alloc(&idx->tr_alpha, b * mr, "training alpha")) != IFVS_OK ||
        (st = dev_alloc(&idx->tr_wf, b * idx->dim, "training w_f")) != IFVS_OK ||
        (st = dev_alloc(&idx->tr_lut, b * idx->m * kKsub, "training tables")) != IFVS_OK ||
        (st = dev_alloc(&idx->tr_gdelta, b * idx->m * kKsub * idx->dsub, "training Delta gradients")) != IFVS_OK ||
        (st = dev_alloc(&idx->tr_galpha, b * mr, "training alpha gradients")) != IFVS_OK ||
        (st = dev_alloc(&idx->tr_rows, b * idx->h, "training bank rows")) != IFVS_OK) {
      for (void* p : {static_cast<void*>(idx->tr_alpha), static_cast<void*>(idx->tr_wf),
                      static_cast<void*>(idx->tr_lut), static_cast<void*>(idx->tr_gdelta),
                      static_cast<void*>(idx->tr_galpha), static_cast<void*>(idx->tr_rows)})
        if (p) hipFree(p);
      idx->tr_alpha = idx->tr_wf = idx->tr_lut = idx->tr_gdelta = idx->tr_galpha = nullptr;
      idx->tr_rows = nullptr;
      return st;
    }
  }
  if (idx->perm && !idx->inv_perm) {
    // Candidates are original ids; the codes are in physical order.
    if (ifvs_status st = dev_alloc(&idx->inv_perm, static_cast<size_t>(idx->n), "inverse permutation"); st != IFVS_OK)
      return st;
    if (hipError_t e = launch_invert_perm(idx->perm, idx->n, idx->inv_perm, s); e != hipSuccess) {
      hipFree(idx->inv_perm);
      idx->inv_perm = nullptr;
      return hip_fail(e, "launching permutation inverse");
    }
  }
  int slot = 0;
  if (ifvs_status st = stage_predicates(idx, nq, preds, false, false, s, &slot); st != IFVS_OK) return st;
  IFVS_LAUNCH(idx, kStCondition, s, "launching condition kernel",
              launch_condition(q, idx->dim, idx->staging_dev[slot], nq, idx->bank, idx->bank_rows, mr, idx->h,
                               idx->hash_seed, w_z, idx->tr_alpha, idx->tr_wf, s, idx->tr_rows));
  if (ifvs_status st = release_slot(idx, slot, s); st != IFVS_OK) return st;
  IFVS_LAUNCH(idx, kStLut, s, "launching LUT kernel",
              launch_build_lut(q, idx->dim, idx->m, idx->dsub, idx->r, idx->cpq, idx->W, idx->tr_alpha, idx->tr_wf,
                               nq, IFVS_LUT_F32, idx->tr_lut, s));
  TrainArgs a{};
  a.codes_t = idx->codes_t;
  a.inv_perm = idx->inv_perm;
  a.n = idx->n;
  a.m = idx->m;
  a.mw = idx->mw;
  a.dsub = idx->dsub;
  a.r = idx->r;
  a.dim = idx->dim;
  a.q = q;
  a.w_z = w_z;
  a.wf = idx->tr_wf;
  a.alpha = idx->tr_alpha;
  a.lut = idx->tr_lut;
  a.cpq = idx->cpq;
  a.W = idx->W;
  a.cand = cand;
  a.nq = nq;
  a.n_cand = n_cand;
  a.n_pos = n_pos;
  a.tau = tau;
  a.lam = lambda;
  a.loss = loss_out;
  a.gdelta = idx->tr_gdelta;
  a.galpha = idx->tr_galpha;
  a.dwz = dwz_out;
  IFVS_HIP(launch_train_query(a, s), "launching training gradient kernel");
  IFVS_HIP(launch_train_update_w(idx->W, idx->tr_gdelta, idx->tr_alpha, nq, idx->m, idx->r, idx->dsub, lr, s),
           "launching W update");
  IFVS_HIP(launch_train_update_bank(idx->bank, mr, idx->tr_rows, idx->h, idx->tr_galpha, nq, lr, s),
           "launching memory bank update");
  return IFVS_OK;
}

ifvs_status ifvs_read_params(const ifvs_index* idx, float* bank_out, float* W_out, void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (idx->bank_rows == 0) return fail(IFVS_E_STATE, "the index has no memory bank and W");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  if (bank_out)
    IFVS_HIP(hipMemcpyAsync(bank_out, idx->bank, sizeof(float) * idx->bank_rows * idx->m * idx->r,
                            hipMemcpyDefault, s), "copying the memory bank");
  if (W_out)
    IFVS_HIP(hipMemcpyAsync(W_out, idx->W, sizeof(float) * idx->m * idx->r * kKsub * idx->dsub,
                            hipMemcpyDefault, s), "copying W");
  return IFVS_OK;
}

ifvs_status ifvs_last_plan(const ifvs_index* idx, int64_t* out5) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (!out5) return fail(IFVS_E_INVALID, "out5 is NULL");
  out5[0] = idx->last_plan.qtile;
  out5[1] = idx->last_plan.splits;
  out5[2] = idx->last_plan.min_chunk;
  out5[3] = static_cast<int64_t>(idx->last_plan.lds_bytes);
  out5[4] = idx->last_plan.chunk_tiles;
  return IFVS_OK;
}

ifvs_status ifvs_last_coarse(const ifvs_index* idx, int32_t* used_out) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (!used_out) return fail(IFVS_E_INVALID, "used_out is NULL");
  *used_out = idx->last_coarse ? 1 : 0;
  return IFVS_OK;
}

ifvs_status ifvs_build_coarse(ifvs_index* idx, int32_t n_centroids, int32_t iters) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (n_centroids < 1 || n_centroids > kCoarseMax || n_centroids > idx->n)
    return fail(IFVS_E_INVALID, "n_centroids outside 1.." + std::to_string(kCoarseMax) + " (and at most n)");
  if (iters < 0 || iters > 1000) return fail(IFVS_E_INVALID, "iters outside 0..1000");
  if (idx->dim > kCoarseMaxDim)
    return fail(IFVS_E_UNSUPPORTED, "a coarse quantizer needs dim <= " + std::to_string(kCoarseMaxDim));
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  const int C = n_centroids, D = idx->dim, mw = idx->mw;
  const int64_t n = idx->n, n_pad = idx->n_tiles * kTileRows;
  const int64_t S = coarse_samples(n, C);
  float* X = nullptr;
  float* cent = nullptr;
  float* chat = nullptr;
  int32_t* assign = nullptr;
  uint32_t* cc = nullptr;
  CoarseLists nl;
  nl.C = C;
  auto cleanup = [&](ifvs_status st) {
    for (void* p : {static_cast<void*>(X), static_cast<void*>(cent), static_cast<void*>(chat),
                    static_cast<void*>(assign), static_cast<void*>(cc)})
      if (p) (void)hipFree(p);
    nl.release();
    return st;
  };
  auto alloc = [&](auto** p, size_t count, const char* what) { return dev_alloc(p, count, what); };
  if (ifvs_status st = alloc(&X, static_cast<size_t>(S) * D, "coarse samples"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&cent, static_cast<size_t>(C) * D, "coarse centroids"); st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&chat, static_cast<size_t>(C) * D, "encoded centroids"); st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&assign, static_cast<size_t>(S), "coarse assignment"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&cc, static_cast<size_t>(C) * mw, "centroid codes"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.words, static_cast<size_t>(n_pad), "coarse row words"); st != IFVS_OK)
    return cleanup(st);
  hipStream_t s = nullptr;
  auto step = [&](hipError_t e, const char* what) -> ifvs_status {
    return e == hipSuccess ? IFVS_OK : hip_fail(e, what);
  };
  // Samples: evenly spaced rows; first centroids: C evenly spaced rows.
  if (ifvs_status st = step(launch_coarse_sample(idx->codes_t, mw, idx->m, idx->dsub, idx->cpq, S, n / S, X, s),
                            "launching coarse sample kernel");
      st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = step(launch_coarse_sample(idx->codes_t, mw, idx->m, idx->dsub, idx->cpq, C, n / C, cent, s),
                            "launching coarse sample kernel");
      st != IFVS_OK)
    return cleanup(st);
  for (int it = 0; it < iters; ++it)
    if (ifvs_status st = step(launch_coarse_kmeans_step(X, S, D, cent, C, assign, s), "launching k-means kernels");
        st != IFVS_OK)
      return cleanup(st);
  if (ifvs_status st = step(launch_coarse_encode(cent, C, idx->m, mw, idx->dsub, idx->cpq, cc, chat, s),
                            "launching centroid encoding kernel");
      st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = step(launch_coarse_rows(idx->codes_t, n, n_pad, idx->m, mw, idx->dsub, idx->cpq, chat, C,
                                               nl.words, s),
                            "launching coarse assignment kernel");
      st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = step(hipDeviceSynchronize(), "building the coarse quantizer"); st != IFVS_OK)
    return cleanup(st);

  // Sub-lists (host).  Each row's radius band within its list: the list's
  // radii at the quantiles kBandQuantiles split it into kBands bands (equal
  // radii share a band).  Then a stable counting sort of the layout rows by
  // sub-list s = c * kBands + b, the largest radius of each sub-list, and
  // the rank table every 2^f_shift rows.
  std::vector<uint32_t> hw(static_cast<size_t>(n));
  std::vector<uint32_t> hcc(static_cast<size_t>(C) * mw);
  if (ifvs_status st = step(hipMemcpy(hw.data(), nl.words, hw.size() * 4, hipMemcpyDeviceToHost), "reading row words");
      st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = step(hipMemcpy(hcc.data(), cc, hcc.size() * 4, hipMemcpyDeviceToHost), "reading centroids");
      st != IFVS_OK)
    return cleanup(st);
  const int NS = C * kBands;
  auto radius_of = [&](int64_t r) {
    const uint32_t bits = hw[static_cast<size_t>(r)] & 0xFFFF0000u;
    float rad;
    std::memcpy(&rad, &bits, 4);
    return rad;
  };
  std::vector<int32_t> coff(static_cast<size_t>(C) + 1, 0);
  for (int64_t r = 0; r < n; ++r) ++coff[static_cast<size_t>(hw[static_cast<size_t>(r)] & 0xFFFFu) + 1];
  for (int c = 0; c < C; ++c) coff[static_cast<size_t>(c) + 1] += coff[static_cast<size_t>(c)];
  std::vector<float> radii(static_cast<size_t>(n));
  {
    std::vector<int32_t> pos(coff.begin(), coff.end() - 1);
    for (int64_t r = 0; r < n; ++r)
      radii[static_cast<size_t>(pos[hw[static_cast<size_t>(r)] & 0xFFFFu]++)] = radius_of(r);
  }
  std::vector<float> cut(static_cast<size_t>(C) * (kBands - 1));
  for (int c = 0; c < C; ++c) {
    auto b = radii.begin() + coff[static_cast<size_t>(c)], e = radii.begin() + coff[static_cast<size_t>(c) + 1];
    std::sort(b, e);
    const int64_t cnt = e - b;
    for (int j = 0; j < kBands - 1; ++j)
      cut[static_cast<size_t>(c) * (kBands - 1) + j] =
          cnt > 0 ? *(b + std::min<int64_t>(cnt - 1, static_cast<int64_t>(kBandQuantiles[j] * cnt))) : 0.0f;
  }
  std::vector<uint8_t> hband(static_cast<size_t>(n));
  std::vector<int32_t> off(static_cast<size_t>(NS) + 1, 0), hrow(static_cast<size_t>(n));
  std::vector<float> rmax(static_cast<size_t>(NS), 0.0f);
  for (int64_t r = 0; r < n; ++r) {
    const int c = static_cast<int>(hw[static_cast<size_t>(r)] & 0xFFFFu);
    const float rad = radius_of(r);
    int b = 0;
    while (b < kBands - 1 && rad > cut[static_cast<size_t>(c) * (kBands - 1) + b]) ++b;
    hband[static_cast<size_t>(r)] = static_cast<uint8_t>(b);
    const int sub = c * kBands + b;
    ++off[static_cast<size_t>(sub) + 1];
    rmax[static_cast<size_t>(sub)] = std::max(rmax[static_cast<size_t>(sub)], rad);
  }
  for (int sub = 0; sub < NS; ++sub) off[static_cast<size_t>(sub) + 1] += off[static_cast<size_t>(sub)];
  nl.f_shift = 12;
  while (((n >> nl.f_shift) + 1) * NS > (int64_t{1} << 24)) ++nl.f_shift;
  const int64_t nb = (n >> nl.f_shift) + 1;
  std::vector<int32_t> cnt_f(static_cast<size_t>(nb * NS));
  {
    std::vector<int32_t> run(static_cast<size_t>(NS), 0), pos(off.begin(), off.end() - 1);
    const int64_t fmask = (int64_t{1} << nl.f_shift) - 1;
    for (int64_t r = 0; r < n; ++r) {
      if ((r & fmask) == 0) std::copy(run.begin(), run.end(), cnt_f.begin() + (r >> nl.f_shift) * NS);
      const int sub = static_cast<int>(hw[static_cast<size_t>(r)] & 0xFFFFu) * kBands + hband[static_cast<size_t>(r)];
      hrow[static_cast<size_t>(pos[static_cast<size_t>(sub)]++)] = static_cast<int32_t>(r);
      ++run[static_cast<size_t>(sub)];
    }
    if ((n & fmask) == 0) std::copy(run.begin(), run.end(), cnt_f.begin() + (n >> nl.f_shift) * NS);
  }
  std::vector<uint32_t> cc_t(hcc.size());
  for (int c = 0; c < C; ++c)
    for (int w = 0; w < mw; ++w)
      cc_t[static_cast<size_t>(w) * C + c] = hcc[static_cast<size_t>(c) * mw + w];

  const size_t items = static_cast<size_t>(idx->max_batch) * NS;
  if (ifvs_status st = alloc(&nl.cc_t, cc_t.size(), "centroid codes"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.sub_off, off.size(), "sub-list offsets"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.rmax, rmax.size(), "sub-list radii"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.cnt_f, cnt_f.size(), "sub-list rank table"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.band, hband.size(), "radius bands"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.codes_t, static_cast<size_t>(n_pad) * mw, "list-order codes"); st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&nl.ids, static_cast<size_t>(n_pad), "list-order ids"); st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&nl.lrow, hrow.size(), "list rows"); st != IFVS_OK) return cleanup(st);
  for (int32_t** a : {&nl.it_r0, &nl.it_r1, &nl.it_t})
    if (ifvs_status st = alloc(a, items, "list plan"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.it_lb, items, "list plan"); st != IFVS_OK) return cleanup(st);
  if (ifvs_status st = alloc(&nl.hdr, static_cast<size_t>(idx->max_batch) * 4, "list plan"); st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&nl.slots, static_cast<size_t>(idx->max_batch) * kListSlots, "list scan bound slots");
      st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&nl.jobs, static_cast<size_t>(idx->max_batch) * kListJobs, "list scan jobs");
      st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&nl.n_keys, static_cast<size_t>(idx->max_batch), "list scan jobs"); st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = alloc(&nl.job_ctr, 2, "list scan jobs"); st != IFVS_OK) return cleanup(st);
  const struct {
    void* dst;
    const void* src;
    size_t bytes;
  } uploads[] = {{nl.cc_t, cc_t.data(), cc_t.size() * 4},   {nl.sub_off, off.data(), off.size() * 4},
                 {nl.rmax, rmax.data(), rmax.size() * 4},    {nl.cnt_f, cnt_f.data(), cnt_f.size() * 4},
                 {nl.band, hband.data(), hband.size()},      {nl.lrow, hrow.data(), hrow.size() * 4}};
  for (const auto& u : uploads)
    if (ifvs_status st = step(hipMemcpy(u.dst, u.src, u.bytes, hipMemcpyHostToDevice), "uploading the lists");
        st != IFVS_OK)
      return cleanup(st);
  if (ifvs_status st = step(launch_gather_list(idx->codes_t, mw, idx->perm, nl.lrow, n, idx->n_tiles, nl.codes_t,
                                               nl.ids, s),
                            "launching list gather kernels");
      st != IFVS_OK)
    return cleanup(st);
  if (ifvs_status st = step(hipDeviceSynchronize(), "building the lists"); st != IFVS_OK) return cleanup(st);
  idx->coarse.release();
  idx->coarse = nl;
  nl = CoarseLists{};
  return cleanup(IFVS_OK);
}

ifvs_status ifvs_lut_bounds(ifvs_index* idx, int32_t nq, const float* alpha, const float* wf, float* bounds_out,
                            void* stream) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  if (ifvs_status st = check_nq(idx, nq); st != IFVS_OK) return st;
  if (nq == 0) return IFVS_OK;
  if (!bounds_out) return fail(IFVS_E_INVALID, "bounds_out is NULL");
  if (alpha && idx->bank_rows == 0) return fail(IFVS_E_INVALID, "alpha given but the index has no memory bank");
  hipStream_t s = static_cast<hipStream_t>(stream);
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  IFVS_LAUNCH(idx, kStCoarse, s, "launching table bounds kernel",
              launch_lut_bounds(alpha, wf, idx->cpq, idx->W, nq, idx->m, idx->r, idx->dsub, idx->bound_parts,
                                bounds_out, s));
  return IFVS_OK;
}

ifvs_status ifvs_read_coarse(const ifvs_index* idx, int32_t* n_centroids_out, int32_t* assign_out,
                             float* radius_out, uint8_t* codes_out) {
  if (ifvs_status st = check_index(idx); st != IFVS_OK) return st;
  const CoarseLists& cl = idx->coarse;
  if (!cl.words) return fail(IFVS_E_STATE, "no coarse quantizer built (ifvs_build_coarse)");
  IFVS_HIP(hipSetDevice(idx->device), "hipSetDevice");
  IFVS_HIP(hipDeviceSynchronize(), "waiting for the device");
  if (n_centroids_out) *n_centroids_out = cl.C;
  if (assign_out || radius_out) {
    std::vector<uint32_t> w(static_cast<size_t>(idx->n));
    IFVS_HIP(hipMemcpy(w.data(), cl.words, w.size() * 4, hipMemcpyDeviceToHost), "reading coarse words");
    std::vector<int32_t> perm;
    if (idx->perm) {
      perm.resize(static_cast<size_t>(idx->n));
      IFVS_HIP(hipMemcpy(perm.data(), idx->perm, perm.size() * 4, hipMemcpyDeviceToHost), "reading the row order");
    }
    for (int64_t r = 0; r < idx->n; ++r) {
      const int64_t id = idx->perm ? perm[static_cast<size_t>(r)] : r;
      const uint32_t v = w[static_cast<size_t>(r)];
      if (assign_out) assign_out[id] = static_cast<int32_t>(v & 0xFFFFu);
      if (radius_out) {
        const uint32_t bits = v & 0xFFFF0000u;
        float f;
        std::memcpy(&f, &bits, 4);
        radius_out[id] = f;
      }
    }
  }
  if (codes_out) {
    std::vector<uint32_t> cw(static_cast<size_t>(cl.C) * idx->mw);
    IFVS_HIP(hipMemcpy(cw.data(), cl.cc_t, cw.size() * 4, hipMemcpyDeviceToHost), "reading centroid codes");
    for (int c = 0; c < cl.C; ++c)
      for (int m = 0; m < idx->m; ++m)
        codes_out[static_cast<size_t>(c) * idx->m + m] =
            static_cast<uint8_t>((cw[static_cast<size_t>(m / 4) * cl.C + c] >> (8 * (m % 4))) & 0xFFu);
  }
  return IFVS_OK;
}

}  // extern "C"
