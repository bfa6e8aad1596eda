// Internal declarations shared by the host runtime and the HIP kernels of
// libifvs.  Not part of the public ABI (include/ifvs.h).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <cstdint>

namespace ifvs {

constexpr int kKsub = 256;
constexpr int kMaxClauses = 4;
constexpr int kTileRows = 64;              // vectors per code tile = one wavefront
constexpr int kLdsBudget = 160 * 1024;     // LDS bytes per workgroup on gfx950
constexpr int kScanWaves = 8;              // wavefronts per scan workgroup
constexpr int kScanPub = 2;                // best keys per (wavefront, query) published for the workgroup bound
constexpr int kScanSeed = 8;               // seed candidates per wavefront (kScanWaves * kScanSeed = 64 >= k)
constexpr int kFilterQueries = 16;         // predicates evaluated per attribute read
constexpr int kReadHistEntries = 66;       // read-counting builds: tiles, reads by 1..64 lanes, tiles fetched whole
constexpr int kLookupHistBytes = 272;      // LDS of the scan's read-counting build: 66 counters, padded
constexpr int kCoarseMaxDim = 128;         // largest D with a coarse quantizer (a row held in registers)
constexpr int kCoarseMax = 4096;           // most coarse centroids
constexpr int kBands = 4;                  // radius bands per coarse list (sub-lists)
constexpr int kMaxItems = kCoarseMax * kBands;   // sub-lists a list plan sorts in one workgroup
constexpr int kItemBits = 14;                    // sub-list index bits of a plan's sort entry
constexpr int kItemMask = (1 << kItemBits) - 1;
static_assert(kMaxItems <= (1 << kItemBits), "sub-list index must fit the plan's entry");
constexpr int kPlanBuckets = 4096;               // list plan: bucket 0 (no bound) and 4095 bound buckets
constexpr int kSeedRows = 4096;                  // rows of the nearest list a plan scores for its seed

// A predicate as the device sees it.  The raw fields are the caller's clauses
// exactly as given (they are hashed into the memory bank); the effective
// fields are the same conjunction normalized for evaluation on int32
// attributes: each kept clause tests (uint32)(attr - lo) < width, clauses that
// admit every int32 value are dropped, and n_eff = -1 marks a predicate that
// no value satisfies.
//
// On an index whose rows are clustered by attribute columns (c0 major, c1
// minor), the clauses on the cluster key become one interval of rows
// (iv_mode 1: c0 in [iv_lo0, iv_hi0); iv_mode 2: c0 == iv_lo0 and c1 in
// [iv_lo1, iv_hi1)); iv_mode 0 is the whole index.  Effective clauses whose
// bit is set in residual_mask are still tested row by row (selection bitmap).
struct DevPred {
  int32_t n_raw;
  int32_t n_eff;
  int32_t raw_col[kMaxClauses];
  int64_t raw_lo[kMaxClauses];
  int64_t raw_hi[kMaxClauses];
  int32_t col[kMaxClauses];
  int32_t lo[kMaxClauses];
  uint32_t width[kMaxClauses];
  int32_t residual_mask;
  int32_t iv_mode;
  int64_t iv_lo0, iv_hi0, iv_lo1, iv_hi1;
  // The residual clauses alone, packed (n_res of them), in the same form.
  int32_t n_res;
  int32_t res_col[kMaxClauses];
  int32_t res_lo[kMaxClauses];
  uint32_t res_width[kMaxClauses];
};

// Copy one predicate with a wavefront (lane i moves dword i): a single round
// trip when the source is the pinned host staging slot.
__device__ inline void copy_pred(const DevPred* __restrict__ src, DevPred* __restrict__ dst, int lane) {
  constexpr int kWords = static_cast<int>(sizeof(DevPred) / 4);
  static_assert(sizeof(DevPred) % 4 == 0 && sizeof(DevPred) / 4 <= 64, "one dword per lane");
  if (lane < kWords) reinterpret_cast<uint32_t*>(dst)[lane] = reinterpret_cast<const uint32_t*>(src)[lane];
}

// Kernel launchers (each defined next to its kernel).  All return the HIP
// error of the launch.

// Rows sorted by (attr[c0], attr[c1], id) as order-preserving 64-bit keys
// (stable LSD radix sort): perm[row] = original id of physical row `row`.
hipError_t cluster_permutation(const int32_t* attrs, int64_t n, int n_cluster, int c0, int c1,
                               int32_t* perm, hipStream_t s);
hipError_t launch_gather_attrs(const int32_t* attrs, int64_t n, int n_attr, const int32_t* perm,
                               int32_t* attrs_phys, hipStream_t s);
// Row interval [iv[2q], iv[2q+1]) of every query on the clustered layout
// (whole index for predicates without a cluster-key interval).  Reads the
// predicates and the scan order from the staging slot (pinned host memory)
// and leaves device copies in preds_out / order_out for the kernels that
// follow; resets each query's shared scan threshold gthr[q] to all ones;
// copies n_slots words of the scan's dispatch order from the staging slot
// (slots_src) to slots_dst.  vstart (may be null): vstart[t] = first
// physical row whose leading cluster key is >= vmin + t, for t < vcount (the
// last entry is n).
struct IntervalArgs {
  const int32_t* attrs_phys = nullptr;
  int64_t n = 0;
  int c0 = 0, c1 = 0;
  const int32_t* vstart = nullptr;
  int64_t vmin = 0, vcount = 0;
  const DevPred* staged_preds = nullptr;
  const int32_t* staged_order = nullptr;
  int nq = 0;
  DevPred* preds_out = nullptr;
  int32_t* order_out = nullptr;
  int64_t* iv = nullptr;
  uint64_t* gthr = nullptr;
  const int32_t* slots_src = nullptr;
  int32_t* slots_dst = nullptr;
  int64_t n_slots = 0;
};
hipError_t launch_intervals(const IntervalArgs& a, hipStream_t s);

// codes (row-major [n][m]) -> 64-row tiles, physical row r taken from
// original row perm[r] (perm may be null: identity).
hipError_t launch_relayout_codes(const uint8_t* codes, int64_t n, int m, int mw, const int32_t* perm,
                                 uint32_t* codes_t, int64_t n_tiles, hipStream_t s);

// Selection bitmaps; residual_only evaluates only the clauses in each
// predicate's residual_mask.
// Selection bitmaps (physical row order) and, when counts is not null, pool
// sizes; count_parts ([nq][filter_count_parts(n)] words) then holds, per
// query, the exclusive prefix sums of the selected rows of consecutive
// kFilterPartRows-row parts.
constexpr int64_t kFilterPartRows = 4 * 64 * 64;
int64_t filter_count_parts(int64_t n);
hipError_t launch_filter(const int32_t* attrs, int64_t n, int n_attr, const DevPred* preds,
                         int nq, bool residual_only, uint64_t* bitmap, int64_t stride64,
                         unsigned long long* counts, uint32_t* count_parts, hipStream_t s);

// rows_out (optional, [nq][h]): the hashed bank rows of each query.
hipError_t launch_condition(const float* q, int dim, const DevPred* preds, int nq,
                            const float* bank, int bank_rows, int mr, int h, uint64_t seed,
                            const float* w_z, float* alpha_out, float* wf_out, hipStream_t s,
                            int32_t* rows_out = nullptr);

// One training step of the conditioning (Section 2, training paragraph).
struct TrainArgs {
  const uint32_t* codes_t;   // [n_tiles][mw][64] code words, physical order
  const int32_t* inv_perm;   // original id -> physical row (null: identity)
  int64_t n;
  int m, mw, dsub, r, dim;
  const float* q;            // [nq][dim]
  const float* w_z;          // [nq][dim] or null (w_f = 1)
  const float* wf;           // [nq][dim]
  const float* alpha;        // [nq][m*r]
  const float* lut;          // [nq][m][256] fp32
  const float* cpq;          // [m][256][dsub]
  const float* W;            // [m][r][256][dsub]
  const int32_t* cand;       // [nq][n_cand] original ids (-1: absent), the first n_pos positives
  int nq, n_cand, n_pos;
  float tau, lam;
  float* loss;               // [nq]
  float* gdelta;             // [nq][m][256][dsub]
  float* galpha;             // [nq][m*r]
  float* dwz;                // [nq][dim] or null
};
size_t train_query_lds_bytes(int m, int dim, int n_cand, int mr);
hipError_t launch_train_query(const TrainArgs& a, hipStream_t s);
// W -= lr * sum_q gdelta_q (x) alpha_q, one thread per W entry.
hipError_t launch_train_update_w(float* W, const float* gdelta, const float* alpha, int nq, int m, int r,
                                 int dsub, float lr, hipStream_t s);
// bank[rows_q[i]] -= lr * galpha_q for every query and hash function.
hipError_t launch_train_update_bank(float* bank, int mr, const int32_t* rows, int h, const float* galpha,
                                    int nq, float lr, hipStream_t s);
// inv[perm[r]] = r.
hipError_t launch_invert_perm(const int32_t* perm, int64_t n, int32_t* inv, hipStream_t s);

// A word in pinned host memory that a kernel sets to `seq` as it starts: the
// kernels enqueued before it on the stream have all run (the host waits on
// the word instead of an event, whose record costs the stream a few
// microseconds).  flag null: nothing to signal.
struct StageDone {
  uint64_t* flag = nullptr;
  uint64_t seq = 0;
};
__device__ __forceinline__ void signal_stage_done(const StageDone& d) {
  if (d.flag && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
    __hip_atomic_store(d.flag, d.seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// parts: optional [nq][2][m] coarse-bound factors (launch_bound_parts's
// output, the same bits), written by the table kernel itself when
// lut_emits_bound_parts holds for the shape (hipErrorInvalidValue otherwise).
// done: signalled as the table kernel starts.
hipError_t launch_build_lut(const float* q, int dim, int m, int dsub, int r,
                            const float* cpq, const float* W, const float* alpha,
                            const float* wf, int nq, int lut_dtype, void* lut_out,
                            hipStream_t s, float* parts = nullptr, StageDone done = {});
bool lut_emits_bound_parts(int dsub, int r, bool has_alpha);

struct ScanPlan {
  int qtile;        // queries sharing one LDS residency and one pass over the codes
  int splits;       // code chunks per query tile (grid.x)
  int min_chunk;    // fewest 64-row tiles per chunk
  int pool_stride;  // candidate pool keys per (wave, query): >= k + 64
  int kpl;          // pool keys per lane when it is sorted
  size_t lds_bytes;
  int64_t chunk_tiles;  // > 0: chunk grid cell in tiles (interval scans); 0: equal chunks
  bool abs_cells;       // chunk c is absolute grid cell c (splits = cells of the whole index)
  bool shared_bound;    // wavefronts publish their best keys for a workgroup bound (k <= 16)
  int seed_tiles;       // > 0: seeded bound from up to this many tiles per wavefront
};

// Largest query tile whose tables and pools fit the LDS budget (0 if none).
int scan_max_qtile(int m, int lut_bytes, int k);
// Dynamic LDS of one scan workgroup.
size_t scan_lds_bytes(int m, int qtile, int lut_bytes, int pool_stride);
// Round a requested tile down to one this build instantiates.
int scan_supported_qtile(int want);
int pool_kpl(int k);
int pool_stride_for(int k);

// Everything the scan needs about the batch.
struct ScanBatch {
  const uint32_t* codes_t;
  int64_t n, n_tiles;
  int m, mw;
  const void* lut;              // [nq][m][256] by original query index
  int lut_dtype;
  int nq;
  const int32_t* qorder;        // tile position -> original query index
  const int64_t* iv;            // [nq][2] row interval per original query
  const DevPred* preds;         // residual_mask per original query
  const uint64_t* bitmap;       // [nq][stride64] physical-order selection words
  int64_t stride64;
  const int32_t* perm;          // physical row -> original id (null: identity)
  int k;
  uint64_t* partials;           // [nq positions][splits][waves][k]
  uint64_t* gthr;               // [nq] shared thresholds, all-ones before the scan
  const int32_t* mode;          // [nq] 1: the query is scored by the gather scan (null: none is)
  const int32_t* slot_order;    // chunk-grid dispatch order (null: slots in index order)
  unsigned long long* lookup_hist;  // [65] non-null: run the read-counting build (see scan_can_count)
};

// Gather scan of compacted row lists (masked batches, few selected rows).
struct GatherBatch {
  const uint32_t* codes_rm;     // [n][rw] row-major code words, physical order
  int rw;                       // words per row (16-byte multiple)
  int m;
  const void* lut;
  int lut_dtype;
  int nq;
  const int32_t* qorder;
  const int32_t* mode;
  const int32_t* lists;         // [nq][list_cap] ascending physical rows
  const int32_t* list_n;
  int64_t list_cap;
  int gblocks;                  // workgroups per query position (<= splits)
  int splits;
  const int32_t* perm;
  int k, pool_stride, kpl;
  uint64_t* partials;
  uint64_t* gthr;
};
bool gather_supported(int m, int lut_dtype);
int gather_row_words(int m);
size_t gather_lds_bytes(int pool_stride);
int gather_blocks_per_query(int64_t list_cap, int splits);
hipError_t launch_rowmajor_codes(const uint32_t* codes_t, int64_t n, int mw, int rw, uint32_t* codes_rm,
                                 hipStream_t s);
// Per query: mode (1 when its pool holds at most max_rows rows; max_rows < 0:
// never) and, for those, the ascending list of selected physical rows.
hipError_t launch_compact(const uint64_t* bitmap, int64_t stride64, const unsigned long long* counts,
                          const uint32_t* count_prefix, int64_t parts, int nq, int64_t max_rows,
                          int64_t list_cap, int32_t* lists, int32_t* list_n, int32_t* mode, hipStream_t s);
hipError_t launch_gather_scan(const GatherBatch& b, hipStream_t s);

hipError_t launch_scan(const ScanBatch& b, const ScanPlan& plan, hipStream_t s);
// Predicate encoder (k_encoder.hip): w_z [nq][D] of the predicates in
// `preds` (device-readable DevPred records) through the packed parameters
// (layout in ifvs.h), H <= 128 a multiple of 16, F <= 256 a multiple of 16.
// With cond, the launch also writes what launch_condition would for the
// same queries and w_z (bit for bit): w_f = softplus(w_z), and alpha when
// cond->alpha is set (h hash functions over the bank).
struct EncCondition {
  const float* q = nullptr;      // [nq][D] queries (for the fingerprint)
  const float* bank = nullptr;   // [bank_rows][mr]
  int bank_rows = 0, mr = 0, h = 0;
  uint64_t seed = 0;
  float* alpha = nullptr;        // [nq][mr], or null: w_f only
  float* wf = nullptr;           // [nq][D]
};
size_t encoder_lds_bytes(int H, int F, int layers);
// Whether the encoder can condition in-launch: any index without a bank,
// else h of at most 4.
bool encoder_conditions(int h, bool has_bank);
// With iv, the launch also does launch_intervals' work for the batch (in
// workgroups of its own beside the encoder's).
hipError_t launch_encoder(const float* params, const double* off, const double* scale, int H, int heads, int layers,
                          int F, int D, int n_attr, const DevPred* preds, int nq, float* wz, hipStream_t s,
                          const EncCondition* cond = nullptr, const IntervalArgs* iv = nullptr);

// Whether a read-counting build of the scan exists for this plan (one query
// per tile, M of 16, 48 or 120).
bool scan_can_count(int m, int qtile, int lut_dtype);
// Coarse quantizer (k_coarse.hip).  Per layout row one word: centroid id in
// the low 16 bits, the radius ||c0 - x0|| rounded up to a bfloat16 in the
// high 16.
int64_t coarse_samples(int64_t n, int C);
float coarse_keep(int m, int dsub, int lut_dtype);   // 1 - eps on squared distances
float coarse_abs(int m, int lut_dtype);              // absolute rounding allowance of a table sum
hipError_t launch_coarse_sample(const uint32_t* codes_t, int mw, int m, int dsub, const float* cpq, int64_t S,
                                int64_t stride, float* X, hipStream_t s);
hipError_t launch_coarse_kmeans_step(const float* X, int64_t S, int D, float* cent, int C, int32_t* assign,
                                     hipStream_t s);
hipError_t launch_coarse_encode(const float* cent, int C, int m, int mw, int dsub, const float* cpq, uint32_t* cc,
                                float* chat, hipStream_t s);
hipError_t launch_coarse_rows(const uint32_t* codes_t, int64_t n, int64_t n_pad, int m, int mw, int dsub,
                              const float* cpq, const float* chat, int C, uint32_t* words, hipStream_t s);
// Per query: bounds [nq][2] = {sqrt(max w) widened, delta widened} of tables
// built with alpha (null: no conditioning) and wf (null: w = 1); parts is a
// [nq][2][m] workspace.
hipError_t launch_lut_bounds(const float* alpha, const float* wf, const float* cpq, const float* W, int nq, int m,
                             int r, int dsub, float* parts, float* bounds, hipStream_t s);
// The first of those two kernels alone (the list plan finishes the bounds).
hipError_t launch_bound_parts(const float* alpha, const float* wf, const float* cpq, const float* W, int nq, int m,
                              int r, int dsub, float* parts, hipStream_t s);
float bound_grow(int m, int dsub);   // delta's rounding allowance
// List order: rows grouped by sub-list s = (centroid c, radius band b),
// s = c * kBands + b, positions [sub_off[s], sub_off[s+1]), each sub-list in
// layout order.  Code tiles and original ids gathered through src_rows[p] =
// layout row of position p.
hipError_t launch_gather_list(const uint32_t* src_t, int mw, const int32_t* perm, const int32_t* src_rows, int64_t n,
                              int64_t n_tiles, uint32_t* dst_t, int32_t* ids, hipStream_t s);

// List scan (k_listscan.hip): the Rank and Select stages over the items of
// each query in bound order, persistent workgroups taking jobs (chunks of a
// query's tiles) from a table built after the plan.
constexpr int kListJobs = 16;     // most jobs (and partial-list slots) per query
constexpr int kJobTiles = 1024;   // tiles per job before a query is split further
constexpr int kListPreGroups = 3; // subspace groups whose code words the list scan fetches ahead
struct ListJobArgs {
  const float* hdr;         // [nq][4] list plan headers ([1]: tiles to scan, int bits)
  const int32_t* qorder;
  int nq, np2;              // np2: power of two >= nq
  int k, max_jobs;          // max_jobs <= kListJobs
  int4* jobs;               // [nq * kListJobs] (position, chunk, first tile position, end)
  int32_t* n_keys;          // [positions] partial keys written per position
  int* job_next;
  int* job_total;
};
// Per-query list plan (one workgroup per original query index).
struct ListPlanArgs {
  const void* lut;          // [nq][m][256] tables (fp32 or binary16)
  int m, nq;
  const uint32_t* cc_t;     // [mw][C] centroid code words
  int mw, C, n_sub;         // n_sub = C * kBands sub-lists
  const float* parts;       // [nq][2][m] bound_parts output; the plan reduces it to sqrt(max w), delta
  float grow;               // delta's rounding allowance (launch_lut_bounds)
  const int64_t* iv;        // [nq][2] layout row interval of each query
  const int32_t* cnt_f;     // [(n >> f_shift) + 1][n_sub]: rows of sub-list s among layout rows [0, b << f_shift)
  int f_shift;
  const uint32_t* words;    // [n] layout row words (centroid id in the low 16 bits)
  const uint8_t* band;      // [n] layout row radius band
  const int32_t* sub_off;   // [n_sub + 1]
  const float* rmax;        // [n_sub] largest radius of each sub-list
  const int32_t* lrow;      // [n] list position -> layout row
  const uint32_t* codes_t;  // list-order code tiles (the seed's rows)
  int k;
  uint64_t* gthr;           // [nq] the queries' shared thresholds (the seed lowers them)
  float keep, abs_m;
  // Outputs by original query: items [nq][n_sub] in increasing bound order,
  // and a header [nq][4] = {items (int bits), tiles (int bits), sqrt(max w),
  // delta}.
  int32_t* it_r0;           // first list position of the item's rows
  int32_t* it_r1;           // one past the last
  int32_t* it_t;            // 64-row tiles the items before it touch
  float* it_lb;             // lower bound of the distance of every row of the sub-list (NaN: none)
  float* hdr;
  uint32_t* slots;          // [nq][kListSlots] the list scan's union-bound slots, reset here
};
size_t list_plan_lds_bytes(int m, int lut_dtype, int C);
hipError_t launch_list_plan(const ListPlanArgs& a, int lut_dtype, hipStream_t s);
// The job table from the plan's headers (one workgroup).
hipError_t launch_list_jobs(const ListJobArgs& a, hipStream_t s);

size_t list_jobs_lds_bytes(int nq);   // the job table's LDS (one workgroup sorts the batch)
struct ListScanArgs {
  const uint32_t* codes_t;  // [n_tiles][mw][64] list-order code words
  const int32_t* ids;       // list position -> original id
  int m, mw;
  const void* lut;          // [nq][m][256] by original query
  int nq, max_jobs;         // max_jobs: the partial-list slots per query (<= kListJobs)
  const int32_t* qorder;    // position -> original query
  const int4* jobs;         // job table (launch_list_jobs)
  int* job_next;            // job counter (0 before the scan)
  const int* job_total;
  const int32_t* it_r0;
  const int32_t* it_r1;
  const int32_t* it_t;
  const float* it_lb;
  const float* hdr;
  int C;                    // item stride per query (sub-lists)
  float keep, abs_m;
  int k, pool_stride, kpl;
  uint64_t* partials;       // [positions][max_jobs][kScanWaves][k]
  uint64_t* gthr;           // [nq] shared thresholds, all ones before the scan
  uint32_t* slots;          // [nq][kListSlots] union-bound slots, all ones before the scan (list plan)
  unsigned long long* lookup_hist;  // [kReadHistEntries] non-null: the counting build (table reads by lanes,
                                    // [0] tiles, [65] tiles whose later code words were fetched)
  int union_bound;          // 1: the query-wide union bound of the wavefronts' best distances
};
constexpr int kListSlots = 2 * kScanWaves * kListJobs;   // two per wavefront of each job of a query
bool list_scan_supported(int m, int lut_dtype);
size_t list_scan_lds_bytes(int m, int lut_dtype, int pool_stride);
hipError_t launch_list_scan(const ListScanArgs& a, int lut_dtype, hipStream_t s);

// LDS gather probe (k_probe.hip): wavefront-level 4-byte random LDS reads per
// second, chip-wide, with `active` lanes (1..64) per read, measured over
// `reps` launches of wg_per_cu eight-wavefront workgroups per CU.
hipError_t lds_gather_probe(int active, int iters, int wg_per_cu, int reps, hipStream_t s, double* wave_reads_per_s);

hipError_t launch_topk_merge(const uint64_t* partials, int nq, int64_t per_query, int k,
                             const int64_t* iv, int64_t cell_tiles, int64_t slot_keys,
                             const int32_t* qorder, int32_t* ids_out, float* dist_out,
                             hipStream_t s, const int32_t* n_keys = nullptr);   // n_keys: keys per position

// Symmetric distance computation (k_sdc.hip): the codeword table
// T[m][a][b] (at load) and a query's table, the rows T[m][enc(q)_m] laid
// out as [nq][m][256] fp32 (lut_dtype 0) or binary16 (1).
hipError_t launch_sdc_table(const float* cpq, int m, int dsub, float* T, hipStream_t s);
hipError_t launch_sdc_lut(const float* q, int dim, int m, int dsub, const float* cpq, const float* T, int nq,
                          int lut_dtype, void* lut_out, hipStream_t s);

// Exact filtered kNN over the full-precision vectors (k_exact.hip).
int exact_ksteps(int dim);                 // 16-dimension MFMA steps
int64_t exact_bins_per_query(int splits, int bin_lanes);  // pass-1 values per query position
int64_t exact_chunk_quantum();             // screening chunks are multiples of this many rows
// Per physical row r (original row perm[r]): fp32 copies in 64-row tiles
// xt[(r / 64 * dim + j) * 64 + r % 64] and row-major xr[r * dim + j], bf16
// MFMA fragments xb, |x|^2 xn
// ([ceil(n/32)*32], zero past n); the largest row norm as fp32 bits
// (*max_norm_bits must start at 0) and the count of non-finite values (*bad,
// starts at 0).
hipError_t launch_exact_stage(const float* x, int64_t n, int dim, const int32_t* perm, float* xt, float* xr,
                              uint4* xb, float* xn, unsigned* max_norm_bits, unsigned long long* bad, hipStream_t s);
// Reconstructions x[r][m * dsub + j] = C_PQ[m][code of physical row r][j]
// (physical row order) from the 64-row code tiles.
hipError_t launch_decode(const uint32_t* codes_t, int64_t n, int m, int mw, int dsub, const float* cpq, float* x,
                         hipStream_t s);
// Query fragments (ceil(nq/32) tiles), |q|^2, error bounds; clears cand_n.
hipError_t launch_exact_queries(const float* q, int dim, int nq, const int32_t* qorder, const unsigned* max_norm_bits,
                                uint4* qb, float* qn, float* eps, int32_t* cand_n, hipStream_t s);
struct ExactScreen {
  const uint4* xb;
  const float* xn;
  int dim;
  const uint4* qb;
  const float* qn;
  const float* thr;
  const int32_t* qorder;
  const int64_t* iv;
  const DevPred* preds;
  const uint64_t* bitmap;
  int64_t stride64;
  int nq;
  int64_t chunk_rows;
  int splits;
  int bin_lanes;          // lanes (power of two <= 32) whose row minima share a bin
  float* bins;            // [positions][exact_bins_per_query(splits, bin_lanes)]
  int32_t* cand;          // [positions][cand_cap]
  int32_t* cand_n;
  int64_t cand_cap;
};
hipError_t launch_exact_screen(const ExactScreen& e, int pass, hipStream_t s);
hipError_t launch_exact_threshold(const float* bins, int64_t n_bins, int nq, int k, const float* eps, float* thr,
                                  hipStream_t s);
struct ExactRerank {
  const float* xt;        // [ceil(n/64)][dim][64] fp32, physical order
  const float* xr;        // [n][dim] fp32, physical order
  int dim;
  const float* q;         // [nq original][dim]
  const int32_t* qorder;
  const int64_t* iv;
  const DevPred* preds;
  const uint64_t* bitmap;
  int64_t stride64;
  const int32_t* perm;
  const int32_t* cand;    // null cand_n: score every selected row of the interval
  const int32_t* cand_n;
  int64_t cand_cap;
  int nq, k, chunks;
  uint64_t* partials;     // [positions][chunks][k]
};
hipError_t launch_exact_rerank(const ExactRerank& e, hipStream_t s);

}  // namespace ifvs
