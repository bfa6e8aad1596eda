/*
 * ifvs.h -- C ABI of the iFVS filtered vector search hot path for AMD MI355X
 * (gfx950).
 *
 * The method (iFVS, "Towards Instance-Optimized Filtered Vector Search",
 * Section 2) answers a filtered query <q, f> over a fixed PQ-quantized dataset
 * in three stages -- Filter, Rank, Select -- using a codebook conditioned on
 * the query and its predicate:
 *
 *   alpha = sum of h memory-bank rows chosen by hashing <q, f>   (Section 2, opening paragraph)
 *   w_f   = softplus(w_z),  Delta = alpha . W,  C_iFVS = C_PQ + Delta   (Section 2, first display)
 *   Filter: evaluate f over each vector's attributes -> candidate pool P
 *   Rank:   weighted distance of q to each candidate reconstructed from C_iFVS
 *           (the score display of Section 2 equals sum w q^2 minus this distance)
 *   Select: the k best candidates (Section 1 SQL listing: ORDER BY ... LIMIT K)
 *
 * Conventions shared by every call
 *  - Every call returns an ifvs_status; nothing throws across the boundary.
 *    On a non-OK status ifvs_last_error() describes the failure.
 *  - Host-side validation runs before anything is enqueued: a call that fails
 *    validation enqueues no work and writes no output.
 *  - Per-call arrays are caller-owned DEVICE memory unless stated otherwise;
 *    the library never frees caller memory.  Predicates are HOST arrays.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *    the call returns; outputs are valid once the stream has synchronized.
 *    One index handle serves one stream at a time: calls on one handle from
 *    different streams or threads concurrently race on its workspace.
 *  - Device faults surface as IFVS_E_HIP at a later synchronizing call.
 *  - The hot calls (select_codebook, build_lut, filter, filtered_search)
 *    allocate nothing: their scratch lives in the index's workspace, sized at
 *    load by max_batch and max_k.
 */
#ifndef IFVS_H
#define IFVS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ifvs_status;
#define IFVS_OK             0
#define IFVS_E_INVALID     (-1)   /* bad argument (pointer, size, shape, k, column, ...) */
#define IFVS_E_NOMEM       (-2)   /* device or pinned host allocation failed (load only)  */
#define IFVS_E_HIP         (-3)   /* a HIP runtime call failed; see ifvs_last_error()     */
#define IFVS_E_UNSUPPORTED (-4)   /* valid request this build cannot serve (e.g. LDS budget) */
#define IFVS_E_STATE       (-5)   /* call on a NULL handle                                */

#define IFVS_MEM_HOST   0
#define IFVS_MEM_DEVICE 1

#define IFVS_LUT_F32 0            /* distance table entries in fp32 (the exact mode)        */
#define IFVS_LUT_F16 1            /* entries rounded to binary16 (nearest even), summed in fp32 */

#define IFVS_KSUB        256      /* codewords per subspace: 8-bit PQ codes                 */
#define IFVS_MAX_CLAUSES 4
#define IFVS_MAX_K       1024
#define IFVS_MAX_ATTR    16

typedef struct ifvs_index ifvs_index;   /* opaque; library-owned device state */

/* Everything ifvs_load_index needs.  All arrays live in the memory named by
 * mem_kind (all host or all device).  Shapes follow Section 2: D = dim,
 * M = m subspaces of d = dim/m dimensions, K = ksub = 256 codewords, r
 * adjustment directions, a bank of B = bank_rows rows, h hash functions. */
typedef struct {
  int64_t n;                 /* number of base vectors, 1 <= n < 2^31                     */
  int32_t dim;               /* D, 1 <= dim <= 4096                                        */
  int32_t m;                 /* M, dim % m == 0, m <= 256                                  */
  int32_t ksub;              /* must be 256                                                */
  int32_t n_attr;            /* relational attribute columns, 0..IFVS_MAX_ATTR             */
  const uint8_t* codes;      /* [n][m] row-major PQ codes                                  */
  const float*   codebook;   /* C_PQ [m][256][dim/m]                                       */
  const int32_t* attrs;      /* [n_attr][n] column-major attribute values (NULL if n_attr==0) */
  int32_t bank_rows;         /* B; 0 = no memory bank (alpha = 0, the identity of Section 2) */
  int32_t r;                 /* adjustment directions, 1..64 when bank_rows > 0             */
  int32_t h;                 /* hash functions, 1..16 when bank_rows > 0                    */
  int32_t mem_kind;          /* IFVS_MEM_HOST or IFVS_MEM_DEVICE                           */
  uint64_t hash_seed;        /* seeds the h hash functions                                 */
  const float* bank;         /* memory bank [bank_rows][m*r] (NULL if bank_rows == 0)      */
  const float* W;            /* direction tensor [m][r][256][dim/m] (NULL if bank_rows == 0) */
  int32_t max_batch;         /* largest nq of any later call (sizes the workspace), >= 1    */
  int32_t max_k;             /* largest k of any later call, 1..IFVS_MAX_K                 */
  int32_t n_cluster;         /* 0: rows stay in id order; 1 or 2: rows are stored sorted by */
  int32_t cluster_col[2];    /*   attribute columns cluster_col[0] (major), [1] (minor), id */
} ifvs_index_desc;

/* One clause lo <= attr[col] < hi (half-open, int64 bounds so that any int32
 * attribute value can be included or excluded).  lo >= hi is an empty clause
 * (nothing passes), not an error.  =v is [v, v+1); >v is [v+1, INT64_MAX);
 * <=v is [INT64_MIN, v+1). */
typedef struct {
  int32_t col;               /* attribute column, 0 <= col < n_attr */
  int32_t reserved;          /* must be 0 */
  int64_t lo;
  int64_t hi;
} ifvs_clause;

/* A predicate f: the conjunction of n_clauses clauses (Section 1 SQL listing:
 * WHERE col1 > v1 AND col2 = v2); n_clauses == 0 is TRUE. */
typedef struct {
  int32_t n_clauses;         /* 0..IFVS_MAX_CLAUSES */
  int32_t reserved;          /* must be 0 */
  ifvs_clause c[IFVS_MAX_CLAUSES];
} ifvs_predicate;

/* ifvs_load_index -- make a quantized dataset resident on the current device
 * (Abstract and Section 2: a fixed, quantized vector dataset).
 *  desc: shapes and arrays, see ifvs_index_desc.  The arrays are deep-copied
 *        into library-owned device memory (codes are re-laid out into 64-row
 *        interleaved tiles for coalesced reads); the caller may free them
 *        after return.  The index is immutable afterwards.
 *        With n_cluster > 0 the rows are stored in the order of their
 *        cluster-key attribute values (an instance-optimized layout: the
 *        paper tailors components to a dataset and its query workload).  A
 *        clause on cluster_col[0] -- or an equality on it plus a clause on
 *        cluster_col[1] -- then selects one contiguous run of rows, so the
 *        search reads only those rows; other clauses are still tested row
 *        by row.  Results (ids, order, ties) are identical on both layouts.
 *  out:  receives the handle; free it with ifvs_free_index.
 * Errors: IFVS_E_INVALID for shapes outside the ranges above or NULL arrays,
 * IFVS_E_NOMEM if an allocation fails (nothing is leaked), IFVS_E_HIP. */
ifvs_status ifvs_load_index(const ifvs_index_desc* desc, ifvs_index** out);

/* Release every device and host resource of the handle (NULL is a no-op).
 * Synchronizes the device first so no enqueued work still uses the index. */
void ifvs_free_index(ifvs_index* idx);

/* ifvs_select_codebook -- per-query conditioning (Section 2, opening
 * paragraph and first display).  For each query i < nq:
 *   key   = FNV-1a-64 over q_i's fp32 bytes, then preds[i].n_clauses (int32),
 *           then each clause as (col int32, lo int64, hi int64), little-endian
 *   row_j = SplitMix64(key XOR SplitMix64(hash_seed + j)) mod B,  j < h
 *   alpha_i = bank[row_0] + bank[row_1] + ... (fp32, in j order, from +0)
 *   w_f_i   = softplus(w_z_i) evaluated in fp64, rounded once to fp32
 *  q:         device [nq][dim] fp32
 *  preds:     HOST [nq] predicates (hashed exactly as given)
 *  w_z:       device [nq][dim] fp32, or NULL: w_f = 1 exactly
 *  alpha_out: device [nq][m*r] fp32; may be NULL only when bank_rows == 0
 *             (then nothing is written for alpha)
 *  wf_out:    device [nq][dim] fp32
 * Errors: IFVS_E_INVALID (nq outside 1..max_batch, NULL q / wf_out, bad
 * predicate), IFVS_E_STATE (NULL handle), IFVS_E_HIP. */
ifvs_status ifvs_select_codebook(ifvs_index* idx, int32_t nq, const float* q,
                                 const ifvs_predicate* preds, const float* w_z,
                                 float* alpha_out, float* wf_out, void* stream);

/* ifvs_build_lut -- each query's asymmetric distance table over its
 * conditioned codebook (Section 2 first display and Rank stage):
 *   C[m][c][j]  = C_PQ[m][c][j] + sum_{t<r} alpha[m*r+t] * W[m][t][c][j]
 *   LUT[m][c]   = sum_{j<d} w_f[m*d+j] * (q[m*d+j] - C[m][c][j])^2
 * in fp32 with every operation rounded (no fused multiply-add), t and j summed
 * in index order from +0.
 *  q:       device [nq][dim] fp32
 *  alpha:   device [nq][m*r] fp32, or NULL: Delta = 0 (C_iFVS = C_PQ)
 *  wf:      device [nq][dim] fp32, or NULL: w_f = 1
 *  lut_dtype: IFVS_LUT_F32 or IFVS_LUT_F16 (entries rounded to nearest even
 *           binary16; values beyond its range become +inf)
 *  lut_out: device [nq][m][256] of fp32 or binary16
 * Errors: IFVS_E_INVALID (nq, NULL q / lut_out, alpha given with no bank,
 * unknown dtype), IFVS_E_STATE, IFVS_E_HIP. */
ifvs_status ifvs_build_lut(ifvs_index* idx, int32_t nq, const float* q, const float* alpha,
                           const float* wf, int32_t lut_dtype, void* lut_out, void* stream);

/* ifvs_build_sdc_lut -- the symmetric distance table of each query, for the
 * pre-filtering SDC baselines (iv) and (v) of Section 3.2: the query is
 * quantized with the index's codebook C_PQ,
 *   code[m]     = the c minimizing sum_{j<d} (q[m*d+j] - C_PQ[m][c][j])^2
 *                 (fp32, j order from +0; the lowest c among equals),
 * and LUT[m][c] = T[m][code[m]][c] with the codeword-to-codeword distances
 *   T[m][a][b]  = sum_{j<d} (C_PQ[m][a][j] - C_PQ[m][b][j])^2
 * (fp32, j order from +0; built once by ifvs_load_index).  Passed to
 * ifvs_filtered_search it ranks the pool by SDC distance.
 *  q:         device [nq][dim] fp32
 *  lut_dtype: IFVS_LUT_F32 or IFVS_LUT_F16 (as ifvs_build_lut)
 *  lut_out:   device [nq][m][256]
 * Errors: IFVS_E_INVALID (nq, NULL q / lut_out, unknown dtype), IFVS_E_STATE,
 * IFVS_E_HIP. */
ifvs_status ifvs_build_sdc_lut(ifvs_index* idx, int32_t nq, const float* q, int32_t lut_dtype, void* lut_out,
                               void* stream);

/* ifvs_filter -- the Filter stage alone (Section 2, stage 1): selection
 * bitmaps and pool sizes.
 *  preds:      HOST [nq]
 *  bitmap_out: device [nq][ceil(n/32)] uint32; vector i of query q is bit
 *              (i mod 32) of word (i div 32), least significant bit first;
 *              bits past n are 0
 *  count_out:  device [nq] int64 pool sizes |P_q|, or NULL
 * Errors: IFVS_E_INVALID (nq, NULL bitmap_out, column out of range,
 * n_clauses > 4, nonzero reserved fields), IFVS_E_STATE, IFVS_E_HIP. */
ifvs_status ifvs_filter(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                        uint32_t* bitmap_out, int64_t* count_out, void* stream);

/* ifvs_filtered_search -- Filter, Rank and Select for a batch (Section 2,
 * stages 1-3).  For each query q: the candidate pool P_q = vectors whose
 * attributes satisfy preds[q]; dist(v) = sum_{m<M} LUT_q[m][code_v[m]]
 * (fp32, m in index order from +0; an fp16 table is widened entry by entry);
 * the k smallest (dist, id) pairs in ascending order, ties to the smaller id.
 *  preds:      HOST [nq]
 *  lut:        device [nq][m][256] in lut_dtype (from ifvs_build_lut)
 *  k:          1..max_k
 *  ids_out:    device [nq][k] int32; rows with |P_q| < k end in id -1
 *  dist_out:   device [nq][k] fp32; +inf where the id is -1
 *  bitmap_out: device [nq][ceil(n/32)] uint32: the batch's selection
 *              bitmaps exactly as ifvs_filter writes them, or NULL
 * Errors: IFVS_E_INVALID (nq, k, NULL lut / ids_out / dist_out, predicate
 * errors as in ifvs_filter, unknown dtype), IFVS_E_UNSUPPORTED (one query's
 * fp32 table plus its top-k pool exceeds the 160 KB LDS budget: use
 * IFVS_LUT_F16), IFVS_E_STATE, IFVS_E_HIP. */
ifvs_status ifvs_filtered_search(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                                 const void* lut, int32_t lut_dtype, int32_t k,
                                 int32_t* ids_out, float* dist_out, uint32_t* bitmap_out,
                                 void* stream);

/* ifvs_filtered_search_noalloc -- ifvs_filtered_search for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation calls.  Same arguments and the same
 * results, bit for bit; the call allocates nothing.  Its workspace is a
 * static array of 64 MiB of device memory, one copy per GPU, placed with the
 * library's code object and held until the process ends.
 *  - Every call on one GPU uses that GPU's array: calls that overlap on one
 *    GPU (other streams or threads, any index handle) race and corrupt each
 *    other's results, so serialize them.  The array keeps the last call's
 *    contents; nothing in it has to start at zero.
 *  - A batch takes 256 + 28 bytes per query (predicates, order, intervals,
 *    thresholds), 1 MiB of scan dispatch order, ceil(n/64) * 8 bytes of
 *    selection words per query when a predicate has clauses the row order
 *    does not resolve (or bitmap_out is given), and k * 64 bytes per query
 *    and code chunk of top-k partials; the number of chunks adapts to the
 *    room that is left.
 *  - Masked batches score every query by the tiled scan (no row-list gather).
 * Errors: as ifvs_filtered_search, plus IFVS_E_INVALID when the batch does not
 * fit the 64 MiB with one code chunk per query (send fewer queries per call,
 * or use ifvs_filtered_search). */
ifvs_status ifvs_filtered_search_noalloc(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                                         const void* lut, int32_t lut_dtype, int32_t k,
                                         int32_t* ids_out, float* dist_out, uint32_t* bitmap_out,
                                         void* stream);

/* ---- Coarse bound: exact pruning of the Rank stage ---------------------
 * The Rank stage (Section 2, stage 2) sums M table entries per candidate.  A
 * coarse quantizer of the index's reconstructions gives, per query, a lower
 * bound on every candidate's distance, so candidates that cannot enter the
 * top k are dropped without reading their codes.  With C_c the candidate's
 * coarse centroid (itself a vector of PQ codes) and the triangle inequality
 * in the weighted norm of w_f:
 *   sqrt(dist(v)) >= sqrt(dist(C_c)) - sqrt(max_j w_f[j]) * (r_v + delta)
 * where r_v = ||C_PQ(v) - C_PQ(C_c)|| (stored per row at build) and delta =
 * sqrt(sum over m of (2 max_c ||Delta[m][c]||)^2) bounds what the
 * conditioning Delta = alpha . W (Section 2, first display) adds between two
 * code vectors.  The index keeps a second copy of its codes grouped by
 * centroid and radius band (each centroid's rows split at its radius
 * quantiles 0.5, 0.85 and 0.97), so a group's largest radius bounds all of
 * its rows.  The list scan visits a query's groups in increasing order of
 * that bound and stops at the first one whose bound exceeds the query's
 * current k-th distance.  Every term carries a rounding allowance, so a
 * dropped candidate's computed distance exceeds the query's k-th: results
 * are identical, bit for bit, to ifvs_filtered_search. */

/* ifvs_build_coarse -- k-means over the reconstructions of evenly spaced
 * rows (max(64 n_centroids, 65536) of them, at most n), starting from
 * n_centroids evenly spaced rows and running `iters` iterations (sums in a
 * fixed order: the build is deterministic); the centroids are then encoded
 * with C_PQ and every row gets its nearest encoded centroid and its
 * distance to it, rounded up to a bfloat16; then the grouped copy of the
 * codes.  Synchronous; replaces any earlier coarse quantizer.  Costs about
 * n * (4 ceil(m/4) + 13) bytes of device memory (codes, ids, row words,
 * bands and list positions), a rank table of at most 64 MiB, and max_batch *
 * n_centroids * 64 + max_batch * 1300 bytes of list-plan workspace.
 * Errors: IFVS_E_INVALID (n_centroids outside 1..4096 or above n, iters
 * outside 0..1000), IFVS_E_UNSUPPORTED (dim > 128), IFVS_E_STATE,
 * IFVS_E_NOMEM, IFVS_E_HIP. */
ifvs_status ifvs_build_coarse(ifvs_index* idx, int32_t n_centroids, int32_t iters);

/* ifvs_lut_bounds -- the two per-query factors of the coarse bound (what
 * ifvs_filtered_search_bounded computes inside), for tables built by
 * ifvs_build_lut with the same alpha and wf (NULL and NULL for
 * ifvs_build_sdc_lut's tables):
 *   bounds_out[2i]     >= sqrt(max_j wf_i[j]) (1 when wf is NULL; NaN, which
 *                         disables the bound for that query, when a weight
 *                         is negative or not finite)
 *   bounds_out[2i + 1] >= delta_i, the conditioned codewords recomputed with
 *                         the table build's own operations (0 when alpha is
 *                         NULL)
 *  alpha: device [nq][m*r] or NULL;  wf: device [nq][dim] or NULL
 *  bounds_out: device [nq][2] fp32, caller-owned
 * Enqueued on `stream`.  Errors: IFVS_E_INVALID (nq, NULL bounds_out, alpha
 * given with no bank), IFVS_E_STATE, IFVS_E_HIP. */
ifvs_status ifvs_lut_bounds(ifvs_index* idx, int32_t nq, const float* alpha, const float* wf, float* bounds_out,
                            void* stream);

/* ifvs_filtered_search_bounded -- ifvs_filtered_search with the coarse
 * bound.  alpha and wf are the operands the tables were built with
 * (ifvs_build_lut's; either may be NULL, and both are NULL for
 * ifvs_build_sdc_lut's tables): when the list scan runs, the call computes
 * the bound's factors from them as ifvs_lut_bounds does and drops
 * candidates by the bound.  Same results as ifvs_filtered_search, bit for
 * bit, whenever alpha and wf are the tables' operands; others can drop true
 * neighbours.  The list scan runs once ifvs_build_coarse has run, when every
 * query's selection is a run of rows of the index's layout (no clause
 * tested row by row), M is 16, 48 or 120, nq is at most 16384 and its
 * workspace holds the batch
 * (IFVS_OPT_COARSE: automatic for batches whose widest interval spans 8192
 * or more 64-row tiles, on indexes of 32 or more subspaces); otherwise the
 * call is ifvs_filtered_search.  The
 * list scan adds the bound kernels, one planning kernel per call (one
 * workgroup per query orders the query's groups by their bound) and a job
 * table kernel; the scan's workgroups take chunks of the queries' work from
 * the table, the queries with the most work first.  IFVS_OPT_SPLITS caps a
 * query's chunks (at most 16, the default).
 * Errors: as ifvs_filtered_search, plus IFVS_E_INVALID for alpha given on an
 * index without a memory bank. */
ifvs_status ifvs_filtered_search_bounded(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds,
                                         const void* lut, int32_t lut_dtype, const float* alpha, const float* wf,
                                         int32_t k, int32_t* ids_out, float* dist_out, uint32_t* bitmap_out,
                                         void* stream);

/* ifvs_query_batch -- the whole path of Section 2 for a batch in one call:
 * the predicate encoder (f -> w_z, when w_z is NULL), the condition (alpha,
 * w_f), the distance tables, then ifvs_filtered_search_bounded with those
 * tables and their operands.  Same outputs, bit for bit, as
 * ifvs_encode_predicates + ifvs_select_codebook + ifvs_build_lut +
 * ifvs_filtered_search_bounded on the same arguments, in fewer launches:
 * the predicates are validated and staged once for all four (each separate
 * call stages them and marks its staging with an event, a few microseconds
 * of the stream's time each); when the encoder runs, its launch also
 * conditions the queries (indexes without a bank, or h of at most 4) and
 * finds their row intervals, and the table kernel then releases the
 * staging slot through a pinned word instead of an event; and when the list
 * scan runs, the table kernel also writes the coarse bound's factors.
 *  q: device [nq][dim];  preds: HOST [nq]
 *  w_z: device [nq][dim], or NULL to encode the predicates with the attached
 *       encoder into wz_out (device [nq][dim], caller-owned; unused when w_z
 *       is given)
 *  alpha_out: device [nq][m*r] (may be NULL on an index without a bank);
 *  wf_out: device [nq][dim];  lut_out: device [nq][m][256] of lut_dtype,
 *  16-byte aligned;  ids_out, dist_out: device [nq][k] -- all caller-owned,
 *  written in stream order.
 * Errors: IFVS_E_INVALID (nq, k, NULL arrays, predicate errors, unknown
 * dtype), IFVS_E_STATE (NULL handle; w_z NULL with no encoder attached),
 * IFVS_E_UNSUPPORTED, IFVS_E_HIP. */
ifvs_status ifvs_query_batch(ifvs_index* idx, int32_t nq, const float* q, const ifvs_predicate* preds,
                             const float* w_z, float* wz_out, float* alpha_out, float* wf_out, int32_t lut_dtype,
                             void* lut_out, int32_t k, int32_t* ids_out, float* dist_out, void* stream);

/* ifvs_read_coarse -- the coarse quantizer, for inspection and tests
 * (synchronous; every output may be NULL): *n_centroids_out; assign_out
 * HOST [n] centroid of each vector id; radius_out HOST [n] its stored
 * radius (an upper bound of ||C_PQ(v) - C_PQ(centroid)||); codes_out HOST
 * [n_centroids][m] the centroids' PQ codes.
 * Errors: IFVS_E_STATE (NULL handle or no coarse quantizer), IFVS_E_HIP. */
ifvs_status ifvs_read_coarse(const ifvs_index* idx, int32_t* n_centroids_out, int32_t* assign_out,
                             float* radius_out, uint8_t* codes_out);

/* ifvs_last_coarse -- *used_out = 1 when the most recent filtered search on
 * this index ran the scan with the coarse bound, else 0.
 * Errors: IFVS_E_INVALID (NULL used_out), IFVS_E_STATE. */
ifvs_status ifvs_last_coarse(const ifvs_index* idx, int32_t* used_out);

/* ifvs_load_vectors -- attach the full-precision base vectors, for exact
 * filtered kNN (ifvs_exact_search).  The paper takes the exact top-k over
 * the predicate-passing vectors as its ground truth (Section 3.1), and its
 * pre-filtering baseline (i) computes exact L2 distances over the
 * full-precision vectors of the candidate set (Section 3.2).
 *  x:        [n][dim] fp32, row i = vector id i, in the memory named by
 *            mem_kind; deep-copied (stored in the index's row order as fp32
 *            twice, in 64-row tiles and row by row, and as bf16 matrix-core
 *            fragments, with each row's squared norm), so the caller may
 *            free it after return.  Costs n * dim * 10 bytes of device
 *            memory plus a workspace sized by
 *            max_batch and max_k (a few hundred MB at most).
 * Errors: IFVS_E_INVALID (NULL x, unknown mem_kind, a NaN or infinite
 * value: nothing is kept), IFVS_E_STATE (NULL handle, or vectors already
 * attached), IFVS_E_NOMEM, IFVS_E_HIP. */
ifvs_status ifvs_load_vectors(ifvs_index* idx, const float* x, int32_t mem_kind);

/* ifvs_train_step -- one training step of the filter-aware conditioning
 * (Section 2, training paragraph): the memory bank and W of the index are
 * updated in place by plain SGD, so later calls use the trained values.
 *
 * For each of the nq training queries (q, preds, w_z as for
 * ifvs_select_codebook), cand[i][0..n_cand) are original vector ids, the
 * first n_pos the query's ground-truth positives and the rest its hard
 * negatives (the caller mines them, e.g. with ifvs_filtered_search); an id
 * outside 0..n-1 (such as -1) is an absent slot.  With d_v the weighted
 * distance of candidate v under the current conditioned codebook
 * (ifvs_build_lut's table, subspaces summed in order) and P the present
 * positives, the query's loss is
 *   L_i = (1/P) sum_{positives p} [ logsumexp_v(-d_v / tau) + d_p / tau ]
 *         + lambda * mean over (m, c, j) of Delta_i[m][c][j]^2
 * (cross-entropy 0 when P = 0) and the step descends the batch mean of L_i:
 *   bank[row] -= lr * dL/dalpha_i for each of query i's h hashed rows,
 *   W -= lr * dL/dW.
 * C_PQ and the codes are not changed.  The arithmetic is fp32 with fp64
 * softmax statistics; the bank update uses atomics, so the order of its
 * additions (and the last bits of the result) may vary between runs.
 *
 * q: device [nq][dim]; preds: host [nq]; w_z: device [nq][dim] or NULL
 * (w_f = 1); cand: device [nq][n_cand] int32; loss_out: device [nq], L_i;
 * dwz_out: device [nq][dim] or NULL, dL/dw_z (the gradient a predicate
 * encoder would receive; requires w_z).  Enqueued on `stream`.  The first
 * call allocates a training workspace sized by max_batch
 * (max_batch * (2 M r + dim + 256 M (1 + dsub)) floats + h ints, and n ints
 * on a clustered index).
 * Errors: IFVS_E_STATE (no memory bank), IFVS_E_INVALID (nq > max_batch,
 * n_cand not in 1..4096, n_pos not in 0..n_cand, tau <= 0, lambda < 0,
 * non-finite tau/lambda/lr, NULL q/cand/loss_out, dwz_out without w_z, bad
 * predicate), IFVS_E_UNSUPPORTED (table + candidates + gradients of one
 * query beyond 160 KB of LDS), IFVS_E_NOMEM, IFVS_E_HIP. */
ifvs_status ifvs_train_step(ifvs_index* idx, int32_t nq, const float* q, const ifvs_predicate* preds,
                            const float* w_z, const int32_t* cand, int32_t n_cand, int32_t n_pos, float tau,
                            float lambda, float lr, float* loss_out, float* dwz_out, void* stream);

/* ifvs_read_params -- copy the index's current memory bank ([bank_rows][m*r])
 * and W ([m][r][256][dim/m]) into caller memory (host or device; either
 * pointer may be NULL), enqueued on `stream`.
 * Errors: IFVS_E_STATE (no memory bank), IFVS_E_HIP. */
ifvs_status ifvs_read_params(const ifvs_index* idx, float* bank_out, float* W_out, void* stream);

/* ifvs_load_reconstructions -- attach, in place of full-precision vectors,
 * the reconstructions of the index's own codes: row i becomes the
 * concatenation over m of codeword C_PQ[m][code_i[m]].  ifvs_exact_search
 * then ranks by exact L2 to the reconstructions -- the pre-filtering
 * baseline (ii) of Section 3.2 (reconstruct from PQ codes, then exact L2).
 * Same memory and workspace as ifvs_load_vectors.
 * Errors: IFVS_E_STATE (NULL handle, or vectors already attached),
 * IFVS_E_NOMEM, IFVS_E_HIP. */
ifvs_status ifvs_load_reconstructions(ifvs_index* idx);

/* ifvs_exact_search -- exact filtered kNN (Section 3.1 ground truth; Section
 * 3.2 pre-filtering baseline (i)).  For each query q: the pool P_q of
 * vectors whose attributes satisfy preds[q] (as in ifvs_filter), ranked by
 *   d(v) = sum_{j<dim} (x_v[j] - q[j])^2
 * summed in j order from +0 in fp32, the difference, its square and each
 * addition rounded separately (no fused multiply-add); the k smallest
 * (d, id) pairs ascending, ties to the smaller id.  Results equal that
 * definition exactly: where many queries share rows, a bf16 matrix-core pass
 * with a rigorous error bound only decides which rows need scoring, and
 * every returned distance is computed as defined.
 *  q:        device [nq][dim] fp32
 *  preds:    HOST [nq]
 *  k:        1..max_k
 *  ids_out:  device [nq][k] int32; rows with |P_q| < k end in id -1
 *  dist_out: device [nq][k] fp32; +inf where the id is -1
 * Errors: IFVS_E_INVALID (nq, k, NULL q / ids_out / dist_out, predicate
 * errors as in ifvs_filter), IFVS_E_STATE (NULL handle, no vectors
 * attached), IFVS_E_HIP.  Non-finite query values give unspecified
 * rankings. */
ifvs_status ifvs_exact_search(ifvs_index* idx, int32_t nq, const float* q, const ifvs_predicate* preds,
                              int32_t k, int32_t* ids_out, float* dist_out, void* stream);

/* ---- Predicate encoder (Section 2, opening paragraph) ------------------
 * The relational predicate f is encoded by a light-weight Transformer into
 * the filter-aware weight vector w_z in R^D (then w_f = softplus(w_z),
 * Section 2 first display).  The paper gives no architecture; this library
 * implements the following one, with caller-supplied (trained) weights:
 *   tokens: a summary token `cls`, then one token per clause (col, lo, hi)
 *     in the predicate's order: col_embed[col] + a * feat_w[0] + b * feat_w[1]
 *     + feat_b, where a = clip((lo - col_offset[col]) * col_scale[col], -1, 2)
 *     and b likewise of hi, computed in double and rounded to float; no
 *     positional encoding.
 *   `layers` pre-norm encoder layers over all tokens:
 *     Z = LN1(X); Q|K|V = Z Wqkv + bqkv; per head (width H / heads)
 *     A = softmax over keys of Q K^T / sqrt(H / heads);
 *     X += concat(A V) Wo + bo;  X += relu(LN2(X) W1 + b1) W2 + b2
 *   w_z = LNf(X[summary]) Wout + bout.
 *   LN(x) = (x - mean) / sqrt(biased variance + 1e-5) * g + b over H;
 *   matrices map row vectors (y = x W + b) and are stored [in][out].
 * `params` packs, as consecutive float arrays: col_embed [n_attr][H],
 * feat_w [2][H], feat_b [H], cls [H]; per layer: ln1_g [H], ln1_b [H],
 * Wqkv [H][3H] (columns: Q, then K, then V), bqkv [3H], Wo [H][H], bo [H],
 * ln2_g [H], ln2_b [H], W1 [H][F], b1 [F], W2 [F][H], b2 [H]; then lnf_g [H],
 * lnf_b [H], Wout [H][dim], bout [dim] -- n_params floats in all
 * (ifvs_encoder_params gives the count).  Arithmetic is fp32 (the
 * projections on matrix cores); results are within 1e-4 relative of the
 * definition in exact arithmetic at the shapes the tests use. */
typedef struct {
  int32_t hidden;             /* H: 16..128, a multiple of 16                    */
  int32_t heads;              /* 1..16, divides H                                */
  int32_t layers;             /* 1..8                                            */
  int32_t ffn;                /* F: 16..256, a multiple of 16                    */
  int64_t n_params;           /* floats in params (must equal ifvs_encoder_params) */
  const float* params;        /* packed weights, layout above                    */
  const double* col_offset;   /* [n_attr] bound offset of each attribute column  */
  const double* col_scale;    /* [n_attr] bound scale of each column (finite)    */
  int32_t mem_kind;           /* IFVS_MEM_HOST | IFVS_MEM_DEVICE, all three arrays */
  int32_t reserved;           /* must be 0 */
} ifvs_encoder_desc;

/* Floats in the packed parameters of an encoder of these sizes for an index
 * of `n_attr` attribute columns and `dim` dimensions; -1 when a size is out
 * of range. */
int64_t ifvs_encoder_params(int32_t hidden, int32_t heads, int32_t layers, int32_t ffn, int32_t n_attr,
                            int32_t dim);

/* ifvs_load_encoder -- attaches an encoder to the index: deep-copies the
 * desc's arrays into library-owned device memory (the caller may free its
 * arrays after return), replacing any earlier encoder.  Synchronous.
 * Errors: IFVS_E_INVALID (sizes out of range, n_params mismatch, NULL
 * arrays, non-finite offset or scale, reserved != 0), IFVS_E_STATE (NULL
 * handle), IFVS_E_NOMEM, IFVS_E_HIP.  On error the earlier encoder (if any)
 * stays attached. */
ifvs_status ifvs_load_encoder(ifvs_index* idx, const ifvs_encoder_desc* desc);

/* ifvs_encode_predicates -- w_z of each predicate through the attached
 * encoder (Section 2, opening paragraph), ready for ifvs_select_codebook.
 *  preds:  HOST [nq], validated as in ifvs_filter (copied inside the call)
 *  wz_out: device [nq][dim] fp32, caller-owned
 * Enqueued on `stream`; nq = 0 writes nothing.
 * Errors: IFVS_E_INVALID (nq outside 0..max_batch, NULL wz_out, predicate
 * errors), IFVS_E_STATE (NULL handle, no encoder attached), IFVS_E_HIP. */
ifvs_status ifvs_encode_predicates(ifvs_index* idx, int32_t nq, const ifvs_predicate* preds, float* wz_out,
                                   void* stream);

/* Tuning knobs, never needed for correctness.  IFVS_OPT_QTILE forces the
 * number of queries whose tables share one LDS residency and one pass over
 * the codes (0 = automatic); IFVS_OPT_SPLITS forces the number of code chunks
 * a query tile is cut into (0 = automatic).  IFVS_OPT_GRID_TILES forces the
 * chunk grid of clustered-index scans (0 = automatic: a grid of about 5120
 * tiles when the widest interval spans 8192 or more 64-row tiles, else none):
 * chunk c of a query tile is then absolute grid cell c (every XCD walks the
 * same cells), or with IFVS_OPT_GRID_RELATIVE grid cell (first cell of its
 * span) + c; a span needing more cells than there are chunks is cut into
 * equal chunks instead.  Results never depend on these knobs.
 * Errors: IFVS_E_INVALID for an unknown option or a negative value. */
#define IFVS_OPT_QTILE  1
#define IFVS_OPT_SPLITS 2
#define IFVS_OPT_PROFILE 3        /* 1: time every kernel launch with HIP events (see below);
                                     2: time only the scan kernels' launches;
                                     3: time only the list scan's launches (coarse bound) */
#define IFVS_OPT_MIN_CHUNK 4      /* fewest 64-row code tiles per chunk (0 = automatic)      */
#define IFVS_OPT_GRID_TILES 5     /* chunk grid cell in 64-row tiles (0 = automatic)         */
#define IFVS_OPT_GRID_RELATIVE 7  /* 1: chunk c of a query tile is cell (its first cell) + c
                                     instead of absolute cell c of the grid                 */
#define IFVS_OPT_GATHER 6         /* masked batches: 0 automatic (queries selecting up to 30% of
                                     the rows, within the row-list capacity, are scored from
                                     their compacted row list), 1 every query whose list fits,
                                     2 never (every query takes the tiled scan)               */
#define IFVS_OPT_SLOT_ORDER 8     /* chunk-grid scans: 0 dispatch whole-cell slots first in cell
                                     order, then the others by decreasing estimated work (the
                                     last workgroups are short), 1 slots in index order       */
#define IFVS_OPT_SHARED_BOUND 9   /* k <= 16: the wavefronts of a scan workgroup publish their
                                     two smallest distances and prune with the k-th smallest
                                     published one: 0 automatic (on for chunk-grid scans whose
                                     widest interval spans 32768 or more 64-row tiles, and for
                                     the list scan, where all wavefronts of the query share
                                     them for k up to twice their number), 1 never, 2 always */
#define IFVS_OPT_SEED_TILES 11   /* one-query scans of M = 16, 48 or 120 with k <= 64: before
                                     scanning, each wavefront ranks the selected rows of its first
                                     n selected tiles by their partial sums over the first
                                     subspace group and computes the full distance of its 8 best;
                                     the k-th smallest of the workgroup's candidate distances
                                     bounds the query's answer from the first tile on.  On a
                                     chunk grid the tiles are the wavefront's first n of its
                                     cell, otherwise 8n tiles drawn evenly from the query's
                                     whole interval (all of them if it has fewer).
                                     0 automatic (n = 64 on chunk-grid cells, off otherwise),
                                     1 never, n > 1 at most n tiles                           */
#define IFVS_OPT_EXACT_PLAN 10    /* ifvs_exact_search: 0 automatic (matrix-core screening when
                                     the batch's queries share rows), 1 score every selected row
                                     exactly, 2 always screen first                           */
#define IFVS_OPT_COARSE 13       /* ifvs_filtered_search_bounded: 0 automatic (the list scan for
                                     batches whose widest interval spans 8192 or more 64-row
                                     tiles, M >= 32), 1 never, 2 whenever the batch allows it  */
#define IFVS_OPT_COUNT_READS 12  /* measurement only: 1 = scans run a build of the scan kernel
                                     that also counts its table reads (one per subspace and
                                     wavefront instruction, and one per coarse-bound lookup)
                                     by the number of active lanes, and the code tiles it sums,
                                     read back with ifvs_read_scan_reads; needs one query per
                                     tile and M of 16, 48 or 120, or the list scan (else the
                                     search fails with IFVS_E_UNSUPPORTED).  Results are unchanged; the counting
                                     adds LDS atomics, so it is not the build to time.  0 = off */
ifvs_status ifvs_set_option(ifvs_index* idx, int32_t option, int64_t value);

/* ifvs_read_profile -- with IFVS_OPT_PROFILE on, every kernel the index
 * launches is bracketed by HIP events recorded on the caller's stream.  This
 * call waits for the recorded events, writes the summed kernel time (ms) and
 * the launch count of each stage, and clears the totals.  Stages, in array
 * order (IFVS_N_STAGES entries each): condition, distance table, filter,
 * scan, top-k merge, predicate encoder, coarse bound (ifvs_lut_bounds and
 * the centroid distances of a bounded search).  Errors: IFVS_E_INVALID
 * (NULL arrays), IFVS_E_STATE, IFVS_E_HIP. */
#define IFVS_N_STAGES 7
ifvs_status ifvs_read_profile(ifvs_index* idx, double* ms_out, int64_t* launches_out);

/* ifvs_read_scan_reads -- with IFVS_OPT_COUNT_READS on: hist_out[n] (66
 * entries) = table reads the scans issued with n of a wavefront's 64 lanes
 * active (a read is one LDS instruction of a wavefront; it fetches n table
 * entries), for n = 1..64, hist_out[0] = the 64-row code tiles the scans
 * summed and hist_out[65] = the tiles the list scan read past their first
 * three groups of subspaces (it fetches those code words only for tiles with
 * a row still live), all summed over the scans since the last call, which
 * it then clears.
 * Waits for `stream`.  The LDS cost of the Rank stage's distance-table
 * lookups (Section 2, stage 2) follows from it and ifvs_probe_lds_gather.
 * All zero when counting was never on.
 * Errors: IFVS_E_INVALID (NULL hist_out), IFVS_E_STATE, IFVS_E_HIP. */
ifvs_status ifvs_read_scan_reads(ifvs_index* idx, int64_t* hist_out, void* stream);

/* ifvs_probe_lds_gather -- a measurement of the current GPU, not a step of
 * the method: the chip-wide rate (*wave_reads_per_s, wavefront instructions
 * per second) of 4-byte LDS reads at random addresses of a 48 KB table, with
 * active_lanes (1..64) lanes per instruction, the access the Rank stage's
 * table lookups make (Section 2, stage 2).  Three workgroups of eight
 * wavefronts per CU; enqueued on `stream`, waited for.  Allocates and frees
 * 4 bytes of device memory.
 * Errors: IFVS_E_INVALID (active_lanes out of range, NULL output), IFVS_E_HIP. */
ifvs_status ifvs_probe_lds_gather(int32_t active_lanes, double* wave_reads_per_s, void* stream);

/* ifvs_last_plan -- the launch plan of the most recent ifvs_filtered_search
 * on this index (all zero before the first): out5[0] queries per tile
 * (tables sharing one LDS residency and one pass over the codes), out5[1]
 * code chunks per query tile, out5[2] fewest 64-row code tiles per chunk,
 * out5[3] LDS bytes per workgroup, out5[4] chunk grid cell in tiles (0: no
 * grid).  For measurement and tests.
 * Errors: IFVS_E_INVALID (NULL out5), IFVS_E_STATE. */
ifvs_status ifvs_last_plan(const ifvs_index* idx, int64_t* out5);

/* Text of the last failure on the calling thread; valid until the next call
 * on this thread.  Never NULL. */
const char* ifvs_last_error(void);

#ifdef __cplusplus
}  /* extern "C" */
#endif

#endif /* IFVS_H */
