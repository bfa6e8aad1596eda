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
constexpr int kScanWaves = 4;              // wavefronts per scan workgroup
constexpr int kFilterQueries = 16;         // predicates evaluated per attribute read

// A predicate as the device sees it.  The raw fields are the caller's clauses
// exactly as given (they are hashed into the memory bank); the effective
// fields are the same conjunction normalized for evaluation on int32
// attributes: each kept clause tests (uint32)(attr - lo) < width, clauses that
// admit every int32 value are dropped, and n_eff = -1 marks a predicate that
// no value satisfies.
struct DevPred {
  int32_t n_raw;
  int32_t n_eff;
  int32_t raw_col[kMaxClauses];
  int64_t raw_lo[kMaxClauses];
  int64_t raw_hi[kMaxClauses];
  int32_t col[kMaxClauses];
  int32_t lo[kMaxClauses];
  uint32_t width[kMaxClauses];
};

// Kernel launchers (each defined next to its kernel).  All return the HIP
// error of the launch.
hipError_t launch_relayout_codes(const uint8_t* codes, int64_t n, int m, int mw,
                                 uint32_t* codes_t, int64_t n_tiles, hipStream_t s);

hipError_t launch_filter(const int32_t* attrs, int64_t n, int n_attr, const DevPred* preds,
                         int nq, uint64_t* bitmap, int64_t stride64,
                         unsigned long long* counts, hipStream_t s);

hipError_t launch_condition(const float* q, int dim, const DevPred* preds, int nq,
                            const float* bank, int bank_rows, int mr, int h, uint64_t seed,
                            const float* w_z, float* alpha_out, float* wf_out, hipStream_t s);

hipError_t launch_build_lut(const float* q, int dim, int m, int dsub, int r,
                            const float* cpq, const float* W, const float* alpha,
                            const float* wf, int nq, int lut_dtype, void* lut_out,
                            hipStream_t s);

struct ScanPlan {
  int qtile;        // queries sharing one LDS residency and one pass over the codes
  int splits;       // code chunks per query tile (grid.x)
  int64_t tiles_per_block;
  int pool_stride;  // candidate pool keys per (wave, query): 64*kpl >= k + 64
  int kpl;          // pool keys per lane when it is sorted
  size_t lds_bytes;
};

// Largest query tile whose tables and pools fit the LDS budget (0 if none).
int scan_max_qtile(int m, int lut_bytes, int k);
// Round a requested tile down to one this build instantiates.
int scan_supported_qtile(int want);
int pool_kpl(int k);

hipError_t launch_scan_dense(const uint32_t* codes_t, int64_t n_tiles, int m, int mw,
                             const void* lut, int lut_dtype, int nq,
                             const uint64_t* bitmap, int64_t stride64, int k,
                             const ScanPlan& plan, uint64_t* partials, hipStream_t s);

hipError_t launch_topk_merge(const uint64_t* partials, int nq, int64_t per_query, int k,
                             int32_t* ids_out, float* dist_out, hipStream_t s);

}  // namespace ifvs
