// Distance-table build (Section 2, first display and Rank stage): for each
// query and subspace m, the conditioned codeword
//     C[c][j] = C_PQ[m][c][j] + sum_{t<r} alpha[m*r+t] * W[m][t][c][j]
// and the table entry
//     LUT[m][c] = sum_{j<d} w_f[m*d+j] * (q[m*d+j] - C[c][j])^2 .
// Every product and sum is a separately rounded fp32 operation (explicit
// round-to-nearest intrinsics, so no fused multiply-add), t and j summed in
// index order from +0: the table is bit-identical to the plain definition.
//
// Layout: one workgroup per (subspace, chunk of queries), one thread per
// centroid c.  A thread keeps its codeword C_PQ[m][c] and its r x d slice of
// W in registers for the whole query chunk, so W and C_PQ are read once per
// chunk.  The chunk's q, w_f and alpha values (the same for every thread)
// are loaded once, all in flight together, into LDS and read back as
// broadcasts.  The 256 entries of one (query, m) row are one coalesced 1 KB
// (fp32) or 512 B (binary16) store.  The contraction over r is
// 8 deep and d is 2..8, far too shallow for matrix cores; the kernel is
// store-bound in the identity mode and a few microseconds per batch otherwise.
//
// With a parts array the fixed-shape kernel also writes the coarse bound's
// per-subspace factors of each query, from the conditioned codewords it has
// just formed (the same operations as the separate bound kernel, so the same
// bits): parts[q][0][m] = max_c ||C[c] - C_PQ[m][c]||^2 and parts[q][1][m] =
// max_j w_f[m*d+j] (NaN for a negative or non-finite weight; 1 without
// weights).
#include <cfloat>

#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr int kQueriesPerBlock = 16;

__device__ __forceinline__ float nan_max(float a, float b) {
  return (a != a || b != b) ? __builtin_nanf("") : fmaxf(a, b);
}

__device__ __forceinline__ void store_entry(float* out, int64_t i, float v) { out[i] = v; }
__device__ __forceinline__ void store_entry(__half* out, int64_t i, float v) {
  out[i] = __float2half_rn(v);
}

// d and r known at compile time (R == 0: no alpha, C_iFVS = C_PQ); kParts:
// the bound factors too.
template <int DSUB, int R, typename OutT, bool kParts = false>
__global__ __launch_bounds__(256) void lut_fixed_kernel(
    const float* __restrict__ q, int dim, int M, const float* __restrict__ cpq,
    const float* __restrict__ W, const float* __restrict__ alpha, const float* __restrict__ wf,
    int nq, OutT* __restrict__ out, float* __restrict__ parts, StageDone done) {
  const int m = blockIdx.x;
  const int c = threadIdx.x;
  signal_stage_done(done);
  float creg[DSUB];
#pragma unroll
  for (int j = 0; j < DSUB; ++j) creg[j] = cpq[(static_cast<int64_t>(m) * kKsub + c) * DSUB + j];
  float wreg[R > 0 ? R : 1][DSUB];
  if constexpr (R > 0) {
#pragma unroll
    for (int t = 0; t < R; ++t)
#pragma unroll
      for (int j = 0; j < DSUB; ++j)
        wreg[t][j] = W[((static_cast<int64_t>(m) * R + t) * kKsub + c) * DSUB + j];
  }
  // Per-query operands of the chunk: q and w_f (DSUB each) and alpha (R).
  constexpr int kPer = 2 * DSUB + R;
  __shared__ float s_op[kQueriesPerBlock][kPer];
  const int q_begin = blockIdx.y * kQueriesPerBlock;
  const int q_end = min(nq, q_begin + kQueriesPerBlock);
#pragma unroll
  for (int idx = c; idx < kQueriesPerBlock * kPer; idx += 256) {
    const int k = idx / kPer, o = idx % kPer;
    const int qi = q_begin + k;
    if (qi < q_end) {
      float v;
      if (o < DSUB) v = q[static_cast<int64_t>(qi) * dim + m * DSUB + o];
      else if (o < 2 * DSUB) v = wf ? wf[static_cast<int64_t>(qi) * dim + m * DSUB + (o - DSUB)] : 1.0f;
      else v = alpha[(static_cast<int64_t>(qi) * M + m) * R + (o - 2 * DSUB)];
      s_op[k][o] = v;
    }
  }
  __syncthreads();
  __shared__ float s_red[kParts ? kQueriesPerBlock : 1][4];
  for (int qi = q_begin; qi < q_end; ++qi) {
    const float* op = s_op[qi - q_begin];
    float acc = 0.0f, n2 = 0.0f;
#pragma unroll
    for (int j = 0; j < DSUB; ++j) {
      float C = creg[j];
      if constexpr (R > 0) {
        float delta = 0.0f;
#pragma unroll
        for (int t = 0; t < R; ++t) delta = __fadd_rn(delta, __fmul_rn(op[2 * DSUB + t], wreg[t][j]));
        C = __fadd_rn(C, delta);
        if constexpr (kParts) {
          const float sh = __fsub_rn(C, creg[j]);
          n2 = __fadd_rn(n2, __fmul_rn(sh, sh));
        }
      }
      const float e = __fsub_rn(op[j], C);
      acc = __fadd_rn(acc, __fmul_rn(op[DSUB + j], __fmul_rn(e, e)));
    }
    store_entry(out, (static_cast<int64_t>(qi) * M + m) * kKsub + c, acc);
    if constexpr (kParts) {
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) n2 = nan_max(n2, __shfl_xor(n2, o, 64));
      if ((c & 63) == 0) s_red[qi - q_begin][c >> 6] = n2;
    }
  }
  if constexpr (kParts) {
    __syncthreads();
    const int qi = q_begin + c;
    if (c < kQueriesPerBlock && qi < q_end) {
      const float mx = nan_max(nan_max(s_red[c][0], s_red[c][1]), nan_max(s_red[c][2], s_red[c][3]));
      float wm = 1.0f;
      if (wf) {
        wm = 0.0f;
#pragma unroll
        for (int j = 0; j < DSUB; ++j) {
          const float v = s_op[c][DSUB + j];
          wm = (v >= 0.0f && v <= FLT_MAX && wm == wm) ? fmaxf(wm, v) : __builtin_nanf("");
        }
      }
      parts[(static_cast<size_t>(qi) * 2) * M + m] = mx;
      parts[(static_cast<size_t>(qi) * 2 + 1) * M + m] = wm;
    }
  }
}

// Any d and r: the same arithmetic with operands read from memory.
template <typename OutT>
__global__ __launch_bounds__(256) void lut_generic_kernel(
    const float* __restrict__ q, int dim, int M, int dsub, int r, const float* __restrict__ cpq,
    const float* __restrict__ W, const float* __restrict__ alpha, const float* __restrict__ wf,
    int nq, OutT* __restrict__ out, StageDone done) {
  const int m = blockIdx.x;
  const int c = threadIdx.x;
  signal_stage_done(done);
  const int q_begin = blockIdx.y * kQueriesPerBlock;
  const int q_end = min(nq, q_begin + kQueriesPerBlock);
  for (int qi = q_begin; qi < q_end; ++qi) {
    const float* qv = q + static_cast<int64_t>(qi) * dim + static_cast<int64_t>(m) * dsub;
    const float* wv = wf ? wf + static_cast<int64_t>(qi) * dim + static_cast<int64_t>(m) * dsub : nullptr;
    float acc = 0.0f;
    for (int j = 0; j < dsub; ++j) {
      float C = cpq[(static_cast<int64_t>(m) * kKsub + c) * dsub + j];
      if (alpha) {
        float delta = 0.0f;
        for (int t = 0; t < r; ++t)
          delta = __fadd_rn(delta, __fmul_rn(alpha[(static_cast<int64_t>(qi) * M + m) * r + t],
                                             W[((static_cast<int64_t>(m) * r + t) * kKsub + c) * dsub + j]));
        C = __fadd_rn(C, delta);
      }
      const float e = __fsub_rn(qv[j], C);
      const float w = wv ? wv[j] : 1.0f;
      acc = __fadd_rn(acc, __fmul_rn(w, __fmul_rn(e, e)));
    }
    store_entry(out, (static_cast<int64_t>(qi) * M + m) * kKsub + c, acc);
  }
}

template <int DSUB, int R, typename OutT>
void launch_fixed(dim3 g, hipStream_t s, const float* q, int dim, int M, const float* cpq, const float* W,
                  const float* alpha, const float* wf, int nq, OutT* out, float* parts, StageDone done) {
  if (parts)
    lut_fixed_kernel<DSUB, R, OutT, true><<<g, dim3(256), 0, s>>>(q, dim, M, cpq, W, alpha, wf, nq, out, parts, done);
  else
    lut_fixed_kernel<DSUB, R, OutT><<<g, dim3(256), 0, s>>>(q, dim, M, cpq, W, alpha, wf, nq, out, nullptr, done);
}

template <int DSUB, typename OutT>
bool launch_fixed_r(int r, bool has_alpha, dim3 g, hipStream_t s, const float* q, int dim, int M,
                    const float* cpq, const float* W, const float* alpha, const float* wf, int nq,
                    OutT* out, float* parts, StageDone done) {
  if (!has_alpha) {
    launch_fixed<DSUB, 0, OutT>(g, s, q, dim, M, cpq, W, nullptr, wf, nq, out, parts, done);
    return true;
  }
  if (r == 8) {
    launch_fixed<DSUB, 8, OutT>(g, s, q, dim, M, cpq, W, alpha, wf, nq, out, parts, done);
    return true;
  }
  return false;
}

template <typename OutT>
void launch_typed(const float* q, int dim, int M, int dsub, int r, const float* cpq,
                  const float* W, const float* alpha, const float* wf, int nq, OutT* out,
                  hipStream_t s, float* parts, StageDone done) {
  const dim3 g(M, (nq + kQueriesPerBlock - 1) / kQueriesPerBlock);
  const bool has_alpha = alpha != nullptr;
  bool launched = false;
  switch (dsub) {
    case 2: launched = launch_fixed_r<2>(r, has_alpha, g, s, q, dim, M, cpq, W, alpha, wf, nq, out, parts, done); break;
    case 4: launched = launch_fixed_r<4>(r, has_alpha, g, s, q, dim, M, cpq, W, alpha, wf, nq, out, parts, done); break;
    case 8: launched = launch_fixed_r<8>(r, has_alpha, g, s, q, dim, M, cpq, W, alpha, wf, nq, out, parts, done); break;
    default: break;
  }
  if (!launched)
    lut_generic_kernel<OutT><<<g, dim3(256), 0, s>>>(q, dim, M, dsub, r, cpq, W, alpha, wf, nq, out, done);
}

}  // namespace

bool lut_emits_bound_parts(int dsub, int r, bool has_alpha) {
  return (dsub == 2 || dsub == 4 || dsub == 8) && (!has_alpha || r == 8);
}

hipError_t launch_build_lut(const float* q, int dim, int m, int dsub, int r, const float* cpq,
                            const float* W, const float* alpha, const float* wf, int nq,
                            int lut_dtype, void* lut_out, hipStream_t s, float* parts, StageDone done) {
  if (parts && !lut_emits_bound_parts(dsub, r, alpha != nullptr)) return hipErrorInvalidValue;
  if (lut_dtype == 1)
    launch_typed(q, dim, m, dsub, r, cpq, W, alpha, wf, nq, static_cast<__half*>(lut_out), s, parts, done);
  else
    launch_typed(q, dim, m, dsub, r, cpq, W, alpha, wf, nq, static_cast<float*>(lut_out), s, parts, done);
  return hipGetLastError();
}

}  // namespace ifvs
