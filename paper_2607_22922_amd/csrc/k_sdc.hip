// Symmetric distance computation, the pre-filtering baselines (iv) and (v)
// of Section 3.2: the query is quantized with the data's codebook too, and a
// candidate's distance is the sum over subspaces of codeword-to-codeword
// squared distances.  The codeword table T[m][a][b] is built once, at load;
// a query's table is the row of its own code, T[m][enc(q)_m][.], laid out
// like an asymmetric distance table, so the scan, its early abandonment and
// the top-k serve SDC unchanged.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

// T[m][a][b] = sum_{j<dsub} (C[m][a][j] - C[m][b][j])^2, fp32 in j order
// from +0.  Block (m, a), thread b.
__global__ __launch_bounds__(256) void sdc_table_kernel(const float* __restrict__ cpq, int dsub,
                                                        float* __restrict__ T) {
  const int m = blockIdx.y, a = blockIdx.x, b = threadIdx.x;
  const float* ca = cpq + (static_cast<size_t>(m) * kKsub + a) * dsub;
  const float* cb = cpq + (static_cast<size_t>(m) * kKsub + b) * dsub;
  float acc = 0.0f;
  for (int j = 0; j < dsub; ++j) {
    const float e = __fsub_rn(ca[j], cb[j]);
    acc = __fadd_rn(acc, __fmul_rn(e, e));
  }
  T[(static_cast<size_t>(m) * kKsub + a) * kKsub + b] = acc;
}

__device__ __forceinline__ void put(float* out, size_t i, float v) { out[i] = v; }
__device__ __forceinline__ void put(__half* out, size_t i, float v) { out[i] = __float2half_rn(v); }

// One workgroup (256 threads) per query.  For each subspace, thread c takes
// the squared distance of the query's sub-vector to codeword c (fp32, j
// order), the workgroup finds the smallest (distance, c) -- the query's
// code, lowest index among equals -- and thread c writes T[m][code][c].
template <typename OutT>
__global__ __launch_bounds__(256) void sdc_lut_kernel(const float* __restrict__ q, int dim, int M, int dsub,
                                                      const float* __restrict__ cpq, const float* __restrict__ T,
                                                      OutT* __restrict__ out) {
  __shared__ uint64_t s_min[4];
  const int qi = blockIdx.x, c = threadIdx.x;
  const int lane = c & 63, wave = c >> 6;
  const float* qv = q + static_cast<size_t>(qi) * dim;
  for (int m = 0; m < M; ++m) {
    const float* cw = cpq + (static_cast<size_t>(m) * kKsub + c) * dsub;
    float acc = 0.0f;
    for (int j = 0; j < dsub; ++j) {
      const float e = __fsub_rn(qv[m * dsub + j], cw[j]);
      acc = __fadd_rn(acc, __fmul_rn(e, e));
    }
    uint64_t key = (static_cast<uint64_t>(ordered_bits(acc)) << 32) | static_cast<uint32_t>(c);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint64_t other = shfl_xor_u64(key, o);
      key = other < key ? other : key;
    }
    if (lane == 0) s_min[wave] = key;
    __syncthreads();
    uint64_t best = s_min[0];
#pragma unroll
    for (int w = 1; w < 4; ++w) best = s_min[w] < best ? s_min[w] : best;
    __syncthreads();   // s_min is rewritten for the next subspace
    const int code = static_cast<int>(static_cast<uint32_t>(best));
    put(out, (static_cast<size_t>(qi) * M + m) * kKsub + c, T[(static_cast<size_t>(m) * kKsub + code) * kKsub + c]);
  }
}

}  // namespace

hipError_t launch_sdc_table(const float* cpq, int m, int dsub, float* T, hipStream_t s) {
  sdc_table_kernel<<<dim3(kKsub, m), kKsub, 0, s>>>(cpq, dsub, T);
  return hipGetLastError();
}

hipError_t launch_sdc_lut(const float* q, int dim, int m, int dsub, const float* cpq, const float* T, int nq,
                          int lut_dtype, void* lut_out, hipStream_t s) {
  if (lut_dtype == 1)
    sdc_lut_kernel<__half><<<nq, kKsub, 0, s>>>(q, dim, m, dsub, cpq, T, static_cast<__half*>(lut_out));
  else
    sdc_lut_kernel<float><<<nq, kKsub, 0, s>>>(q, dim, m, dsub, cpq, T, static_cast<float*>(lut_out));
  return hipGetLastError();
}

}  // namespace ifvs
