// One training step of the filter-aware conditioning (Section 2, training
// paragraph): from the conditioned tables of a batch of training queries,
// the softmax cross-entropy of each query's candidate list (ground-truth
// positives first, then mined hard negatives; score = -distance / tau), the
// anchor regularizer lam * mean(Delta^2), and their gradients carried back
// through the tables and Delta = alpha . W into the memory bank and W, and
// to w_z.  Plain SGD.  C_PQ and the codes stay fixed.
//
// train_query_kernel (one workgroup per query):
//   1. the query's table into LDS; its candidates' distances, summed over
//      subspaces in order as the scan does;
//   2. softmax statistics in fp64; g_v = d(batch loss)/d(distance of v);
//   3. the table gradient g_lut[m][c] = sum over candidates v whose code in
//      subspace m is c of g_v, the candidates added in order by one
//      wavefront (lane = subspace), in the table's LDS;
//   4. one thread per codeword c: for every subspace and sub-dimension j,
//      Delta, e = q - C_PQ - Delta, the Delta gradient
//        gd = g_lut * (-2 w e) + (2 lam / (M K d) / nq) Delta
//      (stored for the W update), and the reductions over c of gd * W
//      (alpha gradient) and g_lut * e^2 (w_f gradient): a wavefront
//      reduction each, the four wavefronts' partials added in wave order.
// train_update_w: W -= lr * sum_q gd_q (x) alpha_q, one thread per entry, the
// queries summed in order.
// train_update_bank: bank[row] -= lr * (sum of g_alpha over the (query, hash
// function) pairs that hit the row, in pair order; a row hit twice gets
// both), applied by the row's first pair.
// Every sum has a fixed order, so a step's results do not depend on
// scheduling: two identical steps give identical bits.
#include <cmath>

#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr int kTrainThreads = 256;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_max_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}

// Original id of a candidate slot, -1 when absent or out of range.
__device__ __forceinline__ int64_t cand_id(const TrainArgs& a, int qi, int v) {
  const int64_t id = a.cand[static_cast<int64_t>(qi) * a.n_cand + v];
  return (id >= 0 && id < a.n) ? id : -1;
}

// Code of physical row `row` in subspace mm.
__device__ __forceinline__ int code_of(const TrainArgs& a, int64_t row, int mm) {
  const uint32_t w = a.codes_t[((row >> 6) * a.mw + (mm >> 2)) * 64 + (row & 63)];
  return static_cast<int>((w >> (8 * (mm & 3))) & 0xFFu);
}

__global__ __launch_bounds__(kTrainThreads) void train_query_kernel(const TrainArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int qi = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = a.m, d = a.dsub, r = a.r, mr = a.m * a.r;
  float* s_tab = reinterpret_cast<float*>(smem);                 // [M][256]: table, then its gradient
  float* s_v = s_tab + M * kKsub;                                 // [n_cand]: distances, then g_v
  float* s_gw = s_v + a.n_cand;                                   // [4][dim]: w_f gradient, per wavefront
  float* s_ga = s_gw + 4 * a.dim;                                 // [4][M*r]: alpha gradient, per wavefront
  double* s_red = reinterpret_cast<double*>(s_ga + 4 * mr + ((4 * mr + 4 * a.dim + a.n_cand) & 1));   // [3][4]

  const float* lut = a.lut + static_cast<int64_t>(qi) * M * kKsub;
  for (int e = tid; e < M * kKsub; e += kTrainThreads) s_tab[e] = lut[e];
  __syncthreads();

  // 1. Distances.
  for (int v = tid; v < a.n_cand; v += kTrainThreads) {
    const int64_t id = cand_id(a, qi, v);
    float dist = 0.0f;
    if (id >= 0) {
      const int64_t row = a.inv_perm ? a.inv_perm[id] : id;
      for (int mm = 0; mm < M; ++mm) dist = __fadd_rn(dist, s_tab[mm * kKsub + code_of(a, row, mm)]);
    }
    s_v[v] = dist;
  }
  __syncthreads();

  // 2. Softmax statistics over the present candidates (fp64).
  const double inv_tau = 1.0 / static_cast<double>(a.tau);
  double mx = -INFINITY, pos_sum = 0.0, n_p = 0.0;
  for (int v = tid; v < a.n_cand; v += kTrainThreads) {
    if (cand_id(a, qi, v) < 0) continue;
    mx = fmax(mx, -static_cast<double>(s_v[v]) * inv_tau);
    if (v < a.n_pos) {
      pos_sum += static_cast<double>(s_v[v]);
      n_p += 1.0;
    }
  }
  mx = wave_max_d(mx);
  pos_sum = wave_sum_d(pos_sum);
  n_p = wave_sum_d(n_p);
  if (lane == 0) {
    s_red[wave] = mx;
    s_red[4 + wave] = pos_sum;
    s_red[8 + wave] = n_p;
  }
  __syncthreads();
  mx = fmax(fmax(s_red[0], s_red[1]), fmax(s_red[2], s_red[3]));
  pos_sum = s_red[4] + s_red[5] + s_red[6] + s_red[7];
  n_p = s_red[8] + s_red[9] + s_red[10] + s_red[11];
  __syncthreads();
  double z = 0.0;
  for (int v = tid; v < a.n_cand; v += kTrainThreads)
    if (cand_id(a, qi, v) >= 0) z += exp(-static_cast<double>(s_v[v]) * inv_tau - mx);
  z = wave_sum_d(z);
  if (lane == 0) s_red[wave] = z;
  __syncthreads();
  z = s_red[0] + s_red[1] + s_red[2] + s_red[3];
  const double lse = mx + log(z);
  const double ce = n_p > 0.0 ? lse + pos_sum * inv_tau / n_p : 0.0;
  // g_v = -(softmax_v - [v positive] / P) / tau / nq (0 without positives).
  for (int v = tid; v < a.n_cand; v += kTrainThreads) {
    float g = 0.0f;
    if (n_p > 0.0 && cand_id(a, qi, v) >= 0) {
      const double p = exp(-static_cast<double>(s_v[v]) * inv_tau - lse);
      const double share = v < a.n_pos ? 1.0 / n_p : 0.0;
      g = static_cast<float>(-(p - share) * inv_tau / a.nq);
    }
    s_v[v] = g;
  }
  __syncthreads();

  // 3. Table gradient: wavefront 0 adds the candidates in order, lane mm
  // updating subspace mm (one candidate touches one entry per subspace, and
  // a lane's updates to an entry are in program order).
  for (int e = tid; e < M * kKsub; e += kTrainThreads) s_tab[e] = 0.0f;
  __syncthreads();
  if (wave == 0) {
    for (int v = 0; v < a.n_cand; ++v) {
      const float g = s_v[v];
      const int64_t id = cand_id(a, qi, v);
      if (g == 0.0f || id < 0) continue;
      const int64_t row = a.inv_perm ? a.inv_perm[id] : id;
      for (int mm = lane; mm < M; mm += 64) {
        const int at = mm * kKsub + code_of(a, row, mm);
        s_tab[at] = __fadd_rn(s_tab[at], g);
      }
    }
  }
  __syncthreads();

  // 4. Delta gradient (thread = codeword), alpha and w_f gradients.
  const int c = tid;
  const float anchor = static_cast<float>(2.0 * a.lam / (static_cast<double>(M) * kKsub * d) / a.nq);
  const float* qrow = a.q + static_cast<int64_t>(qi) * a.dim;
  const float* wrow = a.wf + static_cast<int64_t>(qi) * a.dim;
  const float* arow = a.alpha + static_cast<int64_t>(qi) * mr;
  float* gdq = a.gdelta + static_cast<int64_t>(qi) * M * kKsub * d;
  double reg = 0.0;
  for (int mm = 0; mm < M; ++mm) {
    const float gl = s_tab[mm * kKsub + c];
    for (int j = 0; j < d; ++j) {
      float delta = 0.0f;
      for (int t = 0; t < r; ++t)
        delta = __fadd_rn(delta, __fmul_rn(arow[mm * r + t], a.W[((static_cast<int64_t>(mm) * r + t) * kKsub + c) * d + j]));
      const float cq = __fadd_rn(a.cpq[(static_cast<int64_t>(mm) * kKsub + c) * d + j], delta);
      const float e = __fsub_rn(qrow[mm * d + j], cq);
      const float gd = __fadd_rn(__fmul_rn(gl, __fmul_rn(-2.0f * wrow[mm * d + j], e)), __fmul_rn(anchor, delta));
      gdq[(static_cast<int64_t>(mm) * kKsub + c) * d + j] = gd;
      reg += static_cast<double>(delta) * delta;
      const float gw = wave_sum(__fmul_rn(gl, __fmul_rn(e, e)));
      if (lane == 0) s_gw[wave * a.dim + mm * d + j] = gw;
    }
    for (int t = 0; t < r; ++t) {
      float ga = 0.0f;
      for (int j = 0; j < d; ++j)
        ga = __fadd_rn(ga, __fmul_rn(gdq[(static_cast<int64_t>(mm) * kKsub + c) * d + j],
                                     a.W[((static_cast<int64_t>(mm) * r + t) * kKsub + c) * d + j]));
      ga = wave_sum(ga);
      if (lane == 0) s_ga[wave * mr + mm * r + t] = ga;
    }
  }
  reg = wave_sum_d(reg);
  if (lane == 0) s_red[wave] = reg;
  __syncthreads();
  if (tid == 0) {
    const double rsum = s_red[0] + s_red[1] + s_red[2] + s_red[3];
    a.loss[qi] = static_cast<float>(ce + a.lam * rsum / (static_cast<double>(M) * kKsub * d));
  }
  float* garow = a.galpha + static_cast<int64_t>(qi) * mr;
  for (int e = tid; e < mr; e += kTrainThreads)
    garow[e] = __fadd_rn(__fadd_rn(__fadd_rn(s_ga[e], s_ga[mr + e]), s_ga[2 * mr + e]), s_ga[3 * mr + e]);
  if (a.dwz) {
    const float* zrow = a.w_z + static_cast<int64_t>(qi) * a.dim;
    float* drow = a.dwz + static_cast<int64_t>(qi) * a.dim;
    for (int e = tid; e < a.dim; e += kTrainThreads) {
      const double x = static_cast<double>(zrow[e]);
      const float gw = __fadd_rn(__fadd_rn(__fadd_rn(s_gw[e], s_gw[a.dim + e]), s_gw[2 * a.dim + e]),
                                 s_gw[3 * a.dim + e]);
      drow[e] = static_cast<float>(static_cast<double>(gw) / (1.0 + exp(-x)));
    }
  }
}

__global__ __launch_bounds__(256) void train_update_w_kernel(float* __restrict__ W, const float* __restrict__ gdelta,
                                                             const float* __restrict__ alpha, int nq, int m, int r,
                                                             int dsub, float lr) {
  const int64_t per_t = static_cast<int64_t>(kKsub) * dsub;
  const int64_t total = static_cast<int64_t>(m) * r * per_t;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const int64_t cj = e % per_t;                // (c, j) inside a (m, t) slab
  const int64_t mt = e / per_t;
  const int mm = static_cast<int>(mt / r), t = static_cast<int>(mt % r);
  float g = 0.0f;
  for (int q = 0; q < nq; ++q)
    g = __fadd_rn(g, __fmul_rn(gdelta[(static_cast<int64_t>(q) * m + mm) * per_t + cj], alpha[static_cast<int64_t>(q) * m * r + mm * r + t]));
  W[e] = __fsub_rn(W[e], __fmul_rn(lr, g));
}

// One workgroup per (query, hash function) pair p; the first pair that hits
// a row sums the alpha gradients of all pairs hitting it, in pair order, and
// applies them (the other pairs of the row return).
__global__ __launch_bounds__(256) void train_update_bank_kernel(float* __restrict__ bank, int mr,
                                                                const int32_t* __restrict__ rows, int h,
                                                                const float* __restrict__ galpha, int pairs,
                                                                float lr) {
  const int p = blockIdx.x;
  const int32_t row = rows[p];
  for (int p2 = 0; p2 < p; ++p2)
    if (rows[p2] == row) return;
  for (int e = threadIdx.x; e < mr; e += blockDim.x) {
    float g = 0.0f;
    for (int p2 = p; p2 < pairs; ++p2)
      if (rows[p2] == row) g = __fadd_rn(g, galpha[static_cast<int64_t>(p2 / h) * mr + e]);
    const int64_t at = static_cast<int64_t>(row) * mr + e;
    bank[at] = __fsub_rn(bank[at], __fmul_rn(lr, g));
  }
}

__global__ void invert_perm_kernel(const int32_t* __restrict__ perm, int64_t n, int32_t* __restrict__ inv) {
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r < n) inv[perm[r]] = static_cast<int32_t>(r);
}

}  // namespace

size_t train_query_lds_bytes(int m, int dim, int n_cand, int mr) {
  const size_t floats = static_cast<size_t>(m) * kKsub + n_cand + 4 * static_cast<size_t>(dim) + 4 * mr;
  return (floats + 1) / 2 * 8 + 12 * sizeof(double);
}

hipError_t launch_train_query(const TrainArgs& a, hipStream_t s) {
  const size_t lds = train_query_lds_bytes(a.m, a.dim, a.n_cand, a.m * a.r);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&train_query_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  train_query_kernel<<<dim3(a.nq), dim3(kTrainThreads), lds, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_train_update_w(float* W, const float* gdelta, const float* alpha, int nq, int m, int r,
                                 int dsub, float lr, hipStream_t s) {
  const int64_t total = static_cast<int64_t>(m) * r * kKsub * dsub;
  train_update_w_kernel<<<dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, s>>>(W, gdelta, alpha, nq,
                                                                                           m, r, dsub, lr);
  return hipGetLastError();
}

hipError_t launch_train_update_bank(float* bank, int mr, const int32_t* rows, int h, const float* galpha,
                                    int nq, float lr, hipStream_t s) {
  if (nq * h <= 0) return hipSuccess;
  train_update_bank_kernel<<<dim3(nq * h), dim3(256), 0, s>>>(bank, mr, rows, h, galpha, nq * h, lr);
  return hipGetLastError();
}

hipError_t launch_invert_perm(const int32_t* perm, int64_t n, int32_t* inv, hipStream_t s) {
  invert_perm_kernel<<<dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s>>>(perm, n, inv);
  return hipGetLastError();
}

}  // namespace ifvs
