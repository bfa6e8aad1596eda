// Predicate encoder (Section 2, opening paragraph): the relational predicate
// f becomes the filter-aware weight vector w_z in R^D through a light-weight
// Transformer; w_f = softplus(w_z) then weighs the distance (first display).
//
// The architecture is this library's reading (the paper gives none): a
// summary token and one token per clause (column embedding plus the two
// normalized bounds through a 2 x H projection, no positional encoding),
// `layers` pre-norm encoder layers (multi-head self-attention over all the
// predicate's tokens, ReLU feed-forward), and a final layer norm of the
// summary token mapped by an H x D matrix to w_z.
//
// One workgroup encodes kEncQ predicates: their tokens are the rows of a
// 32 x H matrix in LDS (8 slots per predicate: summary + at most 4 clauses,
// the rest padding that attention never reads).  Every projection (Q/K/V,
// output, both feed-forward matrices) is a dense 32 x K x N contraction done
// with fp32 matrix-core instructions (v_mfma_f32_16x16x4_f32), the weights
// read from global memory (they stay in L2 across the workgroups); layer
// norms, the per-head softmax and the final H x D map run on the vector ALU.
#include <cmath>

#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr int kEncQ = 4;                       // predicates per workgroup
constexpr int kEncSlots = 8;                   // token slots per predicate
constexpr int kEncRows = kEncQ * kEncSlots;    // token rows per workgroup (two 16-row MFMA blocks)
constexpr int kEncThreads = 256;
constexpr int kEncWaves = kEncThreads / 64;
constexpr int kPad = 4;                        // LDS row padding (floats): spreads a 16 x 4 operand over the banks

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct EncArgs {
  const float* p;          // packed parameters (layout in ifvs.h)
  const double* off;       // [n_attr] bound offsets
  const double* scale;     // [n_attr] bound scales
  int H, heads, layers, F, D, n_attr;
  const DevPred* preds;    // [nq] (pinned staging slot)
  int nq;
  float* wz;               // [nq][D]
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Y = (accumulate ? Y : 0) + A W + bias (then ReLU if relu), for the 32 token
// rows: A [32][K] in LDS (row stride lda), W [K][N] row-major in global
// memory, bias [N]; K a multiple of 4, N of 16.  Wave w computes the 16-column
// blocks w, w + 4, ...; for each, both 16-row blocks share the B operand.
// Operand layout of v_mfma_f32_16x16x4_f32: lane l holds A[l % 16][l / 16]
// and B[l / 16][l % 16]; result register i of lane l is D[4 (l / 16) + i][l % 16].
__device__ void gemm_rows(const float* A, int lda, int K, const float* __restrict__ W,
                          const float* __restrict__ bias, int N, float* Y, int ldy, bool accumulate, bool relu) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  for (int cb = wave; cb < N / 16; cb += kEncWaves) {
    const int col = cb * 16 + r16;
    floatx4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f};
    floatx4 acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int k0 = 0; k0 < K; k0 += 16) {
      float b[4], a0[4], a1[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = k0 + 4 * u + kq;
        const bool in = k < K;
        b[u] = in ? W[static_cast<size_t>(k) * N + col] : 0.0f;
        a0[u] = in ? A[r16 * lda + k] : 0.0f;
        a1[u] = in ? A[(16 + r16) * lda + k] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[u], b[u], acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[u], b[u], acc1, 0, 0, 0);
      }
    }
    const float bc = bias[col];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r0 = 4 * kq + i, r1 = 16 + 4 * kq + i;
      float y0 = acc0[i] + bc, y1 = acc1[i] + bc;
      if (relu) {
        y0 = fmaxf(y0, 0.0f);
        y1 = fmaxf(y1, 0.0f);
      }
      if (accumulate) {
        y0 = Y[r0 * ldy + col] + y0;
        y1 = Y[r1 * ldy + col] + y1;
      }
      Y[r0 * ldy + col] = y0;
      Y[r1 * ldy + col] = y1;
    }
  }
}

// Z[r] = LN(X[r]) * g + b for `rows` rows (H <= 128: lane l holds elements
// l and l + 64), one wavefront per row.
__device__ void layer_norm_rows(const float* X, int ldx, float* Z, int ldz, const float* __restrict__ g,
                                const float* __restrict__ bt, int H, int rows) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const bool h0 = lane < H, h1 = lane + 64 < H;
  for (int r = wave; r < rows; r += kEncWaves) {
    const float v0 = h0 ? X[r * ldx + lane] : 0.0f;
    const float v1 = h1 ? X[r * ldx + lane + 64] : 0.0f;
    const float mean = wave_sum(v0 + v1) / static_cast<float>(H);
    const float d0 = h0 ? v0 - mean : 0.0f;
    const float d1 = h1 ? v1 - mean : 0.0f;
    const float var = wave_sum(d0 * d0 + d1 * d1) / static_cast<float>(H);
    const float rstd = 1.0f / sqrtf(var + 1e-5f);
    if (h0) Z[r * ldz + lane] = d0 * rstd * g[lane] + bt[lane];
    if (h1) Z[r * ldz + lane + 64] = d1 * rstd * g[lane + 64] + bt[lane + 64];
  }
}

__global__ __launch_bounds__(kEncThreads) void encoder_kernel(const EncArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int H = a.H, F = a.F;
  const int ldh = H + kPad, ldq = 3 * H + kPad, ldf = F + kPad;
  float* X = reinterpret_cast<float*>(smem);          // [32][ldh] token states
  float* Z = X + kEncRows * ldh;                      // [32][ldh] normalized tokens / attention output
  float* QKV = Z + kEncRows * ldh;                    // [32][ldq]
  float* Hd = QKV + kEncRows * ldq;                   // [32][ldf] feed-forward hidden
  DevPred* sp = reinterpret_cast<DevPred*>(Hd + kEncRows * ldf);   // [kEncQ]
  float* fa = reinterpret_cast<float*>(sp + kEncQ);   // [32] normalized lower bound of the row's clause
  float* fb = fa + kEncRows;                          // [32] normalized upper bound
  int* kind = reinterpret_cast<int*>(fb + kEncRows);  // [32] 0 padding, 1 summary, 2 clause
  int* col = kind + kEncRows;                         // [32] clause column
  int* seq = col + kEncRows;                          // [kEncQ] tokens of each predicate

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int q0 = blockIdx.x * kEncQ;
  if (wave < kEncQ && q0 + wave < a.nq) copy_pred(a.preds + q0 + wave, sp + wave, lane);
  __syncthreads();

  // Tokens: the summary token, then one per clause (bounds normalized in
  // fp64, clipped to [-1, 2], rounded to fp32).
  if (threadIdx.x < kEncRows) {
    const int r = threadIdx.x, qi = r / kEncSlots, i = r % kEncSlots;
    int kd = 0, c = 0;
    float xa = 0.0f, xb = 0.0f;
    if (q0 + qi < a.nq) {
      const DevPred& p = sp[qi];
      if (i == 0) {
        kd = 1;
      } else if (i <= p.n_raw) {
        kd = 2;
        c = p.raw_col[i - 1];
        const double off = a.off[c], sc = a.scale[c];
        const double lo = fmin(fmax((static_cast<double>(p.raw_lo[i - 1]) - off) * sc, -1.0), 2.0);
        const double hi = fmin(fmax((static_cast<double>(p.raw_hi[i - 1]) - off) * sc, -1.0), 2.0);
        xa = static_cast<float>(lo);
        xb = static_cast<float>(hi);
      }
    }
    kind[r] = kd;
    col[r] = c;
    fa[r] = xa;
    fb[r] = xb;
    if (i == 0) seq[qi] = q0 + qi < a.nq ? 1 + sp[qi].n_raw : 0;
  }
  __syncthreads();
  const float* P = a.p;
  const float* col_embed = P;
  const float* feat_w = col_embed + static_cast<size_t>(a.n_attr) * H;
  const float* feat_b = feat_w + 2 * H;
  const float* cls = feat_b + H;
  for (int e = threadIdx.x; e < kEncRows * H; e += kEncThreads) {
    const int r = e / H, h = e % H;
    float v = 0.0f;
    if (kind[r] == 1) {
      v = cls[h];
    } else if (kind[r] == 2) {
      v = col_embed[static_cast<size_t>(col[r]) * H + h] + fa[r] * feat_w[h];
      v = v + fb[r] * feat_w[H + h];
      v = v + feat_b[h];
    }
    X[r * ldh + h] = v;
  }
  __syncthreads();

  const float* L = cls + H;
  const int dh = H / a.heads;
  const float inv_sqrt_dh = 1.0f / sqrtf(static_cast<float>(dh));
  for (int layer = 0; layer < a.layers; ++layer) {
    const float* ln1_g = L;
    const float* ln1_b = ln1_g + H;
    const float* Wqkv = ln1_b + H;
    const float* bqkv = Wqkv + static_cast<size_t>(H) * 3 * H;
    const float* Wo = bqkv + 3 * H;
    const float* bo = Wo + static_cast<size_t>(H) * H;
    const float* ln2_g = bo + H;
    const float* ln2_b = ln2_g + H;
    const float* W1 = ln2_b + H;
    const float* b1 = W1 + static_cast<size_t>(H) * F;
    const float* W2 = b1 + F;
    const float* b2 = W2 + static_cast<size_t>(F) * H;
    L = b2 + H;

    layer_norm_rows(X, ldh, Z, ldh, ln1_g, ln1_b, H, kEncRows);
    __syncthreads();
    gemm_rows(Z, ldh, H, Wqkv, bqkv, 3 * H, QKV, ldq, false, false);
    __syncthreads();
    // Attention of token i of predicate qi in head hd over the predicate's
    // tokens; the output (head slices side by side) goes to Z.  Padding rows
    // get zeros.
    for (int t = threadIdx.x; t < kEncQ * a.heads * kEncSlots; t += kEncThreads) {
      const int qi = t / (a.heads * kEncSlots);
      const int hd = (t / kEncSlots) % a.heads;
      const int i = t % kEncSlots;
      const int S = seq[qi];
      const int ri = qi * kEncSlots + i;
      float* o = Z + ri * ldh + hd * dh;
      if (i >= S) {
        for (int d = 0; d < dh; ++d) o[d] = 0.0f;
        continue;
      }
      const float* qv = QKV + ri * ldq + hd * dh;
      float s[kEncSlots];
      float mx = -INFINITY;
      for (int j = 0; j < S; ++j) {
        const float* kv = QKV + (qi * kEncSlots + j) * ldq + H + hd * dh;
        float acc = 0.0f;
        for (int d = 0; d < dh; ++d) acc += qv[d] * kv[d];
        s[j] = acc * inv_sqrt_dh;
        mx = fmaxf(mx, s[j]);
      }
      float sum = 0.0f;
      for (int j = 0; j < S; ++j) {
        s[j] = expf(s[j] - mx);
        sum += s[j];
      }
      const float inv = 1.0f / sum;
      for (int d = 0; d < dh; ++d) {
        float acc = 0.0f;
        for (int j = 0; j < S; ++j) acc += s[j] * QKV[(qi * kEncSlots + j) * ldq + 2 * H + hd * dh + d];
        o[d] = acc * inv;
      }
    }
    __syncthreads();
    gemm_rows(Z, ldh, H, Wo, bo, H, X, ldh, true, false);
    __syncthreads();
    layer_norm_rows(X, ldh, Z, ldh, ln2_g, ln2_b, H, kEncRows);
    __syncthreads();
    gemm_rows(Z, ldh, H, W1, b1, F, Hd, ldf, false, true);
    __syncthreads();
    gemm_rows(Hd, ldf, F, W2, b2, H, X, ldh, true, false);
    __syncthreads();
  }

  // w_z = LN_f(summary token) W_out + b_out, the kEncQ predicates side by
  // side so every W_out row is read once per workgroup.
  const float* lnf_g = L;
  const float* lnf_b = lnf_g + H;
  const float* out_w = lnf_b + H;
  const float* out_b = out_w + static_cast<size_t>(H) * a.D;
  // (row r of the normalization is predicate r's summary token: input row
  // stride kEncSlots rows)
  layer_norm_rows(X, kEncSlots * ldh, Z, ldh, lnf_g, lnf_b, H, kEncQ);
  __syncthreads();
  const int nv = min(kEncQ, a.nq - q0);
  for (int d = threadIdx.x; d < a.D; d += kEncThreads) {
    float acc[kEncQ] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int h = 0; h < H; ++h) {
      const float w = out_w[static_cast<size_t>(h) * a.D + d];
#pragma unroll
      for (int qi = 0; qi < kEncQ; ++qi) acc[qi] += Z[qi * ldh + h] * w;
    }
    for (int qi = 0; qi < nv; ++qi) a.wz[static_cast<size_t>(q0 + qi) * a.D + d] = acc[qi] + out_b[d];
  }
}

}  // namespace

size_t encoder_lds_bytes(int H, int F) {
  const size_t floats = static_cast<size_t>(kEncRows) * (2 * (H + kPad) + (3 * H + kPad) + (F + kPad));
  return floats * sizeof(float) + kEncQ * sizeof(DevPred) + kEncRows * 2 * sizeof(float) +
         (2 * kEncRows + kEncQ) * sizeof(int);
}

hipError_t launch_encoder(const float* params, const double* off, const double* scale, int H, int heads, int layers,
                          int F, int D, int n_attr, const DevPred* preds, int nq, float* wz, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  EncArgs a{};
  a.p = params;
  a.off = off;
  a.scale = scale;
  a.H = H;
  a.heads = heads;
  a.layers = layers;
  a.F = F;
  a.D = D;
  a.n_attr = n_attr;
  a.preds = preds;
  a.nq = nq;
  a.wz = wz;
  const size_t lds = encoder_lds_bytes(H, F);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&encoder_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(encoder_kernel, dim3((nq + kEncQ - 1) / kEncQ), dim3(kEncThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace ifvs
