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
// 16 x H matrix in LDS (8 slots per predicate: summary + at most 4 clauses,
// the rest padding that attention never reads).  Every projection (Q/K/V,
// output, both feed-forward matrices) is a dense 16 x K x N contraction done
// with fp32 matrix-core instructions (v_mfma_f32_16x16x4_f32).  The weights
// (the same for every workgroup, so L2-resident) are staged into LDS in
// column chunks of up to 34 KB, every thread moving 16-byte words with eight
// loads in flight, so a projection waits for memory once or twice rather
// than once per 16-deep step; layer norms, the per-head softmax and the
// final H x D map run on the vector ALU.
//
// Optionally the launch also conditions the queries it encodes (the
// condition kernel's work, the same bits): w_f = softplus(w_z) as w_z is
// written, and alpha from side workgroups after the encoder's, a wavefront
// per query (fingerprint, bank-row hashes, sum).  The fingerprint is a
// sequential chain of several microseconds per query; on CUs of their own
// these workgroups run beside the encoder's instead of lengthening them.
// The same side workgroups can also find the batch's row intervals (the
// interval kernel's work, a wavefront per bound).
#include <cmath>

#include "condition_device.h"
#include "ifvs_internal.h"
#include "intervals_device.h"

namespace ifvs {

namespace {

constexpr int kEncQ = 2;                       // predicates per workgroup
constexpr int kEncSlots = 8;                   // token slots per predicate
constexpr int kEncRows = kEncQ * kEncSlots;    // token rows per workgroup (one 16-row MFMA block)
constexpr int kEncThreads = 256;
constexpr int kEncWaves = kEncThreads / 64;
constexpr int kPad = 4;                        // LDS row padding (floats): spreads a 16 x 4 operand over the banks
constexpr int kWbuf = 9216;                    // floats of the weight staging buffer: 8192 + padding (36 KB)

// Floats of every layer's gains and biases and the final layer norm's.
__host__ __device__ constexpr int vec_floats(int H, int F, int layers) { return layers * (9 * H + F) + 2 * H; }
constexpr int kEncCondMaxH = 4;                // hash functions the in-launch condition handles

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct EncArgs {
  const float* p;          // packed parameters (layout in ifvs.h)
  const double* off;       // [n_attr] bound offsets
  const double* scale;     // [n_attr] bound scales
  int H, heads, layers, F, D, n_attr;
  const DevPred* preds;    // [nq] (pinned staging slot)
  int nq;
  float* wz;               // [nq][D]
  EncCondition cond;       // the in-launch condition (cond.wf null: none)
  IntervalArgs iv;         // the in-launch intervals (iv.nq 0: none)
  int enc_blocks;          // workgroups of the encoder; the side workgroups follow
  int n_cond;              // side items: n_cond queries' alpha, then 2 iv.nq interval bounds
  int n_side_waves;        // wavefronts of the side workgroups
};

// alpha of query qi (one wavefront), as the condition kernel computes it.
__device__ void condition_alpha(const EncArgs& a, int qi, int lane) {
  const EncCondition& cd = a.cond;
  constexpr int kPredWords = static_cast<int>(sizeof(DevPred) / 4);
  const uint32_t pw = lane < kPredWords ? reinterpret_cast<const uint32_t*>(a.preds + qi)[lane] : 0u;
  uint32_t lo, hi;
  fingerprint_query(cd.q + static_cast<size_t>(qi) * a.D, a.D, lo, hi);
  const uint64_t key = fingerprint_key(lo, hi, pw);
  const uint32_t row = hashed_bank_row(key, cd.seed, lane, cd.h, cd.bank_rows);
  float* arow = cd.alpha + static_cast<size_t>(qi) * cd.mr;
  switch (cd.h) {
    case 1: gather_alpha<1>(cd.bank, row, cd.mr, lane, arow); break;
    case 2: gather_alpha<2>(cd.bank, row, cd.mr, lane, arow); break;
    case 3: gather_alpha<3>(cd.bank, row, cd.mr, lane, arow); break;
    case 4: gather_alpha<4>(cd.bank, row, cd.mr, lane, arow); break;
    default: break;
  }
}

// Weight chunks.  A matrix W [K][N] (row-major, rows 16-byte aligned) goes
// through the LDS buffer in chunks of chunk_cols(K, N) columns, at most 8192
// floats each, so one chunk is eight 16-byte words per thread.  The next
// chunk is loaded into registers (Prefetch) while the current one is
// multiplied, so a projection seldom waits for memory.
struct Chunk {
  const float* W;
  int K, N, n0, cols;
};

// Columns of the chunk starting at n0: the largest power of two (>= 16) that
// fits both 8192 / K and the columns left (N - n0, a multiple of 16), so a
// word's row and column follow from shifts.
__device__ __forceinline__ int chunk_cols(int K, int N, int n0) {
  const int lim = min(8192 / K, N - n0);
  int c = 16;
  while (2 * c <= lim) c *= 2;
  return c;
}

__device__ __forceinline__ Chunk first_chunk(const float* W, int K, int N) { return {W, K, N, 0, chunk_cols(K, N, 0)}; }

struct Prefetch {
  float4 v0, v1, v2, v3, v4, v5, v6, v7;   // eight named words: they stay in registers
};

__device__ __forceinline__ float4 chunk_word(const Chunk& c, int u) {
  const int sh = __builtin_ctz(c.cols / 4), words = c.K << sh;   // words per row: a power of two
  // past the end: load the last word again (in bounds; not stored)
  const int e = min(u * kEncThreads + static_cast<int>(threadIdx.x), words - 1);
  return *reinterpret_cast<const float4*>(c.W + static_cast<size_t>(e >> sh) * c.N + c.n0 +
                                          4 * (e & ((1 << sh) - 1)));
}

__device__ __forceinline__ void prefetch(const Chunk& c, Prefetch& pf) {
  if (!c.W) return;
  pf.v0 = chunk_word(c, 0);
  pf.v1 = chunk_word(c, 1);
  pf.v2 = chunk_word(c, 2);
  pf.v3 = chunk_word(c, 3);
  pf.v4 = chunk_word(c, 4);
  pf.v5 = chunk_word(c, 5);
  pf.v6 = chunk_word(c, 6);
  pf.v7 = chunk_word(c, 7);
}

// Words past the chunk's end go to the 16-byte sink after the buffer.
__device__ __forceinline__ void commit_word(const Chunk& c, float* Wb, int ldw, int u, const float4& v) {
  const int sh = __builtin_ctz(c.cols / 4), words = c.K << sh;
  const int e = u * kEncThreads + static_cast<int>(threadIdx.x);
  const int at = e < words ? (e >> sh) * ldw + 4 * (e & ((1 << sh) - 1)) : kWbuf;
  *reinterpret_cast<float4*>(Wb + at) = v;
}

__device__ __forceinline__ void commit(const Chunk& c, const Prefetch& pf, float* Wb, int ldw) {
  commit_word(c, Wb, ldw, 0, pf.v0);
  commit_word(c, Wb, ldw, 1, pf.v1);
  commit_word(c, Wb, ldw, 2, pf.v2);
  commit_word(c, Wb, ldw, 3, pf.v3);
  commit_word(c, Wb, ldw, 4, pf.v4);
  commit_word(c, Wb, ldw, 5, pf.v5);
  commit_word(c, Wb, ldw, 6, pf.v6);
  commit_word(c, Wb, ldw, 7, pf.v7);
}

// Y = (accumulate ? Y : 0) + A W + bias (then ReLU if relu), for the 16
// token rows: A [16][K] in LDS (row stride lda), W [K][N], bias [N] (LDS); K a
// multiple of 4, N of 16.  On entry pf holds W's first chunk; on return it
// holds the first chunk of `next` (the following projection's matrix).
// Wave w computes the 16-column blocks w, w + 4, ... of each chunk.
// Operand layout of v_mfma_f32_16x16x4_f32: lane l holds A[l % 16][l / 16]
// and B[l / 16][l % 16]; result register i of lane l is D[4 (l / 16) + i][l % 16].
__device__ __forceinline__ void gemm_rows(const float* A, int lda, const Chunk& w0, const float* bias, float* Y,
                          int ldy, bool accumulate, bool relu, float* Wb, Prefetch& pf, const Chunk& next) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  const int K = w0.K, N = w0.N;
  for (Chunk c = w0; c.n0 < N;) {
    const int ldw = c.cols + kPad;
    __syncthreads();                      // the buffer's readers are done, A is written
    commit(c, pf, Wb, ldw);
    __syncthreads();
    Chunk nx = c;
    nx.n0 = c.n0 + c.cols;
    nx.cols = nx.n0 < N ? chunk_cols(K, N, nx.n0) : 16;
    prefetch(nx.n0 < N ? nx : next, pf);
    // Two column blocks per wave at a time (two independent accumulator
    // chains); a wave with one block left multiplies it twice and keeps one.
    const int nb = c.cols / 16;
    for (int cb = wave; cb < nb; cb += 2 * kEncWaves) {
      const bool two = cb + kEncWaves < nb;
      const int cb1 = two ? cb + kEncWaves : cb;
      floatx4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f};
      floatx4 acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
      // 64 of K at a time: all operands of 16 steps are read from LDS
      // first (one wait), then the 32 matrix instructions run back to back;
      // steps past K read row 0 and multiply by a zero A operand.
      for (int kb = 0; kb < K; kb += 64) {
        float av[16], b0[16], b1[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int k = kb + 4 * u + kq;
          const bool in = k < K;
          const int kk = in ? k : 0;
          av[u] = in ? A[r16 * lda + kk] : 0.0f;
          b0[u] = Wb[kk * ldw + cb * 16 + r16];
          b1[u] = Wb[kk * ldw + cb1 * 16 + r16];
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], b0[u], acc0, 0, 0, 0);
          acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], b1[u], acc1, 0, 0, 0);
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (h == 1 && !two) break;
        const int col = c.n0 + (h == 0 ? cb : cb1) * 16 + r16;
        const float bc = bias[col];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 4 * kq + i;
          float y = (h == 0 ? acc0[i] : acc1[i]) + bc;
          if (relu) y = fmaxf(y, 0.0f);
          if (accumulate) y = Y[r * ldy + col] + y;
          Y[r * ldy + col] = y;
        }
      }
    }
    c = nx;
  }
  __syncthreads();
}

// Z[r] = LN(X[r]) * g + b for `rows` rows (X row r at X + r * ldx), H a
// multiple of 16 up to 128: a row per 16-lane group (lane j of the group
// holds elements j, j + 16, ...), the four groups of a wavefront on four
// rows at once, so the reductions' shuffles of four rows overlap.
__device__ __forceinline__ void layer_norm_rows(const float* X, int ldx, float* Z, int ldz, const float* g,
                                                const float* bt, int H, int rows) {
  const int lane = threadIdx.x & 63;
  const int grp = threadIdx.x >> 4;          // 16 groups in the workgroup
  const int j = lane & 15;
  const int nt = H >> 4;
  for (int r = grp; r < rows; r += kEncThreads / 16) {
    float v[8];
    float sum = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      v[t] = t < nt ? X[r * ldx + j + 16 * t] : 0.0f;
      sum += v[t];
    }
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 16);
    const float mean = sum / static_cast<float>(H);
    float sq = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      v[t] = t < nt ? v[t] - mean : 0.0f;
      sq += v[t] * v[t];
    }
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) sq += __shfl_xor(sq, o, 16);
    const float rstd = 1.0f / sqrtf(sq / static_cast<float>(H) + 1e-5f);
#pragma unroll
    for (int t = 0; t < 8; ++t)
      if (t < nt) Z[r * ldz + j + 16 * t] = v[t] * rstd * g[j + 16 * t] + bt[j + 16 * t];
  }
}

// One layer's parameters inside the packed array.
struct LayerPtrs {
  const float *ln1_g, *ln1_b, *Wqkv, *bqkv, *Wo, *bo, *ln2_g, *ln2_b, *W1, *b1, *W2, *b2;
};

__device__ __forceinline__ LayerPtrs layer_ptrs(const float* L, int H, int F) {
  LayerPtrs p;
  p.ln1_g = L;
  p.ln1_b = p.ln1_g + H;
  p.Wqkv = p.ln1_b + H;
  p.bqkv = p.Wqkv + static_cast<size_t>(H) * 3 * H;
  p.Wo = p.bqkv + 3 * H;
  p.bo = p.Wo + static_cast<size_t>(H) * H;
  p.ln2_g = p.bo + H;
  p.ln2_b = p.ln2_g + H;
  p.W1 = p.ln2_b + H;
  p.b1 = p.W1 + static_cast<size_t>(H) * F;
  p.W2 = p.b1 + F;
  p.b2 = p.W2 + static_cast<size_t>(F) * H;
  return p;
}

__global__ __launch_bounds__(kEncThreads) void encoder_kernel(const EncArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int H = a.H, F = a.F;
  const int ldh = H + kPad, ldq = 3 * H + kPad, ldf = F + kPad;
  float* X = reinterpret_cast<float*>(smem);          // [16][ldh] token states
  float* Z = X + kEncRows * ldh;                      // [16][ldh] normalized tokens / attention output
  float* QKV = Z + kEncRows * ldh;                    // [16][ldq]
  float* Hd = QKV + kEncRows * ldq;                   // [16][ldf] feed-forward hidden
  float* Wb = Hd + kEncRows * ldf;                    // [kWbuf + 4] weight staging (+ a 16-byte sink)
  float* sv = Wb + kWbuf + 4;                         // [layers * (9H + F) + 2H] gains and biases
  DevPred* sp = reinterpret_cast<DevPred*>(sv + vec_floats(H, F, a.layers));   // [kEncQ]
  float* fa = reinterpret_cast<float*>(sp + kEncQ);   // [16] normalized lower bound of the row's clause
  float* fb = fa + kEncRows;                          // [16] normalized upper bound
  int* kind = reinterpret_cast<int*>(fb + kEncRows);  // [16] 0 padding, 1 summary, 2 clause
  int* col = kind + kEncRows;                         // [16] clause column
  int* seq = col + kEncRows;                          // [kEncQ] tokens of each predicate

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  if (static_cast<int>(blockIdx.x) >= a.enc_blocks) {
    // a side workgroup: no barrier below, the whole group leaves here
    const int item = (static_cast<int>(blockIdx.x) - a.enc_blocks) * kEncWaves + __builtin_amdgcn_readfirstlane(wave);
    copy_slot_order(a.iv, item, a.n_side_waves, lane);
    if (item < a.n_cond) {
      condition_alpha(a, item, lane);
    } else if (item - a.n_cond < 2 * a.iv.nq) {
      const int j = item - a.n_cond;
      interval_bound(a.iv, j >> 1, j & 1, lane);
    }
    return;
  }
  const int q0 = blockIdx.x * kEncQ;
  const float* col_embed = a.p;
  const float* feat_w = col_embed + static_cast<size_t>(a.n_attr) * H;
  const float* feat_b = feat_w + 2 * H;
  const float* cls = feat_b + H;
  const float* layer0 = cls + H;
  const size_t layer_floats = static_cast<size_t>(2 * H) + 3 * H * H + 3 * H + H * H + H + 2 * H + H * F + F +
                              F * H + H;
  // The first projection's weights are on their way, and every layer's gains
  // and biases go to LDS, while the predicates come from host memory.  sv
  // holds per layer ln1_g, ln1_b | bqkv | bo, ln2_g, ln2_b | b1 | b2, then
  // lnf_g, lnf_b.
  Prefetch pf;
  prefetch(first_chunk(layer_ptrs(layer0, H, F).Wqkv, H, 3 * H), pf);
  if (wave < kEncQ && q0 + wave < a.nq) copy_pred(a.preds + q0 + wave, sp + wave, lane);
  {
    const int vs = 9 * H + F, n = vec_floats(H, F, a.layers);
    const float* lnf = layer0 + a.layers * layer_floats;
    for (int i0 = 0; i0 < n; i0 += 8 * kEncThreads) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + static_cast<int>(threadIdx.x) + u * kEncThreads;
        const int l = i / vs, e = i - l * vs;
        const LayerPtrs w = layer_ptrs(layer0 + l * layer_floats, H, F);
        const float* src = l >= a.layers ? lnf + e
                           : e < 2 * H   ? w.ln1_g + e
                           : e < 5 * H   ? w.bqkv + (e - 2 * H)
                           : e < 8 * H   ? w.bo + (e - 5 * H)
                           : e < 8 * H + F ? w.b1 + (e - 8 * H)
                                           : w.b2 + (e - 8 * H - F);
        v[u] = i < n ? *src : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + static_cast<int>(threadIdx.x) + u * kEncThreads;
        if (i < n) sv[i] = v[u];
      }
    }
  }
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

  const int dh = H / a.heads;
  const float inv_sqrt_dh = 1.0f / sqrtf(static_cast<float>(dh));
  for (int layer = 0; layer < a.layers; ++layer) {
    const LayerPtrs w = layer_ptrs(layer0 + layer * layer_floats, H, F);
    const Chunk none{nullptr, 1, 1, 0, 16};
    const Chunk after_ffn =
        layer + 1 < a.layers ? first_chunk(layer_ptrs(layer0 + (layer + 1) * layer_floats, H, F).Wqkv, H, 3 * H)
                             : none;

    const float* lv = sv + layer * (9 * H + F);
    const float* s_ln1_g = lv;
    const float* s_ln1_b = lv + H;
    const float* s_bqkv = lv + 2 * H;
    const float* s_bo = lv + 5 * H;
    const float* s_ln2_g = lv + 6 * H;
    const float* s_ln2_b = lv + 7 * H;
    const float* s_b1 = lv + 8 * H;
    const float* s_b2 = lv + 8 * H + F;
    layer_norm_rows(X, ldh, Z, ldh, s_ln1_g, s_ln1_b, H, kEncRows);
    gemm_rows(Z, ldh, first_chunk(w.Wqkv, H, 3 * H), s_bqkv, QKV, ldq, false, false, Wb, pf,
              first_chunk(w.Wo, H, H));
    // Attention, one item per (predicate, head, token i, dimension d): the
    // scores of row i against the predicate's tokens (the dh threads of a
    // (row, head) compute them alike; their reads are broadcasts), the
    // softmax over them, then the weighted sum of V, into Z (head slices side
    // by side); padding rows get zeros.
    for (int t = threadIdx.x; t < kEncRows * H; t += kEncThreads) {
      const int d = t % dh, hd = (t / dh) % a.heads, r = t / H;   // r = qi * kEncSlots + i
      const int qi = r / kEncSlots, i = r % kEncSlots;
      const int S = seq[qi];
      float out = 0.0f;
      if (i < S) {
        const float* qv = QKV + r * ldq + hd * dh;
        float sc[kEncSlots];
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < kEncSlots; ++j) {
          sc[j] = -INFINITY;
          if (j < S) {
            const float* kv = QKV + (qi * kEncSlots + j) * ldq + H + hd * dh;
            float acc = 0.0f;
#pragma unroll 4
            for (int e = 0; e < dh; ++e) acc += qv[e] * kv[e];
            sc[j] = acc * inv_sqrt_dh;
            mx = fmaxf(mx, sc[j]);
          }
        }
        float sum = 0.0f, acc = 0.0f;
#pragma unroll
        for (int j = 0; j < kEncSlots; ++j) {
          if (j < S) {
            const float e = expf(sc[j] - mx);
            sum += e;
            acc += e * QKV[(qi * kEncSlots + j) * ldq + 2 * H + hd * dh + d];
          }
        }
        out = acc / sum;
      }
      Z[r * ldh + hd * dh + d] = out;
    }
    gemm_rows(Z, ldh, first_chunk(w.Wo, H, H), s_bo, X, ldh, true, false, Wb, pf, first_chunk(w.W1, H, F));
    layer_norm_rows(X, ldh, Z, ldh, s_ln2_g, s_ln2_b, H, kEncRows);
    gemm_rows(Z, ldh, first_chunk(w.W1, H, F), s_b1, Hd, ldf, false, true, Wb, pf, first_chunk(w.W2, F, H));
    gemm_rows(Hd, ldf, first_chunk(w.W2, F, H), s_b2, X, ldh, true, false, Wb, pf, after_ffn);
  }
  const float* L = layer0 + a.layers * layer_floats;

  // w_z = LN_f(summary token) W_out + b_out, the kEncQ predicates side by
  // side so every W_out row is read once per workgroup.
  const float* lnf_g = L;
  const float* lnf_b = lnf_g + H;
  const float* out_w = lnf_b + H;
  const float* out_b = out_w + static_cast<size_t>(H) * a.D;
  // (row r of the normalization is predicate r's summary token: input row
  // stride kEncSlots rows)
  const float* s_lnf = sv + a.layers * (9 * H + F);
  layer_norm_rows(X, kEncSlots * ldh, Z, ldh, s_lnf, s_lnf + H, H, kEncQ);
  __syncthreads();
  const int nv = min(kEncQ, a.nq - q0);
  for (int d = threadIdx.x; d < a.D; d += kEncThreads) {
    float acc[kEncQ] = {};
#pragma unroll 16
    for (int h = 0; h < H; ++h) {
      const float w = out_w[static_cast<size_t>(h) * a.D + d];
#pragma unroll
      for (int qi = 0; qi < kEncQ; ++qi) acc[qi] += Z[qi * ldh + h] * w;
    }
    for (int qi = 0; qi < nv; ++qi) {
      const float wz = acc[qi] + out_b[d];
      a.wz[static_cast<size_t>(q0 + qi) * a.D + d] = wz;
      if (a.cond.wf) a.cond.wf[static_cast<size_t>(q0 + qi) * a.D + d] = softplus_weight(wz);
    }
  }
}

}  // namespace

size_t encoder_lds_bytes(int H, int F, int layers) {
  const size_t floats = static_cast<size_t>(kEncRows) * (2 * (H + kPad) + (3 * H + kPad) + (F + kPad)) + kWbuf + 4 +
                        vec_floats(H, F, layers);
  return floats * sizeof(float) + kEncQ * sizeof(DevPred) + kEncRows * 2 * sizeof(float) +
         (2 * kEncRows + kEncQ) * sizeof(int);
}

bool encoder_conditions(int h, bool has_bank) { return !has_bank || (h >= 1 && h <= kEncCondMaxH); }

hipError_t launch_encoder(const float* params, const double* off, const double* scale, int H, int heads, int layers,
                          int F, int D, int n_attr, const DevPred* preds, int nq, float* wz, hipStream_t s,
                          const EncCondition* cond, const IntervalArgs* iv) {
  if (nq <= 0) return hipSuccess;
  if (iv && iv->nq != nq) return hipErrorInvalidValue;
  if (cond && (!cond->wf || !encoder_conditions(cond->h, cond->alpha != nullptr) ||
               (cond->alpha && (!cond->q || !cond->bank || cond->bank_rows <= 0))))
    return hipErrorInvalidValue;
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
  if (cond) a.cond = *cond;
  if (iv) a.iv = *iv;
  a.enc_blocks = (nq + kEncQ - 1) / kEncQ;
  a.n_cond = cond && cond->alpha ? nq : 0;
  const int side_items = a.n_cond + 2 * a.iv.nq;
  const int side_blocks = (side_items + kEncWaves - 1) / kEncWaves;
  a.n_side_waves = side_blocks * kEncWaves;
  const size_t lds = encoder_lds_bytes(H, F, layers);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&encoder_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(encoder_kernel, dim3(a.enc_blocks + side_blocks), dim3(kEncThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace ifvs
