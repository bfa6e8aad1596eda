// Rank stage (Section 2, stage 2) as an asymmetric-distance scan over the
// 8-bit PQ codes of the selected vectors, feeding the Select stage's
// per-wavefront candidate pools.
//
// For a candidate v of query q: dist(v) = sum_{m<M} LUT_q[m][code_v[m]],
// summed in m order from +0 with separately rounded fp32 additions.
//
// Workgroup = kScanWaves wavefronts; grid = (code chunks, query tiles).
//  * The tables of QT queries live in LDS as [m][qi][256] so that, once a
//    lane has turned its vector's M code bytes into M LDS addresses, the
//    same addresses serve every query of the tile (query qi adds a constant
//    qi*256 that folds into the instruction's offset field).
//  * Codes are stored in 64-row tiles ("word j of all 64 rows" contiguous),
//    so each of the ceil(M/4) dword loads of a wavefront reads 256
//    consecutive bytes.  A tile is loaded once and reused by all QT queries.
//  * The selection bitmap supplies one 64-bit word per (query, tile): a zero
//    word skips the tile for that query without touching the codes, and a
//    tile no query selects is not loaded at all.
//  * Each lane whose vector is selected sums its M table entries; the lanes
//    beating the wavefront's current k-th best key are appended to that
//    query's pool (ballot + prefix count), which is sorted and cut back to
//    k keys whenever it would overflow.  At the end each wavefront writes its
//    k best keys per query; a separate merge kernel reduces them.
#include "ifvs_internal.h"
#include "topk_device.h"

namespace ifvs {

namespace {

__device__ __forceinline__ float widen(float v) { return v; }
__device__ __forceinline__ float widen(__half v) { return __half2float(v); }

template <int MT, int QT, typename LutT>
__global__ __launch_bounds__(kScanWaves * 64) void scan_dense_kernel(
    const uint32_t* __restrict__ codes_t, int64_t n_tiles, int m_rt, int mw,
    const LutT* __restrict__ lut, int nq, const uint64_t* __restrict__ bitmap,
    int64_t stride64, int k, int pool_stride, int kpl, int64_t tiles_per_block,
    uint64_t* __restrict__ partials) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kMW = MT > 0 ? (MT + 3) / 4 : 1;
  const int M = MT > 0 ? MT : m_rt;
  LutT* slut = reinterpret_cast<LutT*>(smem);
  const size_t lut_bytes = static_cast<size_t>(M) * QT * kKsub * sizeof(LutT);
  uint64_t* pools = reinterpret_cast<uint64_t*>(smem + lut_bytes);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q0 = blockIdx.y * QT;
  const int qn = min(QT, nq - q0);

  // Stage the query tile's tables: global [q][m][c] -> LDS [m][qi][c].
  constexpr int kVec = 16 / sizeof(LutT);
  const int vec_per_query = M * kKsub / kVec;
  for (int qi = 0; qi < qn; ++qi) {
    const uint4* src = reinterpret_cast<const uint4*>(lut + static_cast<size_t>(q0 + qi) * M * kKsub);
    for (int v = threadIdx.x; v < vec_per_query; v += kScanWaves * 64) {
      const int e = v * kVec;
      const int m = e / kKsub, c = e % kKsub;
      *reinterpret_cast<uint4*>(slut + (static_cast<size_t>(m) * QT + qi) * kKsub + c) = src[v];
    }
  }
  __syncthreads();

  int cnt[QT];
  uint64_t thr[QT];
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    cnt[qi] = 0;
    thr[qi] = kNoKey;
  }
  uint64_t* my_pools = pools + static_cast<size_t>(wave) * QT * pool_stride;

  const int64_t t_begin = static_cast<int64_t>(blockIdx.x) * tiles_per_block;
  const int64_t t_end = min(n_tiles, t_begin + tiles_per_block);
  for (int64_t t = t_begin + wave; t < t_end; t += kScanWaves) {
    uint64_t bm[QT];
    uint64_t any = 0;
#pragma unroll
    for (int qi = 0; qi < QT; ++qi) {
      bm[qi] = qi < qn ? bitmap[static_cast<size_t>(q0 + qi) * stride64 + t] : 0;
      any |= bm[qi];
    }
    if (any == 0) continue;
    const uint32_t id = static_cast<uint32_t>(t * 64 + lane);

    if constexpr (MT > 0) {
      uint32_t w[kMW];
#pragma unroll
      for (int j = 0; j < kMW; ++j) w[j] = codes_t[(t * kMW + j) * 64 + lane];
      int addr[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m)
        addr[m] = m * QT * kKsub + static_cast<int>((w[m >> 2] >> (8 * (m & 3))) & 0xFFu);
#pragma unroll
      for (int qi = 0; qi < QT; ++qi) {
        if (bm[qi] == 0) continue;
        const bool act = (bm[qi] >> lane) & 1ull;
        uint64_t key = kNoKey;
        bool cand = false;
        if (act) {
          float d = 0.0f;
#pragma unroll
          for (int m = 0; m < MT; ++m) d = __fadd_rn(d, widen(slut[addr[m] + qi * kKsub]));
          key = make_key(d, id);
          cand = key < thr[qi];
        }
        pool_push(my_pools + qi * pool_stride, cnt[qi], thr[qi], key, cand, k, kpl);
      }
    } else {
#pragma unroll
      for (int qi = 0; qi < QT; ++qi) {
        if (bm[qi] == 0) continue;
        const bool act = (bm[qi] >> lane) & 1ull;
        uint64_t key = kNoKey;
        bool cand = false;
        if (act) {
          float d = 0.0f;
          for (int m = 0; m < M; ++m) {
            const uint32_t wv = codes_t[(t * mw + (m >> 2)) * 64 + lane];
            const int c = static_cast<int>((wv >> (8 * (m & 3))) & 0xFFu);
            d = __fadd_rn(d, widen(slut[(static_cast<size_t>(m) * QT + qi) * kKsub + c]));
          }
          key = make_key(d, id);
          cand = key < thr[qi];
        }
        pool_push(my_pools + qi * pool_stride, cnt[qi], thr[qi], key, cand, k, kpl);
      }
    }
  }

  // Each wavefront's k best keys per query, ascending, padded with kNoKey.
#pragma unroll
  for (int qi = 0; qi < QT; ++qi) {
    if (qi >= qn) break;
    uint64_t* pool = my_pools + qi * pool_stride;
    pool_compact(pool, cnt[qi], thr[qi], k, kpl);
    uint64_t* dst = partials + ((static_cast<size_t>(q0 + qi) * gridDim.x + blockIdx.x) * kScanWaves + wave) * k;
    for (int e = lane; e < k; e += 64) dst[e] = pool[e];
  }
}

template <int MT, int QT, typename LutT>
const void* scan_symbol() {
  return reinterpret_cast<const void*>(&scan_dense_kernel<MT, QT, LutT>);
}

constexpr int kQtiles[] = {1, 2, 3, 4, 6, 8};

template <typename LutT, int MT>
const void* pick_q(int qt) {
  switch (qt) {
    case 1: return scan_symbol<MT, 1, LutT>();
    case 2: return scan_symbol<MT, 2, LutT>();
    case 3: return scan_symbol<MT, 3, LutT>();
    case 4: return scan_symbol<MT, 4, LutT>();
    case 6: return scan_symbol<MT, 6, LutT>();
    case 8: return scan_symbol<MT, 8, LutT>();
    default: return nullptr;
  }
}

template <typename LutT>
const void* pick(int m, int qt) {
  switch (m) {
    case 16: return pick_q<LutT, 16>(qt);
    case 48: return pick_q<LutT, 48>(qt);
    case 120: return pick_q<LutT, 120>(qt);
    default: return pick_q<LutT, 0>(qt);
  }
}

}  // namespace

int pool_kpl(int k) {
  int kpl = 2;
  while (64 * kpl < k + 64) kpl *= 2;
  return kpl;
}

int scan_max_qtile(int m, int lut_bytes, int k) {
  const size_t per_query = static_cast<size_t>(m) * kKsub * lut_bytes +
                           static_cast<size_t>(kScanWaves) * 64 * pool_kpl(k) * sizeof(uint64_t);
  return static_cast<int>(kLdsBudget / per_query);
}

int scan_supported_qtile(int want) {
  int best = 0;
  for (int q : kQtiles)
    if (q <= want) best = q;
  return best;
}

hipError_t launch_scan_dense(const uint32_t* codes_t, int64_t n_tiles, int m, int mw,
                             const void* lut, int lut_dtype, int nq, const uint64_t* bitmap,
                             int64_t stride64, int k, const ScanPlan& plan, uint64_t* partials,
                             hipStream_t s) {
  const void* fn = lut_dtype == 1 ? pick<__half>(m, plan.qtile) : pick<float>(m, plan.qtile);
  if (!fn) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     static_cast<int>(plan.lds_bytes));
  if (e != hipSuccess) return e;
  const dim3 grid(plan.splits, (nq + plan.qtile - 1) / plan.qtile);
  int m_arg = m, mw_arg = mw, nq_arg = nq, k_arg = k, ps = plan.pool_stride, kpl = plan.kpl;
  int64_t nt = n_tiles, st = stride64, tpb = plan.tiles_per_block;
  const uint32_t* c_arg = codes_t;
  const void* l_arg = lut;
  const uint64_t* b_arg = bitmap;
  uint64_t* p_arg = partials;
  void* args[] = {&c_arg, &nt, &m_arg, &mw_arg, &l_arg, &nq_arg, &b_arg, &st,
                  &k_arg, &ps,  &kpl,   &tpb,    &p_arg};
  return hipLaunchKernel(fn, grid, dim3(kScanWaves * 64), args, plan.lds_bytes, s);
}

}  // namespace ifvs
