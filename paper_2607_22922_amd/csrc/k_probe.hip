// LDS gather probe: the rate at which the LDS of every CU serves 4-byte
// reads at random addresses of a distance-table-sized array, the access the
// ADC scan makes once per (selected row, subspace).  It is a measurement of
// the roof that bounds the scan when code bytes arrive faster than they can
// be looked up, not a step of the method.
//
// Every workgroup (eight wavefronts, like a scan workgroup) fills a 48 KB
// table in LDS; each active lane draws 32 random entries, one within each of
// 32 1 KB sub-tables, each address in a register of its own (so every read is
// a single-address instruction, as the scan's are), and then reads them over
// and over: the 32 banks see random, conflicting addresses as in the scan.
// The reads are consumed by integer three-operand adds (half a vector
// instruction per read), so the vector ALU never limits the rate, also with
// few lanes.  `active` lanes of each wavefront take part (chosen by a fixed
// scramble of the lane number, since the lanes that survive early
// abandonment in the scan are scattered), which measures what a read with
// fewer lanes costs.
#include "ifvs_internal.h"

namespace ifvs {

namespace {

constexpr int kProbeThreads = 512;
constexpr int kProbeEntries = 12288;   // 48 KB: one 48-subspace fp32 distance table
constexpr int kProbeReads = 32;        // reads per lane and iteration, one per 1 KB sub-table

__global__ __launch_bounds__(kProbeThreads) void lds_gather_probe_kernel(int active, int iters, uint32_t* sink) {
  __shared__ uint32_t tab[kProbeEntries];
  for (int i = threadIdx.x; i < kProbeEntries; i += kProbeThreads) tab[i] = static_cast<uint32_t>(i & 255);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int rank = (lane * 37 + 11) & 63;   // 37 is odd: a permutation of 0..63
  uint32_t x = 0x9E3779B9u * (blockIdx.x * static_cast<uint32_t>(kProbeThreads) + threadIdx.x + 1u);
  int off[kProbeReads];
#pragma unroll
  for (int u = 0; u < kProbeReads; ++u) {
    x ^= x << 13;
    x ^= x >> 17;
    x ^= x << 5;
    off[u] = u * 256 + static_cast<int>(x & 255u);   // < 32 * 256 <= kProbeEntries
  }
  uint32_t acc = 0;
  if (rank < active) {
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int u = 0; u < kProbeReads; u += 2) acc += tab[off[u]] + tab[off[u + 1]];
      // A compiler barrier: the reads are issued again every iteration.
      __asm__ volatile("" : "+v"(acc) : : "memory");
    }
  }
  // The sum decides a store (into the 4-byte sink), so the reads are kept.
  if (acc == 0xFFFFFFFFu) sink[0] = acc;
}

}  // namespace

hipError_t lds_gather_probe(int active, int iters, int wg_per_cu, int reps, hipStream_t s, double* wave_reads_per_s) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  uint32_t* sink = nullptr;
  if ((e = hipMalloc(&sink, sizeof(uint32_t))) != hipSuccess) return e;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  const unsigned grid = static_cast<unsigned>(cus) * static_cast<unsigned>(wg_per_cu);
  float ms = 0.0f;
  do {
    if ((e = hipEventCreate(&e0)) != hipSuccess) break;
    if ((e = hipEventCreate(&e1)) != hipSuccess) break;
    hipLaunchKernelGGL(lds_gather_probe_kernel, dim3(grid), dim3(kProbeThreads), 0, s, active, iters, sink);
    if ((e = hipGetLastError()) != hipSuccess) break;
    if ((e = hipEventRecord(e0, s)) != hipSuccess) break;
    for (int i = 0; i < reps; ++i)
      hipLaunchKernelGGL(lds_gather_probe_kernel, dim3(grid), dim3(kProbeThreads), 0, s, active, iters, sink);
    if ((e = hipGetLastError()) != hipSuccess) break;
    if ((e = hipEventRecord(e1, s)) != hipSuccess) break;
    if ((e = hipEventSynchronize(e1)) != hipSuccess) break;
    e = hipEventElapsedTime(&ms, e0, e1);
  } while (false);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(sink);
  if (e != hipSuccess) return e;
  const double reads = static_cast<double>(grid) * (kProbeThreads / 64) * iters * kProbeReads * reps;
  *wave_reads_per_s = reads / (static_cast<double>(ms) / 1e3);
  return hipSuccess;
}

}  // namespace ifvs
