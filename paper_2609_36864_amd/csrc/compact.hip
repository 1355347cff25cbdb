// Eligibility compaction: the list of scored rows (mask != 0), in row order.
//
// Only policy-generated tokens are scored (Sec. 3.1: the score is defined for
// each policy-generated token; agent trajectories also contain environment
// observations, Sec. 4.1).  Compacting the mask first means masked rows cost
// no matrix work in the fused lm-head kernel.  Masked rows get log p = 0 and
// lse = 0 (and entropy = 0) here, so every output element is written by
// exactly one kernel.
//
// Two launches, both deterministic: per-block counts, then a scan + scatter
// in which every block sums the counts of the blocks before it.
#include "hdl_internal.h"

namespace hdl {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 16;
constexpr int kPerBlock = kThreads * kPerThread;   // 4096 rows per block
static_assert(kPerBlock == kCountBlockRows, "the workspace holds one count per block");

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  return v;
}

// Exclusive scan of one int per thread over a 256-thread block; *total gets
// the block sum.
__device__ __forceinline__ int block_excl_scan(int v, int* total) {
  __shared__ int wsum[kThreads / 64];
  const int incl = wave_incl_scan(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) wsum[w] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) {
    before += (i < w) ? wsum[i] : 0;
    all += wsum[i];
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

__device__ __forceinline__ bool row_on(const uint8_t* mask, int64_t n) {
  return mask == nullptr || mask[n] != 0;
}

__global__ __launch_bounds__(kThreads) void count_kernel(const uint8_t* __restrict__ mask, int64_t n_rows,
                                                         int32_t* __restrict__ block_counts) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kPerBlock + threadIdx.x * kPerThread;
  int c = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int64_t n = base + i;
    c += (n < n_rows && row_on(mask, n)) ? 1 : 0;
  }
  int total;
  block_excl_scan(c, &total);
  if (threadIdx.x == 0) block_counts[blockIdx.x] = total;
}

__global__ __launch_bounds__(kThreads) void scatter_kernel(const uint8_t* __restrict__ mask, int64_t n_rows,
                                                           const int32_t* __restrict__ block_counts,
                                                           int32_t* __restrict__ rows,
                                                           int32_t* __restrict__ n_scored,
                                                           float* __restrict__ logp,
                                                           float* __restrict__ lse,
                                                           float* __restrict__ entropy) {
  // rows scored by the blocks before this one
  int part = 0;
  for (int b = threadIdx.x; b < static_cast<int>(blockIdx.x); b += kThreads) part += block_counts[b];
  int prefix;
  block_excl_scan(part, &prefix);

  const int64_t base = static_cast<int64_t>(blockIdx.x) * kPerBlock + threadIdx.x * kPerThread;
  bool on[kPerThread];
  int c = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int64_t n = base + i;
    on[i] = n < n_rows && row_on(mask, n);
    c += on[i] ? 1 : 0;
  }
  int block_total;
  int pos = prefix + block_excl_scan(c, &block_total);
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int64_t n = base + i;
    if (n >= n_rows) break;
    if (on[i]) {
      rows[pos++] = static_cast<int32_t>(n);
    } else {
      if (logp) logp[n] = 0.f;
      if (lse) lse[n] = 0.f;
      if (entropy) entropy[n] = 0.f;
    }
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *n_scored = prefix + block_total;
}

}  // namespace

// Scratch for the per-block counts lives right after n_scored in the
// workspace (see layout_workspace in plan.h).
hipError_t launch_compact(const uint8_t* mask, int64_t n_rows, int32_t* rows, int32_t* n_scored,
                          float* logp, float* lse, float* entropy, hipStream_t stream) {
  const int64_t blocks = (n_rows + kPerBlock - 1) / kPerBlock;
  int32_t* block_counts = n_scored + 64;
  hipLaunchKernelGGL(count_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, mask,
                     n_rows, block_counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scatter_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, mask,
                     n_rows, block_counts, rows, n_scored, logp, lse, entropy);
  return hipGetLastError();
}

}  // namespace hdl
