// Measured bf16 MFMA ceilings of the GPU this runs on (a measurement tool for
// the fused lm-head kernel's roofline; not part of libhdl.so).
//
// Three loops, each on every CU with 8 waves (2 per SIMD) and
// v_mfma_f32_32x32x16_bf16 into 4x2 independent 32x32 accumulator blocks per
// wave -- the same instruction, block shape and occupancy as the fused kernel:
//   const  : operands with few set bits (bf16 1.0) -- the instruction-rate ceiling;
//   random : pseudo-random bf16 operands, as real weights and hidden states --
//            MFMA power rises with operand bit activity, so this ceiling is lower;
//   mixed  : random operands re-read from LDS every sub-step (6 ds_read_b128
//            fragments per 8 MFMAs, swizzled as in the fused kernel).
// Prints one JSON object with TFLOP/s for each.  Every LDS index is masked into
// range and every loop is bounded.
#include <hip/hip_runtime.h>

#include <cstdio>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int slot(int row, int chunk) {
  return row * 8 + (chunk ^ ((row & 7) ^ ((row >> 3) & 1)));
}

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  x ^= x >> 15; x *= 0x2c1b3c6du; x ^= x >> 12; x *= 0x297a2d39u; x ^= x >> 15;
  return x;
}

// MODE 0: constant operands, no LDS reads; 1: random operands, no LDS reads;
// 2: random operands re-read from LDS each sub-step.
template <int MODE>
__global__ __launch_bounds__(512) void ceiling_kernel(float* out, int iters) {
  __shared__ uint4 lds[2][2048];   // 64 KB: [A/B][256 rows x 8 chunks]
  for (int i = threadIdx.x; i < 4096; i += 512) {
    uint32_t h[4];
    for (int q = 0; q < 4; ++q) {
      const uint32_t x = mix32(static_cast<uint32_t>(i * 4 + q) * 2654435761u + 0x9e3779b9u * (blockIdx.x + 1));
      // two bf16 values with exponents near 1 and random sign/mantissa bits
      h[q] = MODE == 0 ? 0x3f803f80u : ((0x3e00u | (x & 0x80ffu)) | ((0x3e00u | ((x >> 16) & 0x80ffu)) << 16));
    }
    (&lds[0][0])[i] = make_uint4(h[0], h[1], h[2], h[3]);
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wm = wave & 1, wn = wave >> 1;
  const int col = lane & 31, half = lane >> 5;
  f32x16_t acc[4][2];
  for (int a = 0; a < 4; ++a)
    for (int b = 0; b < 2; ++b)
      for (int q = 0; q < 16; ++q) acc[a][b][q] = 0.f;
  uint4 fa[2][4], fb[2][2];
  for (int bm = 0; bm < 4; ++bm) fa[0][bm] = lds[0][slot(wm * 128 + bm * 32 + col, half)];
  for (int bn = 0; bn < 2; ++bn) fb[0][bn] = lds[1][slot(wn * 64 + bn * 32 + col, half)];
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int cur = kk & 1, nk = (kk + 1) & 3;
      if (MODE == 2) {
#pragma unroll
        for (int bm = 0; bm < 4; ++bm) fa[cur ^ 1][bm] = lds[0][slot(wm * 128 + bm * 32 + col, nk * 2 + half)];
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) fb[cur ^ 1][bn] = lds[1][slot(wn * 64 + bn * 32 + col, nk * 2 + half)];
        __builtin_amdgcn_sched_barrier(0);
      } else {
        for (int bm = 0; bm < 4; ++bm) fa[cur ^ 1][bm] = fa[cur][bm];
        for (int bn = 0; bn < 2; ++bn) fb[cur ^ 1][bn] = fb[cur][bn];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j >> 1][j & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, fa[cur][j >> 1]), __builtin_bit_cast(bf16x8_t, fb[cur][j & 1]),
            acc[j >> 1][j & 1], 0, 0, 0);
    }
  }
  float s = 0.f;
  for (int a = 0; a < 4; ++a)
    for (int b = 0; b < 2; ++b)
      for (int q = 0; q < 16; ++q) s += acc[a][b][q];
  out[blockIdx.x * 512 + threadIdx.x] = s;
}

template <int MODE>
double measure(float* out, int blocks, int iters) {
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return -1.0;
  float ms = 0.f;
  for (int rep = 0; rep < 2; ++rep) {   // the first launch warms clocks and caches
    if (hipEventRecord(e0) != hipSuccess) return -1.0;
    hipLaunchKernelGGL(ceiling_kernel<MODE>, dim3(blocks), dim3(512), 0, 0, out, iters);
    if (hipGetLastError() != hipSuccess || hipEventRecord(e1) != hipSuccess) return -1.0;
    if (hipEventSynchronize(e1) != hipSuccess) return -1.0;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) return -1.0;
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  const double flops = static_cast<double>(blocks) * 8 * iters * 4 * 8 * (2.0 * 32 * 32 * 16);
  return flops / (ms * 1e-3) / 1e12;
}

}  // namespace

int main() {
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, 0) != hipSuccess) {
    std::fprintf(stderr, "no GPU\n");
    return 1;
  }
  const int blocks = prop.multiProcessorCount * 2;
  const int iters = 3000;
  float* out = nullptr;
  if (hipMalloc(&out, static_cast<size_t>(blocks) * 512 * sizeof(float)) != hipSuccess) return 1;
  const double c = measure<0>(out, blocks, iters);
  const double r = measure<1>(out, blocks, iters);
  const double m = measure<2>(out, blocks, iters);
  (void)hipFree(out);
  if (c < 0 || r < 0 || m < 0) {
    std::fprintf(stderr, "kernel failed\n");
    return 1;
  }
  std::printf("{\"instruction\": \"v_mfma_f32_32x32x16_bf16\", \"cus\": %d, "
              "\"const_operands_tflops\": %.1f, \"random_operands_tflops\": %.1f, "
              "\"random_operands_with_lds_reads_tflops\": %.1f}\n",
              prop.multiProcessorCount, c, r, m);
  return 0;
}
