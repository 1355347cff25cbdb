// Measured ceilings of the fused lm-head kernel's main loop on the GPU this
// runs on (a measurement tool for the kernel's roofline; not part of
// libhdl.so).
//
// Every loop runs on every CU with the kernel's shape: 8 waves (2 per SIMD),
// each 128 x 64 of a 256 x 256 tile as 8 x 4 blocks of
// v_mfma_f32_16x16x32_bf16, a K-slice being 2 K-steps x 4 quarters of 8
// MFMAs.  Step by step towards the kernel:
//   const      : operands held in registers, few set bits (bf16 1.0) -- the
//                instruction-rate ceiling;
//   random     : random bf16 operands in registers -- MFMA power rises with
//                operand bit activity, so the clock and this ceiling are lower;
//   lds        : random operands read from a 2-stage LDS ring every quarter
//                with the kernel's swizzle, fragment mapping and read-ahead,
//                one workgroup barrier per slice;
//   lds_write  : as lds, plus the ring's write traffic alone: each wave
//                writes its 8 x 1 KB of the stage just read from registers
//                (ds_write_b128), no global reads;
//   dma_l2     : as lds, plus the kernel's per-slice global -> LDS DMA of the
//                stage just freed (8 x 1 KB per wave, 128-byte runs of rows
//                4 KB apart) from a 4 MB source that stays in L2;
//   dma_hbm    : the same from a 1 GiB source (L2 misses to HBM).
// Prints one JSON object with TFLOP/s for each.  Every LDS index is in range
// by construction, every DMA source address lies inside its buffer, and every
// loop is bounded.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kSlots = 2048;                 // 256 rows x 8 sixteen-byte chunks per operand stage
constexpr uint64_t kRegion = 256ull * 4096;  // DMA source of one slice: 256 rows 4 KB apart

__device__ __forceinline__ int row_xor(int r) { return (r & 7) ^ ((r >> 3) & 1); }

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  x ^= x >> 15; x *= 0x2c1b3c6du; x ^= x >> 12; x *= 0x297a2d39u; x ^= x >> 15;
  return x;
}

// two bf16 values with exponents near 1 and random sign and mantissa bits
__device__ __forceinline__ uint32_t rand_pair(uint32_t x) {
  return (0x3e00u | (x & 0x80ffu)) | ((0x3e00u | ((x >> 16) & 0x80ffu)) << 16);
}

__device__ __forceinline__ void dma16(uint64_t sbase, uint32_t voff, uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(voff), "s"(sbase)
      : "memory");
}

__global__ void fill_random(uint32_t* p, uint64_t n) {
  for (uint64_t i = blockIdx.x * 256ull + threadIdx.x; i < n; i += 256ull * gridDim.x)
    p[i] = rand_pair(mix32(static_cast<uint32_t>(i) * 2654435761u + 0x9e3779b9u));
}

// MODE 0 const, 1 random (registers only); 2 lds; 3 lds + DMA (the source
// size decides L2 or HBM); 4 lds + register -> LDS writes of the same bytes.
template <int MODE>
__global__ __launch_bounds__(512, 1) void ceiling_kernel(const char* __restrict__ src, uint64_t n_regions,
                                                          float* out, int slices) {
  __shared__ uint4 lds[2][2][kSlots];   // [stage][A/B], 128 KB like the kernel's ring
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1, r16 = lane & 15, grp = lane >> 4;
  for (int i = tid; i < 2 * 2 * kSlots; i += 512) {
    uint32_t h[4];
    for (int q = 0; q < 4; ++q)
      h[q] = MODE == 0 ? 0x3f803f80u : rand_pair(mix32(static_cast<uint32_t>(i * 4 + q) * 2654435761u +
                                                       0x9e3779b9u * (blockIdx.x + 1)));
    (&lds[0][0][0])[i] = make_uint4(h[0], h[1], h[2], h[3]);
  }
  __syncthreads();
  f32x4_t acc[8][4];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int kchunk = ((grp & 1) << 1) | (grp >> 1);
  const int frag[2] = {r16 * 8 + ((0 + kchunk) ^ row_xor(r16)), r16 * 8 + ((4 + kchunk) ^ row_xor(r16))};
  auto load_a = [&](int st, int ks, int pr, uint4 (&d)[2]) {
#pragma unroll
    for (int j = 0; j < 2; ++j) d[j] = lds[st][0][frag[ks] + (wm * 128 + (2 * pr + j) * 16) * 8];
  };
  auto load_b = [&](int st, int ks, int bn, uint4& d) { d = lds[st][1][frag[ks] + (wn * 64 + bn * 16) * 8]; };
  auto mfma = [&](const uint4& a, const uint4& b, f32x4_t& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                0, 0, 0);
  };
  // (the kernel's MFMA order: B fragments 0..3 with the first A fragment,
  // 3..0 with the second)
  auto quarter = [&](const uint4 (&a)[2], const uint4 (&b)[4], int pr) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int bn = j ? 3 - i : i;
        mfma(a[j], b[bn], acc[2 * pr + j][bn]);
      }
  };
  const uint32_t lds_base = static_cast<uint32_t>(
      reinterpret_cast<size_t>((__attribute__((address_space(3))) uint4*)(&lds[0][0][0])));
  // DMA block i of this wave: rows 8 (4 w + i) .. + 7 of the region, lane l
  // at row + l / 8, 16-byte chunk l % 8 (the kernel's pattern); < kRegion
  uint32_t off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) off[i] = static_cast<uint32_t>(((wave * 4 + i) * 8 + lane / 8) * 4096 + (lane % 8) * 16);

  uint4 fa[2][2], fb[2][4];
  load_a(0, 0, 0, fa[0]);
#pragma unroll
  for (int bn = 0; bn < 4; ++bn) load_b(0, 0, bn, fb[0][bn]);
  for (int it = 0; it < slices; ++it) {
    const int st = MODE >= 2 ? (it & 1) : 0;
#pragma unroll
    for (int pr = 0; pr < 4; ++pr) {
      if (MODE >= 2) {
        if (pr < 3) load_a(st, 0, pr + 1, fa[(pr + 1) & 1]);
        else load_a(st, 1, 0, fa[0]);
        load_b(st, 1, pr, fb[1][pr]);
      } else {
        fa[(pr + 1) & 1][0] = fa[pr & 1][0]; fa[(pr + 1) & 1][1] = fa[pr & 1][1];
        fb[1][pr] = fb[0][pr];
      }
      __builtin_amdgcn_sched_barrier(0);
      quarter(fa[pr & 1], fb[0], pr);
    }
#pragma unroll
    for (int pr = 0; pr < 3; ++pr) {
      if (MODE >= 2) load_a(st, 1, pr + 1, fa[(pr + 1) & 1]);
      else { fa[(pr + 1) & 1][0] = fa[pr & 1][0]; fa[(pr + 1) & 1][1] = fa[pr & 1][1]; }
      __builtin_amdgcn_sched_barrier(0);
      quarter(fa[pr & 1], fb[1], pr);
    }
    // slice boundary: wait for this wave's DMA, workgroup barrier, then the
    // DMA of the slice after next into the stage just read
    if (MODE == 3) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (MODE >= 2) asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (MODE >= 2) {
      load_a(st ^ 1, 0, 0, fa[0]);
#pragma unroll
      for (int bn = 0; bn < 4; ++bn) load_b(st ^ 1, 0, bn, fb[0][bn]);
    } else {
      fa[0][0] = fa[1][0]; fa[0][1] = fa[1][1];
#pragma unroll
      for (int bn = 0; bn < 4; ++bn) fb[0][bn] = fb[1][bn];
    }
    __builtin_amdgcn_sched_barrier(0);
    const uint64_t sbase = reinterpret_cast<uint64_t>(src) +
                           ((static_cast<uint64_t>(blockIdx.x) + it) % n_regions) * kRegion;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int bn = (j / 4) ? 3 - j % 4 : j % 4;
      mfma(fa[1][j / 4], fb[1][bn], acc[6 + j / 4][bn]);
      if (MODE == 4) {
        const int op = j / 4, blk = j % 4;
        lds[st][op][(wave * 4 + blk) * 64 + lane] = fa[1][j & 1];
      }
      if (MODE == 3) {
        const int op = j / 4, blk = j % 4;
        dma16(sbase, off[blk],
              __builtin_amdgcn_readfirstlane(lds_base + static_cast<uint32_t>(((st * 2 + op) * kSlots +
                                                                               (wave * 4 + blk) * 64) * 16)));
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  float s = 0.f;
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) s += acc[a][b][0] + acc[a][b][1] + acc[a][b][2] + acc[a][b][3];
  out[blockIdx.x * 512 + threadIdx.x] = s;
}

template <int MODE>
double measure(const char* src, uint64_t n_regions, float* out, int blocks, int slices) {
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return -1.0;
  float ms = 0.f, best = 1e30f;
  for (int rep = 0; rep < 3; ++rep) {   // the first launch warms clocks and caches
    if (hipEventRecord(e0) != hipSuccess) return -1.0;
    hipLaunchKernelGGL(ceiling_kernel<MODE>, dim3(blocks), dim3(512), 0, 0, src, n_regions, out, slices);
    if (hipGetLastError() != hipSuccess || hipEventRecord(e1) != hipSuccess) return -1.0;
    if (hipEventSynchronize(e1) != hipSuccess) return -1.0;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) return -1.0;
    if (rep > 0 && ms < best) best = ms;
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  const double flops = static_cast<double>(blocks) * slices * (2.0 * 256 * 256 * 64);
  return flops / (best * 1e-3) / 1e12;
}

}  // namespace

int main() {
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, 0) != hipSuccess) {
    std::fprintf(stderr, "no GPU\n");
    return 1;
  }
  const int blocks = prop.multiProcessorCount * 4;
  const int slices = 1500;
  const uint64_t big = 1ull << 30, small = 4ull << 20;
  char* src = nullptr;
  float* out = nullptr;
  if (hipMalloc(&src, big) != hipSuccess) return 1;
  if (hipMalloc(&out, static_cast<size_t>(blocks) * 512 * sizeof(float)) != hipSuccess) return 1;
  hipLaunchKernelGGL(fill_random, dim3(4096), dim3(256), 0, 0, reinterpret_cast<uint32_t*>(src), big / 4);
  if (hipDeviceSynchronize() != hipSuccess) return 1;
  const double c = measure<0>(src, 1, out, blocks, slices);
  const double r = measure<1>(src, 1, out, blocks, slices);
  const double l = measure<2>(src, 1, out, blocks, slices);
  const double lw = measure<4>(src, 1, out, blocks, slices);
  const double d2 = measure<3>(src, small / kRegion, out, blocks, slices);
  const double dh = measure<3>(src, big / kRegion, out, blocks, slices);
  (void)hipFree(out);
  (void)hipFree(src);
  if (c < 0 || r < 0 || l < 0 || lw < 0 || d2 < 0 || dh < 0) {
    std::fprintf(stderr, "kernel failed\n");
    return 1;
  }
  std::printf("{\"instruction\": \"v_mfma_f32_16x16x32_bf16\", \"cus\": %d, "
              "\"const_operands_tflops\": %.1f, \"random_operands_tflops\": %.1f, "
              "\"slice_loop_lds_tflops\": %.1f, \"slice_loop_lds_write_tflops\": %.1f, "
              "\"slice_loop_dma_l2_tflops\": %.1f, \"slice_loop_dma_hbm_tflops\": %.1f}\n",
              prop.multiProcessorCount, c, r, l, lw, d2, dh);
  return 0;
}
