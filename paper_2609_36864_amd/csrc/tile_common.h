// Building blocks shared by the MFMA tile kernels of libhdl.so (the fused
// lm-head kernel and the plain GEMM of the backward pass): the 256 x 256
// workgroup tile, its LDS ring of K-slices with XOR-swizzled 16-byte chunks,
// the direct global -> LDS DMA, explicit memory-counter waits, and the MFMA
// step for bf16 and fp32 operands.  Not part of the public ABI.
#pragma once

#include "hdl_internal.h"

namespace hdl {
namespace tile {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;                           // two waves per SIMD
constexpr int kThreads = 64 * kWaves;
constexpr int kVB = 8;                              // 16-row MFMA blocks per wave along M (128 rows)
constexpr int kTB = 4;                              // 16-column MFMA blocks per wave along N
constexpr int kWaveN = 16 * kTB;                    // N columns per wave
constexpr int kChunks = 8;                          // 16-byte chunks per LDS row per stage (128-byte K-slices)
constexpr int kKSteps = kChunks / 4;                // MFMA K-steps (4 chunks each) per K-slice
constexpr int kStages = 2;                          // LDS ring depth (K-slices)
constexpr int kSlots = kTileV * kChunks;            // uint4 slots per operand per stage
constexpr int kBlockRows = 64 / kChunks;            // rows per 1 KB DMA block
constexpr int kBlocksPerWave = kTileV / kBlockRows / kWaves;   // DMA blocks per operand per wave
constexpr int kDmaPerSlice = 2 * kBlocksPerWave;    // DMA instructions per lane per slice
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

static_assert(kTileV == kTileN, "square workgroup tile assumed");
static_assert(2 * 16 * kVB == kTileV && 4 * kWaveN == kTileN, "8 waves as 2 (M) x 4 (N)");
static_assert(kStages * 2 * kSlots * 16 <= 160 * 1024, "LDS ring exceeds 160 KB");
static_assert(kDmaPerSlice * (kStages - 1) <= 63, "vmcnt range");

// XOR pattern of a row of 128 bytes: 8 consecutive rows get 8 distinct
// chunks, and rows r and r + 8 differ too, so a fragment read (16 rows; see
// frag_chunk) touches every bank at most once per pass.
__device__ __forceinline__ int row_xor(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// Slot of (row, logical 16-byte chunk) in a [rows][kChunks] LDS tile.
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * kChunks + (chunk ^ row_xor(row));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 16 bytes per lane from global memory straight into LDS at lds_base + 16*lane.
// The global address is a wave-uniform 64-bit base (SGPRs) plus a per-lane
// 32-bit byte offset, so issuing a DMA costs no vector ALU work.  M0 carries
// the LDS base; it is saved and restored around the DMA so the compiler's own
// use of M0 is unaffected.
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

// Wait until at most N of this lane's memory loads (DMAs) are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Wait until at most `slices` K-slices (0 or 1 with a 2-stage ring) of this
// lane's DMA are outstanding.
__device__ __forceinline__ void wait_dma(int slices) {
  if (slices >= 1) wait_vmcnt<kDmaPerSlice>();
  else wait_vmcnt<0>();
}

// Workgroup barrier without the memory fence __syncthreads() implies (the
// fence would wait for every in-flight DMA).  LDS reads issued before it
// are complete: callers wait lgkmcnt(0) first.
__device__ __forceinline__ void raw_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// The MFMA shape of the tile kernels: v_mfma_f32_16x16x32_bf16 (fp32
// inputs: four v_mfma_f32_16x16x4_f32 over one 16-byte fragment).  A
// fragment is 16 rows (M or N indices) of one operand: lane l holds row
// (l mod 16) and 16 bytes of consecutive K values, which lane group
// g = l div 16 takes from 16-byte chunk 4 ks + frag_chunk(g) of K-step ks.
// A and B fragments take the same K positions, so the contraction is exact
// whatever order the hardware sums them in.  The 16 x 16 fp32 result block
// sits in 4 registers per lane: column (l mod 16), rows 4 (l div 16) + i.
template <bool BF16> struct Mma16;

template <> struct Mma16<true> {
  __device__ __forceinline__ static void run(const uint4& a, const uint4& b, f32x4_t& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                0, 0, 0);
  }
};

template <> struct Mma16<false> {
  // Four K = 4 steps; lane group g supplies K offset 4 g + j in step j, the
  // same for both operands, so the four steps cover the fragment's 16 K values.
  __device__ __forceinline__ static void run(const uint4& a, const uint4& b, f32x4_t& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  }
};

// Order of the MFMAs of a quarter (two A fragments j = 0, 1 times kTB B
// fragments): B fragment snake(j, i) is the i-th for A fragment j, i.e.
// 0 .. kTB-1 for the first and kTB-1 .. 0 for the second, so that the B
// operand is the same on both sides of the change of A and fewer operand
// bits switch between consecutive MFMAs (with random data the matrix pipes
// then sustain about 2 % more under the power limit).  The accumulator
// blocks are independent, so the order does not change any result.
__device__ __forceinline__ constexpr int snake(int j, int i) { return (j & 1) ? kTB - 1 - i : i; }

// Which of a K-step's four 16-byte chunks lane group g reads: (0, 2, 1, 3).
// A ds_read_b128 serves lanes i..i+7 together with lanes i+32..i+39, i.e.
// lane groups g and g + 2 of the same 8 rows; they must read chunks c and
// c ^ 1, which the row swizzle keeps in disjoint banks (chunks c and c + 2,
// the identity mapping, collide two-way).
__device__ __forceinline__ int frag_chunk(int grp) { return ((grp & 1) << 1) | (grp >> 1); }

}  // namespace tile
}  // namespace hdl
