// Kernels of the backward pass of the fused lm-head log-probability.
//
// For L = sum_n g_n log p_n(y_n) (g_n: the upstream gradient of each scored
// row's log-likelihood, from the policy loss of Sec. 3.3), with
// G[n][v] = g_n (1[v == y_n] - p_n(v)) the gradient with respect to the logits:
//
//     dL/dh_n = sum_v G[n][v] W[v]        (dH = G W)
//     dL/dW_v = sum_n G[n][v] h_n         (dW = G^T H)
//
// G is produced chunk by chunk (at most a few thousand rows at a time, so the
// rows x vocabulary tensor never exists whole) by the fused lm-head kernel in
// its gradient mode, which recomputes the logits tile by tile.  The two
// contractions are plain bf16 GEMMs on the same 256 x 256 MFMA tile as the
// forward kernel (gemm_nt_kernel below); both of their operands must be
// contiguous along the contracted index, so G, W and the chunk's hidden rows
// are also written transposed (transpose_kernel).  dH is split along the
// vocabulary for parallelism and its partial sums are added in a fixed order
// (splitk_scatter_kernel): the whole pass is deterministic.
#include "tile_common.h"

namespace hdl {
namespace {

using namespace tile;

constexpr int kGemmSliceK = 8 * kChunks;   // bf16 elements per K-slice

// C[s][m][n] (=|+=) sum_k A[m][k] B[n][k] over the K range of split s, for
// one 256 x 256 tile of C per workgroup.  Same data path as the fused
// kernel: K-slices of 128 bytes per row stream into a 2-stage LDS ring by
// direct DMA; eight waves each own 128 x 64 of the tile as 4 x 2 MFMA blocks.
__global__ __launch_bounds__(kThreads, 1) void gemm_nt_kernel(GemmArgs p) {
  using M = Mma<true>;
  static_assert(kWaves == 8 && kNB == 2, "8-wave tile layout assumed");
  __shared__ uint4 lds[kStages][2][kSlots];   // [stage][0 = A, 1 = B]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int half = lane >> 5;
  const int col = lane & 31;

  // ---- work item: XCD-aware (m-tile, n-tile, split) ----------------------
  // The j-th workgroup of an XCD belongs to launch group j / 32 of that XCD;
  // a group is gm x gn tiles of one split, sharing A and B rows through L2.
  const int64_t b = blockIdx.x;
  const int64_t xcd = b % kNumXcd;
  const int64_t j = b / kNumXcd;
  const int64_t grp = (j / (p.gm * p.gn)) * kNumXcd + xcd;
  const int64_t loc = j % (p.gm * p.gn);
  const int64_t n_gm = (p.tiles_m + p.gm - 1) / p.gm;
  const int64_t n_gn = (p.tiles_n + p.gn - 1) / p.gn;
  // (the runtime divisions run on the vector ALU; readfirstlane puts the
  // wave-uniform results back in scalar registers for the DMA base)
  const int64_t split = __builtin_amdgcn_readfirstlane(static_cast<int>(grp / (n_gm * n_gn)));
  const int64_t rem = grp % (n_gm * n_gn);
  const int64_t tm = __builtin_amdgcn_readfirstlane(static_cast<int>((rem % n_gm) * p.gm + loc % p.gm));
  const int64_t tn = __builtin_amdgcn_readfirstlane(static_cast<int>((rem / n_gm) * p.gn + loc / p.gm));
  if (split >= p.splits || tm >= p.tiles_m || tn >= p.tiles_n) return;

  int64_t m_valid = p.m, k_valid = p.k;
  if (p.dyn_dim != 0) {
    int64_t dv = *p.dyn - p.dyn_base;
    const int64_t cap = p.dyn_dim == 1 ? p.m : p.k;
    dv = dv < 0 ? 0 : (dv > cap ? cap : dv);
    if (p.dyn_dim == 1) m_valid = dv;
    else k_valid = (dv + kGemmSliceK - 1) / kGemmSliceK * kGemmSliceK;
  }
  if (tm * kTileV >= m_valid) return;
  const int64_t k0 = split * p.k_split;
  const int64_t k1 = (k0 + p.k_split < k_valid) ? k0 + p.k_split : k_valid;
  const int n_iter = k1 > k0 ? static_cast<int>((k1 - k0) / kGemmSliceK) : 0;
  if (n_iter == 0 && p.beta) return;   // nothing to add

  f32x16_t acc[4][kNB];
#pragma unroll
  for (int bm = 0; bm < 4; ++bm)
#pragma unroll
    for (int bn = 0; bn < kNB; ++bn)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[bm][bn][q] = 0.f;

  if (n_iter > 0) {
    // ---- DMA addressing (tile-relative 32-bit offsets, uniform 64-bit base)
    const int lrow = lane / kChunks;
    auto dma_chunk = [&](int i) {
      const int row = (wave * kBlocksPerWave + i) * kBlockRows + lrow;
      return (lane % kChunks) ^ row_xor(row);
    };
    const int64_t a_row_bytes = p.lda * 2, b_row_bytes = p.ldb * 2;
    uint32_t aoff[kBlocksPerWave], boff[kBlocksPerWave];
#pragma unroll
    for (int i = 0; i < kBlocksPerWave; ++i) {
      const int r = wave * (kTileV / kWaves) + i * kBlockRows + lrow;
      int64_t ra = tm * kTileV + r;
      ra = ra < m_valid ? ra : m_valid - 1;
      int64_t rb = tn * kTileN + r;
      rb = rb < p.n ? rb : p.n - 1;
      aoff[i] = static_cast<uint32_t>((ra - tm * kTileV) * a_row_bytes + dma_chunk(i) * 16);
      boff[i] = static_cast<uint32_t>((rb - tn * kTileN) * b_row_bytes + dma_chunk(i) * 16);
    }
    const uint64_t atile = reinterpret_cast<uint64_t>(p.a) + static_cast<uint64_t>(tm * kTileV * a_row_bytes);
    const uint64_t btile = reinterpret_cast<uint64_t>(p.b) + static_cast<uint64_t>(tn * kTileN * b_row_bytes);
    const uint32_t lds_base = static_cast<uint32_t>(
        reinterpret_cast<size_t>((__attribute__((address_space(3))) uint4*)(&lds[0][0][0])));
    auto lds_addr = [&](int stage, int op, int block) -> uint32_t {
      return __builtin_amdgcn_readfirstlane(
          lds_base + static_cast<uint32_t>(((stage * 2 + op) * kSlots + block * 64) * 16));
    };
    uint32_t issue_kbytes = 0;
    int issue_stage = 0;
    auto prep_issue = [&](int slice) {
      issue_stage = slice % kStages;
      issue_kbytes = static_cast<uint32_t>((k0 + static_cast<int64_t>(slice) * kGemmSliceK) * 2);
    };
    auto issue_one = [&](int jj) {
      const int i = jj % kBlocksPerWave;
      const bool is_a = jj < kBlocksPerWave;
      dma16((is_a ? atile : btile) + issue_kbytes, is_a ? aoff[i] : boff[i],
            lds_addr(issue_stage, is_a ? 0 : 1, wave * kBlocksPerWave + i));
    };
    auto load_frags = [&](int slice, int kk, uint4 (&fa)[4], uint4 (&fb)[kNB]) {
      const int stage = slice % kStages;
#pragma unroll
      for (int bm = 0; bm < 4; ++bm) fa[bm] = lds[stage][0][swz(wm * 128 + bm * 32 + col, kk * 2 + half)];
#pragma unroll
      for (int bn = 0; bn < kNB; ++bn) fb[bn] = lds[stage][1][swz(wn * kWaveN + bn * 32 + col, kk * 2 + half)];
    };

    const int n_pre = n_iter < kStages ? n_iter : kStages;
    for (int sl = 0; sl < n_pre; ++sl) {
      prep_issue(sl);
#pragma unroll
      for (int jj = 0; jj < kDmaPerSlice; ++jj) issue_one(jj);
    }
    wait_dma(n_pre - 1);
    raw_barrier();

    uint4 fa[2][4], fb[2][kNB];
    load_frags(0, 0, fa[0], fb[0]);
    for (int it = 0; it < n_iter; ++it) {
#pragma unroll
      for (int kk = 0; kk < kSub; ++kk) {
        const int cur = kk & 1;
        if (kk + 1 < kSub) {
          load_frags(it, kk + 1, fa[cur ^ 1], fb[cur ^ 1]);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < 4 * kNB; ++q) M::run(fa[cur][q / kNB], fb[cur][q % kNB], acc[q / kNB][q % kNB]);
        } else {
          // Every read of slice `it` is issued: wait for slice it+1, then
          // refill this slice's stage with slice it+kStages (past the end:
          // the last slice again, into a stage nothing reads any more; the
          // fragment reads of the call's last step fetch stale, unused LDS).
          wait_dma(kStages - 2);
          raw_barrier();
          prep_issue(it + kStages < n_iter ? it + kStages : n_iter - 1);
          load_frags(it + 1, 0, fa[cur ^ 1], fb[cur ^ 1]);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < 4 * kNB; ++q) {
            M::run(fa[cur][q / kNB], fb[cur][q % kNB], acc[q / kNB][q % kNB]);
            issue_one(q);   // 8 MFMAs, 8 DMAs per slice
          }
        }
      }
    }
    wait_vmcnt<0>();
  }

  // ---- store: lanes of one accumulator element cover 32 consecutive n ----
  float* cbase = p.c + split * p.c_split_stride;
#pragma unroll
  for (int bn = 0; bn < kNB; ++bn) {
    const int64_t n = tn * kTileN + wn * kWaveN + bn * 32 + col;
    if (n >= p.n) continue;
#pragma unroll
    for (int bm = 0; bm < 4; ++bm)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int64_t m = tm * kTileV + wm * 128 + bm * 32 + acc_row(q, half);
        if (m < m_valid) {
          float* dst = cbase + m * p.ldc + n;
          *dst = p.beta ? *dst + acc[bm][bn][q] : acc[bm][bn][q];
        }
      }
  }
}

// 64 x 64 tiles through LDS: coalesced 16-byte reads of input rows and
// 16-byte writes of output rows.
__global__ __launch_bounds__(256) void transpose_kernel(TransposeArgs p) {
  __shared__ __align__(16) uint16_t t[64][72];   // [input row][input column], rows padded to 144 bytes
  int64_t r_valid = p.r_cap;
  if (p.dyn) {
    r_valid = *p.dyn - p.dyn_base;
    r_valid = r_valid < 0 ? 0 : (r_valid > p.r_cap ? p.r_cap : r_valid);
  }
  const int64_t r_end = (r_valid + 63) / 64 * 64;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * 64;
  const int64_t c0 = static_cast<int64_t>(blockIdx.y) * 64;
  if (r0 >= r_end || c0 >= p.out_rows) return;
  for (int q = threadIdx.x; q < 512; q += 256) {
    const int i = q >> 3, cc = (q & 7) * 8;
    const int64_t r = r0 + i, c = c0 + cc;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < r_valid && c < p.c_valid) {
      const int64_t src = p.map ? p.map[r] : r;
      v = *reinterpret_cast<const uint4*>(p.in + src * p.ld_in + c);
    }
    *reinterpret_cast<uint4*>(&t[i][cc]) = v;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < 512; q += 256) {
    const int i = q >> 3, rr = (q & 7) * 8;
    if (c0 + i >= p.out_rows) continue;
    uint32_t w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      w[u] = static_cast<uint32_t>(t[rr + 2 * u][i]) | (static_cast<uint32_t>(t[rr + 2 * u + 1][i]) << 16);
    *reinterpret_cast<uint4*>(p.out + (c0 + i) * p.ld_out + r0 + rr) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// dh[map[e]][j] = sum over splits s (in order) of part[s][e][j].
__global__ __launch_bounds__(256) void splitk_scatter_kernel(const float* __restrict__ part, int64_t splits,
                                                             int64_t split_stride, int64_t d,
                                                             const int32_t* __restrict__ map,
                                                             const int32_t* __restrict__ dyn, int64_t dyn_base,
                                                             int64_t cap, float* __restrict__ dh) {
  int64_t n_valid = *dyn - dyn_base;
  n_valid = n_valid < 0 ? 0 : (n_valid > cap ? cap : n_valid);
  const int64_t e = blockIdx.y;
  if (e >= n_valid) return;
  const int64_t j = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (j >= d) return;
  const float* src = part + e * d + j;
  float4 acc = *reinterpret_cast<const float4*>(src);
  for (int64_t s = 1; s < splits; ++s) {
    const float4 v = *reinterpret_cast<const float4*>(src + s * split_stride);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  *reinterpret_cast<float4*>(dh + static_cast<int64_t>(map[e]) * d + j) = acc;
}

__global__ __launch_bounds__(256) void zero_masked_rows_kernel(const uint8_t* __restrict__ mask, int64_t d,
                                                               float* __restrict__ dh) {
  const int64_t row = blockIdx.x;
  if (mask[row] != 0) return;
  float4* dst = reinterpret_cast<float4*>(dh + row * d);
  for (int64_t q = threadIdx.x; q < d / 4; q += 256) dst[q] = make_float4(0.f, 0.f, 0.f, 0.f);
}

}  // namespace

hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t stream) {
  const int64_t per_group = a.gm * a.gn;
  const int64_t groups = ((a.tiles_m + a.gm - 1) / a.gm) * ((a.tiles_n + a.gn - 1) / a.gn) * a.splits;
  const int64_t grid = (groups + kNumXcd - 1) / kNumXcd * kNumXcd * per_group;
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(gemm_nt_kernel, dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_transpose(const TransposeArgs& a, hipStream_t stream) {
  const int64_t gx = (a.r_cap + 63) / 64, gy = (a.out_rows + 63) / 64;
  if (gx <= 0 || gy <= 0) return hipSuccess;
  hipLaunchKernelGGL(transpose_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy)), dim3(256), 0,
                     stream, a);
  return hipGetLastError();
}

hipError_t launch_splitk_scatter(const float* part, int64_t splits, int64_t split_stride, int64_t d,
                                 const int32_t* map, const int32_t* dyn, int64_t dyn_base, int64_t cap,
                                 float* dh, hipStream_t stream) {
  const int64_t gx = (d / 4 + 255) / 256;
  if (gx <= 0 || cap <= 0) return hipSuccess;
  hipLaunchKernelGGL(splitk_scatter_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(cap)), dim3(256),
                     0, stream, part, splits, split_stride, d, map, dyn, dyn_base, cap, dh);
  return hipGetLastError();
}

hipError_t launch_zero_masked_rows(const uint8_t* mask, int64_t n_rows, int64_t d, float* dh,
                                   hipStream_t stream) {
  if (!mask || n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_masked_rows_kernel, dim3(static_cast<unsigned>(n_rows)), dim3(256), 0, stream, mask, d,
                     dh);
  return hipGetLastError();
}

}  // namespace hdl
