// Kernels of the backward pass of the fused lm-head log-probability.
//
// For L = sum_n g_n log p_n(y_n) (g_n: the upstream gradient of each scored
// row's log-likelihood, from the policy loss of Sec. 3.3), with
// G[n][v] = g_n (1[v == y_n] - p_n(v)) the gradient with respect to the logits:
//
//     dL/dh_n = sum_v G[n][v] W[v]        (dH = G W)
//     dL/dW_v = sum_n G[n][v] h_n         (dW = G^T H)
//
// G is produced chunk by chunk (at most 32,768 rows at a time, so the rows x
// vocabulary tensor is bounded) by the fused lm-head kernel in its gradient
// mode, which recomputes the logits tile by tile and stores G chunk-major
// (8 vocabulary entries of a row, then the same 8 of the next row).  The two
// contractions are plain bf16 GEMMs on the same 256 x 256 MFMA tile as the
// forward kernel (gemm_kernel below), each operand read as stored: G in
// either role, W, and the chunk's hidden rows (gathered into a dense block,
// chunk-major along the row index, by gather_rows_cm_kernel).  Operands whose
// stored rows run along the contracted index (W in dH, G in dW) are staged in
// LDS as stored and turned into MFMA fragments by gfx950's transposing LDS
// reads, so nothing large is transposed in memory.  dH is
// split along the vocabulary when it has too few tiles for the chip, and its
// partial sums are added in a fixed order (splitk_scatter_kernel): the whole
// pass is deterministic.
#include "tile_common.h"

namespace hdl {
namespace {

using namespace tile;

constexpr int kGemmSliceK = 8 * kChunks;   // bf16 elements per K-slice
// K-row operand tiles: a K-slice is 64 stored rows of kTileV bf16 (512 bytes,
// 32 chunks of 16 bytes), 32 KB like every operand stage.
constexpr int kKRowChunks = kTileV * 2 / 16;
static_assert(kGemmSliceK * kKRowChunks == kSlots, "K-row slice must fill one operand stage");
static_assert(2 * kKRowChunks == 64, "one DMA block must hold two stored K rows");

typedef short i16x4_t __attribute__((ext_vector_type(4)));

// XOR pattern of the 16-byte chunks of K-row r.  A transposing read by 16
// lanes touches 32 bytes (two chunks) in each of 4 consecutive rows, and 32
// lanes touch 64 bytes in each of those rows; with 512-byte rows every row
// starts on the same bank, so the pattern must give the 4 rows distinct
// 32-byte bank positions within 128 bytes (bits 1-2 of the chunk index) and
// distinct 64-byte positions within 256 bytes (bits 2-3): (j0, j1) = the two
// low bits of r map to bits (2, 1) and bit 3 takes j0 ^ j1.
__device__ __forceinline__ int krow_xor(int r) {
  const int j0 = r & 1, j1 = (r >> 1) & 1;
  return 2 * j1 + 4 * j0 + 8 * (j0 ^ j1);
}

// Chunk-major tiles in the K-row role: stored row r of the slice in chunk
// c sits at slot c * 64 + (r ^ cm_xor(c)).  A transposing read by 32 lanes
// touches 4 consecutive rows (64 bytes) in each of 4 consecutive chunks,
// which start 1 KB apart (same bank): XOR-ing bits 2-3 of the row with the
// chunk's two low bits puts the 4 segments in distinct 64-byte bank ranges
// (and any 2 consecutive chunks in distinct 32-byte ranges of 128 bytes).
__device__ __forceinline__ int cm_xor(int c) { return 4 * (c & 3); }

// Per-lane DMA and fragment addressing of one operand of the tile, by
// stored layout (GemmArgs::a_layout / b_layout):
//   kLayoutKRow   X(i, k) at k * ld + i: row k holds the tile's columns;
//                 LDS slot of (row r, chunk c) = r * 32 + (c ^ krow_xor(r)).
//   kLayoutCmRow  X(i, k) at ((k / 8) * ld + i) * 8 + k % 8 (chunk-major,
//                 K split into chunks); LDS slot of (row i, chunk c) =
//                 c * 256 + i, read with plain 16-byte loads.
//   kLayoutCmKRow X(i, k) at ((i / 8) * ld + k) * 8 + i % 8 (chunk-major,
//                 the tile's columns split into chunks); LDS slot as for
//                 cm_xor above, read with transposing loads.
// In every case one DMA block of 64 lanes fills 64 consecutive LDS slots,
// and a K-slice fills 2048 slots (32 KB).
template <int LAY>
struct Operand {
  uint32_t off[kBlocksPerWave];   // per-lane byte offset of each DMA block (kLayoutCmRow: final)
  uint64_t tile;                  // uniform base of the tile
  int64_t ld;                     // elements between stored rows (chunk-major: rows per chunk plane)
  int64_t krows;                  // stored K rows (K-row roles)
  uint32_t frag_lo[4], frag_hi[4];   // transposing reads: per-lane LDS byte offset of each 32-wide block

  // t0: first column (tile index) of the tile; rows / cols: valid extent
  // of that index (row role) or stored columns (K-row roles; a multiple of 8).
  __device__ __forceinline__ void init(const void* ptr, int64_t ld_, int64_t t0, int64_t rows, int64_t cols,
                                       int64_t krows_, int wave, int lane, int nblk, int blk0) {
    ld = ld_;
    krows = krows_;
    const int a = lane & 15, gi = (lane >> 4) & 1, half = lane >> 5;
    if (LAY == kLayoutKRow) {
      tile = reinterpret_cast<uint64_t>(ptr) + static_cast<uint64_t>(t0 * 2);
#pragma unroll
      for (int i = 0; i < kBlocksPerWave; ++i) {
        const int r = 2 * (wave * kBlocksPerWave + i) + (lane >> 5);   // stored row within the slice
        const int chunk = (lane & 31) ^ krow_xor(r);
        int64_t c = t0 + 8 * chunk;
        c = c < cols - 8 ? c : cols - 8;
        off[i] = static_cast<uint32_t>((c - t0) * 2);   // + row * ld * 2 at issue
      }
      // lane l of a 16-lane group reads stored row 4 j + l / 4 (j: which half
      // of the 8 K values) at columns 4 (l % 4) .. +3 of its group's 16
      // columns; lanes 32-63 take K values 8-15 of the sub-step
#pragma unroll
      for (int bk = 0; bk < nblk; ++bk) {
        const int c = (((blk0 + bk * 32) >> 3) + 2 * gi + ((a & 3) >> 1)) ^ krow_xor(a >> 2);
        frag_lo[bk] = static_cast<uint32_t>(((a >> 2) + 8 * half) * (kKRowChunks * 16) + c * 16 + (a & 1) * 8);
        frag_hi[bk] = frag_lo[bk] + 4 * kKRowChunks * 16;
      }
    } else if (LAY == kLayoutCmRow) {
      tile = reinterpret_cast<uint64_t>(ptr) + static_cast<uint64_t>(t0 * 16);
#pragma unroll
      for (int i = 0; i < kBlocksPerWave; ++i) {
        // block wave*4 + i = slots (wave * 4 + i) * 64 ..: chunk `wave`, rows i * 64 + lane
        int64_t row = t0 + i * 64 + lane;
        row = row < rows ? row : rows - 1;
        off[i] = static_cast<uint32_t>((wave * ld + (row - t0)) * 16);
      }
    } else {
      const int64_t c0 = t0 / 8;
      tile = reinterpret_cast<uint64_t>(ptr) + static_cast<uint64_t>(c0 * ld * 16);
#pragma unroll
      for (int i = 0; i < kBlocksPerWave; ++i) {
        // block wave*4 + i = chunk c = wave * 4 + i, slot lane = row lane ^ cm_xor(c)
        int64_t c = c0 + wave * kBlocksPerWave + i;
        c = c < cols / 8 - 1 ? c : cols / 8 - 1;
        off[i] = static_cast<uint32_t>((c - c0) * ld * 16);   // + row * 16 at issue
      }
#pragma unroll
      for (int bk = 0; bk < nblk; ++bk) {
        const int c = ((blk0 + bk * 32) >> 3) + 2 * gi + ((a & 3) >> 1);
        const int r = 8 * half + (a >> 2);   // bits 2-3: 0 / half; + 4 j for the second read
        frag_lo[bk] = static_cast<uint32_t>((c * 64 + (r ^ cm_xor(c))) * 16 + (a & 1) * 8);
        frag_hi[bk] = static_cast<uint32_t>((c * 64 + ((r + 4) ^ cm_xor(c))) * 16 + (a & 1) * 8);
      }
    }
  }
  // uniform address of the K-slice starting at element k
  __device__ __forceinline__ uint64_t slice_base(int64_t k) const {
    if (LAY == kLayoutKRow) return tile + static_cast<uint64_t>(k * ld * 2);
    if (LAY == kLayoutCmRow) return tile + static_cast<uint64_t>((k / 8) * ld * 16);
    return tile + static_cast<uint64_t>(k * 16);
  }
  // last stored row of the K-slice starting at element k, relative to it
  // (>= 0: every slice starts at a stored row; 63 when the slice is whole)
  __device__ __forceinline__ int slice_rmax(int64_t k) const {
    const int64_t r = krows - 1 - k;
    return r < kGemmSliceK - 1 ? static_cast<int>(r) : kGemmSliceK - 1;
  }
  // per-lane offset of DMA block i of a K-slice whose last stored row is rmax
  __device__ __forceinline__ uint32_t block_off(int i, int rmax, int wave, int lane) const {
    if (LAY == kLayoutCmRow) return off[i];
    const int r = LAY == kLayoutKRow ? 2 * (wave * kBlocksPerWave + i) + (lane >> 5) : lane ^ (4 * i);
    const int rr = r < rmax ? r : rmax;
    return LAY == kLayoutKRow ? static_cast<uint32_t>(rr) * static_cast<uint32_t>(ld * 2) + off[i]
                              : static_cast<uint32_t>(rr) * 16u + off[i];
  }
  // the 16-byte MFMA fragment of 32-wide block bk (first column mbase of the
  // tile) for sub-step kk: 8 consecutive K values of column mbase + lane % 32
  __device__ __forceinline__ uint4 frag(const uint4* stage_op, int bk, int mbase, int kk, int lane) const {
    if (LAY == kLayoutCmRow) return stage_op[(kk * 2 + (lane >> 5)) * kTileV + mbase + (lane & 31)];
    typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
    const char __attribute__((address_space(3)))* base =
        (const char __attribute__((address_space(3)))*)(
            (const __attribute__((address_space(3))) uint4*)stage_op);
    // sub-step kk covers stored rows 16 kk .. 16 kk + 15 (untouched by the XOR patterns)
    const uint32_t ks = static_cast<uint32_t>(kk * 16 * (LAY == kLayoutKRow ? kKRowChunks * 16 : 16));
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + frag_lo[bk] + ks));
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + frag_hi[bk] + ks));
    const uint2 l = __builtin_bit_cast(uint2, lo), h = __builtin_bit_cast(uint2, hi);
    return make_uint4(l.x, l.y, h.x, h.y);
  }
};

// C[s][m][n] (=|+=) sum_k A(m, k) B(n, k) over the K range of split s, for
// one 256 x 256 tile of C per workgroup.  Same data path as the fused
// kernel: K-slices of 64 K values stream into a 2-stage LDS ring by direct
// DMA; eight waves each own 128 x 64 of the tile as 4 x 2 MFMA blocks.
// LA / LB: stored layouts of A and B (see Operand).
template <int LA, int LB>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(GemmArgs p) {
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
    Operand<LA> A;
    Operand<LB> B;
    A.init(p.a, p.lda, tm * kTileV, m_valid, p.a_cols, p.a_krows, wave, lane, 4, wm * 128);
    B.init(p.b, p.ldb, tn * kTileN, p.n, p.b_cols, p.b_krows, wave, lane, kNB, wn * kWaveN);
    const uint32_t lds_base = static_cast<uint32_t>(
        reinterpret_cast<size_t>((__attribute__((address_space(3))) uint4*)(&lds[0][0][0])));
    auto lds_addr = [&](int stage, int op, int block) -> uint32_t {
      return __builtin_amdgcn_readfirstlane(
          lds_base + static_cast<uint32_t>(((stage * 2 + op) * kSlots + block * 64) * 16));
    };
    int issue_stage = 0, a_rmax = 0, b_rmax = 0;
    uint64_t a_slice = 0, b_slice = 0;
    auto prep_issue = [&](int slice) {
      issue_stage = slice % kStages;
      const int64_t k = k0 + static_cast<int64_t>(slice) * kGemmSliceK;
      a_slice = A.slice_base(k);
      b_slice = B.slice_base(k);
      if (LA != kLayoutCmRow) a_rmax = A.slice_rmax(k);
      if (LB != kLayoutCmRow) b_rmax = B.slice_rmax(k);
    };
    auto issue_one = [&](int jj) {
      const int i = jj % kBlocksPerWave;
      if (jj < kBlocksPerWave)
        dma16(a_slice, A.block_off(i, a_rmax, wave, lane), lds_addr(issue_stage, 0, wave * kBlocksPerWave + i));
      else
        dma16(b_slice, B.block_off(i, b_rmax, wave, lane), lds_addr(issue_stage, 1, wave * kBlocksPerWave + i));
    };
    auto load_frags = [&](int slice, int kk, uint4 (&fa)[4], uint4 (&fb)[kNB]) {
      const int stage = slice % kStages;
#pragma unroll
      for (int bm = 0; bm < 4; ++bm) fa[bm] = A.frag(lds[stage][0], bm, wm * 128 + bm * 32, kk, lane);
#pragma unroll
      for (int bn = 0; bn < kNB; ++bn) fb[bn] = B.frag(lds[stage][1], bn, wn * kWaveN + bn * 32, kk, lane);
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

// The chunk's scored hidden rows, chunk-major along the row index (the dense
// B operand of dW = G^T H with K = rows, read with plain 16-byte loads):
// out[(e / 8) * d + j][e % 8] = in[map[e]][j] for the e < n scored rows,
// zeros for n <= e < round_up(n, 64).  Each thread moves an 8 x 8 block
// (8 rows x 8 columns): eight 16-byte row reads, eight 16-byte writes of one
// column's 8 rows each.
__global__ __launch_bounds__(256) void gather_rows_cm_kernel(const uint16_t* __restrict__ in, int64_t ld_in,
                                                             const int32_t* __restrict__ map,
                                                             const int32_t* __restrict__ dyn, int64_t dyn_base,
                                                             int64_t cap, int64_t d, uint16_t* __restrict__ out) {
  int64_t n = *dyn - dyn_base;
  n = n < 0 ? 0 : (n > cap ? cap : n);
  int64_t n_pad = (n + 63) / 64 * 64;
  n_pad = n_pad < cap ? n_pad : cap;
  const int64_t e0 = static_cast<int64_t>(blockIdx.y) * 8;
  if (e0 >= n_pad) return;
  const int64_t j = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (j >= d) return;
  uint4 rows[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    rows[r] = make_uint4(0, 0, 0, 0);
    if (e0 + r < n) rows[r] = *reinterpret_cast<const uint4*>(in + static_cast<int64_t>(map[e0 + r]) * ld_in + j);
  }
  // element (r, c): 16-bit half c % 2 (low half first) of 32-bit word c / 2 of row r
  auto elem = [&](int r, int c) -> uint32_t {
    const uint32_t w = (c >> 1) == 0 ? rows[r].x : (c >> 1) == 1 ? rows[r].y : (c >> 1) == 2 ? rows[r].z : rows[r].w;
    return (c & 1) ? (w >> 16) : (w & 0xffffu);
  };
  uint4* dst = reinterpret_cast<uint4*>(out + ((e0 / 8) * d + j) * 8);
#pragma unroll
  for (int c = 0; c < 8; ++c)
    dst[c] = make_uint4(elem(0, c) | (elem(1, c) << 16), elem(2, c) | (elem(3, c) << 16),
                        elem(4, c) | (elem(5, c) << 16), elem(6, c) | (elem(7, c) << 16));
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

hipError_t launch_gemm(const GemmArgs& a, hipStream_t stream) {
  const int64_t per_group = a.gm * a.gn;
  const int64_t groups = ((a.tiles_m + a.gm - 1) / a.gm) * ((a.tiles_n + a.gn - 1) / a.gn) * a.splits;
  const int64_t grid = (groups + kNumXcd - 1) / kNumXcd * kNumXcd * per_group;
  if (grid <= 0) return hipSuccess;
  const dim3 g(static_cast<unsigned>(grid)), blk(kThreads);
  if (a.a_layout == kLayoutCmRow && a.b_layout == kLayoutKRow)
    hipLaunchKernelGGL((gemm_kernel<kLayoutCmRow, kLayoutKRow>), g, blk, 0, stream, a);
  else if (a.a_layout == kLayoutCmKRow && a.b_layout == kLayoutCmRow)
    hipLaunchKernelGGL((gemm_kernel<kLayoutCmKRow, kLayoutCmRow>), g, blk, 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_gather_rows_cm(const uint16_t* in, int64_t ld_in, const int32_t* map, const int32_t* dyn,
                                 int64_t dyn_base, int64_t cap, int64_t d, uint16_t* out, hipStream_t stream) {
  const int64_t gx = (d / 8 + 255) / 256;
  const int64_t gy = (cap + 7) / 8;
  if (gx <= 0 || gy <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_cm_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy)), dim3(256), 0,
                     stream, in, ld_in, map, dyn, dyn_base, cap, d, out);
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
