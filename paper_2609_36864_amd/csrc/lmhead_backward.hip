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
static_assert(kKSteps * 32 == kGemmSliceK, "a K-slice is two K-steps of 32");

typedef short i16x4_t __attribute__((ext_vector_type(4)));

// Operands whose stored rows run along K (W in dH, G in dW) are turned into
// MFMA fragments by gfx950's transposing read ds_read_b64_tr_b16: within
// each 16-lane group, lane i receives element i mod 4 of the 8-byte pieces
// addressed by lanes i/4, i/4 + 4, i/4 + 8 and i/4 + 12.  For the fragment
// of 16 columns m0 .. m0+15 at K-step ks, lane a of lane group g addresses
// stored K row 32 ks + 8 frag_chunk(g) + 4 j + a/4 at columns
// m0 + 4 (a mod 4) .. +3 (read j = 0, 1): lane a then holds column m0 + a,
// K values 8 frag_chunk(g) + 4 j + 0..3 of the K-step, as the MFMA wants.
// A read touches 4 rows x 32 bytes per lane group; the groups read rows
// whose bits 3-4 are (0, 0), (0, 1), (1, 0), (1, 1) (g = 0, 1, 2, 3).

// XOR pattern of the 16-byte chunks of K row r (512-byte rows, so every
// row starts on the same bank): the 32-byte pieces that 4 rows x 4 groups
// read must fall in distinct 32-byte bank positions of 128 bytes (one
// group) and of 256 bytes (two groups, whichever two the LDS serves
// together): bits 1-3 of the chunk take r mod 4 and bit 3 ^ bit 4 of r.
__device__ __forceinline__ int krow_xor(int r) { return 2 * ((r & 3) | ((((r >> 3) ^ (r >> 4)) & 1) << 2)); }

// Chunk-major tiles in the K-row role: stored row r of the slice in chunk c
// sits at slot c * 64 + (r ^ cm_xor(c, r)) (1 KB per chunk, so chunks start
// on the same bank).  A lane group reads 4 rows of 2 chunks (c even, c + 1):
// bit 2 of the row takes c mod 2, bit 3 takes bit 4 of the row, so 8 pieces
// of one group and 16 of any two groups land in distinct 16-byte positions.
// Only bits 2-3 change, so the pattern is its own inverse.
__device__ __forceinline__ int cm_xor(int c, int r) { return (4 * (c & 1)) ^ (8 * ((r >> 4) & 1)); }

// Per-lane DMA and fragment addressing of one operand of the tile, by
// stored layout (GemmArgs::a_layout / b_layout):
//   kLayoutKRow   X(i, k) at k * ld + i: row k holds the tile's columns;
//                 LDS slot of (K row r, chunk c) = r * 32 + (c ^ krow_xor(r)).
//   kLayoutCmRow  X(i, k) at ((k / 8) * ld + i) * 8 + k % 8 (chunk-major,
//                 K split into chunks); LDS slot of (row i, chunk c) =
//                 c * 256 + i, so that each DMA block reads 1 KB contiguous
//                 (with the fused kernel's row-major tiles a DMA block would
//                 read 8 runs of 128 bytes from 8 chunk planes a power of
//                 two apart, which ran the GEMMs 13 % slower); read with
//                 plain 16-byte loads.  Lane groups g and g + 2 (served
//                 together) read chunks 2 m and 2 m + 1 of the same rows,
//                 4 KB apart: 0 bank conflicts measured, as for the 32-row
//                 fragments of the same layout.
//   kLayoutCmKRow X(i, k) at ((i / 8) * ld + k) * 8 + i % 8 (chunk-major,
//                 the tile's columns split into chunks); LDS slot as for
//                 cm_xor above, read with transposing loads.
// In every case one DMA block of 64 lanes fills 64 consecutive LDS slots,
// and a K-slice fills 2048 slots (32 KB).  NBLK: the operand's 16-column
// fragments per wave (kVB as A, kTB as B).
template <int LAY, int NBLK>
struct Operand {
  static constexpr int kFragOffs = LAY == kLayoutKRow ? NBLK : 2;
  uint32_t off[kBlocksPerWave];   // per-lane byte offset of each DMA block (kLayoutCmRow: final)
  uint64_t tile;                  // uniform base of the tile
  int64_t ld;                     // elements between stored rows (chunk-major: rows per chunk plane)
  int64_t krows;                  // stored K rows (K-row roles)
  // per-lane LDS offsets of the fragment reads: kLayoutCmRow: 16-byte slot
  // per K-step; kLayoutKRow: byte offset per fragment; kLayoutCmKRow: byte
  // offset per read j
  uint32_t frag_off[kFragOffs];

  // t0: first column (tile index) of the tile; rows / cols: valid extent
  // of that index (row role) or stored columns (K-row roles; a multiple of
  // 8); fbase: the wave's first column within the tile.
  __device__ __forceinline__ void init(const void* ptr, int64_t ld_, int64_t t0, int64_t rows, int64_t cols,
                                       int64_t krows_, int wave, int lane, int fbase) {
    ld = ld_;
    krows = krows_;
    const int a = lane & 15, grp = lane >> 4;
    const int r0 = 8 * frag_chunk(grp) + (a >> 2);   // fragment K row of read j = 0 at K-step 0
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
      // krow_xor of the rows read depends on bits 0, 1, 3, 4 only: the same
      // for both reads and both K-steps
#pragma unroll
      for (int b = 0; b < NBLK; ++b) {
        const int c = ((fbase + 16 * b) >> 3) + ((a & 3) >> 1);
        frag_off[b] = static_cast<uint32_t>((r0 * kKRowChunks + (c ^ krow_xor(r0))) * 16 + (a & 1) * 8);
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
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        frag_off[ks] = static_cast<uint32_t>((4 * ks + frag_chunk(grp)) * kTileV + fbase + a);
    } else {
      const int64_t c0 = t0 / 8;
      tile = reinterpret_cast<uint64_t>(ptr) + static_cast<uint64_t>(c0 * ld * 16);
#pragma unroll
      for (int i = 0; i < kBlocksPerWave; ++i) {
        // block wave * 4 + i = chunk c = wave * 4 + i, slot lane = row lane ^ cm_xor(c, lane)
        int64_t c = c0 + wave * kBlocksPerWave + i;
        c = c < cols / 8 - 1 ? c : cols / 8 - 1;
        off[i] = static_cast<uint32_t>((c - c0) * ld * 16);   // + row * 16 at issue
      }
      // chunk of the lane's columns: fbase / 8 + 2 b + (a mod 4) / 2, whose
      // parity is that of (a mod 4) / 2; bit 4 of the rows read is
      // frag_chunk(g) / 2 for both reads and both K-steps
      const int cpar = (a & 3) >> 1;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int r = r0 + 4 * j;
        frag_off[j] = static_cast<uint32_t>(((fbase >> 3) + cpar) * 64 * 16 + (r ^ cm_xor(cpar, r)) * 16 +
                                            (a & 1) * 8);
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
    const int r = LAY == kLayoutKRow ? 2 * (wave * kBlocksPerWave + i) + (lane >> 5)
                                     : lane ^ cm_xor(wave * kBlocksPerWave + i, lane);
    const int rr = r < rmax ? r : rmax;
    return LAY == kLayoutKRow ? static_cast<uint32_t>(rr) * static_cast<uint32_t>(ld * 2) + off[i]
                              : static_cast<uint32_t>(rr) * 16u + off[i];
  }
  // The MFMA fragment of 16-column block b of the wave at K-step ks.
  __device__ __forceinline__ uint4 frag(const uint4* stage_op, int b, int ks) const {
    if (LAY == kLayoutCmRow) return stage_op[frag_off[ks] + b * 16];
    typedef __attribute__((address_space(3))) char lds_char;
    const lds_char* base = (const lds_char*)((const __attribute__((address_space(3))) uint4*)stage_op);
    typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
    uint32_t o0, o1;
    if (LAY == kLayoutKRow) {
      // K-step ks: rows + 32 ks; read 1: rows + 4
      o0 = frag_off[b] + ks * 32 * kKRowChunks * 16;
      o1 = o0 + 4 * kKRowChunks * 16;
    } else {
      // fragment b: chunks + 2 b; K-step ks: rows + 32 ks
      o0 = frag_off[0] + b * 2 * 64 * 16 + ks * 32 * 16;
      o1 = frag_off[1] + b * 2 * 64 * 16 + ks * 32 * 16;
    }
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + o0));
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + o1));
    const uint2 l = __builtin_bit_cast(uint2, lo), h = __builtin_bit_cast(uint2, hi);
    return make_uint4(l.x, l.y, h.x, h.y);
  }
};

// C[s][m][n] (=|+=) sum_k A(m, k) B(n, k) over the K range of split s, for
// one 256 x 256 tile of C per workgroup.  Same data path as the fused
// kernel: K-slices of 64 K values stream into a 2-stage LDS ring by direct
// DMA; eight waves each own 128 x 64 of the tile as 8 x 4 blocks of
// v_mfma_f32_16x16x32_bf16, with the fused kernel's quarter schedule.
// LA / LB: stored layouts of A and B (see Operand).
template <int LA, int LB>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(GemmArgs p) {
  using M = Mma16<true>;
  __shared__ uint4 lds[kStages][2][kSlots];   // [stage][0 = A, 1 = B]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int r16 = lane & 15;
  const int grp = lane >> 4;

  // ---- work item: XCD-aware (m-tile, n-tile, split) ----------------------
  // The j-th workgroup of an XCD belongs to launch group j / 32 of that XCD;
  // a group is gm x gn tiles of one split, sharing A and B rows through L2.
  // Consecutive groups (which run at the same time on neighbouring XCDs)
  // take the n-groups of one m-group first, so the XCDs that read the same
  // rows of A (the large logit gradient) read them together and all but the
  // first find them in the memory-side cache (3.7 % faster at c2 than
  // m-groups first).
  const int64_t b = blockIdx.x;
  const int64_t xcd = b % kNumXcd;
  const int64_t j = b / kNumXcd;
  const int64_t grp_id = (j / (p.gm * p.gn)) * kNumXcd + xcd;
  const int64_t loc = j % (p.gm * p.gn);
  const int64_t n_gm = (p.tiles_m + p.gm - 1) / p.gm;
  const int64_t n_gn = (p.tiles_n + p.gn - 1) / p.gn;
  // (the runtime divisions run on the vector ALU; readfirstlane puts the
  // wave-uniform results back in scalar registers for the DMA base)
  const int64_t split = __builtin_amdgcn_readfirstlane(static_cast<int>(grp_id / (n_gm * n_gn)));
  const int64_t rem = grp_id % (n_gm * n_gn);
  const int64_t tm = __builtin_amdgcn_readfirstlane(static_cast<int>((rem / n_gn) * p.gm + loc % p.gm));
  const int64_t tn = __builtin_amdgcn_readfirstlane(static_cast<int>((rem % n_gn) * p.gn + loc / p.gm));
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

  f32x4_t acc[kVB][kTB];
#pragma unroll
  for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[bm][bn][q] = 0.f;

  if (n_iter > 0) {
    Operand<LA, kVB> A;
    Operand<LB, kTB> B;
    A.init(p.a, p.lda, tm * kTileV, m_valid, p.a_cols, p.a_krows, wave, lane, wm * 16 * kVB);
    B.init(p.b, p.ldb, tn * kTileN, p.n, p.b_cols, p.b_krows, wave, lane, wn * kWaveN);
    const uint32_t lds_base = static_cast<uint32_t>(
        reinterpret_cast<size_t>((__attribute__((address_space(3))) uint4*)(&lds[0][0][0])));
    auto lds_addr = [&](int stage, int op, int block) -> uint32_t {
      return __builtin_amdgcn_readfirstlane(
          lds_base + static_cast<uint32_t>(((stage * 2 + op) * kSlots + block * 64) * 16));
    };
    int issue_stage = 0, a_rmax = 0, b_rmax = 0;
    uint64_t a_slice = 0, b_slice = 0;
    // slot: the ring position (its stage); slice: the data fetched into it
    // (they differ only for the copies of the last slice past the end)
    auto prep_issue = [&](int slot, int slice) {
      issue_stage = slot % kStages;
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
    // the two A fragments (M blocks 2 pr, 2 pr + 1) of quarter pr of K-step ks
    auto load_a = [&](int slice, int ks, int pr, uint4 (&dst)[2]) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) dst[jj] = A.frag(lds[slice % kStages][0], 2 * pr + jj, ks);
    };
    auto load_b = [&](int slice, int ks, int bn, uint4& dst) { dst = B.frag(lds[slice % kStages][1], bn, ks); };
    auto quarter_mfma = [&](const uint4 (&fa_)[2], const uint4 (&fb_)[kTB], int pr) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int i = 0; i < kTB; ++i) M::run(fa_[jj], fb_[snake(jj, i)], acc[2 * pr + jj][snake(jj, i)]);
    };

    const int n_pre = n_iter < kStages ? n_iter : kStages;
    for (int sl = 0; sl < n_pre; ++sl) {
      prep_issue(sl, sl);
#pragma unroll
      for (int jj = 0; jj < kDmaPerSlice; ++jj) issue_one(jj);
    }
    wait_dma(n_pre - 1);
    raw_barrier();

    // The fused kernel's schedule: a K-slice is 2 K-steps x 4 quarters;
    // each quarter first reads what the next one needs (the next two A
    // fragments, and during K-step 0 one B fragment of K-step 1), and the
    // slice's last quarter crosses the barrier into the next slice and
    // issues the DMA of the slice after next between its MFMAs.
    uint4 fa[2][2], fb[2][kTB];
    load_a(0, 0, 0, fa[0]);
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn) load_b(0, 0, bn, fb[0][bn]);
    for (int it = 0; it < n_iter; ++it) {
#pragma unroll
      for (int pr = 0; pr < 4; ++pr) {
        if (pr < 3) load_a(it, 0, pr + 1, fa[(pr + 1) & 1]);
        else load_a(it, 1, 0, fa[0]);
        load_b(it, 1, pr, fb[1][pr]);
        __builtin_amdgcn_sched_barrier(0);
        quarter_mfma(fa[pr & 1], fb[0], pr);
      }
#pragma unroll
      for (int pr = 0; pr < 3; ++pr) {
        load_a(it, 1, pr + 1, fa[(pr + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        quarter_mfma(fa[pr & 1], fb[1], pr);
      }
      // Every read of slice `it` is issued: wait for slice it+1, then refill
      // this slice's stage with slice it+kStages (past the end: a copy of
      // the last slice, into a stage nothing reads any more; the fragment
      // reads of the call's last step fetch stale, unused LDS).
      wait_dma(kStages - 2);
      raw_barrier();
      prep_issue(it + kStages, it + kStages < n_iter ? it + kStages : n_iter - 1);
      load_a(it + 1, 0, 0, fa[0]);
#pragma unroll
      for (int bn = 0; bn < kTB; ++bn) load_b(it + 1, 0, bn, fb[0][bn]);
      __builtin_amdgcn_sched_barrier(0);
      constexpr int kM = 2 * kTB;   // MFMAs per quarter, one DMA after each
      static_assert(kM == kDmaPerSlice, "one DMA per MFMA of the last quarter");
#pragma unroll
      for (int q = 0; q < kM; ++q) {
        M::run(fa[1][q / kTB], fb[1][snake(q / kTB, q % kTB)], acc[6 + q / kTB][snake(q / kTB, q % kTB)]);
        issue_one(q);
      }
    }
    wait_vmcnt<0>();
  }

  // ---- store: in each block, lane l holds column l mod 16 of rows
  // 4 (l div 16) + q, so one store instruction covers 4 rows x 64 bytes ----
  float* cbase = p.c + split * p.c_split_stride;
#pragma unroll
  for (int bn = 0; bn < kTB; ++bn) {
    const int64_t n = tn * kTileN + wn * kWaveN + bn * 16 + r16;
    if (n >= p.n) continue;
#pragma unroll
    for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t m = tm * kTileV + wm * 16 * kVB + bm * 16 + 4 * grp + q;
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
