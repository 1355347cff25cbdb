// Fused lm-head log-probability kernel for gfx950 (MI355X).
//
// For every scored row n (a final hidden state h_n) and its sampled token y_n
// it computes, in one pass over the vocabulary projection W [V, d]:
//
//     z_n[v] = sum_j W[v, j] h_n[j]            (lm-head contraction, Eq. 1)
//     lse_n  = log sum_v exp(z_n[v])           (softmax normaliser)
//     log p_n(y_n) = z_n[y_n] - lse_n          (sampled-token log-likelihood)
//
// without ever storing z.  The vocabulary is cut into chunks; each work item
// (row tile x chunk) leaves a partial (max, sum of exp, captured z_y) per row,
// and merge_kernel combines the chunk partials in a fixed order.
//
// Work item: 256 vocabulary rows x 256 token rows per V-tile, looping over
// the V-tiles of one chunk.  Eight waves per workgroup (two per SIMD, so one
// wave's memory and epilogue work overlaps the other's MFMAs), each owning
// 128 vocab x 64 tokens as a 4x2 grid of 32x32 MFMA blocks with fp32
// accumulators (HDL_WAVES=4 selects one wave per SIMD with 128 x 128 each).
// W is the MFMA "A" operand (vocabulary on the M axis) and the hidden states
// are the "B" operand (tokens on the N axis), so each lane's accumulators
// hold one token column and 64 vocabulary rows: the online max / sum-of-exp
// update of a V-tile is entirely lane-local, and lanes and waves are merged
// only once per work item.
//
// Operands stream through LDS in K-slices of 128 bytes per row (64 bf16 or
// 32 fp32; HDL_LDS_CHUNKS=4 selects 64-byte slices) through a ring of
// HDL_LDS_STAGES stages (default 2, 128 KB): the next slice is in flight
// (global -> LDS DMA, no VGPR staging) while slice i is multiplied.  16-byte
// chunks are XOR swizzled so that the 32-row fragment reads are bank-conflict
// free.  The DMA is issued from inline assembly (wave-uniform 64-bit base +
// per-lane 32-bit offset) and waited for with explicit vmcnt counts: the
// compiler cannot see that a DMA into one stage does not alias the reads of
// another, and would otherwise wait for every outstanding DMA before each LDS
// read.
//
// Both operands are contiguous in K.  MFMA lane l takes row (l mod 32) and a
// 16-byte K fragment chosen by (l div 32); A and B fragments use the same K
// assignment, so the contraction is exact whatever order the hardware sums
// the K values in.
#include "hdl_internal.h"

#include <type_traits>

namespace hdl {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

#ifndef HDL_WAVES
#define HDL_WAVES 8
#endif
constexpr int kWaves = HDL_WAVES;                   // 4: one wave per SIMD; 8: two
constexpr int kThreads = 64 * kWaves;
constexpr int kNB = kWaves == 4 ? 4 : 2;            // 32-token MFMA blocks per wave
constexpr int kWaveN = 32 * kNB;                    // tokens per wave (128 or 64)
#ifndef HDL_LDS_CHUNKS
#define HDL_LDS_CHUNKS 8
#endif
#ifndef HDL_LDS_STAGES
#define HDL_LDS_STAGES 2
#endif
constexpr int kChunks = HDL_LDS_CHUNKS;             // 16-byte chunks per LDS row per stage
constexpr int kStages = HDL_LDS_STAGES;             // LDS ring depth (K-slices)
constexpr int kSlots = kTileV * kChunks;            // uint4 slots per operand per stage
constexpr int kBlockRows = 64 / kChunks;            // rows per 1 KB DMA block
constexpr int kBlocksPerWave = kTileV / kBlockRows / kWaves;   // DMA blocks per operand per wave
constexpr int kDmaPerSlice = 2 * kBlocksPerWave;    // DMA instructions per lane per slice
constexpr int kSub = kChunks / 2;                   // MFMA sub-steps per slice
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

static_assert(kTileV == kTileN, "square workgroup tile assumed");
static_assert(kWaves == 4 || kWaves == 8, "4 or 8 waves");
static_assert(kChunks == 4 || kChunks == 8, "64- or 128-byte K-slices");
static_assert(kStages * 2 * kSlots * 16 <= 160 * 1024, "LDS ring exceeds 160 KB");
static_assert(kDmaPerSlice * (kStages - 1) <= 63, "vmcnt range");

#ifndef HDL_SWZ
#define HDL_SWZ 1
#endif
// XOR pattern of a row: the rows of one 32-row fragment read must land in
// distinct 16-byte bank groups whether the LDS serves 8 or 16 lanes of a
// ds_read_b128 per cycle.  With 128-byte rows, (row & 7) ^ ((row >> 3) & 1)
// does both: 8 consecutive rows get 8 distinct chunks, and rows r and r+8
// (same bank half when two rows share a 256-byte bank line) differ too.
__device__ __forceinline__ int row_xor(int row) {
  if (kChunks == 8) {
    if (HDL_SWZ == 0) return row & 7;
    if (HDL_SWZ == 1) return (row & 7) ^ ((row >> 3) & 1);
    return (row >> 1) & 7;
  }
  if (HDL_SWZ == 0) return (row >> 1) & 3;
  if (HDL_SWZ == 1) return ((row >> 1) & 3) ^ ((row >> 3) & 1);
  return (row >> 2) & 3;
}

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

// Wait until at most `slices` K-slices of this lane's DMA are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_dma(int slices) {
  if (kStages > 3 && slices >= 3) wait_vmcnt<(kStages > 3 ? 3 : 0) * kDmaPerSlice>();
  else if (kStages > 2 && slices >= 2) wait_vmcnt<(kStages > 2 ? 2 : 0) * kDmaPerSlice>();
  else if (slices >= 1) wait_vmcnt<kDmaPerSlice>();
  else wait_vmcnt<0>();
}

// Workgroup barrier without the memory fence __syncthreads() implies (the
// fence would wait for every in-flight DMA).  LDS reads issued before it
// are complete: callers wait lgkmcnt(0) first.
__device__ __forceinline__ void raw_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// One MFMA step over a pair of 16-byte fragments (same K positions in A, B).
template <bool BF16> struct Mma;

template <> struct Mma<true> {
  static constexpr int kElemsPer16B = 8;
  __device__ __forceinline__ static void run(const uint4& a, const uint4& b, f32x16_t& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  }
};

template <> struct Mma<false> {
  static constexpr int kElemsPer16B = 4;
  // Four K=2 steps; lane group g supplies K offset 4g + j in step j, the same
  // for both operands, so the four steps cover the fragment's 8 K values.
  __device__ __forceinline__ static void run(const uint4& a, const uint4& b, f32x16_t& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  }
};

// t of a state, moved from its own max m to a larger max mn:
//   sum exp(z - mn) * (z - mn) log2(e) = f * (t + (m - mn) log2(e) * s),  f = exp(m - mn).
// An empty state (m = -inf, s = t = 0) stays 0.
__device__ __forceinline__ float shift_t(float t, float s, float m, float mn, float f) {
  return (m == mn) ? t : (m == kNegInf ? 0.f : f * __builtin_fmaf((m - mn) * kLog2e, s, t));
}

// Combine two (max m, sum of exp(z - m) s, captured logit z, and for the
// entropy t = sum exp(z - m) * (z - m) log2(e)) states.  t is only
// meaningful when entropy is requested; otherwise it stays 0 and the
// compiler drops it.  t is kept relative to m so that the entropy
// ln s - ln(2) t / s is a sum of two non-negative terms: no cancellation
// against the size of the logits.
__device__ __forceinline__ void combine(float& m, float& s, float& z, float& t, float m2, float s2,
                                        float z2, float t2) {
  const float mn = fmaxf(m, m2);
  const float fa = (m == mn) ? 1.f : fast_exp2((m - mn) * kLog2e);
  const float fb = (m2 == mn) ? 1.f : fast_exp2((m2 - mn) * kLog2e);
  t = shift_t(t, s, m, mn, fa) + shift_t(t2, s2, m2, mn, fb);
  // (an explicit fma: a contractible s * fa + s2 * fb could be fused
  // differently in different instantiations, and log p must not depend on
  // whether the entropy is requested)
  s = __builtin_fmaf(s, fa, s2 * fb);
  m = mn;
  z = fmaxf(z, z2);
}

// Row of the 32x32 accumulator block held in element i of lane l:
// row = 8*(i/4) + 4*(l/32) + (i%4), column = l%32.
__device__ __forceinline__ int acc_row(int i, int half) { return 8 * (i >> 2) + 4 * half + (i & 3); }

// KTAIL: d is not a multiple of the K-slice, so the last slice of every
// row needs zero-filling (a separate instantiation keeps that work out of the
// common case).  ENT: also accumulate sum exp(z - m) * (z - m) for the next-token
// entropy H = ln s - E_p[z - m] (the Entropy localization baseline).
template <bool BF16, bool KTAIL, bool ENT>
__global__ __launch_bounds__(kThreads, 1) void lmhead_logprob_kernel(LmheadArgs p) {
  using M = Mma<BF16>;
  constexpr int kEsz = BF16 ? 2 : 4;
  constexpr int kSliceK = M::kElemsPer16B * kChunks;   // K elements per slice

  __shared__ uint4 lds[kStages][2][kSlots];   // [stage][0 = W, 1 = hidden] = 128 KB

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int wm = wave & 1;      // which 128 vocabulary rows of the tile
  const int wn = wave >> 1;     // which kWaveN token rows of the tile
  const int half = lane >> 5;
  const int col = lane & 31;

  // ---- work item: XCD-aware (row tile, vocabulary chunk) ------------------
  // Workgroups are dealt to the XCDs round-robin.  The j-th workgroup of an
  // XCD belongs to launch group (j / 32) of that XCD; a group is a block of
  // 4 row tiles x 8 vocabulary chunks, so the workgroups resident on one XCD
  // at a time share hidden tiles and W tiles through that XCD's L2.
  const int64_t b = blockIdx.x;
  const int64_t xcd = b % kNumXcd;
  const int64_t j = b / kNumXcd;
  const int64_t grp = (j / (kGroupRT * kGroupCH)) * kNumXcd + xcd;
  const int loc = static_cast<int>(j % (kGroupRT * kGroupCH));
  const int64_t rt = (grp % p.n_grt) * kGroupRT + (loc % kGroupRT);
  const int64_t ch = (grp / p.n_grt) * kGroupCH + (loc / kGroupRT);
  const int64_t n_s = *p.n_scored;
  const int64_t n_rt = (n_s + kTileN - 1) / kTileN;
  if (rt >= n_rt || ch >= p.n_ch) return;

  const int64_t vt0 = ch * p.tpc;
  const int64_t vt1 = (vt0 + p.tpc < p.n_vt) ? vt0 + p.tpc : p.n_vt;
  const int nk = static_cast<int>((p.d + kSliceK - 1) / kSliceK);
  const int n_iter = static_cast<int>(vt1 - vt0) * nk;
  const int64_t d = p.d;
  const int64_t V = p.vocab;

  const char* __restrict__ wbase = static_cast<const char*>(p.w);
  const char* __restrict__ hbase = static_cast<const char*>(p.hidden);

  // ---- this lane's token columns and their sampled tokens ------------------
  int tok[kNB];
#pragma unroll
  for (int bn = 0; bn < kNB; ++bn) {
    int64_t e = rt * kTileN + wn * kWaveN + bn * 32 + col;
    e = e < n_s ? e : n_s - 1;
    tok[bn] = p.tokens[p.rows[e]];
  }

  float run_m[kNB], run_s[kNB], run_z[kNB], run_t[kNB];
#pragma unroll
  for (int bn = 0; bn < kNB; ++bn) { run_m[bn] = kNegInf; run_s[bn] = 0.f; run_z[bn] = kNegInf; run_t[bn] = 0.f; }

  f32x16_t acc[4][kNB];
#pragma unroll
  for (int bm = 0; bm < 4; ++bm)
#pragma unroll
    for (int bn = 0; bn < kNB; ++bn)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[bm][bn][q] = 0.f;

  // ---- direct global -> LDS loads -----------------------------------------
  // A K-slice of one operand tile is made of 1 KB blocks of kBlockRows rows.
  // Wave w fetches blocks w*kBlocksPerWave ..; within a block lane l lands in
  // LDS slot l, i.e. row l/kChunks and physical chunk l%kChunks, so it
  // fetches the logical chunk that the read swizzle maps there.
  const int lrow = lane / kChunks;
  // logical chunk this lane fetches for DMA block i of this wave
  auto dma_chunk = [&](int i) {
    const int row = (wave * kBlocksPerWave + i) * kBlockRows + lrow;
    return (lane % kChunks) ^ row_xor(row);
  };
  constexpr bool k_tail = KTAIL;
  const int64_t row_bytes = d * kEsz;
  // Per-lane byte offsets (row start + 16-byte chunk) of this wave's DMA
  // blocks; a call never spans more than 4 GiB of either operand.
  uint32_t hoff[kBlocksPerWave];
#pragma unroll
  for (int i = 0; i < kBlocksPerWave; ++i) {
    int64_t e = rt * kTileN + wave * (kTileN / kWaves) + i * kBlockRows + lrow;
    e = e < n_s ? e : n_s - 1;
    hoff[i] = static_cast<uint32_t>(static_cast<int64_t>(p.rows[e]) * row_bytes + dma_chunk(i) * 16);
  }
  uint32_t woff[kBlocksPerWave];
  uint64_t wtile = 0;   // address of the current V-tile's first row (uniform)
  auto set_w = [&](int64_t vt) {
    wtile = reinterpret_cast<uint64_t>(wbase) + static_cast<uint64_t>(vt * kTileV * row_bytes);
#pragma unroll
    for (int i = 0; i < kBlocksPerWave; ++i) {
      int64_t v = vt * kTileV + wave * (kTileV / kWaves) + i * kBlockRows + lrow;
      v = v < V ? v : V - 1;
      woff[i] = static_cast<uint32_t>((v - vt * kTileV) * row_bytes + dma_chunk(i) * 16);
    }
  };
  const uint32_t lds_base = static_cast<uint32_t>(
      reinterpret_cast<size_t>((__attribute__((address_space(3))) uint4*)(&lds[0][0][0])));
  auto lds_addr = [&](int stage, int op, int block) -> uint32_t {
    return __builtin_amdgcn_readfirstlane(
        lds_base + static_cast<uint32_t>(((stage * 2 + op) * kSlots + block * 64) * 16));
  };
  // DMA j (0 .. kDmaPerSlice-1) of K-slice `slice`; j < kBlocksPerWave are W
  // blocks, the rest hidden-state blocks.  prep_issue() must run first.
  uint32_t issue_kbytes = 0;
  int issue_stage = 0;
  bool issue_tail = false;
  auto prep_issue = [&](int slice) {
    issue_stage = slice % kStages;
    const int kt = slice % nk;
    if (kt == 0) set_w(vt0 + slice / nk);
    issue_kbytes = static_cast<uint32_t>(kt) * kSliceK * kEsz;
    issue_tail = k_tail && kt == nk - 1;
  };
  auto issue_one = [&](int j, auto tail_tag) {
    constexpr bool kTail = decltype(tail_tag)::value;
    const int i = j % kBlocksPerWave;
    const uint32_t off = j < kBlocksPerWave ? woff[i] : hoff[i];
    const uint64_t base = j < kBlocksPerWave ? wtile : reinterpret_cast<uint64_t>(hbase);
    const uint32_t lds = lds_addr(issue_stage, j < kBlocksPerWave ? 0 : 1, wave * kBlocksPerWave + i);
    if (!kTail) {
      dma16(base + issue_kbytes, off, lds);
    } else {
      // chunks past the end of the row fetch the row start instead (an
      // in-bounds dummy, zeroed after arrival)
      const uint32_t chunk_bytes = dma_chunk(i) * 16;
      const bool in = static_cast<int64_t>(issue_kbytes + chunk_bytes) < row_bytes;
      dma16(base, off - chunk_bytes + (in ? issue_kbytes + chunk_bytes : 0), lds);
    }
  };
  auto issue = [&](int slice) {
    prep_issue(slice);
    if (!issue_tail) {
#pragma unroll
      for (int j = 0; j < kDmaPerSlice; ++j) issue_one(j, std::false_type{});
    } else {
#pragma unroll
      for (int j = 0; j < kDmaPerSlice; ++j) issue_one(j, std::true_type{});
    }
  };

  // On the last K-slice of a row whose length is not a multiple of the
  // slice, clear the chunks past d (between two barriers: the DMA of every
  // wave must have landed before, and no wave may read before it is done).
  auto clear_k_tail = [&](int slice) {
    const int stage = slice % kStages;
    const int kt = slice % nk;
    for (int sidx = tid; sidx < kSlots; sidx += kThreads) {
      const int row = sidx / kChunks;
      const int chunk = (sidx % kChunks) ^ row_xor(row);
      if (static_cast<int64_t>(kt) * kSliceK + chunk * M::kElemsPer16B >= d) {
        lds[stage][0][sidx] = make_uint4(0, 0, 0, 0);
        lds[stage][1][sidx] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto load_frags = [&](int slice, int kk, uint4 (&fa)[4], uint4 (&fb)[kNB]) {
    const int stage = slice % kStages;
#pragma unroll
    for (int bm = 0; bm < 4; ++bm) fa[bm] = lds[stage][0][swz(wm * 128 + bm * 32 + col, kk * 2 + half)];
#pragma unroll
    for (int bn = 0; bn < kNB; ++bn) fb[bn] = lds[stage][1][swz(wn * kWaveN + bn * 32 + col, kk * 2 + half)];
  };

  // Online max / sum-of-exp update of one V-tile, then capture of the
  // sampled token's logit if this lane holds it.  MASKED: the tile runs past
  // the end of the vocabulary and rows >= V are excluded.
  auto epilogue = [&](int64_t vt, auto masked_tag) {
    constexpr bool kMasked = decltype(masked_tag)::value;
    const int64_t vbase = vt * kTileV + wm * 128;   // first vocab row of this wave
#pragma unroll
    for (int bn = 0; bn < kNB; ++bn) {
      if (kMasked) {
#pragma unroll
        for (int bm = 0; bm < 4; ++bm)
#pragma unroll
          for (int q = 0; q < 16; ++q)
            if (vbase + bm * 32 + acc_row(q, half) >= V) acc[bm][bn][q] = kNegInf;
      }
      float mx = acc[0][bn][0];
#pragma unroll
      for (int bm = 0; bm < 4; ++bm)
#pragma unroll
        for (int q = 0; q < 16; ++q) mx = fmaxf(mx, acc[bm][bn][q]);
      const float mnew = fmaxf(run_m[bn], mx);
      if (!kMasked || mnew != kNegInf) {
        const float mb = mnew * kLog2e;
        float s4[4], t4[4];
#pragma unroll
        for (int bm = 0; bm < 4; ++bm) {
          float sacc = 0.f, tacc = 0.f;
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const float zq = acc[bm][bn][q];
            const float zl = __builtin_fmaf(zq, kLog2e, -mb);   // (z - m) log2(e)
            const float e = fast_exp2(zl);
            sacc += e;
            // (masked rows hold -inf and e = 0; their product term is 0)
            if (ENT) tacc = __builtin_fmaf(e, (kMasked && zq == kNegInf) ? 0.f : zl, tacc);
          }
          s4[bm] = sacc;
          t4[bm] = tacc;
        }
        const float tile_sum = (s4[0] + s4[1]) + (s4[2] + s4[3]);
        const float rescale = fast_exp2(__builtin_fmaf(run_m[bn], kLog2e, -mb));
        if (ENT)   // (before run_s changes: shift_t wants the old sum)
          run_t[bn] = shift_t(run_t[bn], run_s[bn], run_m[bn], mnew, rescale) + ((t4[0] + t4[1]) + (t4[2] + t4[3]));
        run_s[bn] = __builtin_fmaf(run_s[bn], rescale, tile_sum);
        run_m[bn] = mnew;
      }
      const int64_t o = static_cast<int64_t>(tok[bn]) - vbase;
      if (o >= 0 && o < 128) {
        const int r = static_cast<int>(o) & 31;
        if (((r >> 2) & 1) == half) {
          const int code = (static_cast<int>(o) >> 5) * 16 + (r >> 3) * 4 + (r & 3);
          float zc = kNegInf;
#pragma unroll
          for (int bm = 0; bm < 4; ++bm)
#pragma unroll
            for (int q = 0; q < 16; ++q)
              if (code == bm * 16 + q) zc = acc[bm][bn][q];
          run_z[bn] = zc;
        }
      }
    }
#pragma unroll
    for (int bm = 0; bm < 4; ++bm)
#pragma unroll
      for (int bn = 0; bn < kNB; ++bn)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[bm][bn][q] = 0.f;
  };

  // ---- pipelined main loop over (V-tile, K-slice) ------------------------
  const int n_pre = n_iter < kStages ? n_iter : kStages;
  for (int sl = 0; sl < n_pre; ++sl) issue(sl);
  wait_dma(n_pre - 1);
  raw_barrier();
  if (k_tail && nk == 1) { clear_k_tail(0); raw_barrier(); }

  // The 4 x kNB MFMAs of one sub-step.
  auto mfma_step = [&](const uint4 (&a)[4], const uint4 (&b)[kNB]) {
#pragma unroll
    for (int j = 0; j < 4 * kNB; ++j) M::run(a[j / kNB], b[j % kNB], acc[j / kNB][j % kNB]);
  };

  uint4 fa[2][4], fb[2][kNB];
  int it = 0;   // global slice counter
  for (int64_t vt = vt0; vt < vt1; ++vt) {
    load_frags(it, 0, fa[0], fb[0]);
    for (int kt = 0; kt < nk; ++kt, ++it) {
#pragma unroll
      for (int kk = 0; kk < kSub; ++kk) {
        const int cur = kk & 1;
        if (kk + 1 < kSub) {
          load_frags(it, kk + 1, fa[cur ^ 1], fb[cur ^ 1]);
          // keep the fragment reads for the next sub-step ahead of this
          // sub-step's MFMAs, so their LDS latency hides under matrix work
          __builtin_amdgcn_sched_barrier(0);
          mfma_step(fa[cur], fb[cur]);
        } else if (KTAIL) {
          // every read of slice `it` is issued: wait for slice it+1, then
          // recycle this slice's stage for slice it+kStages.  On the call's
          // last slice this waits for nothing and the fragment reads below
          // fetch stale (in-bounds, unused) LDS: keeping this path
          // unconditional leaves no control-flow join before the MFMAs.
          const int after = n_iter - 2 - it;
          wait_dma(after < kStages - 2 ? after : kStages - 2);
          raw_barrier();
          if (((it + 1) % nk) == nk - 1) { clear_k_tail(it + 1); raw_barrier(); }
          if (it + kStages < n_iter) issue(it + kStages);
          load_frags(it + 1, 0, fa[cur ^ 1], fb[cur ^ 1]);
          __builtin_amdgcn_sched_barrier(0);
          mfma_step(fa[cur], fb[cur]);
        } else {
          // As above, but the DMAs for slice it+kStages are spread between
          // this sub-step's MFMAs so their issue overlaps matrix work.  They
          // are unconditional: past the end of the work item they re-fetch
          // the last slice into the stage just freed, which nothing reads.
          wait_dma(kStages - 2);
          raw_barrier();
          const int nxt = it + kStages < n_iter ? it + kStages : n_iter - 1;
          prep_issue(nxt);
          load_frags(it + 1, 0, fa[cur ^ 1], fb[cur ^ 1]);
          __builtin_amdgcn_sched_barrier(0);
          constexpr int kM = 4 * kNB;                          // MFMAs per sub-step
          constexpr int kEvery = kM / kDmaPerSlice > 0 ? kM / kDmaPerSlice : 1;
#pragma unroll
          for (int j = 0; j < kM; ++j) {
            M::run(fa[cur][j / kNB], fb[cur][j % kNB], acc[j / kNB][j % kNB]);
            if (j % kEvery == kEvery - 1 && j / kEvery < kDmaPerSlice) issue_one(j / kEvery, std::false_type{});
          }
#pragma unroll
          for (int j = kM / kEvery; j < kDmaPerSlice; ++j) issue_one(j, std::false_type{});
        }
      }
    }
    if ((vt + 1) * kTileV <= V) epilogue(vt, std::false_type{});
    else epilogue(vt, std::true_type{});
  }
  wait_vmcnt<0>();   // (dummy DMAs past the end may still be landing)
  __syncthreads();

  // ---- merge the two lane halves, then the two vocabulary waves -----------
#pragma unroll
  for (int bn = 0; bn < kNB; ++bn) {
    const float m2 = __shfl_xor(run_m[bn], 32);
    const float s2 = __shfl_xor(run_s[bn], 32);
    const float z2 = __shfl_xor(run_z[bn], 32);
    const float t2 = ENT ? __shfl_xor(run_t[bn], 32) : 0.f;
    combine(run_m[bn], run_s[bn], run_z[bn], run_t[bn], m2, s2, z2, t2);
  }
  float* xm = reinterpret_cast<float*>(&lds[0][0][0]);
  float* xs = xm + kTileN;
  float* xz = xs + kTileN;
  float* xt = xz + kTileN;
  if (wm == 1 && half == 0) {
#pragma unroll
    for (int bn = 0; bn < kNB; ++bn) {
      const int tcol = wn * kWaveN + bn * 32 + col;
      xm[tcol] = run_m[bn];
      xs[tcol] = run_s[bn];
      xz[tcol] = run_z[bn];
      if (ENT) xt[tcol] = run_t[bn];
    }
  }
  __syncthreads();
  if (wm == 0 && half == 0) {
#pragma unroll
    for (int bn = 0; bn < kNB; ++bn) {
      const int tcol = wn * kWaveN + bn * 32 + col;
      float m = run_m[bn], s = run_s[bn], z = run_z[bn], t = run_t[bn];
      combine(m, s, z, t, xm[tcol], xs[tcol], xz[tcol], ENT ? xt[tcol] : 0.f);
      const int64_t e = rt * kTileN + tcol;
      if (e < n_s) {
        const int64_t o = ch * p.part_stride + e;
        p.part_m[o] = m;
        p.part_s[o] = s;
        p.part_z[o] = z;
        if (ENT) p.part_t[o] = t;
      }
    }
  }
}

// Combine the chunk partials of each scored row in chunk order and write
// log p = z_y - (m + ln s); non-finite or out-of-range tokens give NaN.
// With entropy requested, also H = ln s - E_p[z - m] = ln s - ln(2) t / s.
__global__ __launch_bounds__(256) void merge_kernel(LmheadArgs p, float* __restrict__ logp,
                                                    float* __restrict__ lse_out,
                                                    float* __restrict__ entropy) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t n_s = *p.n_scored;
  if (e >= n_s) return;
  const bool ent = p.part_t != nullptr;
  float m = p.part_m[e], s = p.part_s[e], z = p.part_z[e], t = ent ? p.part_t[e] : 0.f;
  for (int64_t c = 1; c < p.n_ch; ++c) {
    const int64_t o = c * p.part_stride + e;
    combine(m, s, z, t, p.part_m[o], p.part_s[o], p.part_z[o], ent ? p.part_t[o] : 0.f);
  }
  const float lse = m + __builtin_amdgcn_logf(s) * 0.6931471805599453f;
  const int row = p.rows[e];
  const int y = p.tokens[row];
  float lp = z - lse;
  // The exact value is <= 0; rounding in the fp32 normaliser can leave a
  // positive residue of a few ulps when one logit dominates.
  lp = lp < 0.f ? lp : 0.f;
  if (y < 0 || y >= p.vocab) lp = __builtin_nanf("");
  logp[row] = lp;
  if (lse_out) lse_out[row] = lse;
  if (ent) {
    // The exact value is >= 0; clamp the rounding residue of a near one-hot
    // distribution.
    const float h = __builtin_fmaf(-0.6931471805599453f, t / s, __builtin_amdgcn_logf(s) * 0.6931471805599453f);
    entropy[row] = h > 0.f ? h : 0.f;
  }
}

}  // namespace

hipError_t launch_lmhead(const LmheadArgs& a, int64_t grid, bool bf16, hipStream_t stream) {
  if (grid <= 0) return hipSuccess;
  const dim3 g(static_cast<unsigned>(grid)), b(kThreads);
  const bool tail = (a.d % (bf16 ? 8 * kChunks : 4 * kChunks)) != 0;
  const bool ent = a.part_t != nullptr;
  const int which = (bf16 ? 4 : 0) + (tail ? 2 : 0) + (ent ? 1 : 0);
  switch (which) {
    case 0: hipLaunchKernelGGL((lmhead_logprob_kernel<false, false, false>), g, b, 0, stream, a); break;
    case 1: hipLaunchKernelGGL((lmhead_logprob_kernel<false, false, true>), g, b, 0, stream, a); break;
    case 2: hipLaunchKernelGGL((lmhead_logprob_kernel<false, true, false>), g, b, 0, stream, a); break;
    case 3: hipLaunchKernelGGL((lmhead_logprob_kernel<false, true, true>), g, b, 0, stream, a); break;
    case 4: hipLaunchKernelGGL((lmhead_logprob_kernel<true, false, false>), g, b, 0, stream, a); break;
    case 5: hipLaunchKernelGGL((lmhead_logprob_kernel<true, false, true>), g, b, 0, stream, a); break;
    case 6: hipLaunchKernelGGL((lmhead_logprob_kernel<true, true, false>), g, b, 0, stream, a); break;
    default: hipLaunchKernelGGL((lmhead_logprob_kernel<true, true, true>), g, b, 0, stream, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_merge(const LmheadArgs& a, int64_t n_rows, float* logp, float* lse,
                        float* entropy, hipStream_t stream) {
  const int64_t blocks = (n_rows + 255) / 256;
  if (blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(merge_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, a, logp, lse,
                     entropy);
  return hipGetLastError();
}

}  // namespace hdl
