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
// and merge_kernel combines the chunk partials in a fixed order.  Two more
// epilogues share the same main loop: one also accumulates the next-token
// entropy (the Entropy localization baseline), the other writes the gradient
// of log p with respect to the logits for the backward pass (the logits are
// recomputed there, given the forward pass's log-sum-exp).
//
// Work item: 256 vocabulary rows x 256 token rows per V-tile, looping over
// the V-tiles of one chunk.  Eight waves per workgroup (two per SIMD, so one
// wave's LDS reads and DMA issue overlap the other's MFMAs; the per-V-tile
// epilogue, which both reach after the same slice, does not), each owning
// 128 vocab x 64 tokens as an 8 x 4 grid of 16 x 16 MFMA blocks
// (v_mfma_f32_16x16x32_bf16) with fp32 accumulators.
// W is the MFMA "A" operand (vocabulary on the M axis) and the hidden states
// are the "B" operand (tokens on the N axis), so each lane's accumulators
// hold 4 token columns and 32 vocabulary rows each: the online max /
// sum-of-exp update of a V-tile is entirely lane-local, and lanes and waves
// are merged only once per work item.
//
// Operands stream through LDS in K-slices of 128 bytes per row (64 bf16 or
// 32 fp32) through a ring of 2 stages (128 KB): the next slice is in flight
// (global -> LDS DMA, no VGPR staging) while slice i is multiplied.  16-byte
// chunks are XOR swizzled and each lane group reads the chunk frag_chunk()
// assigns it, so that the 16-row fragment reads are bank-conflict free.
// The DMA is issued from inline assembly (wave-uniform 64-bit base +
// per-lane 32-bit offset) and waited for with explicit vmcnt counts: the
// compiler cannot see that a DMA into one stage does not alias the reads of
// another, and would otherwise wait for every outstanding DMA before each LDS
// read.
#include "tile_common.h"

#include <type_traits>

namespace hdl {
namespace {

using namespace tile;

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

static_assert(kKSteps == 2, "a K-slice is two K-steps");
static_assert(kVB % 2 == 0, "the gradient epilogue pairs vocabulary blocks");

// KTAIL: d is not a multiple of the K-slice, so the last slice of every
// row needs zero-filling (a separate instantiation keeps that work out of the
// common case).  EPI selects what each V-tile's logits feed:
//   kEpiStats:   online max / sum of exp and the sampled-token logit;
//   kEpiEntropy: the same plus sum exp(z - m) * (z - m) for the next-token
//                entropy H = ln s - E_p[z - m] (the Entropy localization
//                baseline);
//   kEpiGrad:    the gradient of log p with respect to the logits,
//                g (1[v == y] - exp(z - lse)), written as bf16 (backward pass;
//                lse comes from the forward pass), chunk-major (8 vocabulary
//                entries of a row, then the same 8 of the next row), with
//                zero rows up to the next multiple of 64 rows so that a
//                contraction over rows can run in whole 64-row K-slices.
constexpr int kEpiStats = 0, kEpiEntropy = 1, kEpiGrad = 2;

template <bool BF16, bool KTAIL, int EPI>
__global__ __launch_bounds__(kThreads, 1) void lmhead_logprob_kernel(LmheadArgs p) {
  constexpr bool ENT = EPI == kEpiEntropy;
  constexpr bool GRAD = EPI == kEpiGrad;
  using M = Mma16<BF16>;
  constexpr int kEsz = BF16 ? 2 : 4;
  constexpr int kElemsPer16B = 16 / kEsz;
  constexpr int kSliceK = kElemsPer16B * kChunks;   // K elements per slice

  __shared__ uint4 lds[kStages][2][kSlots];   // [stage][0 = W, 1 = hidden] = 128 KB

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int wm = wave & 1;      // which 128 vocabulary rows of the tile
  const int wn = wave >> 1;     // which kWaveN token rows of the tile
  const int r16 = lane & 15;    // row of a 16-row fragment / column of a result block
  const int grp = lane >> 4;    // lane group: K chunk of a fragment, row quad of a result block

  // ---- work item: XCD-aware (row tile, vocabulary chunk), see plan.h -----
  int64_t rt, ch;
  work_item(blockIdx.x, p.n_grt, &rt, &ch);
  int64_t n_s = *p.n_scored - p.row_base;
  n_s = n_s < 0 ? 0 : (n_s > p.row_cap ? p.row_cap : n_s);
  const int64_t n_rt = (n_s + kTileN - 1) / kTileN;
  const int64_t n_s_pad = (n_s + 63) / 64 * 64;   // gradient mode: rows written (row_cap % 64 == 0)
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
  int tok[kTB];
  float g_lse[kTB], g_up[kTB];   // gradient mode: lse * log2(e) and upstream gradient
#pragma unroll
  for (int bn = 0; bn < kTB; ++bn) {
    int64_t e = rt * kTileN + wn * kWaveN + bn * 16 + r16;
    e = e < n_s ? e : n_s - 1;
    const int row = p.rows[e];
    tok[bn] = p.tokens[row];
    if (GRAD) {
      // no indicator term for a token outside [0, V): padding columns of G stay 0
      tok[bn] = (tok[bn] >= 0 && tok[bn] < V) ? tok[bn] : -1;
      g_lse[bn] = p.lse_in[row] * kLog2e;
      g_up[bn] = p.grad_in[row];
    }
  }

  float run_m[kTB], run_s[kTB], run_z[kTB], run_t[kTB];
#pragma unroll
  for (int bn = 0; bn < kTB; ++bn) { run_m[bn] = kNegInf; run_s[bn] = 0.f; run_z[bn] = kNegInf; run_t[bn] = 0.f; }

  f32x4_t acc[kVB][kTB];
#pragma unroll
  for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[bm][bn][q] = 0.f;

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
  // blocks; a launch never spans more than 4 GiB of hidden states, and W is
  // addressed from the current V-tile's first row.
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
  // slot: the ring position (its stage); slice: the data fetched into it
  // (they differ only for the copies of the last slice past the end)
  auto prep_issue = [&](int slot, int slice) {
    issue_stage = slot % kStages;
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
    prep_issue(slice, slice);
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
      if (static_cast<int64_t>(kt) * kSliceK + chunk * kElemsPer16B >= d) {
        lds[stage][0][sidx] = make_uint4(0, 0, 0, 0);
        lds[stage][1][sidx] = make_uint4(0, 0, 0, 0);
      }
    }
  };

  // ---- fragment reads ------------------------------------------------------
  // Fragments start at multiples of 16 rows, so a fragment row's swizzle is
  // that of (lane mod 16): one per-lane offset per K-step, plus immediates.
  // Lane group g reads chunk 4 ks + frag_chunk(g) of the K-step (A and B
  // alike, so the K positions pair up).
  const int kchunk = frag_chunk(grp);
  const int frag_lane[kKSteps] = {(r16 * kChunks + ((0 + kchunk) ^ row_xor(r16))),
                                  (r16 * kChunks + ((4 + kchunk) ^ row_xor(r16)))};
  // the two W fragments (vocabulary blocks 2 pr, 2 pr + 1) of quarter pr of K-step ks
  auto load_a = [&](int slice, int ks, int pr, uint4 (&dst)[2]) {
    const uint4* base = &lds[slice % kStages][0][frag_lane[ks]];
#pragma unroll
    for (int j = 0; j < 2; ++j) dst[j] = base[(wm * 128 + (2 * pr + j) * 16) * kChunks];
  };
  // hidden-state fragment of token block bn, K-step ks
  auto load_b = [&](int slice, int ks, int bn, uint4& dst) {
    dst = lds[slice % kStages][1][frag_lane[ks] + (wn * kWaveN + bn * 16) * kChunks];
  };
  // the 2 x kTB MFMAs of quarter pr
  auto quarter_mfma = [&](const uint4 (&a)[2], const uint4 (&b)[kTB], int pr) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < kTB; ++i) M::run(a[j], b[snake(j, i)], acc[2 * pr + j][snake(j, i)]);
  };

  // Online max / sum-of-exp update of one V-tile, then capture of the
  // sampled token's logit if this lane holds it.  MASKED: the tile runs past
  // the end of the vocabulary and rows >= V are excluded.
  auto epilogue = [&](int64_t vt, auto masked_tag) {
    constexpr bool kMasked = decltype(masked_tag)::value;
    const int64_t vbase = vt * kTileV + wm * 128;   // first vocab row of this wave
    const int64_t vlane = vbase + 4 * grp;          // + 16 bm + i: this lane's rows
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn) {
      if (kMasked) {
#pragma unroll
        for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (vlane + bm * 16 + q >= V) acc[bm][bn][q] = kNegInf;
      }
      float mx = acc[0][bn][0];
#pragma unroll
      for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
        for (int q = 0; q < 4; ++q) mx = fmaxf(mx, acc[bm][bn][q]);
      const float mnew = fmaxf(run_m[bn], mx);
      if (!kMasked || mnew != kNegInf) {
        const float mb = mnew * kLog2e;
        float s4[4], t4[4];
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          float sacc = 0.f, tacc = 0.f;
#pragma unroll
          for (int bm = 2 * g4; bm < 2 * g4 + 2; ++bm)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float zq = acc[bm][bn][q];
              const float zl = __builtin_fmaf(zq, kLog2e, -mb);   // (z - m) log2(e)
              const float e = fast_exp2(zl);
              sacc += e;
              // (masked rows hold -inf and e = 0; their product term is 0)
              if (ENT) tacc = __builtin_fmaf(e, (kMasked && zq == kNegInf) ? 0.f : zl, tacc);
            }
          s4[g4] = sacc;
          t4[g4] = tacc;
        }
        const float tile_sum = (s4[0] + s4[1]) + (s4[2] + s4[3]);
        const float rescale = fast_exp2(__builtin_fmaf(run_m[bn], kLog2e, -mb));
        if (ENT)   // (before run_s changes: shift_t wants the old sum)
          run_t[bn] = shift_t(run_t[bn], run_s[bn], run_m[bn], mnew, rescale) + ((t4[0] + t4[1]) + (t4[2] + t4[3]));
        run_s[bn] = __builtin_fmaf(run_s[bn], rescale, tile_sum);
        run_m[bn] = mnew;
      }
      const int64_t o = static_cast<int64_t>(tok[bn]) - vbase;
      if (o >= 0 && o < 128 && ((static_cast<int>(o) >> 2) & 3) == grp) {
        const int code = (static_cast<int>(o) >> 4) * 4 + (static_cast<int>(o) & 3);   // 4 bm + i
        float zc = kNegInf;
#pragma unroll
        for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (code == bm * 4 + q) zc = acc[bm][bn][q];
        run_z[bn] = zc;
      }
    }
#pragma unroll
    for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
      for (int bn = 0; bn < kTB; ++bn)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[bm][bn][q] = 0.f;
  };

  // Gradient mode: G = g (1[v == y] - p) for the kVB x kTB blocks of this
  // wave, rounded to bf16.  In each block a lane holds 4 consecutive
  // vocabulary entries of its token row: half of an 8-entry chunk (lane
  // groups 0 and 1 hold the two halves of one chunk, groups 2 and 3 those of
  // the next).  Blocks are taken in pairs: v_permlane16_swap_b32 trades the
  // odd lane groups' halves of the first block for the even groups' halves
  // of the second, so that every lane then holds one whole chunk, chunk
  // frag_chunk(g) of the pair's four, and stores it with one 16-byte store
  // (stores of 8 bytes per lane drained about 1.6 times slower: all work
  // items reach this epilogue together, and the next K-slice's DMA wait
  // also waits for these stores).  G is stored chunk-major, so a store
  // instruction covers four runs of 256 contiguous bytes (16 token rows x one
  // chunk each).  Rows >= V hold -inf, so p = 0 and G = 0 there, which
  // zero-fills the columns up to g_cols.
  auto grad_epilogue = [&](int64_t vt) {
    const int vbase = static_cast<int>(vt * kTileV) + wm * 128;   // V < 2^31
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn) {
      const int64_t e = rt * kTileN + wn * kWaveN + bn * 16 + r16;
      const bool live = e < n_s;   // rows n_s .. round_up(n_s, 64) - 1 are written as zeros
      uint16_t* gcol = p.g_out + e * 8;   // chunk c of this row: gcol + c * g_ld * 8
      const float gneg = -g_up[bn];
      // The sampled token's column gets g (1 - p), computed as g - g p (one
      // rounding); `code` is its place 4 bm + q among this lane's elements of
      // the column, -1 if the lane does not hold it.
      const int o = tok[bn] - vbase;
      const int code = (o >= 0 && o < 128 && ((o >> 2) & 3) == grp) ? (o >> 4) * 4 + (o & 3) : -1;
#pragma unroll
      for (int bp = 0; bp < kVB; bp += 2) {
        uint32_t pk[2][2];   // [block of the pair][bf16 pair]: entries v0 .. v0 + 3
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int bm = bp + h;
          float gv[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float pv = fast_exp2(__builtin_fmaf(acc[bm][bn][q], kLog2e, -g_lse[bn]));
            gv[q] = __builtin_fmaf(gneg, pv, code == bm * 4 + q ? g_up[bn] : 0.f);
          }
#pragma unroll
          for (int r = 0; r < 4; r += 2) {
            const uint32_t w = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{gv[r], gv[r + 1]}, bf16x2_t));
            pk[h][r / 2] = live ? w : 0u;
          }
        }
        // even lane groups keep their first-block half and receive the
        // partner's (the chunk's upper half); odd groups receive the
        // partner's second-block half (the lower half) and keep their own
        const auto s0 = __builtin_amdgcn_permlane16_swap(pk[0][0], pk[1][0], false, false);
        const auto s1 = __builtin_amdgcn_permlane16_swap(pk[0][1], pk[1][1], false, false);
        const int chunk = (vbase + bp * 16) / 8 + frag_chunk(grp);
        // (the pair's 32 columns lie wholly below g_cols, a multiple of 64, or
        // wholly above).  Non-temporal: G is read back only by the two GEMMs,
        // long after it has left the L2, and these write-backs would
        // otherwise evict the tiles the next K-slices' DMAs read.
        if (e < n_s_pad && vbase + bp * 16 < p.g_cols)
          __builtin_nontemporal_store(u32x4_t{s0[0], s1[0], s0[1], s1[1]},
                                      reinterpret_cast<u32x4_t*>(gcol + static_cast<int64_t>(chunk) * p.g_ld * 8));
      }
    }
#pragma unroll
    for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
      for (int bn = 0; bn < kTB; ++bn)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[bm][bn][q] = 0.f;
  };

  // ---- pipelined main loop over (V-tile, K-slice) ------------------------
  // A K-slice is 2 K-steps x 4 quarters; quarter pr multiplies the W
  // fragments of vocabulary blocks 2 pr, 2 pr + 1 with the kTB hidden-state
  // fragments.  Each quarter first reads what the next one needs: the next
  // quarter's two W fragments (alternating buffers fa[0], fa[1]) and, during
  // K-step 0, one hidden-state fragment of K-step 1 (fb[1]).  The slice's
  // last quarter waits for the next slice's DMA and the workgroup barrier,
  // reads the next slice's first W fragments and all of its K-step-0 hidden
  // fragments (fb[0]), and issues the DMA of the slice after next into the
  // stage just released, spread between its MFMAs.
  const int n_pre = n_iter < kStages ? n_iter : kStages;
  for (int sl = 0; sl < n_pre; ++sl) issue(sl);
  wait_dma(n_pre - 1);
  raw_barrier();
  if (k_tail && nk == 1) { clear_k_tail(0); raw_barrier(); }

  uint4 fa[2][2], fb[2][kTB];
  int it = 0;   // global slice counter
  for (int64_t vt = vt0; vt < vt1; ++vt) {
    load_a(it, 0, 0, fa[0]);
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn) load_b(it, 0, bn, fb[0][bn]);
    for (int kt = 0; kt < nk; ++kt, ++it) {
      // K-step 0
#pragma unroll
      for (int pr = 0; pr < 4; ++pr) {
        if (pr < 3) load_a(it, 0, pr + 1, fa[(pr + 1) & 1]);
        else load_a(it, 1, 0, fa[0]);
        load_b(it, 1, pr, fb[1][pr]);
        // keep the fragment reads for the next quarter ahead of this
        // quarter's MFMAs, so their LDS latency hides under matrix work
        __builtin_amdgcn_sched_barrier(0);
        quarter_mfma(fa[pr & 1], fb[0], pr);
      }
      // K-step 1, quarters 0-2
#pragma unroll
      for (int pr = 0; pr < 3; ++pr) {
        load_a(it, 1, pr + 1, fa[(pr + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        quarter_mfma(fa[pr & 1], fb[1], pr);
      }
      // K-step 1, quarter 3: the slice boundary.  Every read of slice `it`
      // is issued: wait for slice it+1, then recycle this slice's stage.  On
      // the work item's last slice this waits for nothing and the reads of
      // "slice it+1" fetch stale (in-bounds, unused) LDS: keeping this path
      // unconditional leaves no control-flow join before the MFMAs.
      if (KTAIL) {
        const int after = n_iter - 2 - it;
        wait_dma(after < kStages - 2 ? after : kStages - 2);
        raw_barrier();
        if (((it + 1) % nk) == nk - 1) { clear_k_tail(it + 1); raw_barrier(); }
        if (it + kStages < n_iter) issue(it + kStages);
        load_a(it + 1, 0, 0, fa[0]);
#pragma unroll
        for (int bn = 0; bn < kTB; ++bn) load_b(it + 1, 0, bn, fb[0][bn]);
        __builtin_amdgcn_sched_barrier(0);
        quarter_mfma(fa[1], fb[1], 3);
      } else {
        // As above, but the DMAs for slice it+kStages are spread between
        // this quarter's MFMAs so their issue overlaps matrix work.  They are
        // unconditional: past the end of the work item they fetch a copy of
        // the last slice into the stage just freed, which nothing reads.
        wait_dma(kStages - 2);
        raw_barrier();
        prep_issue(it + kStages, it + kStages < n_iter ? it + kStages : n_iter - 1);
        load_a(it + 1, 0, 0, fa[0]);
#pragma unroll
        for (int bn = 0; bn < kTB; ++bn) load_b(it + 1, 0, bn, fb[0][bn]);
        __builtin_amdgcn_sched_barrier(0);
        constexpr int kM = 2 * kTB;                          // MFMAs per quarter
        constexpr int kEvery = kM / kDmaPerSlice > 0 ? kM / kDmaPerSlice : 1;
#pragma unroll
        for (int j = 0; j < kM; ++j) {
          M::run(fa[1][j / kTB], fb[1][snake(j / kTB, j % kTB)], acc[6 + j / kTB][snake(j / kTB, j % kTB)]);
          if (j % kEvery == kEvery - 1 && j / kEvery < kDmaPerSlice) issue_one(j / kEvery, std::false_type{});
        }
#pragma unroll
        for (int j = kM / kEvery; j < kDmaPerSlice; ++j) issue_one(j, std::false_type{});
      }
    }
    if (GRAD) {
      if ((vt + 1) * kTileV > V) {
        // rows >= V: -inf, so that they contribute G = 0
#pragma unroll
        for (int bm = 0; bm < kVB; ++bm)
#pragma unroll
          for (int bn = 0; bn < kTB; ++bn)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              if (vt * kTileV + wm * 128 + bm * 16 + 4 * grp + q >= V) acc[bm][bn][q] = kNegInf;
      }
      grad_epilogue(vt);
    } else if ((vt + 1) * kTileV <= V) {
      epilogue(vt, std::false_type{});
    } else {
      epilogue(vt, std::true_type{});
    }
  }
  wait_vmcnt<0>();   // (dummy DMAs past the end may still be landing)
  __syncthreads();
  if (GRAD) return;

  // ---- merge the four lane groups, then the two vocabulary waves ----------
#pragma unroll
  for (int bn = 0; bn < kTB; ++bn) {
#pragma unroll
    for (int x = 16; x <= 32; x <<= 1) {
      const float m2 = __shfl_xor(run_m[bn], x);
      const float s2 = __shfl_xor(run_s[bn], x);
      const float z2 = __shfl_xor(run_z[bn], x);
      const float t2 = ENT ? __shfl_xor(run_t[bn], x) : 0.f;
      combine(run_m[bn], run_s[bn], run_z[bn], run_t[bn], m2, s2, z2, t2);
    }
  }
  float* xm = reinterpret_cast<float*>(&lds[0][0][0]);
  float* xs = xm + kTileN;
  float* xz = xs + kTileN;
  float* xt = xz + kTileN;
  if (wm == 1 && grp == 0) {
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn) {
      const int tcol = wn * kWaveN + bn * 16 + r16;
      xm[tcol] = run_m[bn];
      xs[tcol] = run_s[bn];
      xz[tcol] = run_z[bn];
      if (ENT) xt[tcol] = run_t[bn];
    }
  }
  __syncthreads();
  if (wm == 0 && grp == 0) {
#pragma unroll
    for (int bn = 0; bn < kTB; ++bn) {
      const int tcol = wn * kWaveN + bn * 16 + r16;
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
  // positive residue of a few ulps when one logit dominates.  (Written so
  // that a NaN -- a non-finite hidden state -- stays NaN.)
  lp = lp > 0.f ? 0.f : lp;
  if (y < 0 || y >= p.vocab) lp = __builtin_nanf("");
  logp[row] = lp;
  if (lse_out) lse_out[row] = lse;
  if (ent) {
    // The exact value is >= 0; clamp the rounding residue of a near one-hot
    // distribution.
    const float h = __builtin_fmaf(-0.6931471805599453f, t / s, __builtin_amdgcn_logf(s) * 0.6931471805599453f);
    entropy[row] = h < 0.f ? 0.f : h;
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
    case 0: hipLaunchKernelGGL((lmhead_logprob_kernel<false, false, kEpiStats>), g, b, 0, stream, a); break;
    case 1: hipLaunchKernelGGL((lmhead_logprob_kernel<false, false, kEpiEntropy>), g, b, 0, stream, a); break;
    case 2: hipLaunchKernelGGL((lmhead_logprob_kernel<false, true, kEpiStats>), g, b, 0, stream, a); break;
    case 3: hipLaunchKernelGGL((lmhead_logprob_kernel<false, true, kEpiEntropy>), g, b, 0, stream, a); break;
    case 4: hipLaunchKernelGGL((lmhead_logprob_kernel<true, false, kEpiStats>), g, b, 0, stream, a); break;
    case 5: hipLaunchKernelGGL((lmhead_logprob_kernel<true, false, kEpiEntropy>), g, b, 0, stream, a); break;
    case 6: hipLaunchKernelGGL((lmhead_logprob_kernel<true, true, kEpiStats>), g, b, 0, stream, a); break;
    default: hipLaunchKernelGGL((lmhead_logprob_kernel<true, true, kEpiEntropy>), g, b, 0, stream, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_lmhead_grad(const LmheadArgs& a, int64_t grid, hipStream_t stream) {
  if (grid <= 0) return hipSuccess;
  const dim3 g(static_cast<unsigned>(grid)), b(kThreads);
  if (a.d % (8 * kChunks) != 0)
    hipLaunchKernelGGL((lmhead_logprob_kernel<true, true, kEpiGrad>), g, b, 0, stream, a);
  else
    hipLaunchKernelGGL((lmhead_logprob_kernel<true, false, kEpiGrad>), g, b, 0, stream, a);
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
