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
// the V-tiles of one chunk.  Four waves per workgroup, each owning 128 vocab x
// 128 tokens as a 4x4 grid of 32x32 MFMA blocks (fp32 accumulators).  W is
// the MFMA "A" operand (vocabulary on the M axis) and the hidden states are
// the "B" operand (tokens on the N axis), so each lane's accumulators hold one
// token column and 64 vocabulary rows: the online max / sum-of-exp update of
// a V-tile is entirely lane-local, and lanes and waves are merged only once
// per work item.
//
// Operands stream through LDS in K-slices of 128 bytes per row (64 bf16 or 32
// fp32), double-buffered, with an XOR swizzle of the 16-byte chunks so that
// the 32-row fragment reads are bank-conflict free.  Global loads for slice
// i+1 are in flight while slice i is multiplied.
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

constexpr int kThreads = 256;
constexpr int kChunks = 8;                          // 16-byte chunks per LDS row
constexpr int kRowsPerPass = kThreads / kChunks;    // 32 rows per cooperative load
constexpr int kLoads = kTileV / kRowsPerPass;       // 8 loads per operand per slice
constexpr int kTileElems = kTileV * kChunks;        // uint4 slots per operand tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

static_assert(kTileV == kTileN, "square workgroup tile assumed");

__device__ __forceinline__ int swz(int row, int chunk) {
  return row * kChunks + (chunk ^ (row & 7));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

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

// Combine two (max, sum-of-exp, captured logit) states.  Symmetric in its
// arguments, so partner lanes obtain bitwise-identical results.
__device__ __forceinline__ void combine(float& m, float& s, float& z, float m2, float s2, float z2) {
  const float mn = fmaxf(m, m2);
  const float a = (m == mn) ? s : s * fast_exp2((m - mn) * kLog2e);
  const float b = (m2 == mn) ? s2 : s2 * fast_exp2((m2 - mn) * kLog2e);
  s = a + b;
  m = mn;
  z = fmaxf(z, z2);
}

// Row of the 32x32 accumulator block held in element i of lane l:
// row = 8*(i/4) + 4*(l/32) + (i%4), column = l%32.
__device__ __forceinline__ int acc_row(int i, int half) { return 8 * (i >> 2) + 4 * half + (i & 3); }

template <bool BF16>
__global__ __launch_bounds__(kThreads, 1) void lmhead_logprob_kernel(LmheadArgs p) {
  using M = Mma<BF16>;
  constexpr int kEsz = BF16 ? 2 : 4;
  constexpr int kSliceK = M::kElemsPer16B * kChunks;   // K elements per slice

  __shared__ uint4 lds[2][2][kTileElems];   // [stage][0 = W, 1 = hidden]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 1;      // which 128 vocabulary rows of the tile
  const int wn = wave >> 1;     // which 128 token rows of the tile
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
  int tok[4];
#pragma unroll
  for (int bn = 0; bn < 4; ++bn) {
    int64_t e = rt * kTileN + wn * 128 + bn * 32 + col;
    e = e < n_s ? e : n_s - 1;
    tok[bn] = p.tokens[p.rows[e]];
  }

  float run_m[4], run_s[4], run_z[4];
#pragma unroll
  for (int bn = 0; bn < 4; ++bn) { run_m[bn] = kNegInf; run_s[bn] = 0.f; run_z[bn] = kNegInf; }

  f32x16_t acc[4][4];
#pragma unroll
  for (int bm = 0; bm < 4; ++bm)
#pragma unroll
    for (int bn = 0; bn < 4; ++bn)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[bm][bn][q] = 0.f;

  // ---- direct global -> LDS loads -----------------------------------------
  // A K-slice of one operand tile is 32 blocks of 8 rows x 128 bytes.  Wave
  // w fetches blocks 8w .. 8w+7; within a block lane l lands in LDS slot l,
  // i.e. row l/8 and physical chunk l%8, so it fetches logical chunk
  // (l%8) ^ (l/8) of that row (the inverse of the read swizzle).
  const int lrow = lane >> 3;
  const int lchunk = (lane & 7) ^ lrow;
  const bool k_tail = (d % kSliceK) != 0;
  const char* hp[kLoads];
#pragma unroll
  for (int i = 0; i < kLoads; ++i) {
    int64_t e = rt * kTileN + wave * 64 + i * 8 + lrow;
    e = e < n_s ? e : n_s - 1;
    hp[i] = hbase + static_cast<int64_t>(p.rows[e]) * d * kEsz;
  }
  const char* wp[kLoads];
  auto set_w = [&](int64_t vt) {
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      int64_t v = vt * kTileV + wave * 64 + i * 8 + lrow;
      v = v < V ? v : V - 1;
      wp[i] = wbase + v * d * kEsz;
    }
  };
  auto issue = [&](int it, int stage) {
    const int kt = it % nk;
    if (kt == 0) set_w(vt0 + it / nk);
    int64_t koff = (static_cast<int64_t>(kt) * kSliceK + lchunk * M::kElemsPer16B);
    if (k_tail && koff >= d) koff = 0;   // in-bounds dummy; zeroed after arrival
    koff *= kEsz;
#pragma unroll
    for (int i = 0; i < kLoads; ++i)
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(wp[i] + koff),
          (__attribute__((address_space(3))) void*)(&lds[stage][0][(wave * kLoads + i) * 64]),
          16, 0, 0);
#pragma unroll
    for (int i = 0; i < kLoads; ++i)
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(hp[i] + koff),
          (__attribute__((address_space(3))) void*)(&lds[stage][1][(wave * kLoads + i) * 64]),
          16, 0, 0);
  };
  // Wait for this thread's LDS-bound loads; on the last K-slice of a row
  // whose length is not a multiple of the slice, clear the chunks past d.
  auto arrive = [&](int it, int stage) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (k_tail && (it % nk) == nk - 1) {
      for (int sidx = tid; sidx < kTileElems; sidx += kThreads) {
        const int row = sidx >> 3;
        const int chunk = (sidx & 7) ^ (row & 7);
        if (static_cast<int64_t>(it % nk) * kSliceK + chunk * M::kElemsPer16B >= d) {
          lds[stage][0][sidx] = make_uint4(0, 0, 0, 0);
          lds[stage][1][sidx] = make_uint4(0, 0, 0, 0);
        }
      }
    }
    __syncthreads();
  };

  // Online max / sum-of-exp update of one V-tile, then capture of the
  // sampled token's logit if this lane holds it.  MASKED: the tile runs past
  // the end of the vocabulary and rows >= V are excluded.
  auto epilogue = [&](int64_t vt, auto masked_tag) {
    constexpr bool kMasked = decltype(masked_tag)::value;
    const int64_t vbase = vt * kTileV + wm * 128;   // first vocab row of this wave
#pragma unroll
    for (int bn = 0; bn < 4; ++bn) {
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
        float s4[4];
#pragma unroll
        for (int bm = 0; bm < 4; ++bm) {
          float sacc = 0.f;
#pragma unroll
          for (int q = 0; q < 16; ++q) sacc += fast_exp2(__builtin_fmaf(acc[bm][bn][q], kLog2e, -mb));
          s4[bm] = sacc;
        }
        const float tile_sum = (s4[0] + s4[1]) + (s4[2] + s4[3]);
        run_s[bn] = __builtin_fmaf(run_s[bn], fast_exp2(__builtin_fmaf(run_m[bn], kLog2e, -mb)), tile_sum);
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
      for (int bn = 0; bn < 4; ++bn)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[bm][bn][q] = 0.f;
  };

  issue(0, 0);
  arrive(0, 0);

  int it = 0;
  for (int64_t vt = vt0; vt < vt1; ++vt) {
    for (int kt = 0; kt < nk; ++kt, ++it) {
      const int stage = it & 1;
      if (it + 1 < n_iter) issue(it + 1, stage ^ 1);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        uint4 af[4], bf[4];
#pragma unroll
        for (int bm = 0; bm < 4; ++bm)
          af[bm] = lds[stage][0][swz(wm * 128 + bm * 32 + col, kk * 2 + half)];
#pragma unroll
        for (int bn = 0; bn < 4; ++bn)
          bf[bn] = lds[stage][1][swz(wn * 128 + bn * 32 + col, kk * 2 + half)];
#pragma unroll
        for (int bm = 0; bm < 4; ++bm)
#pragma unroll
          for (int bn = 0; bn < 4; ++bn) M::run(af[bm], bf[bn], acc[bm][bn]);
      }
      if (it + 1 < n_iter) arrive(it + 1, stage ^ 1);
      else __syncthreads();
    }
    if ((vt + 1) * kTileV <= V) epilogue(vt, std::false_type{});
    else epilogue(vt, std::true_type{});
  }

  // ---- merge the two lane halves, then the two vocabulary waves -----------
#pragma unroll
  for (int bn = 0; bn < 4; ++bn) {
    const float m2 = __shfl_xor(run_m[bn], 32);
    const float s2 = __shfl_xor(run_s[bn], 32);
    const float z2 = __shfl_xor(run_z[bn], 32);
    combine(run_m[bn], run_s[bn], run_z[bn], m2, s2, z2);
  }
  float* xm = reinterpret_cast<float*>(&lds[0][0][0]);
  float* xs = xm + kTileN;
  float* xz = xs + kTileN;
  if (wm == 1 && half == 0) {
#pragma unroll
    for (int bn = 0; bn < 4; ++bn) {
      const int tcol = wn * 128 + bn * 32 + col;
      xm[tcol] = run_m[bn];
      xs[tcol] = run_s[bn];
      xz[tcol] = run_z[bn];
    }
  }
  __syncthreads();
  if (wm == 0 && half == 0) {
#pragma unroll
    for (int bn = 0; bn < 4; ++bn) {
      const int tcol = wn * 128 + bn * 32 + col;
      float m = run_m[bn], s = run_s[bn], z = run_z[bn];
      combine(m, s, z, xm[tcol], xs[tcol], xz[tcol]);
      const int64_t e = rt * kTileN + tcol;
      if (e < n_s) {
        const int64_t o = ch * p.part_stride + e;
        p.part_m[o] = m;
        p.part_s[o] = s;
        p.part_z[o] = z;
      }
    }
  }
}

// Combine the chunk partials of each scored row in chunk order and write
// log p = z_y - (m + ln s); non-finite or out-of-range tokens give NaN.
__global__ __launch_bounds__(256) void merge_kernel(LmheadArgs p, float* __restrict__ logp,
                                                    float* __restrict__ lse_out) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t n_s = *p.n_scored;
  if (e >= n_s) return;
  float m = p.part_m[e], s = p.part_s[e], z = p.part_z[e];
  for (int64_t c = 1; c < p.n_ch; ++c) {
    const int64_t o = c * p.part_stride + e;
    combine(m, s, z, p.part_m[o], p.part_s[o], p.part_z[o]);
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
}

}  // namespace

hipError_t launch_lmhead(const LmheadArgs& a, int64_t grid, bool bf16, hipStream_t stream) {
  if (grid <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(lmhead_logprob_kernel<true>, dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                       0, stream, a);
  else
    hipLaunchKernelGGL(lmhead_logprob_kernel<false>, dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                       0, stream, a);
  return hipGetLastError();
}

hipError_t launch_merge(const LmheadArgs& a, int64_t n_rows, float* logp, float* lse,
                        hipStream_t stream) {
  const int64_t blocks = (n_rows + 255) / 256;
  if (blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(merge_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, a, logp, lse);
  return hipGetLastError();
}

}  // namespace hdl
