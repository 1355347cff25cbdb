// Hindsight-divergence score and per-root branch-point selection (Eq. 2 and
// the ranking of Sec. 3.2), and the same per-root top-k over an arbitrary
// per-position value (the Entropy localization baseline of Sec. 4.1 ranks
// positions by next-token entropy).
//
// One 1024-thread workgroup per root.  For position t:
//     delta = logp_hind[t] - logp_orig[t]   (one fp32 subtraction)
//     s     = |delta|,  eligible = mask[t] != 0 and delta finite.
// (In value mode, s is the value itself.)  Scores map to 32-bit keys that
// order like the floats (sign-magnitude flipped to an unsigned order, -0
// folded onto +0).  The k largest s are found by a radix select on the
// keys: four 8-bit digits, most
// significant first, each resolved from an LDS histogram (the first one
// built while the keys are staged).  That yields the threshold score S and
// how many positions at exactly S are needed; those are the lowest-indexed
// ties, found in one ordered pass in which every thread owns a contiguous
// range of positions.  The kk <= 1024
// winners are then sorted by the composite key (s, ~t) with a bitonic sort
// in LDS, giving the order (s descending, t ascending).
//
// Branch-point constraints (the paper applies the same ones to every
// localization method, Sec. 4.3): candidates may be restricted to a per-root
// index range [lo, hi], and retained points must lie at least min_gap
// positions apart.  The spacing filter walks the ranked winners and keeps a
// point only if it is far enough from every point kept before it; without
// refill the walk sees only the top k (a point too close to a better one is
// dropped, so a root can end with fewer than k points), with refill it sees
// up to the best 1024 candidates and keeps going until k points are kept.
#include "hdl_internal.h"

namespace hdl {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
// Roots with at most this many positions keep their candidate keys in LDS
// after the first pass (128 KB), so the radix passes and the collect scan
// do not re-read global memory; longer roots recompute them each pass.
constexpr int kStageMax = 32768;

struct Scratch {
  int wsum[kWaves];
  int hist[256];
  int digit;
  int rank;
  unsigned long long keys[kThreads];
  int kept;
  unsigned staged[kStageMax];   // candidate key per position, 0 = not a candidate
};

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  return v;
}

// Exclusive block scan; *total receives the block sum.  Contains barriers:
// every thread of the block must call it.
__device__ __forceinline__ int block_excl_scan(int v, int* total, Scratch& sh) {
  const int incl = wave_incl_scan(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) sh.wsum[w] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) {
    const int x = sh.wsum[i];
    before += (i < w) ? x : 0;
    all += x;
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

struct Pos {
  float delta;
  unsigned key;
  bool elig;
};

// Unsigned key ordered like the float (finite inputs); -0 maps like +0.
__device__ __forceinline__ unsigned float_key(float f) {
  const unsigned u = __float_as_uint(f == 0.f ? 0.f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_float(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// VALUES: the score is lo[t] itself; otherwise |lh[t] - lo[t]| (one fp32
// subtraction).
template <bool VALUES>
__device__ __forceinline__ Pos load_pos(const float* lo, const float* lh, const uint8_t* mask,
                                        int64_t base, int64_t t) {
  Pos p;
  const float d = VALUES ? lo[base + t] : lh[base + t] - lo[base + t];
  const bool on = (mask == nullptr) || (mask[base + t] != 0);
  p.elig = on && __builtin_isfinite(d);
  p.delta = p.elig ? d : 0.f;
  p.key = float_key(VALUES ? p.delta : __builtin_fabsf(p.delta));
  return p;
}

// Candidate for ranking: eligible and inside the root's index range.
__device__ __forceinline__ Pos load_cand(bool values, const float* lo, const float* lh, const uint8_t* mask,
                                         int64_t base, int64_t t, int64_t t_lo, int64_t t_hi) {
  Pos p = values ? load_pos<true>(lo, lh, mask, base, t) : load_pos<false>(lo, lh, mask, base, t);
  p.elig = p.elig && t >= t_lo && t <= t_hi;
  return p;
}

// Candidate key of position t: from LDS when the root is staged, else
// recomputed from global memory (0: not a candidate; every candidate's key
// is at least 0x00800000, the key of the most negative finite float).
template <bool VALUES>
__device__ __forceinline__ unsigned cand_key(const Scratch& sh, bool staged, const float* lo, const float* lh,
                                             const uint8_t* mask, int64_t base, int64_t t, int64_t t_lo,
                                             int64_t t_hi) {
  if (staged) return sh.staged[t];
  const Pos p = load_cand(VALUES, lo, lh, mask, base, t, t_lo, t_hi);
  return p.elig ? p.key : 0u;
}

// pool: winners ranked before the spacing filter (k without refill);
// min_gap <= 1 disables the filter; r_lo / r_hi (optional) bound the range.
template <bool VALUES>
__global__ __launch_bounds__(kThreads) void select_kernel(const float* __restrict__ lo,
                                                          const float* __restrict__ lh,
                                                          const uint8_t* __restrict__ mask,
                                                          int64_t T, int k,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ score,
                                                          int32_t* __restrict__ count,
                                                          float* __restrict__ delta_out,
                                                          const int32_t* __restrict__ r_lo,
                                                          const int32_t* __restrict__ r_hi,
                                                          int min_gap, int pool) {
  __shared__ Scratch sh;
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t base = static_cast<int64_t>(r) * T;
  const int64_t t_lo = r_lo ? r_lo[r] : 0;
  const int64_t t_hi = r_hi ? r_hi[r] : T - 1;

  // ---- eligibility count (and the optional signed delta) -----------------
  // A staged root also gets the histogram of its keys' top digit here, the
  // first radix pass's, so that pass needs no sweep of its own.
  const bool staged = T <= kStageMax;
  for (int i = tid; i < 256; i += kThreads) sh.hist[i] = 0;
  __syncthreads();
  int c = 0;
  for (int64_t t = tid; t < T; t += kThreads) {
    const Pos p = load_pos<VALUES>(lo, lh, mask, base, t);
    if (delta_out) delta_out[base + t] = p.delta;
    const bool cand = p.elig && t >= t_lo && t <= t_hi;
    if (staged) {
      sh.staged[t] = cand ? p.key : 0u;
      if (cand) atomicAdd(&sh.hist[p.key >> 24], 1);
    }
    c += cand ? 1 : 0;
  }
  int n_elig;
  block_excl_scan(c, &n_elig, sh);   // (its barriers also publish the histogram)
  const int kk = n_elig < pool ? n_elig : pool;

  if (kk > 0) {
    // ---- radix select of the kk-th largest score --------------------------
    unsigned prefix = 0, pmask = 0;
    int rank = kk;   // rank of the threshold among positions matching prefix
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (!(staged && shift == 24)) {
        for (int i = tid; i < 256; i += kThreads) sh.hist[i] = 0;
        __syncthreads();
        for (int64_t t = tid; t < T; t += kThreads) {
          const unsigned key = cand_key<VALUES>(sh, staged, lo, lh, mask, base, t, t_lo, t_hi);
          if (key != 0u && (key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shift) & 255], 1);
        }
        __syncthreads();
      }
      // Inclusive scan over bins from the top digit down; the bin in which
      // the running count reaches `rank` holds the threshold.
      const int h = (tid < 256) ? sh.hist[255 - tid] : 0;
      int tot;
      const int above = block_excl_scan(h, &tot, sh);
      if (tid < 256 && above < rank && above + h >= rank) {
        sh.digit = 255 - tid;
        sh.rank = rank - above;
      }
      __syncthreads();
      prefix |= static_cast<unsigned>(sh.digit) << shift;
      pmask |= 255u << shift;
      rank = sh.rank;
      __syncthreads();
    }
    const unsigned thr = prefix;   // bit pattern of the kk-th largest score
    const int need_ties = rank;    // positions scoring exactly thr to take

    // ---- collect: all above the threshold, then the lowest-indexed ties ---
    // Thread i owns the contiguous positions [i per, (i + 1) per): one scan
    // of the per-thread tie counts gives every thread the ties at lower
    // positions, one scan of the per-thread takes gives its output slots.
    const int64_t per = (T + kThreads - 1) / kThreads;
    const int64_t t_beg = tid * per;
    const int64_t t_end = t_beg + per < T ? t_beg + per : T;
    int my_eq = 0;
    for (int64_t t = t_beg; t < t_end; ++t)
      my_eq += cand_key<VALUES>(sh, staged, lo, lh, mask, base, t, t_lo, t_hi) == thr ? 1 : 0;
    int n_eq_all;
    const int eq_before = block_excl_scan(my_eq, &n_eq_all, sh);
    int my_take = 0;
    {
      int eq_seen = eq_before;
      for (int64_t t = t_beg; t < t_end; ++t) {
        const unsigned key = cand_key<VALUES>(sh, staged, lo, lh, mask, base, t, t_lo, t_hi);
        if (key > thr) ++my_take;
        else if (key == thr && key != 0u) my_take += (eq_seen++ < need_ties) ? 1 : 0;
      }
    }
    int n_take_all;
    int slot = block_excl_scan(my_take, &n_take_all, sh);
    {
      int eq_seen = eq_before;
      for (int64_t t = t_beg; t < t_end; ++t) {
        const unsigned key = cand_key<VALUES>(sh, staged, lo, lh, mask, base, t, t_lo, t_hi);
        bool take = key > thr;
        if (key == thr && key != 0u) take = eq_seen++ < need_ties;
        if (take) {
          if (slot < kThreads)
            sh.keys[slot] = (static_cast<unsigned long long>(key) << 32) |
                            static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<unsigned>(t));
          ++slot;
        }
      }
    }
    __syncthreads();

    // ---- bitonic sort, descending, of the kk winners ----------------------
    // (padding keys are 0, below every real key: a finite score's key is at
    // least 0x00800000, so every real composite key is positive)
    int P = 1;
    while (P < kk) P <<= 1;
    for (int i = kk + tid; i < P; i += kThreads) sh.keys[i] = 0ull;
    __syncthreads();
    for (int size = 2; size <= P; size <<= 1) {
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int i = tid; i < P; i += kThreads) {
          const int jx = i ^ stride;
          if (jx > i) {
            const unsigned long long a = sh.keys[i], bb = sh.keys[jx];
            const bool desc = (i & size) == 0;
            if (desc ? (a < bb) : (a > bb)) {
              sh.keys[i] = bb;
              sh.keys[jx] = a;
            }
          }
        }
        __syncthreads();
      }
    }
  }

  // ---- spacing filter over the ranked winners ----------------------------
  int n_out = kk < k ? kk : k;
  if (min_gap > 1 && kk > 0) {
    if (tid == 0) {
      int kept = 0;
      for (int j = 0; j < kk && kept < k; ++j) {
        const unsigned long long key = sh.keys[j];
        const int64_t t = 0xFFFFFFFFu - static_cast<unsigned>(key & 0xFFFFFFFFull);
        bool ok = true;
        for (int q = 0; q < kept && ok; ++q) {
          const int64_t u = 0xFFFFFFFFu - static_cast<unsigned>(sh.keys[q] & 0xFFFFFFFFull);
          ok = (t > u ? t - u : u - t) >= min_gap;
        }
        if (ok) sh.keys[kept++] = key;   // kept <= j: compaction in place
      }
      sh.kept = kept;
    }
    __syncthreads();
    n_out = sh.kept;
  }

  for (int j = tid; j < k; j += kThreads) {
    if (j < n_out) {
      const unsigned long long key = sh.keys[j];
      idx[static_cast<int64_t>(r) * k + j] = static_cast<int32_t>(0xFFFFFFFFu - static_cast<unsigned>(key & 0xFFFFFFFFull));
      score[static_cast<int64_t>(r) * k + j] = key_float(static_cast<unsigned>(key >> 32));
    } else {
      idx[static_cast<int64_t>(r) * k + j] = -1;
      score[static_cast<int64_t>(r) * k + j] = 0.f;
    }
  }
  if (tid == 0) count[r] = n_out;
}

}  // namespace

hipError_t launch_select(const float* lo, const float* lh, const uint8_t* mask, int64_t n_roots,
                         int64_t T, int k, int32_t* idx, float* score, int32_t* count, float* delta,
                         bool values, hipStream_t stream, const int32_t* r_lo, const int32_t* r_hi,
                         int min_gap, int pool) {
  if (pool < k) pool = k;
  if (values)
    hipLaunchKernelGGL(select_kernel<true>, dim3(static_cast<unsigned>(n_roots)), dim3(kThreads), 0,
                       stream, lo, lh, mask, T, k, idx, score, count, delta, r_lo, r_hi, min_gap, pool);
  else
    hipLaunchKernelGGL(select_kernel<false>, dim3(static_cast<unsigned>(n_roots)), dim3(kThreads), 0,
                       stream, lo, lh, mask, T, k, idx, score, count, delta, r_lo, r_hi, min_gap, pool);
  return hipGetLastError();
}

}  // namespace hdl
