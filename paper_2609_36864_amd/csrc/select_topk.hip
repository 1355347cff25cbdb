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
// keys: four 8-bit digits, most significant first, each resolved from an LDS
// histogram (the first one built while the keys are staged) by one wave.
// That yields the threshold score S and how many positions at exactly S are
// needed.  Each wave then sweeps a contiguous range of positions, its lanes
// on consecutive positions (coalesced, and spread over the LDS banks), and
// takes every score above S and, when only some of the positions at S are
// needed, the lowest-indexed ones (the ties of lower wave ranges are counted
// first).  The kk <= 1024 winners are sorted by the composite key (s, ~t)
// with a bitonic network -- in one wave's registers for kk <= 64, else in
// LDS -- giving the order (s descending, t ascending).
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

#include <type_traits>

namespace hdl {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
// Roots with at most this many positions keep their candidate keys in LDS
// after the first pass (128 KB), so the radix passes and the collect pass
// do not re-read global memory; longer roots recompute them each pass.
constexpr int kStageMax = 32768;

struct Scratch {
  int welig[kWaves];    // candidates per wave
  int weq[kWaves];      // positions at the threshold per wave range
  int hist[2][256];     // radix histograms, alternating between digits
  int digit;
  int rank;
  int n_thr;            // candidates scoring exactly the threshold
  int n_taken;          // winner slots handed out so far
  unsigned long long keys[kThreads];
  int kept;
  unsigned staged[kStageMax];   // candidate key per position, 0 = not a candidate
};

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Lanes below this one whose bit is set in a wave-wide mask.
__device__ __forceinline__ int lanes_below(unsigned long long m) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<unsigned>(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<unsigned>(m), 0u));
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

// Score of a position from its loaded inputs: in VALUES mode the value a
// itself, otherwise |b - a| (one fp32 subtraction).
template <bool VALUES>
__device__ __forceinline__ Pos make_pos(float a, float b, bool on) {
  Pos p;
  const float d = VALUES ? a : b - a;
  p.elig = on && __builtin_isfinite(d);
  p.delta = p.elig ? d : 0.f;
  p.key = float_key(VALUES ? p.delta : __builtin_fabsf(p.delta));
  return p;
}

template <bool VALUES>
__device__ __forceinline__ Pos load_pos(const float* lo, const float* lh, const uint8_t* mask,
                                        int64_t base, int64_t t) {
  return make_pos<VALUES>(lo[base + t], VALUES ? 0.f : lh[base + t], (mask == nullptr) || (mask[base + t] != 0));
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
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t base = static_cast<int64_t>(r) * T;
  const int64_t t_lo = r_lo ? r_lo[r] : 0;
  const int64_t t_hi = r_hi ? r_hi[r] : T - 1;

  // ---- eligibility count (and the optional signed delta) -----------------
  // A staged root also gets the histogram of its keys' top digit here, the
  // first radix pass's, so that pass needs no sweep of its own.
  const bool staged = T <= kStageMax;
  for (int i = tid; i < 2 * 256; i += kThreads) (&sh.hist[0][0])[i] = 0;
  if (tid == 0) sh.n_taken = 0;
  __syncthreads();
  // kBatch positions per thread are loaded (unconditionally, from clamped
  // in-bounds positions) before any is used, so that their memory latencies
  // overlap.
  constexpr int kBatch = 8;
  int c = 0;
  auto first_pass = [&](auto has_mask) {
    constexpr bool kMask = decltype(has_mask)::value;
    for (int64_t t0 = tid; t0 < T; t0 += kBatch * kThreads) {
      float a[kBatch], b[kBatch];
      uint8_t mk[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        int64_t t = t0 + j * kThreads;
        t = t < T ? t : T - 1;
        a[j] = lo[base + t];
        b[j] = VALUES ? 0.f : lh[base + t];
        mk[j] = kMask ? mask[base + t] : uint8_t{1};
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int64_t t = t0 + j * kThreads;
        if (t < T) {
          const Pos p = make_pos<VALUES>(a[j], b[j], mk[j] != 0);
          if (delta_out) delta_out[base + t] = p.delta;
          const bool cand = p.elig && t >= t_lo && t <= t_hi;
          if (staged) {
            sh.staged[t] = cand ? p.key : 0u;
            if (cand) atomicAdd(&sh.hist[0][p.key >> 24], 1);
          }
          c += cand ? 1 : 0;
        }
      }
    }
  };
  if (mask != nullptr) first_pass(std::true_type{});
  else first_pass(std::false_type{});
  c = wave_sum(c);
  if (lane == 0) sh.welig[wave] = c;
  __syncthreads();   // (also publishes the staged keys and the first histogram)
  int n_elig = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) n_elig += sh.welig[i];
  const int kk = n_elig < pool ? n_elig : pool;

  if (kk > 0) {
    // ---- radix select of the kk-th largest score --------------------------
    // Per digit: one sweep adds the positions that match the prefix so far
    // to this digit's histogram (and clears the other one for the next
    // digit), then wave 0 finds the bin in which the count from the top
    // reaches `rank`.
    unsigned prefix = 0, pmask = 0;
    int rank = kk;   // rank of the threshold among positions matching prefix
#pragma unroll
    for (int dg = 0; dg < 4; ++dg) {
      const int shift = 24 - 8 * dg;
      int* hist = sh.hist[dg & 1];
      if (dg > 0 || !staged) {
        if (dg > 0 && tid < 256) sh.hist[(dg + 1) & 1][tid] = 0;
        for (int64_t t0 = tid; t0 < T; t0 += kBatch * kThreads) {
          unsigned key[kBatch];
#pragma unroll
          for (int j = 0; j < kBatch; ++j) {
            const int64_t t = t0 + j * kThreads;
            key[j] = t < T ? cand_key<VALUES>(sh, staged, lo, lh, mask, base, t, t_lo, t_hi) : 0u;
          }
#pragma unroll
          for (int j = 0; j < kBatch; ++j)
            if (key[j] != 0u && (key[j] & pmask) == prefix) atomicAdd(&hist[(key[j] >> shift) & 255], 1);
        }
        __syncthreads();
      }
      if (wave == 0) {
        // lane l holds bins 255 - 4 l - j, j = 0..3 (from the top)
        int h[4], hs = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) { h[j] = hist[255 - 4 * lane - j]; hs += h[j]; }
        int incl = hs;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int u = __shfl_up(incl, o);
          if (lane >= o) incl += u;
        }
        int above = incl - hs;
        if (above < rank && incl >= rank) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (above < rank && above + h[j] >= rank) {
              sh.digit = 255 - 4 * lane - j;
              sh.rank = rank - above;
              sh.n_thr = h[j];
            }
            above += h[j];
          }
        }
      }
      __syncthreads();
      prefix |= static_cast<unsigned>(sh.digit) << shift;
      pmask |= 255u << shift;
      rank = sh.rank;
    }
    const unsigned thr = prefix;   // bit pattern of the kk-th largest score
    const int need_ties = rank;    // positions scoring exactly thr to take
    const bool all_ties = need_ties == sh.n_thr;

    // ---- collect: all above the threshold, then the lowest-indexed ties ---
    // Wave w owns positions [w per_w, (w + 1) per_w), its lanes taking
    // consecutive positions.  When only some of the positions at the
    // threshold are needed, a first sweep counts them per wave range, so
    // every wave knows how many lie at lower positions.  Winners go to
    // slots in any order: the sort below orders them.
    const int64_t per_w = ((T + kWaves - 1) / kWaves + 63) / 64 * 64;
    const int64_t w_beg = wave * per_w;
    const int64_t w_end = w_beg + per_w < T ? w_beg + per_w : T;
    int eq_before = 0;
    if (!all_ties) {
      int n_eq = 0;
      for (int64_t t0 = w_beg; t0 < w_end; t0 += 64) {
        const int64_t t = t0 + lane;
        const unsigned key = t < w_end ? cand_key<VALUES>(sh, staged, lo, lh, mask, base, t, t_lo, t_hi) : 0u;
        n_eq += __popcll(__ballot(key == thr));
      }
      if (lane == 0) sh.weq[wave] = n_eq;
      __syncthreads();
      for (int i = 0; i < wave; ++i) eq_before += sh.weq[i];
    }
    for (int64_t t0 = w_beg; t0 < w_end; t0 += 64) {
      const int64_t t = t0 + lane;
      const unsigned key = t < w_end ? cand_key<VALUES>(sh, staged, lo, lh, mask, base, t, t_lo, t_hi) : 0u;
      // (thr >= 0x00800000, so key == thr implies a candidate)
      const unsigned long long eq = __ballot(key == thr);
      bool take = key > thr;
      if (key == thr) take = all_ties || eq_before + lanes_below(eq) < need_ties;
      eq_before += __popcll(eq);
      const unsigned long long tk = __ballot(take);
      if (tk != 0ull) {
        int slot0 = 0;
        if (lane == 0) slot0 = atomicAdd(&sh.n_taken, __popcll(tk));
        slot0 = __shfl(slot0, 0);
        if (take) {
          const int slot = slot0 + lanes_below(tk);
          if (slot < kThreads)
            sh.keys[slot] = (static_cast<unsigned long long>(key) << 32) |
                            static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<unsigned>(t));
        }
      }
    }
    __syncthreads();

    // ---- sort, descending, of the kk winners on the key (s, ~t) -----------
    // (padding keys are 0, below every real key: a finite score's key is at
    // least 0x00800000, so every real composite key is positive)
    if (kk <= 64) {
      // one wave, one key per lane: a key's place is the number of larger
      // keys (all composite keys differ in t)
      if (wave == 0) {
        const unsigned long long a = lane < kk ? sh.keys[lane] : 0ull;
        int place = 0;
        for (int j = 0; j < kk; ++j) {
          const unsigned hi = static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(a >> 32), j));
          const unsigned lo32 = static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(a), j));
          const unsigned long long bj = (static_cast<unsigned long long>(hi) << 32) | lo32;
          place += bj > a ? 1 : 0;
        }
        if (lane < kk) sh.keys[place] = a;
      }
      __syncthreads();
    } else {
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
