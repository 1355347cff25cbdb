// Internal declarations shared by the host-side entry points and the kernel
// translation units of libhdl.so.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "plan.h"

namespace hdl {

struct LmheadArgs {
  const void* hidden;
  const void* w;
  const int32_t* tokens;
  const int32_t* rows;      // compacted scored-row list
  const int32_t* n_scored;  // device-side count of scored rows
  int64_t d;
  int64_t vocab;
  int64_t n_vt, tpc, n_ch, n_grt;
  int64_t part_stride;      // elements between chunk planes of the partials
  float* part_m;            // running max (natural-log units)
  float* part_s;            // sum of exp(z - m)
  float* part_z;            // sampled-token logit, -inf where not captured
  float* part_t;            // sum of exp(z - m) * (z - m), or nullptr (no entropy)
  // Scored rows handled by this launch: rows[0 .. n) with
  // n = clamp(*n_scored - row_base, 0, row_cap) (`rows` already offset).
  int64_t row_base, row_cap;
  // Gradient mode (backward pass): instead of partial statistics, write
  // G[e][v] = g_e (1[v == y_e] - exp(z_ev - lse_e)) as bf16 for scored row e
  // of this launch, columns v < g_cols (zero for v >= vocab), and zero rows
  // for n <= e < round_up(n, 64).  G is stored chunk-major: the 8 entries
  // v = 8c .. 8c+7 of row e are the 16 bytes at element (c * g_ld + e) * 8,
  // so consecutive rows' chunks are adjacent (g_ld >= row_cap).
  const float* lse_in;      // [n_rows] log-sum-exp from the forward pass
  const float* grad_in;     // [n_rows] upstream gradient of log p
  uint16_t* g_out;          // [g_cols / 8][g_ld][8] bf16, or nullptr (statistics mode)
  int64_t g_ld, g_cols;
};

// Plain bf16 GEMM on the same 256 x 256 MFMA tile:
//   C[s][m][n] (=|+=) sum_{k in split s} A(m, k) B(n, k)
// Each operand X (A indexed by m, B by n) is used as stored, in one of:
//   kLayoutKRow    X(i, k) at k * ld + i (row k holds every i; W and hidden
//                  rows for a contraction over the vocabulary or the rows);
//   kLayoutCmRow   X(i, k) at ((k / 8) * ld + i) * 8 + k % 8 (chunk-major
//                  along k: the logit gradient contracted over the vocabulary);
//   kLayoutCmKRow  X(i, k) at ((i / 8) * ld + k) * 8 + i % 8 (chunk-major
//                  along i: the logit gradient contracted over its rows).
// K ranges are multiples of 64.
constexpr int kLayoutKRow = 1, kLayoutCmRow = 2, kLayoutCmKRow = 3;
struct GemmArgs {
  const void* a;
  int64_t lda;
  int a_layout;
  // K-row roles only: stored extent along i (a multiple of 8; reads past it
  // are clamped) and stored K rows (reads of K rows past them are clamped;
  // the other operand must hold zeros at those K).
  int64_t a_cols, a_krows;
  const void* b;
  int64_t ldb;
  int b_layout;
  int64_t b_cols, b_krows;
  int64_t m, n, k;          // sizes (upper bounds when a dimension is dynamic)
  // Dynamic dimension: dyn_dim 1 makes M = clamp(*dyn - dyn_base, 0, m);
  // dyn_dim 2 makes K = round_up(clamp(*dyn - dyn_base, 0, k), 64).
  const int32_t* dyn;
  int64_t dyn_base;
  int dyn_dim;
  int64_t k_split;          // K elements per split (multiple of 64)
  int64_t tiles_m, tiles_n, splits, gm, gn;   // launch grouping (host-computed)
  float* c;
  int64_t ldc, c_split_stride;
  int beta;                 // 0: store, 1: accumulate
};

hipError_t launch_compact(const uint8_t* mask, int64_t n_rows, int32_t* rows,
                          int32_t* n_scored, float* logp, float* lse, float* entropy,
                          hipStream_t stream);
hipError_t launch_lmhead(const LmheadArgs& a, int64_t grid, bool bf16, hipStream_t stream);
hipError_t launch_lmhead_grad(const LmheadArgs& a, int64_t grid, hipStream_t stream);
// Supported layouts (a, b): (kLayoutCmRow, kLayoutKRow), (kLayoutCmKRow, kLayoutCmRow).
hipError_t launch_gemm(const GemmArgs& a, hipStream_t stream);
// Row e < min(round_up(n, 64), cap) of X = (e < n ? in[map[e]][:] : 0), where
// n = clamp(*dyn - dyn_base, 0, cap), stored chunk-major along e:
// X[e][j] at ((e / 8) * d + j) * 8 + e % 8 (kLayoutCmRow with ld = d).
// out holds cap * d bf16; d % 8 == 0, cap % 8 == 0.
hipError_t launch_gather_rows_cm(const uint16_t* in, int64_t ld_in, const int32_t* map, const int32_t* dyn,
                                 int64_t dyn_base, int64_t cap, int64_t d, uint16_t* out, hipStream_t stream);
// dh[map[e]][j] = sum_s part[s][e][j] for e < clamp(*dyn - dyn_base, 0, cap)
hipError_t launch_splitk_scatter(const float* part, int64_t splits, int64_t split_stride, int64_t d,
                                 const int32_t* map, const int32_t* dyn, int64_t dyn_base, int64_t cap,
                                 float* dh, hipStream_t stream);
// dh[n][:] = 0 for rows with mask[n] == 0
hipError_t launch_zero_masked_rows(const uint8_t* mask, int64_t n_rows, int64_t d, float* dh,
                                   hipStream_t stream);
hipError_t launch_merge(const LmheadArgs& a, int64_t n_rows, float* logp, float* lse,
                        float* entropy, hipStream_t stream);
// values == true: rank `lo` itself (lh unused); otherwise rank |lh - lo|.
hipError_t launch_select(const float* lo, const float* lh, const uint8_t* mask,
                         int64_t n_roots, int64_t T, int k, int32_t* idx, float* score,
                         int32_t* count, float* delta, bool values, hipStream_t stream,
                         const int32_t* r_lo = nullptr, const int32_t* r_hi = nullptr, int min_gap = 0,
                         int pool = 0);
// Group construction (group.hip).
hipError_t launch_allocate(const int32_t* idx, const int32_t* count, int64_t n_roots, int k,
                           const int32_t* alloc, int total, int32_t fallback, int32_t* branch_pos,
                           int32_t* branch_rank, hipStream_t stream);
hipError_t launch_advantages(const float* rewards, int64_t n_groups, int group_size, float* adv,
                             hipStream_t stream);
hipError_t launch_policy_grad(const float* adv, const int32_t* traj, const int32_t* pos, const int32_t* start,
                              const float* logp_new, const float* logp_old, const uint8_t* loss_mask,
                              int64_t n_tokens, int64_t n_traj, float eps_low, float eps_high, float scale,
                              float* grad, float* loss, int64_t* n_trained, hipStream_t stream);

}  // namespace hdl
