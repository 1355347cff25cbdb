// Internal declarations shared by the host-side entry points and the kernel
// translation units of libhdl.so.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hdl {

// Fused lm-head tile geometry (see lmhead_logprob.hip).
constexpr int kTileV = 256;         // vocabulary rows per workgroup tile
constexpr int kTileN = 256;         // token rows per workgroup tile
#ifndef HDL_GROUP_RT
#define HDL_GROUP_RT 8
#endif
constexpr int kGroupRT = HDL_GROUP_RT;   // row tiles per per-XCD launch group
constexpr int kGroupCH = 32 / kGroupRT; // vocabulary chunks per per-XCD launch group
constexpr int kNumXcd = 8;          // XCDs per MI355X; workgroups go round-robin

// How one hdl_token_logprobs call is cut into work items.  Every quantity
// depends on the sizes only, so the workspace size can be computed up front.
struct LmheadPlan {
  int64_t n_rows;       // rows per launch (upper bound of scored rows)
  int64_t rows_per_launch;  // a call is cut into launches of at most this many rows
  int64_t n_vt;         // vocabulary tiles of kTileV rows
  int64_t tpc;          // vocabulary tiles per chunk (one work item's span)
  int64_t n_ch;         // vocabulary chunks
  int64_t n_rt_max;     // row tiles if every row is scored
  int64_t n_grt;        // row-tile groups
  int64_t n_gch;        // chunk groups
  int64_t grid;         // workgroups launched
  // workspace layout (byte offsets)
  size_t off_rows, off_count, off_part, bytes;
};

// Largest number of rows one launch may cover: every hidden-state byte offset
// of a launch must fit in 32 bits (the DMA uses a 64-bit base + 32-bit offset).
int64_t rows_per_launch(int64_t d, int esz);
LmheadPlan make_plan(int64_t n_rows, int64_t vocab, int64_t d, int esz);

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
  float* part_t;            // sum of exp(z - m) * z, or nullptr (no entropy)
};

hipError_t launch_compact(const uint8_t* mask, int64_t n_rows, int32_t* rows,
                          int32_t* n_scored, float* logp, float* lse, float* entropy,
                          hipStream_t stream);
hipError_t launch_lmhead(const LmheadArgs& a, int64_t grid, bool bf16, hipStream_t stream);
hipError_t launch_merge(const LmheadArgs& a, int64_t n_rows, float* logp, float* lse,
                        float* entropy, hipStream_t stream);
// values == true: rank `lo` itself (lh unused); otherwise rank |lh - lo|.
hipError_t launch_select(const float* lo, const float* lh, const uint8_t* mask,
                         int64_t n_roots, int64_t T, int k, int32_t* idx, float* score,
                         int32_t* count, float* delta, bool values, hipStream_t stream);

}  // namespace hdl
