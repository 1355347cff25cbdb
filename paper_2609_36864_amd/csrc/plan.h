// Work planning of the fused lm-head kernel: how one hdl_token_logprobs call
// is cut into launches and work items, and where the caller's workspace holds
// what.  Everything here depends on the sizes only (never on the mask), so the
// workspace size is known before the call.  Host code and the kernel share
// the work-item mapping below; tests compile this header on the CPU to check
// the arithmetic over wide ranges of sizes.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hdl {

// Fused lm-head tile geometry (see lmhead_logprob.hip).
constexpr int kTileV = 256;              // vocabulary rows per workgroup tile
constexpr int kTileN = 256;              // token rows per workgroup tile
constexpr int kGroupRT = 4;              // row tiles per per-XCD launch group
constexpr int kGroupCH = 32 / kGroupRT;  // vocabulary chunks per per-XCD launch group
constexpr int kNumXcd = 8;               // XCDs per MI355X; workgroups go round-robin
constexpr int kCountBlockRows = 4096;    // rows per block of the compaction's count pass

// How one call is cut up.  A call of n_rows rows runs in launches of at most
// rows_per_launch rows (every hidden-state byte offset of a launch must fit
// in 32 bits: the DMA takes a 64-bit base plus a 32-bit per-lane offset).
// All launches of a call share the vocabulary chunking (tpc, n_ch), so the
// partials of any launch, n_ch planes of at most n_rows rows each, fit the
// workspace sized for the first.
struct LmheadPlan {
  int64_t n_rows;           // rows of the largest launch (upper bound of its scored rows)
  int64_t rows_per_launch;  // a call is cut into launches of at most this many rows
  int64_t n_vt;             // vocabulary tiles of kTileV rows
  int64_t tpc;              // vocabulary tiles per chunk (one work item's span)
  int64_t n_ch;             // vocabulary chunks
  // workspace layout (byte offsets): compacted rows int32 [n_rows] | scored
  // count + count-pass block sums | partials fp32 [planes][n_ch][n_rows]
  size_t off_rows, off_count, off_part, bytes;
  int planes;               // partial planes: max, sum of exp, sampled logit (+ entropy)
};

// Geometry of one launch over n <= plan.n_rows rows.
struct LmheadLaunch {
  int64_t n_rt_max;  // row tiles if every row is scored
  int64_t n_grt;     // row-tile groups
  int64_t n_gch;     // chunk groups
  int64_t grid;      // workgroups launched
};

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline size_t round_up_sz(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Largest number of rows one launch may cover (a multiple of the row tile;
// 0 when a single row tile would already exceed 4 GiB).
inline int64_t rows_per_launch(int64_t d, int esz) {
  const int64_t row_bytes = d * esz;
  return ((int64_t{1} << 32) / row_bytes) / kTileN * kTileN;
}

// Vocabulary tiles per work item for a launch of `rows` rows: long items
// amortise the per-item pipeline fill and partial write, short ones balance
// the tail across 256 CUs.  Aim for about 32 items per CU (measured: at
// 16,384 rows this runs 6 % faster than 8 items per CU; at 65,536 rows both
// give 16 tiles).
inline int64_t default_tpc(int64_t rows, int64_t n_vt) {
  int64_t tpc = ceil_div(rows, kTileN) * n_vt / 8192;
  if (tpc < 1) tpc = 1;
  if (tpc > 16) tpc = 16;
  return tpc;
}

// Workspace layout for launches of at most `rows` rows with n_ch chunks.
inline void layout_workspace(LmheadPlan& p, int64_t rows, int planes) {
  p.n_rows = rows;
  p.planes = planes;
  size_t off = 0;
  p.off_rows = off;
  off = round_up_sz(off + sizeof(int32_t) * static_cast<size_t>(rows), 256);
  p.off_count = off;
  off = round_up_sz(off + sizeof(int32_t) * (64 + static_cast<size_t>(ceil_div(rows, kCountBlockRows))), 256);
  p.off_part = off;
  off = round_up_sz(off + sizeof(float) * static_cast<size_t>(planes) * static_cast<size_t>(p.n_ch) *
                              static_cast<size_t>(rows), 256);
  p.bytes = off;
}

// The plan of a call over n_rows_total rows (4 partial planes: room for the
// entropy accumulator, so one workspace serves both entry points).
inline LmheadPlan make_plan(int64_t n_rows_total, int64_t vocab, int64_t d, int esz) {
  LmheadPlan p{};
  p.rows_per_launch = rows_per_launch(d, esz);
  const int64_t rows = n_rows_total < p.rows_per_launch ? n_rows_total : p.rows_per_launch;
  p.n_vt = ceil_div(vocab, kTileV);
  p.tpc = default_tpc(rows, p.n_vt);
  p.n_ch = ceil_div(p.n_vt, p.tpc);
  layout_workspace(p, rows, 4);
  return p;
}

// The plan of a call whose whole workspace must fit in `total_bytes`, with
// `planes` partial planes: the default chunking where it fits (then the
// results equal those of the default plan bit for bit), else fewer, longer
// chunks.  Returns false when not even one chunk fits.
inline bool make_plan_bounded(int64_t n_rows_total, int64_t vocab, int64_t d, int esz, int planes,
                              size_t total_bytes, LmheadPlan* out) {
  LmheadPlan p{};
  p.rows_per_launch = rows_per_launch(d, esz);
  if (p.rows_per_launch < kTileN) return false;
  const int64_t rows = n_rows_total < p.rows_per_launch ? n_rows_total : p.rows_per_launch;
  p.n_vt = ceil_div(vocab, kTileV);
  // the part of the workspace that does not depend on the chunking
  p.n_ch = 0;
  layout_workspace(p, rows, planes);
  const size_t fixed = p.off_part;
  const size_t per_chunk = sizeof(float) * static_cast<size_t>(planes) * static_cast<size_t>(rows);
  if (total_bytes < fixed + per_chunk) return false;
  const int64_t n_ch_fit = static_cast<int64_t>((total_bytes - fixed) / per_chunk);
  p.tpc = default_tpc(rows, p.n_vt);
  if (ceil_div(p.n_vt, p.tpc) > n_ch_fit) p.tpc = ceil_div(p.n_vt, n_ch_fit);   // fewer, longer chunks
  p.n_ch = ceil_div(p.n_vt, p.tpc);   // <= n_ch_fit
  layout_workspace(p, rows, planes);
  if (p.bytes > total_bytes) return false;
  *out = p;
  return true;
}

// Geometry of one launch over n rows (n <= plan.n_rows) with the call's
// chunking.  Work items are (row tile, chunk) pairs, dealt in groups of
// kGroupRT x kGroupCH per XCD (see work_item).
inline LmheadLaunch plan_launch(const LmheadPlan& p, int64_t n) {
  LmheadLaunch l{};
  l.n_rt_max = ceil_div(n, kTileN);
  l.n_grt = ceil_div(l.n_rt_max, kGroupRT);
  l.n_gch = ceil_div(p.n_ch, kGroupCH);
  const int64_t groups = l.n_grt * l.n_gch;
  l.grid = ceil_div(groups, kNumXcd) * kNumXcd * (kGroupRT * kGroupCH);
  return l;
}

// Work item of workgroup b.  Workgroups are dealt to the XCDs round-robin;
// the j-th workgroup of an XCD belongs to launch group (j / 32) of that XCD,
// and a group is a block of kGroupRT row tiles x kGroupCH vocabulary chunks,
// so the workgroups resident on one XCD at a time share hidden-state and W
// tiles through that XCD's L2.  Items past the problem (row tile >= n_rt or
// chunk >= n_ch) have nothing to do.
__host__ __device__ inline void work_item(int64_t b, int64_t n_grt, int64_t* rt, int64_t* ch) {
  const int64_t xcd = b % kNumXcd;
  const int64_t j = b / kNumXcd;
  const int64_t grp = (j / (kGroupRT * kGroupCH)) * kNumXcd + xcd;
  const int64_t loc = j % (kGroupRT * kGroupCH);
  *rt = (grp % n_grt) * kGroupRT + (loc % kGroupRT);
  *ch = (grp / n_grt) * kGroupCH + (loc / kGroupRT);
}

}  // namespace hdl
