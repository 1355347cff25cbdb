// Host side of libhdl.so: argument validation, work planning, workspace
// layout and kernel launches behind the C ABI declared in include/hdl.h.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "../../include/hdl.h"
#include "hdl_internal.h"

// ---- the allocation-free entry point's scratch ---------------------------
// A fixed device array holds hdl_token_logprobs_noalloc's workspace (the
// compacted row list, the scored-row count and the chunk partials), so that
// callers that cannot allocate (code under graph capture, serving loops)
// still get the fused path.  Every GPU the library runs on holds its own
// copy until the process ends.  Its host-side name is not a device address:
// the address is taken once per device with hipGetSymbolAddress and only
// that address is passed to kernels.  Nothing in it needs clearing between
// calls: every call writes each element it reads first.  Calls that overlap
// on one GPU (different streams or threads) share it and race.

constexpr size_t kScratchBytes = size_t{32} << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(HDL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---- kernel timing (measurement tools only) ------------------------------
// Kinds: HDL_PROFILE_LMHEAD (fused lm-head kernel, statistics or entropy),
// HDL_PROFILE_GRAD (its gradient mode), HDL_PROFILE_GEMM (backward GEMMs),
// HDL_PROFILE_SELECT (the per-root selection kernel).
constexpr int kProfileKinds = 4;
using EventPair = std::pair<hipEvent_t, hipEvent_t>;
struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<EventPair> pending[kProfileKinds];
  std::vector<EventPair> spare;
};
Profiler g_prof;

// A timed launch: start() records the first event on the stream if timing
// is on, stop() the second one and files the pair under its kind.
struct TimedLaunch {
  EventPair ev{nullptr, nullptr};
  bool timed = false;
  hipError_t start(hipStream_t s) {
    {
      std::lock_guard<std::mutex> lk(g_prof.mu);
      if (!g_prof.on) return hipSuccess;
      if (!g_prof.spare.empty()) {
        ev = g_prof.spare.back();
        g_prof.spare.pop_back();
      } else {
        hipError_t e = hipEventCreate(&ev.first);
        if (e == hipSuccess) e = hipEventCreate(&ev.second);
        if (e != hipSuccess) return e;
      }
      timed = true;
    }
    return hipEventRecord(ev.first, s);
  }
  hipError_t stop(int kind, hipStream_t s) {
    if (!timed) return hipSuccess;
    hipError_t e = hipEventRecord(ev.second, s);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lk(g_prof.mu);
    g_prof.pending[kind].push_back(ev);
    return hipSuccess;
  }
};

}  // namespace


extern "C" {

size_t hdl_token_logprobs_workspace_size(int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype) {
  if (n_rows <= 0 || d <= 0 || vocab <= 0 || n_rows > INT32_MAX || vocab > INT32_MAX) return 0;
  if (dtype != HDL_F32 && dtype != HDL_BF16) return 0;
  const int esz = dtype == HDL_BF16 ? 2 : 4;
  if (hdl::rows_per_launch(d, esz) < hdl::kTileN) return 0;
  return hdl::make_plan(n_rows, vocab, d, esz).bytes;
}

}  // extern "C"

namespace {

// Argument checks shared by the log-probability entry points; on success
// *esz is the element size.  Nothing is launched.
int check_stats_args(const char* fn, const void* hidden, const void* w_vocab, const int32_t* tokens,
                     float* logp, int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype, int* esz) {
  if (!hidden || !w_vocab || !tokens || !logp)
    return fail(HDL_ERR_INVALID_ARG, "%s: null hidden, w_vocab, tokens or logp", fn);
  if (n_rows <= 0 || d <= 0 || vocab <= 0)
    return fail(HDL_ERR_INVALID_ARG, "%s: sizes must be positive (n_rows=%lld d=%lld vocab=%lld)",
                fn, static_cast<long long>(n_rows), static_cast<long long>(d), static_cast<long long>(vocab));
  if (n_rows > INT32_MAX || vocab > INT32_MAX)
    return fail(HDL_ERR_UNSUPPORTED, "%s: n_rows and vocab must fit in int32", fn);
  if (dtype != HDL_F32 && dtype != HDL_BF16)
    return fail(HDL_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
  if (d % 8 != 0)
    return fail(HDL_ERR_UNSUPPORTED, "%s: d=%lld is not a multiple of 8", fn, static_cast<long long>(d));
  if (!aligned(hidden, 16) || !aligned(w_vocab, 16))
    return fail(HDL_ERR_INVALID_ARG, "%s: hidden and w_vocab must be 16-byte aligned", fn);
  *esz = dtype == HDL_BF16 ? 2 : 4;
  if (hdl::rows_per_launch(d, *esz) < hdl::kTileN)
    return fail(HDL_ERR_UNSUPPORTED, "%s: hidden rows larger than 16 MiB", fn);
  return HDL_OK;
}

// Shared implementation of the log-probability entry points: compaction,
// fused kernel and merge for each launch of the call, in the workspace `ws`
// laid out by `plan`.  `timed`: bracket the fused kernel with the timing
// hook's events when it is on.
int token_stats(const char* fn, const void* hidden, const void* w_vocab, const int32_t* tokens,
                const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab, int esz, int dtype,
                float* logp, float* lse_out, float* entropy, const hdl::LmheadPlan& plan, char* ws,
                bool timed, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* rows = reinterpret_cast<int32_t*>(ws + plan.off_rows);
  int32_t* n_scored = reinterpret_cast<int32_t*>(ws + plan.off_count);
  float* part = reinterpret_cast<float*>(ws + plan.off_part);
  const size_t plane = static_cast<size_t>(plan.n_ch) * static_cast<size_t>(plan.n_rows);
  const int64_t row_bytes = d * esz;
  if (entropy && plan.planes < 4) return fail(HDL_ERR_UNSUPPORTED, "%s: no entropy plane in the plan", fn);

  // Launches of at most plan.rows_per_launch rows each (one launch for every
  // configuration up to 4 GiB of hidden states), all with the call's
  // vocabulary chunking, so every launch's partials fit the planes.  Checked
  // for every launch before anything is enqueued.
  for (int64_t r0 = 0; r0 < n_rows; r0 += plan.rows_per_launch) {
    const int64_t n = (n_rows - r0) < plan.rows_per_launch ? (n_rows - r0) : plan.rows_per_launch;
    if (n > plan.n_rows || static_cast<size_t>(plan.n_ch) * static_cast<size_t>(n) > plane ||
        hdl::plan_launch(plan, n).grid > INT32_MAX)
      return fail(HDL_ERR_UNSUPPORTED, "%s: a launch of %lld rows does not fit the plan", fn,
                  static_cast<long long>(n));
  }
  for (int64_t r0 = 0; r0 < n_rows; r0 += plan.rows_per_launch) {
    const int64_t n = (n_rows - r0) < plan.rows_per_launch ? (n_rows - r0) : plan.rows_per_launch;
    const hdl::LmheadLaunch lp = hdl::plan_launch(plan, n);
    float* logp_c = logp + r0;
    float* lse_c = lse_out ? lse_out + r0 : nullptr;
    float* ent_c = entropy ? entropy + r0 : nullptr;
    hipError_t e = hdl::launch_compact(mask ? mask + r0 : nullptr, n, rows, n_scored, logp_c, lse_c, ent_c, s);
    if (e != hipSuccess) return hip_fail(e, "compaction launch");

    hdl::LmheadArgs a{};
    a.hidden = static_cast<const char*>(hidden) + r0 * row_bytes;
    a.w = w_vocab;
    a.tokens = tokens + r0;
    a.rows = rows;
    a.n_scored = n_scored;
    a.d = d;
    a.vocab = vocab;
    a.n_vt = plan.n_vt;
    a.tpc = plan.tpc;
    a.n_ch = plan.n_ch;
    a.n_grt = lp.n_grt;
    a.part_stride = n;
    a.part_m = part;
    a.part_s = part + plane;
    a.part_z = part + 2 * plane;
    a.part_t = entropy ? part + 3 * plane : nullptr;
    a.row_base = 0;
    a.row_cap = n;

    TimedLaunch tl;
    if (timed && (e = tl.start(s)) != hipSuccess) return hip_fail(e, "timing event");
    e = hdl::launch_lmhead(a, lp.grid, dtype == HDL_BF16, s);
    if (e != hipSuccess) return hip_fail(e, "lm-head kernel launch");
    if ((e = tl.stop(HDL_PROFILE_LMHEAD, s)) != hipSuccess) return hip_fail(e, "timing event");
    e = hdl::launch_merge(a, n, logp_c, lse_c, ent_c, s);
    if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
  }
  return HDL_OK;
}

// The workspace entry points: the caller's workspace, the default plan.
int token_stats_ws(const char* fn, const void* hidden, const void* w_vocab, const int32_t* tokens,
                   const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype, float* logp,
                   float* lse_out, float* entropy, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error[0] = '\0';
  int esz = 0;
  int st = check_stats_args(fn, hidden, w_vocab, tokens, logp, n_rows, d, vocab, dtype, &esz);
  if (st != HDL_OK) return st;
  const hdl::LmheadPlan plan = hdl::make_plan(n_rows, vocab, d, esz);
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(HDL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given",
                fn, plan.bytes, workspace ? workspace_bytes : static_cast<size_t>(0));
  if (!aligned(workspace, 256))
    return fail(HDL_ERR_INVALID_ARG, "%s: workspace must be 256-byte aligned", fn);
  return token_stats(fn, hidden, w_vocab, tokens, mask, n_rows, d, vocab, esz, dtype, logp, lse_out, entropy,
                     plan, static_cast<char*>(workspace), true, stream);
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

int scratch_on_current_device(const char* fn, char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(HDL_ERR_UNSUPPORTED, "%s: device %d", fn, dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || !aligned(p, 256)) return fail(HDL_ERR_HIP, "%s: scratch address %p", fn, p);
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return HDL_OK;
}

}  // namespace

extern "C" {

int hdl_token_logprobs(const void* hidden, const void* w_vocab, const int32_t* tokens,
                       const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype,
                       float* logp, float* lse_out, void* workspace, size_t workspace_bytes,
                       void* stream) {
  return token_stats_ws("hdl_token_logprobs", hidden, w_vocab, tokens, mask, n_rows, d, vocab, dtype,
                        logp, lse_out, nullptr, workspace, workspace_bytes, stream);
}

int hdl_token_logprobs_entropy(const void* hidden, const void* w_vocab, const int32_t* tokens,
                               const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab,
                               hdl_dtype dtype, float* logp, float* lse_out, float* entropy,
                               void* workspace, size_t workspace_bytes, void* stream) {
  if (!entropy) {
    g_last_error[0] = '\0';
    return fail(HDL_ERR_INVALID_ARG, "hdl_token_logprobs_entropy: null entropy");
  }
  return token_stats_ws("hdl_token_logprobs_entropy", hidden, w_vocab, tokens, mask, n_rows, d, vocab,
                        dtype, logp, lse_out, entropy, workspace, workspace_bytes, stream);
}

int hdl_token_logprobs_noalloc(const void* hidden, const void* w_vocab, const int32_t* tokens,
                               const uint8_t* mask, int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype,
                               float* logp, float* lse_out, void* stream) {
  const char* fn = "hdl_token_logprobs_noalloc";
  g_last_error[0] = '\0';
  int esz = 0;
  int st = check_stats_args(fn, hidden, w_vocab, tokens, logp, n_rows, d, vocab, dtype, &esz);
  if (st != HDL_OK) return st;
  hdl::LmheadPlan plan{};
  if (!hdl::make_plan_bounded(n_rows, vocab, d, esz, 3, kScratchBytes, &plan))
    return fail(HDL_ERR_UNSUPPORTED,
                "%s: a launch of %lld rows needs more than the library's fixed %zu-byte scratch "
                "(16 bytes per row of a launch: at most about %zu rows)",
                fn, static_cast<long long>(n_rows < hdl::rows_per_launch(d, esz) ? n_rows : hdl::rows_per_launch(d, esz)),
                kScratchBytes, (kScratchBytes - 4096) / 16);
  char* ws = nullptr;
  if ((st = scratch_on_current_device(fn, &ws)) != HDL_OK) return st;
  return token_stats(fn, hidden, w_vocab, tokens, mask, n_rows, d, vocab, esz, dtype, logp, lse_out, nullptr,
                     plan, ws, false, stream);
}

int hdl_select_branch_points(const float* logp_orig, const float* logp_hind, const uint8_t* mask,
                             int64_t n_roots, int64_t T, int32_t k, int32_t* idx, float* score,
                             int32_t* count, float* delta_signed, void* stream) {
  g_last_error[0] = '\0';
  if (!logp_orig || !logp_hind || !idx || !score || !count)
    return fail(HDL_ERR_INVALID_ARG, "hdl_select_branch_points: null required pointer");
  if (n_roots <= 0 || T <= 0)
    return fail(HDL_ERR_INVALID_ARG, "hdl_select_branch_points: n_roots and T must be positive");
  if (k < 1)
    return fail(HDL_ERR_INVALID_ARG, "hdl_select_branch_points: k=%d must be >= 1", k);
  if (k > HDL_MAX_K)
    return fail(HDL_ERR_UNSUPPORTED, "hdl_select_branch_points: k=%d exceeds %d", k, HDL_MAX_K);
  if (n_roots > INT32_MAX || T > INT32_MAX)
    return fail(HDL_ERR_UNSUPPORTED, "hdl_select_branch_points: n_roots and T must fit in int32");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch tl;
  hipError_t e = tl.start(s);
  if (e != hipSuccess) return hip_fail(e, "timing event");
  e = hdl::launch_select(logp_orig, logp_hind, mask, n_roots, T, k, idx, score, count, delta_signed,
                         false, s);
  if (e != hipSuccess) return hip_fail(e, "selection kernel launch");
  if ((e = tl.stop(HDL_PROFILE_SELECT, s)) != hipSuccess) return hip_fail(e, "timing event");
  return HDL_OK;
}

int hdl_select_top_k(const float* values, const uint8_t* mask, int64_t n_roots, int64_t T,
                     int32_t k, int32_t* idx, float* score, int32_t* count, void* stream) {
  g_last_error[0] = '\0';
  if (!values || !idx || !score || !count)
    return fail(HDL_ERR_INVALID_ARG, "hdl_select_top_k: null required pointer");
  if (n_roots <= 0 || T <= 0)
    return fail(HDL_ERR_INVALID_ARG, "hdl_select_top_k: n_roots and T must be positive");
  if (k < 1) return fail(HDL_ERR_INVALID_ARG, "hdl_select_top_k: k=%d must be >= 1", k);
  if (k > HDL_MAX_K) return fail(HDL_ERR_UNSUPPORTED, "hdl_select_top_k: k=%d exceeds %d", k, HDL_MAX_K);
  if (n_roots > INT32_MAX || T > INT32_MAX)
    return fail(HDL_ERR_UNSUPPORTED, "hdl_select_top_k: n_roots and T must fit in int32");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch tl;
  hipError_t e = tl.start(s);
  if (e != hipSuccess) return hip_fail(e, "timing event");
  e = hdl::launch_select(values, nullptr, mask, n_roots, T, k, idx, score, count, nullptr, true, s);
  if (e != hipSuccess) return hip_fail(e, "selection kernel launch");
  if ((e = tl.stop(HDL_PROFILE_SELECT, s)) != hipSuccess) return hip_fail(e, "timing event");
  return HDL_OK;
}

const char* hdl_status_string(int status) {
  switch (status) {
    case HDL_OK: return "ok";
    case HDL_ERR_INVALID_ARG: return "invalid argument";
    case HDL_ERR_UNSUPPORTED: return "unsupported argument";
    case HDL_ERR_WORKSPACE: return "workspace missing or too small";
    case HDL_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* hdl_last_hip_error(void) { return g_last_error; }

int hdl_abi_version(void) { return 6; }

int hdl_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = on != 0;
  return HDL_OK;
}

int hdl_profile_read(double* total_ms, int64_t* launches) {
  return hdl_profile_read_kind(HDL_PROFILE_LMHEAD, total_ms, launches);
}

int hdl_profile_read_kind(int kind, double* total_ms, int64_t* launches) {
  if (kind < 0 || kind >= kProfileKinds) return fail(HDL_ERR_INVALID_ARG, "hdl_profile_read_kind: kind %d", kind);
  std::lock_guard<std::mutex> lk(g_prof.mu);
  double tot = 0.0;
  int64_t n = 0;
  for (auto& ev : g_prof.pending[kind]) {
    hipError_t e = hipEventSynchronize(ev.second);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, ev.first, ev.second);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    tot += ms;
    ++n;
    g_prof.spare.push_back(ev);
  }
  g_prof.pending[kind].clear();
  if (total_ms) *total_ms = tot;
  if (launches) *launches = n;
  return HDL_OK;
}

}  // extern "C"

// ---- backward pass --------------------------------------------------------
namespace {

// How one hdl_token_logprobs_backward call is cut up.  Scored rows are taken
// in chunks of `nc`; the gradient with respect to the logits, G [nc][v_pad]
// (bf16), exists for one chunk at a time, never more.
struct BwdPlan {
  int64_t nc, v_pad, n_chunks;
  int64_t splits, k_split;      // vocabulary split of the dH contraction
  hdl::LmheadPlan fwd;          // gradient-mode lm-head launches (nc rows)
  size_t off_rows, off_count, off_g, off_hc, off_hpart, bytes;
};

constexpr int64_t kBwdChunkRows = 32768;
// The GEMMs address a 64-row K-slice of W or of the gathered hidden rows
// with 32-bit byte offsets; vocabulary indices stay well inside int32.
constexpr int64_t kBwdMaxVocab = int64_t{1} << 30;
constexpr int64_t kBwdMaxD = int64_t{1} << 23;

BwdPlan make_bwd_plan(int64_t n_rows, int64_t vocab, int64_t d) {
  BwdPlan p{};
  p.nc = n_rows < kBwdChunkRows ? static_cast<int64_t>(round_up(static_cast<size_t>(n_rows), 256))
                                : kBwdChunkRows;
  p.v_pad = static_cast<int64_t>(round_up(static_cast<size_t>(vocab), 64));
  p.n_chunks = (n_rows + p.nc - 1) / p.nc;
  // dH = G W has nc/256 x d/256 output tiles; split the vocabulary so that
  // about 512 workgroups run.
  const int64_t tiles = (p.nc / hdl::kTileN) * ((d + hdl::kTileN - 1) / hdl::kTileN);
  int64_t s = (512 + tiles - 1) / tiles;
  s = s < 1 ? 1 : (s > 8 ? 8 : s);
  const int64_t slices = p.v_pad / 64;
  if (s > slices) s = slices;
  p.k_split = (slices + s - 1) / s * 64;
  p.splits = (p.v_pad + p.k_split - 1) / p.k_split;
  p.fwd = hdl::make_plan(p.nc, vocab, d, 2);
  size_t off = 0;
  p.off_rows = off;
  off = round_up(off + sizeof(int32_t) * static_cast<size_t>(n_rows), 256);
  p.off_count = off;
  off = round_up(off + sizeof(int32_t) * (64 + static_cast<size_t>(hdl::ceil_div(n_rows, hdl::kCountBlockRows))), 256);
  p.off_g = off;    // G chunk-major [v_pad / 8][nc][8] bf16
  off = round_up(off + 2 * static_cast<size_t>(p.nc) * static_cast<size_t>(p.v_pad), 256);
  p.off_hc = off;   // the chunk's scored hidden rows, gathered chunk-major [nc / 8][d][8] bf16
  off = round_up(off + 2 * static_cast<size_t>(p.nc) * static_cast<size_t>(d), 256);
  p.off_hpart = off;   // dH partial sums [splits][nc][d] fp32
  off = round_up(off + 4 * static_cast<size_t>(p.splits) * static_cast<size_t>(p.nc) * static_cast<size_t>(d), 256);
  p.bytes = off;
  return p;
}

// Arguments of C = sum_k A(m, k) B(n, k): A is the chunk-major logit
// gradient (layout a_layout), B is W stored with K as its row (kLayoutKRow)
// or the gathered hidden rows, chunk-major along K (kLayoutCmRow).
hdl::GemmArgs gemm_args(const void* a, int64_t lda, int a_layout, int64_t a_cols, int64_t a_krows, const void* b,
                        int64_t ldb, int b_layout, int64_t b_cols, int64_t b_krows, int64_t m, int64_t n, int64_t k, float* c,
                        int64_t ldc) {
  hdl::GemmArgs g{};
  g.a = a;
  g.lda = lda;
  g.a_layout = a_layout;
  g.a_cols = a_cols;
  g.a_krows = a_krows;
  g.b = b;
  g.ldb = ldb;
  g.b_layout = b_layout;
  g.b_cols = b_cols;
  g.b_krows = b_krows;
  g.m = m;
  g.n = n;
  g.k = k;
  g.k_split = k;
  g.splits = 1;
  g.tiles_m = (m + hdl::kTileV - 1) / hdl::kTileV;
  g.tiles_n = (n + hdl::kTileN - 1) / hdl::kTileN;
  g.gn = g.tiles_n < 4 ? g.tiles_n : 4;
  g.gm = 32 / g.gn;
  g.c = c;
  g.ldc = ldc;
  return g;
}

}  // namespace

extern "C" {

size_t hdl_token_logprobs_backward_workspace_size(int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype) {
  if (n_rows <= 0 || d <= 0 || vocab <= 0 || n_rows > INT32_MAX || vocab > INT32_MAX) return 0;
  if (dtype != HDL_BF16 || d % 8 != 0) return 0;
  if (vocab > kBwdMaxVocab || d > kBwdMaxD) return 0;
  const int64_t rpl = hdl::rows_per_launch(d, 2);
  if (rpl < hdl::kTileN) return 0;
  return make_bwd_plan(n_rows < rpl ? n_rows : rpl, vocab, d).bytes;
}

int hdl_token_logprobs_backward(const void* hidden, const void* w_vocab, const int32_t* tokens,
                                const uint8_t* mask, const float* lse, const float* grad_logp,
                                int64_t n_rows, int64_t d, int64_t vocab, hdl_dtype dtype, float* grad_hidden,
                                float* grad_w, int accumulate_w, void* workspace, size_t workspace_bytes,
                                void* stream) {
  const char* fn = "hdl_token_logprobs_backward";
  g_last_error[0] = '\0';
  if (!hidden || !w_vocab || !tokens || !lse || !grad_logp || !grad_hidden || !grad_w)
    return fail(HDL_ERR_INVALID_ARG, "%s: null required pointer", fn);
  if (n_rows <= 0 || d <= 0 || vocab <= 0)
    return fail(HDL_ERR_INVALID_ARG, "%s: sizes must be positive (n_rows=%lld d=%lld vocab=%lld)", fn,
                static_cast<long long>(n_rows), static_cast<long long>(d), static_cast<long long>(vocab));
  if (n_rows > INT32_MAX || vocab > INT32_MAX)
    return fail(HDL_ERR_UNSUPPORTED, "%s: n_rows and vocab must fit in int32", fn);
  if (dtype != HDL_BF16) return fail(HDL_ERR_UNSUPPORTED, "%s: only bf16 inputs are supported", fn);
  if (d % 8 != 0)
    return fail(HDL_ERR_UNSUPPORTED, "%s: d=%lld is not a multiple of 8", fn, static_cast<long long>(d));
  if (vocab > kBwdMaxVocab || d > kBwdMaxD)
    return fail(HDL_ERR_UNSUPPORTED, "%s: vocab must not exceed %lld and d %lld", fn,
                static_cast<long long>(kBwdMaxVocab), static_cast<long long>(kBwdMaxD));
  // Rows are taken in blocks whose hidden states span at most 4 GiB (the
  // kernels address a block's rows with 32-bit byte offsets).
  const int64_t rpl = hdl::rows_per_launch(d, 2);
  if (rpl < hdl::kTileN) return fail(HDL_ERR_UNSUPPORTED, "%s: d=%lld too large", fn, static_cast<long long>(d));
  if (!aligned(hidden, 16) || !aligned(w_vocab, 16) || !aligned(grad_hidden, 16) || !aligned(grad_w, 16))
    return fail(HDL_ERR_INVALID_ARG, "%s: hidden, w_vocab, grad_hidden and grad_w must be 16-byte aligned", fn);
  const int64_t block_rows = n_rows < rpl ? n_rows : rpl;
  const BwdPlan plan = make_bwd_plan(block_rows, vocab, d);
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(HDL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, plan.bytes,
                workspace ? workspace_bytes : static_cast<size_t>(0));
  if (!aligned(workspace, 256)) return fail(HDL_ERR_INVALID_ARG, "%s: workspace must be 256-byte aligned", fn);
  const hdl::LmheadLaunch grad_launch = hdl::plan_launch(plan.fwd, plan.nc);
  if (grad_launch.grid > INT32_MAX) return fail(HDL_ERR_UNSUPPORTED, "%s: problem too large for one launch", fn);

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  int32_t* rows = reinterpret_cast<int32_t*>(ws + plan.off_rows);
  int32_t* n_scored = reinterpret_cast<int32_t*>(ws + plan.off_count);
  uint16_t* g = reinterpret_cast<uint16_t*>(ws + plan.off_g);
  uint16_t* hc = reinterpret_cast<uint16_t*>(ws + plan.off_hc);
  float* hpart = reinterpret_cast<float*>(ws + plan.off_hpart);

  hipError_t e = hipSuccess;
  for (int64_t b0 = 0; b0 < n_rows; b0 += block_rows) {
    // one block of rows: every pointer below is offset to the block
    const int64_t nb = n_rows - b0 < block_rows ? n_rows - b0 : block_rows;
    const uint8_t* mask_b = mask ? mask + b0 : nullptr;
    const void* hidden_b = static_cast<const char*>(hidden) + b0 * d * 2;
    const int32_t* tokens_b = tokens + b0;
    const float* lse_b = lse + b0;
    const float* grad_b = grad_logp + b0;
    float* dh_b = grad_hidden + b0 * d;
    if ((e = hdl::launch_compact(mask_b, nb, rows, n_scored, nullptr, nullptr, nullptr, s)) != hipSuccess)
      return hip_fail(e, "compaction launch");
    if ((e = hdl::launch_zero_masked_rows(mask_b, nb, d, dh_b, s)) != hipSuccess)
      return hip_fail(e, "row clearing launch");
    const int64_t n_chunks = (nb + plan.nc - 1) / plan.nc;
    for (int64_t c = 0; c < n_chunks; ++c) {
      const int64_t base = c * plan.nc;
      // 1. G for this chunk's scored rows (logits recomputed tile by tile)
      hdl::LmheadArgs a{};
      a.hidden = hidden_b;
      a.w = w_vocab;
      a.tokens = tokens_b;
      a.rows = rows + base;
      a.n_scored = n_scored;
      a.d = d;
      a.vocab = vocab;
      a.n_vt = plan.fwd.n_vt;
      a.tpc = plan.fwd.tpc;
      a.n_ch = plan.fwd.n_ch;
      a.n_grt = grad_launch.n_grt;
      a.row_base = base;
      a.row_cap = plan.nc;
      a.lse_in = lse_b;
      a.grad_in = grad_b;
      a.g_out = g;
      a.g_ld = plan.nc;   // chunk-major: nc rows per 8-column plane
      a.g_cols = plan.v_pad;
      TimedLaunch tg_;
      if ((e = tg_.start(s)) != hipSuccess) return hip_fail(e, "timing event");
      if ((e = hdl::launch_lmhead_grad(a, grad_launch.grid, s)) != hipSuccess)
        return hip_fail(e, "gradient kernel launch");
      if ((e = tg_.stop(HDL_PROFILE_GRAD, s)) != hipSuccess) return hip_fail(e, "timing event");
      // 2. the chunk's scored hidden rows, gathered chunk-major along the row
      // index (zeros up to the next 64 rows)
      if ((e = hdl::launch_gather_rows_cm(static_cast<const uint16_t*>(hidden_b), d, rows + base, n_scored, base,
                                          plan.nc, d, hc, s)) != hipSuccess)
        return hip_fail(e, "row gather launch");
      // 3. dH rows of the chunk: G W (W read as stored, K = vocabulary rows past
      // V clamped: G is zero there), split along the vocabulary, partials summed in order
      hdl::GemmArgs gh = gemm_args(g, plan.nc, hdl::kLayoutCmRow, 0, 0, w_vocab, d, hdl::kLayoutKRow, d, vocab,
                                   plan.nc, d, plan.v_pad, hpart, d);
      gh.dyn = n_scored;
      gh.dyn_base = base;
      gh.dyn_dim = 1;
      gh.k_split = plan.k_split;
      gh.splits = plan.splits;
      gh.c_split_stride = plan.nc * d;
      TimedLaunch th_;
      if ((e = th_.start(s)) != hipSuccess) return hip_fail(e, "timing event");
      if ((e = hdl::launch_gemm(gh, s)) != hipSuccess) return hip_fail(e, "GEMM launch");
      if ((e = th_.stop(HDL_PROFILE_GEMM, s)) != hipSuccess) return hip_fail(e, "timing event");
      if ((e = hdl::launch_splitk_scatter(hpart, plan.splits, plan.nc * d, d, rows + base, n_scored, base,
                                          plan.nc, dh_b, s)) != hipSuccess)
        return hip_fail(e, "split-K sum launch");
      // 4. dW (+)= G^T H over the chunk's rows (both read with the row index as
      // K); the call's first chunk overwrites dW unless the caller accumulates
      hdl::GemmArgs gw = gemm_args(g, plan.nc, hdl::kLayoutCmKRow, plan.v_pad, plan.nc, hc, d, hdl::kLayoutCmRow, 0,
                                   0, vocab, d, plan.nc, grad_w, d);
      gw.dyn = n_scored;
      gw.dyn_base = base;
      gw.dyn_dim = 2;
      gw.beta = (b0 > 0 || c > 0 || accumulate_w) ? 1 : 0;
      TimedLaunch tw_;
      if ((e = tw_.start(s)) != hipSuccess) return hip_fail(e, "timing event");
      if ((e = hdl::launch_gemm(gw, s)) != hipSuccess) return hip_fail(e, "GEMM launch");
      if ((e = tw_.stop(HDL_PROFILE_GEMM, s)) != hipSuccess) return hip_fail(e, "timing event");
    }
  }
  return HDL_OK;
}

}  // extern "C"

// ---- branch-point constraints and group construction ---------------------
extern "C" {

int hdl_select_constrained(const float* a, const float* b, const uint8_t* mask, int64_t n_roots, int64_t T,
                           int32_t k, const int32_t* lo, const int32_t* hi, int32_t min_gap, int refill,
                           int32_t* idx, float* score, int32_t* count, void* stream) {
  const char* fn = "hdl_select_constrained";
  g_last_error[0] = '\0';
  if (!a || !idx || !score || !count) return fail(HDL_ERR_INVALID_ARG, "%s: null required pointer", fn);
  if (n_roots <= 0 || T <= 0) return fail(HDL_ERR_INVALID_ARG, "%s: n_roots and T must be positive", fn);
  if (k < 1) return fail(HDL_ERR_INVALID_ARG, "%s: k=%d must be >= 1", fn, k);
  if (k > HDL_MAX_K) return fail(HDL_ERR_UNSUPPORTED, "%s: k=%d exceeds %d", fn, k, HDL_MAX_K);
  if (n_roots > INT32_MAX || T > INT32_MAX)
    return fail(HDL_ERR_UNSUPPORTED, "%s: n_roots and T must fit in int32", fn);
  if (min_gap < 0) return fail(HDL_ERR_INVALID_ARG, "%s: min_gap=%d must be >= 0", fn, min_gap);
  const int pool = refill ? HDL_MAX_K : k;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  TimedLaunch tl;
  hipError_t e = tl.start(s);
  if (e != hipSuccess) return hip_fail(e, "timing event");
  e = hdl::launch_select(a, b, mask, n_roots, T, k, idx, score, count, nullptr, b == nullptr, s, lo,
                         hi, min_gap, pool);
  if (e != hipSuccess) return hip_fail(e, "selection kernel launch");
  if ((e = tl.stop(HDL_PROFILE_SELECT, s)) != hipSuccess) return hip_fail(e, "timing event");
  return HDL_OK;
}

int hdl_allocate_continuations(const int32_t* idx, const int32_t* count, int64_t n_roots, int32_t k,
                               const int32_t* alloc, int32_t fallback_pos, int32_t* branch_pos,
                               int32_t* branch_rank, void* stream) {
  const char* fn = "hdl_allocate_continuations";
  g_last_error[0] = '\0';
  if (!idx || !count || !alloc || !branch_pos) return fail(HDL_ERR_INVALID_ARG, "%s: null required pointer", fn);
  if (n_roots <= 0 || k < 1) return fail(HDL_ERR_INVALID_ARG, "%s: n_roots and k must be positive", fn);
  if (k > 16) return fail(HDL_ERR_UNSUPPORTED, "%s: k=%d exceeds 16 branch points per root", fn, k);
  if (n_roots > INT32_MAX) return fail(HDL_ERR_UNSUPPORTED, "%s: n_roots must fit in int32", fn);
  int64_t total = 0;
  for (int j = 0; j < k; ++j) {
    if (alloc[j] < 0) return fail(HDL_ERR_INVALID_ARG, "%s: alloc[%d]=%d is negative", fn, j, alloc[j]);
    total += alloc[j];
  }
  if (total < 1 || total > 4096)
    return fail(HDL_ERR_INVALID_ARG, "%s: %lld continuations per root (1 .. 4096)", fn, static_cast<long long>(total));
  hipError_t e = hdl::launch_allocate(idx, count, n_roots, k, alloc, static_cast<int>(total), fallback_pos,
                                      branch_pos, branch_rank, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "allocation kernel launch");
  return HDL_OK;
}

int hdl_group_advantages(const float* rewards, int64_t n_groups, int32_t group_size, float* adv, void* stream) {
  const char* fn = "hdl_group_advantages";
  g_last_error[0] = '\0';
  if (!rewards || !adv) return fail(HDL_ERR_INVALID_ARG, "%s: null required pointer", fn);
  if (n_groups <= 0 || group_size <= 0)
    return fail(HDL_ERR_INVALID_ARG, "%s: n_groups and group_size must be positive", fn);
  if (n_groups > INT32_MAX) return fail(HDL_ERR_UNSUPPORTED, "%s: n_groups must fit in int32", fn);
  hipError_t e = hdl::launch_advantages(rewards, n_groups, group_size, adv, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "advantage kernel launch");
  return HDL_OK;
}

int hdl_policy_loss_grad(const float* adv, int64_t n_traj, const int32_t* traj, const int32_t* pos,
                         const int32_t* start, const float* logp_new, const float* logp_old,
                         const uint8_t* loss_mask, int64_t n_tokens, float eps_low, float eps_high, float scale,
                         float* grad_logp, float* loss, int64_t* n_trained, void* stream) {
  const char* fn = "hdl_policy_loss_grad";
  g_last_error[0] = '\0';
  if (!adv || !traj || !logp_new || !logp_old || !grad_logp)
    return fail(HDL_ERR_INVALID_ARG, "%s: null required pointer", fn);
  if ((pos == nullptr) != (start == nullptr))
    return fail(HDL_ERR_INVALID_ARG, "%s: pos and start must be given together", fn);
  if (n_traj <= 0 || n_tokens <= 0) return fail(HDL_ERR_INVALID_ARG, "%s: sizes must be positive", fn);
  if (n_tokens > (int64_t{1} << 38)) return fail(HDL_ERR_UNSUPPORTED, "%s: too many tokens", fn);
  if (!(eps_low >= 0.f) || !(eps_high >= 0.f)) return fail(HDL_ERR_INVALID_ARG, "%s: negative clip range", fn);
  if (scale != scale) return fail(HDL_ERR_INVALID_ARG, "%s: scale is NaN", fn);
  if (!(scale > 0.f) && !n_trained)
    return fail(HDL_ERR_INVALID_ARG, "%s: scale <= 0 (token-level mean) needs n_trained", fn);
  if (n_trained && !aligned(n_trained, 8)) return fail(HDL_ERR_INVALID_ARG, "%s: n_trained must be 8-byte aligned", fn);
  hipError_t e = hdl::launch_policy_grad(adv, traj, pos, start, logp_new, logp_old, loss_mask, n_tokens, n_traj,
                                         eps_low, eps_high, scale, grad_logp, loss, n_trained,
                                         static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "policy-gradient kernel launch");
  return HDL_OK;
}

}  // extern "C"
