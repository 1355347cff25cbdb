// A native consumer of libhdl.so's C ABI (include/hdl.h): plain HIP device
// buffers, no Python or torch.  It runs the re-scoring path on seeded inputs
// and checks properties the results must have whatever the numbers are:
//
//  * log p <= 0 and finite on scored rows, exactly 0 on masked rows (Eq. 1);
//  * roots whose two contexts are identical get |delta| == 0 bit for bit
//    (Eq. 1 uses the same parameters and prefix for both contexts), so their
//    branch points are the first k eligible positions (ties go to the lower
//    position);
//  * every root returns k eligible, distinct positions in (score descending,
//    position ascending) order, with score == |delta| at each (Eq. 2);
//  * argument errors come back synchronously as negative statuses.
//
// Prints "abi_check: ok" and exits 0, or names the first failed check and
// exits 1.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "hdl.h"

namespace {

constexpr int kRoots = 4, kT = 1000, kD = 256, kV = 5000, kK = 4, kSkip = 16;

uint64_t g_state = 0x9e3779b97f4a7c15ull;
double uniform() {   // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return static_cast<double>((g_state * 0x2545f4914f6cdd1dull) >> 11) * (1.0 / 9007199254740992.0);
}
double normal() {
  const double u = uniform() + 1e-300, v = uniform();
  return std::sqrt(-2.0 * std::log(u)) * std::cos(6.283185307179586 * v);
}
uint16_t to_bf16(float f) {   // round to nearest even
  uint32_t x;
  std::memcpy(&x, &f, 4);
  return static_cast<uint16_t>((x + 0x7fffu + ((x >> 16) & 1u)) >> 16);
}

int g_failed = 0;
void check(bool ok, const char* what) {
  if (!ok && !g_failed) {
    std::printf("abi_check: FAILED: %s\n", what);
    g_failed = 1;
  }
}

template <typename T>
T* upload(const std::vector<T>& h) {
  T* d = nullptr;
  if (hipMalloc(&d, h.size() * sizeof(T)) != hipSuccess) return nullptr;
  if (hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice) != hipSuccess) return nullptr;
  return d;
}

}  // namespace

int main() {
  const int64_t n_rows = 2LL * kRoots * kT;   // rows ordered [context][root][t]
  std::vector<uint16_t> w(static_cast<size_t>(kV) * kD), hidden(static_cast<size_t>(n_rows) * kD);
  for (auto& x : w) x = to_bf16(static_cast<float>(0.05 * normal()));
  for (int r = 0; r < kRoots; ++r)
    for (int t = 0; t < kT; ++t)
      for (int j = 0; j < kD; ++j) {
        const float h0 = static_cast<float>(normal());
        // roots 0 and 1: identical contexts; roots 2 and 3: the hindsight state differs
        const float h1 = r < 2 ? h0 : static_cast<float>(h0 + 0.3 * normal());
        hidden[(static_cast<size_t>(r) * kT + t) * kD + j] = to_bf16(h0);
        hidden[(static_cast<size_t>(kRoots + r) * kT + t) * kD + j] = to_bf16(h1);
      }
  std::vector<int32_t> tokens(n_rows);
  std::vector<uint8_t> mask(n_rows), mask_rt(static_cast<size_t>(kRoots) * kT);
  for (int r = 0; r < kRoots; ++r)
    for (int t = 0; t < kT; ++t) {
      const int32_t y = static_cast<int32_t>(uniform() * kV) % kV;
      const uint8_t m = t < kSkip ? 0 : 1;
      tokens[static_cast<size_t>(r) * kT + t] = tokens[static_cast<size_t>(kRoots + r) * kT + t] = y;
      mask[static_cast<size_t>(r) * kT + t] = mask[static_cast<size_t>(kRoots + r) * kT + t] = m;
      mask_rt[static_cast<size_t>(r) * kT + t] = m;
    }

  uint16_t* d_w = upload(w);
  uint16_t* d_h = upload(hidden);
  int32_t* d_tok = upload(tokens);
  uint8_t* d_mask = upload(mask);
  uint8_t* d_mask_rt = upload(mask_rt);
  float *d_logp = nullptr, *d_lse = nullptr, *d_score = nullptr, *d_delta = nullptr;
  int32_t *d_idx = nullptr, *d_count = nullptr;
  void* d_ws = nullptr;
  const size_t ws = hdl_token_logprobs_workspace_size(n_rows, kD, kV, HDL_BF16);
  if (!d_w || !d_h || !d_tok || !d_mask || !d_mask_rt || ws == 0 ||
      hipMalloc(&d_logp, n_rows * 4) != hipSuccess || hipMalloc(&d_lse, n_rows * 4) != hipSuccess ||
      hipMalloc(&d_score, kRoots * kK * 4) != hipSuccess || hipMalloc(&d_delta, kRoots * kT * 4) != hipSuccess ||
      hipMalloc(&d_idx, kRoots * kK * 4) != hipSuccess || hipMalloc(&d_count, kRoots * 4) != hipSuccess ||
      hipMalloc(&d_ws, ws) != hipSuccess) {
    std::printf("abi_check: FAILED: setup (%s)\n", hdl_last_hip_error());
    return 1;
  }

  // argument errors: synchronous, nothing enqueued
  check(hdl_token_logprobs(nullptr, d_w, d_tok, d_mask, n_rows, kD, kV, HDL_BF16, d_logp, d_lse, d_ws, ws,
                           nullptr) == HDL_ERR_INVALID_ARG, "null hidden is an invalid argument");
  check(hdl_token_logprobs(d_h, d_w, d_tok, d_mask, n_rows, kD, kV, HDL_BF16, d_logp, d_lse, d_ws, ws - 1,
                           nullptr) == HDL_ERR_WORKSPACE, "a short workspace is reported");
  check(hdl_select_branch_points(d_logp, d_logp, d_mask_rt, kRoots, kT, 0, d_idx, d_score, d_count, nullptr,
                                 nullptr) == HDL_ERR_INVALID_ARG, "k = 0 is an invalid argument");

  // the path: both contexts in one call, then the per-root selection
  const float* lp0 = d_logp;
  const float* lp1 = d_logp + static_cast<int64_t>(kRoots) * kT;
  check(hdl_token_logprobs(d_h, d_w, d_tok, d_mask, n_rows, kD, kV, HDL_BF16, d_logp, d_lse, d_ws, ws,
                           nullptr) == HDL_OK, "hdl_token_logprobs");
  check(hdl_select_branch_points(lp0, lp1, d_mask_rt, kRoots, kT, kK, d_idx, d_score, d_count, d_delta,
                                 nullptr) == HDL_OK, "hdl_select_branch_points");
  if (hipDeviceSynchronize() != hipSuccess) {
    std::printf("abi_check: FAILED: synchronize\n");
    return 1;
  }
  std::vector<float> logp(n_rows), score(kRoots * kK), delta(kRoots * kT);
  std::vector<int32_t> idx(kRoots * kK), count(kRoots);
  (void)hipMemcpy(logp.data(), d_logp, n_rows * 4, hipMemcpyDeviceToHost);
  (void)hipMemcpy(score.data(), d_score, score.size() * 4, hipMemcpyDeviceToHost);
  (void)hipMemcpy(delta.data(), d_delta, delta.size() * 4, hipMemcpyDeviceToHost);
  (void)hipMemcpy(idx.data(), d_idx, idx.size() * 4, hipMemcpyDeviceToHost);
  (void)hipMemcpy(count.data(), d_count, count.size() * 4, hipMemcpyDeviceToHost);

  for (int64_t n = 0; n < n_rows; ++n) {
    if (mask[n]) check(std::isfinite(logp[n]) && logp[n] <= 0.f, "log p finite and <= 0 on scored rows");
    else check(logp[n] == 0.f, "log p = 0 on masked rows");
  }
  for (int r = 0; r < kRoots; ++r) {
    check(count[r] == kK, "k branch points per root");
    for (int j = 0; j < kK; ++j) {
      const int t = idx[r * kK + j];
      check(t >= kSkip && t < kT, "branch points are eligible positions");
      if (t < kSkip || t >= kT) continue;
      check(score[r * kK + j] == std::fabs(delta[r * kT + t]), "score = |delta| at the branch point");
      if (j > 0) {
        const int tp = idx[r * kK + j - 1];
        const float sp = score[r * kK + j - 1], s = score[r * kK + j];
        check(sp > s || (sp == s && tp < t), "order: score descending, position ascending");
      }
      if (r < 2) check(t == kSkip + j && score[r * kK + j] == 0.f, "identical contexts: first k positions, score 0");
    }
    if (r < 2)
      for (int t = kSkip; t < kT; ++t) check(delta[r * kT + t] == 0.f, "identical contexts: delta == 0 bit for bit");
  }
  (void)hipFree(d_w); (void)hipFree(d_h); (void)hipFree(d_tok); (void)hipFree(d_mask); (void)hipFree(d_mask_rt);
  (void)hipFree(d_logp); (void)hipFree(d_lse); (void)hipFree(d_score); (void)hipFree(d_delta);
  (void)hipFree(d_idx); (void)hipFree(d_count); (void)hipFree(d_ws);
  if (g_failed) return 1;
  std::printf("abi_check: ok (%d roots x 2 contexts x %d positions, d=%d, V=%d, k=%d)\n", kRoots, kT, kD, kV, kK);
  return 0;
}
