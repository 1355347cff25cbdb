// CPU check of the fused lm-head kernel's work planning (csrc/plan.h), the
// header the library itself compiles: for a sweep of (n_rows, d, vocab,
// element size) every launch of a call must fit the workspace the call's
// plan sizes (partials of n_ch chunks x launch rows inside one plane), the
// grid must fit a launch, and the workgroup -> (row tile, chunk) mapping
// must cover every work item exactly once.  Built and run by
// tests/test_plan.py; prints one line per failure and "plan_check: ok N".
#include <cstdint>
#include <cstdio>
#include <vector>

#include "../paper_2609_36864_amd/csrc/plan.h"

using namespace hdl;

static int g_fail = 0;
static long g_cases = 0;

#define CHECK(cond, ...)                      \
  do {                                        \
    if (!(cond)) {                            \
      if (g_fail < 50) {                      \
        std::printf("FAIL %s: ", #cond);      \
        std::printf(__VA_ARGS__);             \
        std::printf("\n");                    \
      }                                       \
      ++g_fail;                               \
    }                                         \
  } while (0)

// Every (rt, ch) with rt < n_rt, ch < n_ch is produced by exactly one
// workgroup of the launch; the others fall outside the problem.
static void check_coverage(const LmheadPlan& p, const LmheadLaunch& l) {
  const int64_t n_rt = l.n_rt_max;
  std::vector<int> seen(static_cast<size_t>(n_rt * p.n_ch), 0);
  for (int64_t b = 0; b < l.grid; ++b) {
    int64_t rt, ch;
    work_item(b, l.n_grt, &rt, &ch);
    CHECK(rt >= 0 && ch >= 0, "negative item at b=%lld", (long long)b);
    if (rt < n_rt && ch < p.n_ch) ++seen[static_cast<size_t>(rt * p.n_ch + ch)];
  }
  for (size_t i = 0; i < seen.size(); ++i)
    CHECK(seen[i] == 1, "item %zu covered %d times (n_rt=%lld n_ch=%lld grid=%lld)", i, seen[i],
          (long long)n_rt, (long long)p.n_ch, (long long)l.grid);
}

static void check_call(int64_t n_rows, int64_t d, int64_t vocab, int esz, bool coverage) {
  ++g_cases;
  const int64_t rpl = rows_per_launch(d, esz);
  if (rpl < kTileN) return;   // rejected by the library before planning
  const LmheadPlan p = make_plan(n_rows, vocab, d, esz);
  const size_t plane = static_cast<size_t>(p.n_ch) * static_cast<size_t>(p.n_rows);
  CHECK(p.tpc >= 1 && p.n_ch >= 1 && p.tpc * p.n_ch >= p.n_vt && (p.n_ch - 1) * p.tpc < p.n_vt,
        "chunking n_vt=%lld tpc=%lld n_ch=%lld", (long long)p.n_vt, (long long)p.tpc, (long long)p.n_ch);
  CHECK(p.off_part + sizeof(float) * 4 * plane <= p.bytes, "partials exceed the workspace");
  CHECK(p.off_count + sizeof(int32_t) * (64 + ceil_div(p.n_rows, kCountBlockRows)) <= p.off_part,
        "count scratch overlaps the partials");
  CHECK(p.off_rows + sizeof(int32_t) * p.n_rows <= p.off_count, "row list overlaps the counts");
  for (int64_t r0 = 0; r0 < n_rows; r0 += p.rows_per_launch) {
    const int64_t n = n_rows - r0 < p.rows_per_launch ? n_rows - r0 : p.rows_per_launch;
    const LmheadLaunch l = plan_launch(p, n);
    CHECK(n <= p.n_rows, "launch rows %lld > plan rows %lld", (long long)n, (long long)p.n_rows);
    CHECK(static_cast<size_t>(p.n_ch) * static_cast<size_t>(n) <= plane,
          "n_rows=%lld d=%lld V=%lld esz=%d: launch at %lld needs %lld x %lld partials, plane %zu",
          (long long)n_rows, (long long)d, (long long)vocab, esz, (long long)r0, (long long)p.n_ch,
          (long long)n, plane);
    CHECK(l.grid <= INT32_MAX && l.grid > 0, "grid %lld", (long long)l.grid);
    // hidden-state byte offsets of a launch stay below 4 GiB
    CHECK(n * d * esz <= (int64_t{1} << 32), "launch spans %lld bytes", (long long)(n * d * esz));
    if (coverage) check_coverage(p, l);
  }
}

static void check_bounded(int64_t n_rows, int64_t d, int64_t vocab, int esz, size_t total) {
  ++g_cases;
  LmheadPlan p{};
  if (!make_plan_bounded(n_rows, vocab, d, esz, 3, total, &p)) {
    // must really not fit: the fixed part plus one chunk exceeds the bound
    const int64_t rpl = rows_per_launch(d, esz);
    if (rpl < kTileN) return;
    const int64_t rows = n_rows < rpl ? n_rows : rpl;
    LmheadPlan q{};
    q.n_ch = 1;
    layout_workspace(q, rows, 3);
    CHECK(q.bytes > total, "bounded plan refused a call that fits (rows=%lld)", (long long)rows);
    return;
  }
  CHECK(p.bytes <= total, "bounded plan of %zu bytes exceeds %zu", p.bytes, total);
  CHECK(p.tpc * p.n_ch >= p.n_vt && (p.n_ch - 1) * p.tpc < p.n_vt, "bounded chunking");
  const LmheadPlan def = make_plan(n_rows, vocab, d, esz);
  CHECK(p.n_ch <= def.n_ch, "bounded plan has more chunks than the default");
  // where the default chunking fits, the bounded plan keeps it
  LmheadPlan def3 = def;
  layout_workspace(def3, def.n_rows, 3);
  if (def3.bytes <= total) CHECK(p.tpc == def.tpc && p.n_ch == def.n_ch, "bounded plan changed a chunking that fits");
  const size_t plane = static_cast<size_t>(p.n_ch) * static_cast<size_t>(p.n_rows);
  for (int64_t r0 = 0; r0 < n_rows; r0 += p.rows_per_launch) {
    const int64_t n = n_rows - r0 < p.rows_per_launch ? n_rows - r0 : p.rows_per_launch;
    CHECK(static_cast<size_t>(p.n_ch) * static_cast<size_t>(n) <= plane, "bounded launch overflows");
    CHECK(p.off_part + sizeof(float) * 3 * plane <= p.bytes, "bounded partials exceed the workspace");
  }
}

int main() {
  // The case that overflowed when every launch re-planned its own chunking:
  // bf16, V = 32000, d = 5120 -> 419,328 rows per launch; the 26,880-row
  // remainder launch would get 125 chunks (3,360,000 partials) against a
  // plane of 8 x 419,328 = 3,354,624.
  {
    const LmheadPlan p = make_plan(446208, 32000, 5120, 2);
    const LmheadPlan tail = make_plan(446208 - p.rows_per_launch, 32000, 5120, 2);
    CHECK(p.rows_per_launch == 419328, "rows per launch %lld", (long long)p.rows_per_launch);
    CHECK(static_cast<size_t>(tail.n_ch) * static_cast<size_t>(tail.n_rows) >
              static_cast<size_t>(p.n_ch) * static_cast<size_t>(p.n_rows),
          "the remainder launch's own chunking no longer exceeds the plane (update this example)");
    check_call(446208, 5120, 32000, 2, false);
  }
  const int64_t ds[] = {8, 24, 72, 256, 2048, 2056, 4096, 5120, 8192, 12288, 16384, 65536};
  const int64_t vs[] = {1, 2, 255, 257, 4096, 32000, 151936, 152064, 262400};
  for (int esz : {2, 4})
    for (int64_t d : ds)
      for (int64_t v : vs) {
        const int64_t rpl = rows_per_launch(d, esz);
        std::vector<int64_t> ns = {1, 255, 256, 257, 4096, 65536, 65537, 131072, 524288};
        if (rpl >= kTileN) {
          for (int64_t m : {int64_t{1}, int64_t{2}, int64_t{3}}) {
            ns.push_back(m * rpl - 1);
            ns.push_back(m * rpl);
            ns.push_back(m * rpl + 1);
            ns.push_back(m * rpl + 26880);
          }
        }
        for (int64_t n : ns) {
          if (n <= 0 || n > INT32_MAX) continue;
          check_call(n, d, v, esz, n <= 65537 && v <= 32000);
          check_bounded(n, d, v, esz, size_t{32} << 20);
          check_bounded(n, d, v, esz, size_t{1} << 20);
        }
      }
  // exhaustive coverage on small grids
  for (int64_t n = 1; n <= 5000; n += 37)
    for (int64_t v : {1, 300, 2000, 9000}) check_call(n, 64, v, 2, true);
  if (g_fail) {
    std::printf("plan_check: %d failures in %ld cases\n", g_fail, g_cases);
    return 1;
  }
  std::printf("plan_check: ok %ld\n", g_cases);
  return 0;
}
