// Minimum-threshold prediction (XAttention Sec. 3.3): the dynamic program
// over heads and threshold adjustments. Host code; the per-head performance
// table comes from the caller (e.g. the output error of each head at each
// adjusted threshold, measured with xattn_head_error).
//
// D[h][m] = best total performance with exactly m adjustments over heads
// 0 .. h-1, each adjustment lowering one head's threshold by 10 %. Head h
// takes a = 0 .. min(m, A) adjustments on top of D[h-1][m-a]; a = 0 or 1 is
// the paper's two-way recurrence (A = 1). On equal values the smaller a is
// kept. The configuration of D[H][M] is traced back.
#include <cmath>
#include <cstdio>
#include <limits>
#include <vector>

#include "xattn.h"

namespace xattn_host {
int fail(int code, const char* fmt, ...);
}

namespace {

// Validates the table shape shared by the dynamic-program entry points.
int check_table(const double* table, int heads, int max_adjust, int adjustments) {
  using xattn_host::fail;
  if (!table) return fail(XATTN_ERR_ARG, "the per-head table must be non-NULL");
  if (heads < 1 || max_adjust < 1)
    return fail(XATTN_ERR_ARG, "heads (%d) and max_adjust (%d) must be >= 1", heads, max_adjust);
  if ((long long)heads * (max_adjust + 1) > (1ll << 26) ||
      (long long)heads * max_adjust > (1ll << 20))
    return fail(XATTN_ERR_UNSUPPORTED, "table of %d heads x %d adjustments too large", heads,
                max_adjust);
  if (adjustments < 0 || adjustments > heads * max_adjust)
    return fail(XATTN_ERR_ARG, "adjustments (%d) must lie in [0, heads * max_adjust = %d]",
                adjustments, heads * max_adjust);
  for (long long i = 0; i < (long long)heads * (max_adjust + 1); ++i)
    if (!std::isfinite(table[i]))
      return fail(XATTN_ERR_ARG, "table entry %lld is not finite", i);
  return XATTN_OK;
}

// D[h][m] over heads in index order; value(h, a) is head h's performance
// after a adjustments (sign = +1: the table itself, -1: minus an error
// table). Fills adjust[] and returns D[H][M].
double run_dp(const double* table, double sign, int heads, int A, int M, int32_t* adjust) {
  const double NEG = -std::numeric_limits<double>::infinity();
  std::vector<double> prev(M + 1, NEG), cur(M + 1);
  std::vector<int32_t> take((size_t)heads * (M + 1));
  prev[0] = 0.0;
  for (int h = 0; h < heads; ++h) {
    const double* row = table + (size_t)h * (A + 1);
    int32_t* th = take.data() + (size_t)h * (M + 1);
    for (int m = 0; m <= M; ++m) {
      double bestv = NEG;
      int arg = 0;
      const int amax = m < A ? m : A;
      for (int a = 0; a <= amax; ++a) {
        if (prev[m - a] == NEG) continue;
        const double v = prev[m - a] + sign * row[a];
        if (v > bestv) {
          bestv = v;
          arg = a;
        }
      }
      cur[m] = bestv;
      th[m] = arg;
    }
    prev.swap(cur);
  }
  int m = M;
  for (int h = heads - 1; h >= 0; --h) {
    adjust[h] = take[(size_t)h * (M + 1) + m];
    m -= adjust[h];
  }
  return prev[M];
}

// The threshold after a reductions of 10 %: tau0 * 0.9^a in fp64, rounded
// once to the fp32 value the selection receives.
float level(double tau0, int a) { return (float)(tau0 * std::pow(0.9, (double)a)); }

}  // namespace

extern "C" int xattn_threshold_dp(const double* perf, int heads, int max_adjust,
                                  int adjustments, int32_t* adjust, double* best) {
  using xattn_host::fail;
  if (!perf || !adjust) return fail(XATTN_ERR_ARG, "perf and adjust must be non-NULL");
  if (int rc = check_table(perf, heads, max_adjust, adjustments)) return rc;
  const double v = run_dp(perf, 1.0, heads, max_adjust, adjustments, adjust);
  if (best) *best = v;
  return XATTN_OK;
}

extern "C" int xattn_threshold_levels(double tau0, int max_adjust, float* levels) {
  using xattn_host::fail;
  if (!levels) return fail(XATTN_ERR_ARG, "levels must be non-NULL");
  if (!(tau0 > 0.0) || !std::isfinite(tau0))
    return fail(XATTN_ERR_ARG, "tau0 must be finite and > 0 (got %g)", tau0);
  if (max_adjust < 0 || max_adjust > (1 << 20))
    return fail(XATTN_ERR_ARG, "max_adjust (%d) must lie in [0, 2^20]", max_adjust);
  for (int a = 0; a <= max_adjust; ++a) levels[a] = level(tau0, a);
  return XATTN_OK;
}

extern "C" int xattn_threshold_predict(const double* err, int heads, int max_adjust,
                                       int adjustments, double tau0, int32_t* adjust,
                                       float* tau_h, double* total_err) {
  using xattn_host::fail;
  if (!err || !adjust || !tau_h)
    return fail(XATTN_ERR_ARG, "err, adjust and tau_h must be non-NULL");
  if (!(tau0 > 0.0) || !std::isfinite(tau0))
    return fail(XATTN_ERR_ARG, "tau0 must be finite and > 0 (got %g)", tau0);
  if (int rc = check_table(err, heads, max_adjust, adjustments)) return rc;
  const double v = run_dp(err, -1.0, heads, max_adjust, adjustments, adjust);
  for (int h = 0; h < heads; ++h) tau_h[h] = level(tau0, adjust[h]);
  if (total_err) *total_err = -v;
  return XATTN_OK;
}
