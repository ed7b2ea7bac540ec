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

extern "C" int xattn_threshold_dp(const double* perf, int heads, int max_adjust,
                                  int adjustments, int32_t* adjust, double* best) {
  using xattn_host::fail;
  if (!perf || !adjust) return fail(XATTN_ERR_ARG, "perf and adjust must be non-NULL");
  if (heads < 1 || max_adjust < 1)
    return fail(XATTN_ERR_ARG, "heads (%d) and max_adjust (%d) must be >= 1", heads, max_adjust);
  if ((long long)heads * (max_adjust + 1) > (1ll << 26) ||
      (long long)heads * max_adjust > (1ll << 20))
    return fail(XATTN_ERR_UNSUPPORTED, "table of %d heads x %d adjustments too large", heads,
                max_adjust);
  if (adjustments < 0 || adjustments > heads * max_adjust)
    return fail(XATTN_ERR_ARG, "adjustments (%d) must lie in [0, heads * max_adjust = %d]",
                adjustments, heads * max_adjust);
  const int A = max_adjust, M = adjustments;
  for (long long i = 0; i < (long long)heads * (A + 1); ++i)
    if (!std::isfinite(perf[i]))
      return fail(XATTN_ERR_ARG, "perf[%lld] is not finite", i);

  const double NEG = -std::numeric_limits<double>::infinity();
  std::vector<double> prev(M + 1, NEG), cur(M + 1);
  std::vector<int32_t> take((size_t)heads * (M + 1));
  prev[0] = 0.0;
  for (int h = 0; h < heads; ++h) {
    const double* row = perf + (size_t)h * (A + 1);
    int32_t* th = take.data() + (size_t)h * (M + 1);
    for (int m = 0; m <= M; ++m) {
      double bestv = NEG;
      int arg = 0;
      const int amax = m < A ? m : A;
      for (int a = 0; a <= amax; ++a) {
        if (prev[m - a] == NEG) continue;
        const double v = prev[m - a] + row[a];
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
  if (best) *best = prev[M];
  return XATTN_OK;
}
