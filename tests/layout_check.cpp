// Host check of the scoring scratch layout (score_rows.h): for the causal
// (packed) and non-causal layouts, every slot the kernels write maps to a
// distinct index inside the buffer that score_scratch_bytes sizes, and the
// slots cover that buffer exactly. Built host-only by tests/test_layout_host.py.
#include <cstdio>
#include <vector>

#include "score_rows.h"

using namespace xattn;

static int check(int HQ, int L, int S, bool causal) {
  const int NB = L / kBlock, nrb = kBlock / S, NR = L / S, NT = (NR + kTsub - 1) / kTsub;
  const size_t np = part_elems(HQ, NB, nrb, causal);
  std::vector<unsigned char> seen(np, 0);
  for (int h = 0; h < HQ; ++h)
    for (int b = 0; b < NB; ++b)
      for (int j = 0; j < (causal ? b + 1 : NB); ++j)
        for (int r = 0; r < nrb; ++r) {
          const size_t i = part_row(h, b, NB, causal) * nrb + (size_t)j * nrb + r;
          if (i >= np || seen[i]++) {
            std::printf("part: slot (%d %d %d %d) -> %zu of %zu\n", h, b, j, r, i, np);
            return 1;
          }
        }
  for (size_t i = 0; i < np; ++i)
    if (!seen[i]) { std::printf("part: index %zu unused\n", i); return 1; }
  const size_t ns = (size_t)HQ * stats_per_head(NR, NT, causal);
  std::vector<unsigned char> sseen(ns, 0);
  for (int h = 0; h < HQ; ++h)
    for (int t = 0; t < NT; ++t)
      for (int R = causal ? kTsub * t : 0; R < NR; ++R) {
        const size_t i = stats_at(h, t, R, NR, NT, causal);
        if (i >= ns || sseen[i]++) {
          std::printf("stats: slot (%d %d %d) -> %zu of %zu\n", h, t, R, i, ns);
          return 1;
        }
      }
  for (size_t i = 0; i < ns; ++i)
    if (!sseen[i]) { std::printf("stats: index %zu unused\n", i); return 1; }
  return 0;
}

int main() {
  const int cases[][3] = {{1, 128, 16}, {2, 1280, 8}, {3, 4736, 4}, {2, 128 * 37, 2},
                          {1, 8192, 64}, {2, 128 * 21, 1}, {1, 32768, 16}};
  for (auto& c : cases)
    for (int causal = 0; causal < 2; ++causal)
      if (check(c[0], c[1], c[2], causal != 0)) {
        std::printf("FAIL HQ=%d L=%d S=%d causal=%d\n", c[0], c[1], c[2], causal);
        return 1;
      }
  std::printf("layout ok\n");
  return 0;
}
