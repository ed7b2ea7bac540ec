// Step 2: threshold block selection, find_blocks (XAttention Sec. 3.2).
//
// find_blocks asks for the smallest set of key blocks whose mass reaches tau.
// Masses are integers u_j = floor(clamp(score_j, 0, 1) * 2^32), so every sum
// below is exact and the result does not depend on summation order; the
// target is ceil(tau * T) with T the row total (one fp64 product).
//
// The same search serves the fixed-size selections of the Top-K / Top-Ratio
// ablation (Sec. 4.5, Table 6) with block counts instead of masses, and
// thresholds may differ per head (the consumer side of Sec. 3.3).
//
// One wave64 per (head, query block) row. Instead of sorting, the wave finds
// the mass v* of the last block the sorted prefix needs: the largest v with
// F(v) = sum_{u_j >= v} u_j >= target (binary search, F non-increasing).
// The shortest prefix of the (u desc, j asc) order that reaches the target is
// then every block with u_j > v* plus the first ceil((target - F(v*+1)) / v*)
// blocks with u_j == v* in ascending j. Emitting in ascending j with ballot /
// popcount yields the index list already sorted. After the first search steps
// the few values still inside the search interval are gathered one per lane,
// so the remaining steps no longer scan every candidate.
#include "common.h"

using namespace xattn;

namespace {

// Sum over the wave, returned uniform (in a scalar register): prefix sums
// inside each row of 16 lanes by DPP row shifts, then the four row totals.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  return __builtin_amdgcn_readlane(x, 15) + __builtin_amdgcn_readlane(x, 31) +
         __builtin_amdgcn_readlane(x, 47) + __builtin_amdgcn_readlane(x, 63);
}

// Exact wave sum of per-lane values below 2^42: the high and low 21-bit parts
// are summed separately (each total stays below 2^27).
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
  const uint32_t hi = wave_sum_u32((uint32_t)(x >> 21));
  const uint32_t lo = wave_sum_u32((uint32_t)x & ((1u << 21) - 1u));
  return ((uint64_t)hi << 21) + lo;
}

constexpr int kFullSteps = 10;  // search steps over every value before narrowing

// One row with at most 64 NPL candidates; lane l holds j = l + 64 i. Every
// per-lane partial sum below is at most NPL * 2^32 <= 2^37.
//   COUNT = false (find_blocks): target = ceil(tau * T), F(v) = sum_{u >= v} u.
//   COUNT = true (Top-K / Top-Ratio): target = k, F(v) = #{u >= v}.
// v* = the largest v with F(v) >= target; the selection is every u > v* plus
// the first ties (u == v*) in ascending j that bring it to the target.
template <int NPL, bool COUNT>
__device__ __forceinline__ void select_row(const float* __restrict__ s, int m, float tau,
                                           int k, int lane, int32_t* __restrict__ out,
                                           int32_t* __restrict__ cnt_out,
                                           uint64_t* __restrict__ stage) {
  uint64_t u[NPL];
  uint64_t tl = 0;
#pragma unroll
  for (int i = 0; i < NPL; ++i) {
    const int j = lane + 64 * i;
    float v = j < m ? s[j] : 0.f;
    v = v > 0.f ? (v < 1.f ? v : 1.f) : 0.f;  // NaN -> 0
    u[i] = (uint64_t)floor((double)v * 4294967296.0);
    tl += u[i];
  }
  uint64_t target;
  if constexpr (COUNT) {
    target = (uint64_t)k;  // 1 <= k < m
  } else {
    const uint64_t T = wave_sum_u64(tl);
    if (T == 0) {  // every candidate has zero mass: the first in (u desc, j asc) order is j = 0
      if (lane == 0) {
        out[0] = 0;
        *cnt_out = 1;
      }
      return;
    }
    const double prod = (double)tau * (double)T;
    target = (uint64_t)ceil(prod);
  }
  auto F = [&](uint64_t v, bool strict) -> uint64_t {
    uint64_t f = 0;
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
      const bool in = strict ? u[i] > v : u[i] >= v;
      f += in ? (COUNT ? 1 : u[i]) : 0;
    }
    return wave_sum_u64(f);
  };

  // largest v in [0, 2^32] with F(v) >= target; F(0) >= target, F(2^32 + 1) = 0
  uint64_t lo = 0, hi = (1ull << 32) + 1;
  for (int it = 0; it < kFullSteps && hi - lo > 1; ++it) {
    const uint64_t mid = (lo + hi) >> 1;
    if (F(mid, false) >= target) lo = mid;
    else hi = mid;
  }
  if (hi - lo > 1) {
    // For v in (lo, hi) only the values in [lo, hi) can change F(v): F(v) =
    // A + sum of those >= v, A = F(hi). When at most 64 remain they are
    // gathered one per lane (through LDS) and the search ends on them alone,
    // visiting the same midpoints with the same F values.
    uint64_t a = 0;
    uint32_t n = 0;
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
      a += u[i] >= hi ? (COUNT ? 1 : u[i]) : 0;
      n += (lane + 64 * i < m && u[i] >= lo && u[i] < hi) ? 1u : 0u;
    }
    if (NPL > 2 && wave_sum_u32(n) <= 64) {
      const uint64_t A = wave_sum_u64(a);
      const uint64_t below = (1ull << lane) - 1ull;
      uint32_t pos = 0;
#pragma unroll
      for (int i = 0; i < NPL; ++i) {
        const bool in = lane + 64 * i < m && u[i] >= lo && u[i] < hi;
        const uint64_t msk = __ballot(in);
        if (in) stage[pos + __popcll(msk & below)] = u[i];
        pos += __popcll(msk);
      }
      __builtin_amdgcn_wave_barrier();
      const uint64_t c = lane < (int)pos ? stage[lane] : 0;  // 0 never counts: v >= 1
      while (hi - lo > 1) {
        const uint64_t mid = (lo + hi) >> 1;
        const uint64_t f = A + wave_sum_u64(c >= mid ? (COUNT ? 1 : c) : 0);
        if (f >= target) lo = mid;
        else hi = mid;
      }
    } else {
      while (hi - lo > 1) {
        const uint64_t mid = (lo + hi) >> 1;
        if (F(mid, false) >= target) lo = mid;
        else hi = mid;
      }
    }
  }
  const uint64_t vstar = lo;
  const uint64_t base = F(vstar, true);  // < target by maximality of v*
  // find_blocks: v* >= 1 because F(1) = T >= target
  const uint64_t ties_needed = COUNT ? target - base : (target - base + vstar - 1) / vstar;

  const uint64_t below = (1ull << lane) - 1ull;
  uint32_t written = 0;
  uint64_t ties_seen = 0;
#pragma unroll
  for (int i = 0; i < NPL; ++i) {
    const int j = lane + 64 * i;
    const bool tie = (j < m) && (u[i] == vstar);
    const uint64_t tmask = __ballot(tie);
    const uint64_t rank = ties_seen + (uint64_t)__popcll(tmask & below);
    const bool sel = (j < m) && (u[i] > vstar || (tie && rank < ties_needed));
    const uint64_t smask = __ballot(sel);
    if (sel) out[written + __popcll(smask & below)] = j;
    written += __popcll(smask);
    ties_seen += __popcll(tmask);
  }
  if (lane == 0) *cnt_out = (int32_t)written;
}

template <int NPL, bool COUNT>
__device__ __forceinline__ void select_row_sized(const float* s, int m, float tau, int k,
                                                 int lane, int32_t* out, int32_t* cnt_out,
                                                 uint64_t* stage) {
  const int nact = (m + 63) >> 6;
  if (NPL <= 1 || nact <= 1) select_row<1, COUNT>(s, m, tau, k, lane, out, cnt_out, stage);
  else if (NPL <= 2 || nact <= 2) select_row<(NPL < 2 ? NPL : 2), COUNT>(s, m, tau, k, lane, out, cnt_out, stage);
  else if (NPL <= 4 || nact <= 4) select_row<(NPL < 4 ? NPL : 4), COUNT>(s, m, tau, k, lane, out, cnt_out, stage);
  else if (NPL <= 8 || nact <= 8) select_row<(NPL < 8 ? NPL : 8), COUNT>(s, m, tau, k, lane, out, cnt_out, stage);
  else if (NPL <= 16 || nact <= 16) select_row<(NPL < 16 ? NPL : 16), COUNT>(s, m, tau, k, lane, out, cnt_out, stage);
  else select_row<NPL, COUNT>(s, m, tau, k, lane, out, cnt_out, stage);
}

// One wave64 per (head, query block) row. NPL = slots per lane for the
// longest row (64 NPL >= NB); a causal row with m = b + 1 candidates runs the
// smallest power-of-two slot count that holds them. Per-head parameters are
// indexed by the row's head modulo hq (the same for every batch element).
template <int NPL, bool CAUSAL>
__global__ __launch_bounds__(256) void select_kernel(const float* __restrict__ scores,
                                                     int n_rows, int NB, SelectParams p,
                                                     int32_t* __restrict__ idx,
                                                     int32_t* __restrict__ cnt) {
  __shared__ uint64_t stage_all[4][64];  // per wave: the values left for the search's end
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;  // uniform per wave
  const int b = row % NB;
  const int hp = p.uniform ? 0 : (row / NB) % p.hq;
  const int m = CAUSAL ? b + 1 : NB;
  const float* s = scores + (size_t)row * NB;
  int32_t* out = idx + (size_t)row * NB;

  int k = m;  // blocks a fixed-size mode keeps
  if (p.mode == kSelectTopK) {
    k = p.k[hp];
  } else if (p.mode == kSelectRatio) {
    const double want = floor((double)p.v[hp] * (double)m + 0.5);
    k = want < 1.0 ? 1 : (want > (double)m ? m : (int)want);
  }
  k = k < 1 ? 1 : k;
  const bool all = p.mode == kSelectThreshold ? p.v[hp] >= 1.f : k >= m;
  if (all) {
    for (int j = lane; j < m; j += 64) out[j] = j;
    if (lane == 0) cnt[row] = m;
    return;
  }
  uint64_t* stage = stage_all[threadIdx.x >> 6];
  if (p.mode == kSelectThreshold)
    select_row_sized<NPL, false>(s, m, p.v[hp], 0, lane, out, cnt + row, stage);
  else
    select_row_sized<NPL, true>(s, m, 0.f, k, lane, out, cnt + row, stage);
}

template <int NPL>
hipError_t launch_npl(const float* scores, const XattnShape& s, const SelectParams& p,
                      int32_t* idx, int32_t* cnt, hipStream_t st) {
  const int n_rows = s.HQ() * s.NB();
  const dim3 grid((n_rows + 3) / 4);
  if (s.causal)
    hipLaunchKernelGGL((select_kernel<NPL, true>), grid, dim3(256), 0, st, scores, n_rows,
                       s.NB(), p, idx, cnt);
  else
    hipLaunchKernelGGL((select_kernel<NPL, false>), grid, dim3(256), 0, st, scores, n_rows,
                       s.NB(), p, idx, cnt);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select(const float* scores, const XattnShape& s, const SelectParams& p,
                         int32_t* idx, int32_t* cnt, hipStream_t st) {
  const int NB = s.NB();
  if (NB <= 64) return launch_npl<1>(scores, s, p, idx, cnt, st);
  if (NB <= 128) return launch_npl<2>(scores, s, p, idx, cnt, st);
  if (NB <= 256) return launch_npl<4>(scores, s, p, idx, cnt, st);
  if (NB <= 512) return launch_npl<8>(scores, s, p, idx, cnt, st);
  if (NB <= 1024) return launch_npl<16>(scores, s, p, idx, cnt, st);
  if (NB <= 2048) return launch_npl<32>(scores, s, p, idx, cnt, st);
  return hipErrorInvalidValue;
}
