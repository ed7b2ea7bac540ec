// Scoring scratch layout and the per-row finalisation of the block scores
// (XAttention Sec. 3.2, Algorithm 1: reduced-row softmax, then the mean over
// each query block's B/S reduced rows of the per-key-block sums). Used by the
// scoring kernels (score.hip); the layout functions are host-callable too.
#pragma once

#include "common.h"

namespace xattn {

constexpr int kTsub = 128;      // reduced-column sub-tile owning one (max, sum) per row
constexpr int kStatMax = 2048;  // (row, sub-tile) stats staged in LDS (16 KB) when they fit
constexpr int kFinUnroll = 4;   // independent 16-byte partial-sum loads per thread
constexpr int kFinThreads = 256;

// Partial block masses, fp32: row (h, query block b) holds nrb floats per key
// block j, j < b + 1 when causal (the rows packed as a lower triangle), j <
// NB otherwise; element (h, b, j, r) at part_row(h, b) * nrb + j * nrb + r.
__host__ __device__ inline size_t part_row(int h, int b, int NB, bool causal) {
  return causal ? (size_t)h * ((size_t)NB * (NB + 1) / 2) + (size_t)b * (b + 1) / 2
                : ((size_t)h * NB + b) * NB;
}
__host__ __device__ inline size_t part_elems(int HQ, int NB, int nrb, bool causal) {
  return part_row(HQ, 0, NB, causal) * nrb;
}

// Row statistics (max, sum) per reduced row R and column sub-tile t, float2.
// Causal: only sub-tiles that start at or before the row (t * kTsub <= R)
// are kept, sub-tile t holding rows t * kTsub .. NR - 1; otherwise every
// (t, R). NT = ceil(NR / kTsub).
__host__ __device__ inline size_t stats_per_head(int NR, int NT, bool causal) {
  return causal ? (size_t)NT * NR - (size_t)kTsub * NT * (NT - 1) / 2 : (size_t)NT * NR;
}
__host__ __device__ inline size_t stats_at(int h, int t, int R, int NR, int NT, bool causal) {
  const size_t head = (size_t)h * stats_per_head(NR, NT, causal);
  return causal ? head + (size_t)t * NR - (size_t)kTsub * t * (t - 1) / 2 + (R - kTsub * t)
                : head + (size_t)t * NR + R;
}

__device__ __forceinline__ float fin_wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}
__device__ __forceinline__ float fin_wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// LDS of one finalisation (one workgroup of kFinThreads per row).
struct FinalizeLds {
  float mR[kBlock], ilR[kBlock];
  float sm[kStatMax], sl[kStatMax];  // sm[t * nrb + r]: m, then the factor f
};

// Block scores of row (h, b), nrb = B/S reduced rows R = b nrb + r and tn
// column sub-tiles per row:
//   m_R = max_t m[t][R],  l_R = sum_t l[t][R] 2^(m[t][R] - m_R),
//   f[r][t] = 2^(m[t][R] - m_R) / l_R,
//   out[j] = (1/nrb) sum_r part[j][r] f[r][t(j)]   for the candidates j,
//   out[j] = 0 for the other j < NB (causal: j > b).
// The (r, t) stats are read r-fastest (the nrb rows of one sub-tile are
// adjacent in memory) into LDS; one wave per reduced row reduces them in a
// fixed order. The row's partial-sum slab [j][r] is streamed as float4 (or
// float2 when nrb = 2), kFinUnroll loads in flight per thread; the nrb / 4
// lanes of one block then reduce with shuffles in a fixed order. Rows whose
// stats exceed the LDS stage use the same arithmetic with the stats read from
// global memory. Called by all kFinThreads threads of the workgroup.
template <bool CAUSAL>
__device__ __forceinline__ void finalize_row(const float* __restrict__ part,
                                             const float2* __restrict__ stats, int NR, int NB,
                                             int NT, int nrb, int h, int b,
                                             float* __restrict__ out, FinalizeLds& L) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int ncand = CAUSAL ? b + 1 : NB;
  const int tn = CAUSAL ? (b * nrb) / kTsub + 1 : NT;  // sub-tiles of this row's stats
  const int R0 = b * nrb;
  auto st = [&](int t, int r) -> float2 { return stats[stats_at(h, t, R0 + r, NR, NT, CAUSAL)]; };
  const bool staged = nrb * tn <= kStatMax;
  if (staged) {
    for (int i = tid; i < nrb * tn; i += kFinThreads) {
      const int t = i / nrb, r = i - t * nrb;
      const float2 v = st(t, r);
      L.sm[i] = v.x;
      L.sl[i] = v.y;
    }
    __syncthreads();
  }
  for (int r = wv; r < nrb; r += kFinThreads / 64) {
    float m = -INFINITY;
    for (int t = lane; t < tn; t += 64) m = fmaxf(m, staged ? L.sm[t * nrb + r] : st(t, r).x);
    m = fin_wave_max(m);
    float l = 0.f;
    for (int t = lane; t < tn; t += 64) {
      const float2 v = staged ? make_float2(L.sm[t * nrb + r], L.sl[t * nrb + r]) : st(t, r);
      l += v.y * fast_exp2(v.x - m);
    }
    l = fin_wave_sum(l);
    if (lane == 0) {
      L.mR[r] = m;
      L.ilR[r] = 1.f / l;
    }
  }
  __syncthreads();
  if (staged) {
    for (int i = tid; i < nrb * tn; i += kFinThreads) {
      const int r = i % nrb;
      L.sm[i] = fast_exp2(L.sm[i] - L.mR[r]) * L.ilR[r];
    }
    __syncthreads();
  }
  auto factor = [&](int r, int t) -> float {
    return staged ? L.sm[t * nrb + r] : fast_exp2(st(t, r).x - L.mR[r]) * L.ilR[r];
  };

  const float inv_nrb = 1.f / (float)nrb;
  const float* pb = part + part_row(h, b, NB, CAUSAL) * nrb;  // this row's slab [j][r]
  if (nrb >= 4) {
    // chunk q = 4 consecutive floats = rows 4 (q % (nrb/4)) .. +3 of block q / (nrb/4)
    const int cpb = nrb / 4;  // chunks (lanes) per block, a power of two <= 32
    const int nq = ncand * cpb;
    const float4* p4 = (const float4*)pb;
    for (int q0 = 0; q0 < nq; q0 += kFinThreads * kFinUnroll) {
      float4 v[kFinUnroll];
#pragma unroll
      for (int u = 0; u < kFinUnroll; ++u) {
        const int q = q0 + kFinThreads * u + tid;
        v[u] = q < nq ? p4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < kFinUnroll; ++u) {
        const int q = q0 + kFinThreads * u + tid;
        const int j = q / cpb, r0 = 4 * (q % cpb);
        const int t = (j * nrb) / kTsub;
        float acc = 0.f;
        if (q < nq)
          acc = v[u].x * factor(r0, t) + v[u].y * factor(r0 + 1, t) +
                v[u].z * factor(r0 + 2, t) + v[u].w * factor(r0 + 3, t);
        for (int off = cpb / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
        if (q < nq && (q % cpb) == 0) out[j] = acc * inv_nrb;
      }
    }
  } else {  // nrb == 2: one float2 per block
    const float2* p2 = (const float2*)pb;
    for (int j0 = 0; j0 < ncand; j0 += kFinThreads * kFinUnroll) {
      float2 v[kFinUnroll];
#pragma unroll
      for (int u = 0; u < kFinUnroll; ++u) {
        const int j = j0 + kFinThreads * u + tid;
        v[u] = j < ncand ? p2[j] : make_float2(0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < kFinUnroll; ++u) {
        const int j = j0 + kFinThreads * u + tid;
        if (j < ncand) {
          const int t = (j * nrb) / kTsub;
          out[j] = (v[u].x * factor(0, t) + v[u].y * factor(1, t)) * inv_nrb;
        }
      }
    }
  }
  for (int j = ncand + tid; j < NB; j += kFinThreads) out[j] = 0.f;  // not candidates
}

}  // namespace xattn
