// Step 1: strided antidiagonal block scoring (XAttention Sec. 3.2, Algorithm 1).
//
// The reshapes of Algorithm 1 make reduced row R of Q~ the concatenation
// (along features) of query rows R*S + S-1, ..., R*S and reduced column c of
// K~ the concatenation of key rows c*S, ..., c*S + S-1, so
//   X[R][c] = q~_R . k~_c = sum_{t<S} q[R*S + S-1-t] . k[c*S + t],
// the sum over the antidiagonal of the S x S sub-block (R, c) of Q K^T.
// K~ is a plain view of K ([L/S][S*d], row c at K + c*S*d) and Q~ a view of Q
// with the S sub-rows reversed: no data is moved to build either.
//
// Kernel score_partials computes X^T = K~ Q~^T tile by tile on bf16 MFMA
// (fp32 accumulate) and, in its epilogue, per reduced row R and 128-column
// tile t: the tile max m (log2 domain), l = sum exp2(x - m), and per key
// block j the partial mass sum_{c in j} exp2(x - m). Kernel score_finalize
// merges the tiles of each row (m_R = max_t m, l_R = sum_t l e^(m - m_R)),
// normalises, and averages the B/S reduced rows of each query block.
#include "common.h"

using namespace xattn;

namespace {

constexpr int TR = 128;              // reduced rows per workgroup tile
constexpr int TC = 128;              // reduced columns per workgroup tile
constexpr int KC = 64;               // reduced-K chunk staged through LDS
constexpr int LDS_STRIDE = KC + 8;   // bf16 per LDS row (16-byte pad vs bank conflicts)
constexpr int kThreads = 256;

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ void tri_decode(int t, int& rt, int& ct) {
  int r = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while (r * (r + 1) / 2 > t) --r;
  while ((r + 1) * (r + 2) / 2 <= t) ++r;
  rt = r;
  ct = t - r * (r + 1) / 2;
}

// NRB = reduced rows (and columns) per 128-token block = 128 / S.
template <int NRB, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void score_partials(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int hq, int hkv, int L,
    int NR, int NB, int NT, int tiles_per_head, int n_work, float scale_log2,
    float* __restrict__ part, float2* __restrict__ stats) {
  constexpr int S = kBlock / NRB;
  constexpr int KD = S * kHeadDim;  // reduced inner dimension S*d
  constexpr int NCH = KD / KC;
  __shared__ __attribute__((aligned(16))) uint16_t As[TC * LDS_STRIDE];  // K~ rows (c)
  __shared__ __attribute__((aligned(16))) uint16_t Bs[TR * LDS_STRIDE];  // Q~ rows (R)

  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, lr = lane & 31, lh = lane >> 5;

  // logical order: (kv head, row tile, column tile, query head in group)
  const int w = xcd_remap(blockIdx.x, n_work);
  const int G = hq / hkv;
  const int hh = w % G;
  const int rest = w / G;
  const int tile = rest % tiles_per_head;
  const int gidx = rest / tiles_per_head;
  const int h = (gidx / hkv) * hq + (gidx % hkv) * G + hh;
  int rt, ct;
  if (CAUSAL) {
    tri_decode(tile, rt, ct);
  } else {
    rt = tile / NT;
    ct = tile % NT;
  }
  const int R0 = rt * TR, c0 = ct * TC;
  const uint16_t* Qh = q + (size_t)h * L * kHeadDim;
  const uint16_t* Kg = k + (size_t)gidx * L * kHeadDim;

  // ---- global -> register staging of one K-chunk: 4 + 4 16-byte pieces per thread
  u32x4 ra[4], rb[4];
  auto fetch = [&](int ch) {
    const int kap0 = ch * KC;
    const int tsub = kap0 / kHeadDim, e0 = kap0 % kHeadDim;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = tid + kThreads * i;
      const int row = p >> 3, col = (p & 7) * 8;
      const int c = c0 + row, R = R0 + row;
      ra[i] = c < NR ? *(const u32x4*)(Kg + (size_t)c * KD + kap0 + col) : u32x4{0, 0, 0, 0};
      rb[i] = R < NR ? *(const u32x4*)(Qh + ((size_t)R * S + (S - 1 - tsub)) * kHeadDim + e0 + col)
                     : u32x4{0, 0, 0, 0};
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = tid + kThreads * i;
      const int row = p >> 3, col = (p & 7) * 8;
      *(u32x4*)&As[row * LDS_STRIDE + col] = ra[i];
      *(u32x4*)&Bs[row * LDS_STRIDE + col] = rb[i];
    }
  };

  f32x16 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x16{};

  // Diagonal tile: column sub-tiles entirely right of this wave's rows are masked.
  const bool diag = CAUSAL && (rt == ct);

  fetch(0);
  stash();
  __syncthreads();
  for (int ch = 0; ch < NCH; ++ch) {
    if (ch + 1 < NCH) fetch(ch + 1);
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      const u32x4 bq = *(const u32x4*)&Bs[(32 * wv + lr) * LDS_STRIDE + ks * 16 + lh * 8];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (!diag || t <= wv) {
          const u32x4 ak = *(const u32x4*)&As[(32 * t + lr) * LDS_STRIDE + ks * 16 + lh * 8];
          acc[t] = mfma32(as_bf16x8(ak), as_bf16x8(bq), acc[t]);
        }
      }
    }
    __syncthreads();
    if (ch + 1 < NCH) {
      stash();
      __syncthreads();
    }
  }

  // ---- epilogue: this lane owns reduced row R and 64 of the tile's columns;
  // lane (lr, 1-lh) owns the other 64.
  const int R = R0 + 32 * wv + lr;
  float mloc = -INFINITY;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int c = c0 + 32 * t + 8 * (r >> 2) + 4 * lh + (r & 3);
      const bool valid = (c < NR) && (!CAUSAL || c <= R);
      const float x = valid ? acc[t][r] * scale_log2 : -INFINITY;
      acc[t][r] = x;
      mloc = fmaxf(mloc, x);
    }
  }
  const float m = fmaxf(mloc, __shfl_xor(mloc, 32));
  const float mref = (m == -INFINITY) ? 0.f : m;
  float gsum[16];  // 16 groups of 4 consecutive columns: group gi = 4*t + r/4
  float lloc = 0.f;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = fast_exp2(acc[t][4 * g4 + e] - mref);
        acc[t][4 * g4 + e] = p;
        s += p;
      }
      gsum[4 * t + g4] = s;
      lloc += s;
    }
  }
  const float l = lloc + __shfl_xor(lloc, 32);
  const bool rvalid = R < NR;
  float* prow = part + ((size_t)h * NR + (rvalid ? R : 0)) * NB;
  const int j0 = c0 / NRB;

  if constexpr (NRB >= 8) {
    // group gi covers columns 8*gi + 4*lh + [0, 4): block (local) gi / (NRB / 8)
    constexpr int GPB = NRB / 8;
    constexpr int NBL = TC / NRB;
    float pb[NBL];
#pragma unroll
    for (int jb = 0; jb < NBL; ++jb) {
      float s = 0.f;
#pragma unroll
      for (int x = 0; x < GPB; ++x) s += gsum[jb * GPB + x];
      pb[jb] = s + __shfl_xor(s, 32);
    }
    if (rvalid) {
      if constexpr (NBL >= 2) {
#pragma unroll
        for (int x = 0; x < NBL / 2; ++x) {
          const int jb = lh * (NBL / 2) + x;
          if (j0 + jb < NB) prow[j0 + jb] = pb[jb];
        }
      } else {
        if (lh == 0 && j0 < NB) prow[j0] = pb[0];
      }
    }
  } else if constexpr (NRB == 4) {
    // each group of 4 columns is one block: local block 2*gi + lh
    if (rvalid) {
#pragma unroll
      for (int gi = 0; gi < 16; ++gi) {
        const int j = j0 + 2 * gi + lh;
        if (j < NB) prow[j] = gsum[gi];
      }
    }
  } else {  // NRB == 2: each group holds two blocks
    static_assert(NRB == 2, "stride must divide the block");
    if (rvalid) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int gi = 4 * t + g4;
          const int j = j0 + 4 * gi + 2 * lh;
          if (j < NB) prow[j] = acc[t][4 * g4] + acc[t][4 * g4 + 1];
          if (j + 1 < NB) prow[j + 1] = acc[t][4 * g4 + 2] + acc[t][4 * g4 + 3];
        }
      }
    }
  }
  if (rvalid && lh == 0) stats[((size_t)h * NR + R) * NT + ct] = make_float2(m, l);
}

// One workgroup per (query head, query block) row.
template <bool CAUSAL>
__global__ __launch_bounds__(256) void score_finalize(const float* __restrict__ part,
                                                      const float2* __restrict__ stats, int NR,
                                                      int NB, int NT, int nrb,
                                                      float* __restrict__ scores) {
  const int h = blockIdx.x / NB, b = blockIdx.x % NB;
  __shared__ float mR[kBlock], ilR[kBlock];
  const int tid = threadIdx.x;
  if (tid < nrb) {
    const int R = b * nrb + tid;
    const int tmax = CAUSAL ? R / TC : NT - 1;
    const float2* st = stats + ((size_t)h * NR + R) * NT;
    float m = -INFINITY;
    for (int t = 0; t <= tmax; ++t) m = fmaxf(m, st[t].x);
    float l = 0.f;
    for (int t = 0; t <= tmax; ++t) l += st[t].y * fast_exp2(st[t].x - m);
    mR[tid] = m;
    ilR[tid] = 1.f / l;
  }
  __syncthreads();
  const int ncand = CAUSAL ? b + 1 : NB;
  const float inv_nrb = 1.f / (float)nrb;
  float* out = scores + ((size_t)h * NB + b) * NB;
  for (int j = tid; j < NB; j += 256) {
    float acc = 0.f;
    if (j < ncand) {
      const int t = (j * nrb) / TC;
      for (int r = 0; r < nrb; ++r) {
        const size_t R = (size_t)h * NR + b * nrb + r;
        const float f = fast_exp2(stats[R * NT + t].x - mR[r]) * ilR[r];
        acc += part[R * NB + j] * f;
      }
      acc *= inv_nrb;
    }
    out[j] = acc;
  }
}

template <int NRB, bool CAUSAL>
hipError_t launch_partials(const void* q, const void* k, const XattnShape& s, float* part,
                           float* stats, hipStream_t st) {
  const int S = kBlock / NRB, NR = s.seq / S, NB = s.NB(), NT = ceil_div(NR, TC);
  const int tiles = CAUSAL ? NT * (NT + 1) / 2 : NT * NT;
  const int n_work = s.batch * s.hkv * tiles * (s.hq / s.hkv);
  const float scale_log2 = kLog2e / (sqrtf((float)kHeadDim) * (float)S);
  hipLaunchKernelGGL((score_partials<NRB, CAUSAL>), dim3(n_work), dim3(kThreads), 0, st,
                     (const uint16_t*)q, (const uint16_t*)k, s.hq, s.hkv, s.seq, NR, NB, NT,
                     tiles, n_work, scale_log2, part, (float2*)stats);
  return hipGetLastError();
}

template <int NRB>
hipError_t launch_partials_c(const void* q, const void* k, const XattnShape& s, float* part,
                             float* stats, hipStream_t st) {
  return s.causal ? launch_partials<NRB, true>(q, k, s, part, stats, st)
                  : launch_partials<NRB, false>(q, k, s, part, stats, st);
}

}  // namespace

size_t score_scratch_bytes(const XattnShape& s, int stride) {
  const size_t NR = (size_t)s.seq / stride, NB = s.NB(), NT = ceil_div((int)NR, TC);
  const size_t part = (size_t)s.HQ() * NR * NB * sizeof(float);
  const size_t stats = (size_t)s.HQ() * NR * NT * 2 * sizeof(float);
  return ((part + 255) / 256) * 256 + stats;
}

hipError_t launch_score(const void* q, const void* k, const XattnShape& s, int stride,
                        float* scores, void* scratch, hipStream_t st) {
  const int NR = s.seq / stride, NB = s.NB(), NT = ceil_div(NR, TC);
  const size_t part_bytes = (size_t)s.HQ() * NR * NB * sizeof(float);
  float* part = (float*)scratch;
  float* stats = (float*)((char*)scratch + ((part_bytes + 255) / 256) * 256);
  hipError_t e;
  switch (stride) {
    case 1: e = launch_partials_c<128>(q, k, s, part, stats, st); break;
    case 2: e = launch_partials_c<64>(q, k, s, part, stats, st); break;
    case 4: e = launch_partials_c<32>(q, k, s, part, stats, st); break;
    case 8: e = launch_partials_c<16>(q, k, s, part, stats, st); break;
    case 16: e = launch_partials_c<8>(q, k, s, part, stats, st); break;
    case 32: e = launch_partials_c<4>(q, k, s, part, stats, st); break;
    case 64: e = launch_partials_c<2>(q, k, s, part, stats, st); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  const int nrb = kBlock / stride;
  if (s.causal)
    hipLaunchKernelGGL(score_finalize<true>, dim3(s.HQ() * NB), dim3(256), 0, st, part,
                       (const float2*)stats, NR, NB, NT, nrb, scores);
  else
    hipLaunchKernelGGL(score_finalize<false>, dim3(s.HQ() * NB), dim3(256), 0, st, part,
                       (const float2*)stats, NR, NB, NT, nrb, scores);
  return hipGetLastError();
}
