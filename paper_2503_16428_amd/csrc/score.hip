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
// Kernel score_partials computes X^T = K~ Q~^T in 256 x 256 tiles on bf16
// MFMA (fp32 accumulate; 8 waves of 128 columns x 64 rows; 64-deep K chunks
// streamed by direct-to-LDS loads through a two-stage pipeline) and, in its
// epilogue, per reduced row R and 128-column sub-tile t: the sub-tile max m
// (log2 domain), l = sum exp2(x - m), and per key block j the partial mass
// sum_{c in j} exp2(x - m). Kernel score_finalize
// merges the tiles of each row (m_R = max_t m, l_R = sum_t l e^(m - m_R)),
// normalises, and averages the B/S reduced rows of each query block.
#include "common.h"

using namespace xattn;

namespace {

constexpr int TM = 256;             // reduced rows (R) and columns (c) per workgroup tile
constexpr int TSUB = 128;           // column sub-tile owning one (m, l) pair per row
constexpr int KC = 32;              // reduced-K chunk per pipeline stage
constexpr int NSTAGE = 4;           // pipeline depth (3 chunks in flight)
constexpr int kThreads = 512;       // 8 waves: 2 (columns) x 4 (rows), 128 c x 64 R each
constexpr int kStage = TM * KC;     // bf16 elements of one operand in one stage (32 KB)

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ void tri_decode(int t, int& rt, int& ct) {
  int r = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while (r * (r + 1) / 2 > t) --r;
  while ((r + 1) * (r + 2) / 2 <= t) ++r;
  rt = r;
  ct = t - r * (r + 1) / 2;
}

// LDS rows hold KC = 32 bf16 (4 chunks of 16 B); chunk c of row r sits at
// position c ^ ((r >> 2) & 3), so 16 consecutive rows read at one logical
// chunk hit 16 distinct bank groups.

// NRB = reduced rows (and columns) per 128-token block = 128 / S.
template <int NRB, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 1) void score_partials(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int hq, int hkv, int L,
    int NR, int NB, int NT, int tiles_per_head, int n_work, float scale_log2,
    float* __restrict__ part, float2* __restrict__ stats) {
  constexpr int S = kBlock / NRB;
  constexpr int KD = S * kHeadDim;  // reduced inner dimension S*d
  constexpr int NCH = KD / KC;      // >= 2 (S >= 1)
  // [stage][operand A = K~ rows (c) | B = Q~ rows (R)][256 rows x 32]
  __shared__ __attribute__((aligned(1024))) uint16_t lds[NSTAGE * 2 * kStage];

  const int tid = threadIdx.x, lane = tid & 63, lr = lane & 31, lh = lane >> 5;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wc = wv & 1, wr = wv >> 1;

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
    rt = tile / ceil_div(NR, TM);
    ct = tile % ceil_div(NR, TM);
  }
  const int R0 = rt * TM, c0 = ct * TM;
  const uint16_t* Qh = q + (size_t)h * L * kHeadDim;
  const uint16_t* Kg = k + (size_t)gidx * L * kHeadDim;

  // ---- direct-to-LDS staging: per stage each wave loads rows 32 wv .. +32 of
  // both operands, 2 instructions (16 rows x 64 B) each. Rows beyond NR are
  // clamped to NR - 1 (their results are masked / not stored).
  uint32_t offA[2], offB[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = 32 * wv + 16 * i + (lane >> 2);
    const int c = (lane & 3) ^ ((r >> 2) & 3);
    const int ra = min(c0 + r, NR - 1), rb = min(R0 + r, NR - 1);
    offA[i] = (uint32_t)(((size_t)ra * KD + c * 8) * 2);
    offB[i] = (uint32_t)(((size_t)rb * S * kHeadDim + c * 8) * 2);
  }
  const uint32_t lds0 = XATTN_LDS_ADDR(lds);
  auto issue = [&](int ch) {
    const int kap0 = ch * KC;
    const int tsub = kap0 / kHeadDim, e0 = kap0 % kHeadDim;
    const uint32_t st = lds0 + (uint32_t)((ch % NSTAGE) * 2 * kStage * 2);
    const uint16_t* baseA = Kg + kap0;
    const uint16_t* baseB = Qh + (S - 1 - tsub) * kHeadDim + e0;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t row_lds = (uint32_t)((32 * wv + 16 * i) * KC * 2);
      dma16(baseA, offA[i], st + row_lds);
      dma16(baseB, offB[i], st + kStage * 2 + row_lds);
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int n = 0; n < 2; ++n) acc[t][n] = f32x16{};

  // Diagonal tiles are computed in full (their masked half is ~2% of the MFMA
  // work of a causal layer); a per-MFMA skip would break the inner loop into
  // branches that serialise every LDS read with its MFMA.
  const uint32_t xa = (uint32_t)((lr >> 2) & 3);  // swizzle of this lane's rows
  auto compute = [&](int ch) {
    const uint16_t* A = lds + (ch % NSTAGE) * 2 * kStage;
    const uint16_t* Bm = A + kStage;
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      const uint32_t coff = (uint32_t)((((2 * ks + lh) ^ xa)) << 3);  // elements
      u32x4 bq[2];
#pragma unroll
      for (int n = 0; n < 2; ++n)
        bq[n] = *(const u32x4*)(Bm + (64 * wr + 32 * n + lr) * KC + coff);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const u32x4 ak = *(const u32x4*)(A + (128 * wc + 32 * t + lr) * KC + coff);
#pragma unroll
        for (int n = 0; n < 2; ++n) acc[t][n] = mfma32(as_bf16x8(ak), as_bf16x8(bq[n]), acc[t][n]);
      }
    }
    // Issue order per chunk: the 6 reads of k-step 0, then its 8 MFMAs with the
    // 6 reads of k-step 1 interleaved, then the 8 MFMAs of k-step 1.
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 10, 0);
  };

  // Each wave issues 4 loads per chunk; NCH = S*d/32 >= 4 for every stride.
  // Step ch: wait for chunk ch (chunks ch+1, ch+2 may stay in flight), one
  // barrier (chunk ch visible; every wave finished chunk ch-1, whose stage
  // chunk ch+3 now refills), prefetch ch+3, compute ch.
  issue(0);
  issue(1);
  issue(2);
  for (int ch = 0; ch < NCH - 2; ++ch) {
    wait_vmcnt<8>();
    barrier_nofence();
    if (ch + 3 < NCH) issue(ch + 3);
    compute(ch);
  }
  wait_vmcnt<4>();
  barrier_nofence();
  compute(NCH - 2);
  wait_vmcnt<0>();
  barrier_nofence();
  compute(NCH - 1);

  // ---- epilogue per 32-row slab n: this lane owns reduced row R and 64 of the
  // wave's 128 columns; lane (lr, 1-lh) owns the other 64.
  const int csub = c0 + 128 * wc;  // first column of this wave's sub-tile
  const int tsub_idx = csub / TSUB;
  const int j0 = csub / NRB;
#pragma unroll
  for (int n = 0; n < 2; ++n) {
    const int R = R0 + 64 * wr + 32 * n + lr;
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = csub + 32 * t + 8 * (r >> 2) + 4 * lh + (r & 3);
        const bool valid = (c < NR) && (!CAUSAL || c <= R);
        const float x = valid ? acc[t][n][r] * scale_log2 : -INFINITY;
        acc[t][n][r] = x;
        mloc = fmaxf(mloc, x);
      }
    }
    const float m = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float mref = (m == -INFINITY) ? 0.f : m;
    float gsum[16];  // groups of 4 consecutive columns: group gi = 4 t + r / 4
    float lloc = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = fast_exp2(acc[t][n][4 * g4 + e] - mref);
          acc[t][n][4 * g4 + e] = p;
          sum += p;
        }
        gsum[4 * t + g4] = sum;
        lloc += sum;
      }
    }
    const float l = lloc + __shfl_xor(lloc, 32);
    const bool rvalid = R < NR;
    float* prow = part + ((size_t)h * NR + (rvalid ? R : 0)) * NB;

    if constexpr (NRB >= 8) {
      // group gi covers columns 8 gi + 4 lh + [0, 4): local block gi / (NRB / 8)
      constexpr int GPB = NRB / 8;
      constexpr int NBL = TSUB / NRB;
      float pb[NBL];
#pragma unroll
      for (int jb = 0; jb < NBL; ++jb) {
        float sum = 0.f;
#pragma unroll
        for (int x = 0; x < GPB; ++x) sum += gsum[jb * GPB + x];
        pb[jb] = sum + __shfl_xor(sum, 32);
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
      // each group of 4 columns is one block: local block 2 gi + lh
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
            if (j < NB) prow[j] = acc[t][n][4 * g4] + acc[t][n][4 * g4 + 1];
            if (j + 1 < NB) prow[j + 1] = acc[t][n][4 * g4 + 2] + acc[t][n][4 * g4 + 3];
          }
        }
      }
    }
    if (rvalid && lh == 0 && tsub_idx < NT)
      stats[((size_t)h * NR + R) * NT + tsub_idx] = make_float2(m, l);
  }
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
    const int tmax = CAUSAL ? R / TSUB : NT - 1;
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
      const int t = (j * nrb) / TSUB;
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
  const int S = kBlock / NRB, NR = s.seq / S, NB = s.NB(), NT = ceil_div(NR, TSUB);
  const int T = ceil_div(NR, TM);
  const int tiles = CAUSAL ? T * (T + 1) / 2 : T * T;
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
  const size_t NR = (size_t)s.seq / stride, NB = s.NB(), NT = ceil_div((int)NR, TSUB);
  const size_t part = (size_t)s.HQ() * NR * NB * sizeof(float);
  const size_t stats = (size_t)s.HQ() * NR * NT * 2 * sizeof(float);
  return ((part + 255) / 256) * 256 + stats;
}

hipError_t launch_score(const void* q, const void* k, const XattnShape& s, int stride,
                        float* scores, void* scratch, hipStream_t st) {
  const int NR = s.seq / stride, NB = s.NB(), NT = ceil_div(NR, TSUB);
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
