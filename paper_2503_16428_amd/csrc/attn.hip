// Step 3: block-sparse flash attention over the selected key blocks
// (XAttention Fig. 1 right), and the dense mode (every candidate block).
//
// One workgroup (4 waves) per (query head, query block of 128 rows); wave w
// owns queries 32w .. 32w+31 of the block. Per listed key block j:
//   K_j [128 keys][128 d] and V_j^T [128 d][128 keys] are staged in LDS,
//   S^T = K_j Q^T       (32x32x16 bf16 MFMA; Q stays in registers),
//   online softmax in fp32 in the log2 domain (lane = query, so the row
//   max / sum need one cross-half exchange),
//   O^T += V_j^T P^T    (P rounded to bf16; the key order inside each
//   16-key MFMA step is permuted so that P never leaves registers).
// Keeping the accumulators transposed (lane = query) makes the per-query
// rescale by exp2(m_old - m_new) a purely lane-local multiply.
#include "common.h"

using namespace xattn;

namespace {

constexpr int kThreads = 256;
constexpr int KS = kHeadDim + 8;  // LDS row stride of K_j   (bf16 elements)
constexpr int VS = kBlock + 8;    // LDS row stride of V_j^T (bf16 elements)

template <bool CAUSAL, bool DENSE>
__global__ __launch_bounds__(kThreads, 2) void attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, int hq, int hkv, int L, int NB, int n_work,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt, float scale_log2,
    uint16_t* __restrict__ o, float* __restrict__ lse) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kBlock * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kHeadDim * VS];

  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, lr = lane & 31, lh = lane >> 5;

  // logical order: (kv head, query block descending, query head in group):
  // heavy causal rows first, and the query heads sharing K/V run together.
  const int w = xcd_remap(blockIdx.x, n_work);
  const int G = hq / hkv;
  const int hh = w % G;
  const int rest = w / G;
  const int b = NB - 1 - rest % NB;
  const int gidx = rest / NB;
  const int h = (gidx / hkv) * hq + (gidx % hkv) * G + hh;
  const uint16_t* Qh = q + (size_t)h * L * kHeadDim;
  const uint16_t* Kg = k + (size_t)gidx * L * kHeadDim;
  const uint16_t* Vg = v + (size_t)gidx * L * kHeadDim;
  const int q0 = b * kBlock + 32 * wv;  // first query of this wave
  const int qi = q0 + lr;               // this lane's query

  // Q^T as the B operand: lane holds Q[qi][16 s + 8 lh .. +8] for k-step s
  bf16x8 qb[8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
    qb[s] = as_bf16x8(*(const u32x4*)(Qh + (size_t)qi * kHeadDim + 16 * s + 8 * lh));

  int n_kb;
  const int32_t* list = nullptr;
  if (DENSE) {
    n_kb = CAUSAL ? b + 1 : NB;
  } else {
    n_kb = cnt[(size_t)h * NB + b];
    n_kb = n_kb < 0 ? 0 : (n_kb > NB ? NB : n_kb);
    list = idx + ((size_t)h * NB + b) * NB;
  }

  f32x16 oacc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) oacc[i] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  for (int it = 0; it < n_kb; ++it) {
    const int j = DENSE ? it : list[it];
    if (j < 0 || j >= NB) continue;  // malformed list entry: skip (uniform)
    const int key0 = j * kBlock;
    __syncthreads();
    // K_j -> LDS: 2048 16-byte pieces, 8 per thread, 16 threads per key row
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int p = tid + kThreads * i;
      const int row = p >> 4, col = (p & 15) * 8;
      *(u32x4*)&Ks[row * KS + col] = *(const u32x4*)(Kg + (size_t)(key0 + row) * kHeadDim + col);
    }
    // V_j^T -> LDS: groups of 4 keys x 8 features, written as 8 x (4 keys)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int gI = tid + kThreads * i;
      const int dc = gI & 15, k4 = gI >> 4;
      u32x4 r[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        r[kk] = *(const u32x4*)(Vg + (size_t)(key0 + 4 * k4 + kk) * kHeadDim + 8 * dc);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int wd = e >> 1, sh = 16 * (e & 1);
        const uint32_t x0 = (r[0][wd] >> sh) & 0xFFFFu, x1 = (r[1][wd] >> sh) & 0xFFFFu;
        const uint32_t x2 = (r[2][wd] >> sh) & 0xFFFFu, x3 = (r[3][wd] >> sh) & 0xFFFFu;
        *(u32x2*)&Vt[(8 * dc + e) * VS + 4 * k4] = u32x2{x0 | (x1 << 16), x2 | (x3 << 16)};
      }
    }
    __syncthreads();

    // S^T = K_j Q^T: tile kt covers keys 32 kt .. 32 kt + 31
    f32x16 sacc[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      sacc[kt] = f32x16{};
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const u32x4 a = *(const u32x4*)&Ks[(32 * kt + lr) * KS + 16 * s + 8 * lh];
        sacc[kt] = mfma32(as_bf16x8(a), qb[s], sacc[kt]);
      }
    }

    // online softmax (log2 domain); register r of tile kt is key
    // key0 + 32 kt + 8 (r/4) + 4 lh + r%4 of query qi
    const bool mask = CAUSAL && (j >= b);
    float mt = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = sacc[kt][r] * scale_log2;
        if (mask) {
          const int key = key0 + 32 * kt + 8 * (r >> 2) + 4 * lh + (r & 3);
          if (key > qi) x = -INFINITY;
        }
        sacc[kt][r] = x;
        mt = fmaxf(mt, x);
      }
    }
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) oacc[dt] *= alpha;

    uint32_t pk[4][8];
    float ls = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const float p0 = fast_exp2(sacc[kt][r] - m_use);
        const float p1 = fast_exp2(sacc[kt][r + 1] - m_use);
        ls += p0 + p1;
        pk[kt][r >> 1] = pack_bf16x2(p0, p1);
      }
    }
    l_run += ls;

    // O^T += V_j^T P^T. MFMA step u covers keys 16u .. 16u+15; slot
    // 8 lh + jj of both operands is key 16u + 8 (jj/4) + 4 lh + jj%4.
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int kt = u >> 1, hf = u & 1;
      const bf16x8 pb = as_bf16x8(
          u32x4{pk[kt][4 * hf], pk[kt][4 * hf + 1], pk[kt][4 * hf + 2], pk[kt][4 * hf + 3]});
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int d = 32 * dt + lr;
        const u32x2 lo = *(const u32x2*)&Vt[d * VS + 16 * u + 4 * lh];
        const u32x2 hi = *(const u32x2*)&Vt[d * VS + 16 * u + 8 + 4 * lh];
        oacc[dt] = mfma32(as_bf16x8(u32x4{lo[0], lo[1], hi[0], hi[1]}), pb, oacc[dt]);
      }
    }
  }

  // normalise and store: register r of tile dt is feature 32 dt + 8 (r/4) + 4 lh + r%4
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  uint16_t* orow = o + ((size_t)h * L + qi) * kHeadDim;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = 32 * dt + 8 * g4 + 4 * lh;
      const u32x2 val{pack_bf16x2(oacc[dt][4 * g4] * inv, oacc[dt][4 * g4 + 1] * inv),
                      pack_bf16x2(oacc[dt][4 * g4 + 2] * inv, oacc[dt][4 * g4 + 3] * inv)};
      *(u32x2*)(orow + d0) = val;
    }
  }
  if (lse != nullptr && lh == 0)
    lse[(size_t)h * L + qi] =
        l_tot > 0.f ? (m_run + __builtin_log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
}

template <bool CAUSAL, bool DENSE>
hipError_t launch_t(const void* q, const void* k, const void* v, const XattnShape& s,
                    const int32_t* idx, const int32_t* cnt, void* o, float* lse,
                    hipStream_t st) {
  const int n_work = s.HQ() * s.NB();
  const float scale_log2 = kLog2e / sqrtf((float)kHeadDim);
  hipLaunchKernelGGL((attn_kernel<CAUSAL, DENSE>), dim3(n_work), dim3(kThreads), 0, st,
                     (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, s.hq, s.hkv,
                     s.seq, s.NB(), n_work, idx, cnt, scale_log2, (uint16_t*)o, lse);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const void* q, const void* k, const void* v, const XattnShape& s,
                       const int32_t* idx, const int32_t* cnt, bool dense, void* o,
                       float* lse, hipStream_t st) {
  if (s.causal)
    return dense ? launch_t<true, true>(q, k, v, s, idx, cnt, o, lse, st)
                 : launch_t<true, false>(q, k, v, s, idx, cnt, o, lse, st);
  return dense ? launch_t<false, true>(q, k, v, s, idx, cnt, o, lse, st)
               : launch_t<false, false>(q, k, v, s, idx, cnt, o, lse, st);
}
