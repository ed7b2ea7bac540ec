// Step 3: block-sparse flash attention over the selected key blocks
// (XAttention Fig. 1 right), and the dense mode (every candidate block).
//
// One workgroup (4 waves) per (query head, query block of 128 rows); wave w
// owns queries 32w .. 32w+31 of the block. Per listed key block j:
//   S^T = K_j Q^T       (32x32x16 bf16 MFMA; Q stays in registers),
//   online softmax in fp32 in the log2 domain (lane = query, so the row
//   max / sum need one cross-half exchange),
//   O^T += V_j^T P^T    (P rounded to bf16; the key order inside each
//   16-key MFMA step is permuted so that P never leaves registers).
// Keeping the accumulators transposed (lane = query) makes the per-query
// rescale by exp2(m_old - m_new) a lane-local multiply.
//
// Data movement: K_j and V_j (32 KB each, row-major [key][d]) go straight
// from global memory into LDS with global_load_lds_dwordx4 (no registers),
// with the 16-byte chunk index XOR-swizzled by (row mod 16) against bank
// conflicts. One K buffer and one V buffer form a two-stage pipeline: the
// next K tile streams in during softmax + PV, the next V tile during the
// next QK^T + softmax. The V^T operand of PV is read with ds_read_b64_tr_b16,
// which hands each lane four keys of one feature from a 4 x 16 patch.
// 64 KB of LDS per workgroup: two workgroups share a CU.
#include <type_traits>

#include "common.h"

using namespace xattn;

namespace {

constexpr int kThreads = 256;
constexpr float kRescaleSlack = 8.f;  // log2 units: probabilities stay <= 256

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4;
typedef __attribute__((ext_vector_type(2))) float f32v2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16v2;
#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

__device__ __forceinline__ uint32_t cvt_pk_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32v2{a, b}, bf16v2));
}

// Element offset of logical 16-byte chunk c of row r in a swizzled [128][128]
// tile. K tiles are read 16 rows at one chunk (ds_read_b128): chunk ^ (r mod 16)
// spreads them over 16 bank groups. V tiles are read as 4-row x 32-byte
// patches (ds_read_b64_tr_b16): chunk ^ (4 (r mod 4) | (r / 4) mod 4) puts the
// 8 row/chunk pairs of a patch, and of two patches side by side, on distinct
// bank groups.
__device__ __forceinline__ int swz_k(int r, int c) { return r * kHeadDim + ((c ^ (r & 15)) << 3); }
__device__ __forceinline__ int swz_v_mask(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int swz_v(int r, int c) {
  return r * kHeadDim + ((c ^ swz_v_mask(r)) << 3);
}

// This wave's share of one 128 x 128 bf16 tile: 8 x (4 rows x 256 B).
// Per-lane byte offsets of this wave's 8 loads of a 128 x 128 bf16 tile: load
// i covers rows 4i .. 4i+3 of the wave's 32 rows, lane l filling physical
// chunk l mod 16 of row 4i + l / 16. Rows 16 apart share the swizzle (both
// layouts), so loads i and i+4 use the same offset (+4 KB on the scalar base).
template <bool VTILE>
__device__ __forceinline__ void tile_offsets(int lane, uint32_t voff[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * i + (lane >> 4);
    const int c = (lane & 15) ^ (VTILE ? swz_v_mask(r) : (r & 15));
    voff[i] = (uint32_t)((r * kHeadDim + c * 8) * 2);
  }
}

// This wave's share (rows 32 wv .. 32 wv + 31) of tile src -> LDS (swizzled).
__device__ __forceinline__ void issue_tile(uint32_t lds_base, const uint16_t* src, int wv,
                                           const uint32_t voff[4]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint16_t* base = src + (size_t)(32 * wv + (i >= 4 ? 16 : 0)) * kHeadDim;
    dma16(base, voff[i & 3], lds_base + (uint32_t)((32 * wv + 4 * i) * kHeadDim * 2));
  }
}

// The LDS tiles arrive as distinct __restrict__ pointers: once inlined, the
// compiler knows a K-tile prefetch cannot alias a V-tile read (and vice versa)
// and does not stall LDS reads on the other buffer's loads in flight.
template <bool CAUSAL>
__device__ __forceinline__ void attn_body(bool dense,
    uint16_t* __restrict__ Ks, uint16_t* __restrict__ Vs, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, int hq, int hkv, int L,
    int NB, const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt,
    float scale_log2, uint16_t* __restrict__ o, float* __restrict__ lse) {
  const int tid = threadIdx.x, lane = tid & 63, lr = lane & 31, lh = lane >> 5;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (SGPR)

  // Work order (kv head, query block descending, query head in group), in
  // dispatch order: the workgroups resident at any time read the K/V of one
  // group (64 MB at 128K tokens), which then stays in the Infinity Cache;
  // heavy causal rows start first.
  const int w = blockIdx.x;
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

  int n_kb;
  const int32_t* list = nullptr;
  if (dense) {
    n_kb = CAUSAL ? b + 1 : NB;
  } else {
    n_kb = cnt[(size_t)h * NB + b];
    n_kb = n_kb < 0 ? 0 : (n_kb > NB ? NB : n_kb);
    list = idx + ((size_t)h * NB + b) * NB;
  }
  // The block list is held 64 entries at a time in one register (lane l holds
  // entry 64c + l) and read with v_readlane: a per-step memory load would make
  // the compiler wait for every load in flight, prefetches included.
  auto list_chunk = [&](int c0) -> int {
    const int i = c0 + lane;
    return (!dense && i < n_kb) ? list[i] : 0;
  };
  int lreg = list_chunk(0);
  auto block_at = [&](int it) -> int {
    if (dense) return it;
    if ((it & 63) == 0 && it > 0) {  // calls come in increasing it
      lreg = list_chunk(it);
      asm volatile("" ::"v"(lreg));  // wait for the reload here, not on every step
    }
    const int j = __builtin_amdgcn_readlane(lreg, it & 63);
    return j < 0 ? 0 : (j >= NB ? NB - 1 : j);  // memory-safe on malformed lists
  };

  uint32_t koff[4], voff[4];
  tile_offsets<false>(lane, koff);
  tile_offsets<true>(lane, voff);
  const uint32_t ks_lds = XATTN_LDS_ADDR(Ks);
  const uint32_t vs_lds = XATTN_LDS_ADDR(Vs);
  int j = n_kb > 0 ? block_at(0) : 0;
  if (n_kb > 0) {
    issue_tile(ks_lds, Kg + (size_t)j * kBlock * kHeadDim, wv, koff);
    issue_tile(vs_lds, Vg + (size_t)j * kBlock * kHeadDim, wv, voff);
  }

  // Q^T as the B operand: lane holds Q[qi][16 s + 8 lh .. +8] for k-step s
  bf16x8 qb[8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
    qb[s] = as_bf16x8(*(const u32x4*)(Qh + (size_t)qi * kHeadDim + 16 * s + 8 * lh));
  // consume Q here, so the compiler's own wait for it stays out of the loop
#pragma unroll
  for (int s = 0; s < 8; ++s) asm volatile("" ::"v"(qb[s]));

  f32x16 oacc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) oacc[i] = f32x16{};
  float m_ref = -INFINITY, l_run = 0.f;  // exponent reference (log2 domain), row sum

  // ds_read_b64_tr_b16 source addresses (see header): lane = (group G, index i)
  const int tj = lane & 15, tg2 = (lane >> 4) & 1;

  // One pipeline step on key block j; when NEXT, the tiles of key block jn are
  // prefetched into the buffers as soon as these are free. The last step is
  // peeled off so that every wait below has one fixed count.
  auto step = [&](auto next_tag, int jn) {
    constexpr bool NEXT = decltype(next_tag)::value;
    const int key0 = j * kBlock;

    // ---- K_j ready (V_j may still be in flight)
    wait_vmcnt<8>();
    barrier_nofence();
    f32x16 sacc[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      sacc[kt] = f32x16{};
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const u32x4 a = *(const u32x4*)&Ks[swz_k(32 * kt + lr, 2 * s + lh)];
        sacc[kt] = mfma32(as_bf16x8(a), qb[s], sacc[kt]);
      }
    }
    // keep LDS reads next to their MFMAs (bounds the registers held by reads in flight)
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    }
    barrier_nofence();  // every wave is done with Ks
    if constexpr (NEXT) issue_tile(ks_lds, Kg + (size_t)jn * kBlock * kHeadDim, wv, koff);

    // ---- online softmax (log2 domain); register r of tile kt is key
    // key0 + 32 kt + 8 (r/4) + 4 lh + r%4 of query qi. Only blocks j >= b (the
    // diagonal) need the causal mask; the empty asm keeps the compiler from
    // turning this uniform branch into selects executed on every block.
    if (CAUSAL && j >= b) {
      asm volatile("");
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + 32 * kt + 8 * (r >> 2) + 4 * lh + (r & 3);
          if (key > qi) sacc[kt][r] = -INFINITY;
        }
      }
    }
    float mraw = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) mraw = fmaxf(mraw, sacc[kt][r]);
    }
    mraw = fmaxf(mraw, __shfl_xor(mraw, 32));
    const float mt = mraw * scale_log2;  // scale > 0: max commutes with it
    // Lazy rescaling: the exponent reference m_ref only moves when some lane's
    // tile max exceeds it by more than kRescaleSlack, so p = exp2(s - m_ref)
    // stays <= 2^kRescaleSlack; the result is the same softmax (the common
    // factor cancels in O / l), and the 64 rescale multiplies are skipped
    // whenever no lane needs them.
    if (__ballot(mt > m_ref + kRescaleSlack) != 0) {
      const float m_new = fmaxf(m_ref, mt);
      const float alpha = fast_exp2(m_ref - m_new);  // m_ref = -inf -> 0
      m_ref = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) oacc[dt] *= alpha;
    }
    const float neg_m = (m_ref == -INFINITY) ? 0.f : -m_ref;

    uint32_t pk[4][8];
    float ls = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const float p0 = fast_exp2(fmaf(sacc[kt][r], scale_log2, neg_m));
        const float p1 = fast_exp2(fmaf(sacc[kt][r + 1], scale_log2, neg_m));
        ls += p0 + p1;
        pk[kt][r >> 1] = cvt_pk_bf16(p0, p1);
      }
    }
    l_run += ls;

    // ---- V_j ready (K_jn may be in flight)
    if constexpr (NEXT) wait_vmcnt<8>();
    else wait_vmcnt<0>();
    barrier_nofence();
    // O^T += V_j^T P^T. MFMA step u covers keys 16u .. 16u+15; slot
    // 8 lh + jj of both operands is key 16u + 8 (jj/4) + 4 lh + jj%4.
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int kt = u >> 1, hf = u & 1;
      const bf16x8 pb = as_bf16x8(
          u32x4{pk[kt][4 * hf], pk[kt][4 * hf + 1], pk[kt][4 * hf + 2], pk[kt][4 * hf + 3]});
      const int row = 16 * u + 4 * lh + (tj >> 2);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int c = 4 * dt + 2 * tg2 + ((tj & 3) >> 1);
        const int off = 4 * (tj & 1);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)&Vs[swz_v(row, c) + off]);
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)&Vs[swz_v(row + 8, c) + off]);
        const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
        oacc[dt] = mfma32(as_bf16x8(u32x4{lo2[0], lo2[1], hi2[0], hi2[1]}), pb, oacc[dt]);
      }
    }
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // two DS transpose reads
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    }
    if constexpr (NEXT) {
      barrier_nofence();  // every wave is done with Vs
      issue_tile(vs_lds, Vg + (size_t)jn * kBlock * kHeadDim, wv, voff);
      j = jn;
    }
  };

  for (int it = 0; it + 1 < n_kb; ++it) step(std::true_type{}, block_at(it + 1));
  if (n_kb > 0) step(std::false_type{}, 0);

  // normalise and store: register r of tile dt is feature 32 dt + 8 (r/4) + 4 lh + r%4
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  uint16_t* orow = o + ((size_t)h * L + qi) * kHeadDim;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = 32 * dt + 8 * g4 + 4 * lh;
      const u32x2 val{cvt_pk_bf16(oacc[dt][4 * g4] * inv, oacc[dt][4 * g4 + 1] * inv),
                      cvt_pk_bf16(oacc[dt][4 * g4 + 2] * inv, oacc[dt][4 * g4 + 3] * inv)};
      *(u32x2*)(orow + d0) = val;
    }
  }
  if (lse != nullptr && lh == 0)
    lse[(size_t)h * L + qi] =
        l_tot > 0.f ? (m_ref + __builtin_log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
}

// Dense mode is a runtime flag of the same kernel (not a separate
// instantiation): both modes execute identical code and so give bitwise equal
// results on equal block lists.
template <bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void attn_kernel(
    int dense, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, int hq, int hkv, int L, int NB,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt, float scale_log2,
    uint16_t* __restrict__ o, float* __restrict__ lse) {
  __shared__ __attribute__((aligned(1024))) uint16_t Ks[kBlock * kHeadDim];
  __shared__ __attribute__((aligned(1024))) uint16_t Vs[kBlock * kHeadDim];
  attn_body<CAUSAL>(dense != 0, Ks, Vs, q, k, v, hq, hkv, L, NB, idx, cnt, scale_log2, o, lse);
}

template <bool CAUSAL>
hipError_t launch_t(const void* q, const void* k, const void* v, const XattnShape& s,
                    const int32_t* idx, const int32_t* cnt, bool dense, void* o, float* lse,
                    hipStream_t st) {
  const int n_work = s.HQ() * s.NB();
  const float scale_log2 = kLog2e / sqrtf((float)kHeadDim);
  hipLaunchKernelGGL((attn_kernel<CAUSAL>), dim3(n_work), dim3(kThreads), 0, st, dense ? 1 : 0,
                     (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, s.hq, s.hkv,
                     s.seq, s.NB(), idx, cnt, scale_log2, (uint16_t*)o, lse);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const void* q, const void* k, const void* v, const XattnShape& s,
                       const int32_t* idx, const int32_t* cnt, bool dense, void* o,
                       float* lse, hipStream_t st) {
  return s.causal ? launch_t<true>(q, k, v, s, idx, cnt, dense, o, lse, st)
                  : launch_t<false>(q, k, v, s, idx, cnt, dense, o, lse, st);
}
