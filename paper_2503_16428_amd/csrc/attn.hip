// Step 3: block-sparse flash attention over the selected key blocks
// (XAttention Fig. 1 right), and the dense mode (every candidate block).
//
// One workgroup (4 waves) per (query head, query block of 128 rows); wave w
// owns queries 32w .. 32w+31 of the block. Each listed 128-key block is
// processed as two 64-key half-tiles; per half-tile:
//   S^T = K_h Q^T       (32x32x16 bf16 MFMA; Q stays in registers),
//   online softmax in fp32 in the log2 domain (lane = query, so the row
//   max / sum need one cross-half exchange), with lazy rescaling,
//   O^T += V_h^T P^T    (P rounded to bf16; the key order inside each
//   16-key MFMA step is permuted so that P never leaves registers; the row
//   sum l adds the same rounded P, so O / l normalises consistently).
// Keeping the accumulators transposed (lane = query) makes the per-query
// rescale a lane-local multiply.
//
// Software pipeline inside each wave: the step on half-tile i issues the
// QK^T MFMAs of half-tile i+1 interleaved with the exponentials of half-tile
// i (independent work, so the matrix cores and the VALU run side by side),
// then the PV MFMAs of i.
//
// Data movement: K and V half-tiles (16 KB each, row-major [key][d]) go
// straight from global memory into LDS with global_load_lds_dwordx4, double
// buffered (64 KB of LDS per workgroup, two workgroups per CU): during the
// step on half-tile i, K of i+2 and V of i+1 are loading. The 16-byte chunk
// index is XOR-swizzled per row: K tiles are read 16 rows at one chunk
// (ds_read_b128), V tiles as 4-row x 32-byte patches by ds_read_b64_tr_b16,
// which hands each lane four keys of one feature.
#include <type_traits>

#include "common.h"

using namespace xattn;

namespace {

constexpr int kThreads = 256;
constexpr int kHalf = 64;                      // keys per half-tile
constexpr int kHalfElems = kHalf * kHeadDim;   // bf16 elements per half-tile
constexpr uint32_t kHalfBytes = kHalfElems * 2;
constexpr float kRescaleSlack = 8.f;  // log2 units: probabilities stay <= 256

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4;
typedef __attribute__((ext_vector_type(2))) float f32v2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16v2;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// max over lanes l and l ^ 32 (the two halves of the wave hold the two key
// halves of each query's scores)
__device__ __forceinline__ float half_max(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}

// this lane's max over the 32 scores of a half-tile
__device__ __forceinline__ float lane_max(const f32x16 (&s)[2]) {
  float m = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
    for (int r = 0; r < 16; ++r) m = fmaxf(m, s[kt][r]);
  }
  return m;
}

__device__ __forceinline__ uint32_t cvt_pk_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32v2{a, b}, bf16v2));
}

// acc + the two bf16 values packed in pk (one v_dot2c_f32_bf16 against 1.0, 1.0)
__device__ __forceinline__ float sum_pk_bf16(uint32_t pk, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16v2, pk),
                                         __builtin_bit_cast(bf16v2, 0x3F803F80u), acc, false);
}

// Element offset of logical 16-byte chunk c of row r in a swizzled [64][128]
// half-tile. K: chunk ^ (r mod 16) spreads 16 rows read at one chunk over 16
// bank groups. V: chunk ^ (4 (r mod 4) | (r / 4) mod 4) puts the 8 row/chunk
// pairs of a transposed-read patch, and of two patches side by side, on
// distinct bank groups.
__device__ __forceinline__ int swz_k(int r, int c) { return r * kHeadDim + ((c ^ (r & 15)) << 3); }
__device__ __forceinline__ int swz_v_mask(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int swz_v(int r, int c) {
  return r * kHeadDim + ((c ^ swz_v_mask(r)) << 3);
}

// Per-lane byte offsets of a wave's 4 loads of a half-tile: wave wv fills
// rows 16 wv .. 16 wv + 15; load i covers rows 16 wv + 4i .. +3, lane l
// filling physical chunk l mod 16 of row 16 wv + 4i + l / 16. Both swizzles
// depend only on the row mod 16, so the offsets are the same for every wave.
template <bool VTILE>
__device__ __forceinline__ void tile_offsets(int lane, uint32_t off[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * i + (lane >> 4);
    const int c = (lane & 15) ^ (VTILE ? swz_v_mask(r) : (r & 15));
    off[i] = (uint32_t)((r * kHeadDim + c * 8) * 2);
  }
}

// This wave's share (rows 16 wv .. 16 wv + 15) of the half-tile whose first
// row is src -> LDS half-tile buffer at byte address lds_base.
__device__ __forceinline__ void issue_half(uint32_t lds_base, const uint16_t* src, int wv,
                                           const uint32_t off[4]) {
  const uint16_t* base = src + (size_t)(16 * wv) * kHeadDim;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    dma16(base, off[i], lds_base + (uint32_t)((16 * wv + 4 * i) * kHeadDim * 2));
}

// The LDS buffers arrive as distinct __restrict__ pointers of an inlined body.
template <bool CAUSAL>
__device__ __forceinline__ void attn_body(
    bool dense, uint16_t* __restrict__ Ks, uint16_t* __restrict__ Vs,
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, int hq, int hkv, int L, int NB,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ cnt, float scale_log2,
    uint16_t* __restrict__ o, float* __restrict__ lse) {
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
  auto block_at = [&](int it) -> int {  // calls come in increasing it
    if (dense) return it;
    if ((it & 63) == 0 && it > 0) {
      lreg = list_chunk(it);
      asm volatile("" ::"v"(lreg));  // wait for the reload here, not on every step
    }
    const int j = __builtin_amdgcn_readlane(lreg, it & 63);
    return j < 0 ? 0 : (j >= NB ? NB - 1 : j);  // memory-safe on malformed lists
  };

  uint32_t koff[4], voff[4];
  tile_offsets<false>(lane, koff);
  tile_offsets<true>(lane, voff);
  const uint32_t ks_lds = XATTN_LDS_ADDR(Ks), vs_lds = XATTN_LDS_ADDR(Vs);
  auto krow = [&](int key) { return Kg + (size_t)key * kHeadDim; };
  auto vrow = [&](int key) { return Vg + (size_t)key * kHeadDim; };

  // jc: block of the current pair of half-tiles, jn: block of the next pair
  int jc = 0;
  if (n_kb > 0) {
    jc = block_at(0);
    issue_half(ks_lds, krow(jc * kBlock), wv, koff);                       // K(0)
    issue_half(vs_lds, vrow(jc * kBlock), wv, voff);                       // V(0)
    issue_half(ks_lds + kHalfBytes, krow(jc * kBlock + kHalf), wv, koff);  // K(1)
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

  // ds_read_b64_tr_b16 source addresses: lane = (group lane/16, index tj)
  const int tj = lane & 15, tg2 = (lane >> 4) & 1;

  // S^T of the half-tile in K buffer kb; tile kt covers keys 32 kt .. 32 kt + 31
  // (hook(t) runs after the t-th MFMA: the step spreads its prefetches there)
  auto qk = [&](int kb, f32x16 (&s)[2], auto hook) {
    const uint16_t* Kb = Ks + kb * kHalfElems;
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const u32x4 a = *(const u32x4*)&Kb[swz_k(32 * kt + lr, 2 * ks + lh)];
        s[kt] = mfma32(as_bf16x8(a), qb[ks], s[kt]);
        hook(2 * ks + kt);
      }
    }
  };

  // One step on half-tile i = 2p + PAR, whose scores are in sc (register r of
  // tile kt is key key0 + 32 kt + 8 (r/4) + 4 lh + r%4 of query qi). K(i+1)
  // and V(i) were issued one step earlier. Prefetches K(i+2) into the K
  // buffer of i and V(i+1) into the other V buffer, computes S(i+1) into sn
  // (from stale data on the last step: never used) and accumulates PV(i).
  // PAR fixes the buffers at compile time (the loop is unrolled by 2).
  auto step = [&](auto par_tag, bool has_next, int jn, f32x16 (&sc)[2], f32x16 (&sn)[2],
                  float& mpre) {
    constexpr int PAR = decltype(par_tag)::value;
    const int key0 = jc * kBlock + PAR * kHalf;
    wait_vmcnt<0>();    // this wave's loads of K(i+1) and V(i) have landed
    barrier_nofence();  // ... everyone's; all waves are done with step i-1
    // Prefetch sources; past the last pair the current block is loaded again
    // (in bounds, never read), which keeps the step free of branches.
    const int jp = has_next ? jn : jc;
    const uint16_t* ksrc = krow(jp * kBlock + PAR * kHalf) + (size_t)(16 * wv) * kHeadDim;
    const uint16_t* vsrc =
        vrow(PAR == 0 ? jc * kBlock + kHalf : jp * kBlock) + (size_t)(16 * wv) * kHeadDim;
    const uint32_t kdst = ks_lds + PAR * kHalfBytes + (uint32_t)(16 * wv * kHeadDim * 2);
    const uint32_t vdst = vs_lds + (PAR ^ 1) * kHalfBytes + (uint32_t)(16 * wv * kHeadDim * 2);
    // one 1 KB load after every other QK^T MFMA: a burst of loads at the
    // step start would stall the wave at issue
    auto prefetch = [&](int t) {
      if (t & 1) {
        const int n = t >> 1;
        if (n < 4) dma16(ksrc, koff[n], kdst + (uint32_t)(4 * n * kHeadDim * 2));
        else dma16(vsrc, voff[n - 4], vdst + (uint32_t)(4 * (n - 4) * kHeadDim * 2));
      }
    };

    // causal mask: only half-tiles reaching past this wave's first query (the
    // empty asm keeps this uniform branch from becoming selects on every step)
    // (mpre is this lane's max of sc, taken during the previous step; on
    // masked half-tiles it is taken again here)
    float mraw = mpre;
    if (CAUSAL && key0 + kHalf - 1 > q0) {
      asm volatile("");
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + 32 * kt + 8 * (r >> 2) + 4 * lh + (r & 3);
          if (key > qi) sc[kt][r] = -INFINITY;
        }
      }
      mraw = lane_max(sc);
    }
    mraw = half_max(mraw);
    const float mt = mraw * scale_log2;  // scale > 0: max commutes with it
    // Lazy rescaling: the exponent reference m_ref only moves when some lane's
    // tile max exceeds it by more than kRescaleSlack, so p = exp2(s - m_ref)
    // stays <= 2^kRescaleSlack; the result is the same softmax (the common
    // factor cancels in O / l), and the rescale multiplies are skipped
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

    // ---- one scheduling region: S(i+1) MFMAs beside the exponentials of i,
    // then PV(i)
    qk(PAR ^ 1, sn, prefetch);
    // The row sum adds the bf16-rounded probabilities that the PV product
    // uses, so O / l is a weighted mean with consistent weights: a query
    // whose mass sits on one key gets that key's value exactly (up to the
    // output rounding), whatever the rounding of its probability.
    uint32_t pk[2][8];
    float ls[2] = {0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const float p0 = fast_exp2(fmaf(sc[kt][r], scale_log2, neg_m));
        const float p1 = fast_exp2(fmaf(sc[kt][r + 1], scale_log2, neg_m));
        const uint32_t pp = cvt_pk_bf16(p0, p1);
        pk[kt][r >> 1] = pp;
        ls[kt] = sum_pk_bf16(pp, ls[kt]);
      }
    }
    l_run += ls[0] + ls[1];
    // O^T += V^T P^T. MFMA step u covers keys 16u .. 16u+15 of the half-tile;
    // slot 8 lh + jj of both operands is key 16u + 8 (jj/4) + 4 lh + jj%4.
    const uint16_t* Vb = Vs + PAR * kHalfElems;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int kt = u >> 1, hf = u & 1;
      const bf16x8 pb = as_bf16x8(
          u32x4{pk[kt][4 * hf], pk[kt][4 * hf + 1], pk[kt][4 * hf + 2], pk[kt][4 * hf + 3]});
      const int row = 16 * u + 4 * lh + (tj >> 2);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int c = 4 * dt + 2 * tg2 + ((tj & 3) >> 1);
        const int off = 4 * (tj & 1);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)&Vb[swz_v(row, c) + off]);
        const s16x4 hi =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)&Vb[swz_v(row + 8, c) + off]);
        const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
        oacc[dt] = mfma32(as_bf16x8(u32x4{lo2[0], lo2[1], hi2[0], hi2[1]}), pb, oacc[dt]);
      }
    }
    mpre = lane_max(sn);  // for the next step, beside the last PV MFMAs
    asm volatile("" ::"v"(mpre));  // (not sunk past the next step's mask branch)
    // Schedule: LDS reads run two MFMAs ahead of their use. The softmax work
    // is spread over all 32 MFMAs so that the VALU between two MFMAs stays
    // well inside one MFMA's 32 cycles: the QK^T MFMAs carry the exponentials
    // of PV steps 0-2 (1.5 per MFMA, with their fma / add / convert), the
    // first 8 PV MFMAs those of PV step 3, the last 8 the max of S(i+1).
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);    // DS read (K operand)
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // QK^T MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
      if (t >= 14) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // VALU
      if (t & 1) __builtin_amdgcn_sched_group_barrier(0x400, 1, 0);  // exp2
      else __builtin_amdgcn_sched_group_barrier(0x400, 2, 0);
    }
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // PV MFMA
      if (t < 14) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS transpose reads
      if (t < 8) {
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        __builtin_amdgcn_sched_group_barrier(0x400, 1, 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
      }
    }
  };

  if (n_kb > 0) {
    f32x16 sa[2], sb[2];
    wait_vmcnt<0>();
    barrier_nofence();
    qk(0, sa, [](int) {});
    float mpre = lane_max(sa);
    for (int p = 0; p < n_kb; ++p) {
      const bool has_next = p + 1 < n_kb;
      const int jn = has_next ? block_at(p + 1) : jc;
      step(std::integral_constant<int, 0>{}, has_next, jn, sa, sb, mpre);
      step(std::integral_constant<int, 1>{}, has_next, jn, sb, sa, mpre);
      jc = jn;
    }
    wait_vmcnt<0>();  // the last prefetches land before the LDS is released
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
  __shared__ __attribute__((aligned(1024))) uint16_t Ks[2 * kHalfElems];
  __shared__ __attribute__((aligned(1024))) uint16_t Vs[2 * kHalfElems];
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
