// Internal helpers of the gfx950 XAttention library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xattn {

typedef __bf16 bf16_t;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

constexpr int kBlock = 128;     // B: attention / selection block size
constexpr int kHeadDim = 128;   // d
constexpr int kWave = 64;
constexpr int kNumXcd = 8;      // MI355X: 8 XCDs, workgroups dispatched round-robin
constexpr float kLog2e = 1.4426950408889634f;

// 32x32x16 bf16 MFMA, fp32 accumulate. Lane i supplies A[i%32][8*(i/32) .. +8]
// and B[8*(i/32) .. +8][i%32]; accumulator register r of lane i holds
// D[8*(r/4) + 4*(i/32) + r%4][i%32].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Direct-to-LDS load of 16 bytes per lane: lane l's bytes land at LDS byte
// address lds + 16 l (lds wave-uniform, passed through M0); the global address
// is sbase (scalar) + voff (per lane, bytes). Issued as inline asm so the
// compiler does not track it: lacking alias information it would otherwise
// stall every LDS read on every such load in flight. Kernels order these
// loads themselves (explicit vmcnt waits + barriers).
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}

// Wait until at most N of this wave's vector-memory loads are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier that does not wait for vector-memory loads (prefetches
// into LDS stay in flight; __syncthreads would drain them). Each wave first
// waits for its own outstanding LDS reads (lgkmcnt(0)): the compiler may sink
// the instruction consuming a ds_read below the barrier, and without the wait
// another wave could refill the buffer before that read returns. Waiting for
// a wave's own direct-to-LDS loads (vmcnt) is left to the caller.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

#define XATTN_LDS_ADDR(p) ((uint32_t)(uintptr_t)((__attribute__((address_space(3))) void*)(p)))

}  // namespace xattn

// Kernel launchers (one per .hip file), called by the C ABI layer after the
// arguments have been validated. They return hipSuccess or the launch error.
struct XattnShape {
  int batch, hq, hkv, seq, head_dim, causal;
  int HQ() const { return batch * hq; }
  int NB() const { return seq / xattn::kBlock; }
};

// Query sub-row paired with key sub-row t inside each S x S sub-block of the
// scoring: S-1-t is the antidiagonal of Algorithm 1 (qsub == nullptr); other
// permutations give the diagonal / random patterns. Passed by value.
struct SubRowPairing {
  int q[64];
};
hipError_t launch_score(const void* q, const void* k, const XattnShape& s, int stride,
                        const int32_t* qsub, float* scores, void* scratch, hipStream_t st);
size_t score_scratch_bytes(const XattnShape& s, int stride);
// Views of the scoring scratch: partial block masses and row statistics.
struct ScoreScratch {
  float* part;   // partial block masses (layout in score_rows.h)
  float* stats;  // float2 (max, sum) per reduced row and column sub-tile
};
ScoreScratch score_scratch_views(const XattnShape& s, int stride, void* scratch);
// Selection rule of one launch: find_blocks with a threshold per head, or a
// fixed block count per head (Top-K) or fraction of the candidates
// (Top-Ratio). Passed by value as a kernel argument; with uniform != 0 every
// head uses entry 0 (then hq may exceed kMaxSelectHeads).
constexpr int kMaxSelectHeads = 256;
enum { kSelectThreshold = 0, kSelectTopK = 1, kSelectRatio = 2 };
struct SelectParams {
  int mode, hq, uniform;
  float v[kMaxSelectHeads];  // tau (threshold) or ratio (Top-Ratio)
  int k[kMaxSelectHeads];    // blocks (Top-K)
};
hipError_t launch_select(const float* scores, const XattnShape& s, const SelectParams& p,
                         int32_t* idx, int32_t* cnt, hipStream_t st);
size_t head_error_scratch_bytes(const XattnShape& s);
hipError_t launch_head_error(const void* o, const void* o_ref, const XattnShape& s, double* err,
                             void* scratch, bool mean_over_batch, hipStream_t st);
hipError_t launch_attn(const void* q, const void* k, const void* v, const XattnShape& s,
                       const int32_t* idx, const int32_t* cnt, bool dense, void* o,
                       float* lse, hipStream_t st);
// The static scratch of xattn_forward_noalloc (XATTN_NOALLOC_SCRATCH_BYTES
// bytes per device): its device address on the current device, fetched on
// the first call per device.
constexpr size_t kNoallocScratchBytes = (size_t)64 << 20;
hipError_t noalloc_scratch(void** ptr);
