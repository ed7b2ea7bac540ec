// Measurement probe (not part of the XAttention ABI; built into its own
// library, libxattn_probe.so, and used by the benchmark only).
//
// xattn_probe_gather: the data movement of the block-sparse attention kernel
// without its arithmetic. Each workgroup (4 waves, two resident per CU like the attention kernel)
// streams a list of 64 KB blocks -- a block stands for one key block's K
// and V, 128 rows x 128 bf16 each -- as four 16 KB half-tiles into a double-
// buffered 64 KB LDS region with the same direct-to-LDS loads, vmcnt waits
// and fence-free barriers, so the rate it reaches is the rate at which that
// load pattern can feed the attention kernel from wherever the blocks live
// (L2, Infinity Cache or HBM, depending on the buffer size).
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "common.h"

using namespace xattn;

namespace {

constexpr int kThreads = 256;
constexpr uint32_t kHalfBytes = 64 * 128 * 2;  // one 64-row x 128-column bf16 half-tile

// Rows 16 wv .. 16 wv + 15 of the half-tile at src (row-major, 256 B rows)
// into LDS at byte address dst: four 1 KB loads per wave.
__device__ __forceinline__ void load_half(const uint16_t* src, uint32_t dst, int wv, int lane) {
  const uint16_t* base = src + (size_t)(16 * wv) * 128;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t off = (uint32_t)(((4 * i + (lane >> 4)) * 128 + (lane & 15) * 8) * 2);
    dma16(base, off, dst + (uint32_t)((16 * wv + 4 * i) * 128 * 2));
  }
}

__global__ __launch_bounds__(kThreads, 2) void gather_probe_kernel(
    const uint16_t* __restrict__ buf, int nblk, const int32_t* __restrict__ blocks, int per_wg,
    uint32_t* __restrict__ sink) {
  __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * 2 * 64 * 128];  // 2 stages x 32 KB
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t l0 = XATTN_LDS_ADDR(lds);
  const int32_t* list = blocks + (size_t)blockIdx.x * per_wg;
  // step s loads half-tile pair s (block s / 2: its K rows for even s, its V
  // rows for odd s) into stage s % 2 while the previous pair is "consumed"
  const int steps = 2 * per_wg;
  for (int s = 0; s < steps; ++s) {
    int j = list[s >> 1];
    j = j < 0 ? 0 : (j >= nblk ? nblk - 1 : j);
    const uint16_t* src = buf + (size_t)j * (64 * 1024 / 2) + (size_t)(s & 1) * (128 * 128);
    const uint32_t st = l0 + (uint32_t)((s & 1) * 2 * kHalfBytes);
    load_half(src, st, wv, lane);
    load_half(src + 64 * 128, st + kHalfBytes, wv, lane);
    wait_vmcnt<8>();    // this wave's loads of the previous pair have landed
    barrier_nofence();  // ... everyone's
  }
  wait_vmcnt<0>();
  barrier_nofence();
  if (threadIdx.x == 0) sink[blockIdx.x] = lds[(blockIdx.x * 97) & (2 * 2 * 64 * 128 - 1)];
}

}  // namespace

// buf: nblk 64 KB blocks (device); blocks: n_wg * per_wg block indices
// (device int32, clamped to [0, nblk)); sink: n_wg uint32 (device). Returns
// a hipError_t as int.
extern "C" int xattn_probe_gather(const void* buf, int nblk, const int32_t* blocks, int per_wg,
                                  int n_wg, uint32_t* sink, void* stream) {
  if (!buf || !blocks || !sink || nblk < 1 || per_wg < 1 || n_wg < 1)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_probe_kernel, dim3(n_wg), dim3(kThreads), 0, (hipStream_t)stream,
                     (const uint16_t*)buf, nblk, blocks, per_wg, sink);
  return (int)hipGetLastError();
}
