// Per-head output error, the performance proxy of the minimum-threshold
// prediction (Sec. 3.3): err[h] = sum (o - o_ref)^2 / sum o_ref^2 over the
// head's [L][D] bf16 outputs, accumulated in fp64.
//
// Pass 1: grid (chunk, head); each 256-thread workgroup streams one chunk of
// a head with 16-byte loads, every thread sums in fp64, the workgroup reduces
// in a fixed order and writes (num, den) for its chunk. Pass 2: one wave per
// head adds its chunks in index order and divides (for the batch mean, one
// wave per query head then adds the batch's ratios in batch order and
// divides by the batch). Deterministic.
#include "common.h"

using namespace xattn;

namespace {

constexpr int kThreads = 256;
constexpr int kChunkElems = 1 << 17;  // bf16 elements per workgroup (256 KB of o + o_ref)

__device__ __forceinline__ float bf2f(uint32_t bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

__device__ __forceinline__ double wave_sum_f64(double x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__global__ __launch_bounds__(kThreads) void head_error_partials(
    const uint16_t* __restrict__ o, const uint16_t* __restrict__ r, long long per_head,
    int n_chunks, double2* __restrict__ part) {
  const int c = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const long long base = (long long)h * per_head + (long long)c * kChunkElems;
  const long long rem = per_head - (long long)c * kChunkElems;
  const int n = rem < kChunkElems ? (int)rem : kChunkElems;  // multiple of 8 (D = 128)
  const u32x4* o4 = (const u32x4*)(o + base);
  const u32x4* r4 = (const u32x4*)(r + base);
  double num = 0.0, den = 0.0;
  for (int i = tid; i < n / 8; i += kThreads) {
    const u32x4 a = o4[i], b = r4[i];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float a0 = bf2f(a[w] & 0xFFFFu), a1 = bf2f(a[w] >> 16);
      const float b0 = bf2f(b[w] & 0xFFFFu), b1 = bf2f(b[w] >> 16);
      const double d0 = (double)a0 - (double)b0, d1 = (double)a1 - (double)b1;
      num += d0 * d0 + d1 * d1;
      den += (double)b0 * (double)b0 + (double)b1 * (double)b1;
    }
  }
  __shared__ double sn[kThreads / 64], sd[kThreads / 64];
  num = wave_sum_f64(num);
  den = wave_sum_f64(den);
  if ((tid & 63) == 0) {
    sn[tid >> 6] = num;
    sd[tid >> 6] = den;
  }
  __syncthreads();
  if (tid == 0) {
    double tn = 0.0, td = 0.0;
    for (int w = 0; w < kThreads / 64; ++w) {
      tn += sn[w];
      td += sd[w];
    }
    part[(size_t)h * n_chunks + c] = make_double2(tn, td);
  }
}

__device__ __forceinline__ double head_ratio(const double2* __restrict__ part, int n_chunks,
                                             int h) {
  double tn = 0.0, td = 0.0;
  for (int c = 0; c < n_chunks; ++c) {
    const double2 v = part[(size_t)h * n_chunks + c];
    tn += v.x;
    td += v.y;
  }
  return td > 0.0 ? tn / td : (tn > 0.0 ? INFINITY : 0.0);
}

// err[h] for every (batch, query head) row h; with mean_over_batch, err[h]
// for h < hq is instead the mean of the batch's errors of query head h, added
// in batch order.
__global__ __launch_bounds__(64) void head_error_finish(const double2* __restrict__ part,
                                                        int n_chunks, int batch, int hq,
                                                        int mean_over_batch,
                                                        double* __restrict__ err) {
  const int h = blockIdx.x;
  if (threadIdx.x != 0) return;
  if (!mean_over_batch) {
    err[h] = head_ratio(part, n_chunks, h);
    return;
  }
  double sum = 0.0;
  for (int n = 0; n < batch; ++n) sum += head_ratio(part, n_chunks, n * hq + h);
  err[h] = sum / (double)batch;
}

}  // namespace

size_t head_error_scratch_bytes(const XattnShape& s) {
  const long long per_head = (long long)s.seq * s.head_dim;
  const long long n_chunks = (per_head + kChunkElems - 1) / kChunkElems;
  return (size_t)s.HQ() * (size_t)n_chunks * sizeof(double2);
}

hipError_t launch_head_error(const void* o, const void* o_ref, const XattnShape& s, double* err,
                             void* scratch, bool mean_over_batch, hipStream_t st) {
  const long long per_head = (long long)s.seq * s.head_dim;
  const int n_chunks = (int)((per_head + kChunkElems - 1) / kChunkElems);
  hipLaunchKernelGGL(head_error_partials, dim3(n_chunks, s.HQ()), dim3(kThreads), 0, st,
                     (const uint16_t*)o, (const uint16_t*)o_ref, per_head, n_chunks,
                     (double2*)scratch);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_error_finish, dim3(mean_over_batch ? s.hq : s.HQ()), dim3(64), 0, st,
                     (const double2*)scratch, n_chunks, s.batch, s.hq, mean_over_batch ? 1 : 0,
                     err);
  return hipGetLastError();
}
