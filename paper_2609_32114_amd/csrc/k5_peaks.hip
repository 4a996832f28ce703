// k5_peaks.hip -- measured ceilings for the roofline fractions: a streaming
// device copy (the HBM bandwidth a plain kernel reaches on this device) and a
// loop of independent bf16 MFMAs (the matrix-core rate).  Measurement aids
// only: no prefill or decode call launches them.
#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kPeakThreads = 256;

// dst[i] = src[i] for n 16-byte vectors, grid-stride, nontemporal so that the
// stream bypasses the caches the way a first touch of HBM data does.
__global__ __launch_bounds__(kPeakThreads) void copy_kernel(const u32x4 *__restrict__ src, u32x4 *__restrict__ dst,
                                                          size_t n) {
  const size_t stride = (size_t)gridDim.x * kPeakThreads;
  for (size_t i = (size_t)blockIdx.x * kPeakThreads + threadIdx.x; i < n; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(src + i);
    __builtin_nontemporal_store(v, dst + i);
  }
}

// Every wave runs `iters` rounds of 8 independent 16x16x32 bf16 MFMA chains
// (8 x 16 x 16 x 32 multiply-adds per round); lane 0 of each wave stores a
// sum so the chains are live.
__global__ __launch_bounds__(kPeakThreads) void mfma_loop_kernel(int iters, float *sink) {
  const int lane = threadIdx.x & 63;
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = 1e-3f * (float)(lane + j);
  const bf16x8 a = make_frag<bf16_t>(x);
  f32x4 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = zero4();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = mma(acc[j], a, a);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  if (lane == 0) sink[(size_t)blockIdx.x * (kPeakThreads / 64) + (threadIdx.x >> 6)] = s;
}

hipError_t launch_copy(const void *src, void *dst, size_t bytes, int cus, hipStream_t stream) {
  const size_t n = bytes / 16;
  const unsigned blocks = (unsigned)(cus > 0 ? cus * 8 : 2048);
  hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(kPeakThreads), 0, stream, static_cast<const u32x4 *>(src),
                     static_cast<u32x4 *>(dst), n);
  return hipGetLastError();
}

hipError_t launch_mfma_loop(int blocks, int iters, float *sink, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_loop_kernel, dim3((unsigned)blocks), dim3(kPeakThreads), 0, stream, iters, sink);
  return hipGetLastError();
}

}  // namespace hagdn
