// Read-stream probe: how fast this GPU delivers a plain sequential read with
// the 16-byte nontemporal loads the expert-FFN kernels use.  A diagnostic
// beside the FFN roofline, not a step of the verify pass.
#include "common.h"
#include "kernels.h"

namespace s2moe {

namespace {

// Each wave owns one contiguous range of the 16-byte chunks (a multiple of
// 8 KB) and reads it front to back, 8 KB per iteration (lane L takes chunks
// L, L + 64, ...: each load instruction covers 1 KB); the XOR of everything
// a block read goes to one sink word so the loads cannot be dropped.
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ src,
                                                          size_t n16, uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & (kWave - 1);
  const size_t waves = (size_t)gridDim.x * (blockDim.x / kWave);
  const size_t wave = (size_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
  const size_t per = ((n16 + waves - 1) / waves + 511) & ~(size_t)511;
  size_t i = wave * per;
  const size_t end = min(n16, i + per);
  uint32_t acc = 0;
  for (; i + 512 <= end; i += 512) {
    u32x4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = __builtin_nontemporal_load(src + i + q * kWave + lane);
#pragma unroll
    for (int q = 0; q < 8; ++q) acc ^= v[q][0] ^ v[q][1] ^ v[q][2] ^ v[q][3];
  }
  for (; i < end; i += kWave) {
    if (i + lane < end) {
      const u32x4 v = __builtin_nontemporal_load(src + i + lane);
      acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
  }
  __shared__ uint32_t red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
    for (int t = 0; t < 256; ++t) r ^= red[t];
    sink[blockIdx.x] = r;
  }
}

}  // namespace

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, int blocks,
                              hipStream_t s) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(256), 0, s,
                     static_cast<const u32x4*>(src), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace s2moe
