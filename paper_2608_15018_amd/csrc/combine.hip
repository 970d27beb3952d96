// Combine: y_b = sum_j gate_w[b,j] out[b*k+j] + sum_s out[B*k + s*B + b],
// summed in that order in fp32 (no atomics, so the result is deterministic).
#include "common.h"
#include "kernels.h"

namespace s2moe {

__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  const int b = blockIdx.y;
  const int c = blockIdx.x * blockDim.x + threadIdx.x;  // float4 column
  if (c * 4 >= a.H) return;
  const f32x4* eo = reinterpret_cast<const f32x4*>(a.expert_out);
  const int ldq = a.H / 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < a.k; ++j) {
    const float w = a.gate_w[b * a.k + j];
    const f32x4 v = eo[(size_t)(b * a.k + j) * ldq + c];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = fmaf(w, v[q], acc[q]);
  }
  for (int s = 0; s < a.S; ++s) {
    const f32x4 v = eo[(size_t)(a.B * a.k + s * a.B + b) * ldq + c];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] += v[q];
  }
  reinterpret_cast<f32x4*>(a.y)[(size_t)b * ldq + c] = acc;
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  const int cols = a.H / 4;
  hipLaunchKernelGGL(combine_kernel, dim3((cols + 255) / 256, a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
