// Combine: y_b = sum_j gate_w[b,j] out[b*k+j] + sum_s out[B*k + s*B + b],
// summed in that order in fp32 (no atomics, so the result is deterministic).
#include "common.h"
#include "kernels.h"

namespace s2moe {

// kG terms are loaded together before they are added (the loads of a group
// are all in flight at once; the additions keep the order above).
template <int kG>
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  const int b = blockIdx.y;
  const int c = blockIdx.x * blockDim.x + threadIdx.x;  // float4 column
  if (c * 4 >= a.H) return;
  const f32x4* eo = reinterpret_cast<const f32x4*>(a.expert_out);
  const int ldq = a.H / 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < a.k; j0 += kG) {
    f32x4 v[kG];
    float w[kG];
#pragma unroll
    for (int u = 0; u < kG; ++u) {
      const int j = min(j0 + u, a.k - 1);
      w[u] = a.gate_w[b * a.k + j];
      v[u] = eo[(size_t)(b * a.k + j) * ldq + c];
    }
#pragma unroll
    for (int u = 0; u < kG; ++u)
      if (j0 + u < a.k) {
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = fmaf(w[u], v[u][q], acc[q]);
      }
  }
  for (int s0 = 0; s0 < a.S; s0 += kG) {
    f32x4 v[kG];
#pragma unroll
    for (int u = 0; u < kG; ++u)
      v[u] = eo[(size_t)(a.B * a.k + min(s0 + u, a.S - 1) * a.B + b) * ldq + c];
#pragma unroll
    for (int u = 0; u < kG; ++u)
      if (s0 + u < a.S) {
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] += v[u][q];
      }
  }
  reinterpret_cast<f32x4*>(a.y)[(size_t)b * ldq + c] = acc;
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  const dim3 grid((a.H / 4 + 255) / 256, a.B);
  const int terms = a.k > a.S ? a.k : a.S;
  if (terms <= 2)
    hipLaunchKernelGGL(combine_kernel<2>, grid, dim3(256), 0, s, a);
  else if (terms <= 4)
    hipLaunchKernelGGL(combine_kernel<4>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(combine_kernel<8>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
