// Router logits and plain top-(k+1) per draft token (Sec. "Reuse-aware
// Expert Gating": target gating logits ell_b; gap_b = ell_(1) - ell_(k+1)).
#include "common.h"
#include "kernels.h"

namespace s2moe {

// One wave per (expert, block of 8 tokens).  Lanes split H in 16-byte
// chunks, so a wave reads one router row and one token row coalesced; the
// lane partial sums are added by a butterfly (fixed order, fp32).
template <bool kBf16>
__global__ __launch_bounds__(256) void router_logits_kernel(const void* __restrict__ x,
                                                            const void* __restrict__ router,
                                                            float* __restrict__ logits, int B,
                                                            int H, int E) {
  const int lane = threadIdx.x & (kWave - 1);
  const int e = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (e >= E) return;
  constexpr int kPer = kBf16 ? 8 : 4;  // elements per 16-byte chunk
  const int b0 = blockIdx.y * 8;
  const int b1 = min(B, b0 + 8);
  const int n_chunks = H / kPer;
  for (int b = b0; b < b1; ++b) {
    float acc = 0.f;
    for (int c = lane; c < n_chunks; c += kWave) {
      if (kBf16) {
        const u32x4 w = reinterpret_cast<const u32x4*>(
            static_cast<const uint16_t*>(router) + (size_t)e * H)[c];
        const u32x4 v = reinterpret_cast<const u32x4*>(
            static_cast<const uint16_t*>(x) + (size_t)b * H)[c];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc = fmaf(bf16_to_f32(w[q] & 0xFFFFu), bf16_to_f32(v[q] & 0xFFFFu), acc);
          acc = fmaf(bf16_to_f32(w[q] >> 16), bf16_to_f32(v[q] >> 16), acc);
        }
      } else {
        const f32x4 w = reinterpret_cast<const f32x4*>(
            static_cast<const float*>(router) + (size_t)e * H)[c];
        const f32x4 v = reinterpret_cast<const f32x4*>(
            static_cast<const float*>(x) + (size_t)b * H)[c];
#pragma unroll
        for (int q = 0; q < 4; ++q) acc = fmaf(w[q], v[q], acc);
      }
    }
    acc = wave_sum(acc);
    if (lane == 0) logits[(size_t)b * E + e] = acc;
  }
}

// One wave per token: k+1 rounds of wave argmax give the plain top-k (listed
// in ascending expert id) and the (k+1)-th value for the gap.
__global__ __launch_bounds__(256) void plain_topk_kernel(const float* __restrict__ logits,
                                                         int32_t* __restrict__ plain_idx,
                                                         float* __restrict__ gap, int B, int E,
                                                         int k) {
  const int lane = threadIdx.x & (kWave - 1);
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + kWave * j;
    v[j] = e < E ? logits[(size_t)b * E + e] : 0.f;
  }
  uint32_t bits;
  float top1, kth1;
  wave_topn(v, E, k + 1, k, &bits, &top1, &kth1);
  int rank[4];
  wave_rank_flagged(bits, rank);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if ((bits >> j) & 1u) plain_idx[(size_t)b * k + rank[j]] = lane + kWave * j;
  if (lane == 0) gap[b] = top1 - kth1;
}

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  dim3 g1((a.E + 3) / 4, (a.B + 7) / 8);
  if (a.bf16)
    hipLaunchKernelGGL(router_logits_kernel<true>, g1, dim3(256), 0, s, a.x, a.router, a.logits,
                       a.B, a.H, a.E);
  else
    hipLaunchKernelGGL(router_logits_kernel<false>, g1, dim3(256), 0, s, a.x, a.router,
                       a.logits, a.B, a.H, a.E);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(plain_topk_kernel, dim3((a.B + 3) / 4), dim3(256), 0, s, a.logits,
                     a.plain_idx, a.gap, a.B, a.E, a.k);
  return hipGetLastError();
}

}  // namespace s2moe
