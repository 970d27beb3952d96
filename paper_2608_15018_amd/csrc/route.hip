// Router logits and plain top-(k+1) per draft token (Sec. "Reuse-aware
// Expert Gating": target gating logits ell_b; gap_b = ell_(1) - ell_(k+1)).
//
// One workgroup of up to 16 waves per token.  Waves take experts
// round-robin; for each, the lanes split H in 16-byte chunks (one router row
// and the token row read coalesced, several chunks in flight) and a DPP
// reduction adds the lane partials in a fixed order.  Wave 0 then ranks the
// E logits with a bitwise threshold search for the (k+1)-th largest key.
#include "common.h"
#include "kernels.h"

namespace s2moe {

namespace {

template <bool kBf16>
__device__ __forceinline__ float dot_row(const void* x, const void* w, int H, int lane) {
  float acc = 0.f;
  if (kBf16) {
    const u32x4* wr = reinterpret_cast<const u32x4*>(w);
    const u32x4* xr = reinterpret_cast<const u32x4*>(x);
    const int n = H / 8;
#pragma unroll 4
    for (int c = lane; c < n; c += kWave) {
      const u32x4 wc = wr[c], xc = xr[c];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc = fmaf(bf16_to_f32(wc[q] & 0xFFFFu), bf16_to_f32(xc[q] & 0xFFFFu), acc);
        acc = fmaf(bf16_to_f32(wc[q] >> 16), bf16_to_f32(xc[q] >> 16), acc);
      }
    }
  } else {
    const f32x4* wr = reinterpret_cast<const f32x4*>(w);
    const f32x4* xr = reinterpret_cast<const f32x4*>(x);
    const int n = H / 4;
#pragma unroll 4
    for (int c = lane; c < n; c += kWave) {
      const f32x4 wc = wr[c], xc = xr[c];
#pragma unroll
      for (int q = 0; q < 4; ++q) acc = fmaf(wc[q], xc[q], acc);
    }
  }
  return wave_sum_dpp(acc);
}

template <bool kBf16>
__global__ __launch_bounds__(1024) void route_kernel(RouteArgs a) {
  __shared__ float ell_s[kMaxExperts];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x >> 6;
  const int n_waves = blockDim.x >> 6;
  const int b = blockIdx.x;
  const int H = a.H, E = a.E, k = a.k;
  const size_t esz = kBf16 ? 2 : 4;
  const char* xb = static_cast<const char*>(a.x) + (size_t)b * H * esz;
  const char* wr = static_cast<const char*>(a.router);

  for (int e = wave; e < E; e += n_waves) {
    const float l = dot_row<kBf16>(xb, wr + (size_t)e * H * esz, H, lane);
    if (lane == 0) {
      ell_s[e] = l;
      a.logits[(size_t)b * E + e] = l;
    }
  }
  __syncthreads();
  if (wave != 0) return;

  const int nj = (E + kWave - 1) / kWave;
  uint64_t key[4];
  float vmax = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + kWave * j;
    key[j] = 0;
    if (e < E) {
      const float v = ell_s[e];
      key[j] = rank_key(v, e);
      vmax = fmaxf(vmax, v);
    }
  }
  // (k+1)-th largest key: the plain top-k are exactly the keys above it.
  const uint64_t kth1 = wave_kth_key(key, nj, k + 1);
  const float top1 = wave_max_dpp(vmax);
  uint32_t bits = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (key[j] > kth1) bits |= 1u << j;
  int rank[4];
  wave_rank_flagged(bits, rank);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if ((bits >> j) & 1u) a.plain_idx[(size_t)b * k + rank[j]] = lane + kWave * j;
  if (lane == 0) a.gap[b] = top1 - key_value((uint32_t)(kth1 >> 16));
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  const int waves = a.E >= 16 ? 16 : a.E;  // at most one wave per expert
  const dim3 block(64 * waves);
  if (a.bf16)
    hipLaunchKernelGGL(route_kernel<true>, dim3(a.B), block, 0, s, a);
  else
    hipLaunchKernelGGL(route_kernel<false>, dim3(a.B), block, 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
