// Router logits and plain top-(k+1) per draft token (Sec. "Reuse-aware
// Expert Gating": target gating logits ell_b; gap_b = ell_(1) - ell_(k+1)).
//
// One workgroup of up to 16 waves per token.  Each wave takes 4 experts per
// pass; the lanes split H in 16-byte chunks (the token row and 4 router rows
// read coalesced, all in flight together) and DPP reductions add the lane
// partials in a fixed order.  Wave 0 then ranks the E logits with a bitwise
// threshold search for the (k+1)-th largest value.
#include "common.h"
#include "kernels.h"

namespace s2moe {

namespace {

// Dot products of the token row with 4 router rows (e0 .. e0+3, those < E):
// lanes split H in 16-byte chunks, so each iteration has 5 loads in flight.
template <bool kBf16>
__device__ __forceinline__ void dot_rows4(const char* x, const char* w, int H, int e0, int E,
                                          int lane, float acc[4]) {
  const size_t row = (size_t)H * (kBf16 ? 2 : 4);
  const int n = H / (kBf16 ? 8 : 4);
  const u32x4* xr = reinterpret_cast<const u32x4*>(x);
  const u32x4* wr[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    acc[q] = 0.f;
    wr[q] = reinterpret_cast<const u32x4*>(w + (size_t)min(e0 + q, E - 1) * row);
  }
#pragma unroll 2
  for (int c = lane; c < n; c += kWave) {
    const u32x4 xc = xr[c];
    u32x4 wc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) wc[q] = wr[q][c];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (kBf16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[q] = fmaf(bf16_to_f32(wc[q][i] & 0xFFFFu), bf16_to_f32(xc[i] & 0xFFFFu), acc[q]);
          acc[q] = fmaf(bf16_to_f32(wc[q][i] >> 16), bf16_to_f32(xc[i] >> 16), acc[q]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[q] = fmaf(__uint_as_float(wc[q][i]), __uint_as_float(xc[i]), acc[q]);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) acc[q] = wave_sum_dpp(acc[q]);
}

template <bool kBf16>
__global__ __launch_bounds__(1024) void route_kernel(RouteArgs a) {
  __shared__ float ell_s[kMaxExperts];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x >> 6;
  const int n_waves = blockDim.x >> 6;
  const int b = blockIdx.x;
  const int H = a.H, E = a.E, k = a.k;
  const char* xb = static_cast<const char*>(a.x) + (size_t)b * H * (kBf16 ? 2 : 4);
  const char* wr = static_cast<const char*>(a.router);

  for (int e0 = wave * 4; e0 < E; e0 += n_waves * 4) {
    float l[4];
    dot_rows4<kBf16>(xb, wr, H, e0, E, lane, l);
    if (lane == 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (e0 + q < E) {
          ell_s[e0 + q] = l[q];
          a.logits[(size_t)b * E + e0 + q] = l[q];
        }
      }
    }
  }
  __syncthreads();
  if (wave != 0) return;

  uint32_t key[4];
  float vmax = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + kWave * j;
    key[j] = 0;
    if (e < E) {
      const float v = ell_s[e];
      key[j] = order_key(v);
      vmax = fmaxf(vmax, v);
    }
  }
  // ell_(k+1) is the (k+1)-th largest value; the plain top-k are the k best
  // entries, which all rank at or above it.
  const uint32_t kth1 = wave_kth_key(key, k + 1);
  const float top1 = wave_max_dpp(vmax);
  const uint32_t bits = wave_select_top(key, kth1, k);
  int rank[4];
  wave_rank_flagged(bits, rank);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if ((bits >> j) & 1u) a.plain_idx[(size_t)b * k + rank[j]] = lane + kWave * j;
  if (lane == 0) a.gap[b] = top1 - key_value(kth1);
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  const int waves = min(16, (a.E + 3) / 4);  // 4 experts per wave and pass
  const dim3 block(64 * waves);
  if (a.bf16)
    hipLaunchKernelGGL(route_kernel<true>, dim3(a.B), block, 0, s, a);
  else
    hipLaunchKernelGGL(route_kernel<false>, dim3(a.B), block, 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
