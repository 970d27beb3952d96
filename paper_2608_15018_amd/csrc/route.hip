// Router logits and plain top-(k+1) per draft token (Sec. "Reuse-aware
// Expert Gating": target gating logits ell_b; gap_b = ell_(1) - ell_(k+1)).
//
// Two paths.  Small batches, and batches over many experts, compute the
// logits with one wave per (router row, token) pair and rank them in a second
// launch, one wave per token.  Otherwise one workgroup of up to 16 waves per
// token does both.  There a wave takes 4 experts and a
// slice of H per item (H is sliced when there are few experts, so that all
// waves load at once); its lanes split the slice in 16-byte chunks (the
// token row and 4 router rows read coalesced, all in flight together), DPP
// reductions add the lane partials and the slices are summed in order.
// Wave 0 then ranks the E logits: an exact top-(k+1) by ballots over the
// order keys, as in the gating kernel.
#include "q4_layout.h"
#include "small_batch.h"

namespace s2moe {

namespace {

// Partial dot products of the token row with 4 router rows (e0 .. e0+3,
// those < E) over the 16-byte chunks [c_lo, c_hi) of H: lanes split the
// chunks, so up to 4 iterations x 5 loads are in flight together.
template <bool kBf16>
__device__ __forceinline__ void dot_rows4(const char* x, const char* w, int H, int e0, int E,
                                          int c_lo, int c_hi, int lane, float acc[4]) {
  const size_t row = (size_t)H * (kBf16 ? 2 : 4);
  const u32x4* xr = reinterpret_cast<const u32x4*>(x);
  const u32x4* wr[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    acc[q] = 0.f;
    wr[q] = reinterpret_cast<const u32x4*>(w + (size_t)min(e0 + q, E - 1) * row);
  }
#pragma unroll 4
  for (int c = c_lo + lane; c < c_hi; c += kWave) {
    const u32x4 xc = xr[c];
    u32x4 wc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) wc[q] = wr[q][c];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = dot_chunk<kBf16>(xc, wc[q], acc[q]);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) acc[q] = wave_sum_dpp(acc[q]);
}

// Number of H slices: as many as keep every wave busy (slices x expert
// groups <= 16) while each slice still spans at least 64 chunks.
__host__ __device__ inline int route_slices(int E, int chunks) {
  const int groups = (E + 3) / 4;
  int S = 1;
  while (S * 2 * groups <= 16 && chunks / (S * 2) >= kWave) S *= 2;
  return S;
}

// Small batches and many experts: one wave per (router row, token) pair
// (grid: E / 4 x B workgroups of 4 waves), so the E rows are streamed by
// waves spread over the GPU instead of by one workgroup per token.
template <bool kBf16>
__global__ __launch_bounds__(256) void route_rows_kernel(RouteArgs a) {
  if ((int)blockIdx.y >= a.B) {
    // Rows of workgroups past the B tokens convert x (a.x16 set).
    const int blk = (blockIdx.y - a.B) * gridDim.x + blockIdx.x;
    prep_x8(static_cast<const uint16_t*>(a.x), a.x16, blk * 256 + threadIdx.x, a.n8);
    return;
  }
  route_row_logit<kBf16>(a, blockIdx.x * 4 + wave_id(), blockIdx.y);
}

// Small batches, second launch: one wave per token ranks the logits
// route_rows_kernel wrote.
template <int NJ>
__global__ __launch_bounds__(kWave) void route_select_wave_kernel(RouteArgs a) {
  const int b = blockIdx.x;
  wave_select_plain<NJ>(a.E, a.k, a.logits + (size_t)b * a.E, a.plain_idx + (size_t)b * a.k,
                        a.gap + b, static_cast<int32_t*>(nullptr), nullptr);
}

template <bool kBf16, int NJ>
__global__ __launch_bounds__(1024) void route_kernel(RouteArgs a) {
  if ((int)blockIdx.x >= a.B) {
    // Workgroups past the B tokens convert x (a.x16 set).
    prep_x8(static_cast<const uint16_t*>(a.x), a.x16,
            (blockIdx.x - a.B) * blockDim.x + threadIdx.x, a.n8);
    return;
  }
  __shared__ float part_s[kMaxExperts];  // [slice][E]: slices * E <= 256
  __shared__ float ell_s[kMaxExperts];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = wave_id();
  const int n_waves = blockDim.x >> 6;
  const int b = blockIdx.x;
  const int H = a.H, E = a.E;
  const char* xb = static_cast<const char*>(a.x) + (size_t)b * H * (kBf16 ? 2 : 4);
  const char* wr = static_cast<const char*>(a.router);
  const int chunks = H / (kBf16 ? 8 : 4);
  const int groups = (E + 3) / 4;
  const int S = route_slices(E, chunks);
  const int per_slice = (chunks + S - 1) / S;

  // Work item p = (slice, group of 4 experts), p = slice * groups + group.
  for (int p = wave; p < S * groups; p += n_waves) {
    const int slice = p / groups, e0 = (p - slice * groups) * 4;
    const int c_lo = slice * per_slice, c_hi = min(chunks, c_lo + per_slice);
    float l[4];
    dot_rows4<kBf16>(xb, wr, H, e0, E, c_lo, c_hi, lane, l);
    if (lane == 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (e0 + q < E) part_s[slice * E + e0 + q] = l[q];
    }
  }
  __syncthreads();
  if (tid < E) {
    float v = part_s[tid];
    for (int sl = 1; sl < S; ++sl) v += part_s[sl * E + tid];
    ell_s[tid] = v;
    a.logits[(size_t)b * E + tid] = v;
  }
  __syncthreads();
  if (wave == 0)
    wave_select_plain<NJ>(E, a.k, ell_s, a.plain_idx + (size_t)b * a.k, a.gap + b,
                          static_cast<int32_t*>(nullptr), nullptr);
}

}  // namespace

// The two-launch path (router rows spread over the GPU, then one wave per
// token ranking its logits) serves batches up to this many tokens, and every
// batch when there are more than S2MOE_ROUTE_ROWS_MIN_E experts (the one
// workgroup per token of route_kernel would stream the whole router through
// each token's compute unit).
#ifndef S2MOE_ROUTE_ROWS_MAX_B
#define S2MOE_ROUTE_ROWS_MAX_B 8
#endif
#ifndef S2MOE_ROUTE_ROWS_MIN_E
#define S2MOE_ROUTE_ROWS_MIN_E 64
#endif

hipError_t launch_route_rows(const RouteArgs& a, hipStream_t s) {
  const int gx = (a.E + 3) / 4;
  const int prep_rows = a.x16 ? (a.n8 + 256 * gx - 1) / (256 * gx) : 0;
  const dim3 grid(gx, a.B + prep_rows);
  if (a.bf16)
    hipLaunchKernelGGL(route_rows_kernel<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(route_rows_kernel<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

bool route_ranks_separately(const RouteArgs& a) {
  return a.B <= S2MOE_ROUTE_ROWS_MAX_B || a.E > S2MOE_ROUTE_ROWS_MIN_E;
}

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  if (route_ranks_separately(a)) {
    const hipError_t e = launch_route_rows(a, s);
    if (e != hipSuccess) return e;
    if (a.E <= 64)
      hipLaunchKernelGGL(route_select_wave_kernel<1>, dim3(a.B), dim3(kWave), 0, s, a);
    else if (a.E <= 128)
      hipLaunchKernelGGL(route_select_wave_kernel<2>, dim3(a.B), dim3(kWave), 0, s, a);
    else
      hipLaunchKernelGGL(route_select_wave_kernel<4>, dim3(a.B), dim3(kWave), 0, s, a);
    return hipGetLastError();
  }
  // One wave per (H slice, 4 experts) item, at most 16; with 4 experts per
  // wave there is a thread per expert to add the slices.
  const int chunks = a.H / (a.bf16 ? 8 : 4);
  const int waves = min(16, route_slices(a.E, chunks) * ((a.E + 3) / 4));
  const dim3 block(64 * waves);
  const dim3 grid(a.B + (a.x16 ? (a.n8 + 64 * waves - 1) / (64 * waves) : 0));
  if (a.E <= 64) {
    if (a.bf16) hipLaunchKernelGGL((route_kernel<true, 1>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((route_kernel<false, 1>), grid, block, 0, s, a);
  } else if (a.E <= 128) {
    if (a.bf16) hipLaunchKernelGGL((route_kernel<true, 2>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((route_kernel<false, 2>), grid, block, 0, s, a);
  } else {
    if (a.bf16) hipLaunchKernelGGL((route_kernel<true, 4>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((route_kernel<false, 4>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace s2moe
