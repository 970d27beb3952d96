// Grouped SwiGLU experts over the verify batch: the fp32 path and the
// dispatch to the matrix-core paths (ffn_bf16.hip, ffn_q4.hip).
//
// For every activated expert e (and every shared expert) the tokens routed
// to it are processed together, so each weight row is read from HBM once
// per verify batch however many tokens use the expert -- the parameter
// reuse that reuse-aware gating is designed to raise.
//
//   gate-up:  Hh[t, f] = silu(W_g[f,:] . x_t) * (W_u[f,:] . x_t)
//   down:     out[t, h] = W_d[h,:] . Hh_t
//
// fp32 weights use a VALU path: one wave per weight row, lanes split K, up
// to 8 tokens per pass, butterfly reduction.
#include "ffn_common.h"

namespace s2moe {

using namespace ffn;

namespace {

// ---------------------------------------------------------------- fp32 path
template <int kMode>
__global__ __launch_bounds__(256) void ffn_f32_kernel(FfnArgs a) {
  Segment seg;
  int rb;
  if (!resolve_block(a, kMode, 4, &seg, &rb)) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int row = rb * 4 + wave_id();
  const int rows = kMode == 0 ? (seg.shared ? a.Fs : a.F) : a.H;
  const int K = kMode == 0 ? a.H : (seg.shared ? a.Fs : a.F);
  const float* W0;
  const float* W1 = nullptr;
  const size_t mat = (size_t)rows * K;
  if (kMode == 0) {
    W0 = static_cast<const float*>(seg.shared ? a.sh_gate : a.gate) + seg.id * mat;
    W1 = static_cast<const float*>(seg.shared ? a.sh_up : a.up) + seg.id * mat;
  } else {
    W0 = static_cast<const float*>(seg.shared ? a.sh_down : a.down) + seg.id * mat;
  }
  W0 += (size_t)row * K;
  if (kMode == 0) W1 += (size_t)row * K;
  const float* X = kMode == 0 ? static_cast<const float*>(a.x) : static_cast<const float*>(a.hh);
  const int ldx = kMode == 0 ? a.H : a.ldh;

  for (int t0 = 0; t0 < seg.n; t0 += 8) {
    float acc0[8], acc1[8];
    const float* xr[8];
#pragma unroll
    for (int tt = 0; tt < 8; ++tt) {
      acc0[tt] = 0.f;
      acc1[tt] = 0.f;
      xr[tt] = X + (size_t)x_row(a, kMode, seg, min(t0 + tt, seg.n - 1)) * ldx;
    }
    for (int c = lane * 4; c < K; c += 4 * kWave) {
      const f32x4 w0 = *reinterpret_cast<const f32x4*>(W0 + c);
      f32x4 w1 = w0;
      if (kMode == 0) w1 = *reinterpret_cast<const f32x4*>(W1 + c);
#pragma unroll
      for (int tt = 0; tt < 8; ++tt) {
        const f32x4 xv = *reinterpret_cast<const f32x4*>(xr[tt] + c);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc0[tt] = fmaf(w0[q], xv[q], acc0[tt]);
          if (kMode == 0) acc1[tt] = fmaf(w1[q], xv[q], acc1[tt]);
        }
      }
    }
#pragma unroll
    for (int tt = 0; tt < 8; ++tt) {
      acc0[tt] = wave_sum(acc0[tt]);
      if (kMode == 0) acc1[tt] = wave_sum(acc1[tt]);
    }
    if (lane == 0) {
#pragma unroll
      for (int tt = 0; tt < 8; ++tt) {
        const int t = t0 + tt;
        if (t >= seg.n) break;
        if (kMode == 0)
          static_cast<float*>(a.hh)[(size_t)(seg.base + t) * a.ldh + row] =
              silu(acc0[tt]) * acc1[tt];
        else
          a.out[(size_t)out_row(a, seg, t) * a.H + row] = acc0[tt];
      }
    }
  }
}

}  // namespace

hipError_t launch_ffn(const FfnArgs& a, hipStream_t s) {
  if (a.wf == kWF32) {
    hipLaunchKernelGGL(ffn_f32_kernel<0>, dim3(n_blocks(a, 0, 4)), dim3(256), 0, s, a);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(ffn_f32_kernel<1>, dim3(n_blocks(a, 1, 4)), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (a.wf == kWBf16) return launch_ffn_bf16(a, s);
  return launch_ffn_q4(a, s);
}

}  // namespace s2moe
