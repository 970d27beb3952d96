// Grouped SwiGLU experts over the verify batch.
//
// For every activated expert e (and every shared expert) the tokens routed
// to it are processed together, so each weight row is read from HBM once
// per verify batch however many tokens use the expert -- the parameter
// reuse that reuse-aware gating is designed to raise.
//
//   gate-up:  Hh[t, f] = silu(W_g[f,:] . x_t) * (W_u[f,:] . x_t)
//   down:     out[t, h] = W_d[h,:] . Hh_t
//
// Both are skinny products out[t, r] = sum_k W[r, k] X[t, k] with K
// contiguous in W.  The bf16 / int4 path runs them on the matrix cores with
// v_mfma_f32_16x16x32_bf16: a wave owns 16 weight rows (the A operand, read
// straight from HBM) and up to 64 tokens (four B tiles of 16, read from
// L2-resident activations); columns of B beyond the expert's token count
// hold copies of a valid token and are never stored.  fp32 weights use a
// VALU path (lanes split K, butterfly reduction).
//
// int4 (4-bit codes, 32-element groups, fp16 scales): one MFMA step covers
// exactly one group of 32 K elements.  The codes are expanded to the exact
// bf16 values 128 + q with one and-or per pair, the MFMA gives
// P = sum (128 + q) x and a second MFMA with an all-ones A gives Sx = sum x,
// and the group contributes s * (P - 136 Sx) = s * sum (q - 8) x in fp32.
// No dequantised weight ever reaches memory.
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
  const int row = rb * 4 + (threadIdx.x >> 6);
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

template <int T, int kMode>
__device__ __forceinline__ void mfma_tile_q4(const FfnArgs& a, const Segment& seg, int t0,
                                             int r0, int K, const uint8_t* C0,
                                             const uint8_t* C1, const uint16_t* S0,
                                             const uint16_t* S1) {
  constexpr bool kDual = kMode == 0;
  constexpr int U = 8;  // steps (= groups) per block; K % 256 == 0
  const int lane = threadIdx.x & (kWave - 1);
  const int rA = lane & 15, gK = lane >> 4;
  const int nks = K / 32;
  const int srow = K / 32;  // scales per row
  const uint16_t* X = static_cast<const uint16_t*>(kMode == 0 ? a.x : a.hh);
  const int ldx = kMode == 0 ? a.H : a.ldh;
  const u32x4* xb[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int t = min(t0 + tt * 16 + rA, seg.n - 1);
    xb[tt] = reinterpret_cast<const u32x4*>(X + (size_t)x_row(a, kMode, seg, t) * ldx) + gK;
  }
  // codes: 16 bytes per group per row; the lane's 8 elements are bytes 4 gK..4 gK+3
  const uint32_t* pc0 =
      reinterpret_cast<const uint32_t*>(C0 + (size_t)(r0 + rA) * (K / 2)) + gK;
  const uint32_t* pc1 =
      kDual ? reinterpret_cast<const uint32_t*>(C1 + (size_t)(r0 + rA) * (K / 2)) + gK : pc0;
  // scales of the lane's four output rows 4 gK + i
  const int m0 = r0 + 4 * gK;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  u32x4 ones_u;
#pragma unroll
  for (int q = 0; q < 4; ++q) ones_u[q] = 0x3F803F80u;
  const bf16x8 ones = as_bf16x8(ones_u);

  f32x4 acc0[T], acc1[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    acc0[tt] = zero;
    acc1[tt] = zero;
  }
  for (int ks = 0; ks < nks; ks += U) {
    uint32_t c0[U], c1[U];
    u32x4 sc0[4], sc1[4], Bn[T][U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      c0[u] = pc0[4 * (ks + u)];
      if (kDual) c1[u] = pc1[4 * (ks + u)];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc0[i] = *reinterpret_cast<const u32x4*>(S0 + (size_t)(m0 + i) * srow + ks);
      if (kDual) sc1[i] = *reinterpret_cast<const u32x4*>(S1 + (size_t)(m0 + i) * srow + ks);
    }
#pragma unroll
    for (int tt = 0; tt < T; ++tt)
#pragma unroll
      for (int u = 0; u < U; ++u) Bn[tt][u] = xb[tt][4 * (ks + u)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bf16x8 A0 = q4_expand(c0[u]);
      const bf16x8 A1 = kDual ? q4_expand(c1[u]) : A0;
      float s0[4], s1[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t pair0 = sc0[i][u >> 1];
        s0[i] = f16_bits_to_f32((uint16_t)((u & 1) ? (pair0 >> 16) : (pair0 & 0xFFFFu)));
        if (kDual) {
          const uint32_t pair1 = sc1[i][u >> 1];
          s1[i] = f16_bits_to_f32((uint16_t)((u & 1) ? (pair1 >> 16) : (pair1 & 0xFFFFu)));
        }
      }
#pragma unroll
      for (int tt = 0; tt < T; ++tt) {
        const bf16x8 Bp = q4_permute_x(Bn[tt][u]);
        const f32x4 sx = mfma(ones, Bp, zero);
        const f32x4 p0 = mfma(A0, Bp, zero);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc0[tt][i] = fmaf(s0[i], fmaf(-136.f, sx[i], p0[i]), acc0[tt][i]);
        if (kDual) {
          const f32x4 p1 = mfma(A1, Bp, zero);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc1[tt][i] = fmaf(s1[i], fmaf(-136.f, sx[i], p1[i]), acc1[tt][i]);
        }
      }
    }
  }
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int t = t0 + tt * 16 + rA;
    if (t >= seg.n) continue;
    if (kMode == 0) {
      uint32_t h[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) h[i] = f32_to_bf16(silu(acc0[tt][i]) * acc1[tt][i]);
      uint2 v;
      v.x = h[0] | (h[1] << 16);
      v.y = h[2] | (h[3] << 16);
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.hh) + (size_t)(seg.base + t) * a.ldh +
                                m0) = v;
    } else {
      *reinterpret_cast<f32x4*>(a.out + (size_t)out_row(a, seg, t) * a.H + m0) = acc0[tt];
    }
  }
}

template <int kMode>
__global__ __launch_bounds__(256) void ffn_q4_kernel(FfnArgs a) {
  Segment seg;
  int rb;
  if (!resolve_block(a, kMode, 64, &seg, &rb)) return;
  const int r0 = rb * 64 + (threadIdx.x >> 6) * 16;
  const int rows = kMode == 0 ? (seg.shared ? a.Fs : a.F) : a.H;
  const int K = kMode == 0 ? a.H : (seg.shared ? a.Fs : a.F);
  const void* M0;
  const void* M1 = nullptr;
  const void* Q0 = nullptr;
  const void* Q1 = nullptr;
  if (kMode == 0) {
    M0 = seg.shared ? a.sh_gate : a.gate;
    M1 = seg.shared ? a.sh_up : a.up;
    Q0 = seg.shared ? a.sh_gate_s : a.gate_s;
    Q1 = seg.shared ? a.sh_up_s : a.up_s;
  } else {
    M0 = seg.shared ? a.sh_down : a.down;
    Q0 = seg.shared ? a.sh_down_s : a.down_s;
  }
  const size_t mat = (size_t)rows * K;  // weights per expert matrix
  for (int t0 = 0; t0 < seg.n; t0 += 64) {
    const int T = min(4, (seg.n - t0 + 15) / 16);
    const uint8_t* C0 = static_cast<const uint8_t*>(M0) + seg.id * (mat / 2);
    const uint8_t* C1 = kMode == 0 ? static_cast<const uint8_t*>(M1) + seg.id * (mat / 2) : C0;
    const uint16_t* S0 = static_cast<const uint16_t*>(Q0) + seg.id * (mat / 32);
    const uint16_t* S1 =
        kMode == 0 ? static_cast<const uint16_t*>(Q1) + seg.id * (mat / 32) : S0;
    switch (T) {
      case 1: mfma_tile_q4<1, kMode>(a, seg, t0, r0, K, C0, C1, S0, S1); break;
      case 2: mfma_tile_q4<2, kMode>(a, seg, t0, r0, K, C0, C1, S0, S1); break;
      case 3: mfma_tile_q4<3, kMode>(a, seg, t0, r0, K, C0, C1, S0, S1); break;
      default: mfma_tile_q4<4, kMode>(a, seg, t0, r0, K, C0, C1, S0, S1); break;
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
  hipLaunchKernelGGL(ffn_q4_kernel<0>, dim3(n_blocks(a, 0, 64)), dim3(256), 0, s, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(ffn_q4_kernel<1>, dim3(n_blocks(a, 1, 64)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
