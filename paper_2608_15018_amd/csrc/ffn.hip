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
#include "common.h"
#include "kernels.h"

namespace s2moe {

namespace {

struct Segment {
  int n;      // tokens
  int base;   // routed: offset[e] (row of its first token in Hh); shared: B*k + s*B
  int id;     // expert e or shared expert s
  bool shared;
};

// Grid layout: shared-expert blocks first (always live), then routed blocks
// u-major (u = position in uniq), so blocks of inactive experts come last
// and exit at once.
__device__ __forceinline__ bool resolve_block(const FfnArgs& a, int mode, int rows_per_block,
                                              Segment* seg, int* rb) {
  const int rows_r = mode == 0 ? a.F : a.H;
  const int rows_s = mode == 0 ? a.Fs : a.H;
  const int nbs = a.S > 0 ? rows_s / rows_per_block : 0;
  const int nbr = rows_r / rows_per_block;
  int bid = blockIdx.x;
  if (bid < a.S * nbs) {
    seg->shared = true;
    seg->id = bid / nbs;
    *rb = bid % nbs;
    seg->n = a.B;
    seg->base = a.B * a.k + seg->id * a.B;
    return true;
  }
  bid -= a.S * nbs;
  const int u = bid / nbr;
  *rb = bid % nbr;
  if (u >= min(*a.n_uniq, a.E)) return false;
  // The routing arrays come from the gating step; values outside their
  // ranges (routing never computed) make the block idle instead of faulting.
  const int e = a.uniq[u];
  if (e < 0 || e >= a.E) return false;
  seg->shared = false;
  seg->id = e;
  seg->n = a.count[e];
  seg->base = a.offset[e];
  return seg->n > 0 && seg->base >= 0 && seg->base + seg->n <= a.B * a.k;
}

__device__ __forceinline__ int slot_at(const FfnArgs& a, int i) {
  const int v = a.slot[i];
  return min(max(v, 0), a.B * a.k - 1);
}

// Row of the X source feeding token t of the segment: x for gate-up
// (gathered through slot), the segment's own Hh rows for down.
__device__ __forceinline__ int x_row(const FfnArgs& a, int mode, const Segment& s, int t) {
  if (mode == 0) return s.shared ? t : slot_at(a, s.base + t) / a.k;
  return s.base + t;
}

// Row of expert_out written for token t (down only).
__device__ __forceinline__ int out_row(const FfnArgs& a, const Segment& s, int t) {
  return s.shared ? s.base + t : slot_at(a, s.base + t);
}

__device__ __forceinline__ float silu(float z) { return z / (1.f + expf(-z)); }

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

// ---------------------------------------------------------------- MFMA path
__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  bf16x8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// 8 codes of one dword -> the bf16 values 128 + q, in the element order
// (0, 4, 2, 6, 1, 5, 3, 7) of K offsets within the lane's 8.
__device__ __forceinline__ bf16x8 q4_expand(uint32_t w) {
  u32x4 d;
  d[0] = (w & 0x000F000Fu) | 0x43004300u;
  d[1] = ((w >> 8) & 0x000F000Fu) | 0x43004300u;
  d[2] = ((w >> 4) & 0x000F000Fu) | 0x43004300u;
  d[3] = ((w >> 12) & 0x000F000Fu) | 0x43004300u;
  return as_bf16x8(d);
}

// Natural-order activations (k0..k7) -> the element order of q4_expand.
__device__ __forceinline__ bf16x8 q4_permute_x(u32x4 x) {
  u32x4 d;
  d[0] = (x[0] & 0xFFFFu) | (x[2] << 16);          // k0, k4
  d[1] = (x[1] & 0xFFFFu) | (x[3] << 16);          // k2, k6
  d[2] = (x[0] >> 16) | (x[2] & 0xFFFF0000u);      // k1, k5
  d[3] = (x[1] >> 16) | (x[3] & 0xFFFF0000u);      // k3, k7
  return as_bf16x8(d);
}

template <int T, int kMode, int U>
__device__ __forceinline__ void mfma_tile_bf16(const FfnArgs& a, const Segment& seg, int t0,
                                               int r0, int K, const uint16_t* W0,
                                               const uint16_t* W1) {
  constexpr bool kDual = kMode == 0;
  const int lane = threadIdx.x & (kWave - 1);
  const int rA = lane & 15, gK = lane >> 4;
  const int nks = K / 32;
  const uint16_t* X = static_cast<const uint16_t*>(kMode == 0 ? a.x : a.hh);
  const int ldx = kMode == 0 ? a.H : a.ldh;
  const u32x4* xb[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int t = min(t0 + tt * 16 + rA, seg.n - 1);
    xb[tt] = reinterpret_cast<const u32x4*>(X + (size_t)x_row(a, kMode, seg, t) * ldx) + gK;
  }
  const u32x4* pa0 = reinterpret_cast<const u32x4*>(W0 + (size_t)(r0 + rA) * K) + gK;
  const u32x4* pa1 = kDual ? reinterpret_cast<const u32x4*>(W1 + (size_t)(r0 + rA) * K) + gK
                           : pa0;
  f32x4 acc0[T], acc1[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    acc0[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc1[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int ks = 0; ks < nks; ks += U) {
    u32x4 A0[U], A1[U], Bf[T][U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      A0[u] = pa0[4 * (ks + u)];
      if (kDual) A1[u] = pa1[4 * (ks + u)];
    }
#pragma unroll
    for (int tt = 0; tt < T; ++tt)
#pragma unroll
      for (int u = 0; u < U; ++u) Bf[tt][u] = xb[tt][4 * (ks + u)];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int tt = 0; tt < T; ++tt) {
        acc0[tt] = mfma(as_bf16x8(A0[u]), as_bf16x8(Bf[tt][u]), acc0[tt]);
        if (kDual) acc1[tt] = mfma(as_bf16x8(A1[u]), as_bf16x8(Bf[tt][u]), acc1[tt]);
      }
  }
  // Epilogue.  Lane holds D[m][n] for token n = rA, rows m = 4 gK + i.
  const int m0 = r0 + 4 * gK;
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

template <int kMode, bool kQ4>
__global__ __launch_bounds__(256) void ffn_mfma_kernel(FfnArgs a) {
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
    if (kQ4) {
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
    } else {
      const uint16_t* W0 = static_cast<const uint16_t*>(M0) + seg.id * mat;
      const uint16_t* W1 = kMode == 0 ? static_cast<const uint16_t*>(M1) + seg.id * mat : W0;
      const bool u8 = ((K / 32) % 8) == 0;
      switch (T * 2 + (u8 ? 1 : 0)) {
        case 2: mfma_tile_bf16<1, kMode, 2>(a, seg, t0, r0, K, W0, W1); break;
        case 3: mfma_tile_bf16<1, kMode, 8>(a, seg, t0, r0, K, W0, W1); break;
        case 4: mfma_tile_bf16<2, kMode, 2>(a, seg, t0, r0, K, W0, W1); break;
        case 5: mfma_tile_bf16<2, kMode, 8>(a, seg, t0, r0, K, W0, W1); break;
        case 6: mfma_tile_bf16<3, kMode, 2>(a, seg, t0, r0, K, W0, W1); break;
        case 7: mfma_tile_bf16<3, kMode, 8>(a, seg, t0, r0, K, W0, W1); break;
        case 8: mfma_tile_bf16<4, kMode, 2>(a, seg, t0, r0, K, W0, W1); break;
        default: mfma_tile_bf16<4, kMode, 8>(a, seg, t0, r0, K, W0, W1); break;
      }
    }
  }
}

int n_blocks(const FfnArgs& a, int mode, int rows_per_block) {
  const int rows_r = mode == 0 ? a.F : a.H;
  const int rows_s = mode == 0 ? a.Fs : a.H;
  return (a.S > 0 ? a.S * (rows_s / rows_per_block) : 0) + a.E * (rows_r / rows_per_block);
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
  if (a.wf == kWBf16) {
    hipLaunchKernelGGL((ffn_mfma_kernel<0, false>), dim3(n_blocks(a, 0, 64)), dim3(256), 0, s, a);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((ffn_mfma_kernel<1, false>), dim3(n_blocks(a, 1, 64)), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((ffn_mfma_kernel<0, true>), dim3(n_blocks(a, 0, 64)), dim3(256), 0, s, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((ffn_mfma_kernel<1, true>), dim3(n_blocks(a, 1, 64)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
