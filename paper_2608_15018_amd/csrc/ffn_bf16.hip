// bf16 expert FFN on the matrix cores, one 16-row weight tile per workgroup.
//
// Unit of work: 16 rows of one expert matrix pair (gate and up) or of one
// down matrix, for all tokens routed to that expert.  The W waves of the
// workgroup split the reduction dimension K into W contiguous ranges; each
// wave streams its range with a double-buffered register pipeline (chunk c+1
// is in flight while chunk c feeds the MFMAs), and the W partial tiles are
// added through LDS in wave order, so results do not depend on timing.
//
// Per 32-wide K step a lane loads 16 bytes of its weight row (the A operand
// of v_mfma_f32_16x16x32_bf16: row = lane % 16, K slice = lane / 16) and 16
// bytes of each token tile (B operand, from the L2-resident activations).
// Small units keep the tail short: the hardware dispatcher starts the next
// tile on any CU that frees up.
#include "ffn_common.h"

namespace s2moe {

using namespace ffn;

namespace {

template <int T, int NM, int U>
struct Stage {
  u32x4 a[NM][U];
  u32x4 b[T][U];
};

template <int T, int NM, int U>
__device__ __forceinline__ void load_stage(Stage<T, NM, U>& st, const u32x4* pa0,
                                           const u32x4* pa1, const u32x4* const* xb, int s0,
                                           int hi) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int s = min(s0 + u, hi - 1);  // steps past the range reload a valid one
    st.a[0][u] = pa0[4 * s];
    if (NM > 1) st.a[NM - 1][u] = pa1[4 * s];
  }
#pragma unroll
  for (int tt = 0; tt < T; ++tt)
#pragma unroll
    for (int u = 0; u < U; ++u) st.b[tt][u] = xb[tt][4 * min(s0 + u, hi - 1)];
}

template <int T, int NM, int U>
__device__ __forceinline__ void compute_stage(const Stage<T, NM, U>& st, f32x4* acc0,
                                              f32x4* acc1, int s0, int hi) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (s0 + u < hi) {
#pragma unroll
      for (int tt = 0; tt < T; ++tt) {
        acc0[tt] = mfma(as_bf16x8(st.a[0][u]), as_bf16x8(st.b[tt][u]), acc0[tt]);
        if (NM > 1) acc1[tt] = mfma(as_bf16x8(st.a[NM - 1][u]), as_bf16x8(st.b[tt][u]), acc1[tt]);
      }
    }
  }
}

// One pass over up to 16*T tokens of the unit, all of the wave's K range.
template <int kMode, int T, int TMAX, int W, int U>
__device__ __forceinline__ void unit_pass(const FfnArgs& a, const Segment& seg, int t0, int r0,
                                          int K, const uint16_t* W0, const uint16_t* W1,
                                          f32x4* red) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x >> 6;
  const int rA = lane & 15, gK = lane >> 4;
  const int nks = K / 32;
  const int lo = wave * nks / W, hi = (wave + 1) * nks / W;

  const uint16_t* X = static_cast<const uint16_t*>(kMode == 0 ? a.x : a.hh);
  const int ldx = kMode == 0 ? a.H : a.ldh;
  const u32x4* xb[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int t = min(t0 + tt * 16 + rA, seg.n - 1);
    xb[tt] = reinterpret_cast<const u32x4*>(X + (size_t)x_row(a, kMode, seg, t) * ldx) + gK;
  }
  const u32x4* pa0 = reinterpret_cast<const u32x4*>(W0 + (size_t)(r0 + rA) * K) + gK;
  const u32x4* pa1 = reinterpret_cast<const u32x4*>(W1 + (size_t)(r0 + rA) * K) + gK;

  f32x4 acc0[T], acc1[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    acc0[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc1[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  if (hi > lo) {
    const int nch = (hi - lo + U - 1) / U;
    Stage<T, NM, U> st0, st1;
    load_stage(st0, pa0, pa1, xb, lo, hi);
    for (int c = 0; c < nch; c += 2) {
      if (c + 1 < nch) load_stage(st1, pa0, pa1, xb, lo + (c + 1) * U, hi);
      compute_stage(st0, acc0, acc1, lo + c * U, hi);
      if (c + 1 >= nch) break;
      if (c + 2 < nch) load_stage(st0, pa0, pa1, xb, lo + (c + 2) * U, hi);
      compute_stage(st1, acc0, acc1, lo + (c + 1) * U, hi);
    }
  }

  if (W > 1) {
    // Partial tiles of all waves -> LDS, summed by wave 0 in wave order.
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
      red[((wave * TMAX + tt) * NM) * kWave + lane] = acc0[tt];
      if (NM > 1) red[((wave * TMAX + tt) * NM + 1) * kWave + lane] = acc1[tt];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int tt = 0; tt < T; ++tt) {
        for (int w = 1; w < W; ++w) {
          const f32x4 p0 = red[((w * TMAX + tt) * NM) * kWave + lane];
#pragma unroll
          for (int i = 0; i < 4; ++i) acc0[tt][i] += p0[i];
          if (NM > 1) {
            const f32x4 p1 = red[((w * TMAX + tt) * NM + 1) * kWave + lane];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc1[tt][i] += p1[i];
          }
        }
      }
    }
  }
  if (wave == 0) {
    // Lane holds D[m][n] for token n = rA and rows m = 4 gK + i.
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
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.hh) +
                                  (size_t)(seg.base + t) * a.ldh + m0) = v;
      } else {
        *reinterpret_cast<f32x4*>(a.out + (size_t)out_row(a, seg, t) * a.H + m0) = acc0[tt];
      }
    }
  }
  if (W > 1) __syncthreads();  // LDS is reused by the next pass
}

template <int kMode, int TMAX, int W, int U>
__global__ __launch_bounds__(W * 64) void ffn_bf16_kernel(FfnArgs a) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  __shared__ f32x4 red[W > 1 ? W * TMAX * NM * kWave : 1];
  Segment seg;
  int tile;
  if (!resolve_block(a, kMode, 16, &seg, &tile)) return;
  const int r0 = tile * 16;
  const int rows = kMode == 0 ? (seg.shared ? a.Fs : a.F) : a.H;
  const int K = kMode == 0 ? a.H : (seg.shared ? a.Fs : a.F);
  const size_t mat = (size_t)rows * K;
  const uint16_t* W0;
  const uint16_t* W1;
  if (kMode == 0) {
    W0 = static_cast<const uint16_t*>(seg.shared ? a.sh_gate : a.gate) + seg.id * mat;
    W1 = static_cast<const uint16_t*>(seg.shared ? a.sh_up : a.up) + seg.id * mat;
  } else {
    W0 = static_cast<const uint16_t*>(seg.shared ? a.sh_down : a.down) + seg.id * mat;
    W1 = W0;
  }
  for (int t0 = 0; t0 < seg.n; t0 += 16 * TMAX) {
    const int T = min(TMAX, (seg.n - t0 + 15) / 16);
    if (T >= 4 && TMAX >= 4)
      unit_pass<kMode, (TMAX >= 4 ? 4 : 1), TMAX, W, U>(a, seg, t0, r0, K, W0, W1, red);
    else if (T == 3 && TMAX >= 3)
      unit_pass<kMode, (TMAX >= 3 ? 3 : 1), TMAX, W, U>(a, seg, t0, r0, K, W0, W1, red);
    else if (T == 2 && TMAX >= 2)
      unit_pass<kMode, (TMAX >= 2 ? 2 : 1), TMAX, W, U>(a, seg, t0, r0, K, W0, W1, red);
    else
      unit_pass<kMode, 1, TMAX, W, U>(a, seg, t0, r0, K, W0, W1, red);
  }
}

#ifndef S2MOE_STEPS_PER_WAVE
#define S2MOE_STEPS_PER_WAVE 32
#endif
#ifndef S2MOE_MAX_WAVES
#define S2MOE_MAX_WAVES 8
#endif
#ifndef S2MOE_STAGE_STEPS
#define S2MOE_STAGE_STEPS 4
#endif

// Waves per tile: enough that each streams >= S2MOE_STEPS_PER_WAVE K steps,
// a power of two, and the reduction buffer stays within 32 KB of LDS.
int pick_waves(int nks, int tmax, int nm) {
  int w = 1;
  while (w * 2 <= S2MOE_MAX_WAVES && nks / (w * 2) >= S2MOE_STEPS_PER_WAVE &&
         (w * 2) * tmax * nm <= 32)
    w *= 2;
  return w;
}

template <int kMode, int TMAX>
hipError_t launch_mode(const FfnArgs& a, hipStream_t s) {
  constexpr int U = S2MOE_STAGE_STEPS;
  const int nm = kMode == 0 ? 2 : 1;
  int nks = kMode == 0 ? a.H / 32 : a.F / 32;
  if (kMode == 1 && a.S > 0) nks = min(nks, a.Fs / 32);
  const int w = pick_waves(nks, TMAX, nm);
  const dim3 grid(n_blocks(a, kMode, 16));
  switch (w) {
    case 1: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, 1, U>), grid, dim3(64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, 2, U>), grid, dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, 4, U>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, 8, U>), grid, dim3(512), 0, s, a); break;
  }
  return hipGetLastError();
}

template <int TMAX>
hipError_t launch_both(const FfnArgs& a, hipStream_t s) {
  hipError_t err = launch_mode<0, TMAX>(a, s);
  if (err != hipSuccess) return err;
  return launch_mode<1, TMAX>(a, s);
}

}  // namespace

hipError_t launch_ffn_bf16(const FfnArgs& a, hipStream_t s) {
  // Token tiles held at once: up to 4 (64 tokens); larger buckets take
  // several passes over the same weight rows.
  const int tmax = a.B <= 16 ? 1 : (a.B <= 32 ? 2 : 4);
  if (tmax == 1) return launch_both<1>(a, s);
  if (tmax == 2) return launch_both<2>(a, s);
  return launch_both<4>(a, s);
}

}  // namespace s2moe
