// bf16 expert FFN on the matrix cores.
//
// Unit of work: R consecutive 16-row tiles of one expert matrix pair (gate
// and up) or one down matrix, for all tokens routed to that expert.  The W
// waves of the workgroup split the reduction dimension K into W contiguous
// ranges; each wave streams its range with a double-buffered register
// pipeline (the next chunk of steps is in flight while the current one
// feeds the MFMAs), and the W partial tiles are added through LDS in wave
// order, so results do not depend on timing.
//
// Per 32-wide K step a lane loads 16 bytes of each of its R weight rows (the
// A operand of v_mfma_f32_16x16x32_bf16: row = lane % 16, K slice =
// lane / 16) and 16 bytes of each token tile (B operand, from the
// L2-resident activations); the R row tiles share the token fragments.
#include "small_layer.h"

namespace s2moe {

using namespace ffn;

namespace {

template <int T, int R, int NM, int U>
struct Stage {
  u32x4 a[NM][R][U];
  u32x4 b[T][U];
};

// Weights of step s: plain layout -> 16 bytes at u32x4 index 4 s of the
// lane's row pointer; packed layout -> 1 KB tile s (u32x4 index 64 s), read
// with a nontemporal hint since each weight byte is used once per call.
template <bool kPacked>
__device__ __forceinline__ u32x4 load_weights(const u32x4* p, int s) {
  if (kPacked) return __builtin_nontemporal_load(p + 64 * s);
  return p[4 * s];
}

template <bool kPacked, int T, int R, int NM, int U>
__device__ __forceinline__ void load_stage(Stage<T, R, NM, U>& st, const u32x4* const* pa,
                                           const u32x4* const* xb, int s0, int hi) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int s = min(s0 + u, hi - 1);  // steps past the range reload a valid one
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < R; ++r) st.a[m][r][u] = load_weights<kPacked>(pa[m * R + r], s);
  }
#pragma unroll
  for (int tt = 0; tt < T; ++tt)
#pragma unroll
    for (int u = 0; u < U; ++u) st.b[tt][u] = xb[tt][4 * min(s0 + u, hi - 1)];
}

template <int T, int R, int NM, int U>
__device__ __forceinline__ void compute_stage(const Stage<T, R, NM, U>& st,
                                              f32x4 (&acc)[NM][R][T], int s0, int hi) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (s0 + u < hi) {
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int tt = 0; tt < T; ++tt)
            acc[m][r][tt] =
                mfma(as_bf16x8(st.a[m][r][u]), as_bf16x8(st.b[tt][u]), acc[m][r][tt]);
    }
  }
}

// One pass over up to 16*T tokens of the unit, all of the wave's K range.
template <int kMode, int T, int TMAX, int R, int W, int U, bool kPacked>
__device__ __forceinline__ void unit_pass(const FfnArgs& a, const Segment& seg, int t0, int r0,
                                          int K, const uint16_t* W0, const uint16_t* W1,
                                          f32x4* red) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
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
  const u32x4* pa[NM * R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (kPacked) {
      const size_t tile0 = (size_t)(r0 / 16 + r) * nks;  // first tile of the row tile
      pa[r] = reinterpret_cast<const u32x4*>(W0) + tile0 * 64 + lane;
      if (NM > 1) pa[R + r] = reinterpret_cast<const u32x4*>(W1) + tile0 * 64 + lane;
    } else {
      pa[r] = reinterpret_cast<const u32x4*>(W0 + (size_t)(r0 + 16 * r + rA) * K) + gK;
      if (NM > 1)
        pa[R + r] = reinterpret_cast<const u32x4*>(W1 + (size_t)(r0 + 16 * r + rA) * K) + gK;
    }
  }

  f32x4 acc[NM][R][T];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int tt = 0; tt < T; ++tt) acc[m][r][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (hi > lo) {
    pipeline2<Stage<T, R, NM, U>>(
        (hi - lo + U - 1) / U,
        [&](Stage<T, R, NM, U>& st, int c) { load_stage<kPacked>(st, pa, xb, lo + c * U, hi); },
        [&](const Stage<T, R, NM, U>& st, int c) { compute_stage(st, acc, lo + c * U, hi); });
  }

  if (W > 1) {
    // Partial tiles of all waves -> LDS, summed by wave 0 in wave order.
    constexpr int kTiles = NM * R * TMAX;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int tt = 0; tt < T; ++tt)
          red[(wave * kTiles + (m * R + r) * TMAX + tt) * kWave + lane] = acc[m][r][tt];
    __syncthreads();
    if (wave == 0) {
      for (int w = 1; w < W; ++w) {
#pragma unroll
        for (int m = 0; m < NM; ++m)
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int tt = 0; tt < T; ++tt) {
              const f32x4 p = red[(w * kTiles + (m * R + r) * TMAX + tt) * kWave + lane];
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[m][r][tt][i] += p[i];
            }
      }
    }
  }
  if (wave == 0) {
    // Lane holds D[m][n] for token n = rA and rows 4 gK + i of each tile.
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
      const int t = t0 + tt * 16 + rA;
      if (t >= seg.n) continue;
      if (kMode == 0) {
        uint16_t* dst = static_cast<uint16_t*>(a.hh) + (size_t)(seg.base + t) * a.ldh;
#pragma unroll
        for (int r = 0; r < R; ++r) {
          uint32_t h[4];
#pragma unroll
          for (int i = 0; i < 4; ++i)
            h[i] = f32_to_bf16(silu(acc[0][r][tt][i]) * acc[NM - 1][r][tt][i]);
          uint2 v;
          v.x = h[0] | (h[1] << 16);
          v.y = h[2] | (h[3] << 16);
          *reinterpret_cast<uint2*>(dst + r0 + 16 * r + 4 * gK) = v;
        }
      } else {
        float* dst = a.out + (size_t)out_row(a, seg, t) * a.H;
#pragma unroll
        for (int r = 0; r < R; ++r)
          *reinterpret_cast<f32x4*>(dst + r0 + 16 * r + 4 * gK) = acc[0][r][tt];
      }
    }
  }
  if (W > 1) __syncthreads();  // LDS is reused by the next pass
}

// The workgroup's unit: resolve it from the buckets (count, offset, slot,
// uniq, n_uniq: global, or LDS in the fused small-batch kernel) and run its
// passes over the tokens.  red: W > 1 ? W NM R TMAX x 64 f32x4 of LDS.
template <int kMode, int TMAX, int R, int W, int U, bool kPacked>
__device__ __forceinline__ void ffn_bf16_unit(const FfnArgs& a, f32x4* red) {
  Segment seg;
  int unit;
  if (!resolve_block(a, kMode, 16 * R, &seg, &unit)) return;
  const int r0 = unit * 16 * R;
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
    if (TMAX >= 4 && T >= 4)
      unit_pass<kMode, (TMAX >= 4 ? 4 : 1), TMAX, R, W, U, kPacked>(a, seg, t0, r0, K, W0, W1, red);
    else if (TMAX >= 3 && T == 3)
      unit_pass<kMode, (TMAX >= 3 ? 3 : 1), TMAX, R, W, U, kPacked>(a, seg, t0, r0, K, W0, W1, red);
    else if (TMAX >= 2 && T == 2)
      unit_pass<kMode, (TMAX >= 2 ? 2 : 1), TMAX, R, W, U, kPacked>(a, seg, t0, r0, K, W0, W1, red);
    else
      unit_pass<kMode, 1, TMAX, R, W, U, kPacked>(a, seg, t0, r0, K, W0, W1, red);
  }
}

template <int kMode, int TMAX, int R, int W, int U, bool kPacked>
__global__ __launch_bounds__(W * 64) void ffn_bf16_kernel(FfnArgs a) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  __shared__ f32x4 red[W > 1 ? W * NM * R * TMAX * kWave : 1];
  ffn_bf16_unit<kMode, TMAX, R, W, U, kPacked>(a, red);
}

// ------------------------------------------------- fused small-batch layer
// A whole MoE layer of B <= kSmallMaxTokens tokens whose gating keeps the
// plain top-k runs as three launches: the router rows (route.hip), then the
// two kernels below.  Each computes exactly what the unfused kernels
// compute, so the results are the same bit for bit.

// Gate-up with the routing in its prologue (small_layer_routing): one extra
// workgroup, the last, publishes the routing and exits; the unit work of the
// others is ffn_bf16_kernel<0, ...>'s, resolved from the LDS buckets.
template <int NJ, int TMAX, int R, int W, int U, bool kPacked>
__global__ __launch_bounds__(W * 64) void ffn_bf16_gate_up_routed_kernel(FfnArgs a,
                                                                        RouteArgs ra,
                                                                        GateArgs ga) {
  __shared__ SmallGateLds rt;
  __shared__ f32x4 red[W > 1 ? W * 2 * R * TMAX * kWave : 1];
  const bool pub = blockIdx.x == gridDim.x - 1;
  if (wave_id() == 0) small_layer_routing<NJ>(ra, ga, rt, pub);
  __syncthreads();
  if (pub) return;
  ffn_bf16_unit<0, TMAX, R, W, U, kPacked>(with_lds_buckets(a, rt), red);
}

// Down projection and combine in one launch.  A workgroup takes 16 R rows of
// H for every segment (small_down_segment); wave w works on segment w / KW
// over K part w % KW with the down kernel's K ranges, and small_down_finish
// adds the parts in the down kernel's order, writes expert_out and forms y.
template <int R, int KW, int U, bool kPacked>
__global__ __launch_bounds__(1024) void ffn_bf16_down_combine_kernel(FfnArgs a,
                                                                     const int32_t* idx,
                                                                     const float* gate_w,
                                                                     float* y) {
  __shared__ SmallDownLds<R> lds;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
  const int rA = lane & 15, gK = lane >> 4;
  const int seg_i = wave / KW, part = wave - seg_i * KW;
  const int r0 = blockIdx.x * 16 * R;
  Segment seg;
  uint64_t members;
  const bool live = small_down_segment<R>(a, idx, gate_w, seg_i, lds, &seg, &members);

  f32x4 acc[1][R][1];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[0][r][0] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (live) {
    const int K = seg.shared ? a.Fs : a.F;
    const int nks = K / 32;
    const int lo = part * nks / KW, hi = (part + 1) * nks / KW;
    const uint16_t* W0 = static_cast<const uint16_t*>(seg.shared ? a.sh_down : a.down) +
                         (size_t)seg.id * a.H * K;
    const u32x4* xb[1];
    xb[0] = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.hh) +
                                           (size_t)x_row(a, 1, seg, min(rA, seg.n - 1)) *
                                               a.ldh) +
            gK;
    const u32x4* pa[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (kPacked)
        pa[r] = reinterpret_cast<const u32x4*>(W0) + (size_t)(r0 / 16 + r) * nks * 64 + lane;
      else
        pa[r] = reinterpret_cast<const u32x4*>(W0 + (size_t)(r0 + 16 * r + rA) * K) + gK;
    }
    if (hi > lo) {
      pipeline2<Stage<1, R, 1, U>>(
          (hi - lo + U - 1) / U,
          [&](Stage<1, R, 1, U>& st, int c) { load_stage<kPacked>(st, pa, xb, lo + c * U, hi); },
          [&](const Stage<1, R, 1, U>& st, int c) { compute_stage(st, acc, lo + c * U, hi); });
    }
  }
  small_down_finish<R, KW>(a, seg, live, part, members, acc, lds, y, r0);
}

#ifndef S2MOE_MAX_WAVES
#define S2MOE_MAX_WAVES 8
#endif

#ifndef S2MOE_MAX_RED_TILES
#define S2MOE_MAX_RED_TILES 32
#endif

// Waves per unit: enough that each streams >= spw K steps, a power of two,
// and the reduction buffer stays within S2MOE_MAX_RED_TILES KB of LDS.
int pick_waves(int nks, int tiles, int spw) {
  int w = 1;
  while (w * 2 <= S2MOE_MAX_WAVES && nks / (w * 2) >= spw &&
         (w * 2) * tiles <= S2MOE_MAX_RED_TILES)
    w *= 2;
  return w;
}

template <int kMode, int TMAX, int R, int U, bool kPacked>
hipError_t launch_mode_p(const FfnArgs& a, int spw, hipStream_t s) {
  const int nm = kMode == 0 ? 2 : 1;
  int nks = kMode == 0 ? a.H / 32 : a.F / 32;
  if (kMode == 1 && a.S > 0) nks = min(nks, a.Fs / 32);
  const int w = pick_waves(nks, nm * R * TMAX, spw);
  const dim3 grid(n_blocks(a, kMode, 16 * R));
  switch (w) {
    case 1: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, R, 1, U, kPacked>), grid, dim3(64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, R, 2, U, kPacked>), grid, dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, R, 4, U, kPacked>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((ffn_bf16_kernel<kMode, TMAX, R, 8, U, kPacked>), grid, dim3(512), 0, s, a); break;
  }
  return hipGetLastError();
}

template <int kMode, int TMAX, int R, int U>
hipError_t launch_mode(const FfnArgs& a, int spw, hipStream_t s) {
  return a.packed ? launch_mode_p<kMode, TMAX, R, U, true>(a, spw, s)
                  : launch_mode_p<kMode, TMAX, R, U, false>(a, spw, s);
}

// Token tiles held at once (TMAX) follow the batch size; larger buckets take
// several passes over the same weight rows.  Row tiles per wave (R) grow
// with TMAX so that activation reads from L2 stay below the weight stream.
// Each choice is (TMAX, R gate-up, steps per stage gate-up, R down, steps
// per stage down, minimum K steps per wave [, the same for down alone]).
// For 17-32 tokens the down projection (a short K: 24 steps at F = 768)
// splits K over 4 waves of 6 steps: measured on MI355X at 32 tokens over
// 128 experts, its launch then takes 2 us less than with one wave (8 waves:
// 15 us more).
#ifndef S2MOE_BF16_TINY
#define S2MOE_BF16_TINY 1, 1, 2, 1, 4, 16
#endif
#ifndef S2MOE_BF16_SMALL
#define S2MOE_BF16_SMALL 1, 1, 2, 1, 4, 16
#endif
#ifndef S2MOE_BF16_MEDIUM
#define S2MOE_BF16_MEDIUM 2, 2, 2, 2, 2, 32, 4
#endif
#ifndef S2MOE_BF16_LARGE
#define S2MOE_BF16_LARGE 4, 2, 1, 4, 1, 16
#endif

template <int TMAX, int RG, int UG, int RD, int UD, int SPW, int SPWD = SPW>
hipError_t launch_bf16_pair(const FfnArgs& a, hipStream_t s) {
  hipError_t err = launch_mode<0, TMAX, RG, UG>(a, SPW, s);
  return err != hipSuccess ? err : launch_mode<1, TMAX, RD, UD>(a, SPWD, s);
}

// The fused small-batch layer with the tiny-batch configuration above: the
// gate-up and down launches take the waves, rows and stages the unfused
// launches take, so the arithmetic is the same.
constexpr int kFusedMaxWaves = 16;

template <int TMAX, int RG, int UG, int RD, int UD, int SPW, int SPWD = SPW>
struct SmallLayer {
  static_assert(TMAX == 1, "one token tile");
  static int down_waves(const FfnArgs& a) {
    int nks = a.F / 32;
    if (a.S > 0) nks = min(nks, a.Fs / 32);
    return pick_waves(nks, RD * TMAX, SPWD);
  }
  static bool fits(const FfnArgs& a) {
    return (a.S + min(a.E, a.B * a.k)) * down_waves(a) <= kFusedMaxWaves;
  }

  template <int NJ, bool kPacked>
  static hipError_t gate_up(const FfnArgs& a, const RouteArgs& ra, const GateArgs& ga,
                            hipStream_t s) {
    const int w = pick_waves(a.H / 32, 2 * RG * TMAX, SPW);
    const dim3 grid(n_blocks(a, 0, 16 * RG) + 1);
    switch (w) {
      case 1: hipLaunchKernelGGL((ffn_bf16_gate_up_routed_kernel<NJ, TMAX, RG, 1, UG, kPacked>), grid, dim3(64), 0, s, a, ra, ga); break;
      case 2: hipLaunchKernelGGL((ffn_bf16_gate_up_routed_kernel<NJ, TMAX, RG, 2, UG, kPacked>), grid, dim3(128), 0, s, a, ra, ga); break;
      case 4: hipLaunchKernelGGL((ffn_bf16_gate_up_routed_kernel<NJ, TMAX, RG, 4, UG, kPacked>), grid, dim3(256), 0, s, a, ra, ga); break;
      default: hipLaunchKernelGGL((ffn_bf16_gate_up_routed_kernel<NJ, TMAX, RG, 8, UG, kPacked>), grid, dim3(512), 0, s, a, ra, ga); break;
    }
    return hipGetLastError();
  }

  template <bool kPacked>
  static hipError_t down(const FfnArgs& a, const int32_t* idx, const float* gate_w, float* y,
                         hipStream_t s) {
    const int kw = down_waves(a);
    const dim3 grid(a.H / (16 * RD));
    const dim3 block(64 * kw * (a.S + min(a.E, a.B * a.k)));
    switch (kw) {
      case 1: hipLaunchKernelGGL((ffn_bf16_down_combine_kernel<RD, 1, UD, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
      case 2: hipLaunchKernelGGL((ffn_bf16_down_combine_kernel<RD, 2, UD, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
      case 4: hipLaunchKernelGGL((ffn_bf16_down_combine_kernel<RD, 4, UD, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
      default: hipLaunchKernelGGL((ffn_bf16_down_combine_kernel<RD, 8, UD, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
    }
    return hipGetLastError();
  }

  template <bool kPacked>
  static hipError_t layer(const RouteArgs& ra, const GateArgs& ga, const FfnArgs& a, float* y,
                          hipStream_t s) {
    hipError_t err = launch_route_rows(ra, s);
    if (err != hipSuccess) return err;
    if (a.E <= 64) err = gate_up<1, kPacked>(a, ra, ga, s);
    else if (a.E <= 128) err = gate_up<2, kPacked>(a, ra, ga, s);
    else err = gate_up<4, kPacked>(a, ra, ga, s);
    if (err != hipSuccess) return err;
    return down<kPacked>(a, ga.idx, ga.gate_w, y, s);
  }
};

using TinyLayer = SmallLayer<S2MOE_BF16_TINY>;

}  // namespace

bool moe_layer_small_fits_bf16(const FfnArgs& a) { return TinyLayer::fits(a); }

hipError_t launch_moe_layer_small_bf16(const RouteArgs& ra, const GateArgs& ga,
                                       const FfnArgs& a, float* y, hipStream_t s) {
  return a.packed ? TinyLayer::layer<true>(ra, ga, a, y, s)
                  : TinyLayer::layer<false>(ra, ga, a, y, s);
}

hipError_t launch_ffn_bf16(const FfnArgs& a, hipStream_t s) {
  if (a.B <= 4) return launch_bf16_pair<S2MOE_BF16_TINY>(a, s);
  if (a.B <= 16) return launch_bf16_pair<S2MOE_BF16_SMALL>(a, s);
  if (a.B <= 32) return launch_bf16_pair<S2MOE_BF16_MEDIUM>(a, s);
  return launch_bf16_pair<S2MOE_BF16_LARGE>(a, s);
}

}  // namespace s2moe
