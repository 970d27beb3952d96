// int4 expert FFN (4-bit codes, one fp16 scale per 32 K elements) on the
// matrix cores, decoding inside the weight stream.
//
// A lane reads one whole 32-code group (16 bytes) of its weight row per
// 128-wide "super-step" (lanes 16 apart take consecutive groups, so a row's
// 64 bytes arrive in one load) plus that group's scale.  Each code dword (8
// codes, nibble slots 0..7) becomes 4 fp16 pairs with one shift and four
// and-or operations: slots (0,4) and (2,6) land in the low mantissa bits of
// 0x6400 (the fp16 number 1024 + q), slots (1,5) and (3,7) four bits higher
// (1024 + 16 q).  Exact packed fp16 steps take them to q - 8 (a subtract of
// 1032, or a fused (h / 16) - 72), and a packed multiply by the group scale
// gives round_fp16(s * (q - 8)).  The four dwords are the A operands of four
// v_mfma_f32_16x16x32_f16, accumulated in fp32, so no dequantised weight is
// ever written to memory and no per-group epilogue is needed.  The decode
// yields the slot order (0,4,1,5,2,6,3,7) inside each 8-element block; the
// activations are kept in fp16 in that same order (a prep kernel converts x,
// the gate-up epilogue writes Hh so), with the 8-blocks of each super-step
// stored so that every B-operand load reads 64 contiguous bytes per token.
//
// Work decomposition as in the bf16 kernel: R 16-row tiles per unit, W waves
// split K, two-stage register pipeline, LDS reduction in wave order.  Above
// 8 tokens the gate-up launch instead uses a row-split kernel whose waves
// share LDS-staged activations (ffn_q4_rows_kernel).
#include <atomic>

#include "ffn_common.h"

namespace s2moe {

using namespace ffn;

namespace {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef _Float16 half8v __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4 mfma16(half8v a, half8v b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ half8v as_half8(u32x4 v) {
  half8v r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// Position of element e of an 8-element block in the decode order
// (0,4,1,5,2,6,3,7).
__device__ __forceinline__ int pos8(int e) { return ((e & 3) << 1) | (e >> 2); }

// Where 8-block c of a row of activations is stored: inside each 128-wide
// super-step (16 blocks, block 4 g + j = dword j of code group g) the blocks
// are stored j-major, so that the four lanes of one token that feed MFMA j
// read 64 contiguous bytes.
__host__ __device__ __forceinline__ int block_pos(int c) {
  return (c & ~15) | ((c & 3) << 2) | ((c >> 2) & 3);
}

// The value unchanged but held in a register the compiler cannot see through,
// so that "(w & mask) | magic" becomes one v_and_or_b32 (a VOP3 instruction
// takes at most one literal).
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

// 8 codes (one dword) -> s * (q - 8) as fp16, in decode order.
__device__ __forceinline__ half8v q4_decode(uint32_t w, half2v s2, uint32_t magic) {
  const half2v off = {(_Float16)-1032.0f, (_Float16)-1032.0f};
  const half2v sixteenth = {(_Float16)0.0625f, (_Float16)0.0625f};
  const half2v off16 = {(_Float16)-72.0f, (_Float16)-72.0f};
  const uint32_t w8 = w >> 8;
  const uint32_t d[4] = {(w & 0x000F000Fu) | magic, (w & 0x00F000F0u) | magic,
                         (w8 & 0x000F000Fu) | magic, (w8 & 0x00F000F0u) | magic};
  half8v r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    half2v h;
    __builtin_memcpy(&h, &d[i], 4);
    // 1024 + q - 1032, or (1024 + 16 q) / 16 - 72: both exactly q - 8
    h = (i & 1) ? __builtin_elementwise_fma(h, sixteenth, off16) : h + off;
    h = h * s2;
    r[2 * i] = h[0];
    r[2 * i + 1] = h[1];
  }
  return r;
}

template <int T, int R, int NM>
struct StageQ {
  u32x4 c[NM][R];     // one 32-code group per lane
  uint32_t s[NM][R];  // its fp16 scale (low half)
  u32x4 b[T][4];      // 4 x 8 activations per token tile
};

// Codes and scale of super-step s: plain layout -> u32x4 index 4 s and
// scale index 4 s of the lane's row pointers; packed layout -> 1 KB code
// tile s and 128-byte scale tile s (nontemporal: read once per call).
template <bool kPacked, int T, int R, int NM>
__device__ __forceinline__ void load_q(StageQ<T, R, NM>& st, const u32x4* const* pc,
                                       const uint16_t* const* ps, const u32x4* const* xb,
                                       int s) {
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (kPacked) {
        st.c[m][r] = __builtin_nontemporal_load(pc[m * R + r] + 64 * s);
        st.s[m][r] = __builtin_nontemporal_load(ps[m * R + r] + 64 * s);
      } else {
        st.c[m][r] = pc[m * R + r][4 * s];
        st.s[m][r] = ps[m * R + r][4 * s];
      }
    }
#pragma unroll
  for (int tt = 0; tt < T; ++tt)
#pragma unroll
    for (int j = 0; j < 4; ++j) st.b[tt][j] = xb[tt][16 * s + 4 * j];
}

template <int T, int R, int NM>
__device__ __forceinline__ void compute_q(const StageQ<T, R, NM>& st, f32x4 (&acc)[NM][R][T],
                                          uint32_t magic) {
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      _Float16 sh;
      const uint16_t bits = (uint16_t)st.s[m][r];
      __builtin_memcpy(&sh, &bits, 2);
      const half2v s2 = {sh, sh};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const half8v a = q4_decode(st.c[m][r][j], s2, magic);
#pragma unroll
        for (int tt = 0; tt < T; ++tt)
          acc[m][r][tt] = mfma16(a, as_half8(st.b[tt][j]), acc[m][r][tt]);
      }
    }
}

template <int kMode, int T, int TMAX, int R, int W, bool kPacked>
__device__ __forceinline__ void unit_pass_q(const FfnArgs& a, const Segment& seg, int t0, int r0,
                                            int K, const uint8_t* C0, const uint8_t* C1,
                                            const uint16_t* S0, const uint16_t* S1, f32x4* red) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
  const int rA = lane & 15, gK = lane >> 4;
  const int nss = K / 128;
  const int lo = wave * nss / W, hi = (wave + 1) * nss / W;

  // fp16 activations in decode order: x16 for gate-up, Hh for down.
  const uint16_t* X = static_cast<const uint16_t*>(kMode == 0 ? a.x16 : a.hh);
  const int ldx = kMode == 0 ? a.H : a.ldh;
  const u32x4* xb[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int t = min(t0 + tt * 16 + rA, seg.n - 1);
    xb[tt] = reinterpret_cast<const u32x4*>(X + (size_t)x_row(a, kMode, seg, t) * ldx) + gK;
  }
  const u32x4* pc[NM * R];
  const uint16_t* ps[NM * R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (kPacked) {
      const size_t tile0 = (size_t)(r0 / 16 + r) * nss;  // first tile of the row tile
      pc[r] = reinterpret_cast<const u32x4*>(C0) + tile0 * 64 + lane;
      ps[r] = S0 + tile0 * 64 + lane;
      if (NM > 1) {
        pc[R + r] = reinterpret_cast<const u32x4*>(C1) + tile0 * 64 + lane;
        ps[R + r] = S1 + tile0 * 64 + lane;
      }
    } else {
      const size_t row = (size_t)(r0 + 16 * r + rA);
      pc[r] = reinterpret_cast<const u32x4*>(C0 + row * (K / 2)) + gK;
      ps[r] = S0 + row * (K / 32) + gK;
      if (NM > 1) {
        pc[R + r] = reinterpret_cast<const u32x4*>(C1 + row * (K / 2)) + gK;
        ps[R + r] = S1 + row * (K / 32) + gK;
      }
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
    const uint32_t magic = opaque(0x64006400u);
    pipeline2<StageQ<T, R, NM>>(
        hi - lo,
        [&](StageQ<T, R, NM>& st, int i) { load_q<kPacked>(st, pc, ps, xb, lo + i); },
        [&](const StageQ<T, R, NM>& st, int) { compute_q(st, acc, magic); });
  }

  if (W > 1) {
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
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
      const int t = t0 + tt * 16 + rA;
      if (t >= seg.n) continue;
      if (kMode == 0) {
        _Float16* dst = static_cast<_Float16*>(a.hh) + (size_t)(seg.base + t) * a.ldh;
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int f = r0 + 16 * r + 4 * gK + i;
            dst[(block_pos(f >> 3) << 3) | pos8(f & 7)] =
                (_Float16)(silu(acc[0][r][tt][i]) * acc[NM - 1][r][tt][i]);
          }
      } else {
        float* dst = a.out + (size_t)out_row(a, seg, t) * a.H;
#pragma unroll
        for (int r = 0; r < R; ++r)
          *reinterpret_cast<f32x4*>(dst + r0 + 16 * r + 4 * gK) = acc[0][r][tt];
      }
    }
  }
  if (W > 1) __syncthreads();
}

template <int kMode, int TMAX, int R, int W, bool kPacked>
__global__ __launch_bounds__(W * 64) void ffn_q4_kernel(FfnArgs a) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  __shared__ f32x4 red[W > 1 ? W * NM * R * TMAX * kWave : 1];
  Segment seg;
  int unit;
  if (!resolve_block(a, kMode, 16 * R, &seg, &unit)) return;
  const int r0 = unit * 16 * R;
  const int rows = kMode == 0 ? (seg.shared ? a.Fs : a.F) : a.H;
  const int K = kMode == 0 ? a.H : (seg.shared ? a.Fs : a.F);
  const size_t mat = (size_t)rows * K;
  const void *M0, *M1, *Q0, *Q1;
  if (kMode == 0) {
    M0 = seg.shared ? a.sh_gate : a.gate;
    M1 = seg.shared ? a.sh_up : a.up;
    Q0 = seg.shared ? a.sh_gate_s : a.gate_s;
    Q1 = seg.shared ? a.sh_up_s : a.up_s;
  } else {
    M0 = M1 = seg.shared ? a.sh_down : a.down;
    Q0 = Q1 = seg.shared ? a.sh_down_s : a.down_s;
  }
  const uint8_t* C0 = static_cast<const uint8_t*>(M0) + seg.id * (mat / 2);
  const uint8_t* C1 = static_cast<const uint8_t*>(M1) + seg.id * (mat / 2);
  const uint16_t* S0 = static_cast<const uint16_t*>(Q0) + seg.id * (mat / 32);
  const uint16_t* S1 = static_cast<const uint16_t*>(Q1) + seg.id * (mat / 32);
  for (int t0 = 0; t0 < seg.n; t0 += 16 * TMAX) {
    const int T = min(TMAX, (seg.n - t0 + 15) / 16);
    if (TMAX >= 4 && T >= 4)
      unit_pass_q<kMode, (TMAX >= 4 ? 4 : 1), TMAX, R, W, kPacked>(a, seg, t0, r0, K, C0, C1, S0, S1, red);
    else if (TMAX >= 3 && T == 3)
      unit_pass_q<kMode, (TMAX >= 3 ? 3 : 1), TMAX, R, W, kPacked>(a, seg, t0, r0, K, C0, C1, S0, S1, red);
    else if (TMAX >= 2 && T == 2)
      unit_pass_q<kMode, (TMAX >= 2 ? 2 : 1), TMAX, R, W, kPacked>(a, seg, t0, r0, K, C0, C1, S0, S1, red);
    else
      unit_pass_q<kMode, 1, TMAX, R, W, kPacked>(a, seg, t0, r0, K, C0, C1, S0, S1, red);
  }
}

// Row-split variant (one or two token tiles per pass): the W waves of a
// workgroup take different row tiles over all of K, and share the
// activations, which the workgroup stages in LDS two super-steps at a time
// (double-buffered, one barrier per two super-steps).  The B operands then
// come from LDS instead of one global load per wave, which at two token
// tiles would move twice the weight bytes through the texture units.
constexpr int kChunkU4 = 32;       // u32x4 of one token row per chunk (2 super-steps)
constexpr int kLdsRowU4 = kChunkU4 + 1;  // padded: the 16 rows of a tile hit distinct banks

template <int R, int NM>
struct CodesQ {
  u32x4 c[NM][R];
  uint32_t s[NM][R];
};

template <bool kPacked, int R, int NM>
__device__ __forceinline__ void load_codes(CodesQ<R, NM>& st, const u32x4* const* pc,
                                           const uint16_t* const* ps, int s) {
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (kPacked) {
        st.c[m][r] = __builtin_nontemporal_load(pc[m * R + r] + 64 * s);
        st.s[m][r] = __builtin_nontemporal_load(ps[m * R + r] + 64 * s);
      } else {
        st.c[m][r] = pc[m * R + r][4 * s];
        st.s[m][r] = ps[m * R + r][4 * s];
      }
    }
}

// One super-step: codes from registers, B operands from LDS half h of the
// staged chunk.
template <int T, int R, int NM>
__device__ __forceinline__ void compute_rows(const CodesQ<R, NM>& st, const u32x4* buf, int h,
                                             f32x4 (&acc)[NM][R][T], uint32_t magic) {
  const int lane = threadIdx.x & (kWave - 1);
  const int rA = lane & 15, gK = lane >> 4;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    half8v b[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) b[tt] = as_half8(buf[(tt * 16 + rA) * kLdsRowU4 + 16 * h + 4 * j + gK]);
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < R; ++r) {
        _Float16 sh;
        const uint16_t bits = (uint16_t)st.s[m][r];
        __builtin_memcpy(&sh, &bits, 2);
        const half2v s2 = {sh, sh};
        const half8v a = q4_decode(st.c[m][r][j], s2, magic);
#pragma unroll
        for (int tt = 0; tt < T; ++tt) acc[m][r][tt] = mfma16(a, b[tt], acc[m][r][tt]);
      }
  }
}

template <int kMode, int T, int R, int W, bool kPacked>
__device__ __forceinline__ void rows_pass_q(const FfnArgs& a, const Segment& seg, int t0, int r0,
                                            int K, const uint8_t* C0, const uint8_t* C1,
                                            const uint16_t* S0, const uint16_t* S1, u32x4* lds) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  constexpr int kBuf = T * 16 * kLdsRowU4;       // u32x4 per LDS buffer
  constexpr int kStg = T * 16 * kChunkU4 / (W * kWave);  // staged u32x4 per thread
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = wave_id();
  const int rA = lane & 15, gK = lane >> 4;
  const int nss = K / 128, nch = (nss + 1) / 2;
  const int rw = r0 + wave * 16 * R;  // the wave's first row

  // Staging map: thread item q covers token row tok, 16-byte block blk of the
  // chunk (16 blocks per super-step).
  const uint16_t* X = static_cast<const uint16_t*>(kMode == 0 ? a.x16 : a.hh);
  const int ldx = kMode == 0 ? a.H : a.ldh;
  const u32x4* xs[kStg];
  int ld_off[kStg], blk_h[kStg], blk_l[kStg];
#pragma unroll
  for (int q = 0; q < kStg; ++q) {
    const int idx = tid + q * W * kWave;
    const int tok = idx / kChunkU4, blk = idx % kChunkU4;
    const int t = min(t0 + tok, seg.n - 1);
    xs[q] = reinterpret_cast<const u32x4*>(X + (size_t)x_row(a, kMode, seg, t) * ldx);
    ld_off[q] = tok * kLdsRowU4 + blk;
    blk_h[q] = blk >> 4;
    blk_l[q] = blk & 15;
  }
  // Chunk c holds super-steps 2c and 2c + 1 (the latter clamped to the last).
  auto load_stage = [&](u32x4 (&v)[kStg], int c) {
#pragma unroll
    for (int q = 0; q < kStg; ++q) v[q] = xs[q][16 * min(2 * c + blk_h[q], nss - 1) + blk_l[q]];
  };
  auto store_stage = [&](const u32x4 (&v)[kStg], u32x4* buf) {
#pragma unroll
    for (int q = 0; q < kStg; ++q) buf[ld_off[q]] = v[q];
  };

  const u32x4* pc[NM * R];
  const uint16_t* ps[NM * R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (kPacked) {
      const size_t tile0 = (size_t)(rw / 16 + r) * nss;
      pc[r] = reinterpret_cast<const u32x4*>(C0) + tile0 * 64 + lane;
      ps[r] = S0 + tile0 * 64 + lane;
      if (NM > 1) {
        pc[R + r] = reinterpret_cast<const u32x4*>(C1) + tile0 * 64 + lane;
        ps[R + r] = S1 + tile0 * 64 + lane;
      }
    } else {
      const size_t row = (size_t)(rw + 16 * r + rA);
      pc[r] = reinterpret_cast<const u32x4*>(C0 + row * (K / 2)) + gK;
      ps[r] = S0 + row * (K / 32) + gK;
      if (NM > 1) {
        pc[R + r] = reinterpret_cast<const u32x4*>(C1 + row * (K / 2)) + gK;
        ps[R + r] = S1 + row * (K / 32) + gK;
      }
    }
  }

  f32x4 acc[NM][R][T];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int tt = 0; tt < T; ++tt) acc[m][r][tt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const uint32_t magic = opaque(0x64006400u);
  u32x4 stg[kStg];
  CodesQ<R, NM> cA, cB;
  load_stage(stg, 0);
  load_codes<kPacked>(cA, pc, ps, 0);
  store_stage(stg, lds);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    const u32x4* buf = lds + (c & 1) * kBuf;
    load_stage(stg, min(c + 1, nch - 1));
    load_codes<kPacked>(cB, pc, ps, min(2 * c + 1, nss - 1));
    pipe_barrier();
    compute_rows(cA, buf, 0, acc, magic);
    load_codes<kPacked>(cA, pc, ps, min(2 * c + 2, nss - 1));
    pipe_barrier();
    if (2 * c + 1 < nss) compute_rows(cB, buf, 1, acc, magic);
    // The other buffer was last read in chunk c - 1, before the barrier that
    // ended it.
    store_stage(stg, lds + ((c + 1) & 1) * kBuf);
    __syncthreads();
  }

#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int t = t0 + tt * 16 + rA;
    if (t >= seg.n) continue;
    if (kMode == 0) {
      _Float16* dst = static_cast<_Float16*>(a.hh) + (size_t)(seg.base + t) * a.ldh;
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int f = rw + 16 * r + 4 * gK + i;
          dst[(block_pos(f >> 3) << 3) | pos8(f & 7)] =
              (_Float16)(silu(acc[0][r][tt][i]) * acc[NM - 1][r][tt][i]);
        }
    } else {
      float* dst = a.out + (size_t)out_row(a, seg, t) * a.H;
#pragma unroll
      for (int r = 0; r < R; ++r)
        *reinterpret_cast<f32x4*>(dst + rw + 16 * r + 4 * gK) = acc[0][r][tt];
    }
  }
}

template <int kMode, int R, int W, bool kPacked>
__global__ __launch_bounds__(W * 64) void ffn_q4_rows_kernel(FfnArgs a) {
  // Row counts are multiples of 128, so a workgroup's rows must divide 128.
  static_assert(128 % (16 * R * W) == 0, "rows per workgroup must divide 128");
  constexpr int NM = kMode == 0 ? 2 : 1;
  __shared__ u32x4 lds[2 * 2 * 16 * kLdsRowU4];
  Segment seg;
  int unit;
  if (!resolve_block(a, kMode, 16 * R * W, &seg, &unit)) return;
  const int r0 = unit * 16 * R * W;
  const int rows = kMode == 0 ? (seg.shared ? a.Fs : a.F) : a.H;
  const int K = kMode == 0 ? a.H : (seg.shared ? a.Fs : a.F);
  const size_t mat = (size_t)rows * K;
  const void *M0, *M1, *Q0, *Q1;
  if (kMode == 0) {
    M0 = seg.shared ? a.sh_gate : a.gate;
    M1 = seg.shared ? a.sh_up : a.up;
    Q0 = seg.shared ? a.sh_gate_s : a.gate_s;
    Q1 = seg.shared ? a.sh_up_s : a.up_s;
  } else {
    M0 = M1 = seg.shared ? a.sh_down : a.down;
    Q0 = Q1 = seg.shared ? a.sh_down_s : a.down_s;
  }
  const uint8_t* C0 = static_cast<const uint8_t*>(M0) + seg.id * (mat / 2);
  const uint8_t* C1 = static_cast<const uint8_t*>(M1) + seg.id * (mat / 2);
  const uint16_t* S0 = static_cast<const uint16_t*>(Q0) + seg.id * (mat / 32);
  const uint16_t* S1 = static_cast<const uint16_t*>(Q1) + seg.id * (mat / 32);
  for (int t0 = 0; t0 < seg.n; t0 += 32) {
    if (seg.n - t0 > 16)
      rows_pass_q<kMode, 2, R, W, kPacked>(a, seg, t0, r0, K, C0, C1, S0, S1, lds);
    else
      rows_pass_q<kMode, 1, R, W, kPacked>(a, seg, t0, r0, K, C0, C1, S0, S1, lds);
  }
  (void)NM;
}

// x [B, H] bf16 -> x16 [B, H] fp16 in the kernels' order (block_pos, then
// decode order inside each block), one 8-block per thread (H % 128 == 0, so
// a row holds whole super-steps).
__global__ __launch_bounds__(256) void q4_prep_x_kernel(const uint16_t* __restrict__ x,
                                                        uint16_t* __restrict__ x16, int n8) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n8) return;
  const u32x4 v = reinterpret_cast<const u32x4*>(x)[i];
  _Float16 h[8], o[8];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    h[2 * q] = (_Float16)bf16_to_f32(v[q] & 0xFFFFu);
    h[2 * q + 1] = (_Float16)bf16_to_f32(v[q] >> 16);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) o[pos8(e)] = h[e];
  u32x4 r;
  __builtin_memcpy(&r, o, 16);
  reinterpret_cast<u32x4*>(x16)[block_pos(i)] = r;
}

#ifndef S2MOE_Q4_STEPS_PER_WAVE
#define S2MOE_Q4_STEPS_PER_WAVE 8
#endif

int pick_waves_q4(int nss, int tiles) {
  int w = 1;
  while (w * 2 <= 8 && nss / (w * 2) >= S2MOE_Q4_STEPS_PER_WAVE && (w * 2) * tiles <= 32)
    w *= 2;
  return w;
}

template <int kMode, int TMAX, int R, bool kPacked>
hipError_t launch_q4_mode_p(const FfnArgs& a, hipStream_t s) {
  const int nm = kMode == 0 ? 2 : 1;
  int nss = kMode == 0 ? a.H / 128 : a.F / 128;
  if (kMode == 1 && a.S > 0) nss = min(nss, a.Fs / 128);
  const int w = pick_waves_q4(nss, nm * R * TMAX);
  const dim3 grid(n_blocks(a, kMode, 16 * R));
  switch (w) {
    case 1: hipLaunchKernelGGL((ffn_q4_kernel<kMode, TMAX, R, 1, kPacked>), grid, dim3(64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((ffn_q4_kernel<kMode, TMAX, R, 2, kPacked>), grid, dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL((ffn_q4_kernel<kMode, TMAX, R, 4, kPacked>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((ffn_q4_kernel<kMode, TMAX, R, 8, kPacked>), grid, dim3(512), 0, s, a); break;
  }
  return hipGetLastError();
}

template <int kMode, int TMAX, int R>
hipError_t launch_q4_mode(const FfnArgs& a, hipStream_t s) {
  return a.packed ? launch_q4_mode_p<kMode, TMAX, R, true>(a, s)
                  : launch_q4_mode_p<kMode, TMAX, R, false>(a, s);
}

// Compute units of the current device, queried once per device.
hipError_t device_cus(int* cus) {
  static std::atomic<int> cache[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && (*cus = cache[dev].load(std::memory_order_relaxed)) > 0)
    return hipSuccess;
  e = hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64) cache[dev].store(*cus, std::memory_order_relaxed);
  return hipSuccess;
}

template <int kMode, int R, int W>
hipError_t launch_q4_rows(const FfnArgs& a, hipStream_t s) {
  const dim3 grid(n_blocks(a, kMode, 16 * R * W));
  if (a.packed)
    hipLaunchKernelGGL((ffn_q4_rows_kernel<kMode, R, W, true>), grid, dim3(W * 64), 0, s, a);
  else
    hipLaunchKernelGGL((ffn_q4_rows_kernel<kMode, R, W, false>), grid, dim3(W * 64), 0, s, a);
  return hipGetLastError();
}

// Tile choices per batch size.
// - Gate-up above 8 tokens runs on the row-split kernel with one row tile
//   per wave (64 rows per workgroup, activations shared through LDS, up to
//   two token tiles per pass).  One row tile per wave keeps it at four
//   waves per SIMD (two row tiles: two), and the finer work units leave a
//   smaller partly filled last round of workgroups.
// - Gate-up up to 8 tokens and down up to 16 tokens hold one token tile,
//   and the row tiles per wave are the most (gate-up 2, down 4) that still
//   give every compute unit a workgroup: with one or two activated experts
//   (a draft step, or B = 1) fewer rows per workgroup spread the weight
//   stream over the whole GPU.
// - Down above 16 tokens holds two token tiles with 4 row tiles per wave.
//   Buckets larger than 32 tokens take several passes over the same rows.
hipError_t launch_q4_tiles(const FfnArgs& a, hipStream_t s) {
  hipError_t err;
  int cus = 0;
  if (a.B > 8) {
    err = launch_q4_rows<0, 1, 4>(a, s);
  } else {
    err = device_cus(&cus);
    if (err != hipSuccess) return err;
    err = n_blocks(a, 0, 32) >= cus ? launch_q4_mode<0, 1, 2>(a, s) : launch_q4_mode<0, 1, 1>(a, s);
  }
  if (err != hipSuccess) return err;
  if (a.B > 16) return launch_q4_mode<1, 2, 4>(a, s);
  if (cus == 0 && (err = device_cus(&cus)) != hipSuccess) return err;
  if (n_blocks(a, 1, 64) >= cus) return launch_q4_mode<1, 1, 4>(a, s);
  if (n_blocks(a, 1, 32) >= cus) return launch_q4_mode<1, 1, 2>(a, s);
  return launch_q4_mode<1, 1, 1>(a, s);
}

}  // namespace

hipError_t launch_ffn_q4(const FfnArgs& a, hipStream_t s) {
  const int n8 = a.B * a.H / 8;
  hipLaunchKernelGGL(q4_prep_x_kernel, dim3((n8 + 255) / 256), dim3(256), 0, s,
                     static_cast<const uint16_t*>(a.x), static_cast<uint16_t*>(a.x16), n8);
  const hipError_t err = hipGetLastError();
  return err != hipSuccess ? err : launch_q4_tiles(a, s);
}

}  // namespace s2moe
