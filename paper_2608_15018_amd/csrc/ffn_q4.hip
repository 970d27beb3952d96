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
// ever written to memory.  The decode yields the slot order (0,4,1,5,2,6,3,7)
// inside each 8-element block; the activations are kept in fp16 in that same
// order (a prep kernel converts x, the gate-up epilogue writes Hh so), with
// the 8-blocks of each super-step stored so that one token's 16 bytes for
// MFMA j of the four K slots lie side by side.
//
// Work decomposition for batches of more than kQ4KsplitMaxTokens tokens (one
// persistent launch per projection; smaller batches run the K-split kernel
// further down):
// - A work item is 16 R W rows of one expert (W = 4 waves, R row tiles per
//   wave) over one of Q contiguous K parts, for all tokens routed to that
//   expert.  The launch has at most as many workgroups as fit on the GPU at
//   once, a multiple of the 8 XCDs, and deals the items (expert-major)
//   round-robin over all of them, so every XCD gets an equal share of every
//   expert.  Within an expert, the down items one XCD receives form one
//   contiguous run of its (part, row block) list (resolve_item), so that
//   XCD's L2 fetches the activations of at most two of the Q parts.  Buckets
//   of different sizes make items of different cost (a
//   pass over four token tiles costs about twice one over one tile), and a
//   share of each keeps the XCDs equally loaded.  Measured on MI355X, 24
//   int4 layers at 64 tokens, where some layers route 60 tokens to one
//   expert: contiguous per-XCD slices of the items, which keep an expert's
//   activations in one to three L2s, were 17 % slower per layer with equal
//   item counts and 6 % slower with equal estimated costs (items run in
//   discrete rounds of workgroups, so a cost-balanced cut still leaves some
//   XCDs a round longer); a work counter taken with an atomic add per item
//   was 20-35 % slower, the adds of all workgroups serialising on one
//   address, and claims on 8 counters past the first round of items 1-2 %
//   slower; equal runs of consecutive items, or one workgroup per item,
//   were 3-15 % slower.
// - The waves of a workgroup stream different rows over the same K range, so
//   they share the activations: the workgroup stages the tokens' next
//   super-step in LDS while the current one is decoded (double-buffered, one
//   barrier per super-step), and every B operand is an LDS read.  Reading
//   them with one global load per MFMA instead caps the stream at a fraction
//   of HBM bandwidth on MI355X (measured: 3.8 TB/s at one token tile, 1 TB/s
//   at four).
// - Each wave keeps D - 1 super-steps of codes in flight in a register ring
//   (D = 2: the decode, not the memory latency, bounds the stream; deeper
//   rings of 3, 4, 6 and 8 were 2-35 % slower on MI355X as their registers
//   cost occupancy).
// - Up to TMAX = 4 token tiles (64 tokens) share one pass over the weights;
//   larger buckets take further passes.
// - Gate-up items span all of K (Q = 1), so SwiGLU is applied in the
//   epilogue.  Down items split K into Q parts when few experts are active:
//   part 0 writes expert_out, parts 1..Q-1 write partial sums to the
//   workspace, and q4_reduce_kernel adds them in part order afterwards, so
//   the result does not depend on timing.
#include <atomic>
#include <type_traits>

#include "q4_layout.h"
#include "small_layer.h"

namespace s2moe {

using namespace ffn;

namespace {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef _Float16 half8v __attribute__((ext_vector_type(8)));

constexpr int kW = 4;     // waves per workgroup
constexpr int kXcds = 8;  // accelerator dies of an MI355X, each with its own L2

__device__ __forceinline__ f32x4 mfma16(half8v a, half8v b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ half8v as_half8(u32x4 v) {
  half8v r;
  __builtin_memcpy(&r, &v, 16);
  return r;
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

// Codes and scales of one super-step for the wave's NM x R row tiles.
template <int R, int NM>
struct CodesQ {
  u32x4 c[NM][R];     // one 32-code group per lane
  uint32_t s[NM][R];  // its fp16 scale (low half)
};

// Codes and scale of super-step s: plain layout -> u32x4 index 4 s and
// scale index 4 s of the lane's row pointers; packed layout -> 1 KB code
// tile s and 128-byte scale tile s (nontemporal: read once per call).
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

// One super-step: codes from registers, B operands from LDS (token rows of
// kRow u32x4, `buf` at this super-step's first block).
template <int T, int R, int NM, int kRow>
__device__ __forceinline__ void compute_step(const CodesQ<R, NM>& st, const u32x4* buf,
                                             f32x4 (&acc)[NM][R][T], uint32_t magic) {
  const int lane = threadIdx.x & (kWave - 1);
  const int rA = lane & 15, gK = lane >> 4;
  half2v s2[NM][R];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      _Float16 sh;
      const uint16_t bits = (uint16_t)st.s[m][r];
      __builtin_memcpy(&sh, &bits, 2);
      s2[m][r] = half2v{sh, sh};
    }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    half8v b[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) b[tt] = as_half8(buf[(tt * 16 + rA) * kRow + 4 * j + gK]);
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const half8v a = q4_decode(st.c[m][r][j], s2[m][r], magic);
#pragma unroll
        for (int tt = 0; tt < T; ++tt) acc[m][r][tt] = mfma16(a, b[tt], acc[m][r][tt]);
      }
  }
}

// ---------------------------------------------------------------------------
// K-split kernel for tiny batches (B <= kQ4KsplitMaxTokens, one token tile):
// a work unit is R 16-row tiles of one expert over all of K, the W waves of
// the workgroup split K into contiguous ranges, each loads its own B
// operands (the batch's few tokens), and the partial tiles are added through
// LDS in wave order.  Units of 16 R rows (R chosen so the grid still fills
// the GPU) give a draft step's two or three small experts enough workgroups;
// the row-split kernel below needs 64- or 128-row items.
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

// The workgroup's unit of the K-split kernel: resolve it from the buckets
// (global, or LDS in the fused small-batch gate-up) and run its passes.
// red: W > 1 ? W NM R TMAX x 64 f32x4 of LDS.
template <int kMode, int TMAX, int R, int W, bool kPacked>
__device__ __forceinline__ void ffn_q4_ksplit_unit(const FfnArgs& a, f32x4* red) {
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

template <int kMode, int TMAX, int R, int W, bool kPacked>
__global__ __launch_bounds__(W * 64) void ffn_q4_ksplit_kernel(FfnArgs a) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  __shared__ f32x4 red[W > 1 ? W * NM * R * TMAX * kWave : 1];
  ffn_q4_ksplit_unit<kMode, TMAX, R, W, kPacked>(a, red);
}

// Row-split variant (one or two token tiles per pass): the W waves of a
// workgroup take different row tiles over all of K, and share the
// activations, which the workgroup stages in LDS two super-steps at a time
// (double-buffered, one barrier per two super-steps).  The B operands then
// come from LDS instead of one global load per wave, which at two token

constexpr int gcd_c(int x, int y) { return y == 0 ? x : gcd_c(y, x % y); }
constexpr int lcm_c(int x, int y) { return x / gcd_c(x, y) * y; }

// One pass of a work item over T token tiles (tokens t0 .. t0 + 16 T - 1 of
// the segment) and super-steps [lo, hi) of K.  The activations move through
// LDS in chunks of C super-steps (one barrier per chunk); each thread keeps
// the activations of the next A chunks and each wave the codes of the next
// D - 1 super-steps in flight in registers.
template <int kMode, int T, int R, int D, int A, int C, bool kPacked>
__device__ __forceinline__ void q4_pass(const FfnArgs& a, const Segment& seg, int t0, int r0,
                                        int q, int lo, int hi, int K, const uint8_t* C0,
                                        const uint8_t* C1, const uint16_t* S0,
                                        const uint16_t* S1, u32x4* lds) {
  constexpr int NM = kMode == 0 ? 2 : 1;
  constexpr int kRow = 16 * C + 1;      // u32x4 per token row of a chunk (+ pad)
  constexpr int kBuf = T * 16 * kRow;   // u32x4 per LDS buffer
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = wave_id();
  const int rA = lane & 15, gK = lane >> 4;
  const int nss = K / 128;
  const int rw = r0 + wave * 16 * R;  // the wave's first row

  // Staging: thread tid moves 16-byte block tid % 16 of token row
  // tt * 16 + tid / 16 of each super-step (256 threads, one row block each).
  const uint16_t* X = static_cast<const uint16_t*>(kMode == 0 ? a.x16 : a.hh);
  const int ldx = kMode == 0 ? a.H : a.ldh;
  const u32x4* xs[T];
  int ldo[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    const int tok = tt * 16 + (tid >> 4);
    const int t = min(t0 + tok, seg.n - 1);
    xs[tt] = reinterpret_cast<const u32x4*>(X + (size_t)x_row(a, kMode, seg, t) * ldx) + (tid & 15);
    ldo[tt] = tok * kRow + (tid & 15);
  }

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
  // The vector-memory counter completes loads in issue order, so a wait for
  // one load also waits for every older one.  A chunk's activations are
  // requested before the codes of the same step: waiting at the end of
  // chunk c for the activations of chunk c + 1 then forces no codes that
  // are not already due (needs D - 2 <= A C).
  static_assert(D - 2 <= A * C, "activation ring too short for the code ring");
  constexpr int U = lcm_c(D, A * C);  // steps of one loop turn: both rings wrap
  CodesQ<R, NM> ring[D];
  u32x4 stg[A][C][T];
  // Prologue.  Indices past the range reload the last valid super-step, so
  // every load is unconditional and the compiler's wait counts stay exact.
#pragma unroll
  for (int g = 0; g < A; ++g)
#pragma unroll
    for (int cs = 0; cs < C; ++cs)
#pragma unroll
      for (int tt = 0; tt < T; ++tt) stg[g][cs][tt] = xs[tt][16 * min(lo + g * C + cs, hi - 1)];
#pragma unroll
  for (int d = 0; d < D - 1; ++d) load_codes<kPacked>(ring[d], pc, ps, min(lo + d, hi - 1));
#pragma unroll
  for (int cs = 0; cs < C; ++cs)
#pragma unroll
    for (int tt = 0; tt < T; ++tt) lds[ldo[tt] + 16 * cs] = stg[0][cs][tt];
  __syncthreads();
  for (int base = lo; base < hi; base += U) {
#pragma unroll
    for (int d = 0; d < U; ++d) {
      const int s = base + d;
      const int ch = (s - lo) / C;  // chunk of step s (d / C within the turn)
      if (d % C == 0) {
        // Request the activations of chunk ch + A into the slot chunk ch
        // held (staged into LDS at the end of chunk ch - 1).
#pragma unroll
        for (int cs = 0; cs < C; ++cs)
#pragma unroll
          for (int tt = 0; tt < T; ++tt)
            stg[(d / C) % A][cs][tt] = xs[tt][16 * min(s + A * C + cs, hi - 1)];
      }
      load_codes<kPacked>(ring[(d + D - 1) % D], pc, ps, min(s + D - 1, hi - 1));
      pipe_barrier();
      if (s < hi)
        compute_step<T, R, NM, kRow>(ring[d % D], lds + (ch & 1) * kBuf + 16 * (d % C), acc, magic);
      if (d % C == C - 1) {
        // The other buffer was last read in chunk ch - 1, before the barrier
        // that ended it.
#pragma unroll
        for (int cs = 0; cs < C; ++cs)
#pragma unroll
          for (int tt = 0; tt < T; ++tt)
            lds[((ch + 1) & 1) * kBuf + ldo[tt] + 16 * cs] = stg[(d / C + 1) % A][cs][tt];
        __syncthreads();
      }
    }
  }

  // Lane holds D[row][token] for token rA of each tile and rows 4 gK + i.
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
      const size_t rows_out = (size_t)a.B * a.k + (size_t)a.S * a.B;
      float* base_out = q == 0 ? a.out : a.part + (size_t)(q - 1) * rows_out * a.H;
      float* dst = base_out + (size_t)out_row(a, seg, t) * a.H;
#pragma unroll
      for (int r = 0; r < R; ++r)
        *reinterpret_cast<f32x4*>(dst + rw + 16 * r + 4 * gK) = acc[0][r][tt];
    }
  }
}

// Work item `item` of a launch whose items cover 16 R kW rows over one of Q K
// parts: shared experts first, then the activated routed experts in uniq
// order.  False once the items of the activated experts are exhausted.
__device__ __forceinline__ bool resolve_item(const FfnArgs& a, int mode, int rows_per_item,
                                             int Q, int n_act, int item, Segment* seg, int* rb,
                                             int* q) {
  const int rows_r = mode == 0 ? a.F : a.H;
  const int rows_s = mode == 0 ? a.Fs : a.H;
  const int per_s = a.S > 0 ? rows_s / rows_per_item * Q : 0;
  const int per_r = rows_r / rows_per_item * Q;
  int rem;
  if (item < a.S * per_s) {
    seg->shared = true;
    seg->id = item / per_s;
    rem = item % per_s;
    seg->n = a.B;
    seg->base = a.B * a.k + seg->id * a.B;
  } else {
    item -= a.S * per_s;
    const int u = item / per_r;
    if (u >= n_act) return false;
    rem = item % per_r;
    // The routing arrays come from the gating step; values outside their
    // ranges (routing never computed) make the item empty instead of
    // faulting.
    const int e = a.uniq[u];
    seg->shared = false;
    seg->id = e;
    if (e < 0 || e >= a.E) {
      seg->n = 0;
    } else {
      seg->n = a.count[e];
      seg->base = a.offset[e];
      if (seg->n < 0 || seg->base < 0 || seg->base + seg->n > a.B * a.k) seg->n = 0;
    }
  }
  // Items are dealt round-robin over the grid (a multiple of kXcds
  // workgroups), so positions p and p + kXcds of a segment's items run on
  // the same XCD.  With K parts, the positions p = x (mod kXcds) take the
  // x-th of kXcds contiguous chunks of the segment's items in (part, row
  // block) order: each XCD's L2 then holds the activations of at most two of
  // the segment's Q parts, for any Q <= kXcds.
  const int per = seg->shared ? per_s : per_r;
  const int nrb = per / Q;
  const int L = (Q > 1 && per % kXcds == 0) ? (rem % kXcds) * (per / kXcds) + rem / kXcds : rem;
  *q = L / nrb;
  *rb = L % nrb;
  return true;
}

#ifndef S2MOE_Q4_MINWAVES_T4
#define S2MOE_Q4_MINWAVES_T4 2
#endif

template <int kMode, int TMAX, int R, int D, int A, int C, bool kPacked>
__global__ __launch_bounds__(kW * 64, TMAX >= 4 ? S2MOE_Q4_MINWAVES_T4 : 1) void ffn_q4_kernel(FfnArgs a) {
  __shared__ u32x4 lds[2 * TMAX * 16 * (16 * C + 1)];
  constexpr int kRows = 16 * R * kW;
  const int Q = kMode == 0 ? 1 : a.qparts;
  const int n_act = min(*a.n_uniq, min(a.E, a.B * a.k));
  const int rows_r = kMode == 0 ? a.F : a.H;
  const int rows_s = kMode == 0 ? a.Fs : a.H;
  const int n_items = (a.S > 0 ? a.S * (rows_s / kRows) : 0) * Q + max(n_act, 0) * (rows_r / kRows) * Q;
  for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
    Segment seg;
    int rb, q;
    if (!resolve_item(a, kMode, kRows, Q, n_act, item, &seg, &rb, &q)) break;
    if (seg.n <= 0) continue;
    const int r0 = rb * kRows;
    const int rows = kMode == 0 ? (seg.shared ? a.Fs : a.F) : a.H;
    const int K = kMode == 0 ? a.H : (seg.shared ? a.Fs : a.F);
    const int nss = K / 128;
    const int lo = q * nss / Q, hi = (q + 1) * nss / Q;
    if (hi <= lo) continue;  // the host keeps Q <= K / 128, so never taken
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
        q4_pass<kMode, (TMAX >= 4 ? 4 : 1), R, D, A, C, kPacked>(a, seg, t0, r0, q, lo, hi, K, C0, C1, S0, S1, lds);
      else if (TMAX >= 3 && T == 3)
        q4_pass<kMode, (TMAX >= 3 ? 3 : 1), R, D, A, C, kPacked>(a, seg, t0, r0, q, lo, hi, K, C0, C1, S0, S1, lds);
      else if (TMAX >= 2 && T == 2)
        q4_pass<kMode, (TMAX >= 2 ? 2 : 1), R, D, A, C, kPacked>(a, seg, t0, r0, q, lo, hi, K, C0, C1, S0, S1, lds);
      else
        q4_pass<kMode, 1, R, D, A, C, kPacked>(a, seg, t0, r0, q, lo, hi, K, C0, C1, S0, S1, lds);
    }
  }
}

// Element quad i of expert_out plus the partial sums of K parts 1 .. Q - 1
// (part q at part[(q - 1) n4 + i]), added in part order.  The Q loads are all
// issued before the first addition, so a quad costs one memory round trip.
template <int Q>
__device__ __forceinline__ f32x4 q4_sum_parts(const f32x4* out, const f32x4* part, size_t n4,
                                              size_t i) {
  f32x4 p[Q];
  p[0] = out[i];
#pragma unroll
  for (int q = 1; q < Q; ++q) p[q] = part[(size_t)(q - 1) * n4 + i];
  f32x4 v = p[0];
#pragma unroll
  for (int q = 1; q < Q; ++q)
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] += p[q][c];
  return v;
}

// expert_out += the partial sums of K parts 1 .. Q - 1, added in part order.
template <int Q>
__global__ __launch_bounds__(256) void q4_reduce_kernel(float* __restrict__ out,
                                                        const float* __restrict__ part,
                                                        size_t n4) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  reinterpret_cast<f32x4*>(out)[i] = q4_sum_parts<Q>(reinterpret_cast<const f32x4*>(out),
                                                     reinterpret_cast<const f32x4*>(part), n4, i);
}

// The ordered reduce and the combine in one launch (the one-call layer): for
// token b and 4 columns, each of its output rows (the k routed rows b k + j,
// then the shared rows B k + s B + b) gets parts 1 .. Q - 1 added in part
// order and goes back to expert_out, as q4_reduce_kernel does; y is then
// formed from those rows with combine_kernel's arithmetic.
template <int Q>
__global__ __launch_bounds__(256) void q4_reduce_combine_kernel(FfnArgs a, CombineArgs c) {
  const int b = blockIdx.y;
  const int col = blockIdx.x * blockDim.x + threadIdx.x;
  if (col * 4 >= a.H) return;
  const int ldq = a.H / 4;
  const size_t n4 = ((size_t)a.B * a.k + (size_t)a.S * a.B) * ldq;
  f32x4* out = reinterpret_cast<f32x4*>(a.out);
  const f32x4* part = reinterpret_cast<const f32x4*>(a.part);
  auto reduce_row = [&](int r) {
    const size_t i = (size_t)r * ldq + col;
    const f32x4 v = q4_sum_parts<Q>(out, part, n4, i);
    out[i] = v;
    return v;
  };
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < a.k; ++j) {
    const float w = c.gate_w[b * a.k + j];
    const f32x4 v = reduce_row(b * a.k + j);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = fmaf(w, v[e], acc[e]);
  }
  for (int sh = 0; sh < a.S; ++sh) {
    const f32x4 v = reduce_row(a.B * a.k + sh * a.B + b);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] += v[e];
  }
  reinterpret_cast<f32x4*>(c.y)[(size_t)b * ldq + col] = acc;
}

// x [B, H] bf16 -> x16 [B, H] fp16 in the kernels' order (prep_x8).
__global__ __launch_bounds__(256) void q4_prep_x_kernel(const uint16_t* __restrict__ x,
                                                        uint16_t* __restrict__ x16, int n8) {
  prep_x8(x, x16, blockIdx.x * blockDim.x + threadIdx.x, n8);
}

// ------------------------------------------------- fused small-batch layer
// The int4 form of the three-launch small-batch layer (small_layer.h):
// router rows and the fp16 copy of x in one launch; the K-split gate-up with
// the routing in its prologue; the down projection with the combine.  Each
// computes exactly what the unfused launches compute.

// Workgroups [0, gx B) compute the logits (4 per workgroup, as
// route_rows_kernel), the rest convert x as q4_prep_x_kernel.
__global__ __launch_bounds__(256) void route_rows_prep_kernel(RouteArgs ra, uint16_t* x16,
                                                              int n8, int gx) {
  const int n_route = gx * ra.B;
  if ((int)blockIdx.x < n_route) {
    route_row_logit<true>(ra, (blockIdx.x % gx) * 4 + wave_id(), blockIdx.x / gx);
    return;
  }
  prep_x8(static_cast<const uint16_t*>(ra.x), x16, (blockIdx.x - n_route) * 256 + threadIdx.x,
          n8);
}

// K-split gate-up with the routing in its prologue (small_layer_routing): the
// last workgroup publishes the routing and exits; the unit work of the
// others is ffn_q4_ksplit_kernel<0, 1, R, W>'s, resolved from the LDS
// buckets.
template <int NJ, int R, int W, bool kPacked>
__global__ __launch_bounds__(W * 64) void ffn_q4_gate_up_routed_kernel(FfnArgs a, RouteArgs ra,
                                                                      GateArgs ga) {
  __shared__ SmallGateLds rt;
  __shared__ f32x4 red[W > 1 ? W * 2 * R * kWave : 1];
  const bool pub = blockIdx.x == gridDim.x - 1;
  if (wave_id() == 0) small_layer_routing<NJ>(ra, ga, rt, pub);
  __syncthreads();
  if (pub) return;
  ffn_q4_ksplit_unit<0, 1, R, W, kPacked>(with_lds_buckets(a, rt), red);
}

// Down projection and combine: a workgroup takes 16 R rows of H for every
// segment (small_down_segment); wave w works on segment w / KW over the
// super-steps of K part w % KW as the K-split down kernel with KW waves
// does, and small_down_finish adds the parts in that kernel's order,
// writes expert_out and forms y.
template <int R, int KW, bool kPacked>
__global__ __launch_bounds__(1024) void ffn_q4_down_combine_kernel(FfnArgs a, const int32_t* idx,
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
    const int nss = K / 128;
    const int lo = part * nss / KW, hi = (part + 1) * nss / KW;
    const size_t mat = (size_t)a.H * K;
    const uint8_t* C0 = static_cast<const uint8_t*>(seg.shared ? a.sh_down : a.down) +
                        seg.id * (mat / 2);
    const uint16_t* S0 = static_cast<const uint16_t*>(seg.shared ? a.sh_down_s : a.down_s) +
                         seg.id * (mat / 32);
    const u32x4* xb[1];
    xb[0] = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.hh) +
                                           (size_t)x_row(a, 1, seg, min(rA, seg.n - 1)) *
                                               a.ldh) +
            gK;
    const u32x4* pc[R];
    const uint16_t* ps[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (kPacked) {
        const size_t tile0 = (size_t)(r0 / 16 + r) * nss;
        pc[r] = reinterpret_cast<const u32x4*>(C0) + tile0 * 64 + lane;
        ps[r] = S0 + tile0 * 64 + lane;
      } else {
        const size_t row = (size_t)(r0 + 16 * r + rA);
        pc[r] = reinterpret_cast<const u32x4*>(C0 + row * (K / 2)) + gK;
        ps[r] = S0 + row * (K / 32) + gK;
      }
    }
    if (hi > lo) {
      const uint32_t magic = opaque(0x64006400u);
      pipeline2<StageQ<1, R, 1>>(
          hi - lo,
          [&](StageQ<1, R, 1>& st, int i) { load_q<kPacked>(st, pc, ps, xb, lo + i); },
          [&](const StageQ<1, R, 1>& st, int) { compute_q(st, acc, magic); });
    }
  }
  small_down_finish<R, KW>(a, seg, live, part, members, acc, lds, y, r0);
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
    case 1: hipLaunchKernelGGL((ffn_q4_ksplit_kernel<kMode, TMAX, R, 1, kPacked>), grid, dim3(64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((ffn_q4_ksplit_kernel<kMode, TMAX, R, 2, kPacked>), grid, dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL((ffn_q4_ksplit_kernel<kMode, TMAX, R, 4, kPacked>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((ffn_q4_ksplit_kernel<kMode, TMAX, R, 8, kPacked>), grid, dim3(512), 0, s, a); break;
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

// Workgroups of one kernel that fit on a compute unit at once, queried once
// per kernel (the same on every device of one type).  `cache` must be the
// calling kernel's own: every instantiation has the same function type.
template <class Kern>
hipError_t resident_per_cu(Kern kern, std::atomic<int>& cache, int* n) {
  if ((*n = cache.load(std::memory_order_relaxed)) > 0) return hipSuccess;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(n, kern, kW * 64, 0);
  if (e != hipSuccess) return e;
  if (*n < 1) *n = 1;
  cache.store(*n, std::memory_order_relaxed);
  return hipSuccess;
}

// Launch of one projection: the grid holds every work item a batch could
// have (all min(E, B k) routed slots active), capped at the workgroups the
// GPU holds at once.
template <int kMode, int TMAX, int R, int D, int A, int C, bool kPacked>
hipError_t launch_q4(const FfnArgs& a, int Q, hipStream_t s) {
  auto kern = ffn_q4_kernel<kMode, TMAX, R, D, A, C, kPacked>;
  static std::atomic<int> resident{0};  // this instantiation's workgroups per CU
  int cus = 0, per_cu = 0;
  hipError_t err = device_cus(&cus);
  if (err == hipSuccess) err = resident_per_cu(kern, resident, &per_cu);
  if (err != hipSuccess) return err;
  constexpr int kRows = 16 * R * kW;
  const int rows_r = kMode == 0 ? a.F : a.H;
  const int rows_s = kMode == 0 ? a.Fs : a.H;
  const int slots = min(a.E, a.B * a.k);
  const long items = ((long)(a.S > 0 ? a.S * (rows_s / kRows) : 0) + (long)slots * (rows_r / kRows)) * Q;
  // A multiple of kXcds workgroups, so every XCD has the same number.
  const long grid = (min(items + kXcds - 1, (long)cus * per_cu) / kXcds) * kXcds;
  if (grid < kXcds) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kW * 64), 0, s, a);
  return hipGetLastError();
}

template <int kMode, int TMAX, int R, int D, int A, int C>
hipError_t launch_q4_layout(const FfnArgs& a, int Q, hipStream_t s) {
  return a.packed ? launch_q4<kMode, TMAX, R, D, A, C, true>(a, Q, s)
                  : launch_q4<kMode, TMAX, R, D, A, C, false>(a, Q, s);
}

#ifndef S2MOE_Q4_RING
#define S2MOE_Q4_RING 2
#endif
#ifndef S2MOE_Q4_ACT_RING
#define S2MOE_Q4_ACT_RING 1
#endif
#ifndef S2MOE_Q4_CHUNK
#define S2MOE_Q4_CHUNK 1
#endif
#ifndef S2MOE_Q4_TMAX_LARGE
#define S2MOE_Q4_TMAX_LARGE 4
#endif
#ifndef S2MOE_Q4_GATEUP_R
#define S2MOE_Q4_GATEUP_R 1
#endif

template <int TMAX>
hipError_t launch_q4_pair(const FfnArgs& a, hipStream_t s) {
  constexpr int D = S2MOE_Q4_RING;
  static_assert(16 * S2MOE_Q4_DOWN_R * kW == kQ4DownRows, "down rows per item");
  constexpr int A = S2MOE_Q4_ACT_RING, C = S2MOE_Q4_CHUNK;
  hipError_t err = launch_q4_layout<0, TMAX, S2MOE_Q4_GATEUP_R, D, A, C>(a, 1, s);
  if (err != hipSuccess) return err;
  return launch_q4_layout<1, TMAX, S2MOE_Q4_DOWN_R, D, A, C>(a, a.qparts, s);
}

// Tiny batches: the K-split kernel, with the most row tiles per unit (gate-up
// 2 or 1, down 4, 2 or 1) that still give every compute unit a workgroup.
// Row tiles per unit of the K-split launches (launch_q4_ksplit): enough
// units to give every compute unit one.
hipError_t ksplit_rows(const FfnArgs& a, int* rg, int* rd) {
  int cus = 0;
  const hipError_t err = device_cus(&cus);
  if (err != hipSuccess) return err;
  *rg = n_blocks(a, 0, 32) >= cus ? 2 : 1;
  *rd = n_blocks(a, 1, 64) >= cus ? 4 : (n_blocks(a, 1, 32) >= cus ? 2 : 1);
  return hipSuccess;
}

// Waves over K of the K-split down launch with rd row tiles per unit.
int ksplit_down_waves(const FfnArgs& a, int rd) {
  int nss = a.F / 128;
  if (a.S > 0) nss = min(nss, a.Fs / 128);
  return pick_waves_q4(nss, rd);
}

hipError_t launch_q4_ksplit(const FfnArgs& a, hipStream_t s) {
  int rg = 1, rd = 1;
  hipError_t err = ksplit_rows(a, &rg, &rd);
  if (err != hipSuccess) return err;
  err = rg == 2 ? launch_q4_mode<0, 1, 2>(a, s) : launch_q4_mode<0, 1, 1>(a, s);
  if (err != hipSuccess) return err;
  if (rd == 4) return launch_q4_mode<1, 1, 4>(a, s);
  if (rd == 2) return launch_q4_mode<1, 1, 2>(a, s);
  return launch_q4_mode<1, 1, 1>(a, s);
}

constexpr int kFusedMaxWavesQ4 = 16;

template <int NJ, bool kPacked>
hipError_t launch_q4_gate_up_routed(const FfnArgs& a, const RouteArgs& ra, const GateArgs& ga,
                                    int rg, hipStream_t s) {
  const int w = pick_waves_q4(a.H / 128, 2 * rg);
  const dim3 grid(n_blocks(a, 0, 16 * rg) + 1);
  if (rg == 2) {
    switch (w) {
      case 1: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 2, 1, kPacked>), grid, dim3(64), 0, s, a, ra, ga); break;
      case 2: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 2, 2, kPacked>), grid, dim3(128), 0, s, a, ra, ga); break;
      case 4: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 2, 4, kPacked>), grid, dim3(256), 0, s, a, ra, ga); break;
      default: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 2, 8, kPacked>), grid, dim3(512), 0, s, a, ra, ga); break;
    }
  } else {
    switch (w) {
      case 1: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 1, 1, kPacked>), grid, dim3(64), 0, s, a, ra, ga); break;
      case 2: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 1, 2, kPacked>), grid, dim3(128), 0, s, a, ra, ga); break;
      case 4: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 1, 4, kPacked>), grid, dim3(256), 0, s, a, ra, ga); break;
      default: hipLaunchKernelGGL((ffn_q4_gate_up_routed_kernel<NJ, 1, 8, kPacked>), grid, dim3(512), 0, s, a, ra, ga); break;
    }
  }
  return hipGetLastError();
}

template <bool kPacked>
hipError_t launch_q4_down_combine(const FfnArgs& a, const int32_t* idx, const float* gate_w,
                                  float* y, int kw, hipStream_t s) {
  const dim3 grid(a.H / 16);
  const dim3 block(64 * kw * (a.S + min(a.E, a.B * a.k)));
  switch (kw) {
    case 1: hipLaunchKernelGGL((ffn_q4_down_combine_kernel<1, 1, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
    case 2: hipLaunchKernelGGL((ffn_q4_down_combine_kernel<1, 2, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
    case 4: hipLaunchKernelGGL((ffn_q4_down_combine_kernel<1, 4, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
    default: hipLaunchKernelGGL((ffn_q4_down_combine_kernel<1, 8, kPacked>), grid, block, 0, s, a, idx, gate_w, y); break;
  }
  return hipGetLastError();
}

template <bool kPacked>
hipError_t launch_q4_small_layer(const RouteArgs& ra, const GateArgs& ga, const FfnArgs& a,
                                 float* y, hipStream_t s) {
  int rg = 1, rd = 1;
  hipError_t err = ksplit_rows(a, &rg, &rd);
  if (err != hipSuccess) return err;
  const int n8 = a.B * a.H / 8;
  const int gx = (a.E + 3) / 4;
  hipLaunchKernelGGL(route_rows_prep_kernel, dim3(gx * a.B + (n8 + 255) / 256), dim3(256), 0, s,
                     ra, static_cast<uint16_t*>(a.x16), n8, gx);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (a.E <= 64) err = launch_q4_gate_up_routed<1, kPacked>(a, ra, ga, rg, s);
  else if (a.E <= 128) err = launch_q4_gate_up_routed<2, kPacked>(a, ra, ga, rg, s);
  else err = launch_q4_gate_up_routed<4, kPacked>(a, ra, ga, rg, s);
  if (err != hipSuccess) return err;
  return launch_q4_down_combine<kPacked>(a, ga.idx, ga.gate_w, y, ksplit_down_waves(a, rd), s);
}

}  // namespace

bool moe_layer_small_fits_q4(const FfnArgs& a) {
  if (a.B > kQ4KsplitMaxTokens || a.qparts != 1) return false;
  int rg = 1, rd = 1;
  if (ksplit_rows(a, &rg, &rd) != hipSuccess) return false;
  return (a.S + min(a.E, a.B * a.k)) * ksplit_down_waves(a, rd) <= kFusedMaxWavesQ4;
}

hipError_t launch_moe_layer_small_q4(const RouteArgs& ra, const GateArgs& ga, const FfnArgs& a,
                                     float* y, hipStream_t s) {
  return a.packed ? launch_q4_small_layer<true>(ra, ga, a, y, s)
                  : launch_q4_small_layer<false>(ra, ga, a, y, s);
}

// Calls f with std::integral_constant<int, Q> for a launch's part count
// Q = 2 .. 8 (q4_down_parts returns at most 8), then checks the launch.
template <class F>
hipError_t with_q4_parts(int Q, F&& f) {
  switch (Q) {
    case 2: f(std::integral_constant<int, 2>()); break;
    case 3: f(std::integral_constant<int, 3>()); break;
    case 4: f(std::integral_constant<int, 4>()); break;
    case 5: f(std::integral_constant<int, 5>()); break;
    case 6: f(std::integral_constant<int, 6>()); break;
    case 7: f(std::integral_constant<int, 7>()); break;
    case 8: f(std::integral_constant<int, 8>()); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_q4_reduce_combine(const FfnArgs& a, const CombineArgs& c, hipStream_t s) {
  const dim3 grid((a.H / 4 + 255) / 256, a.B);
  return with_q4_parts(a.qparts, [&](auto q) {
    hipLaunchKernelGGL((q4_reduce_combine_kernel<decltype(q)::value>), grid, dim3(256), 0, s, a, c);
  });
}

hipError_t launch_ffn_q4(const FfnArgs& a, hipStream_t s) {
  hipError_t err = hipSuccess;
  if (!a.x16_ready) {
    const int n8 = a.B * a.H / 8;
    hipLaunchKernelGGL(q4_prep_x_kernel, dim3((n8 + 255) / 256), dim3(256), 0, s,
                       static_cast<const uint16_t*>(a.x), static_cast<uint16_t*>(a.x16), n8);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  if (a.B <= kQ4KsplitMaxTokens) return launch_q4_ksplit(a, s);
  // Token tiles held in one pass: the batch bounds every bucket.
  if (a.B <= 16) err = launch_q4_pair<1>(a, s);
  else if (a.B <= 32) err = launch_q4_pair<2>(a, s);
  else err = launch_q4_pair<S2MOE_Q4_TMAX_LARGE>(a, s);
  if (err != hipSuccess || a.qparts <= 1 || a.defer_reduce) return err;
  const size_t n4 = ((size_t)a.B * a.k + (size_t)a.S * a.B) * a.H / 4;
  const dim3 grid((unsigned)((n4 + 255) / 256));
  return with_q4_parts(a.qparts, [&](auto q) {
    hipLaunchKernelGGL((q4_reduce_kernel<decltype(q)::value>), grid, dim3(256), 0, s, a.out,
                       static_cast<const float*>(a.part), n4);
  });
}

}  // namespace s2moe
