// Device helpers shared by the s2moe kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace s2moe {

constexpr int kWave = 64;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}

// Total-order key of a float: larger value -> larger key.  -0 is folded
// into +0 first so that equal values tie (and then break on the index).
__device__ __forceinline__ uint32_t order_key(float v) {
  uint32_t u = __float_as_uint(v + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)v, m, kWave);
    uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, kWave);
    uint64_t o = ((uint64_t)hi << 32) | lo;
    v = o > v ? o : v;
  }
  return v;
}

// Exclusive prefix sum across the wave; returns the lane's exclusive sum and
// writes the wave total.
__device__ __forceinline__ int wave_exclusive_scan(int v, int* total) {
  const int lane = threadIdx.x & (kWave - 1);
  int incl = v;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    int o = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += o;
  }
  *total = __shfl(incl, kWave - 1, kWave);
  return incl - v;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & (kWave - 1);
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Wave-wide reductions through DPP lane moves (quad permutes, row mirrors,
// row broadcasts), finished by reading lane 63.  The combination order is
// fixed, so results are deterministic.
#define S2MOE_DPP_STEP(v, ident, op, ctrl, rmask)                                              \
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(ident), __float_as_int(v), \
                                                        ctrl, rmask, 0xF, false)))

__device__ __forceinline__ float add_f(float a, float b) { return a + b; }
__device__ __forceinline__ float max_f(float a, float b) { return fmaxf(a, b); }

__device__ __forceinline__ float wave_sum_dpp(float v) {
  S2MOE_DPP_STEP(v, 0.f, add_f, 0xB1, 0xF);   // quad_perm [1,0,3,2]
  S2MOE_DPP_STEP(v, 0.f, add_f, 0x4E, 0xF);   // quad_perm [2,3,0,1]
  S2MOE_DPP_STEP(v, 0.f, add_f, 0x141, 0xF);  // row_half_mirror
  S2MOE_DPP_STEP(v, 0.f, add_f, 0x140, 0xF);  // row_mirror
  S2MOE_DPP_STEP(v, 0.f, add_f, 0x142, 0xA);  // row_bcast:15
  S2MOE_DPP_STEP(v, 0.f, add_f, 0x143, 0xC);  // row_bcast:31
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_max_dpp(float v) {
  const float ni = -INFINITY;
  S2MOE_DPP_STEP(v, ni, max_f, 0xB1, 0xF);
  S2MOE_DPP_STEP(v, ni, max_f, 0x4E, 0xF);
  S2MOE_DPP_STEP(v, ni, max_f, 0x141, 0xF);
  S2MOE_DPP_STEP(v, ni, max_f, 0x140, 0xF);
  S2MOE_DPP_STEP(v, ni, max_f, 0x142, 0xA);
  S2MOE_DPP_STEP(v, ni, max_f, 0x143, 0xC);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Value of the k-th largest entry (duplicates counted) among the order keys
// held four per lane: a bit-by-bit search of the largest threshold with at
// least k keys at or above it (ballots count them).  Empty slots hold 0,
// below every real key.  Wave-uniform, branch-free apart from the loop.
__device__ __forceinline__ uint32_t wave_kth_key(const uint32_t key[4], int k) {
  uint32_t prefix = 0;
#pragma unroll 4
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    const int cnt = __popcll(__ballot(key[0] >= cand)) + __popcll(__ballot(key[1] >= cand)) +
                    __popcll(__ballot(key[2] >= cand)) + __popcll(__ballot(key[3] >= cand));
    prefix = cnt >= k ? cand : prefix;
  }
  return prefix;
}

// Flags (bit j of a lane) of the k best entries under (value desc, expert id
// asc), given kth = wave_kth_key(key, k): every key above kth, plus the keys
// equal to kth with the smallest expert ids (expert lane + 64 j) up to k.
__device__ __forceinline__ uint32_t wave_select_top(const uint32_t key[4], uint32_t kth, int k) {
  const int above = __popcll(__ballot(key[0] > kth)) + __popcll(__ballot(key[1] > kth)) +
                    __popcll(__ballot(key[2] > kth)) + __popcll(__ballot(key[3] > kth));
  const int need = k - above;
  const uint64_t lt = lanemask_lt();
  uint32_t bits = 0;
  int before = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint64_t m = __ballot(key[j] == kth);
    const int r = before + __popcll(m & lt);
    if (key[j] > kth || (key[j] == kth && r < need)) bits |= 1u << j;
    before += __popcll(m);
  }
  return bits;
}

// Rank, in ascending expert id, of the flagged experts: expert lane + 64 j
// with bit j set gets position rank[j].  Returns the number flagged.
__device__ __forceinline__ int wave_rank_flagged(uint32_t bits, int rank[4]) {
  int before = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint64_t m = __ballot((bits >> j) & 1u);
    rank[j] = before + __popcll(m & lanemask_lt());
    before += __popcll(m);
  }
  return before;
}

}  // namespace s2moe
