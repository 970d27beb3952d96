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

// Wave-cooperative top-n selection over up to 256 values held four per lane
// (value j of a lane is expert lane + 64 j).  Order: value descending, then
// expert id ascending.  `n_sel` rounds pick the n_sel best; the experts of
// the first `n_mark` rounds are flagged in `taken_bits` (bit j of a lane).
// The values picked in the first and in the last round are returned
// (wave-uniform).
__device__ __forceinline__ void wave_topn(const float v[4], int E, int n_sel, int n_mark,
                                          uint32_t* taken_bits, float* first_val,
                                          float* last_val) {
  const int lane = threadIdx.x & (kWave - 1);
  uint64_t key[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + kWave * j;
    key[j] = (e < E) ? (((uint64_t)order_key(v[j]) << 32) | (uint32_t)(0xFFFFu - e)) : 0ull;
  }
  uint32_t bits = 0;
  float first = 0.f, last = 0.f;
  for (int r = 0; r < n_sel; ++r) {
    uint64_t best = key[0];
#pragma unroll
    for (int j = 1; j < 4; ++j) best = key[j] > best ? key[j] : best;
    best = wave_max_u64(best);
    const int e = 0xFFFF - (int)(uint32_t)(best & 0xFFFFu);
    last = key_value((uint32_t)(best >> 32));
    if (r == 0) first = last;
    if ((e & (kWave - 1)) == lane) {
      const int j = e / kWave;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        if (jj == j) key[jj] = 0ull;
      if (r < n_mark) bits |= 1u << j;
    }
  }
  *taken_bits = bits;
  *first_val = first;
  *last_val = last;
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
