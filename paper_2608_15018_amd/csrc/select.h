// Wave- and workgroup-level ranking helpers of the routing kernels: order
// keys, DPP reductions and scans, exact top-k selection with ties broken
// towards the lower expert id.  Every result is deterministic.
#pragma once

#include "common.h"

namespace s2moe {

// Total-order key of a float: larger value -> larger key.  -0 is folded
// into +0 first so that equal values tie (and then break on the index).
// Finite values map to keys >= 0x00800000, so 0 can mark an empty slot.
__device__ __forceinline__ uint32_t order_key(float v) {
  uint32_t u = __float_as_uint(v + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & (kWave - 1);
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Wave-wide reductions through DPP lane moves (quad permutes, row mirrors,
// row broadcasts), finished by reading lane 63.  The combination order is
// fixed, so results are deterministic.  Lanes a move does not reach take
// the identity.
#define S2MOE_DPP(ident, v, ctrl, rmask) \
  __builtin_amdgcn_update_dpp((ident), (v), (ctrl), (rmask), 0xF, false)

__device__ __forceinline__ float wave_sum_dpp(float x) {
  int v = __float_as_int(x);
  v = __float_as_int(__int_as_float(v) + __int_as_float(S2MOE_DPP(0, v, 0xB1, 0xF)));  // quad [1,0,3,2]
  v = __float_as_int(__int_as_float(v) + __int_as_float(S2MOE_DPP(0, v, 0x4E, 0xF)));  // quad [2,3,0,1]
  v = __float_as_int(__int_as_float(v) + __int_as_float(S2MOE_DPP(0, v, 0x141, 0xF))); // row_half_mirror
  v = __float_as_int(__int_as_float(v) + __int_as_float(S2MOE_DPP(0, v, 0x140, 0xF))); // row_mirror
  v = __float_as_int(__int_as_float(v) + __int_as_float(S2MOE_DPP(0, v, 0x142, 0xA))); // row_bcast:15
  v = __float_as_int(__int_as_float(v) + __int_as_float(S2MOE_DPP(0, v, 0x143, 0xC))); // row_bcast:31
  return __int_as_float(__builtin_amdgcn_readlane(v, 63));
}

// Maximum of unsigned keys (0 is the identity).
__device__ __forceinline__ uint32_t wave_max_key_dpp(uint32_t x) {
  int v = (int)x;
  v = (int)max((uint32_t)v, (uint32_t)S2MOE_DPP(0, v, 0xB1, 0xF));
  v = (int)max((uint32_t)v, (uint32_t)S2MOE_DPP(0, v, 0x4E, 0xF));
  v = (int)max((uint32_t)v, (uint32_t)S2MOE_DPP(0, v, 0x141, 0xF));
  v = (int)max((uint32_t)v, (uint32_t)S2MOE_DPP(0, v, 0x140, 0xF));
  v = (int)max((uint32_t)v, (uint32_t)S2MOE_DPP(0, v, 0x142, 0xA));
  v = (int)max((uint32_t)v, (uint32_t)S2MOE_DPP(0, v, 0x143, 0xC));
  return (uint32_t)__builtin_amdgcn_readlane(v, 63);
}

// Inclusive prefix sum across the wave through DPP row shifts and row
// broadcasts; the total is in lane 63.
__device__ __forceinline__ int wave_inclusive_scan_dpp(int v) {
  v += S2MOE_DPP(0, v, 0x111, 0xF);  // row_shr:1
  v += S2MOE_DPP(0, v, 0x112, 0xF);  // row_shr:2
  v += S2MOE_DPP(0, v, 0x114, 0xF);  // row_shr:4
  v += S2MOE_DPP(0, v, 0x118, 0xF);  // row_shr:8
  v += S2MOE_DPP(0, v, 0x142, 0xA);  // row_bcast:15
  v += S2MOE_DPP(0, v, 0x143, 0xC);  // row_bcast:31
  return v;
}

// Exact top-k of NT independent key sets held NJ per lane (slot j of a lane
// is expert lane + 64 j; empty slots hold key 0, below every real key),
// under (key desc, expert id asc).  Bit j of sel[t] flags slot j.
//
// A bit-by-bit search over the upper 16 key bits finds the largest prefix P
// with at least k keys whose upper half is >= P (ballots count them; the NT
// searches advance together so that their dependency chains overlap).
// Keys above the bucket P are in; when the bucket holds more keys than the
// places left, its members are ranked among themselves exactly (a scalar
// loop over the bucket, which is almost always one or two keys).  A set
// with fewer than k real keys gets an unspecified selection.
template <int NT, int NJ>
__device__ __forceinline__ void wave_top_k(const uint32_t (&key)[NT][NJ], int k,
                                           uint32_t (&sel)[NT]) {
  uint32_t p[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) p[t] = 0;
#pragma unroll 2
  for (int bit = 31; bit >= 16; --bit) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const uint32_t cand = p[t] | (1u << bit);
      int cnt = 0;
#pragma unroll
      for (int j = 0; j < NJ; ++j) cnt += __popcll(__ballot(key[t][j] >= cand));
      p[t] = cnt >= k ? cand : p[t];
    }
  }
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const uint32_t P = p[t] >> 16;
    uint64_t in_bucket[NJ];
    int above = 0, n_bucket = 0;
    sel[t] = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const uint32_t hi = key[t][j] >> 16;
      above += __popcll(__ballot(hi > P));
      in_bucket[j] = __ballot(hi == P);
      n_bucket += __popcll(in_bucket[j]);
      if (hi >= P) sel[t] |= 1u << j;
    }
    const int need = k - above;  // 1 <= need <= n_bucket
    if (need < n_bucket && P != 0) {
      int r[NJ];
#pragma unroll
      for (int j = 0; j < NJ; ++j) r[j] = 0;
#pragma unroll
      for (int j2 = 0; j2 < NJ; ++j2) {
        uint64_t m = in_bucket[j2];
        while (m) {
          const int l2 = __builtin_ctzll(m);
          m &= m - 1;
          const uint32_t k2 = __builtin_amdgcn_readlane(key[t][j2], l2);
          const int e2 = l2 + kWave * j2;
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            r[j] += (k2 > key[t][j]) || (k2 == key[t][j] && e2 < lane + kWave * j);
        }
      }
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        if ((key[t][j] >> 16) == P && r[j] >= need) sel[t] &= ~(1u << j);
    }
  }
}

// Rank, in ascending expert id, of the flagged experts: expert lane + 64 j
// with bit j set gets position rank[j].  Returns the number flagged.
template <int NJ>
__device__ __forceinline__ int wave_rank_flagged(uint32_t bits, int (&rank)[NJ]) {
  int before = 0;
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const uint64_t m = __ballot((bits >> j) & 1u);
    rank[j] = before + __popcll(m & lt);
    before += __popcll(m);
  }
  return before;
}

}  // namespace s2moe
