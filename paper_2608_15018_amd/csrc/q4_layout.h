// Layout of the int4 path's fp16 activations, shared by the expert-FFN
// kernels and the launches that convert x for them.
#pragma once

#include "common.h"

namespace s2moe {

// Position of element e of an 8-element block in the int4 decode order
// (0,4,1,5,2,6,3,7).
__device__ __forceinline__ int pos8(int e) { return ((e & 3) << 1) | (e >> 2); }

// Where 8-block c of a row of activations is stored: inside each 128-wide
// super-step (16 blocks, block 4 g + j = dword j of code group g) the blocks
// are stored j-major, so that the four lanes of one token that feed MFMA j
// read 64 contiguous bytes.
__host__ __device__ __forceinline__ int block_pos(int c) {
  return (c & ~15) | ((c & 3) << 2) | ((c >> 2) & 3);
}

// x [B, H] bf16 -> x16 [B, H] fp16 in the kernels' order (block_pos, then
// decode order inside each block) for the 8 elements of block i < n8 (H is a
// multiple of 128, so a row holds whole super-steps).
__device__ __forceinline__ void prep_x8(const uint16_t* __restrict__ x,
                                        uint16_t* __restrict__ x16, int i, int n8) {
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

}  // namespace s2moe
