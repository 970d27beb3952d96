// Weight packing for the matrix-core FFN kernels.
//
// Packed order of one matrix [rows, K] (per expert):
//   bf16:  tile (rt, s) = rows 16 rt .. 16 rt + 15, K 32 s .. 32 s + 31, 1 KB,
//          stored at ((rt * K/32) + s) KB; inside a tile the 16 bytes of lane L
//          (0..63) are row 16 rt + L % 16, K 32 s + 8 (L / 16) .. + 7 -- the A
//          operand of v_mfma_f32_16x16x32_bf16 for that lane.
//   int4:  codes: tile (rt, S) = rows 16 rt.., the 128-wide K block S, 1 KB at
//          ((rt * K/128) + S) KB; lane L's 16 bytes are the 32 codes of group
//          4 S + L / 16 of row 16 rt + L % 16.  scales: 128 bytes per tile at
//          ((rt * K/128) + S) * 128; lane L's fp16 is that group's scale.
// A wave that streams K steps lo..hi of one row tile therefore reads one
// contiguous range, 1 KB per load instruction.  The element values do not
// change; only their order does.
#include "common.h"
#include "kernels.h"

namespace s2moe {

namespace {

// One thread per 16-byte packed chunk.
__global__ __launch_bounds__(256) void pack_bf16_kernel(const uint16_t* __restrict__ src,
                                                        uint16_t* __restrict__ dst, int n,
                                                        int rows, int K) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t per_mat = (size_t)rows * K / 8;
  if (i >= (size_t)n * per_mat) return;
  const size_t m = i / per_mat;
  const size_t c = i % per_mat;           // chunk within the packed matrix
  const int lane = (int)(c % 64);
  const size_t tile = c / 64;
  const int nks = K / 32;
  const int rt = (int)(tile / nks), s = (int)(tile % nks);
  const int row = 16 * rt + (lane & 15);
  const int k0 = 32 * s + 8 * (lane >> 4);
  const u32x4 v = *reinterpret_cast<const u32x4*>(src + m * rows * K + (size_t)row * K + k0);
  reinterpret_cast<u32x4*>(dst)[i] = v;
}

__global__ __launch_bounds__(256) void pack_q4_kernel(const uint8_t* __restrict__ src,
                                                      const uint16_t* __restrict__ src_s,
                                                      uint8_t* __restrict__ dst,
                                                      uint16_t* __restrict__ dst_s, int n,
                                                      int rows, int K) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t per_mat = (size_t)rows * K / 32;  // one 16-byte group per thread
  if (i >= (size_t)n * per_mat) return;
  const size_t m = i / per_mat;
  const size_t c = i % per_mat;
  const int lane = (int)(c % 64);
  const size_t tile = c / 64;
  const int nss = K / 128;
  const int rt = (int)(tile / nss), S = (int)(tile % nss);
  const int row = 16 * rt + (lane & 15);
  const int grp = 4 * S + (lane >> 4);
  const u32x4 v = *reinterpret_cast<const u32x4*>(src + m * rows * (K / 2) +
                                                   (size_t)row * (K / 2) + (size_t)grp * 16);
  reinterpret_cast<u32x4*>(dst)[i] = v;
  dst_s[i] = src_s[m * rows * (K / 32) + (size_t)row * (K / 32) + grp];
}

}  // namespace

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
  if (a.q4) {
    const size_t n = (size_t)a.n * a.rows * a.K / 32;
    hipLaunchKernelGGL(pack_q4_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       static_cast<const uint8_t*>(a.src), static_cast<const uint16_t*>(a.src_s),
                       static_cast<uint8_t*>(a.dst), static_cast<uint16_t*>(a.dst_s), a.n,
                       a.rows, a.K);
  } else {
    const size_t n = (size_t)a.n * a.rows * a.K / 8;
    hipLaunchKernelGGL(pack_bf16_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       static_cast<const uint16_t*>(a.src), static_cast<uint16_t*>(a.dst), a.n,
                       a.rows, a.K);
  }
  return hipGetLastError();
}

}  // namespace s2moe
