// Reuse-aware expert gating and token->expert bucketing (Sec. "Reuse-aware
// Expert Gating": cross-token expert importance aggregation, global
// preferred expert selection, soft routing bias for reuse promotion).
//
// One workgroup of 16 waves handles the whole verify batch (B <= 256,
// E <= 256): the decisions couple all tokens through g, and the batch is
// small.  Nothing here is a serial loop over assignments:
//   * g: one thread per expert sums w_b * ell_{b,e} over b in order;
//   * TopCap: each expert's rank among the candidates by (g desc, id asc);
//   * per token (one wave): biased order keys, a bitwise threshold search
//     for the k-th largest value (ties to the lower expert id), ballot ranks
//     for ascending-id order, DPP softmax;
//   * buckets: a B-bit token mask per expert (LDS 64-bit ORs), so an
//     assignment's position in its expert's list is the popcount of the mask
//     below its token.
// Every result is deterministic: integer atomics only (bitwise OR), fixed
// floating-point summation orders, rank-based placement.
#include "common.h"
#include "kernels.h"

namespace s2moe {

constexpr int kStage = 10240;  // logits staged in LDS up to B * E = 10240

template <bool kStaged>
__global__ __launch_bounds__(1024) void reuse_gate_kernel(GateArgs a) {
  constexpr int kMaskWords = kMaxTokens / 64;
  __shared__ float ell_s[kStaged ? kStage : 1];
  __shared__ float w_s[kMaxTokens];
  __shared__ float gap_s[kMaxTokens];
  __shared__ __align__(16) float gm_s[kMaxExperts];  // g of candidates, -inf otherwise
  __shared__ int pref_s[kMaxExperts];
  __shared__ int count_s[kMaxExperts];
  __shared__ int offset_s[kMaxExperts + 1];
  __shared__ uint64_t mask_s[kMaxExperts][kMaskWords];
  __shared__ uint8_t idx_s[kMaxTokens * kMaxTopK];
  __shared__ int cand_s[kMaxExperts];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid >> 6;
  const int n_waves = blockDim.x >> 6;
  const int B = a.B, E = a.E, k = a.k;

  // Non-negative confidences w_b; logits to LDS; cleared masks.
  int positive = 0;
  if (tid < B) {
    const float w = fmaxf(a.conf_w[tid], 0.f);
    w_s[tid] = w;
    gap_s[tid] = a.gap[tid];
    positive = w > 0.f;
  }
  if (kStaged) {
    // All loads first, then the LDS writes (10 per thread at most).
    constexpr int kPer = kStage / 1024;
    float v[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int i = tid + q * 1024;
      v[q] = i < B * E ? a.logits[i] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int i = tid + q * 1024;
      if (i < B * E) ell_s[i] = v[q];
    }
  }
  for (int i = tid; i < kMaxExperts * kMaskWords; i += blockDim.x)
    (&mask_s[0][0])[i] = 0ull;
  if (tid < kMaxExperts) cand_s[tid] = (!(a.flags & kPrefActivatedOnly) && tid < E) ? 1 : 0;
  const int active = __syncthreads_or(positive);
  const float* ell = kStaged ? static_cast<const float*>(ell_s) : a.logits;

  // TopCap candidates: all experts, or those in some token's plain top-k.
  if (a.flags & kPrefActivatedOnly) {
    for (int i = tid; i < B * k; i += blockDim.x) {
      const int e = a.plain_idx[i];
      if (e >= 0 && e < E) cand_s[e] = 1;
    }
    __syncthreads();
  }

  // g_e = sum_b w_b * ell_{b,e}, summed over b in order.
  if (tid < E) {
    float s = 0.f;
#pragma unroll 8
    for (int b = 0; b < B; ++b) s = fmaf(w_s[b], ell[(size_t)b * E + tid], s);
    a.g[tid] = s;
    gm_s[tid] = cand_s[tid] ? s : -INFINITY;
  }
  __syncthreads();

  // E* = TopCap(g): rank of each candidate by (g desc, id asc).
  if (tid < E) {
    int p = 0;
    if (active && cand_s[tid]) {
      const float ge = gm_s[tid];
      int rank = 0;
      const f32x4* g4 = reinterpret_cast<const f32x4*>(gm_s);
      for (int q = 0; q < (E + 3) / 4; ++q) {
        const f32x4 g2 = g4[q];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e2 = 4 * q + i;
          rank += (e2 < E) && ((g2[i] > ge) || (g2[i] == ge && e2 < tid));
        }
      }
      p = rank < a.cap;
    }
    pref_s[tid] = p;
    a.pref[tid] = p;
  }
  __syncthreads();

  // Per token: lambda_b, biased keys, biased top-k, gate weights, masks.
  const bool from_biased = (a.flags & kGateFromBiased) != 0;
  for (int b = wave; b < B; b += n_waves) {
    float lam = 0.f;
    if (active) lam = (a.flags & kBiasAbsolute) ? a.alpha : a.alpha * gap_s[b];
    float l[4], lb[4];
    uint32_t key[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane + kWave * j;
      l[j] = 0.f;
      lb[j] = 0.f;
      key[j] = 0;
      if (e < E) {
        l[j] = ell[(size_t)b * E + e];
        lb[j] = pref_s[e] ? l[j] + lam : l[j];
        key[j] = order_key(lb[j]);
      }
    }
    const uint32_t bits = wave_select_top(key, wave_kth_key(key, k), k);
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if ((bits >> j) & 1u) m = fmaxf(m, from_biased ? lb[j] : l[j]);
    int rank[4];
    wave_rank_flagged(bits, rank);
    m = wave_max_dpp(m);
    float ez[4];
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ez[j] = ((bits >> j) & 1u) ? expf((from_biased ? lb[j] : l[j]) - m) : 0.f;
      s += ez[j];
    }
    s = wave_sum_dpp(s);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if ((bits >> j) & 1u) {
        const int pos = b * k + rank[j];
        const int e = lane + kWave * j;
        a.idx[pos] = e;
        a.gate_w[pos] = ez[j] / s;
        idx_s[pos] = (uint8_t)e;
        atomicOr(reinterpret_cast<unsigned long long*>(&mask_s[e][b >> 6]),
                 1ull << (b & 63));
      }
    }
  }
  __syncthreads();

  // Counts from the masks; exclusive offsets and the activated-expert list.
  if (tid < E) {
    int c = 0;
#pragma unroll
    for (int w = 0; w < kMaskWords; ++w) c += __popcll(mask_s[tid][w]);
    count_s[tid] = c;
    a.count[tid] = c;
  }
  __syncthreads();
  if (wave == 0) {
    int c[4], f[4], sum_c = 0, sum_f = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane * 4 + j;
      c[j] = e < E ? count_s[e] : 0;
      f[j] = c[j] > 0;
      sum_c += c[j];
      sum_f += f[j];
    }
    int total_c, total_f;
    int run_c = wave_exclusive_scan(sum_c, &total_c);
    int run_f = wave_exclusive_scan(sum_f, &total_f);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane * 4 + j;
      if (e < E) {
        offset_s[e] = run_c;
        a.offset[e] = run_c;
        if (f[j]) a.uniq[run_f] = e;
      }
      run_c += c[j];
      run_f += f[j];
    }
    for (int i = total_f + lane; i < E; i += kWave) a.uniq[i] = -1;
    if (lane == 0) {
      offset_s[E] = total_c;
      a.offset[E] = total_c;
      *a.n_uniq = total_f;
    }
  }
  __syncthreads();

  // Stable expert-major slot list: assignment (b, j) of expert e goes after
  // the assignments of e by tokens b' < b.
  for (int i = tid; i < B * k; i += blockDim.x) {
    const int b = i / k;
    const int e = idx_s[i];
    int before = 0;
#pragma unroll
    for (int w = 0; w < kMaskWords; ++w) {
      const uint64_t m = mask_s[e][w];
      if (w < (b >> 6)) before += __popcll(m);
      else if (w == (b >> 6)) before += __popcll(m & ((1ull << (b & 63)) - 1ull));
    }
    a.slot[offset_s[e] + before] = i;
  }
}

hipError_t launch_reuse_gate(const GateArgs& a, hipStream_t s) {
  if (a.B * a.E <= kStage)
    hipLaunchKernelGGL(reuse_gate_kernel<true>, dim3(1), dim3(1024), 0, s, a);
  else
    hipLaunchKernelGGL(reuse_gate_kernel<false>, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
