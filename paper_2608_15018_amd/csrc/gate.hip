// Reuse-aware expert gating and token->expert bucketing (Sec. "Reuse-aware
// Expert Gating": cross-token expert importance aggregation, global
// preferred expert selection, soft routing bias for reuse promotion).
//
// One workgroup of 16 waves handles the whole verify batch (B <= 256,
// E <= 256): the gating decisions couple all tokens through g, and the
// batch is small enough that one CU finishes it in a few microseconds.
// Every result is deterministic: integer LDS atomics only, fixed-order
// floating-point sums, rank-based (not atomic-order-based) placement.
#include "common.h"
#include "kernels.h"

namespace s2moe {

__global__ __launch_bounds__(1024) void reuse_gate_kernel(GateArgs a) {
  __shared__ float w_s[kMaxTokens];
  __shared__ float g_s[kMaxExperts];
  __shared__ int cand_s[kMaxExperts];
  __shared__ int pref_s[kMaxExperts];
  __shared__ int count_s[kMaxExperts];
  __shared__ int offset_s[kMaxExperts + 1];
  __shared__ uint8_t idx_s[kMaxTokens * kMaxTopK];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid >> 6;
  const int n_waves = blockDim.x >> 6;
  const int B = a.B, E = a.E, k = a.k;

  // Non-negative confidence weights w_b.
  int positive = 0;
  if (tid < B) {
    const float w = fmaxf(a.conf_w[tid], 0.f);
    w_s[tid] = w;
    positive = w > 0.f;
  }
  if (tid < kMaxExperts) {
    cand_s[tid] = (!(a.flags & kPrefActivatedOnly) && tid < E) ? 1 : 0;
    count_s[tid] = 0;
  }
  const int active = __syncthreads_or(positive);

  // TopCap candidates: all experts, or those in some token's plain top-k.
  if (a.flags & kPrefActivatedOnly)
    for (int i = tid; i < B * k; i += blockDim.x) {
      const int e = a.plain_idx[i];
      if (e >= 0 && e < E) cand_s[e] = 1;
    }

  // g_e = sum_b w_b * ell_{b,e}, summed over b in order.
  if (tid < E) {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s = fmaf(w_s[b], a.logits[(size_t)b * E + tid], s);
    g_s[tid] = s;
    a.g[tid] = s;
  }
  __syncthreads();

  // E* = TopCap(g): rank of e among candidates by (g desc, id asc).
  if (tid < E) {
    int p = 0;
    if (active && cand_s[tid]) {
      const float ge = g_s[tid];
      int rank = 0;
      for (int e2 = 0; e2 < E; ++e2) {
        if (!cand_s[e2]) continue;
        const float g2 = g_s[e2];
        rank += (g2 > ge) || (g2 == ge && e2 < tid);
      }
      p = rank < a.cap;
    }
    pref_s[tid] = p;
    a.pref[tid] = p;
  }
  __syncthreads();

  // Per token: lambda_b, biased logits, biased top-k, gate weights.
  for (int b = wave; b < B; b += n_waves) {
    float lam = 0.f;
    if (active) lam = (a.flags & kBiasAbsolute) ? a.alpha : a.alpha * a.gap[b];
    float l[4], lb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane + kWave * j;
      l[j] = e < E ? a.logits[(size_t)b * E + e] : 0.f;
      lb[j] = (e < E && pref_s[e]) ? l[j] + lam : l[j];
    }
    uint32_t bits;
    float first, last;
    wave_topn(lb, E, k, k, &bits, &first, &last);
    int rank[4];
    wave_rank_flagged(bits, rank);

    const bool from_biased = (a.flags & kGateFromBiased) != 0;
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if ((bits >> j) & 1u) m = fmaxf(m, from_biased ? lb[j] : l[j]);
    m = wave_max(m);
    float ez[4];
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ez[j] = ((bits >> j) & 1u) ? expf((from_biased ? lb[j] : l[j]) - m) : 0.f;
      s += ez[j];
    }
    s = wave_sum(s);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if ((bits >> j) & 1u) {
        const int pos = b * k + rank[j];
        const int e = lane + kWave * j;
        a.idx[pos] = e;
        a.gate_w[pos] = ez[j] / s;
        idx_s[pos] = (uint8_t)e;
      }
    }
  }
  __syncthreads();

  // Bucketing: counts, exclusive offsets, activated experts.
  for (int i = tid; i < B * k; i += blockDim.x) atomicAdd(&count_s[idx_s[i]], 1);
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
        if (f[j]) a.uniq[run_f] = e;
      }
      run_c += c[j];
      run_f += f[j];
    }
    for (int i = total_f + lane; i < E; i += kWave) a.uniq[i] = -1;
    if (lane == 0) {
      offset_s[E] = total_c;
      *a.n_uniq = total_f;
    }
  }
  __syncthreads();

  // Stable expert-major slot list: expert e lists its assignments a = b*k+j
  // in increasing a.
  if (tid < E) {
    int p = offset_s[tid];
    const int c = count_s[tid];
    a.count[tid] = c;
    a.offset[tid] = p;
    if (c > 0)
      for (int i = 0; i < B * k; ++i)
        if (idx_s[i] == tid) a.slot[p++] = i;
  }
  if (tid == 0) a.offset[E] = offset_s[E];
}

hipError_t launch_reuse_gate(const GateArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(reuse_gate_kernel, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

}  // namespace s2moe
