// Reuse-aware expert gating and token->expert bucketing (Sec. "Reuse-aware
// Expert Gating": cross-token expert importance aggregation, global
// preferred expert selection, soft routing bias for reuse promotion).
//
// One workgroup of 16 waves handles the whole verify batch (B <= 256,
// E <= 256): the decisions couple all tokens through g, and the batch is
// small.  Nothing here is a serial loop over assignments:
//   * g: a few threads per expert sum runs of tokens, runs added in order;
//   * TopCap: one wave's exact top-cap of the candidates' g by (g desc, id
//     asc), the threshold search used for the per-token top-k;
//   * per token (one wave, up to 4 tokens at a time): biased order keys, an
//     exact top-k (a bitwise threshold search over the upper key halves,
//     then the boundary bucket ranked; ties to the lower expert id), ballot
//     ranks for ascending-id order, DPP softmax;
//   * buckets: a B-bit token mask per expert (LDS 64-bit ORs), so an
//     assignment's position in its expert's list is the popcount of the mask
//     below its token.
// Every result is deterministic: integer atomics only (bitwise OR), fixed
// floating-point summation orders, rank-based placement.
#include "small_batch.h"

namespace s2moe {

constexpr int kStage = 10240;  // logits staged in LDS up to B * E = 10240

// kNJ = expert slots per lane (E <= 64 kNJ); kNT = tokens a wave takes
// through the threshold search together.  kSelect (with kStaged): the
// kernel first ranks every token's staged logits itself (wave_select_plain,
// the routing kernel's code, one wave per token) and writes plain_idx and
// gap, instead of reading them from a routing launch (ra: the routing
// step's arguments).
template <bool kStaged, int kNJ, int kNT, bool kSelect>
__global__ __launch_bounds__(1024) void reuse_gate_kernel(GateArgs a, RouteArgs ra) {
  static_assert(kStaged || !kSelect, "ranking reads the staged logits");
  constexpr int kMaskWords = kMaxTokens / 64;
  __shared__ float ell_s[kStaged ? kStage : 1];
  __shared__ float w_s[kMaxTokens];
  __shared__ float gap_s[kMaxTokens];
  __shared__ float gm_s[kMaxExperts];                  // g of every expert
  __shared__ int pref_s[kMaxExperts];
  __shared__ int count_s[kMaxExperts];
  __shared__ int offset_s[kMaxExperts + 1];
  __shared__ uint64_t mask_s[kMaxExperts][kMaskWords];
  // [part][E] partial sums of g first, the selected expert ids later.
  static_assert(kMaxTokens * kMaxTopK == 4 * 1024, "shared buffer size");
  __shared__ float gpart_s[1024];
  uint8_t* idx_s = reinterpret_cast<uint8_t*>(gpart_s);
  __shared__ int cand_s[kMaxExperts];
  __shared__ uint8_t plain_s[kSelect ? kMaxTokens * kMaxTopK : 1];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = wave_id();
  const int n_waves = blockDim.x >> 6;
  const int B = a.B, E = a.E, k = a.k;

  // Non-negative confidences w_b; logits to LDS; cleared masks and ranks.
  int positive = 0;
  if (tid < B) {
    const float w = fmaxf(a.conf_w[tid], 0.f);
    w_s[tid] = w;
    if (!kSelect) gap_s[tid] = a.gap[tid];
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
  if (tid < kMaxExperts) {
    cand_s[tid] = (!(a.flags & kPrefActivatedOnly) && tid < E) ? 1 : 0;
  }
  const int active = __syncthreads_or(positive);
  const float* ell = kStaged ? static_cast<const float*>(ell_s) : a.logits;

  if (kSelect) {
    for (int b = wave; b < B; b += n_waves)
      wave_select_plain<kNJ>(E, k, ell + (size_t)b * E, plain_s + b * k, gap_s + b,
                             ra.plain_idx + (size_t)b * k, ra.gap + b);
    __syncthreads();
  }

  // TopCap candidates: all experts, or those in some token's plain top-k.
  if (a.flags & kPrefActivatedOnly) {
    for (int i = tid; i < B * k; i += blockDim.x) {
      const int e = kSelect ? (int)plain_s[i] : a.plain_idx[i];
      if (e >= 0 && e < E) cand_s[e] = 1;
    }
  }

  // g_e = sum_b w_b * ell_{b,e}: `parts` threads per expert each sum a
  // contiguous run of tokens in order, then the runs are added in order.
  int parts = 1;
  while (parts * 2 * E <= 1024 && parts * 2 <= B) parts *= 2;
  const int run = (B + parts - 1) / parts;
  if (tid < parts * E) {
    const int e = tid % E, part = tid / E;
    const int b_lo = part * run, b_hi = min(B, b_lo + run);
    float s = 0.f;
#pragma unroll 4
    for (int b = b_lo; b < b_hi; ++b) s = fmaf(w_s[b], ell[(size_t)b * E + e], s);
    gpart_s[part * E + e] = s;
  }
  __syncthreads();
  if (tid < E) {
    float s = gpart_s[tid];
    for (int part = 1; part < parts; ++part) s += gpart_s[part * E + tid];
    a.g[tid] = s;
    gm_s[tid] = s;
  }
  __syncthreads();

  // E* = TopCap(g): the cap candidates of largest g (ties: lower id), by one
  // wave; all candidates when there are at most cap.
  if (wave == 0) {
    uint32_t key[1][kNJ];
    int n_cand = 0;
#pragma unroll
    for (int j = 0; j < kNJ; ++j) {
      const int e = lane + kWave * j;
      key[0][j] = e < E && cand_s[e] ? order_key(gm_s[e]) : 0u;
      n_cand += __popcll(__ballot(key[0][j] != 0u));
    }
    uint32_t pref_bits = 0;
    if (active) {
      if (n_cand <= a.cap) {
#pragma unroll
        for (int j = 0; j < kNJ; ++j)
          if (key[0][j] != 0u) pref_bits |= 1u << j;
      } else {
        uint32_t sel[1];
        wave_top_k<1, kNJ>(key, a.cap, sel);
        pref_bits = sel[0];
      }
    }
#pragma unroll
    for (int j = 0; j < kNJ; ++j) {
      const int e = lane + kWave * j;
      if (e < E) {
        const int p = (pref_bits >> j) & 1u;
        pref_s[e] = p;
        a.pref[e] = p;
      }
    }
  }
  __syncthreads();

  // Per token: lambda_b, biased keys, biased top-k, gate weights, masks.
  // Wave w takes tokens w, w + 16, ...; kNT of them at a time.
  const bool from_biased = (a.flags & kGateFromBiased) != 0;
  for (int b0 = wave; b0 < B; b0 += n_waves * kNT) {
    float l[kNT][kNJ], lb[kNT][kNJ];
    uint32_t key[kNT][kNJ];
#pragma unroll
    for (int t = 0; t < kNT; ++t) {
      const int b = b0 + t * n_waves;
      float lam = 0.f;
      if (active && b < B) lam = (a.flags & kBiasAbsolute) ? a.alpha : a.alpha * gap_s[b];
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        const int e = lane + kWave * j;
        l[t][j] = 0.f;
        lb[t][j] = 0.f;
        key[t][j] = 0;
        if (b < B && e < E) {
          l[t][j] = ell[(size_t)b * E + e];
          lb[t][j] = pref_s[e] ? l[t][j] + lam : l[t][j];
          key[t][j] = order_key(lb[t][j]);
        }
      }
    }
    uint32_t bits[kNT];
    wave_top_k<kNT, kNJ>(key, k, bits);
    // Softmax over the selected k: max through the order keys (exact),
    // then exp, a DPP sum and one reciprocal.
    float ez[kNT][kNJ], s[kNT], inv_s[kNT];
#pragma unroll
    for (int t = 0; t < kNT; ++t) {
      uint32_t mk = 0;
#pragma unroll
      for (int j = 0; j < kNJ; ++j)
        if ((bits[t] >> j) & 1u) mk = max(mk, from_biased ? key[t][j] : order_key(l[t][j]));
      const float m = key_value(wave_max_key_dpp(mk));
      s[t] = 0.f;
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        // exp(x - m) as 2^((x - m) log2 e) on the hardware exp2 (about 1e-6
        // relative error for |x - m| < 20)
        const float x = from_biased ? lb[t][j] : l[t][j];
        ez[t][j] = ((bits[t] >> j) & 1u) ? __builtin_amdgcn_exp2f((x - m) * kLog2e) : 0.f;
        s[t] += ez[t][j];
      }
    }
#pragma unroll
    for (int t = 0; t < kNT; ++t) inv_s[t] = __builtin_amdgcn_rcpf(wave_sum_dpp(s[t]));
#pragma unroll
    for (int t = 0; t < kNT; ++t) {
      const int b = b0 + t * n_waves;
      if (b >= B) break;
      int rank[kNJ];
      wave_rank_flagged<kNJ>(bits[t], rank);
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        if ((bits[t] >> j) & 1u) {
          const int pos = b * k + rank[j];
          const int e = lane + kWave * j;
          a.idx[pos] = e;
          a.gate_w[pos] = ez[t][j] * inv_s[t];
          idx_s[pos] = (uint8_t)e;
          atomicOr(reinterpret_cast<unsigned long long*>(&mask_s[e][b >> 6]),
                   1ull << (b & 63));
        }
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
    const int incl_c = wave_inclusive_scan_dpp(sum_c);
    const int incl_f = wave_inclusive_scan_dpp(sum_f);
    const int total_c = __builtin_amdgcn_readlane(incl_c, 63);
    const int total_f = __builtin_amdgcn_readlane(incl_f, 63);
    int run_c = incl_c - sum_c, run_f = incl_f - sum_f;
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
  // the assignments of e by tokens b' < b.  Every idx_s entry was written
  // above with an id below E, and offset_s[e] + before < B k for each of
  // them, so the two clamps below never change a result the kernel computes.
  // They are defence only: they keep the addressing inside offset_s and slot
  // should that invariant ever be broken by a change to this kernel.
  for (int i = tid; i < B * k; i += blockDim.x) {
    const int b = i / k;
    const int e = min((int)idx_s[i], E - 1);
    int before = 0;
#pragma unroll
    for (int w = 0; w < kMaskWords; ++w) {
      const uint64_t m = mask_s[e][w];
      if (w < (b >> 6)) before += __popcll(m);
      else if (w == (b >> 6)) before += __popcll(m & ((1ull << (b & 63)) - 1ull));
    }
    a.slot[min(offset_s[e] + before, B * k - 1)] = i;
  }
}

// Small batches without a bias that can change the selection (alpha = 0,
// or a single token): one wave (small_gate) computes g and E* as the kernel
// above does, takes the plain top-k, forms the gate weights with the same
// arithmetic and buckets the B k <= 64 assignments, with no workgroup
// barriers between the phases.
template <int kNJ>
__global__ __launch_bounds__(kWave) void reuse_gate_small_kernel(GateArgs a) {
  __shared__ SmallGateLds s;
  small_gate<kNJ>(a, a.plain_idx, a.gap, s, true);
}

// The same, ranking the tokens' logits first (small_route_gate): the
// routing launch's ranking and this gating in one single-wave launch.
template <int kNJ>
__global__ __launch_bounds__(kWave) void route_gate_small_kernel(RouteArgs ra, GateArgs a) {
  __shared__ SmallGateLds s;
  small_route_gate<kNJ>(ra, a, s, true);
}

template <bool kStaged, int kNJ, bool kSelect>
void launch_gate_nj(const GateArgs& a, const RouteArgs& ra, hipStream_t s) {
  if (a.B <= 16)
    hipLaunchKernelGGL((reuse_gate_kernel<kStaged, kNJ, 1, kSelect>), dim3(1), dim3(1024), 0, s, a, ra);
  else if (a.B <= 32)
    hipLaunchKernelGGL((reuse_gate_kernel<kStaged, kNJ, 2, kSelect>), dim3(1), dim3(1024), 0, s, a, ra);
  else
    hipLaunchKernelGGL((reuse_gate_kernel<kStaged, kNJ, 4, kSelect>), dim3(1), dim3(1024), 0, s, a, ra);
}

template <bool kStaged, bool kSelect>
void launch_gate_staged(const GateArgs& a, const RouteArgs& ra, hipStream_t s) {
  if (a.E <= 64)
    launch_gate_nj<kStaged, 1, kSelect>(a, ra, s);
  else if (a.E <= 128)
    launch_gate_nj<kStaged, 2, kSelect>(a, ra, s);
  else
    launch_gate_nj<kStaged, 4, kSelect>(a, ra, s);
}

bool small_gate_applies(const GateArgs& a) {
  return a.B <= kSmallMaxTokens && (a.alpha == 0.f || a.B == 1);
}

hipError_t launch_reuse_gate(const GateArgs& a, hipStream_t s) {
  if (small_gate_applies(a)) {
    if (a.E <= 64)
      hipLaunchKernelGGL(reuse_gate_small_kernel<1>, dim3(1), dim3(kWave), 0, s, a);
    else if (a.E <= 128)
      hipLaunchKernelGGL(reuse_gate_small_kernel<2>, dim3(1), dim3(kWave), 0, s, a);
    else
      hipLaunchKernelGGL(reuse_gate_small_kernel<4>, dim3(1), dim3(kWave), 0, s, a);
    return hipGetLastError();
  }
  const RouteArgs none{};
  if (a.B * a.E <= kStage)
    launch_gate_staged<true, false>(a, none, s);
  else
    launch_gate_staged<false, false>(a, none, s);
  return hipGetLastError();
}

// The workgroup gating kernel ranks the tokens itself when each of its 16
// waves has at most one token to rank (measured on MI355X: 3.6 us saved at
// 4 tokens, 0.8 us lost at 32, where the routing launch ranks the tokens on
// 32 compute units at once).
constexpr int kGateSelectMaxTokens = 16;

hipError_t launch_route_and_gate(const RouteArgs& ra, const GateArgs& a, hipStream_t s) {
  if (!route_ranks_separately(ra) ||
      (!small_gate_applies(a) && (a.B * a.E > kStage || a.B > kGateSelectMaxTokens))) {
    const hipError_t err = launch_route(ra, s);
    return err != hipSuccess ? err : launch_reuse_gate(a, s);
  }
  const hipError_t err = launch_route_rows(ra, s);
  if (err != hipSuccess) return err;
  if (small_gate_applies(a)) {
    if (a.E <= 64)
      hipLaunchKernelGGL(route_gate_small_kernel<1>, dim3(1), dim3(kWave), 0, s, ra, a);
    else if (a.E <= 128)
      hipLaunchKernelGGL(route_gate_small_kernel<2>, dim3(1), dim3(kWave), 0, s, ra, a);
    else
      hipLaunchKernelGGL(route_gate_small_kernel<4>, dim3(1), dim3(kWave), 0, s, ra, a);
  } else {
    launch_gate_staged<true, true>(a, ra, s);
  }
  return hipGetLastError();
}

}  // namespace s2moe
