// One-wave routing of small batches: the plain top-k ranking of one token
// (Sec. "Reuse-aware Expert Gating": ell_b, its top-k and gap_b =
// ell_(1) - ell_(k+1)) and the gating of a batch whose reuse bias cannot
// move any selection.  The standalone routing and gating kernels and the
// fused small-batch MoE-layer kernels all call these functions, so every
// path computes the same bits.
#pragma once

#include "kernels.h"
#include "select.h"

namespace s2moe {

constexpr float kLog2e = 1.4426950408889634f;

// Dot product of one 16-byte chunk of a token row and of a router row.
template <bool kBf16>
__device__ __forceinline__ float dot_chunk(u32x4 xc, u32x4 wc, float acc) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (kBf16) {
      acc = fmaf(bf16_to_f32(wc[i] & 0xFFFFu), bf16_to_f32(xc[i] & 0xFFFFu), acc);
      acc = fmaf(bf16_to_f32(wc[i] >> 16), bf16_to_f32(xc[i] >> 16), acc);
    } else {
      acc = fmaf(__uint_as_float(wc[i]), __uint_as_float(xc[i]), acc);
    }
  }
  return acc;
}

// Logit e of token b by one wave (e >= E: nothing): lanes take 16-byte
// chunks of H, a DPP reduction adds them, lane 0 writes a.logits[b][e].
template <bool kBf16>
__device__ __forceinline__ void route_row_logit(const RouteArgs& a, int e, int b) {
  const int lane = threadIdx.x & (kWave - 1);
  if (e >= a.E) return;
  const size_t row = (size_t)a.H * (kBf16 ? 2 : 4);
  const u32x4* wr = reinterpret_cast<const u32x4*>(static_cast<const char*>(a.router) + e * row);
  const u32x4* xr = reinterpret_cast<const u32x4*>(static_cast<const char*>(a.x) + b * row);
  const int chunks = a.H / (kBf16 ? 8 : 4);
  float acc = 0.f;
#pragma unroll 4
  for (int c = lane; c < chunks; c += kWave) acc = dot_chunk<kBf16>(xr[c], wr[c], acc);
  acc = wave_sum_dpp(acc);
  if (lane == 0) a.logits[(size_t)b * a.E + e] = acc;
}

// Orders the LDS and global accesses of one wave before and after it (the
// functions below run on a single wave, also inside larger workgroups whose
// other waves are not there to meet a workgroup barrier).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_wave_barrier();
}

// Plain top-k and gap of one token by one wave, from its E logits `ell`
// (LDS or global): the exact top-(k+1) by (value desc, id asc); its last
// member (smallest value, then largest id) is the (k+1)-th, the other k are
// the plain top-k, written in id order to idx[0..k); gap = ell_(1) -
// ell_(k+1) to *gap.  idx2 / gap2, when not null, get the same values.
template <int NJ, class I1, class I2>
__device__ __forceinline__ void wave_select_plain(int E, int k, const float* ell, I1* idx,
                                                  float* gap, I2* idx2, float* gap2) {
  const int lane = threadIdx.x & (kWave - 1);
  uint32_t key[1][NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int e = lane + kWave * j;
    key[0][j] = e < E ? order_key(ell[e]) : 0u;
  }
  uint32_t sel[1];
  wave_top_k<1, NJ>(key, k + 1, sel);
  uint32_t mn = 0xFFFFFFFFu, mx = 0u;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if ((sel[0] >> j) & 1u) mn = min(mn, key[0][j]);
    mx = max(mx, key[0][j]);
  }
  mn = ~wave_max_key_dpp(~mn);
  mx = wave_max_key_dpp(mx);
  int last = -1;
#pragma unroll
  for (int j = NJ - 1; j >= 0; --j) {
    const uint64_t m = __ballot(((sel[0] >> j) & 1u) && key[0][j] == mn);
    if (last < 0 && m) last = kWave * j + 63 - __builtin_clzll(m);
  }
  uint32_t bits = 0;
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (((sel[0] >> j) & 1u) && lane + kWave * j != last) bits |= 1u << j;
  int rank[NJ];
  wave_rank_flagged<NJ>(bits, rank);
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if ((bits >> j) & 1u) {
      idx[rank[j]] = (I1)(lane + kWave * j);
      if (idx2) idx2[rank[j]] = (I2)(lane + kWave * j);
    }
  if (lane == 0) {
    const float gv = key_value(mx) - key_value(mn);
    *gap = gv;
    if (gap2) *gap2 = gv;
  }
}

// LDS of the one-wave gating: its working arrays, and the bucketing every
// caller of small_gate may read afterwards (count, offset, uniq, n_uniq,
// slot: the same values the function publishes to global memory).
struct SmallGateLds {
  int count[kMaxExperts];
  int offset[kMaxExperts + 1];
  int cand[kMaxExperts];
  int idx[kWave];    // plain top-k of the batch, [B k]
  int uniq[kWave];   // activated experts in ascending id (n_uniq <= B k <= 64)
  int slot[kWave];   // assignments grouped by expert
  int plain[kWave];  // plain top-k handed over by a fused caller
  float gap[kSmallMaxTokens];
  int n_uniq;
};

// Gating of B <= kSmallMaxTokens tokens whose biased top-k is the plain
// one: alpha = 0 (then ell' = ell), or a single token (its top-k lies inside
// E* = TopCap(w ell) whatever the flags, and every member of E* gets the
// same lambda).  One wave computes g and E* as the workgroup gating kernel
// does (same runs of tokens, same ranking order), takes the plain top-k
// (`plain` [B k], `gap_in` [B]: global or LDS), forms the gate weights with
// the same arithmetic and buckets the B k assignments.  publish: also
// compute g, E* and the gate weights and write every output of the gating
// step to a's global arrays; without it only the bucketing is computed (it
// is always left in s).
template <int kNJ>
__device__ __forceinline__ void small_gate(const GateArgs& a, const int32_t* plain,
                                           const float* gap_in, SmallGateLds& s, bool publish) {
  const int lane = threadIdx.x & (kWave - 1);
  const int B = a.B, E = a.E, k = a.k, n_asg = B * k;

  // Every global read is issued up front: confidences, gaps and all B x E
  // logits (at most 4 x 4 per lane; only g, E* and the gate weights need
  // them), and the plain top-k.
  float w[kSmallMaxTokens], gap[kSmallMaxTokens], lg[kSmallMaxTokens][kNJ];
  int active = 0;
#pragma unroll
  for (int b = 0; b < kSmallMaxTokens; ++b) {
    const bool use = publish && b < B;
    w[b] = use ? fmaxf(a.conf_w[b], 0.f) : 0.f;
    gap[b] = use ? gap_in[b] : 0.f;
#pragma unroll
    for (int j = 0; j < kNJ; ++j) {
      const int e = lane + kWave * j;
      lg[b][j] = use && e < E ? a.logits[(size_t)b * E + e] : 0.f;
    }
    active |= w[b] > 0.f;
  }
  const int pidx = lane < n_asg ? plain[lane] : 0;
  const bool activated_only = (a.flags & kPrefActivatedOnly) != 0;
#pragma unroll
  for (int j = 0; j < kMaxExperts / kWave; ++j) {
    const int e = lane + kWave * j;
    s.count[e] = 0;
    s.cand[e] = !activated_only && e < E;
  }
  // Ids outside [0, E) (plain_idx never computed) are clamped, so that
  // nothing is addressed out of range.
  int my_e = 0;
  if (lane < n_asg) {
    my_e = min(max(pidx, 0), E - 1);
    s.idx[lane] = my_e;
  }
  wave_sync();
  if (lane < n_asg) {
    if (activated_only) s.cand[my_e] = 1;
    atomicAdd(&s.count[my_e], 1);
  }
  wave_sync();

  // g_e in the same runs of tokens as the workgroup kernel, and E* (only
  // the published outputs and the gate weights need them).
  uint32_t pref_bits = 0;
  if (publish) {
    int parts = 1;
    while (parts * 2 * E <= 1024 && parts * 2 <= B) parts *= 2;
    const int run = (B + parts - 1) / parts;
    uint32_t key[1][kNJ];
    int n_cand = 0;
#pragma unroll
    for (int j = 0; j < kNJ; ++j) {
      const int e = lane + kWave * j;
      key[0][j] = 0;
      if (e < E) {
        float tot = 0.f;
        for (int part = 0; part < parts; ++part) {
          float sum = 0.f;
#pragma unroll
          for (int b = 0; b < kSmallMaxTokens; ++b)
            if (b >= part * run && b < min(B, part * run + run)) sum = fmaf(w[b], lg[b][j], sum);
          tot = part == 0 ? sum : tot + sum;
        }
        a.g[e] = tot;
        if (s.cand[e]) key[0][j] = order_key(tot);
      }
      n_cand += __popcll(__ballot(e < E && s.cand[e]));
    }
    // E* = the cap candidates of largest g (ties: lower id).
    if (active) {
      if (n_cand <= a.cap) {
#pragma unroll
        for (int j = 0; j < kNJ; ++j)
          if (key[0][j] != 0) pref_bits |= 1u << j;
      } else {
        uint32_t sel[1];
        wave_top_k<1, kNJ>(key, a.cap, sel);
        pref_bits = sel[0];
      }
    }
#pragma unroll
    for (int j = 0; j < kNJ; ++j) {
      const int e = lane + kWave * j;
      if (e < E) a.pref[e] = (pref_bits >> j) & 1u;
    }
  }

  // Per token: the plain top-k and its gate weights.
  if (publish) {
    const bool from_biased = (a.flags & kGateFromBiased) != 0;
#pragma unroll
    for (int b = 0; b < kSmallMaxTokens; ++b) {
      if (b >= B) break;
      const float lam = active ? ((a.flags & kBiasAbsolute) ? a.alpha : a.alpha * gap[b]) : 0.f;
      uint32_t bits = 0;
      float x[kNJ];
#pragma unroll
      for (int j = 0; j < kNJ; ++j)
        x[j] = from_biased && ((pref_bits >> j) & 1u) ? lg[b][j] + lam : lg[b][j];
      for (int q = 0; q < k; ++q) {
        const int e = s.idx[b * k + q];
        if ((e & (kWave - 1)) == lane) bits |= 1u << (e / kWave);
      }
      uint32_t mk = 0;
#pragma unroll
      for (int j = 0; j < kNJ; ++j)
        if ((bits >> j) & 1u) mk = max(mk, order_key(x[j]));
      const float m = key_value(wave_max_key_dpp(mk));
      float ez[kNJ], sum = 0.f;
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        ez[j] = ((bits >> j) & 1u) ? __builtin_amdgcn_exp2f((x[j] - m) * kLog2e) : 0.f;
        sum += ez[j];
      }
      const float inv_s = __builtin_amdgcn_rcpf(wave_sum_dpp(sum));
      int rank[kNJ];
      wave_rank_flagged<kNJ>(bits, rank);
#pragma unroll
      for (int j = 0; j < kNJ; ++j)
        if ((bits >> j) & 1u) {
          const int pos = b * k + rank[j];
          a.idx[pos] = lane + kWave * j;
          a.gate_w[pos] = ez[j] * inv_s;
        }
    }
  }

  // Buckets: counts, exclusive offsets, the activated-expert list, slots.
  {
    int c[4], f[4], sum_c = 0, sum_f = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane * 4 + j;
      c[j] = e < E ? s.count[e] : 0;
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
        s.offset[e] = run_c;
        if (publish) {
          a.offset[e] = run_c;
          a.count[e] = c[j];
        }
        if (f[j]) {
          s.uniq[run_f] = e;
          if (publish) a.uniq[run_f] = e;
        }
      }
      run_c += c[j];
      run_f += f[j];
    }
    if (publish)
      for (int i = total_f + lane; i < E; i += kWave) a.uniq[i] = -1;
    if (lane == 0) {
      s.offset[E] = total_c;
      s.n_uniq = total_f;
      if (publish) {
        a.offset[E] = total_c;
        *a.n_uniq = total_f;
      }
    }
  }
  wave_sync();
  if (lane < n_asg) {
    int before = 0;
    for (int q = 0; q < lane; ++q) before += s.idx[q] == my_e;
    s.slot[s.offset[my_e] + before] = lane;
    if (publish) a.slot[s.offset[my_e] + before] = lane;
  }
}

// Plain top-k and gap of each of the B <= kSmallMaxTokens tokens
// (wave_select_plain on the logits ra.logits) into s.plain / s.gap, and,
// when publish, to ra.plain_idx / ra.gap; then, when publish, small_gate on
// them (g, E*, gate weights, buckets, all written to ga's arrays).  One
// wave; the results equal the routing kernel's ranking followed by the
// single-wave gating kernel.
template <int NJ>
__device__ __forceinline__ void small_route_gate(const RouteArgs& ra, const GateArgs& ga,
                                                 SmallGateLds& s, bool publish) {
  for (int b = 0; b < ga.B; ++b)
    wave_select_plain<NJ>(ra.E, ra.k, ra.logits + (size_t)b * ra.E, s.plain + b * ra.k,
                          s.gap + b, publish ? ra.plain_idx + (size_t)b * ra.k : nullptr,
                          publish ? ra.gap + b : nullptr);
  wave_sync();
  if (publish) small_gate<NJ>(ga, s.plain, s.gap, s, true);
}

// Buckets of n <= 64 assignments held one per lane (lane i < n holds the
// expert e_i of assignment i), computed in registers by uniform loops over
// the n lanes: the same bucketing as small_gate (experts in ascending id,
// each expert's assignments in assignment order).
struct LaneBuckets {
  int less;           // assignments to experts below e_i: offset[e_i]
  int before;         // earlier assignments to e_i: slot[less + before] = i
  int count;          // assignments to e_i: count[e_i]
  int distinct_less;  // activated experts below e_i: e_i = uniq[distinct_less]
  bool first;         // i is e_i's first assignment
};

__device__ __forceinline__ LaneBuckets lane_buckets(int e, int n) {
  const int lane = threadIdx.x & (kWave - 1);
  LaneBuckets b{0, 0, 0, 0, false};
  for (int j = 0; j < n; ++j) {
    const int ej = __builtin_amdgcn_readlane(e, j);
    b.less += ej < e;
    b.count += ej == e;
    b.before += ej == e && j < lane;
  }
  b.first = lane < n && b.before == 0;
  uint64_t m = __ballot(b.first);
  while (m) {
    const int j = __builtin_ctzll(m);
    m &= m - 1;
    b.distinct_less += __builtin_amdgcn_readlane(e, j) < e;
  }
  return b;
}

// Segment u of the buckets (the u-th activated expert in ascending id):
// false when fewer experts are activated; else its expert, assignment count
// and offset, and the mask of its assignments (lanes), in order.
__device__ __forceinline__ bool lane_bucket_segment(int e, int n, const LaneBuckets& b, int u,
                                                    int* e_u, int* count, int* offset,
                                                    uint64_t* members) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t m = __ballot(b.first && b.distinct_less == u);
  if (m == 0) return false;
  const int l = __builtin_ctzll(m);
  *e_u = __builtin_amdgcn_readlane(e, l);
  *count = __builtin_amdgcn_readlane(b.count, l);
  *offset = __builtin_amdgcn_readlane(b.less, l);
  *members = __ballot(lane < n && e == *e_u);
  return true;
}

// Index of the t-th set bit of m (t < popcount(m)).
__device__ __forceinline__ int nth_set_bit(uint64_t m, int t) {
  for (int i = 0; i < t; ++i) m &= m - 1;
  return __builtin_ctzll(m);
}

}  // namespace s2moe
