// Pieces of the fused small-batch MoE layer shared by the bf16 and int4
// expert kernels: a layer of B <= kSmallMaxTokens tokens whose gating keeps
// the plain top-k runs as three launches (router rows; gate-up with the
// routing in its prologue; down with the combine), with the same results
// bit for bit as the routing, gating, expert and combine launches.
#pragma once

#include "ffn_common.h"
#include "small_batch.h"

namespace s2moe {
namespace ffn {

// Rows of expert_out a small batch can have: B k + S B.
constexpr int kSmallOutRows = kSmallMaxTokens * kMaxTopK + kMaxShared * kSmallMaxTokens;

// Gate-up prologue, run by wave 0: rank each token's logits (the routing
// kernel's code) and bucket the B k assignments in registers (lane_buckets),
// leaving count, offset, uniq, n_uniq and slot in s for the activated
// experts.  In the publishing workgroup, run the single-wave gating instead
// (g, E*, gate weights, buckets) and write every routing output to global
// memory.  The caller synchronises the workgroup afterwards.
template <int NJ>
__device__ __forceinline__ void small_layer_routing(const RouteArgs& ra, const GateArgs& ga,
                                                    SmallGateLds& s, bool pub) {
  small_route_gate<NJ>(ra, ga, s, pub);
  if (pub) return;
  const int lane = threadIdx.x & (kWave - 1), n = ga.B * ga.k;
  const int e = lane < n ? s.plain[lane] : 0;
  const LaneBuckets lb = lane_buckets(e, n);
  if (lane < n) s.slot[lb.less + lb.before] = lane;
  if (lb.first) {
    s.uniq[lb.distinct_less] = e;
    s.count[e] = lb.count;
    s.offset[e] = lb.less;
  }
  const int nu = __popcll(__ballot(lb.first));
  if (lane == 0) s.n_uniq = nu;
}

// a with its bucket pointers on the LDS buckets of small_layer_routing.
__device__ __forceinline__ FfnArgs with_lds_buckets(const FfnArgs& a, SmallGateLds& s) {
  FfnArgs b = a;
  b.count = s.count;
  b.offset = s.offset;
  b.slot = s.slot;
  b.uniq = s.uniq;
  b.n_uniq = &s.n_uniq;
  return b;
}

// LDS of the fused down launch: partial tiles of every wave, the
// workgroup's columns of expert_out, the gate weights.
template <int R>
struct SmallDownLds {
  f32x4 red[16 * R * kWave];
  float eo[kSmallOutRows][16 * R];
  float gw[kWave];
};

// Segment of wave w = seg_i * KW + part in the fused down launch: the
// shared experts first, then the activated experts in ascending id, found
// by bucketing the published top-k (idx, one id per lane) in registers.  Ids
// outside [0, E) (routing never computed) are clamped.  Wave 0 also stages
// the gate weights in LDS.  members: the segment's assignments (lanes).
template <int R>
__device__ __forceinline__ bool small_down_segment(const FfnArgs& a, const int32_t* idx,
                                                   const float* gate_w, int seg_i,
                                                   SmallDownLds<R>& s, Segment* seg,
                                                   uint64_t* members) {
  const int lane = threadIdx.x & (kWave - 1);
  const int n_asg = a.B * a.k;
  const int e_l = lane < n_asg ? min(max(idx[lane], 0), a.E - 1) : 0;
  const float gw_l = lane < n_asg ? gate_w[lane] : 0.f;
  if (wave_id() == 0) s.gw[lane] = gw_l;
  *members = 0;
  if (seg_i < a.S) {
    seg->shared = true;
    seg->id = seg_i;
    seg->n = a.B;
    seg->base = n_asg + seg_i * a.B;
    return true;
  }
  const LaneBuckets lb = lane_buckets(e_l, n_asg);
  int e = 0, cnt = 0, off = 0;
  if (!lane_bucket_segment(e_l, n_asg, lb, seg_i - a.S, &e, &cnt, &off, members)) return false;
  seg->shared = false;
  seg->id = e;
  seg->n = cnt;
  seg->base = off;
  return true;
}

// After each wave's partial tile acc (its segment, its K part): the K parts
// are added in part order by the part-0 wave as the down kernels do with KW
// waves, the tile goes to expert_out and to LDS, and the workgroup forms y
// for its 16 R rows from r0 with the combine kernel's arithmetic (the k
// routed terms as fmaf in slot order, then the shared terms).  Every wave of
// the workgroup calls it.
template <int R, int KW>
__device__ __forceinline__ void small_down_finish(const FfnArgs& a, const Segment& seg,
                                                  bool live, int part, uint64_t members,
                                                  f32x4 (&acc)[1][R][1], SmallDownLds<R>& s,
                                                  float* y, int r0) {
  constexpr int kRows = 16 * R;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
  const int rA = lane & 15, gK = lane >> 4;
  if (KW > 1) {
#pragma unroll
    for (int r = 0; r < R; ++r) s.red[(wave * R + r) * kWave + lane] = acc[0][r][0];
  }
  __syncthreads();
  if (live && part == 0) {
    for (int w = 1; w < KW; ++w) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const f32x4 p = s.red[((wave + w) * R + r) * kWave + lane];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[0][r][0][i] += p[i];
      }
    }
    if (rA < seg.n) {
      const int row = seg.shared ? seg.base + rA : nth_set_bit(members, rA);
      float* dst = a.out + (size_t)row * a.H;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        *reinterpret_cast<f32x4*>(dst + r0 + 16 * r + 4 * gK) = acc[0][r][0];
#pragma unroll
        for (int i = 0; i < 4; ++i) s.eo[row][16 * r + 4 * gK + i] = acc[0][r][0][i];
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < a.B * kRows; i += blockDim.x) {
    const int b = i / kRows, c = i - b * kRows;
    float v = 0.f;
    for (int j = 0; j < a.k; ++j) v = fmaf(s.gw[b * a.k + j], s.eo[b * a.k + j][c], v);
    for (int sh = 0; sh < a.S; ++sh) v += s.eo[a.B * a.k + sh * a.B + b][c];
    y[(size_t)b * a.H + r0 + c] = v;
  }
}

}  // namespace ffn
}  // namespace s2moe
