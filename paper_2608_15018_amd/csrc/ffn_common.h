// Work decomposition shared by the expert-FFN kernels.
#pragma once

#include "common.h"
#include "kernels.h"

namespace s2moe {
namespace ffn {

struct Segment {
  int n;      // tokens
  int base;   // routed: offset[e] (row of its first token in Hh); shared: B*k + s*B
  int id;     // expert e or shared expert s
  bool shared;
};

// Grid layout: shared-expert blocks first (always live), then routed blocks
// u-major (u = position in uniq), so blocks of inactive experts come last
// and exit at once.
__device__ __forceinline__ bool resolve_block(const FfnArgs& a, int mode, int rows_per_block,
                                              Segment* seg, int* rb) {
  const int rows_r = mode == 0 ? a.F : a.H;
  const int rows_s = mode == 0 ? a.Fs : a.H;
  const int nbs = a.S > 0 ? rows_s / rows_per_block : 0;
  const int nbr = rows_r / rows_per_block;
  int bid = blockIdx.x;
  if (bid < a.S * nbs) {
    seg->shared = true;
    seg->id = bid / nbs;
    *rb = bid % nbs;
    seg->n = a.B;
    seg->base = a.B * a.k + seg->id * a.B;
    return true;
  }
  bid -= a.S * nbs;
  const int u = bid / nbr;
  *rb = bid % nbr;
  if (u >= min(*a.n_uniq, min(a.E, a.B * a.k))) return false;
  // The routing arrays come from the gating step; values outside their
  // ranges (routing never computed) make the block idle instead of faulting.
  const int e = a.uniq[u];
  if (e < 0 || e >= a.E) return false;
  seg->shared = false;
  seg->id = e;
  seg->n = a.count[e];
  seg->base = a.offset[e];
  return seg->n > 0 && seg->base >= 0 && seg->base + seg->n <= a.B * a.k;
}

__device__ __forceinline__ int slot_at(const FfnArgs& a, int i) {
  const int v = a.slot[i];
  return min(max(v, 0), a.B * a.k - 1);
}

// Row of the X source feeding token t of the segment: x for gate-up
// (gathered through slot), the segment's own Hh rows for down.
__device__ __forceinline__ int x_row(const FfnArgs& a, int mode, const Segment& s, int t) {
  if (mode == 0) return s.shared ? t : slot_at(a, s.base + t) / a.k;
  return s.base + t;
}

// Row of expert_out written for token t (down only).
__device__ __forceinline__ int out_row(const FfnArgs& a, const Segment& s, int t) {
  return s.shared ? s.base + t : slot_at(a, s.base + t);
}

__device__ __forceinline__ float silu(float z) { return z / (1.f + expf(-z)); }

// MFMA helpers.
__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  bf16x8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// Streams n >= 1 stages: stage i + 1 is requested before stage i is
// consumed, with two register buffers.  Every load sits on a path without
// conditions of its own (a two-stage loop body, then a one- or two-stage
// tail), so the compiler knows how many loads are in flight at each use and
// waits only for the stage it needs; a load under a condition would make it
// wait for all of them.
// The scheduling barriers keep the compiler from sinking the next stage's
// loads into the current stage's arithmetic.
#ifndef S2MOE_PIPE_BARRIER
#define S2MOE_PIPE_BARRIER 1
#endif
__device__ __forceinline__ void pipe_barrier() {
  if (S2MOE_PIPE_BARRIER) __builtin_amdgcn_sched_barrier(0);
}

template <class Stage, class Load, class Use>
__device__ __forceinline__ void pipeline2(int n, Load&& load, Use&& use) {
  Stage a, b;
  load(a, 0);
  int i = 0;
  for (; i + 2 < n; i += 2) {
    load(b, i + 1);
    pipe_barrier();
    use(a, i);
    load(a, i + 2);
    pipe_barrier();
    use(b, i + 1);
  }
  if (i + 1 < n) {
    load(b, i + 1);
    pipe_barrier();
    use(a, i);
    use(b, i + 1);
  } else {
    use(a, i);
  }
}

// Number of blocks of `rows_per_block` rows a launch covers: the shared
// experts, then one slot per possibly activated expert.  A batch activates
// at most min(E, B k) routed experts, so small batches (a draft step) do not
// launch blocks for experts that cannot be in uniq.
inline int n_blocks(const FfnArgs& a, int mode, int rows_per_block) {
  const int rows_r = mode == 0 ? a.F : a.H;
  const int rows_s = mode == 0 ? a.Fs : a.H;
  const int slots = a.E < a.B * a.k ? a.E : a.B * a.k;
  return (a.S > 0 ? a.S * (rows_s / rows_per_block) : 0) + slots * (rows_r / rows_per_block);
}

}  // namespace ffn
}  // namespace s2moe
