// Internal launch interface between the C-ABI layer (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace s2moe {

constexpr int kMaxTopK = 16;
constexpr int kMaxTokens = 256;
constexpr int kMaxExperts = 256;
constexpr int kMaxShared = 8;  // S2MOE_MAX_SHARED

enum : uint32_t {
  kPrefActivatedOnly = 1u,
  kBiasAbsolute = 2u,
  kGateFromBiased = 4u,
  kPackedWeights = 8u
};
enum WeightFormat : int { kWF32 = 0, kWBf16 = 1, kWQ4 = 2 };

struct RouteArgs {
  const void* x;
  const void* router;
  float* logits;
  int32_t* plain_idx;
  float* gap;
  int B, H, E, k;
  bool bf16;
  // When set (bf16 x, one-call layer with int4 weights): the routing launch
  // also converts x to the int4 path's fp16 copy, n8 8-blocks, in
  // workgroups of its own.
  uint16_t* x16;
  int n8;
};

struct GateArgs {
  const float* logits;
  const float* gap;
  const int32_t* plain_idx;
  const float* conf_w;
  float* g;
  int32_t* pref;
  int32_t* idx;
  float* gate_w;
  int32_t* count;
  int32_t* offset;
  int32_t* slot;
  int32_t* uniq;
  int32_t* n_uniq;
  int B, E, k, cap;
  float alpha;
  uint32_t flags;
};

// Everything the grouped expert FFN needs.  Routed experts use count /
// offset / slot / uniq / n_uniq produced by the gating step; shared experts
// take all B tokens.
struct FfnArgs {
  int B, k, S, E;
  int H, F, Fs;
  int wf;  // WeightFormat
  const int32_t* count;
  const int32_t* offset;
  const int32_t* slot;
  const int32_t* uniq;
  const int32_t* n_uniq;
  const void* x;  // [B, H], fp32 for kWF32 else bf16
  const void *gate, *up, *down;
  const void *gate_s, *up_s, *down_s;
  const void *sh_gate, *sh_up, *sh_down;
  const void *sh_gate_s, *sh_up_s, *sh_down_s;
  void* hh;  // workspace: SwiGLU activations [B*k + S*B, ldh] (fp32, bf16 or fp16)
  int ldh;
  void* x16;  // workspace, int4 weights only: x as fp16 [B, H] in the kernels' order
  float* part;  // workspace, int4 weights only: down partial sums of K parts 1..Q-1,
                // [Q - 1][B*k + S*B][H] fp32 (unused when Q == 1)
  int qparts;   // Q: K parts of the int4 down projection (q4_down_parts)
  bool x16_ready;     // int4: x16 already written (by the routing launch)
  bool defer_reduce;  // int4: leave the K parts' reduce to launch_q4_reduce_combine
  bool packed;  // weights in the packed tile order (pack.hip)
  float* out;  // [B*k + S*B, H]
};

// int4 expert FFN: rows of one down-projection work item (8 row tiles), and
// the number of K parts its reduction dimension is split into.  The parts
// give a launch at least 1024 work items (four per compute unit of a 256-CU
// GPU) when the batch activates so few experts that it would have fewer, up
// to 8 parts; each part spans at least one 128-wide K super-step, and the
// partial sums the parts add stay within 2 % of the down weights' bytes.  Measured
// on MI355X at 16 tokens over 8 experts of F = 14336: targets of 256, 512,
// 1024 and 2048 items gave FFN calls of 135, 125, 118 and 121 us; at 64
// tokens 183, 177, 177 and 184 us.  A bound of 2 % instead of 1 % gives 64
// tokens 3 parts instead of 2 (24 Mixtral-shaped layers: 160 against 165 us
// per layer) and 32 tokens 4 instead of 3.  Host-side: the workspace size
// depends on it.
#ifndef S2MOE_Q4_DOWN_R
#define S2MOE_Q4_DOWN_R 2  // row tiles per wave of a down item (4 waves)
#endif
constexpr int kQ4DownRows = 16 * S2MOE_Q4_DOWN_R * 4;
#ifndef S2MOE_Q4_DOWN_ITEMS
#define S2MOE_Q4_DOWN_ITEMS 1024
#endif

// Batches of at most this many tokens run the int4 FFN on the K-split
// kernel, whose down projection needs no K parts.
constexpr int kQ4KsplitMaxTokens = 8;

inline int q4_down_parts(int B, int k, int E, int H, int F, int S, int Fs) {
  if (B <= kQ4KsplitMaxTokens) return 1;
  const int slots = E < B * k ? E : B * k;
  const int items = (S + slots) * (H / kQ4DownRows);
  int q = (S2MOE_Q4_DOWN_ITEMS + items - 1) / items;
  int nss = F / 128;
  if (S > 0 && Fs / 128 < nss) nss = Fs / 128;
  if (q > 8) q = 8;
  if (q > nss) q = nss;
  // Each part beyond the first writes, and the reduce reads back, fp32 rows
  // of every token's outputs: at most 2 % of the down weights' bytes.
  const double part = (double)(B * k + S * B) * H * 4.0;
  const double down = ((double)slots * F + (double)S * Fs) * H * (0.5 + 2.0 / 32.0);
  const int q_bytes = 1 + (int)(0.02 * down / part);
  if (q > q_bytes) q = q_bytes;
  return q < 1 ? 1 : q;
}

struct CombineArgs {
  const float* gate_w;
  const float* expert_out;
  float* y;
  int B, H, k, S;
};

struct PackArgs {
  const void* src;
  const void* src_s;
  void* dst;
  void* dst_s;
  int n, rows, K;
  bool q4;
};

// Routing-aware adaptive expansion over T padded draft trees of N nodes.
struct ExpandArgs {
  const int32_t* parent;    // [T][N]
  const float* q;           // [T][N]
  const int32_t* eid;       // [T][N][L][k]
  const float* c_draft;     // [T][N]
  const int32_t* root_eid;  // [T][L][k] or nullptr
  const int32_t* n_nodes;   // [T]
  int32_t* order;           // [T][N]
  double* util;             // [T][N]
  int32_t* n_new;           // [T][N]
  int32_t* n_admit;         // [T]
  int32_t* n_pairs;         // [T]
  int32_t* status;          // [T]
  int T, N, L, E, k, max_admit;
  uint64_t k_div;  // ceil(2^42 / k): f / k == (f * k_div) >> 42 for f < 2^22, k <= 32
  double t_ar, t_exp;
};

// Byte offsets of the expansion kernel's LDS regions; host and device use
// the same function so the launch size and the carve-up agree.
struct ExpandLds {
  int ew;  // words of one layer's expert bitset, ceil(E / 32) rounded up to a power of two
  size_t ben, rows, uni, cdr, front, misc, state, total;
};

__host__ __device__ inline int expand_words(int E) {
  int w = 1;
  while (32 * w < E) w <<= 1;
  return w;
}

__host__ __device__ inline ExpandLds expand_lds(int N, int L, int E, int k) {
  (void)k;
  ExpandLds o;
  o.ew = expand_words(E);
  size_t off = 0;
  o.ben = off;    off += (size_t)N * 8;              // p_i, then B_i (double)
  off = (off + 15) & ~(size_t)15;
  o.rows = off;   off += (size_t)N * L * o.ew * 4;   // expert bitset per (node, layer)
  o.uni = off;    off += (size_t)L * o.ew * 4;       // union bitset per layer
  o.cdr = off;    off += (size_t)N * 4;              // C^draft
  o.front = off;  off += (size_t)N * 4;              // candidate list
  off = (off + 15) & ~(size_t)15;
  o.misc = off;   off += 128;                        // reductions and counters
  o.state = off;  off += (size_t)N;                  // per-node flags
  o.total = (off + 15) & ~(size_t)15;
  return o;
}

// Device address of the library's scratch array on the current device
// (S2MOE_NOALLOC_SCRATCH_BYTES bytes, 256-byte aligned).
hipError_t noalloc_scratch(void** ptr);

hipError_t launch_expand(const ExpandArgs& a, size_t lds_bytes, hipStream_t s);
hipError_t launch_route(const RouteArgs& a, hipStream_t s);
// Logits only (the first launch of launch_route's small-batch path).
hipError_t launch_route_rows(const RouteArgs& a, hipStream_t s);
// Whether launch_route computes the logits and ranks them in two launches
// (launch_route_rows, then one wave per token).
bool route_ranks_separately(const RouteArgs& a);
// launch_route then launch_reuse_gate, with the same results bit for bit;
// where the routing ranks in a launch of its own, the gating launch ranks
// the logits itself instead (gate.hip).
hipError_t launch_route_and_gate(const RouteArgs& ra, const GateArgs& a, hipStream_t s);
hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, int blocks,
                              hipStream_t s);
hipError_t launch_pack(const PackArgs& a, hipStream_t s);
hipError_t launch_reuse_gate(const GateArgs& a, hipStream_t s);
hipError_t launch_ffn(const FfnArgs& a, hipStream_t s);
hipError_t launch_ffn_bf16(const FfnArgs& a, hipStream_t s);
hipError_t launch_ffn_q4(const FfnArgs& a, hipStream_t s);
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);
// int4 weights with K parts and defer_reduce: the parts' ordered reduce into
// expert_out and the combine in one launch, the same results bit for bit as
// the reduce in launch_ffn then launch_combine (ffn_q4.hip).
hipError_t launch_q4_reduce_combine(const FfnArgs& a, const CombineArgs& c, hipStream_t s);

// Largest batch the single-wave gating takes (B k <= 64 assignments).
constexpr int kSmallMaxTokens = 4;

// A whole MoE layer of a small batch in three launches (router rows, gate-up
// with the routing in its prologue, down with the combine), the same results
// bit for bit as launch_route, launch_reuse_gate, launch_ffn and
// launch_combine in sequence: ffn_bf16.hip for bf16 weights, ffn_q4.hip for
// int4 (where the first launch also converts x to fp16).  The *_fits
// functions tell whether the layer's segments fit one workgroup of the down
// launch; a carries the same buckets as ga.
bool moe_layer_small_fits_bf16(const FfnArgs& a);
bool moe_layer_small_fits_q4(const FfnArgs& a);
hipError_t launch_moe_layer_small_bf16(const RouteArgs& ra, const GateArgs& ga,
                                       const FfnArgs& a, float* y, hipStream_t s);
hipError_t launch_moe_layer_small_q4(const RouteArgs& ra, const GateArgs& ga, const FfnArgs& a,
                                     float* y, hipStream_t s);

// Whether a layer call takes the three-launch path: B <= 4 tokens whose
// gating keeps the plain top-k (alpha = 0, or one token), bf16 or int4
// weights, few enough segments.
inline bool moe_layer_small_fits(const FfnArgs& a, float alpha) {
  if (a.B < 1 || a.B > kSmallMaxTokens || !(alpha == 0.f || a.B == 1)) return false;
  if (a.wf == kWBf16) return moe_layer_small_fits_bf16(a);
  if (a.wf == kWQ4) return moe_layer_small_fits_q4(a);
  return false;
}

inline hipError_t launch_moe_layer_small(const RouteArgs& ra, const GateArgs& ga,
                                         const FfnArgs& a, float* y, hipStream_t s) {
  return a.wf == kWQ4 ? launch_moe_layer_small_q4(ra, ga, a, y, s)
                      : launch_moe_layer_small_bf16(ra, ga, a, y, s);
}

}  // namespace s2moe
