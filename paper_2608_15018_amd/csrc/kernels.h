// Internal launch interface between the C-ABI layer (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace s2moe {

constexpr int kMaxTopK = 16;
constexpr int kMaxTokens = 256;
constexpr int kMaxExperts = 256;

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
  bool packed;  // weights in the packed tile order (pack.hip)
  float* out;  // [B*k + S*B, H]
};

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

hipError_t launch_route(const RouteArgs& a, hipStream_t s);
hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, int blocks,
                              hipStream_t s);
hipError_t launch_pack(const PackArgs& a, hipStream_t s);
hipError_t launch_reuse_gate(const GateArgs& a, hipStream_t s);
hipError_t launch_ffn(const FfnArgs& a, hipStream_t s);
hipError_t launch_ffn_bf16(const FfnArgs& a, hipStream_t s);
hipError_t launch_ffn_q4(const FfnArgs& a, hipStream_t s);
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

}  // namespace s2moe
