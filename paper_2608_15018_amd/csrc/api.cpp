// C-ABI entry points: argument validation on the host, then kernel launches
// on the caller's stream.  Nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "kernels.h"
#include "s2moe.h"

static_assert(s2moe::kMaxShared == S2MOE_MAX_SHARED, "shared-expert limit");

namespace {

thread_local std::string g_last_error;

s2moe_status fail(s2moe_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

s2moe_status ok() {
  g_last_error.clear();
  return S2MOE_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define S2MOE_REQUIRE_PTR(p)                                                     \
  do {                                                                           \
    if ((p) == nullptr) return fail(S2MOE_EINVAL, "%s: %s is NULL", fn, #p);     \
    if (!aligned16(p)) return fail(S2MOE_EINVAL, "%s: %s is not 16-byte aligned", fn, #p); \
  } while (0)

s2moe_status check_layer(const char* fn, const s2moe_layer* L, int32_t B) {
  if (L == nullptr) return fail(S2MOE_EINVAL, "%s: layer is NULL", fn);
  if (B < 1) return fail(S2MOE_EINVAL, "%s: n_tokens = %d, must be >= 1", fn, B);
  if (B > S2MOE_MAX_TOKENS)
    return fail(S2MOE_EUNSUPPORTED, "%s: n_tokens = %d exceeds %d", fn, B, S2MOE_MAX_TOKENS);
  if (L->hidden < 64 || L->hidden % 64 != 0 || L->hidden > 16384)
    return fail(S2MOE_EINVAL, "%s: hidden = %d must be a multiple of 64 in [64, 16384]", fn,
                L->hidden);
  if (L->ffn < 64 || L->ffn % 64 != 0 || L->ffn > 262144)
    return fail(S2MOE_EINVAL, "%s: ffn = %d must be a multiple of 64 in [64, 262144]", fn,
                L->ffn);
  if (L->n_experts < 2)
    return fail(S2MOE_EINVAL, "%s: n_experts = %d must be >= 2", fn, L->n_experts);
  if (L->n_experts > S2MOE_MAX_EXPERTS)
    return fail(S2MOE_EUNSUPPORTED, "%s: n_experts = %d exceeds %d", fn, L->n_experts,
                S2MOE_MAX_EXPERTS);
  if (L->top_k < 1 || L->top_k >= L->n_experts)
    return fail(S2MOE_EINVAL, "%s: top_k = %d must satisfy 1 <= k < E = %d", fn, L->top_k,
                L->n_experts);
  if (L->top_k > S2MOE_MAX_TOPK)
    return fail(S2MOE_EUNSUPPORTED, "%s: top_k = %d exceeds %d", fn, L->top_k, S2MOE_MAX_TOPK);
  if (L->cap < L->top_k || L->cap > L->n_experts)
    return fail(S2MOE_EINVAL, "%s: cap = %d must satisfy k = %d <= cap <= E = %d", fn, L->cap,
                L->top_k, L->n_experts);
  if (!std::isfinite(L->alpha) || L->alpha < 0.f)
    return fail(S2MOE_EINVAL, "%s: alpha = %g must be finite and >= 0", fn, (double)L->alpha);
  if (L->flags & ~15u) return fail(S2MOE_EINVAL, "%s: unknown flags 0x%x", fn, L->flags);
  if (L->n_shared < 0) return fail(S2MOE_EINVAL, "%s: n_shared = %d < 0", fn, L->n_shared);
  if (L->n_shared > S2MOE_MAX_SHARED)
    return fail(S2MOE_EUNSUPPORTED, "%s: n_shared = %d exceeds %d", fn, L->n_shared,
                S2MOE_MAX_SHARED);
  if (L->n_shared > 0 && (L->ffn_shared < 64 || L->ffn_shared % 64 != 0 ||
                          L->ffn_shared > 262144))
    return fail(S2MOE_EINVAL, "%s: ffn_shared = %d must be a multiple of 64 in [64, 262144]",
                fn, L->ffn_shared);
  const int act = L->act_dtype, wdt = L->w_dtype;
  if (act != S2MOE_F32 && act != S2MOE_BF16)
    return fail(S2MOE_EINVAL, "%s: act_dtype = %d must be F32 or BF16", fn, act);
  if (wdt != S2MOE_F32 && wdt != S2MOE_BF16 && wdt != S2MOE_Q4G32)
    return fail(S2MOE_EINVAL, "%s: w_dtype = %d is not a known dtype", fn, wdt);
  const bool pair_ok = (act == S2MOE_F32 && wdt == S2MOE_F32) ||
                       (act == S2MOE_BF16 && (wdt == S2MOE_BF16 || wdt == S2MOE_Q4G32));
  if (!pair_ok)
    return fail(S2MOE_EUNSUPPORTED,
                "%s: (act_dtype, w_dtype) = (%d, %d); supported: (F32, F32), (BF16, BF16), "
                "(BF16, Q4G32)",
                fn, act, wdt);
  // int4 kernels step through K in 128-wide super-steps and take up to 8
  // 16-row tiles per wave.
  if (wdt == S2MOE_Q4G32 &&
      (L->hidden % 128 || L->ffn % 128 || (L->n_shared > 0 && L->ffn_shared % 128)))
    return fail(S2MOE_EUNSUPPORTED,
                "%s: Q4G32 weights need hidden, ffn and ffn_shared multiples of 128", fn);
  if ((L->flags & S2MOE_PACKED_WEIGHTS) && wdt == S2MOE_F32)
    return fail(S2MOE_EUNSUPPORTED, "%s: S2MOE_PACKED_WEIGHTS needs BF16 or Q4G32 weights", fn);
  return S2MOE_OK;
}

size_t round256(size_t n) { return (n + 255) & ~(size_t)255; }

// Workspace: the SwiGLU activations Hh [B*k + S*B, max(F, F_s)] (fp32 for
// fp32 weights, else 16-bit); for int4 weights then an fp16 copy of x and
// the down projection's partial sums.
size_t hh_rows(const s2moe_layer* L, int32_t B) {
  return (size_t)B * L->top_k + (size_t)L->n_shared * B;
}

size_t hh_ld(const s2moe_layer* L) {
  return (size_t)(L->n_shared > 0 && L->ffn_shared > L->ffn ? L->ffn_shared : L->ffn);
}

size_t hh_bytes(const s2moe_layer* L, int32_t B) {
  const size_t elt = L->w_dtype == S2MOE_F32 ? 4 : 2;
  return round256(hh_rows(L, B) * hh_ld(L) * elt);
}

size_t x16_bytes(const s2moe_layer* L, int32_t B) {
  return round256((size_t)B * L->hidden * 2);
}

int q4_parts(const s2moe_layer* L, int32_t B) {
  return s2moe::q4_down_parts(B, L->top_k, L->n_experts, L->hidden, L->ffn, L->n_shared,
                              L->n_shared > 0 ? L->ffn_shared : 0);
}

// int4 weights: partial sums of the down projection's K parts 1 .. Q-1.
size_t part_bytes(const s2moe_layer* L, int32_t B) {
  if (L->w_dtype != S2MOE_Q4G32) return 0;
  return round256((size_t)(q4_parts(L, B) - 1) * hh_rows(L, B) * L->hidden * sizeof(float));
}

size_t workspace_bytes(const s2moe_layer* L, int32_t B) {
  size_t n = hh_bytes(L, B);
  if (L->w_dtype == S2MOE_Q4G32) n += x16_bytes(L, B) + part_bytes(L, B);
  return n;
}

s2moe_status hip_status(const char* fn, hipError_t err) {
  if (err != hipSuccess) return fail(S2MOE_EHIP, "%s: %s", fn, hipGetErrorString(err));
  return ok();
}

// Checks of each step's arguments, then its launch struct.  The single
// entry points and s2moe_moe_layer share them.
s2moe_status route_args(const char* fn, const s2moe_layer* layer, int32_t n_tokens,
                        const void* x, const void* router, const s2moe_routing* r,
                        s2moe::RouteArgs* out) {
  s2moe_status st = check_layer(fn, layer, n_tokens);
  if (st != S2MOE_OK) return st;
  if (r == nullptr) return fail(S2MOE_EINVAL, "%s: routing is NULL", fn);
  S2MOE_REQUIRE_PTR(x);
  S2MOE_REQUIRE_PTR(router);
  S2MOE_REQUIRE_PTR(r->logits);
  S2MOE_REQUIRE_PTR(r->gap);
  S2MOE_REQUIRE_PTR(r->plain_idx);
  s2moe::RouteArgs& a = *out;
  a.x = x;
  a.router = router;
  a.logits = r->logits;
  a.plain_idx = r->plain_idx;
  a.gap = r->gap;
  a.B = n_tokens;
  a.H = layer->hidden;
  a.E = layer->n_experts;
  a.k = layer->top_k;
  a.bf16 = layer->act_dtype == S2MOE_BF16;
  a.x16 = nullptr;
  a.n8 = 0;
  return S2MOE_OK;
}

s2moe_status gate_args(const char* fn, const s2moe_layer* layer, int32_t n_tokens,
                       const float* conf_w, const s2moe_routing* r, s2moe::GateArgs* out) {
  s2moe_status st = check_layer(fn, layer, n_tokens);
  if (st != S2MOE_OK) return st;
  if (r == nullptr) return fail(S2MOE_EINVAL, "%s: routing is NULL", fn);
  S2MOE_REQUIRE_PTR(conf_w);
  S2MOE_REQUIRE_PTR(r->logits);
  S2MOE_REQUIRE_PTR(r->gap);
  S2MOE_REQUIRE_PTR(r->plain_idx);
  S2MOE_REQUIRE_PTR(r->g);
  S2MOE_REQUIRE_PTR(r->pref);
  S2MOE_REQUIRE_PTR(r->idx);
  S2MOE_REQUIRE_PTR(r->gate_w);
  S2MOE_REQUIRE_PTR(r->count);
  S2MOE_REQUIRE_PTR(r->offset);
  S2MOE_REQUIRE_PTR(r->slot);
  S2MOE_REQUIRE_PTR(r->uniq);
  S2MOE_REQUIRE_PTR(r->n_uniq);
  s2moe::GateArgs& a = *out;
  a.logits = r->logits;
  a.gap = r->gap;
  a.plain_idx = r->plain_idx;
  a.conf_w = conf_w;
  a.g = r->g;
  a.pref = r->pref;
  a.idx = r->idx;
  a.gate_w = r->gate_w;
  a.count = r->count;
  a.offset = r->offset;
  a.slot = r->slot;
  a.uniq = r->uniq;
  a.n_uniq = r->n_uniq;
  a.B = n_tokens;
  a.E = layer->n_experts;
  a.k = layer->top_k;
  a.cap = layer->cap;
  a.alpha = layer->alpha;
  a.flags = layer->flags;
  return S2MOE_OK;
}

s2moe_status combine_args(const char* fn, const s2moe_layer* layer, int32_t n_tokens,
                          const s2moe_routing* r, const float* expert_out, float* y,
                          s2moe::CombineArgs* out) {
  s2moe_status st = check_layer(fn, layer, n_tokens);
  if (st != S2MOE_OK) return st;
  if (r == nullptr) return fail(S2MOE_EINVAL, "%s: routing is NULL", fn);
  S2MOE_REQUIRE_PTR(r->gate_w);
  S2MOE_REQUIRE_PTR(expert_out);
  S2MOE_REQUIRE_PTR(y);
  {
    const size_t H = (size_t)layer->hidden, B = (size_t)n_tokens;
    const char* e0 = reinterpret_cast<const char*>(expert_out);
    const char* y0 = reinterpret_cast<const char*>(y);
    const size_t eb = (B * layer->top_k + (size_t)layer->n_shared * B) * H * sizeof(float);
    const size_t yb = B * H * sizeof(float);
    if (y0 < e0 + eb && e0 < y0 + yb)
      return fail(S2MOE_EINVAL, "%s: y overlaps expert_out", fn);
  }
  s2moe::CombineArgs& a = *out;
  a.gate_w = r->gate_w;
  a.expert_out = expert_out;
  a.y = y;
  a.B = n_tokens;
  a.H = layer->hidden;
  a.k = layer->top_k;
  a.S = layer->n_shared;
  return S2MOE_OK;
}

s2moe_status check_workspace(const char* fn, const s2moe_layer* layer, int32_t n_tokens,
                             const void* workspace, size_t given) {
  const size_t need = workspace_bytes(layer, n_tokens);
  if (workspace == nullptr)
    return fail(S2MOE_EWORKSPACE, "%s: workspace is NULL (%zu bytes needed)", fn, need);
  if (!aligned16(workspace))
    return fail(S2MOE_EINVAL, "%s: workspace is not 16-byte aligned", fn);
  if (given < need)
    return fail(S2MOE_EWORKSPACE, "%s: workspace holds %zu bytes, %zu needed", fn, given, need);
  return S2MOE_OK;
}

}  // namespace

extern "C" {

int32_t s2moe_abi_version(void) { return S2MOE_ABI_VERSION; }

const char* s2moe_last_error(void) { return g_last_error.c_str(); }

const char* s2moe_status_string(s2moe_status st) {
  switch (st) {
    case S2MOE_OK: return "S2MOE_OK";
    case S2MOE_EINVAL: return "S2MOE_EINVAL";
    case S2MOE_EUNSUPPORTED: return "S2MOE_EUNSUPPORTED";
    case S2MOE_EWORKSPACE: return "S2MOE_EWORKSPACE";
    case S2MOE_EHIP: return "S2MOE_EHIP";
  }
  return "S2MOE_UNKNOWN";
}

s2moe_status s2moe_route(const s2moe_layer* layer, int32_t n_tokens, const void* x,
                         const void* router, const s2moe_routing* r, void* stream) {
  const char* fn = "s2moe_route";
  s2moe::RouteArgs a;
  const s2moe_status st = route_args(fn, layer, n_tokens, x, router, r, &a);
  if (st != S2MOE_OK) return st;
  return hip_status(fn, s2moe::launch_route(a, static_cast<hipStream_t>(stream)));
}

s2moe_status s2moe_reuse_gate(const s2moe_layer* layer, int32_t n_tokens, const float* conf_w,
                              const s2moe_routing* r, void* stream) {
  const char* fn = "s2moe_reuse_gate";
  s2moe::GateArgs a;
  const s2moe_status st = gate_args(fn, layer, n_tokens, conf_w, r, &a);
  if (st != S2MOE_OK) return st;
  return hip_status(fn, s2moe::launch_reuse_gate(a, static_cast<hipStream_t>(stream)));
}

size_t s2moe_workspace_bytes(const s2moe_layer* layer, int32_t n_tokens) {
  if (check_layer("s2moe_workspace_bytes", layer, n_tokens) != S2MOE_OK) return 0;
  return workspace_bytes(layer, n_tokens);
}

}  // extern "C"

namespace {

// Checks shared by both verify entry points, then everything of the launch
// except the workspace carve-up.
s2moe_status verify_args(const char* fn, const s2moe_layer* layer, int32_t n_tokens,
                         const void* x, const s2moe_weights* w, const s2moe_routing* r,
                         float* expert_out, s2moe::FfnArgs* out) {
  s2moe_status st = check_layer(fn, layer, n_tokens);
  if (st != S2MOE_OK) return st;
  if (w == nullptr) return fail(S2MOE_EINVAL, "%s: weights is NULL", fn);
  if (r == nullptr) return fail(S2MOE_EINVAL, "%s: routing is NULL", fn);
  S2MOE_REQUIRE_PTR(x);
  S2MOE_REQUIRE_PTR(expert_out);
  S2MOE_REQUIRE_PTR(w->gate);
  S2MOE_REQUIRE_PTR(w->up);
  S2MOE_REQUIRE_PTR(w->down);
  const bool q4 = layer->w_dtype == S2MOE_Q4G32;
  if (q4) {
    S2MOE_REQUIRE_PTR(w->gate_s);
    S2MOE_REQUIRE_PTR(w->up_s);
    S2MOE_REQUIRE_PTR(w->down_s);
  }
  if (layer->n_shared > 0) {
    S2MOE_REQUIRE_PTR(w->sh_gate);
    S2MOE_REQUIRE_PTR(w->sh_up);
    S2MOE_REQUIRE_PTR(w->sh_down);
    if (q4) {
      S2MOE_REQUIRE_PTR(w->sh_gate_s);
      S2MOE_REQUIRE_PTR(w->sh_up_s);
      S2MOE_REQUIRE_PTR(w->sh_down_s);
    }
  }
  S2MOE_REQUIRE_PTR(r->count);
  S2MOE_REQUIRE_PTR(r->offset);
  S2MOE_REQUIRE_PTR(r->slot);
  S2MOE_REQUIRE_PTR(r->uniq);
  S2MOE_REQUIRE_PTR(r->n_uniq);

  s2moe::FfnArgs& a = *out;
  a.B = n_tokens;
  a.k = layer->top_k;
  a.S = layer->n_shared;
  a.E = layer->n_experts;
  a.H = layer->hidden;
  a.F = layer->ffn;
  a.Fs = layer->n_shared > 0 ? layer->ffn_shared : 0;
  a.wf = layer->w_dtype == S2MOE_F32 ? s2moe::kWF32
                                     : (q4 ? s2moe::kWQ4 : s2moe::kWBf16);
  a.count = r->count;
  a.offset = r->offset;
  a.slot = r->slot;
  a.uniq = r->uniq;
  a.n_uniq = r->n_uniq;
  a.x = x;
  a.gate = w->gate;
  a.up = w->up;
  a.down = w->down;
  a.gate_s = w->gate_s;
  a.up_s = w->up_s;
  a.down_s = w->down_s;
  a.sh_gate = w->sh_gate;
  a.sh_up = w->sh_up;
  a.sh_down = w->sh_down;
  a.sh_gate_s = w->sh_gate_s;
  a.sh_up_s = w->sh_up_s;
  a.sh_down_s = w->sh_down_s;
  a.hh = nullptr;
  a.ldh = (int)hh_ld(layer);
  a.x16 = nullptr;
  a.part = nullptr;
  a.qparts = q4 ? q4_parts(layer, n_tokens) : 1;
  a.x16_ready = false;
  a.defer_reduce = false;
  a.out = expert_out;
  a.packed = (layer->flags & S2MOE_PACKED_WEIGHTS) != 0;
  return S2MOE_OK;
}

// Hh at the start of the workspace, then (int4 weights) the fp16 copy of x
// and the down partial sums.
void carve_workspace(const s2moe_layer* layer, int32_t n_tokens, void* workspace,
                     s2moe::FfnArgs* a) {
  char* ws = static_cast<char*>(workspace);
  a->hh = ws;
  const bool q4 = layer->w_dtype == S2MOE_Q4G32;
  a->x16 = q4 ? ws + hh_bytes(layer, n_tokens) : nullptr;
  a->part = q4 ? reinterpret_cast<float*>(ws + hh_bytes(layer, n_tokens) +
                                          x16_bytes(layer, n_tokens))
               : nullptr;
}

}  // namespace

extern "C" {

s2moe_status s2moe_verify_moe(const s2moe_layer* layer, int32_t n_tokens, const void* x,
                              const s2moe_weights* w, const s2moe_routing* r, void* workspace,
                              size_t workspace_bytes_given, float* expert_out, void* stream) {
  const char* fn = "s2moe_verify_moe";
  s2moe::FfnArgs a;
  s2moe_status st = verify_args(fn, layer, n_tokens, x, w, r, expert_out, &a);
  if (st == S2MOE_OK) st = check_workspace(fn, layer, n_tokens, workspace, workspace_bytes_given);
  if (st != S2MOE_OK) return st;
  carve_workspace(layer, n_tokens, workspace, &a);
  return hip_status(fn, s2moe::launch_ffn(a, static_cast<hipStream_t>(stream)));
}

s2moe_status s2moe_verify_moe_noalloc(const s2moe_layer* layer, int32_t n_tokens,
                                      const void* x, const s2moe_weights* w,
                                      const s2moe_routing* r, float* expert_out,
                                      void* stream) {
  const char* fn = "s2moe_verify_moe_noalloc";
  s2moe::FfnArgs a;
  s2moe_status st = verify_args(fn, layer, n_tokens, x, w, r, expert_out, &a);
  if (st != S2MOE_OK) return st;
  const size_t need = workspace_bytes(layer, n_tokens);
  if (need > (size_t)S2MOE_NOALLOC_SCRATCH_BYTES)
    return fail(S2MOE_EUNSUPPORTED,
                "%s: this layer and n_tokens = %d need %zu bytes of scratch; the library's "
                "scratch array holds %zu (use s2moe_verify_moe with a caller workspace)",
                fn, n_tokens, need, (size_t)S2MOE_NOALLOC_SCRATCH_BYTES);
  void* scratch = nullptr;
  const hipError_t err = s2moe::noalloc_scratch(&scratch);
  if (err != hipSuccess) return hip_status(fn, err);
  carve_workspace(layer, n_tokens, scratch, &a);
  return hip_status(fn, s2moe::launch_ffn(a, static_cast<hipStream_t>(stream)));
}

namespace {

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// LDS available to one workgroup on the current device.
s2moe_status device_lds(const char* fn, size_t* bytes) {
  int dev = 0, v = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return fail(S2MOE_EHIP, "%s: %s", fn, hipGetErrorString(e));
  *bytes = (size_t)v;
  return S2MOE_OK;
}

s2moe_status check_expand_dims(const char* fn, int32_t L, int32_t E, int32_t k) {
  if (L < 1 || L > 128) return fail(S2MOE_EINVAL, "%s: n_layers = %d not in [1, 128]", fn, L);
  if (E < 1 || E > 1024) return fail(S2MOE_EINVAL, "%s: n_experts = %d not in [1, 1024]", fn, E);
  if (k < 1 || k > 32) return fail(S2MOE_EINVAL, "%s: k = %d not in [1, 32]", fn, k);
  return S2MOE_OK;
}

}  // namespace

s2moe_status s2moe_expand_max_nodes(int32_t n_layers, int32_t n_experts, int32_t k,
                                    int32_t* max_nodes) {
  const char* fn = "s2moe_expand_max_nodes";
  if (max_nodes == nullptr) return fail(S2MOE_EINVAL, "%s: max_nodes is NULL", fn);
  *max_nodes = 0;
  s2moe_status st = check_expand_dims(fn, n_layers, n_experts, k);
  if (st != S2MOE_OK) return st;
  size_t lds = 0;
  if ((st = device_lds(fn, &lds)) != S2MOE_OK) return st;
  int best = 0;
  for (int n = 1; n <= 1024; ++n)
    if (s2moe::expand_lds(n, n_layers, n_experts, k).total <= lds) best = n;
  *max_nodes = best;
  return ok();
}

s2moe_status s2moe_expand(const s2moe_expand_shape* shape, const int32_t* parent,
                          const float* q, const int32_t* eid, const float* c_draft,
                          const int32_t* root_eid, const int32_t* n_nodes, int32_t* order,
                          double* util, int32_t* n_new, int32_t* n_admit, int32_t* n_pairs,
                          int32_t* status, void* stream) {
  const char* fn = "s2moe_expand";
  if (shape == nullptr) return fail(S2MOE_EINVAL, "%s: shape is NULL", fn);
  const s2moe_expand_shape& sh = *shape;
  if (sh.n_trees < 0 || sh.n_trees > (1 << 24))
    return fail(S2MOE_EINVAL, "%s: n_trees = %d not in [0, 2^24]", fn, sh.n_trees);
  if (sh.max_nodes < 1 || sh.max_nodes > 1024)
    return fail(S2MOE_EINVAL, "%s: max_nodes = %d not in [1, 1024]", fn, sh.max_nodes);
  s2moe_status st = check_expand_dims(fn, sh.n_layers, sh.n_experts, sh.k);
  if (st != S2MOE_OK) return st;
  if (!std::isfinite(sh.t_ar) || sh.t_ar < 0.0 || !std::isfinite(sh.t_exp) || sh.t_exp < 0.0)
    return fail(S2MOE_EINVAL, "%s: t_ar = %g, t_exp = %g must be finite and >= 0", fn, sh.t_ar,
                sh.t_exp);
  if (sh.n_trees == 0) return ok();
  const struct {
    const void* p;
    size_t align;
    const char* name;
  } ptrs[] = {{parent, 4, "parent"}, {q, 4, "q"},           {eid, 4, "eid"},
              {c_draft, 4, "c_draft"}, {n_nodes, 4, "n_nodes"}, {order, 4, "order"},
              {util, 8, "util"},     {n_new, 4, "n_new"},   {n_admit, 4, "n_admit"},
              {n_pairs, 4, "n_pairs"}, {status, 4, "status"}};
  for (const auto& x : ptrs) {
    if (x.p == nullptr) return fail(S2MOE_EINVAL, "%s: %s is NULL", fn, x.name);
    if (!aligned(x.p, x.align))
      return fail(S2MOE_EINVAL, "%s: %s is not %zu-byte aligned", fn, x.name, x.align);
  }
  if (root_eid != nullptr && !aligned(root_eid, 4))
    return fail(S2MOE_EINVAL, "%s: root_eid is not 4-byte aligned", fn);
  if (!aligned(eid, 16)) return fail(S2MOE_EINVAL, "%s: eid is not 16-byte aligned", fn);
  const size_t need = s2moe::expand_lds(sh.max_nodes, sh.n_layers, sh.n_experts, sh.k).total;
  size_t lds = 0;
  if ((st = device_lds(fn, &lds)) != S2MOE_OK) return st;
  if (need > lds)
    return fail(S2MOE_EUNSUPPORTED,
                "%s: N = %d, L = %d, E = %d, k = %d needs %zu bytes of LDS per tree; the device "
                "has %zu (s2moe_expand_max_nodes gives the largest N)",
                fn, sh.max_nodes, sh.n_layers, sh.n_experts, sh.k, need, lds);
  // f / k for f < N L k <= 2^22 as one multiply and shift: the error of
  // f * ceil(2^42 / k) / 2^42 is below f / 2^42 <= 2^-20 < 1 / k.
  const uint64_t kdiv = ((1ull << 42) + (uint64_t)sh.k - 1) / (uint64_t)sh.k;
  s2moe::ExpandArgs a{};
  a.parent = parent;
  a.q = q;
  a.eid = eid;
  a.c_draft = c_draft;
  a.root_eid = root_eid;
  a.n_nodes = n_nodes;
  a.order = order;
  a.util = util;
  a.n_new = n_new;
  a.n_admit = n_admit;
  a.n_pairs = n_pairs;
  a.status = status;
  a.T = sh.n_trees;
  a.N = sh.max_nodes;
  a.L = sh.n_layers;
  a.E = sh.n_experts;
  a.k = sh.k;
  a.max_admit = sh.max_admit;
  a.k_div = kdiv;
  a.t_ar = sh.t_ar;
  a.t_exp = sh.t_exp;
  return hip_status(fn, s2moe::launch_expand(a, need, static_cast<hipStream_t>(stream)));
}

s2moe_status s2moe_stream_read(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  const char* fn = "s2moe_stream_read";
  if (src == nullptr || sink == nullptr) return fail(S2MOE_EINVAL, "%s: NULL pointer", fn);
  if (!aligned16(src) || !aligned16(sink))
    return fail(S2MOE_EINVAL, "%s: pointers must be 16-byte aligned", fn);
  if (bytes == 0 || bytes % 16 != 0)
    return fail(S2MOE_EINVAL, "%s: bytes = %zu, need a nonzero multiple of 16", fn, bytes);
  // 2 waves per SIMD, each streaming one long contiguous range: the
  // fastest plain read pattern measured on MI355X.
  return hip_status(fn, s2moe::launch_stream_read(src, bytes, sink, 512,
                                                  static_cast<hipStream_t>(stream)));
}

s2moe_status s2moe_pack_weights(int32_t w_dtype, int32_t n_mats, int32_t rows, int32_t cols,
                                const void* src, const void* src_scales, void* dst,
                                void* dst_scales, void* stream) {
  const char* fn = "s2moe_pack_weights";
  if (w_dtype != S2MOE_BF16 && w_dtype != S2MOE_Q4G32)
    return fail(w_dtype == S2MOE_F32 ? S2MOE_EUNSUPPORTED : S2MOE_EINVAL,
                "%s: w_dtype = %d; packing applies to BF16 and Q4G32 weights", fn, w_dtype);
  const bool q4 = w_dtype == S2MOE_Q4G32;
  if (n_mats < 1 || rows < 16 || rows % 16 != 0)
    return fail(S2MOE_EINVAL, "%s: n_mats = %d, rows = %d (need n_mats >= 1, rows % 16 == 0)",
                fn, n_mats, rows);
  const int kq = q4 ? 128 : 32;
  if (cols < kq || cols % kq != 0)
    return fail(S2MOE_EINVAL, "%s: cols = %d must be a positive multiple of %d", fn, cols, kq);
  S2MOE_REQUIRE_PTR(src);
  S2MOE_REQUIRE_PTR(dst);
  const size_t bytes = (size_t)n_mats * rows * cols / (q4 ? 2 : 1) * (q4 ? 1 : 2);
  const char* s0 = static_cast<const char*>(src);
  const char* d0 = static_cast<const char*>(dst);
  if (s0 < d0 + bytes && d0 < s0 + bytes)
    return fail(S2MOE_EINVAL, "%s: src and dst overlap (packing is not in place)", fn);
  if (q4) {
    S2MOE_REQUIRE_PTR(src_scales);
    S2MOE_REQUIRE_PTR(dst_scales);
    const size_t sb = (size_t)n_mats * rows * (cols / 32) * 2;
    const char* ss = static_cast<const char*>(src_scales);
    const char* ds = static_cast<const char*>(dst_scales);
    if (ss < ds + sb && ds < ss + sb)
      return fail(S2MOE_EINVAL, "%s: src_scales and dst_scales overlap", fn);
  }
  s2moe::PackArgs a;
  a.src = src;
  a.src_s = src_scales;
  a.dst = dst;
  a.dst_s = dst_scales;
  a.n = n_mats;
  a.rows = rows;
  a.K = cols;
  a.q4 = q4;
  return hip_status(fn, s2moe::launch_pack(a, static_cast<hipStream_t>(stream)));
}

s2moe_status s2moe_combine(const s2moe_layer* layer, int32_t n_tokens, const s2moe_routing* r,
                           const float* expert_out, float* y, void* stream) {
  const char* fn = "s2moe_combine";
  s2moe::CombineArgs a;
  const s2moe_status st = combine_args(fn, layer, n_tokens, r, expert_out, y, &a);
  if (st != S2MOE_OK) return st;
  return hip_status(fn, s2moe::launch_combine(a, static_cast<hipStream_t>(stream)));
}

s2moe_status s2moe_moe_layer(const s2moe_layer* layer, int32_t n_tokens, const void* x,
                             const void* router, const float* conf_w, const s2moe_weights* w,
                             const s2moe_routing* r, void* workspace,
                             size_t workspace_bytes_given, float* expert_out, float* y,
                             void* stream) {
  const char* fn = "s2moe_moe_layer";
  s2moe::RouteArgs ra;
  s2moe::GateArgs ga;
  s2moe::FfnArgs fa;
  s2moe::CombineArgs ca;
  s2moe_status st = route_args(fn, layer, n_tokens, x, router, r, &ra);
  if (st == S2MOE_OK) st = gate_args(fn, layer, n_tokens, conf_w, r, &ga);
  if (st == S2MOE_OK) st = verify_args(fn, layer, n_tokens, x, w, r, expert_out, &fa);
  if (st == S2MOE_OK) st = check_workspace(fn, layer, n_tokens, workspace, workspace_bytes_given);
  if (st == S2MOE_OK) st = combine_args(fn, layer, n_tokens, r, expert_out, y, &ca);
  if (st != S2MOE_OK) return st;
  carve_workspace(layer, n_tokens, workspace, &fa);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (s2moe::moe_layer_small_fits(fa, layer->alpha))
    return hip_status(fn, s2moe::launch_moe_layer_small(ra, ga, fa, y, s));
  if (fa.wf == s2moe::kWQ4) {
    // The routing launch also writes the fp16 copy of x, and the combine
    // launch also adds the down projection's K parts.
    ra.x16 = static_cast<uint16_t*>(fa.x16);
    ra.n8 = n_tokens * layer->hidden / 8;
    fa.x16_ready = true;
    fa.defer_reduce = fa.qparts > 1;
  }
  hipError_t err = s2moe::launch_route_and_gate(ra, ga, s);
  if (err == hipSuccess) err = s2moe::launch_ffn(fa, s);
  if (err == hipSuccess)
    err = fa.defer_reduce ? s2moe::launch_q4_reduce_combine(fa, ca, s)
                          : s2moe::launch_combine(ca, s);
  return hip_status(fn, err);
}

}  // extern "C"
