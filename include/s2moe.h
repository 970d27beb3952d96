/*
 * s2moe.h -- C ABI of the S2-MoE verify-MoE hot path on AMD Instinct MI355X
 * (gfx950).
 *
 * The verification pass of self-speculative decoding runs one MoE layer over
 * the B draft tokens of a verify batch.  The paper (Sec. "Reuse-aware Expert
 * Gating") defines the routing part: the target gating logits ell_b of each
 * draft token, confidence weights w_b >= 0, the cross-token expert importance
 * g_e = sum_b w_b ell_{b,e}, the globally preferred set E* = TopCap(g) with
 * k <= cap, and the additive bias ell'_{b,e} = ell_{b,e} + lambda_b [e in E*]
 * with lambda_b proportional to the gap between the token's top-1 and
 * (k+1)-th logits.  The experts are SwiGLU FFNs; each activated expert's
 * weights are streamed from HBM once for all tokens routed to it (the
 * verification cost the paper counts per newly activated expert, Sec.
 * "Routing-aware Adaptive Speculative Expansion", marginal verification
 * cost).
 *
 * Conventions shared by every entry point
 *   - Tensor arguments are DEVICE pointers, row-major, owned by the caller.
 *     The library never allocates or frees device memory.
 *   - Every pointer must be 16-byte aligned.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls only enqueue work; results are valid once the stream reaches
 *     them.  Nothing synchronises the host.
 *   - Argument errors are detected on the host before anything is enqueued
 *     and returned as S2MOE_EINVAL / S2MOE_EUNSUPPORTED / S2MOE_EWORKSPACE;
 *     a failed launch returns S2MOE_EHIP.  s2moe_last_error() then names the
 *     problem (thread-local string).  No exception crosses the ABI.
 *   - Non-finite inputs are undefined behaviour.
 *   - Calls on one stream are ordered; calls that share output buffers on
 *     different streams race.
 */
#ifndef S2MOE_H
#define S2MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define S2MOE_ABI_VERSION 1
#define S2MOE_MAX_TOKENS 256  /* B: draft tokens per verify batch   */
#define S2MOE_MAX_EXPERTS 256 /* E: routed experts per layer        */
#define S2MOE_MAX_TOPK 16     /* k: experts per token               */
#define S2MOE_MAX_SHARED 8    /* S: always-on shared experts        */

typedef enum s2moe_status {
  S2MOE_OK = 0,
  S2MOE_EINVAL = 1,       /* malformed argument (null, misaligned, out of range) */
  S2MOE_EUNSUPPORTED = 2, /* well-formed but outside what the kernels handle     */
  S2MOE_EWORKSPACE = 3,   /* workspace missing or smaller than required          */
  S2MOE_EHIP = 4          /* a HIP launch or runtime call failed                 */
} s2moe_status;

typedef enum s2moe_dtype {
  S2MOE_F32 = 0,
  S2MOE_BF16 = 1,
  /* weights only: 4-bit codes q in [0,15], two per byte (element 2i in the
     low nibble of byte i), value s * (q - 8) with one fp16 scale s per 32
     consecutive elements along K.  Codes [rows, K/2] u8, scales [rows, K/32]
     f16, per expert.
     Range: with these weights the kernels compute in fp16 with fp32
     accumulation.  x is converted from bf16 to fp16, each weight is rounded
     once to fp16 as s * (q - 8), and the SwiGLU activations
     silu(W_g x) * (W_u x) are stored in fp16.  Every |x|, |s * (q - 8)|
     and activation must therefore stay below 65504 (larger finite values
     become infinite, with no error), and magnitudes below about 6.1e-5
     keep fewer significant bits (fp16 subnormals). */
  S2MOE_Q4G32 = 2
} s2moe_dtype;

/* Readings of the paper's gating where the text leaves a choice (0 = default). */
enum {
  /* TopCap candidates restricted to experts that some token of the batch
     already selects in its plain top-k, so that E* holds at most cap of
     them (Sec. "Reuse-aware Expert Gating", opening paragraph and "Global
     preferred expert selection": the preferred experts are read there as
     ones the batch already activates).  Default: all E experts compete. */
  S2MOE_PREF_ACTIVATED_ONLY = 1u,
  /* lambda_b = alpha instead of alpha * gap_b. */
  S2MOE_BIAS_ABSOLUTE = 2u,
  /* gate weights from the biased logits ell' instead of the original ell. */
  S2MOE_GATE_FROM_BIASED = 4u,
  /* The expert weights passed to s2moe_verify_moe were re-laid by
     s2moe_pack_weights (BF16 and Q4G32 only). */
  S2MOE_PACKED_WEIGHTS = 8u
};

/* One MoE layer.  Supported (act_dtype, w_dtype) pairs: (F32, F32),
   (BF16, BF16), (BF16, Q4G32). */
typedef struct s2moe_layer {
  int32_t hidden;      /* H: 64 <= H <= 16384, H % 64 == 0                  */
  int32_t ffn;         /* F: routed SwiGLU width, 64 <= F <= 262144,
                          F % 64 == 0 (F % 128 == 0 with Q4G32 weights,
                          like H and F_s)                                   */
  int32_t n_experts;   /* E: 2 <= E <= 256                                  */
  int32_t top_k;       /* k: 1 <= k < E, k <= 16                            */
  int32_t n_shared;    /* S: 0 <= S <= 8 always-on experts (weight 1)       */
  int32_t ffn_shared;  /* F_s: 64 <= F_s <= 262144, F_s % 64 == 0 when S > 0 */
  int32_t cap;         /* k <= cap <= E                                     */
  float alpha;         /* lambda_b = alpha * gap_b, alpha >= 0, finite      */
  uint32_t flags;      /* S2MOE_PREF_ACTIVATED_ONLY | ... (default 0)       */
  int32_t act_dtype;   /* s2moe_dtype of x and router: F32 or BF16          */
  int32_t w_dtype;     /* s2moe_dtype of expert weights                     */
} s2moe_layer;

/* Expert weights (device pointers).  Routed:  gate, up [E, F, H] (K = H
   contiguous), down [E, H, F] (K = F contiguous).  Shared: sh_gate, sh_up
   [S, F_s, H], sh_down [S, H, F_s].  For Q4G32 the matrices hold codes with
   K/2 bytes per row and the *_s pointers the fp16 scales with K/32 per row;
   for F32/BF16 the *_s pointers are ignored. */
typedef struct s2moe_weights {
  const void *gate, *up, *down;
  const void *gate_s, *up_s, *down_s;
  const void *sh_gate, *sh_up, *sh_down;
  const void *sh_gate_s, *sh_up_s, *sh_down_s;
} s2moe_weights;

/* Routing state of one verify batch (device memory, caller-owned).  The
   pointers are read from this struct; the arrays they name are written. */
typedef struct s2moe_routing {
  float *logits;      /* [B, E]   ell_b = W_r x_b (fp32)                       */
  float *gap;         /* [B]      ell_(1) - ell_(k+1)                          */
  int32_t *plain_idx; /* [B, k]   unbiased top-k, ascending expert id          */
  float *g;           /* [E]      sum_b max(w_b, 0) ell_{b,e}                  */
  int32_t *pref;      /* [E]      1 iff e in E*                                */
  int32_t *idx;       /* [B, k]   biased top-k, ascending expert id            */
  float *gate_w;      /* [B, k]   softmax over the selected k, sums to 1       */
  int32_t *count;     /* [E]      tokens routed to expert e                    */
  int32_t *offset;    /* [E + 1]  exclusive prefix sum of count                */
  int32_t *slot;      /* [B * k]  assignments a = b*k + j, expert-major, stable */
  int32_t *uniq;      /* [E]      activated experts ascending, tail = -1       */
  int32_t *n_uniq;    /* [1]      |U|                                          */
} s2moe_routing;

/* Router and plain top-k (Sec. "Reuse-aware Expert Gating": the target
   gating logits ell_b, and the top-1 / (k+1)-th gap of "Soft routing bias
   for reuse promotion").
   x [B, H] and router [E, H] in layer->act_dtype.  Writes r->logits
   (fp32 accumulation), r->plain_idx (ties -> lower expert id) and r->gap. */
s2moe_status s2moe_route(const s2moe_layer *layer, int32_t n_tokens, const void *x,
                         const void *router, const s2moe_routing *r, void *stream);

/* Reuse-aware expert gating and token->expert bucketing (same section:
   "Cross-token expert importance aggregation", "Global preferred expert
   selection", "Soft routing bias for reuse promotion").
   conf_w [B] fp32; values below 0 are treated as 0 and if none is positive
   no bias is applied.  Reads r->logits, r->gap, r->plain_idx; writes r->g,
   pref, idx, gate_w, count, offset, slot, uniq, n_uniq.  Deterministic: no
   floating-point atomics, fixed summation order. */
s2moe_status s2moe_reuse_gate(const s2moe_layer *layer, int32_t n_tokens,
                              const float *conf_w, const s2moe_routing *r, void *stream);

/* Bytes of device workspace s2moe_verify_moe needs for n_tokens tokens. */
size_t s2moe_workspace_bytes(const s2moe_layer *layer, int32_t n_tokens);

/* Grouped SwiGLU experts over the verify batch: for every activated expert
   e, FFN_e(x) = W_d,e (silu(W_g,e x) * (W_u,e x)) of each token routed to it,
   each expert's weights read from HBM once for all its tokens; and every
   shared expert over all tokens.
   x [B, H] act_dtype; reads r->count, offset, slot, uniq, n_uniq.  Writes
   expert_out [B*k + S*B, H] fp32, unscaled: row b*k + j for the j-th routed
   expert of token b, row B*k + s*B + b for shared expert s.  workspace must
   hold s2moe_workspace_bytes(layer, n_tokens) bytes; its contents on entry
   do not matter and are clobbered. */
s2moe_status s2moe_verify_moe(const s2moe_layer *layer, int32_t n_tokens, const void *x,
                              const s2moe_weights *w, const s2moe_routing *r,
                              void *workspace, size_t workspace_bytes, float *expert_out,
                              void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
   capture, tight serving loops, harnesses that forbid hipMalloc):
   s2moe_verify_moe without a workspace argument.  The SwiGLU activations
   (and, for Q4G32 weights, the fp16 copy of x) go to a scratch array the
   library holds in device memory, S2MOE_NOALLOC_SCRATCH_BYTES per GPU, from
   the library's load until the process ends; the call itself allocates
   nothing.  Arguments, outputs and results are those of s2moe_verify_moe,
   computed by the same kernels.  A layer and n_tokens whose
   s2moe_workspace_bytes exceed S2MOE_NOALLOC_SCRATCH_BYTES are rejected
   with S2MOE_EUNSUPPORTED before anything is enqueued (c2- to c5-shaped
   layers at up to 64 tokens need at most 8 MiB: the int4 layer at 64
   tokens, with its down projection's partial sums over 3 K parts).  All calls on one
   GPU share its array: calls that can overlap on the device (different
   streams without ordering, several host threads) race and give undefined
   results.  Calls ordered on one stream are safe; the array's contents
   left by a previous call are never read. */
#define S2MOE_NOALLOC_SCRATCH_BYTES (16u << 20)
s2moe_status s2moe_verify_moe_noalloc(const s2moe_layer *layer, int32_t n_tokens, const void *x,
                                      const s2moe_weights *w, const s2moe_routing *r,
                                      float *expert_out, void *stream);

/* Re-lay n_mats expert matrices of [rows, cols] (K = cols contiguous) into
   the tile order the matrix-core kernels stream (layer flag
   S2MOE_PACKED_WEIGHTS).  A one-time transform at model load, not part of
   a verify step: the values are unchanged, only their order, and dst has the
   same size as src.
     BF16:  src, dst [n_mats, rows, cols] bf16; each 16-row x 32-column tile
            becomes one contiguous 1 KB block, tiles ordered row-tile-major.
            rows % 16 == 0, cols % 32 == 0.  *_scales ignored (may be NULL).
     Q4G32: src, dst codes [n_mats, rows, cols/2]; src_scales, dst_scales
            fp16 [n_mats, rows, cols/32]; each 16-row x 128-column block of
            codes becomes 1 KB, its 64 scales 128 bytes.  rows % 16 == 0,
            cols % 128 == 0.
   Apply it to gate and up as [E, F, H], down as [E, H, F], and the shared
   matrices alike.  dst must not overlap src.  Device pointers, enqueued on
   `stream`; F32 weights give S2MOE_EUNSUPPORTED. */
s2moe_status s2moe_pack_weights(int32_t w_dtype, int32_t n_mats, int32_t rows, int32_t cols,
                                const void *src, const void *src_scales, void *dst,
                                void *dst_scales, void *stream);

/* Combine (MoE layer definition: each token's output is the gate-weighted
   sum of its k routed experts' outputs plus, with weight 1, every shared
   expert's output):
   y_b = sum_{j<k} gate_w[b,j] expert_out[b*k+j] +
   sum_{s<S} expert_out[B*k + s*B + b], summed in that order (fp32).
   Reads r->gate_w [B, k] and expert_out [B*k + S*B, H] as written by
   s2moe_reuse_gate and s2moe_verify_moe; writes y [B, H] fp32 (caller-owned,
   must not overlap expert_out).  Errors as for every entry point. */
s2moe_status s2moe_combine(const s2moe_layer *layer, int32_t n_tokens,
                           const s2moe_routing *r, const float *expert_out, float *y,
                           void *stream);

/* One whole MoE layer (the verify pass of Sec. "Reuse-aware Expert Gating"
   over one layer, or a draft step's layer with top_k = k_draft and alpha =
   0, Sec. "System Implementation", "Draft configuration"): s2moe_route,
   s2moe_reuse_gate, s2moe_verify_moe and s2moe_combine on these arguments,
   in that order, with the same results bit for bit in every output (r's
   arrays, expert_out, y) and the same argument checks and errors.
   A batch whose gating cannot move the plain top-k (alpha = 0, or
   n_tokens = 1) and that has at most 4 tokens, BF16 or Q4G32 weights and at
   most 16 waves' worth of segments (S + min(E, B k) segments, each taking
   as many waves as the down launch splits its K into) runs as three
   launches instead of six (seven for Q4G32): the router rows (with Q4G32
   also the fp16 copy of x); the gate-up projection, where every workgroup
   first ranks the logits and buckets the batch itself; and the down
   projection with the combine folded in.  Every other batch runs the four
   calls' kernels one after another, except that the gating launch ranks
   the logits itself where the routing would rank them in a launch of its
   own, and that with Q4G32 weights the routing launch also makes the fp16
   copy of x and the combine launch also adds the down projection's K parts
   (two launches fewer than the four calls).  Layer dispatch cost dominates
   small batches (a draft step runs one per MoE layer and token).
   Workspace, ownership and stream as for s2moe_verify_moe; y as for
   s2moe_combine. */
s2moe_status s2moe_moe_layer(const s2moe_layer *layer, int32_t n_tokens, const void *x,
                             const void *router, const float *conf_w,
                             const s2moe_weights *w, const s2moe_routing *r,
                             void *workspace, size_t workspace_bytes, float *expert_out,
                             float *y, void *stream);

/* ---------------------------------------------------------------------------
   Routing-aware adaptive speculative expansion (Sec. "Routing-aware Adaptive
   Speculative Expansion"): which draft tokens enter the verify batch.

   Each of T draft trees has up to N candidate tokens (nodes 0..n_t-1,
   n_t = n_nodes[t]; a node's parent is an earlier node, or -1 for a child of
   the root, the last verified token).  With
     p_i   = q_i * p_parent(i)  (prefix confidence, "Expected Benefit"),
     B_i   = p_i * T_AR,
     dC_i  = |E_i \ U| * T_exp (Eq. of the marginal verification cost; E_i
             the (layer, expert) pairs predicted for token i, U the union of
             the pairs of the selected tokens, started from the root's),
     U_i   = B_i / (dC_i + C_i^draft)  (Eq. of the utility),
   the call repeatedly selects, among the unselected nodes whose parent is
   selected (or is the root), the one of largest U_i (ties: smaller index),
   while that U_i >= 1, up to max_admit selections.  Everything is computed
   in fp64 as B / (n * T_exp + c) without fused multiply-adds, so results
   are reproducible bit for bit.

   A node is never selected, nor anything below it, if its parent is not -1
   or an earlier node (status bit 1), its q is not in [0, 1] (bit 2) or its
   C^draft is not finite and positive (bit 4); an n_nodes value outside
   [0, N] is clamped (bit 8).  Expert ids outside [0, E) are padding and
   repeated ids count once.

   All arrays are device memory, padded per tree to N nodes, row-major:
     parent   [T][N]       int32
     q        [T][N]       float  draft confidence of node i given its prefix
     eid      [T][N][L][k] int32  predicted experts per MoE layer (16-byte aligned)
     c_draft  [T][N]       float  C_i^draft
     root_eid [T][L][k]    int32  experts of the root token, or NULL (U starts empty)
     n_nodes  [T]          int32
   and written:
     order    [T][N]  int32   selected nodes in selection order, -1 after
     util     [T][N]  double  U_i at each selection, 0 after
     n_new    [T][N]  int32   |E_i \ U| at each selection, 0 after
     n_admit  [T]     int32   number selected
     n_pairs  [T]     int32   |U| at the end (root pairs included)
     status   [T]     int32   bits above, 0 if every node was valid
   Limits: 1 <= N <= 1024, 1 <= L <= 128, 1 <= E <= 1024, 1 <= k <= 32, and
   the tree state (about (N + 1) * L * E' / 8 + 17 N bytes, E' = E rounded
   up to a power of two >= 32) must fit in one
   workgroup's LDS (s2moe_expand_max_nodes); T_AR and T_exp finite and
   >= 0.  Errors: S2MOE_EINVAL for a malformed argument, S2MOE_EUNSUPPORTED
   when the tree state does not fit.  T = 0 is a no-op.  Enqueued on
   `stream`; one workgroup per tree. */
typedef struct s2moe_expand_shape {
  int32_t n_trees;    /* T                                              */
  int32_t max_nodes;  /* N: padded nodes per tree                       */
  int32_t n_layers;   /* L: MoE layers whose experts are predicted      */
  int32_t n_experts;  /* E                                              */
  int32_t k;          /* ids per token and layer (-1 padding allowed)   */
  int32_t max_admit;  /* selections per tree, <= 0: no limit           */
  double t_ar;        /* T_AR: one target decoding step                 */
  double t_exp;       /* T_exp: one more expert at one layer            */
} s2moe_expand_shape;

s2moe_status s2moe_expand(const s2moe_expand_shape *shape, const int32_t *parent,
                          const float *q, const int32_t *eid, const float *c_draft,
                          const int32_t *root_eid, const int32_t *n_nodes, int32_t *order,
                          double *util, int32_t *n_new, int32_t *n_admit, int32_t *n_pairs,
                          int32_t *status, void *stream);

/* Largest N (<= 1024) that s2moe_expand accepts for L layers, E experts and
   k ids per layer on the current device; 0 if none. */
s2moe_status s2moe_expand_max_nodes(int32_t n_layers, int32_t n_experts, int32_t k,
                                    int32_t *max_nodes);

/* Diagnostic, not a step of the verify pass: read `bytes` of device memory
   at `src` once, front to back, with the same 16-byte nontemporal loads the
   expert-FFN kernels stream weights with, so that the rate a caller times
   around it is what this GPU delivers to a plain sequential read.  `bytes`
   must be a nonzero multiple of 16 and `src` 16-byte aligned.  `sink` is a
   device buffer of S2MOE_STREAM_SINK_WORDS uint32; a prefix of it receives
   one checksum word per block (the XOR of all words the block read, so the
   XOR of that prefix is the XOR of the whole buffer).  Enqueued on
   `stream`. */
#define S2MOE_STREAM_SINK_WORDS 2048
s2moe_status s2moe_stream_read(const void *src, size_t bytes, uint32_t *sink, void *stream);

/* Message of the last failed call on this thread ("" if none). */
const char *s2moe_last_error(void);

/* Static name of a status code. */
const char *s2moe_status_string(s2moe_status status);

/* S2MOE_ABI_VERSION of the loaded library. */
int32_t s2moe_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* S2MOE_H */
