"""fp64 CPU oracle of the S2-MoE verify-MoE pass.

TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the benchmark's
CPU-baseline leg use this module.  It shares no code with the HIP library and
neither imports the other; both consume the arrays of `synth`.

What it computes, in the paper's order (Sec. "Reuse-aware Expert Gating"):

  route       ell_b = W_r x_b (target gating logits), plain top-k of ell_b and
              gap_b = ell_(1) - ell_(k+1), the margin between the top-1 and
              the (k+1)-th expert ("Soft routing bias for reuse promotion").
  reuse_gate  w_b = max(conf_w_b, 0) (non-negative confidence weights),
              g_e = sum_b w_b ell_{b,e} (Eq. cross-token expert importance),
              E* = TopCap(g) with |E*| <= cap ("Global preferred expert
              selection"), lambda_b = alpha * gap_b,
              ell'_{b,e} = ell_{b,e} + lambda_b [e in E*] (soft routing bias),
              biased top-k of ell'_b, gate weights softmax over the selected
              experts of the original ell_b, and the token->expert buckets.
  verify_moe  for each activated expert, the SwiGLU FFN
              W_d (silu(W_g x) * (W_u x)) of every token routed to it, and of
              all tokens for each shared expert.
  combine     y_b = sum_j gate_w_{b,j} FFN_{idx_{b,j}}(x_b) + sum_s FFN_s(x_b).

Readings where the paper is silent (all are flags or fixed choices here):
  * ell are raw pre-softmax router logits; gap is taken on them as well.
  * confidences below 0 are clamped to 0; if none is positive no bias is
    applied (E* is empty and the biased top-k is the plain top-k).
  * TopCap takes exactly `cap` experts over all E by default; with
    PREF_ACTIVATED_ONLY only experts in some token's plain top-k compete.
  * lambda_b = alpha * gap_b (alpha >= 0); BIAS_ABSOLUTE gives lambda_b = alpha.
  * gate weights are a softmax of the original logits over the selected k
    (they sum to 1); GATE_FROM_BIASED uses the biased logits instead.
  * every ranking orders by value descending, then expert index ascending;
    idx rows list the selected experts in ascending expert id.
  * the reuse ratio is |U| / (B k): unique activated routed experts over the
    expert activations autoregressive decoding of the same B tokens would make
    (Sec. Motivation, Challenge 2).
  * int4 weights: w = s * (q - 8), q the 4-bit code (element 2i in the low
    nibble of byte i), s the fp16 scale of its 32-element group.

Stored inputs are upcast exactly (bf16 bits -> fp64, fp16 -> fp64) before any
arithmetic; all arithmetic is fp64.
"""

from __future__ import annotations

import numpy as np

PREF_ACTIVATED_ONLY = 1
BIAS_ABSOLUTE = 2
GATE_FROM_BIASED = 4


# --------------------------------------------------------------------------
# exact upcasts of the stored formats
# --------------------------------------------------------------------------
def upcast(a, dtype: str) -> np.ndarray:
    """Stored array -> fp64, exactly."""
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"no upcast for {dtype!r}")


def dequant_q4g32(codes, scales) -> np.ndarray:
    """int4 codes [rows, K/2] + fp16 scales [rows, K/32] -> fp64 [rows, K]."""
    codes = np.asarray(codes, dtype=np.uint8)
    rows, half = codes.shape
    K = 2 * half
    q = np.empty((rows, K), dtype=np.float64)
    q[:, 0::2] = codes & 0x0F
    q[:, 1::2] = codes >> 4
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    assert s.shape == (rows, K // 32)
    return (q - 8.0) * np.repeat(s, 32, axis=1)


def expert_matrix(store: dict, name: str, e: int, wdt: str) -> np.ndarray:
    """One expert's weight matrix (gate, up or down) in fp64."""
    if wdt == "q4g32":
        return dequant_q4g32(store[name][e], store[name + "_s"][e])
    return upcast(store[name][e], wdt)


# --------------------------------------------------------------------------
# rankings
# --------------------------------------------------------------------------
def rank_order(values) -> np.ndarray:
    """Indices ordered by value descending, ties by index ascending."""
    v = np.asarray(values, dtype=np.float64)
    return np.lexsort((np.arange(v.size), -v))


def top_k_ascending(values, k: int) -> np.ndarray:
    """The k best indices under rank_order, listed in ascending index."""
    return np.sort(rank_order(values)[:k]).astype(np.int32)


# --------------------------------------------------------------------------
# the four steps
# --------------------------------------------------------------------------
def route(x, router, k: int, act: str) -> dict:
    """Router logits, plain top-k and the top-1 / (k+1)-th gap."""
    X = upcast(x, act)
    W = upcast(router, act)
    logits = X @ W.T                                   # ell_b = W_r x_b
    B, E = logits.shape
    if not 1 <= k < E:
        raise ValueError("need 1 <= k < E")
    plain_idx = np.empty((B, k), dtype=np.int32)
    gap = np.empty(B, dtype=np.float64)
    for b in range(B):
        o = rank_order(logits[b])
        plain_idx[b] = np.sort(o[:k])
        gap[b] = logits[b, o[0]] - logits[b, o[k]]
    return {"logits": logits, "gap": gap, "plain_idx": plain_idx}


def reuse_gate(logits, gap, plain_idx, conf_w, k: int, cap: int, alpha: float,
               flags: int = 0) -> dict:
    """Reuse-aware expert gating and token->expert bucketing."""
    ell = np.asarray(logits, dtype=np.float64)
    B, E = ell.shape
    if not (k <= cap <= E):
        raise ValueError("need k <= cap <= E")
    w = np.maximum(np.asarray(conf_w, dtype=np.float64), 0.0)
    active = bool(np.any(w > 0.0))

    # cross-token expert importance: g_e = sum_b w_b * ell_{b,e}
    g = np.zeros(E)
    for b in range(B):
        g += w[b] * ell[b]

    # globally preferred experts E* = TopCap(g)
    pref = np.zeros(E, dtype=np.int32)
    if active:
        if flags & PREF_ACTIVATED_ONLY:
            cand = np.unique(np.asarray(plain_idx).reshape(-1))
        else:
            cand = np.arange(E)
        chosen = cand[rank_order(g[cand])][:cap]
        pref[chosen] = 1

    # token-adaptive bias lambda_b, proportional to the top-1 / (k+1)-th gap
    if not active:
        lam = np.zeros(B)
    elif flags & BIAS_ABSOLUTE:
        lam = np.full(B, float(alpha))
    else:
        lam = float(alpha) * np.asarray(gap, dtype=np.float64)
    biased = ell.copy()
    for b in range(B):
        for e in range(E):
            if pref[e]:
                biased[b, e] = ell[b, e] + lam[b]

    # biased top-k and gate weights
    src = biased if flags & GATE_FROM_BIASED else ell
    idx = np.empty((B, k), dtype=np.int32)
    gate_w = np.empty((B, k), dtype=np.float64)
    for b in range(B):
        sel = top_k_ascending(biased[b], k)
        idx[b] = sel
        z = src[b, sel]
        ez = np.exp(z - z.max())
        gate_w[b] = ez / ez.sum()

    bk = bucket(idx, E)
    out = {"g": g, "pref": pref, "lam": lam, "biased": biased, "idx": idx,
           "gate_w": gate_w}
    out.update(bk)
    return out


def bucket(idx, E: int) -> dict:
    """Expert-major stable list of the (token, slot) assignments a = b*k + j."""
    flat = np.asarray(idx, dtype=np.int64).reshape(-1)
    n = flat.size
    count = np.zeros(E, dtype=np.int32)
    for a in range(n):
        count[flat[a]] += 1
    offset = np.zeros(E + 1, dtype=np.int32)
    for e in range(E):
        offset[e + 1] = offset[e] + count[e]
    slot = np.empty(n, dtype=np.int32)
    fill = offset[:E].copy()
    for a in range(n):
        e = flat[a]
        slot[fill[e]] = a
        fill[e] += 1
    uniq = np.full(E, -1, dtype=np.int32)
    n_uniq = 0
    for e in range(E):
        if count[e] > 0:
            uniq[n_uniq] = e
            n_uniq += 1
    return {"count": count, "offset": offset, "slot": slot, "uniq": uniq,
            "n_uniq": n_uniq, "reuse_ratio": n_uniq / n if n else 0.0}


def silu(z):
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu_ffn(X, Wg, Wu, Wd):
    """W_d (silu(W_g x) * (W_u x)) for each row x of X."""
    return (silu(X @ Wg.T) * (X @ Wu.T)) @ Wd.T


def verify_moe(x, experts: dict, shared: dict, gate: dict, k: int, act: str,
               wdt: str, n_shared: int = 0) -> np.ndarray:
    """Unscaled expert outputs: row b*k+j for the j-th routed expert of token
    b, then row B*k + s*B + b for shared expert s."""
    X = upcast(x, act)
    B, H = X.shape
    out = np.zeros((B * k + n_shared * B, H))
    flat = np.asarray(gate["idx"]).reshape(-1)
    for e in np.unique(flat):                 # each activated expert once
        rows = np.nonzero(flat == e)[0]       # assignments a = b*k + j
        toks = rows // k
        Wg = expert_matrix(experts, "gate", int(e), wdt)
        Wu = expert_matrix(experts, "up", int(e), wdt)
        Wd = expert_matrix(experts, "down", int(e), wdt)
        out[rows] = swiglu_ffn(X[toks], Wg, Wu, Wd)
    for s in range(n_shared):
        Wg = expert_matrix(shared, "gate", s, wdt)
        Wu = expert_matrix(shared, "up", s, wdt)
        Wd = expert_matrix(shared, "down", s, wdt)
        out[B * k + s * B: B * k + (s + 1) * B] = swiglu_ffn(X, Wg, Wu, Wd)
    return out


def combine(gate_w, expert_out, k: int, n_shared: int = 0) -> np.ndarray:
    """y_b = sum_j gate_w_{b,j} out_{b*k+j} + sum_s out_{B*k+s*B+b}."""
    gw = np.asarray(gate_w, dtype=np.float64)
    B = gw.shape[0]
    eo = np.asarray(expert_out, dtype=np.float64)
    y = np.zeros((B, eo.shape[1]))
    for b in range(B):
        acc = np.zeros(eo.shape[1])
        for j in range(k):
            acc = acc + gw[b, j] * eo[b * k + j]
        for s in range(n_shared):
            acc = acc + eo[B * k + s * B + b]
        y[b] = acc
    return y


def forward(x, router, conf_w, experts, shared, shape) -> dict:
    """route -> reuse_gate -> verify_moe -> combine for one layer."""
    r = route(x, router, shape.top_k, shape.act)
    gt = reuse_gate(r["logits"], r["gap"], r["plain_idx"], conf_w, shape.top_k,
                    shape.cap, shape.alpha, shape.flags)
    eo = verify_moe(x, experts, shared, gt, shape.top_k, shape.act, shape.wdt,
                    shape.n_shared)
    y = combine(gt["gate_w"], eo, shape.top_k, shape.n_shared)
    out = dict(r)
    out.update(gt)
    out["expert_out"] = eo
    out["y"] = y
    return out


# --------------------------------------------------------------------------
# margins (used by tests to draw inputs whose routing is well posed in fp32)
# --------------------------------------------------------------------------
def routing_margins(logits, conf_w, k: int, cap: int, alphas, flags: int = 0) -> dict:
    """Distances to the nearest decision flip of every ranking the pass makes.

    plain[b]       = ell_(k) - ell_(k+1) of token b
    biased[a][b]   = ell'_(k) - ell'_(k+1) of token b at alpha = alphas[a]
    cap_margin     = g_(cap) - g_(cap+1) among the TopCap candidates
                     (inf when every candidate is selected)
    """
    ell = np.asarray(logits, dtype=np.float64)
    B, E = ell.shape
    r = {"plain": np.empty(B)}
    plain_idx = np.empty((B, k), dtype=np.int32)
    gap = np.empty(B)
    for b in range(B):
        o = rank_order(ell[b])
        srt = ell[b, o]
        r["plain"][b] = srt[k - 1] - srt[k]
        plain_idx[b] = np.sort(o[:k])
        gap[b] = srt[0] - srt[k]
    w = np.maximum(np.asarray(conf_w, dtype=np.float64), 0.0)
    g = np.zeros(E)
    for b in range(B):
        g += w[b] * ell[b]
    cand = (np.unique(plain_idx) if flags & PREF_ACTIVATED_ONLY else np.arange(E))
    gs = np.sort(g[cand])[::-1]
    r["cap_margin"] = (gs[cap - 1] - gs[cap]) if cand.size > cap else np.inf
    r["biased"] = []
    for a in alphas:
        gt = reuse_gate(ell, gap, plain_idx, conf_w, k, cap, a, flags)
        m = np.empty(B)
        for b in range(B):
            s = np.sort(gt["biased"][b])[::-1]
            m[b] = s[k - 1] - s[k]
        r["biased"].append(m)
    return r


def reuse_improvement(ratio_without: float, ratio_with: float) -> float:
    """Relative reduction of the reuse ratio, in percent (Table "Effect of
    reuse-aware expert gating on expert parameter reuse")."""
    return 100.0 * (ratio_without - ratio_with) / ratio_without


def margin_reject(k: int, cap: int, alphas, act: str, flags: int = 0,
                  margin: float = 1e-3):
    """Callback for synth.make_batch: tokens to redraw so that every ranking
    decision (plain top-k, TopCap, biased top-k at each alpha) is separated by
    at least `margin` in fp64 on the stored inputs.  When only the TopCap
    boundary fails, the token with the largest confidence is redrawn (it moves
    g the most)."""

    def reject(x, conf_w, router):
        logits = upcast(x, act) @ upcast(router, act).T
        m = routing_margins(logits, conf_w, k, cap, alphas, flags)
        bad = m["plain"] < margin
        for bm in m["biased"]:
            bad |= bm < margin
        if m["cap_margin"] < margin and not bad.any():
            bad[int(np.argmax(np.asarray(conf_w)))] = True
        return bad

    return reject
