"""Seeded generators for the verify-MoE inputs.

Every array comes from its own NumPy PCG64 stream keyed by
(seed, workload id, layer, tensor, expert), so any subset of experts or layers
can be regenerated on its own and both the HIP path and the oracle see the same
stored bits.

Stored formats:
  * "f32"   : float32
  * "bf16"  : uint16 bit patterns (fp32 rounded to nearest-even, done here)
  * "q4g32" : uint8 [rows, K/2] holding two 4-bit codes per byte (element 2i
              in the low nibble, 2i+1 in the high nibble) and float16 scales
              [rows, K/32], one per 32 consecutive K elements.  The codes and
              scales are drawn directly; nothing here decodes them.

Hidden states follow x_b = sqrt(rho) * u + sqrt(1 - rho) * n_b with a shared
u and per-token n_b, both N(0, I); with router rows ~ N(0, 1/H) this gives
router logits of unit variance and cross-token correlation rho.  Confidence
weights come from a synthetic draft tree: chains of depth min(8, B), edge
confidences ~ Beta(5, 1) (concentrated near 1), and each token's weight the
product of the edge confidences on its path (the prefix confidence of Sec.
Routing-aware Adaptive Speculative Expansion, "Expected Benefit").
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import WORKLOAD_ID, LayerShape, Workload

# tensor ids used in the seed keys
T_XSHARED, T_XNOISE, T_ROUTER, T_GATE, T_UP, T_DOWN = 1, 2, 3, 4, 5, 6
T_CONF, T_RESAMPLE, T_SH_GATE, T_SH_UP, T_SH_DOWN, T_SCALE = 7, 8, 9, 10, 11, 12

_CHUNK = 1 << 24  # elements per conversion chunk (bounds temporaries)


def _rng(seed: int, *key: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=int(seed), spawn_key=tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest, ties to even (finite inputs)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    flat = a.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)
    for s in range(0, flat.size, _CHUNK):
        u = flat[s:s + _CHUNK].view(np.uint32)
        r = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
        out[s:s + _CHUNK] = (r >> np.uint32(16)).astype(np.uint16)
    return out.reshape(a.shape)


def _store(a32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(a32, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_from_f32(a32)
    raise ValueError(f"unsupported storage dtype {dtype!r}")


def _normal_store(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std^2) samples in the storage dtype, generated chunk by chunk."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32 if dtype == "f32" else np.uint16)
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        v = rng.standard_normal(m, dtype=np.float32)
        v *= np.float32(std)
        out[s:s + m] = v if dtype == "f32" else bf16_bits_from_f32(v)
    return out.reshape(shape)


def _q4_store(rng: np.random.Generator, rows: int, K: int, std: float):
    """Random 4-bit codes (uniform 0..15) and fp16 group scales.

    The scale is std / 4.61 with a +-25 % uniform jitter: the codes minus 8
    have an RMS of about 4.6, so the represented weights have std ~ `std`.
    """
    codes = rng.integers(0, 256, size=(rows, K // 2), dtype=np.uint8)
    jit = rng.random((rows, K // 32), dtype=np.float32)
    scales = (np.float32(std / 4.61) * (np.float32(0.75) + np.float32(0.5) * jit)).astype(np.float16)
    return codes, scales


def draft_tree_confidence(B: int, rng: np.random.Generator) -> np.ndarray:
    """Per-token confidence weights w_b of a synthetic draft tree.

    B tokens form ceil(B / D) chains of depth D = min(8, B); token b sits in
    chain b // D at depth b % D.  Edge confidences are Beta(5, 1) and w_b is
    the running product along the chain.
    """
    D = max(1, min(8, B))
    n_chains = -(-B // D)
    q = rng.beta(5.0, 1.0, size=(n_chains, D))
    w = np.cumprod(q, axis=1).reshape(-1)[:B]
    return w.astype(np.float32)


def make_router(shape: LayerShape, seed: int, layer: int = 0, wl_id: int = 0,
                std: float | None = None) -> np.ndarray:
    """Router weights W_r [E, H] in the activation dtype."""
    std = (1.0 / math.sqrt(shape.hidden)) if std is None else std
    rng = _rng(seed, wl_id, layer, T_ROUTER)
    return _normal_store(rng, (shape.n_experts, shape.hidden), std, shape.act)


def make_batch(shape: LayerShape, B: int, seed: int, layer: int = 0, wl_id: int = 0,
               rho: float = 0.0, reject=None, max_rounds: int = 1000):
    """Hidden states x [B, H] (activation dtype) and confidences w [B] (fp32).

    `reject(x_stored, conf_w) -> bool[B]`, if given, names tokens whose noise
    is redrawn (from a per-round sub-stream) until it returns no token; the
    caller supplies it (e.g. a routing-margin check), this module does not
    look at the values.  Returns (x, conf_w, rounds).
    """
    H = shape.hidden
    conf_w = draft_tree_confidence(B, _rng(seed, wl_id, layer, T_CONF))
    u = _rng(seed, wl_id, layer, T_XSHARED).standard_normal(H)
    noise = _rng(seed, wl_id, layer, T_XNOISE).standard_normal((B, H))
    a, c = math.sqrt(rho), math.sqrt(1.0 - rho)

    def assemble():
        x32 = (a * u[None, :] + c * noise).astype(np.float32)
        return _store(x32, shape.act)

    x = assemble()
    rounds = 0
    if reject is not None:
        while True:
            bad = np.asarray(reject(x, conf_w), dtype=bool)
            if not bad.any():
                break
            rounds += 1
            if rounds > max_rounds:
                raise RuntimeError(f"margin resampling did not converge in {max_rounds} rounds")
            for b in np.nonzero(bad)[0]:
                noise[b] = _rng(seed, wl_id, layer, T_RESAMPLE, rounds, int(b)).standard_normal(H)
            x = assemble()
    return x, conf_w, rounds


def _expert_tensors(shape: LayerShape, F: int, n: int, seed: int, layer: int, wl_id: int,
                    std: float, tids, experts):
    """gate/up [n, F, H] and down [n, H, F] (+ scales for q4g32)."""
    H, dt = shape.hidden, shape.wdt
    tg, tu, td = tids
    experts = list(range(n)) if experts is None else list(experts)
    m = len(experts)
    out = {}
    if dt == "q4g32":
        out["gate"] = np.empty((m, F, H // 2), np.uint8)
        out["up"] = np.empty((m, F, H // 2), np.uint8)
        out["down"] = np.empty((m, H, F // 2), np.uint8)
        out["gate_s"] = np.empty((m, F, H // 32), np.float16)
        out["up_s"] = np.empty((m, F, H // 32), np.float16)
        out["down_s"] = np.empty((m, H, F // 32), np.float16)
    else:
        sd = np.float32 if dt == "f32" else np.uint16
        out["gate"] = np.empty((m, F, H), sd)
        out["up"] = np.empty((m, F, H), sd)
        out["down"] = np.empty((m, H, F), sd)

    jobs = []
    for i, e in enumerate(experts):
        for name, tid, rows, K in (("gate", tg, F, H), ("up", tu, F, H), ("down", td, H, F)):
            jobs.append((i, e, name, tid, rows, K))

    def run(job):
        i, e, name, tid, rows, K = job
        rng = _rng(seed, wl_id, layer, tid, e)
        if dt == "q4g32":
            codes, scales = _q4_store(rng, rows, K, std)
            out[name][i] = codes
            out[name + "_s"][i] = scales
        else:
            out[name][i] = _normal_store(rng, (rows, K), std, dt)

    workers = max(1, min(8, os.cpu_count() or 1, len(jobs)))
    if workers == 1:
        for j in jobs:
            run(j)
    else:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(run, jobs))
    return out


def make_experts(shape: LayerShape, seed: int, layer: int = 0, wl_id: int = 0,
                 std: float = 0.02, experts=None) -> dict:
    """Routed-expert weights; `experts` picks a subset (same values as in the full set)."""
    return _expert_tensors(shape, shape.ffn, shape.n_experts, seed, layer, wl_id, std,
                           (T_GATE, T_UP, T_DOWN), experts)


def make_shared_experts(shape: LayerShape, seed: int, layer: int = 0, wl_id: int = 0,
                        std: float = 0.02) -> dict:
    """Shared-expert weights [S, F_s, H] / [S, H, F_s] (+ scales); {} when S = 0."""
    if shape.n_shared == 0:
        return {}
    return _expert_tensors(shape, shape.ffn_shared, shape.n_shared, seed, layer, wl_id, std,
                           (T_SH_GATE, T_SH_UP, T_SH_DOWN), None)


def workload_inputs(wl: Workload, B: int, seed: int, layer: int = 0, reject=None,
                    with_experts: bool = True, experts=None) -> dict:
    """All inputs of one layer of a named workload, as a dict of host arrays."""
    wid = WORKLOAD_ID[wl.name]
    sh = wl.shape
    router = make_router(sh, seed, layer, wid, wl.router_std)
    rej = None if reject is None else (lambda x, w: reject(x, w, router))
    x, conf_w, rounds = make_batch(sh, B, seed, layer, wid, wl.rho, rej)
    d = {"x": x, "conf_w": conf_w, "router": router, "resample_rounds": rounds}
    if with_experts:
        d["experts"] = make_experts(sh, seed, layer, wid, wl.w_std, experts)
        d["shared"] = make_shared_experts(sh, seed, layer, wid, wl.w_std)
    return d
