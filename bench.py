"""Verify-MoE layer benchmark on one MI355X.

A step is one full pass of the hot path -- route, reuse-aware gating, grouped
SwiGLU experts, combine -- over one verify batch of synthetic draft tokens,
enqueued back to back on one HIP stream with all inputs resident in HBM.

    python bench.py [--steps K] [--warmup W] [--workload c2]

Prints one JSON line.  `value` is draft tokens per second of whole steps;
`roofline` covers the expert-FFN launches of s2moe_verify_moe (gate-up and
down), timed with one pair of HIP events on the stream they run on around
back-to-back calls, against the unique expert weight bytes a call must read.
The calls cycle through copies of the expert weights that together exceed
the 256 MB last-level cache, so no weight byte is served from cache.
`stream_read` is a plain read-only pass over 2 GiB on the same GPU (what the
GPU delivers to a simple streaming read), and `cpu_baseline` times the fp64
oracle on the host cores for the same step, repeated for about 10 s.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E


# The oracle baselines repeat their sample until about this many seconds of
# host work have passed (at least once, at most ORACLE_MAX_REPS times).
ORACLE_MIN_S = 10.0
ORACLE_MAX_REPS = 1000


def time_oracle(fn) -> tuple[int, float]:
    """Calls fn() until ORACLE_MIN_S seconds have passed; returns (calls, seconds)."""
    t = time.perf_counter()
    reps = 0
    while reps < 1 or (time.perf_counter() - t < ORACLE_MIN_S and reps < ORACLE_MAX_REPS):
        fn()
        reps += 1
    return reps, time.perf_counter() - t


# Timed launches cycle through input copies totalling more than this, so
# that the 256 MB Infinity Cache cannot hold them between launches.
ROTATE_BYTES = 600_000_000


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def expert_bytes(shape, F: int) -> int:
    """HBM bytes of one expert's gate, up and down weights (int4 scales included)."""
    n = 3 * F * shape.hidden
    if shape.wdt == "bf16":
        return 2 * n
    if shape.wdt == "f32":
        return 4 * n
    return n // 2 + 2 * (n // 32)  # 4-bit codes + one fp16 scale per 32


FFN_SOURCES = {
    "bf16": ["ffn_bf16.hip", "ffn_common.h", "common.h", "kernels.h"],
    "q4g32": ["ffn_q4.hip", "ffn_common.h", "common.h", "kernels.h"],
    "f32": ["ffn.hip", "ffn_common.h", "common.h", "kernels.h"],
}


def _code_only(data: bytes) -> bytes:
    """C/C++ source without comments, whitespace runs collapsed: a comment
    edit leaves the hash of a kernel's sources unchanged."""
    import re
    data = re.sub(rb"/\*.*?\*/", b" ", data, flags=re.S)
    data = re.sub(rb"//[^\n]*", b"", data)
    return b" ".join(data.split())


def ffn_source_hash(wdt: str) -> str:
    """sha256 of the code (comments removed) of the sources the expert-FFN
    kernels of this weight format are built from (identifies the kernel a
    traffic measurement belongs to).  Of kernels.h only the FfnArgs
    definition counts, and for int4 weights also the K-part count of the
    down projection (q4_down_parts): the rest declares other kernels."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in FFN_SOURCES[wdt]:
        with open(os.path.join(ROOT, "paper_2608_15018_amd", "csrc", f), "rb") as fh:
            data = fh.read()
        if f == "kernels.h":
            parts = [rb"struct FfnArgs \{.*?\n\};"]
            if wdt == "q4g32":
                parts.append(rb"#ifndef S2MOE_Q4_DOWN_R.*?inline int q4_down_parts\(.*?\n\}")
            found = [re.search(p, data, re.S) for p in parts]
            data = b"".join(m.group(0) for m in found) if all(found) else data
        h.update(_code_only(data))
    return h.hexdigest()


def expand_source_hash() -> str:
    """sha256 of the code (comments removed) of expand.hip, common.h and the
    ExpandArgs / expand layout definitions of kernels.h (the sources of the
    s2moe_expand kernel)."""
    import hashlib
    import re
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_15018_amd", "csrc")
    for f in ("expand.hip", "common.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(_code_only(fh.read()))
    with open(os.path.join(csrc, "kernels.h"), "rb") as fh:
        data = fh.read()
    for pat in (rb"struct ExpandArgs \{.*?\n\};", rb"struct ExpandLds \{.*?(?=hipError_t launch_expand)"):
        m = re.search(pat, data, re.S)
        h.update(_code_only(m.group(0) if m else data))
    return h.hexdigest()


def _traffic_record(path: str, src_hash: str):
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            key, _, v = line.strip().lstrip("- ").partition(":")
            if key in ("traffic_bytes_per_launch", "kernel_source_sha256"):
                vals[key] = v.strip().strip("`")
    if vals.get("kernel_source_sha256") != src_hash:
        return None
    try:
        return int(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def recorded_expand_traffic(name: str, trees: int):
    """HBM bytes per s2moe_expand launch of `trees` trees of this workload
    from the committed rocprofv3 counter summary, or None if there is none
    or the kernel changed since it was taken."""
    return _traffic_record(os.path.join(ROOT, "profiles", f"expand_{name}_{trees}_traffic.md"),
                           expand_source_hash())


def recorded_traffic(name: str, wdt: str, B: int, default_B: int):
    """HBM bytes per s2moe_verify_moe call from the committed rocprofv3 counter
    summary of this workload at B draft tokens (verify_moe_<name>_b<B>_traffic.md,
    or verify_moe_<name>_traffic.md at the workload's default B), or None if
    there is none or the kernel sources changed since it was taken."""
    names = [f"verify_moe_{name}_b{B}_traffic.md"]
    if B == default_B:
        names.append(f"verify_moe_{name}_traffic.md")
    for n in names:
        v = _traffic_record(os.path.join(ROOT, "profiles", n), ffn_source_hash(wdt))
        if v is not None:
            return v
    return None


# Warm-up lasts at least this long: the shader clock settles under load
# over a few hundred microseconds to milliseconds, and the int4 kernels,
# bound by instruction issue, follow it.
WARMUP_MIN_S = 0.2


def warm(fn, steps: int):
    """Run fn() at least max(1, steps) times and until WARMUP_MIN_S of GPU
    time has passed (untimed)."""
    import torch
    n, t0 = 0, time.perf_counter()
    while n < max(1, steps) or time.perf_counter() - t0 < WARMUP_MIN_S:
        fn()
        n += 1
        if n % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    return n


def _head_start():
    """Queue a short GPU spin so that the host enqueues the timed launches
    while the GPU is still busy: the events then bracket kernels that run
    back to back instead of measuring how fast Python issues launches."""
    import torch
    torch.cuda._sleep(5_000_000)


def expand_bytes(d: dict, L: int, k: int) -> int:
    """Algorithmic HBM bytes of one s2moe_expand launch: each tree's node
    records (parent, q, C^draft: 12 B) and predicted expert ids (L*k int32)
    for its n_t nodes, the root's ids and n_nodes read once; order, util and
    n_new (16 B per padded node) and the three per-tree counts written."""
    T, N = d["parent"].shape
    nodes = int(d["n_nodes"].sum())
    return nodes * (12 + 4 * L * k) + T * (4 * L * k + 4) + T * N * 16 + T * 12


def bench_expand(args) -> int:
    """Routing-aware adaptive expansion: `--trees` draft trees of the named
    model shape per s2moe_expand launch."""
    import torch

    import paper_2608_15018_amd as s2
    from synth.trees import TREE_WORKLOADS, make_trees

    wl = TREE_WORKLOADS[args.workload]
    T = args.trees
    t0 = time.time()
    d = make_trees(wl, T, args.seed)
    _log(f"[bench] {T} trees generated in {time.time() - t0:.1f}s")
    dev = {k: torch.from_numpy(v).cuda() for k, v in d.items()}
    N, L, k = wl.max_nodes, wl.n_layers, wl.k
    out = s2.ExpandOut(T, N)
    stream = torch.cuda.current_stream()

    def launch(o=out, dd=dev):
        s2.expand(dd["parent"], dd["q"], dd["eid"], dd["c_draft"], dd["n_nodes"], o,
                  wl.n_experts, wl.t_ar, wl.t_exp, root_eid=dd["root_eid"])

    warm(launch, args.warmup)
    res = out.host()

    # Timed: K back-to-back launches between one pair of HIP events on the
    # launch stream, cycling through copies of the trees that together exceed
    # the 256 MB Infinity Cache, so every launch reads its ids from HBM.
    nbytes = expand_bytes(d, L, k)
    copies = 1 if args.no_scrub else max(1, min(64, -(-ROTATE_BYTES // nbytes)))
    devs = [dev] + [{kk: v.clone() for kk, v in dev.items()} for _ in range(copies - 1)]
    for dd in devs:
        launch(out, dd)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    _head_start()
    t_start = time.perf_counter()
    e0.record(stream)
    for i in range(args.steps):
        launch(out, devs[i % copies])
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    avg_s = e0.elapsed_time(e1) / 1e3 / args.steps
    achieved = nbytes / avg_s / 1e9
    del devs

    # One tree per launch: the latency a single request sees.
    one = {kk: v[:1].contiguous() for kk, v in dev.items()}
    o1 = s2.ExpandOut(1, N)
    for _ in range(3):
        launch(o1, one)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    _head_start()
    e0.record(stream)
    for _ in range(20):
        launch(o1, one)
    e1.record(stream)
    torch.cuda.synchronize()
    one_us = e0.elapsed_time(e1) / 20 * 1e3

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import expand_oracle
        t = time.perf_counter()
        done = 0
        while done < T and (done < 8 or time.perf_counter() - t < 10.0):
            sl = slice(done, done + 1)
            expand_oracle.expand(d["parent"][sl], d["q"][sl], d["eid"][sl], d["c_draft"][sl],
                                 wl.n_experts, wl.t_ar, wl.t_exp, d["root_eid"][sl],
                                 d["n_nodes"][sl])
            done += 1
        dt = time.perf_counter() - t
        cpu = {"value": done / dt, "unit": "draft trees/s", "cores": 1, "kind": "oracle",
               "sample": f"the first {done} trees of the batch, one at a time, pure Python "
                         f"sets, {dt:.1f}s"}

    line = {
        "metric": "routing-aware expansion: draft trees/s (Eq. U greedy selection per tree)",
        "value": T / avg_s,
        "unit": "draft trees/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": avg_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32 ids, fp64 utilities",
        "data": "synthetic",
        "config": {"workload": wl.description, "name": wl.name, "trees": T, "max_nodes": N,
                   "layers": L, "experts": wl.n_experts, "k": k, "t_ar": wl.t_ar,
                   "t_exp": wl.t_exp, "c_draft": wl.c_draft},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": recorded_expand_traffic(wl.name, T),
                     "kernel": "s2moe_expand", "bytes_per_launch": nbytes,
                     "avg_launch_us": avg_s * 1e6},
        "cpu_baseline": cpu,
        "timing": f"one event pair around {args.steps} back-to-back launches over {copies} "
                  f"input cop{'y' if copies == 1 else 'ies'}",
        "wall_ms_per_step_incl_head_start": wall / args.steps * 1e3,
        "one_tree_us": one_us,
        "mean_nodes": float(d["n_nodes"].mean()),
        "mean_selected": float(res["n_admit"].mean()),
        "mean_union_pairs": float(res["n_pairs"].mean()),
    }
    print(json.dumps(line), flush=True)
    return 0


def bench_draft(args) -> int:
    """Expert-sparse draft step: every MoE layer of the model at k_draft
    experts per token, B = --batch tokens, eager and replayed from a HIP
    graph.  The layers cycle through 8 distinct weight sets drawn on the
    device (each set is far larger than the caches), and each layer has its
    own hidden states and router."""
    import torch

    import paper_2608_15018_amd as s2
    from paper_2608_15018_amd import draft
    from synth import device_gen

    name = args.workload[2:]
    m = draft.DRAFT_MODELS[name]
    B, wdt, L = args.batch or 1, args.wdt, m["layers"]
    H, F, E, k = m["hidden"], m["ffn"], m["n_experts"], m["k_draft"]
    S, Fs = m.get("n_shared", 0), m.get("ffn_shared", 0)
    layer = draft.draft_layer(name, wdt)
    n_sets = min(L, 8)
    t0 = time.time()
    sets = []
    for j in range(n_sets):
        ex = device_gen.expert_weights(E, F, H, wdt, args.seed, j)
        sh = device_gen.expert_weights(S, Fs, H, wdt, args.seed, j, tag=1) if S else {}
        dev, w = s2.pack_expert_weights((ex, sh), wdt)
        del ex, sh
        sets.append((dev, w))
    inputs = [(device_gen.activations(B, H, args.seed, l, rho=0.3),
               device_gen.router(E, H, args.seed, l), sets[l % n_sets][1]) for l in range(L)]
    torch.cuda.synchronize()
    _log(f"[bench] draft {name}: {n_sets} weight sets, {L} layers in {time.time() - t0:.1f}s")
    step = draft.DraftStep(layer, B, inputs)
    warm(step, args.warmup)
    n_uniq = [int(p.rt.n_uniq.item()) for p in step.passes]
    e_bytes = expert_bytes(layer_shape_of(m, wdt), F)
    s_bytes = expert_bytes(layer_shape_of(m, wdt), Fs) if S else 0
    nbytes = sum(n_uniq) * e_bytes + L * S * s_bytes

    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    _head_start()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    eager_s = e0.elapsed_time(e1) / 1e3 / args.steps
    step.capture()
    step.replay()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    graph_s = e0.elapsed_time(e1) / 1e3 / args.steps
    achieved = nbytes / graph_s / 1e9
    # The same step with every layer as four separate calls (route,
    # reuse_gate, verify_moe, combine), replayed from its own graph.
    step4 = draft.DraftStep(layer, B, inputs, fused=False)
    step4.capture()
    step4.replay()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step4.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    graph4_s = e0.elapsed_time(e1) / 1e3 / args.steps
    del step4

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        from synth.configs import LayerShape
        bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)  # noqa: E731
        shape = LayerShape(hidden=H, ffn=F, n_experts=E, top_k=k, cap=k, alpha=0.0, n_shared=S,
                           ffn_shared=Fs, act="bf16", wdt="bf16")
        if wdt == "bf16":
            x, router, _ = inputs[0]
            p0 = step.passes[0]
            used = p0.rt.uniq[: n_uniq[0]]
            dev = sets[0][0]
            ex_raw = device_gen.expert_weights(E, F, H, wdt, args.seed, 0)
            experts = {n: np.zeros((E,) + tuple(v.shape[1:]), np.uint16) for n, v in ex_raw.items()}
            for n, v in ex_raw.items():
                experts[n][used.cpu().numpy()] = bits(v[used.long()])
            del ex_raw
            shared = {n: bits(v) for n, v in (device_gen.expert_weights(
                S, Fs, H, wdt, args.seed, 0, tag=1).items() if S else [])}
            xb, rb, cw = bits(x), bits(router), np.ones(B, np.float32)
            reps, dt = time_oracle(lambda: oracle.forward(xb, rb, cw, experts, shared, shape))
            cpu = {"value": reps * B / (dt * L), "unit": "draft tokens/s", "cores": os.cpu_count(),
                   "kind": "oracle", "sample": f"layer 0 of the step in fp64 numpy, {reps} times "
                                              f"({dt:.1f}s), scaled to {L} layers"}

    line = {
        "metric": "expert-sparse draft step: draft tokens/s over all MoE layers",
        "value": B / graph_s,
        "unit": "draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": graph_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "q4g32": "int4-g32/bf16"}[wdt],
        "data": "synthetic",
        "config": {"workload": f"{name}-shaped draft step: {L} MoE layers, H {H}, F {F}, "
                               f"{E} experts, k_draft {k}" + (f", {S} shared" if S else ""),
                   "name": args.workload, "draft_tokens": B, "layers": L, "k_draft": k,
                   "weights": wdt, "weight_sets": n_sets},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "draft step (route, gate, experts, combine per layer; HIP graph)",
                     "bytes_per_launch": nbytes, "avg_launch_us": graph_s * 1e6},
        "cpu_baseline": cpu,
        "eager_ms_per_step": eager_s * 1e3,
        "four_call_graph_ms_per_step": graph4_s * 1e3,
        "graph_speedup": eager_s / graph_s,
        "experts_per_step": sum(n_uniq),
    }
    print(json.dumps(line), flush=True)
    return 0


def layer_shape_of(m: dict, wdt: str):
    from synth.configs import LayerShape
    return LayerShape(hidden=m["hidden"], ffn=m["ffn"], n_experts=m["n_experts"],
                      top_k=m["k_draft"], cap=m["k_draft"], alpha=0.0,
                      n_shared=m.get("n_shared", 0), ffn_shared=m.get("ffn_shared", 0),
                      act="bf16", wdt=wdt)


def bench_stack(args, wl, shape, B: int, wid: int) -> int:
    """`--layers L` layers of a verify-MoE workload run back to back, each with
    its own router, hidden states and confidences (the host generator, per
    layer) and its own expert weights (drawn on the device: the 24-layer int4
    stack holds 19 GB), all packed.  A step is one full pass (route, gate,
    experts, combine) through every layer; the FFN roofline covers the expert
    launches of all layers, which stream far more than the caches hold."""
    import torch

    import paper_2608_15018_amd as s2
    from synth import device_gen, gen

    L = args.layers
    if L > wl.n_layers:
        raise SystemExit(f"{wl.name} has {wl.n_layers} layer(s)")
    E, F, H, S, Fs = shape.n_experts, shape.ffn, shape.hidden, shape.n_shared, shape.ffn_shared
    layer = s2.make_layer(shape, flags=shape.flags | s2.PACKED_WEIGHTS)
    t0 = time.time()
    keep, passes, ins = [], [], []
    for l in range(L):
        router = gen.make_router(shape, args.seed, l, wid, wl.router_std)
        x, conf_w, _ = gen.make_batch(shape, B, args.seed, l, wid, wl.rho)
        ex = device_gen.expert_weights(E, F, H, shape.wdt, args.seed, l, std=wl.w_std)
        sh = device_gen.expert_weights(S, Fs, H, shape.wdt, args.seed, l, tag=1,
                                       std=wl.w_std) if S else {}
        dev, w = s2.pack_expert_weights((ex, sh), shape.wdt)
        del ex, sh
        keep.append(dev)
        passes.append(s2.VerifyPass(layer, B, fused=True))
        ins.append((s2.to_device(x), s2.to_device(router), s2.to_device(conf_w), w))
    torch.cuda.synchronize()
    _log(f"[bench] {wl.name}: {L} layers generated and packed in {time.time() - t0:.1f}s")

    def step():
        for p, (x, r, c, w) in zip(passes, ins):
            p(x, r, c, w)

    warm(step, args.warmup)
    n_uniq = [int(p.rt.n_uniq.item()) for p in passes]
    nbytes = sum(n_uniq) * expert_bytes(shape, F) + L * S * expert_bytes(shape, Fs)

    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start

    # The expert launches alone: every layer's s2moe_verify_moe, back to back,
    # between one pair of HIP events on the launch stream.
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    _head_start()
    e0.record(stream)
    for _ in range(args.steps):
        for p, (x, _r, _c, w) in zip(passes, ins):
            p.verify_moe(x, w)
    e1.record(stream)
    torch.cuda.synchronize()
    ffn_s = e0.elapsed_time(e1) / 1e3 / args.steps  # per pass through the L layers
    achieved = nbytes / ffn_s / 1e9

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        router = gen.make_router(shape, args.seed, 0, wid, wl.router_std)
        x, conf_w, _ = gen.make_batch(shape, B, args.seed, 0, wid, wl.rho)
        experts = gen.make_experts(shape, args.seed, 0, wid, wl.w_std)
        shared = gen.make_shared_experts(shape, args.seed, 0, wid, wl.w_std)
        reps, dt = time_oracle(lambda: oracle.forward(x, router, conf_w, experts, shared, shape))
        try:
            from threadpoolctl import threadpool_info
            cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        except Exception:  # pragma: no cover
            cores = os.cpu_count()
        cpu = {"value": reps * B / (dt * L), "unit": "draft tokens/s", "cores": cores,
               "kind": "oracle",
               "sample": f"one layer (layer 0, B={B}) of the {L}-layer stack, fp64 numpy, "
                         f"{reps} times ({dt:.1f}s), scaled by {L} layers"}

    out = {
        "metric": "verify-MoE layer: draft tokens/s and achieved HBM GB/s (% of peak) on "
                  "unique experts",
        "value": B * args.steps / elapsed,
        "unit": "draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "f32": "f32", "q4g32": "int4-g32/bf16"}[shape.wdt],
        "data": "synthetic",
        "config": {"workload": wl.description + f" ({L} layers, each its own inputs and weights)",
                   "name": wl.name, "draft_tokens": B, "layers": L,
                   "hidden": H, "ffn": F, "experts": E, "top_k": shape.top_k, "shared": S,
                   "cap": shape.cap, "alpha": shape.alpha, "weights": "packed"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": f"s2moe_verify_moe (expert gate-up + down launches, {L} layers)",
                     "bytes_per_launch": nbytes / L, "avg_launch_us": ffn_s / L * 1e6},
        "cpu_baseline": cpu,
        "n_uniq_per_layer": n_uniq,
        "ffn_timing": f"one event pair around {args.steps} passes through the {L} layers",
        "ms_per_layer": elapsed / args.steps / L * 1e3,
    }
    print(json.dumps(out), flush=True)
    return 0


def stream_read_gbs() -> float:
    """GB/s of s2moe_stream_read over 2 GiB (5 passes between one event pair)."""
    import torch

    import paper_2608_15018_amd as s2
    stream = torch.cuda.current_stream()
    buf = torch.ones(1 << 29, dtype=torch.float32, device="cuda")
    sink = torch.empty(s2.STREAM_SINK_WORDS, dtype=torch.int32, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s2.stream_read(buf, sink)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(5):
        s2.stream_read(buf, sink)
    e1.record(stream)
    torch.cuda.synchronize()
    gbs = 5 * buf.numel() * 4 / (e0.elapsed_time(e1) / 1e3) / 1e9
    del buf, sink
    return gbs


# Extra single-GPU configurations measured by the default run beside the
# headline workload: the Mixtral-shaped int4-g32 layer at 16 and 64 draft
# tokens (layer 0 of the 24-layer stack).
EXTRA_CONFIGS = (("c5", 16), ("c5", 64))


def extra_configs(args) -> dict:
    """FFN roofline of each EXTRA_CONFIGS workload, timed in this run."""
    import gc

    import torch

    from synth.configs import WORKLOAD_ID, WORKLOADS
    res = {}
    for name, B in EXTRA_CONFIGS:
        wl = WORKLOADS[name]
        default_B = wl.batches[-1 if name == "c5" else 0]
        o = bench_layer(args, wl, wl.shape, B, default_B, WORKLOAD_ID[name], stream_ref=False,
                        cpu_baseline=False)
        r = o["roofline"]
        res[f"{name}_b{B}"] = {
            "workload": o["config"]["workload"], "draft_tokens": B, "n_uniq": o["n_uniq"],
            "dtype": o["dtype"], "ms_per_step": o["ms_per_step"],
            "draft_tokens_per_s": o["value"], "ffn_avg_launch_us": r["avg_launch_us"],
            "achieved_gbs": r["achieved"], "frac": r["frac"], "traffic": r["traffic"],
            "bytes_per_launch": r["bytes_per_launch"], "ffn_timing": o["ffn_timing"]}
        _log(f"[bench] extra {name} B={B}: {r['achieved']:.0f} GB/s ({r['frac']:.3f} of peak)")
        gc.collect()
        torch.cuda.empty_cache()
    return res


def bench_layer(args, wl, shape, B: int, default_B: int, wid: int, stream_ref: bool = True,
                cpu_baseline: bool = True) -> dict:
    """One verify-MoE layer (layer 0 of the workload) at B draft tokens: whole
    steps timed on the host, the expert-FFN calls timed with HIP events, the
    read-stream reference and the oracle on the host cores."""
    import torch

    import paper_2608_15018_amd as s2
    from synth import gen

    t0 = time.time()
    router = gen.make_router(shape, args.seed, 0, wid, wl.router_std)
    x, conf_w, _ = gen.make_batch(shape, B, args.seed, 0, wid, wl.rho)
    experts = gen.make_experts(shape, args.seed, 0, wid, wl.w_std)
    shared = gen.make_shared_experts(shape, args.seed, 0, wid, wl.w_std)
    _log(f"[bench] inputs generated in {time.time() - t0:.1f}s")

    # Weights are packed once, as at model load (s2moe_pack_weights); the
    # verify step then streams each activated expert's tiles contiguously.
    packed = shape.wdt != "f32" and not args.plain_weights
    layer = s2.make_layer(shape, flags=shape.flags | (s2.PACKED_WEIGHTS if packed else 0))
    p = s2.VerifyPass(layer, B, fused=True)
    p4 = s2.VerifyPass(layer, B, fused=False)
    xd, rd, cd = s2.to_device(x), s2.to_device(router), s2.to_device(conf_w)
    dev_w, wstruct = s2.weights_to_device(experts, shared)
    if packed:
        dev_w, wstruct = s2.pack_expert_weights(dev_w, shape.wdt)
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    # warm-up (also fixes the routing, which is deterministic)
    warmup_run = warm(lambda: p(xd, rd, cd, wstruct), args.warmup)
    n_uniq = int(p.rt.n_uniq.item())
    unique_bytes = n_uniq * expert_bytes(shape, shape.ffn) + \
        shape.n_shared * expert_bytes(shape, shape.ffn_shared)

    # Timed region 1: K whole steps back to back (no host sync, no events),
    # each one s2moe_moe_layer call.  The same steps as the four calls are
    # timed in blocks of K alternating with blocks of one-call steps, so
    # that the two compare under the same conditions.
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        p(xd, rd, cd, wstruct)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed / args.steps * 1e3
    p4(xd, rd, cd, wstruct)
    torch.cuda.synchronize()
    cmp = {p: 0.0, p4: 0.0}
    for _ in range(2):
        for q in (p4, p):
            tq = time.perf_counter()
            for _ in range(args.steps):
                q(xd, rd, cd, wstruct)
            torch.cuda.synchronize()
            cmp[q] += time.perf_counter() - tq
    four_call_ms = cmp[p4] / (2 * args.steps) * 1e3
    one_call_cmp_ms = cmp[p] / (2 * args.steps) * 1e3

    # Timed region 2: K back-to-back s2moe_verify_moe calls between one pair
    # of HIP events on the launch stream (an event pair costs a few
    # microseconds, paid once here).  The calls cycle through enough copies
    # of the expert weights that each cycle streams > 600 MB, more than the
    # 256 MB Infinity Cache holds, so every call reads its weights from HBM.
    copies = 1 if args.no_scrub else max(1, min(16, -(-ROTATE_BYTES // max(1, unique_bytes))))
    wlist = [wstruct]
    for _ in range(copies - 1):
        ce = {n: t.clone() for n, t in dev_w[0].items()}
        cs = {n: t.clone() for n, t in dev_w[1].items()}
        wlist.append((s2.make_weights(ce, cs), ce, cs))
    wstructs = [wlist[0]] + [w[0] for w in wlist[1:]]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for w in wstructs:
        p.verify_moe(xd, w)
    torch.cuda.synchronize()
    _head_start()
    e0.record(stream)
    for i in range(args.steps):
        p.verify_moe(xd, wstructs[i % copies])
    e1.record(stream)
    torch.cuda.synchronize()
    ffn_avg_s = e0.elapsed_time(e1) / 1e3 / args.steps
    achieved = unique_bytes / ffn_avg_s / 1e9
    del wlist, wstructs

    # Reference: a plain sequential read of 2 GiB with the FFN's load type
    # (s2moe_stream_read, a diagnostic of the library).
    stream_gbs = None
    if stream_ref:
        stream_gbs = stream_read_gbs()
    ffn_note = (f"one event pair around {args.steps} back-to-back calls over {copies} "
                f"weight cop{'y' if copies == 1 else 'ies'}")
    cpu = None
    if cpu_baseline and not args.no_cpu_baseline:
        import oracle
        try:
            from threadpoolctl import threadpool_info
            cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        except Exception:  # pragma: no cover
            cores = os.cpu_count()
        reps, dt = time_oracle(lambda: oracle.forward(x, router, conf_w, experts, shared, shape))
        cpu = {"value": reps * B / dt, "unit": "draft tokens/s", "cores": cores, "kind": "oracle",
               "sample": f"full verify steps of {wl.name} (B={B}, {n_uniq} activated experts"
                         f"{', %d shared' % shape.n_shared if shape.n_shared else ''}), fp64 "
                         f"numpy, {reps} steps in {dt:.1f}s"}

    out = {
        "metric": "verify-MoE layer: draft tokens/s and achieved HBM GB/s (% of peak) on "
                  "unique experts",
        "value": B * args.steps / elapsed,
        "unit": "draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "f32": "f32", "q4g32": "int4-g32/bf16"}[shape.wdt],
        "data": "synthetic",
        "config": {"workload": wl.description + (" (one layer: layer 0)" if wl.n_layers > 1 else ""),
                   "name": wl.name, "draft_tokens": B, "layers": 1,
                   "hidden": shape.hidden, "ffn": shape.ffn, "experts": shape.n_experts,
                   "top_k": shape.top_k, "shared": shape.n_shared, "cap": shape.cap,
                   "alpha": shape.alpha, "weights": "packed" if packed else "row-major"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": recorded_traffic(wl.name, shape.wdt, B, default_B),
                     "kernel": "s2moe_verify_moe (expert gate-up + down launches)",
                     "bytes_per_launch": unique_bytes, "avg_launch_us": ffn_avg_s * 1e6},
        "cpu_baseline": cpu,
        "n_uniq": n_uniq,
        "reuse_ratio": n_uniq / (B * shape.top_k),
        "ffn_timing": ffn_note,
        "step": "one s2moe_moe_layer call (route, gate, experts, combine)",
        "warmup_steps_run": warmup_run,
        "four_call_ms_per_step": four_call_ms,
        "one_call_ms_per_step_alternating": one_call_cmp_ms,
    }
    if stream_gbs is not None:
        out["stream_read"] = {"value": stream_gbs, "unit": "GB/s",
                              "kind": "s2moe_stream_read: one sequential pass over 2 GiB, "
                                      "16-byte nontemporal loads",
                              "ffn_frac_of_stream": achieved / stream_gbs}
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c2",
                    choices=["c1", "c2", "c3", "c4", "c5", "t_qwen3", "t_deepseek", "t_olmoe",
                             "t_gptoss", "d_olmoe", "d_deepseek", "d_qwen3", "d_gptoss"],
                    help="c*: verify-MoE layer; t_*: draft-tree expansion (s2moe_expand); "
                         "d_*: expert-sparse draft step over a model's MoE layers")
    ap.add_argument("--wdt", default="bf16", choices=["bf16", "q4g32"],
                    help="d_* workloads: expert weight format")
    ap.add_argument("--trees", type=int, default=256,
                    help="t_* workloads: draft trees per s2moe_expand launch")
    ap.add_argument("--batch", type=int, default=None, help="draft tokens (default: workload's)")
    ap.add_argument("--alpha", type=float, default=None)
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--layers", type=int, default=1,
                    help="c*: verify this many layers of the workload back to back, each with its "
                         "own router, hidden states, confidences and expert weights (c5: up to 24)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="default run: skip the extra int4 configurations (c5 at B=16 and 64)")
    ap.add_argument("--plain-weights", action="store_true",
                    help="stream the row-major weights instead of the packed tile order")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain device copy of 1 GiB (calibrates HBM byte counters)")
    ap.add_argument("--no-scrub", action="store_true",
                    help="time repeated launches on one copy of the inputs (cache-resident "
                         "when small) instead of cycling through copies larger than the caches")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the verify-MoE path here runs on a single "
              "MI355X (no multi-GPU path is built); run it with --gpus 1.", file=sys.stderr)
        return 2

    import torch

    import paper_2608_15018_amd as s2
    from synth import gen
    from synth.configs import WORKLOAD_ID, WORKLOADS

    torch.cuda.set_device(0)
    if args.copy_probe:
        # A plain copy of known size: each launch reads and writes 1 GiB.
        n = 1 << 30
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n,
                          "launches": 5}))
        return 0
    s2.load()
    if args.workload.startswith("t_"):
        return bench_expand(args)
    if args.workload.startswith("d_"):
        return bench_draft(args)
    wl = WORKLOADS[args.workload]
    shape = wl.shape if args.alpha is None else wl.shape.with_(alpha=args.alpha)
    default_B = wl.batches[-1 if args.workload == "c5" else 0]
    B = args.batch or default_B
    wid = WORKLOAD_ID[wl.name]
    if args.layers > 1:
        return bench_stack(args, wl, shape, B, wid)

    out = bench_layer(args, wl, shape, B, default_B, wid)
    if not args.no_extra and args.workload == "c2" and args.batch is None and args.alpha is None:
        out["extra_configs"] = extra_configs(args)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
