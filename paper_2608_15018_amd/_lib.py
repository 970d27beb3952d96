"""ctypes binding of libs2moe.so: torch tensors in, raw device pointers out.

Every step of the verify-MoE pass runs in the library's HIP kernels; this
module only checks shapes and dtypes, builds the C structs and passes
pointers plus the current HIP stream.  If the library is not built, loading
fails loudly (there is no fallback).
"""

from __future__ import annotations

import ctypes
import os
import re

import torch

# S2MOE_LIBRARY may name another build of the same library (e.g. one built
# with different tuning constants).
LIB_PATH = os.environ.get("S2MOE_LIBRARY") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libs2moe.so")
HEADER_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                           "include", "s2moe.h")

F32, BF16, Q4G32 = 0, 1, 2
DTYPE_CODES = {"f32": F32, "bf16": BF16, "q4g32": Q4G32}
PREF_ACTIVATED_ONLY, BIAS_ABSOLUTE, GATE_FROM_BIASED, PACKED_WEIGHTS = 1, 2, 4, 8
OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP = 0, 1, 2, 3, 4


class S2moeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


class Layer(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("n_shared", ctypes.c_int32), ("ffn_shared", ctypes.c_int32),
                ("cap", ctypes.c_int32), ("alpha", ctypes.c_float),
                ("flags", ctypes.c_uint32), ("act_dtype", ctypes.c_int32),
                ("w_dtype", ctypes.c_int32)]


_WEIGHT_FIELDS = ("gate", "up", "down", "gate_s", "up_s", "down_s",
                  "sh_gate", "sh_up", "sh_down", "sh_gate_s", "sh_up_s", "sh_down_s")


class Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in _WEIGHT_FIELDS]


_ROUTING_FIELDS = ("logits", "gap", "plain_idx", "g", "pref", "idx", "gate_w", "count",
                   "offset", "slot", "uniq", "n_uniq")


class RoutingStruct(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in _ROUTING_FIELDS]


class ExpandShape(ctypes.Structure):
    _fields_ = [("n_trees", ctypes.c_int32), ("max_nodes", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32),
                ("k", ctypes.c_int32), ("max_admit", ctypes.c_int32),
                ("t_ar", ctypes.c_double), ("t_exp", ctypes.c_double)]


_lib = None


def load():
    """Load libs2moe.so (raises ImportError if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing; build it with "
                          "`python -m paper_2608_15018_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    Lp = ctypes.POINTER(Layer)
    lib.s2moe_route.argtypes = [Lp, ctypes.c_int32, P, P, ctypes.POINTER(RoutingStruct), P]
    lib.s2moe_reuse_gate.argtypes = [Lp, ctypes.c_int32, P, ctypes.POINTER(RoutingStruct), P]
    lib.s2moe_workspace_bytes.argtypes = [Lp, ctypes.c_int32]
    lib.s2moe_workspace_bytes.restype = ctypes.c_size_t
    lib.s2moe_verify_moe.argtypes = [Lp, ctypes.c_int32, P, ctypes.POINTER(Weights),
                                     ctypes.POINTER(RoutingStruct), P, ctypes.c_size_t, P, P]
    lib.s2moe_verify_moe_noalloc.argtypes = [Lp, ctypes.c_int32, P, ctypes.POINTER(Weights),
                                             ctypes.POINTER(RoutingStruct), P, P]
    lib.s2moe_combine.argtypes = [Lp, ctypes.c_int32, ctypes.POINTER(RoutingStruct), P, P, P]
    lib.s2moe_moe_layer.argtypes = [Lp, ctypes.c_int32, P, P, P, ctypes.POINTER(Weights),
                                    ctypes.POINTER(RoutingStruct), P, ctypes.c_size_t, P, P, P]
    lib.s2moe_pack_weights.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_int32, P, P, P, P, P]
    lib.s2moe_pack_weights.restype = ctypes.c_int
    lib.s2moe_expand.argtypes = [ctypes.POINTER(ExpandShape)] + [P] * 13
    lib.s2moe_expand.restype = ctypes.c_int
    lib.s2moe_expand_max_nodes.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.POINTER(ctypes.c_int32)]
    lib.s2moe_expand_max_nodes.restype = ctypes.c_int
    lib.s2moe_stream_read.argtypes = [P, ctypes.c_size_t, P, P]
    lib.s2moe_stream_read.restype = ctypes.c_int
    for f in ("s2moe_route", "s2moe_reuse_gate", "s2moe_verify_moe", "s2moe_verify_moe_noalloc",
              "s2moe_combine", "s2moe_moe_layer"):
        getattr(lib, f).restype = ctypes.c_int
    lib.s2moe_last_error.restype = ctypes.c_char_p
    lib.s2moe_last_error.argtypes = []
    lib.s2moe_status_string.restype = ctypes.c_char_p
    lib.s2moe_status_string.argtypes = [ctypes.c_int]
    lib.s2moe_abi_version.restype = ctypes.c_int32
    lib.s2moe_abi_version.argtypes = []
    _lib = lib
    return lib


def header_functions() -> list:
    """Names of the functions include/s2moe.h declares."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(s2moe_[a-z_]+)\s*\(", text)))


def last_error() -> str:
    return load().s2moe_last_error().decode()


def _check(status: int):
    if status != OK:
        raise S2moeError(status, last_error())


def make_layer(shape=None, **kw) -> Layer:
    """A Layer struct from an object with the layer attributes (hidden, ffn,
    n_experts, top_k, n_shared, ffn_shared, cap, alpha, flags, act, wdt)
    and/or keyword overrides."""
    d = {}
    if shape is not None:
        for n in ("hidden", "ffn", "n_experts", "top_k", "n_shared", "ffn_shared", "cap",
                  "alpha", "flags", "act", "wdt"):
            if hasattr(shape, n):
                d[n] = getattr(shape, n)
    d.update(kw)
    act = d.pop("act", "bf16")
    wdt = d.pop("wdt", "bf16")
    L = Layer()
    L.hidden = d["hidden"]
    L.ffn = d["ffn"]
    L.n_experts = d["n_experts"]
    L.top_k = d["top_k"]
    L.n_shared = d.get("n_shared", 0)
    L.ffn_shared = d.get("ffn_shared", 0)
    L.cap = d["cap"]
    L.alpha = d.get("alpha", 0.5)
    L.flags = d.get("flags", 0)
    L.act_dtype = DTYPE_CODES[act] if isinstance(act, str) else act
    L.w_dtype = DTYPE_CODES[wdt] if isinstance(wdt, str) else wdt
    return L


def _ptr(t) -> int | None:
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor")
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


class Routing:
    """Device buffers of the routing state of one verify batch."""

    def __init__(self, layer: Layer, B: int, device="cuda"):
        E, k = layer.n_experts, layer.top_k
        f32, i32 = torch.float32, torch.int32
        mk = lambda shape, dt: torch.empty(shape, dtype=dt, device=device)  # noqa: E731
        self.B = B
        self.logits = mk((B, E), f32)
        self.gap = mk((B,), f32)
        self.plain_idx = mk((B, k), i32)
        self.g = mk((E,), f32)
        self.pref = mk((E,), i32)
        self.idx = mk((B, k), i32)
        self.gate_w = mk((B, k), f32)
        self.count = mk((E,), i32)
        self.offset = mk((E + 1,), i32)
        self.slot = mk((B * k,), i32)
        self.uniq = mk((E,), i32)
        self.n_uniq = mk((1,), i32)
        self.struct = RoutingStruct(*[getattr(self, n).data_ptr() for n in _ROUTING_FIELDS])

    def host(self) -> dict:
        return {n: getattr(self, n).cpu().numpy() for n in _ROUTING_FIELDS}


def route(layer: Layer, x: torch.Tensor, router: torch.Tensor, rt: Routing, stream=None):
    B = x.shape[0]
    _check(load().s2moe_route(ctypes.byref(layer), B, _ptr(x), _ptr(router),
                              ctypes.byref(rt.struct), _stream(stream)))


def reuse_gate(layer: Layer, conf_w: torch.Tensor, rt: Routing, stream=None):
    if conf_w.dtype != torch.float32:
        raise TypeError("conf_w must be float32")
    _check(load().s2moe_reuse_gate(ctypes.byref(layer), rt.B, _ptr(conf_w),
                                   ctypes.byref(rt.struct), _stream(stream)))


def workspace_bytes(layer: Layer, B: int) -> int:
    n = load().s2moe_workspace_bytes(ctypes.byref(layer), B)
    if n == 0:
        raise S2moeError(EINVAL, last_error())
    return int(n)


def make_weights(experts: dict, shared: dict | None = None) -> Weights:
    """Weights struct from dicts of device tensors named like the C fields
    (gate, up, down, gate_s, ...; shared dict keys without the sh_ prefix)."""
    w = Weights()
    for n in ("gate", "up", "down", "gate_s", "up_s", "down_s"):
        t = experts.get(n)
        setattr(w, n, _ptr(t) if t is not None else None)
    for n in ("gate", "up", "down", "gate_s", "up_s", "down_s"):
        t = (shared or {}).get(n)
        setattr(w, "sh_" + n, _ptr(t) if t is not None else None)
    return w


def verify_moe(layer: Layer, x: torch.Tensor, weights: Weights, rt: Routing,
               workspace: torch.Tensor, expert_out: torch.Tensor, stream=None):
    _check(load().s2moe_verify_moe(ctypes.byref(layer), rt.B, _ptr(x), ctypes.byref(weights),
                                   ctypes.byref(rt.struct), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(),
                                   _ptr(expert_out), _stream(stream)))


def verify_moe_noalloc(layer: Layer, x: torch.Tensor, weights: Weights, rt: Routing,
                       expert_out: torch.Tensor, stream=None):
    """s2moe_verify_moe_noalloc: verify_moe on the library's own scratch array."""
    _check(load().s2moe_verify_moe_noalloc(ctypes.byref(layer), rt.B, _ptr(x),
                                           ctypes.byref(weights), ctypes.byref(rt.struct),
                                           _ptr(expert_out), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 16 << 20


def combine(layer: Layer, rt: Routing, expert_out: torch.Tensor, y: torch.Tensor, stream=None):
    _check(load().s2moe_combine(ctypes.byref(layer), rt.B, ctypes.byref(rt.struct),
                                _ptr(expert_out), _ptr(y), _stream(stream)))


def moe_layer(layer: Layer, x: torch.Tensor, router: torch.Tensor, conf_w: torch.Tensor,
              weights: Weights, rt: Routing, workspace: torch.Tensor, expert_out: torch.Tensor,
              y: torch.Tensor, stream=None):
    """s2moe_moe_layer: route, reuse_gate, verify_moe and combine in one call."""
    _check(load().s2moe_moe_layer(ctypes.byref(layer), rt.B, _ptr(x), _ptr(router), _ptr(conf_w),
                                  ctypes.byref(weights), ctypes.byref(rt.struct), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _ptr(expert_out),
                                  _ptr(y), _stream(stream)))


def pack_weights(wdt: str, mats: torch.Tensor, scales: torch.Tensor | None = None,
                 stream=None):
    """Packed copies (s2moe_pack_weights) of matrices [n, rows, cols] (bf16) or
    of int4 codes [n, rows, cols/2] with their scales [n, rows, cols/32]."""
    code = DTYPE_CODES[wdt]
    n, rows = mats.shape[0], mats.shape[1]
    cols = mats.shape[2] * (2 if code == Q4G32 else 1)
    dst = torch.empty_like(mats)
    dst_s = torch.empty_like(scales) if scales is not None else None
    _check(load().s2moe_pack_weights(code, n, rows, cols, _ptr(mats), _ptr(scales), _ptr(dst),
                                     _ptr(dst_s), _stream(stream)))
    return dst, dst_s


class ExpandOut:
    """Device outputs of s2moe_expand for T trees of N nodes."""

    def __init__(self, T: int, N: int, device="cuda"):
        i32 = dict(dtype=torch.int32, device=device)
        self.order = torch.empty((T, N), **i32)
        self.util = torch.empty((T, N), dtype=torch.float64, device=device)
        self.n_new = torch.empty((T, N), **i32)
        self.n_admit = torch.empty(T, **i32)
        self.n_pairs = torch.empty(T, **i32)
        self.status = torch.empty(T, **i32)

    def host(self) -> dict:
        return {k: getattr(self, k).cpu().numpy()
                for k in ("order", "util", "n_new", "n_admit", "n_pairs", "status")}


def _expect(t, name, dtype, shape):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected {dtype} {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")


def expand(parent, q, eid, c_draft, n_nodes, out: ExpandOut, n_experts: int, t_ar: float,
           t_exp: float, root_eid=None, max_admit: int = 0, stream=None):
    """s2moe_expand on device tensors: parent [T, N] int32, q [T, N] f32,
    eid [T, N, L, k] int32, c_draft [T, N] f32, n_nodes [T] int32,
    root_eid [T, L, k] int32 or None; results land in `out`."""
    T, N, L, k = eid.shape
    _expect(parent, "parent", torch.int32, (T, N))
    _expect(q, "q", torch.float32, (T, N))
    _expect(c_draft, "c_draft", torch.float32, (T, N))
    _expect(n_nodes, "n_nodes", torch.int32, (T,))
    _expect(eid, "eid", torch.int32, (T, N, L, k))
    if root_eid is not None:
        _expect(root_eid, "root_eid", torch.int32, (T, L, k))
    for name in ("order", "n_new"):
        _expect(getattr(out, name), name, torch.int32, (T, N))
    _expect(out.util, "util", torch.float64, (T, N))
    for name in ("n_admit", "n_pairs", "status"):
        _expect(getattr(out, name), name, torch.int32, (T,))
    sh = ExpandShape(T, N, L, n_experts, k, max_admit, t_ar, t_exp)
    _check(load().s2moe_expand(ctypes.byref(sh), _ptr(parent), _ptr(q), _ptr(eid), _ptr(c_draft),
                               _ptr(root_eid), _ptr(n_nodes), _ptr(out.order), _ptr(out.util),
                               _ptr(out.n_new), _ptr(out.n_admit), _ptr(out.n_pairs),
                               _ptr(out.status), _stream(stream)))


def expand_max_nodes(n_layers: int, n_experts: int, k: int) -> int:
    v = ctypes.c_int32(0)
    _check(load().s2moe_expand_max_nodes(n_layers, n_experts, k, ctypes.byref(v)))
    return int(v.value)


STREAM_SINK_WORDS = 2048


def stream_read(buf: torch.Tensor, sink: torch.Tensor, stream=None):
    """Diagnostic s2moe_stream_read: one sequential read of buf's bytes; sink
    is a device tensor of at least STREAM_SINK_WORDS int32."""
    _check(load().s2moe_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                                    _stream(stream)))


def abi_version() -> int:
    return int(load().s2moe_abi_version())
