"""C-ABI checks that need no GPU: the library loads, exports every function
the header declares, and rejects malformed arguments on the host before
anything is enqueued (no kernel is launched by these tests)."""

import ctypes
import subprocess

import pytest

import paper_2608_15018_amd as s2
from paper_2608_15018_amd import _lib


@pytest.fixture(scope="module")
def lib():
    return s2.load()


def test_exports_every_declared_function(lib):
    declared = _lib.header_functions()
    assert {"s2moe_route", "s2moe_reuse_gate", "s2moe_verify_moe", "s2moe_combine",
            "s2moe_workspace_bytes", "s2moe_last_error"} <= set(declared)
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in declared:
        assert name in exported, name
        assert hasattr(lib, name)


def test_version_and_status_strings(lib):
    assert s2.abi_version() == 1
    assert lib.s2moe_status_string(0) == b"S2MOE_OK"
    assert lib.s2moe_status_string(3) == b"S2MOE_EWORKSPACE"


def _layer(**kw):
    base = dict(hidden=256, ffn=512, n_experts=8, top_k=2, cap=4, alpha=0.5, act="bf16",
                wdt="bf16")
    base.update(kw)
    return s2.make_layer(**base)


def _route_status(lib, layer, B=4, ptrs=True):
    # Aligned fake addresses; every case below fails validation before use.
    fake = ctypes.c_void_p(0x100000) if ptrs else None
    rt = _lib.RoutingStruct(*([0x200000] * 12))
    st = lib.s2moe_route(ctypes.byref(layer) if layer is not None else None, B, fake, fake,
                         ctypes.byref(rt), None)
    return st, _lib.last_error()


@pytest.mark.parametrize("kw,B,status,needle", [
    ({}, 0, _lib.EINVAL, "n_tokens"),
    ({}, 257, _lib.EUNSUPPORTED, "n_tokens"),
    ({"hidden": 100}, 4, _lib.EINVAL, "hidden"),
    ({"ffn": 96}, 4, _lib.EINVAL, "ffn"),
    ({"n_experts": 300, "cap": 4}, 4, _lib.EUNSUPPORTED, "n_experts"),
    ({"top_k": 8}, 4, _lib.EINVAL, "top_k"),
    ({"n_experts": 64, "top_k": 17, "cap": 20}, 4, _lib.EUNSUPPORTED, "top_k"),
    ({"cap": 1}, 4, _lib.EINVAL, "cap"),
    ({"cap": 9}, 4, _lib.EINVAL, "cap"),
    ({"alpha": -1.0}, 4, _lib.EINVAL, "alpha"),
    ({"alpha": float("inf")}, 4, _lib.EINVAL, "alpha"),
    ({"flags": 16}, 4, _lib.EINVAL, "flags"),
    ({"n_shared": 2, "ffn_shared": 0}, 4, _lib.EINVAL, "ffn_shared"),
    ({"n_shared": 9, "ffn_shared": 64}, 4, _lib.EUNSUPPORTED, "n_shared"),
    ({"act": "f32", "wdt": "bf16"}, 4, _lib.EUNSUPPORTED, "supported"),
    ({"act": "q4g32"}, 4, _lib.EINVAL, "act_dtype"),
    ({"wdt": "q4g32", "ffn": 320}, 4, _lib.EUNSUPPORTED, "Q4G32"),
    ({"hidden": 16384 + 64}, 4, _lib.EINVAL, "hidden"),
    ({"ffn": 262144 + 64}, 4, _lib.EINVAL, "ffn"),
])
def test_invalid_layers_rejected_on_host(lib, kw, B, status, needle):
    st, msg = _route_status(lib, _layer(**kw), B)
    assert st == status, msg
    assert needle in msg


def test_null_and_misaligned_pointers(lib):
    L = _layer()
    st, msg = _route_status(lib, None)
    assert st == _lib.EINVAL and "layer" in msg
    st, msg = _route_status(lib, L, ptrs=False)
    assert st == _lib.EINVAL and "NULL" in msg
    rt = _lib.RoutingStruct(*([0x200000] * 12))
    st = lib.s2moe_route(ctypes.byref(L), 4, ctypes.c_void_p(0x100004), ctypes.c_void_p(0x100000),
                         ctypes.byref(rt), None)
    assert st == _lib.EINVAL and "aligned" in _lib.last_error()
    st = lib.s2moe_reuse_gate(ctypes.byref(L), 4, ctypes.c_void_p(0x100000), None, None)
    assert st == _lib.EINVAL and "routing" in _lib.last_error()


def test_workspace_size_and_errors(lib):
    L = _layer(n_shared=1, ffn_shared=1024)
    B = 8
    need = s2.workspace_bytes(L, B)
    rows = B * 2 + 1 * B
    assert need >= rows * 1024 * 2 and need % 256 == 0
    assert s2.workspace_bytes(_layer(act="f32", wdt="f32"), 8) >= 16 * 512 * 4
    w = _lib.Weights(*([0x300000] * 12))
    rt = _lib.RoutingStruct(*([0x200000] * 12))
    fake = ctypes.c_void_p(0x100000)
    st = lib.s2moe_verify_moe(ctypes.byref(L), B, fake, ctypes.byref(w), ctypes.byref(rt),
                              None, need, fake, None)
    assert st == _lib.EWORKSPACE and "workspace" in _lib.last_error()
    st = lib.s2moe_verify_moe(ctypes.byref(L), B, fake, ctypes.byref(w), ctypes.byref(rt),
                              ctypes.c_void_p(0x400000), need - 1, fake, None)
    assert st == _lib.EWORKSPACE and str(need) in _lib.last_error()
    w.sh_down = None
    st = lib.s2moe_verify_moe(ctypes.byref(L), B, fake, ctypes.byref(w), ctypes.byref(rt),
                              ctypes.c_void_p(0x400000), need, fake, None)
    assert st == _lib.EINVAL and "sh_down" in _lib.last_error()
    Lq = _layer(wdt="q4g32")
    w = _lib.Weights(*([0x300000] * 3 + [None] * 9))
    st = lib.s2moe_verify_moe(ctypes.byref(Lq), B, fake, ctypes.byref(w), ctypes.byref(rt),
                              ctypes.c_void_p(0x400000), 1 << 30, fake, None)
    assert st == _lib.EINVAL and "gate_s" in _lib.last_error()
    assert lib.s2moe_workspace_bytes(ctypes.byref(_layer(cap=0)), 4) == 0


def test_int4_workspace_holds_the_down_k_parts(lib):
    """With int4 weights the workspace holds Hh, the fp16 copy of x and the
    fp32 partial sums of the down projection's K parts 1 .. Q-1.  At the
    Mixtral shape the part rule (at least 1024 down items of 128 rows, at
    most 8 parts, the partial sums within 2 % of the down weights' bytes, one
    part at up to 8 tokens) gives Q = 1, 1, 4, 4 and 3 at 1, 4, 16, 32 and 64
    tokens."""
    H, F, E, k = 4096, 14336, 8, 2
    L = _layer(hidden=H, ffn=F, n_experts=E, top_k=k, cap=4, wdt="q4g32")
    r256 = lambda n: (n + 255) // 256 * 256  # noqa: E731
    down_bytes = E * F * H * (0.5 + 2 / 32)
    for B, Q in ((1, 1), (4, 1), (16, 4), (32, 4), (64, 3)):
        rows = B * k
        part = (Q - 1) * rows * H * 4
        assert part <= 0.02 * down_bytes
        assert s2.workspace_bytes(L, B) == r256(rows * F * 2) + r256(B * H * 2) + r256(part), B


def test_binding_raises_with_message():
    with pytest.raises(s2.S2moeError) as ei:
        s2.workspace_bytes(_layer(top_k=0), 4)
    assert ei.value.status == _lib.EINVAL


@pytest.mark.parametrize("args,status,needle", [
    ((0, 1, 16, 32), _lib.EUNSUPPORTED, "w_dtype"),
    ((5, 1, 16, 32), _lib.EINVAL, "w_dtype"),
    ((1, 0, 16, 32), _lib.EINVAL, "n_mats"),
    ((1, 1, 24, 32), _lib.EINVAL, "rows"),
    ((1, 1, 16, 48), _lib.EINVAL, "cols"),
    ((2, 1, 16, 64), _lib.EINVAL, "cols"),
])
def test_pack_weights_rejects_bad_shapes(lib, args, status, needle):
    fake, other = ctypes.c_void_p(0x100000), ctypes.c_void_p(0x9000000)
    st = lib.s2moe_pack_weights(*args, fake, fake, other, other, None)
    assert st == status
    assert needle in _lib.last_error()


def test_pack_weights_rejects_overlap_and_missing_scales(lib):
    a, b = ctypes.c_void_p(0x100000), ctypes.c_void_p(0x100400)
    assert lib.s2moe_pack_weights(1, 1, 16, 64, a, None, b, None, None) == _lib.EINVAL
    assert "overlap" in _lib.last_error()
    far = ctypes.c_void_p(0x9000000)
    assert lib.s2moe_pack_weights(2, 1, 16, 128, a, None, far, None, None) == _lib.EINVAL
    assert "src_scales" in _lib.last_error()


def test_packed_flag_needs_16bit_or_int4_weights(lib):
    st, msg = _route_status(lib, _layer(act="f32", wdt="f32", flags=8))
    assert st == _lib.EUNSUPPORTED and "PACKED" in msg


def test_stream_read_validation(lib):
    a = ctypes.c_void_p(0x100000)
    assert lib.s2moe_stream_read(a, 0, a, None) == _lib.EINVAL
    assert "multiple of 16" in _lib.last_error()
    assert lib.s2moe_stream_read(a, 24, a, None) == _lib.EINVAL
    assert lib.s2moe_stream_read(ctypes.c_void_p(0x100004), 64, a, None) == _lib.EINVAL
    assert "aligned" in _lib.last_error()
    assert lib.s2moe_stream_read(None, 64, a, None) == _lib.EINVAL


def _expand_call(lib, sh, ptr=0x100000, misalign=None):
    args = [ctypes.c_void_p(ptr)] * 13
    if misalign is not None:
        args[misalign] = ctypes.c_void_p(ptr + 4)
    return lib.s2moe_expand(ctypes.byref(sh) if sh is not None else None, *args)


@pytest.mark.parametrize("field,value,needle", [
    ("max_nodes", 0, "max_nodes"), ("max_nodes", 1025, "max_nodes"),
    ("n_layers", 0, "n_layers"), ("n_layers", 129, "n_layers"),
    ("n_experts", 0, "n_experts"), ("n_experts", 1025, "n_experts"),
    ("k", 0, "k ="), ("k", 33, "k ="), ("n_trees", -1, "n_trees"),
    ("t_ar", -1.0, "t_ar"), ("t_exp", float("nan"), "t_exp"), ("t_ar", float("inf"), "t_ar"),
])
def test_expand_rejects_bad_shapes_on_host(lib, field, value, needle):
    sh = _lib.ExpandShape(4, 116, 48, 128, 8, 0, 512.0, 1.0)
    setattr(sh, field, value)
    assert _expand_call(lib, sh) == _lib.EINVAL
    assert needle in _lib.last_error()


def test_expand_null_misaligned_and_empty(lib):
    assert _expand_call(lib, None) == _lib.EINVAL
    sh = _lib.ExpandShape(0, 116, 48, 128, 8, 0, 512.0, 1.0)
    assert _expand_call(lib, sh, ptr=0) == _lib.OK  # T = 0: no-op, pointers unused
    sh.n_trees = 2
    assert _expand_call(lib, sh, ptr=0) == _lib.EINVAL
    assert "NULL" in _lib.last_error()
    assert _expand_call(lib, sh, misalign=7) == _lib.EINVAL  # util must be 8-byte aligned
    assert "util" in _lib.last_error() and "aligned" in _lib.last_error()
    assert _expand_call(lib, sh, misalign=2) == _lib.EINVAL  # eid must be 16-byte aligned
    assert "eid" in _lib.last_error()
    assert lib.s2moe_expand_max_nodes(48, 128, 8, None) == _lib.EINVAL
    v = ctypes.c_int32(7)
    assert lib.s2moe_expand_max_nodes(0, 128, 8, ctypes.byref(v)) == _lib.EINVAL and v.value == 0


def test_expand_row_index_shortcut_exhaustive():
    """The kernel maps a flat id index f < N*L*k <= 2^22 to its (node, layer)
    row with (f * ceil(2^42 / k)) >> 42; exact for every k <= 32 and f."""
    import numpy as np
    f = np.arange(1 << 22, dtype=np.uint64)
    for k in range(1, 33):
        magic = np.uint64(((1 << 42) + k - 1) // k)
        assert ((f * magic) >> np.uint64(42) == f // np.uint64(k)).all(), k
        assert int(magic) * ((1 << 22) - 1) < 2 ** 64


def test_combine_rejects_overlapping_output(lib):
    L = _layer(n_shared=1, ffn_shared=512)
    B, H = 4, 256
    rt = _lib.RoutingStruct(*([0x200000] * 12))
    eo = 0x1000000
    eo_bytes = (B * 2 + B) * H * 4
    for y in (eo, eo + eo_bytes - 16, eo - B * H * 4 + 16):
        st = lib.s2moe_combine(ctypes.byref(L), B, ctypes.byref(rt), ctypes.c_void_p(eo),
                               ctypes.c_void_p(y), None)
        assert st == _lib.EINVAL and "overlaps" in _lib.last_error()


def test_noalloc_verify_rejects_oversized_scratch_on_host(lib):
    """A layer whose workspace exceeds the library's scratch array is
    rejected before anything touches the device (no GPU needed)."""
    L = _layer(hidden=4096, ffn=32768, n_experts=8, top_k=2, cap=4)
    w = _lib.Weights(*([0x300000] * 12))
    rt = _lib.RoutingStruct(*([0x200000] * 12))
    fake = ctypes.c_void_p(0x100000)
    B = 256
    assert s2.workspace_bytes(L, B) > s2.NOALLOC_SCRATCH_BYTES
    st = lib.s2moe_verify_moe_noalloc(ctypes.byref(L), B, fake, ctypes.byref(w),
                                      ctypes.byref(rt), fake, None)
    assert st == _lib.EUNSUPPORTED and "scratch" in _lib.last_error()
    st = lib.s2moe_verify_moe_noalloc(ctypes.byref(L), 4, fake, ctypes.byref(w),
                                      ctypes.byref(rt), None, None)
    assert st == _lib.EINVAL and "expert_out" in _lib.last_error()


def test_noalloc_scratch_size_matches_header():
    import re
    text = open(_lib.HEADER_PATH).read()
    m = re.search(r"#define S2MOE_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == s2.NOALLOC_SCRATCH_BYTES


def test_moe_layer_validates_like_the_four_calls(lib):
    """s2moe_moe_layer runs the checks of route, reuse_gate, verify_moe (with
    its workspace) and combine before anything is enqueued."""
    L = _layer(n_shared=1, ffn_shared=512)
    B, H = 4, 256
    w = _lib.Weights(*([0x300000] * 12))
    rt = _lib.RoutingStruct(*([0x200000] * 12))
    fake = ctypes.c_void_p(0x100000)
    need = s2.workspace_bytes(L, B)
    ws = ctypes.c_void_p(0x400000)
    eo, y = 0x1000000, 0x2000000

    def call(layer=L, n=B, x=fake, router=fake, conf=fake, weights=w, routing=rt, work=ws,
             nbytes=need, out=eo, yy=y):
        st = lib.s2moe_moe_layer(ctypes.byref(layer) if layer is not None else None, n, x, router,
                                 conf, ctypes.byref(weights), ctypes.byref(routing), work, nbytes,
                                 ctypes.c_void_p(out) if out else None,
                                 ctypes.c_void_p(yy) if yy else None, None)
        return st, _lib.last_error()

    st, msg = call(layer=None)
    assert st == _lib.EINVAL and "layer" in msg and msg.startswith("s2moe_moe_layer")
    assert call(n=0)[0] == _lib.EINVAL
    st, msg = call(router=None)
    assert st == _lib.EINVAL and "router" in msg
    st, msg = call(conf=None)
    assert st == _lib.EINVAL and "conf_w" in msg
    st, msg = call(work=None)
    assert st == _lib.EWORKSPACE and "workspace" in msg
    st, msg = call(nbytes=need - 1)
    assert st == _lib.EWORKSPACE and str(need) in msg
    st, msg = call(out=None)
    assert st == _lib.EINVAL and "expert_out" in msg
    st, msg = call(yy=None)
    assert st == _lib.EINVAL and "y" in msg
    st, msg = call(yy=eo + 16)
    assert st == _lib.EINVAL and "overlaps" in msg
    w2 = _lib.Weights(*([0x300000] * 12))
    w2.sh_up = None
    st, msg = call(weights=w2)
    assert st == _lib.EINVAL and "sh_up" in msg
    rt2 = _lib.RoutingStruct(*([0x200000] * 12))
    rt2.gate_w = None
    st, msg = call(routing=rt2)
    assert st == _lib.EINVAL and "gate_w" in msg
    st, msg = call(layer=_layer(cap=1))
    assert st == _lib.EINVAL and "cap" in msg
