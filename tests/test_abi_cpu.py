"""The C ABI library loads, exports every declared symbol, and validates its
arguments on the host before any HIP call (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2512_14080_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sonicmoe.h")

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="libsonicmoe.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 13
    L = ctypes.CDLL(B.LIB_PATH)
    for name in names:
        assert hasattr(L, name), name
    assert set(B.EXPORTS) == set(names)


def test_binding_constants_match_the_header():
    """Every enumerator the header gives an explicit value (flags, states,
    modes, error codes, kernel classes by position) has the same value in
    the ctypes binding, where the binding defines it."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    explicit = {n: int(v) for n, v in re.findall(r"\b(MOE_[A-Z0-9_]+)\s*=\s*(-?\d+)", text)}
    assert "MOE_ROUTE_SEPARATE_TOPK" in explicit
    checked = 0
    for name, value in explicit.items():
        if hasattr(B, name):
            assert getattr(B, name) == value, name
            checked += 1
    assert checked >= 10
    # kernel classes: the enum's order is the binding's list order
    kc = re.search(r"enum\s*\{\s*(MOE_KC_ROUTER_GEMM[^}]*)\}", text).group(1)
    names = [n for n in re.findall(r"\b(MOE_KC_[A-Z0-9_]+)", kc) if n != "MOE_KC_COUNT"]
    assert len(names) == len(B.KERNEL_CLASSES)


def test_strerror_and_class_names():
    assert B.moe_strerror(0) == "success"
    assert "capacity" in B.moe_strerror(B.MOE_ERR_CAPACITY)
    assert B.lib().moe_kernel_class_name(4).decode() == "up_proj"
    assert [B.lib().moe_kernel_class_name(i).decode() for i in range(len(B.KERNEL_CLASSES))] == B.KERNEL_CLASSES


def test_sizes():
    D = B.dims(32768, 1536, 256, 128, 8)
    assert B.moe_round_capacity(D, 128) == 32768 * 8 + 128 * 127
    assert B.moe_round_capacity(B.dims(10, 128, 64, 8, 2), 128) == 80  # capped at T*E
    assert B.moe_routing_bytes(D, 32768 * 8, 0) > 0
    fwd = B.moe_workspace_bytes(D, 262144, B.MOE_WS_FWD)
    assert fwd >= 262144 * (256 + 1536) * 2
    assert B.moe_workspace_bytes(D, 262144, B.MOE_WS_BWD) >= 262144 * (512 + 256 + 1536) * 2
    assert B.moe_workspace_bytes(D, 262144, 7) == 0


@pytest.mark.parametrize("dims,code", [
    ((0, 128, 64, 8, 2), B.MOE_ERR_INVALID_ARG),
    ((16, 100, 64, 8, 2), B.MOE_ERR_UNSUPPORTED),
    ((16, 128, 48, 8, 2), B.MOE_ERR_UNSUPPORTED),
    ((16, 128, 64, 12, 2), B.MOE_ERR_UNSUPPORTED),
    ((16, 128, 64, 8192, 2), B.MOE_ERR_UNSUPPORTED),
    ((16, 128, 64, 8, 9), B.MOE_ERR_UNSUPPORTED),
    ((16, 128, 64, 64, 17), B.MOE_ERR_UNSUPPORTED),
])
def test_invalid_dims_rejected(dims, code):
    D = B.dims(*dims)
    assert B.moe_routing_bytes(D, 1024, 0) == 0
    r = B.MoeRouting()
    rc = B.lib().moe_route(D, None, None, None, 0, ctypes.byref(r), None)
    assert rc == code, B.moe_last_error()


def _fake_routing(D, capacity):
    # non-null, aligned fake addresses: validation only inspects them
    r = B.MoeRouting()
    r.capacity = capacity
    r.words = (D.T + 63) // 64
    r.state = B.MOE_ROUTING_STATE_BUILT
    for i, name in enumerate(B.MoeRouting.pointer_fields()):
        setattr(r, name, 0x10000000 + 0x1000 * i)
    return r


def test_route_validation_before_any_launch():
    D = B.dims(256, 128, 64, 8, 2)
    L = B.lib()
    r = _fake_routing(D, 512)
    # null X / Wr
    assert L.moe_route(D, None, None, None, 0, ctypes.byref(r), None) == B.MOE_ERR_INVALID_ARG
    assert "X" in B.moe_last_error()
    # misaligned X
    assert L.moe_route(D, 0x1008, 0x2000, None, 0, ctypes.byref(r), None) == B.MOE_ERR_INVALID_ARG
    assert "aligned" in B.moe_last_error()
    # capacity below T*K
    r_small = _fake_routing(D, 511)
    assert L.moe_route(D, 0x1000, 0x2000, None, 0, ctypes.byref(r_small), None) == B.MOE_ERR_CAPACITY
    # wrong word count
    r_bad = _fake_routing(D, 512)
    r_bad.words = 3
    assert L.moe_route(D, 0x1000, 0x2000, None, 0, ctypes.byref(r_bad), None) == B.MOE_ERR_INVALID_ARG
    # a required array missing
    r_null = _fake_routing(D, 512)
    r_null.mask = None
    assert L.moe_route(D, 0x1000, 0x2000, None, 0, ctypes.byref(r_null), None) == B.MOE_ERR_INVALID_ARG
    # flags needing optional arrays
    r_nl = _fake_routing(D, 512)
    r_nl.logits = None
    assert L.moe_route(D, 0x1000, 0x2000, None, B.MOE_ROUTE_WRITE_LOGITS, ctypes.byref(r_nl), None) == B.MOE_ERR_INVALID_ARG
    assert L.moe_route(D, 0x1000, 0x2000, None, 64, ctypes.byref(r), None) == B.MOE_ERR_INVALID_ARG
    # the highest defined flag is MOE_ROUTE_SEPARATE_TOPK (16): the next bit is unknown
    assert B.MOE_ROUTE_SEPARATE_TOPK == 16
    assert L.moe_route(D, 0x1000, 0x2000, None, 32, ctypes.byref(r), None) == B.MOE_ERR_INVALID_ARG
    assert "flags" in B.moe_last_error()


def test_round_validation():
    D = B.dims(256, 128, 64, 8, 2)
    L = B.lib()
    tc = _fake_routing(D, 512)
    tr = _fake_routing(D, B.moe_round_capacity(D, 16))
    assert L.moe_round_tokens(D, 0, 0, None, ctypes.byref(tc), ctypes.byref(tr), None) == B.MOE_ERR_INVALID_ARG
    assert L.moe_round_tokens(D, 16, 9, None, ctypes.byref(tc), ctypes.byref(tr), None) == B.MOE_ERR_INVALID_ARG
    assert L.moe_round_tokens(D, 16, 4, None, ctypes.byref(tc), ctypes.byref(tr), None) == B.MOE_ERR_INVALID_ARG
    small = _fake_routing(D, 512)
    assert L.moe_round_tokens(D, 16, 0, None, ctypes.byref(tc), ctypes.byref(small), None) == B.MOE_ERR_CAPACITY
    tc_nost = _fake_routing(D, 512)
    tc_nost.scores_t = None
    assert L.moe_round_tokens(D, 16, 0, None, ctypes.byref(tc_nost), ctypes.byref(tr), None) == B.MOE_ERR_INVALID_ARG
    big = _fake_routing(D, B.moe_round_capacity(D, 16))
    assert L.moe_round_tokens(D, 16, 0, None, ctypes.byref(big), ctypes.byref(big), None) == B.MOE_ERR_INVALID_ARG
    assert "alias" in B.moe_last_error()


def test_fwd_bwd_validation():
    D = B.dims(256, 128, 64, 8, 2)
    L = B.lib()
    r = _fake_routing(D, 512)
    need = B.moe_workspace_bytes(D, 512, B.MOE_WS_FWD)
    a = 0x100000
    assert L.moe_fwd(D, a, a, a, None, ctypes.byref(r), a, a, a, need - 1, None) == B.MOE_ERR_WORKSPACE
    assert L.moe_fwd(D, a, None, a, None, ctypes.byref(r), a, a, a, need, None) == B.MOE_ERR_INVALID_ARG
    assert L.moe_fwd(D, a, a, a, None, ctypes.byref(r), a + 2, a, a, need, None) == B.MOE_ERR_INVALID_ARG
    needb = B.moe_workspace_bytes(D, 512, B.MOE_WS_BWD)
    args = [D, a, a, a, a, a, None, a, ctypes.byref(r), a, a, a, a, a, a, a, needb - 256, None]
    assert L.moe_bwd(*args) == B.MOE_ERR_WORKSPACE
    args = [D, a, a, a, a, a, None, None, ctypes.byref(r), a, a, a, a, None, None, a, needb, None]
    assert L.moe_bwd(*args) == B.MOE_ERR_INVALID_ARG  # dWr without Wr
    assert "Wr" in B.moe_last_error()


def test_routing_init_layout():
    D = B.dims(1000, 128, 64, 16, 4)
    nbytes = B.moe_routing_bytes(D, 4000, B.MOE_ROUTING_SCORES_T)
    r = B.MoeRouting()
    base = 0x7f0000000000
    assert B.lib().moe_routing_init(D, 4000, B.MOE_ROUTING_SCORES_T, base, nbytes, ctypes.byref(r)) == 0
    assert r.words == 16 and r.capacity == 4000 and r.logits is None and r.scores_t
    assert r.state == B.MOE_ROUTING_STATE_EMPTY
    ptrs = sorted(getattr(r, f) for f in B.MoeRouting.pointer_fields() if getattr(r, f))
    assert all(p % 256 == 0 for p in ptrs)
    assert ptrs[0] >= base and ptrs[-1] < base + nbytes
    assert B.lib().moe_routing_init(D, 4000, 0, base, 10, ctypes.byref(r)) == B.MOE_ERR_INVALID_ARG
    assert B.lib().moe_routing_init(D, 3999, 0, base, nbytes, ctypes.byref(r)) == B.MOE_ERR_CAPACITY


def test_prof_select_validation():
    assert B.lib().moe_prof_select(99) == B.MOE_ERR_INVALID_ARG
    assert B.lib().moe_prof_select(-1) == 0


def test_consumers_need_a_built_routing():
    """moe_fwd and moe_bwd refuse a routing whose metadata was never written
    (fresh from moe_routing_init) or stops at the counts
    (MOE_ROUTE_COUNTS_ONLY); moe_round_tokens needs at least the counts."""
    D = B.dims(256, 128, 64, 8, 2)
    L = B.lib()
    a = 0x100000
    need = B.moe_workspace_bytes(D, 512, B.MOE_WS_FWD)
    needb = B.moe_workspace_bytes(D, 512, B.MOE_WS_BWD)
    for state in (B.MOE_ROUTING_STATE_EMPTY, B.MOE_ROUTING_STATE_COUNTS):
        r = _fake_routing(D, 512)
        r.state = state
        assert L.moe_fwd(D, a, a, a, None, ctypes.byref(r), a, a, a, need, None) == B.MOE_ERR_INVALID_ARG
        assert "not a complete routing" in B.moe_last_error()
        args = [D, a, a, a, a, a, None, a, ctypes.byref(r), a, a, a, a, a, a, a, needb, None]
        assert L.moe_bwd(*args) == B.MOE_ERR_INVALID_ARG
        assert "not a complete routing" in B.moe_last_error()
    tc = _fake_routing(D, 512)
    tc.state = B.MOE_ROUTING_STATE_EMPTY
    tr = _fake_routing(D, B.moe_round_capacity(D, 16))
    assert L.moe_round_tokens(D, 16, 0, None, ctypes.byref(tc), ctypes.byref(tr), None) == B.MOE_ERR_INVALID_ARG
    assert "counts" in B.moe_last_error()


@pytest.mark.parametrize("m_tile", [0, 1, 4, 12, 24, 100, 512, 65536])
def test_m_tile_must_be_power_of_two_in_range(m_tile):
    """m_tile is a power of two in [8, 256], as the header states."""
    D = B.dims(256, 128, 64, 8, 2)
    assert B.moe_round_capacity(D, m_tile) == -1
    tc = _fake_routing(D, 512)
    tr = _fake_routing(D, 256 * 8)
    rc = B.lib().moe_round_tokens(D, m_tile, 0, None, ctypes.byref(tc), ctypes.byref(tr), None)
    assert rc == B.MOE_ERR_INVALID_ARG and "power of two" in B.moe_last_error()


@pytest.mark.parametrize("m_tile", [8, 16, 32, 64, 128, 256])
def test_m_tile_accepted(m_tile):
    D = B.dims(256, 128, 64, 8, 2)
    assert B.moe_round_capacity(D, m_tile) == min(256 * 8, 256 * 2 + 8 * (m_tile - 1))


def test_expert_bias_alignment_checked():
    D = B.dims(256, 128, 64, 8, 2)
    L = B.lib()
    r = _fake_routing(D, 512)
    a = 0x100000
    need = B.moe_workspace_bytes(D, 512, B.MOE_WS_FWD)
    eb = B.MoeExpertBias(a + 4, None, None, None)
    assert L.moe_fwd(D, a, a, a, ctypes.byref(eb), ctypes.byref(r), a, a, a, need, None) == B.MOE_ERR_INVALID_ARG
    assert "eb->b1" in B.moe_last_error()
    needb = B.moe_workspace_bytes(D, 512, B.MOE_WS_BWD)
    eb = B.MoeExpertBias(None, None, None, a + 8)
    args = [D, a, a, a, a, a, ctypes.byref(eb), a, ctypes.byref(r), a, a, a, a, a, a, a, needb, None]
    assert L.moe_bwd(*args) == B.MOE_ERR_INVALID_ARG
    assert "eb->db2" in B.moe_last_error()


def test_static_forward_refuses_oversized_workspace():
    """moe_fwd_static refuses, before any HIP call, a routing whose forward
    workspace exceeds its static array."""
    D = B.dims(32768, 1536, 256, 128, 8)
    r = _fake_routing(D, 32768 * 8)
    assert B.moe_workspace_bytes(D, r.capacity, B.MOE_WS_FWD) > B.lib().moe_fwd_static_max_bytes()
    a = 0x100000
    assert B.lib().moe_fwd_static(D, a, a, a, None, ctypes.byref(r), a, a, None) == B.MOE_ERR_WORKSPACE
    assert "static workspace" in B.moe_last_error()
    assert B.lib().moe_fwd_static_max_bytes() == 64 << 20
