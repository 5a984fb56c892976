"""The C ABI of libbasp on a host without a GPU: the library loads, exports
every function include/basp.h declares, and rejects each host-detectable
misuse with its status code before making any HIP call."""
import ctypes
import os
import re

import pytest

import paper_2609_03151_amd as basp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")

OK, NULL, SHAPE, RANK, UNSUP, ALIGN, WS, HIP, DP = range(9)


def _declared():
    with open(os.path.join(ROOT, "include", "basp.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(basp_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = basp.lib()
    names = _declared()
    assert set(names) == set(basp.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    for code, name in basp.STATUS.items():
        assert basp.status_str(code).startswith(name)
    assert "unknown" in basp.status_str(99)


def test_group_of_matches_paper_example_and_errors():
    with open(os.path.join(GOLDEN, "group_formation_n4_b2.txt")) as f:
        rows = [list(map(int, ln.split())) for ln in f if ln.strip() and not ln.startswith("#")]
    for rank, g, l, K, _seq, _chunk in rows:
        assert basp.group_of(4, 2, rank) == (g, l, K)
    for (N, B, r), code in {(6, 4, 0): SHAPE, (4, 8, 0): DP, (4, 2, 4): RANK,
                            (0, 1, 0): SHAPE, (4, 2, -1): RANK}.items():
        with pytest.raises(basp.BaspError) as e:
            basp.group_of(N, B, r)
        assert e.value.status == code
    g = ctypes.c_int()
    assert basp.lib().basp_group_of(4, 2, 0, None, ctypes.byref(g), ctypes.byref(g)) == NULL


@pytest.mark.parametrize("args,code", [
    ((1, 32768, 32, 8, 128, 4, 1), OK),
    ((1, 65536, 28, 4, 128, 4, 3), OK),
    ((2, 512, 8, 8, 64, 2, 0), OK),
    ((0, 512, 8, 8, 64, 2, 0), OK),          # empty batch is valid
    ((1, 0, 8, 8, 64, 2, 0), OK),            # empty sequence is valid
    ((-1, 512, 8, 8, 64, 2, 0), SHAPE),
    ((1, 510, 8, 8, 64, 4, 0), SHAPE),       # S % G
    ((1, 512, 6, 2, 64, 4, 0), SHAPE),       # H % G
    ((1, 512, 12, 3, 64, 4, 0), SHAPE),      # H_kv neither a multiple nor a divisor of G
    ((1, 512, 8, 2, 64, 4, 0), OK),          # 2 kv heads shared by 4 members
    ((1, 16384, 32, 8, 128, 16, 15), OK),    # 8 kv heads, G = 16
    ((1, 512, 8, 1, 64, 8, 7), OK),          # MQA
    ((1, 512, 12, 8, 64, 4, 0), SHAPE),      # H % H_kv
    ((1, 512, 8, 8, 64, 2, 2), RANK),
    ((1, 512, 8, 8, 64, 2, -1), RANK),
    ((1, 512, 8, 8, 96, 2, 0), OK),          # head dims of Table II
    ((1, 512, 8, 8, 80, 2, 0), OK),
    ((1, 512, 8, 8, 72, 2, 0), UNSUP),       # head dim
    ((1, 512, 8, 8, 256, 2, 0), UNSUP),
])
def test_validate(args, code):
    assert basp.validate(*args) == code


def _fake(addr):
    return ctypes.c_void_p(addr)


def test_pack_rejects_before_any_hip_call():
    """Only invalid (or empty) calls here: the pointers are fake host values,
    so a call that passed validation would launch on them."""
    L = basp.lib()
    vp = ctypes.c_void_p
    good = (vp * 2)(0x1000, 0x2000)
    dst = _fake(0x3000)
    cases = [
        ((good, dst, 1, 63, 8, 64, 2, 0, 0), SHAPE),
        ((good, dst, 1, 64, 7, 64, 2, 0, 0), SHAPE),
        ((good, dst, 1, 64, 8, 64, 2, 2, 0), RANK),
        ((good, dst, 1, 64, 8, 64, 2, 0, 5), UNSUP),
        ((None, dst, 1, 64, 8, 64, 2, 0, 0), NULL),
        (((vp * 2)(0x1000, 0), dst, 1, 64, 8, 64, 2, 0, 0), NULL),
        (((vp * 2)(0x1001, 0x2000), dst, 1, 64, 8, 64, 2, 0, 0), ALIGN),
        (((vp * 2)(0x1002, 0x2000), dst, 1, 64, 8, 64, 2, 0, 1), ALIGN),
        ((good, dst, 0, 64, 8, 64, 2, 0, 0), OK),      # empty: nothing enqueued
    ]
    for args, code in cases:
        assert L.basp_pack(*args, None) == code, args
        src = args[1]
        assert L.basp_unpack(src, args[0], *args[2:], None) == code, args


def test_pack_rejects_group_beyond_maximum():
    L = basp.lib()
    G = 256
    ptrs = (ctypes.c_void_p * G)(*[0x1000 * (j + 1) for j in range(G)])
    assert L.basp_pack(ptrs, _fake(0x100000), 1, G, G, 8, G, 0, 0, None) == UNSUP


def test_permutations_reject_sizes_beyond_block_index():
    """(S/G)*(n/G)*d must stay below 2^31 elements and b*G within a grid
    dimension (65535); both are rejected before the pointers are looked at."""
    L = basp.lib()
    good = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    dst = _fake(0x3000)
    # (S/G)*(n/G)*d = 2^21 * 2^4 * 2^6 = 2^31
    assert L.basp_pack(good, dst, 1, 1 << 22, 32, 64, 2, 0, 0, None) == UNSUP
    assert L.basp_unpack(dst, good, 1, 1 << 22, 32, 64, 2, 0, 0, None) == UNSUP
    assert L.basp_a2a_pack(dst, dst, 1, 1 << 22, 32, 64, 2, 0, None) == UNSUP
    assert L.basp_a2a_unpack(dst, dst, 1, 1 << 22, 32, 64, 2, 0, None) == UNSUP
    assert L.basp_pack(good, dst, 32768, 64, 8, 64, 2, 0, 0, None) == UNSUP   # b*G = 65536
    assert L.basp_a2a_pack(dst, dst, 32768, 64, 8, 64, 2, 0, None) == UNSUP
    assert L.basp_pack(None, dst, 1, 1 << 22, 32, 64, 2, 0, 0, None) == UNSUP  # before NULL


def test_a2a_rejects_before_any_hip_call():
    """Only invalid (or empty) calls: the pointers are fake host values."""
    L = basp.lib()
    a, c = _fake(0x1000), _fake(0x2000)
    for fn in (L.basp_a2a_pack, L.basp_a2a_unpack):
        assert fn(a, c, 1, 63, 8, 64, 2, 0, None) == SHAPE       # S % G
        assert fn(a, c, 1, 64, 7, 64, 2, 0, None) == SHAPE       # n % G
        assert fn(a, c, -1, 64, 8, 64, 2, 0, None) == SHAPE
        assert fn(a, c, 1, 64, 8, 64, 2, 3, None) == UNSUP       # dtype
        assert fn(a, c, 1, 64, 8, 64, 256, 0, None) == SHAPE     # 64 % 256
        assert fn(None, c, 1, 64, 8, 64, 2, 0, None) == NULL
        assert fn(a, None, 1, 64, 8, 64, 2, 0, None) == NULL
        assert fn(_fake(0x1001), c, 1, 64, 8, 64, 2, 0, None) == ALIGN
        assert fn(a, _fake(0x2002), 1, 64, 8, 64, 2, 1, None) == ALIGN
        assert fn(None, None, 0, 64, 8, 64, 2, 0, None) == OK    # empty: nothing enqueued


def test_shared_head_calls_reject_before_any_hip_call():
    """n < G: unpack refuses (a shared head must be added), unpack_add and the
    replica-summing a2a_unpack are fp32 only; n neither a multiple nor a
    divisor of G is a shape error everywhere."""
    L = basp.lib()
    vp = ctypes.c_void_p
    good = (vp * 4)(0x1000, 0x2000, 0x3000, 0x4000)
    a, c = _fake(0x10000), _fake(0x20000)
    assert L.basp_unpack(a, good, 1, 64, 2, 64, 4, 0, 1, None) == SHAPE
    assert L.basp_unpack(a, good, 1, 64, 3, 64, 4, 0, 1, None) == SHAPE
    assert L.basp_pack(good, a, 1, 64, 3, 64, 4, 0, 1, None) == SHAPE
    assert L.basp_a2a_unpack(a, c, 1, 64, 2, 64, 4, 0, None) == UNSUP   # bf16 sum
    assert L.basp_a2a_pack(a, c, 1, 64, 3, 64, 4, 0, None) == SHAPE
    assert L.basp_unpack_add(a, good, 1, 64, 3, 64, 4, 0, None) == SHAPE
    assert L.basp_unpack_add(a, good, 1, 64, 2, 64, 4, 4, None) == RANK
    assert L.basp_unpack_add(None, good, 1, 64, 2, 64, 4, 0, None) == NULL
    assert L.basp_unpack_add(_fake(0x10002), good, 1, 64, 2, 64, 4, 0, None) == ALIGN
    assert L.basp_unpack_add(None, None, 0, 64, 2, 64, 4, 0, None) == OK   # empty
    p = [_fake(0x10000 * (i + 1)) for i in range(5)]
    assert L.basp_attn_fwd(*p, 1, 128, 12, 3, 128, 4, ctypes.c_float(0.1), None) == SHAPE
    assert L.basp_attn_bwd_workspace_bytes(1, 128, 8, 2, 128, 4) > 0


def test_sharded_attn_rejects_before_any_hip_call():
    """Only invalid (or empty) calls: the pointer tables hold fake values."""
    L = basp.lib()
    vp = ctypes.c_void_p
    tab = lambda G, base=0x100000: (vp * G)(*[base * (j + 1) for j in range(G)])
    f = lambda x: ctypes.c_float(x)
    fwd = lambda *a, G=4, t=None, lse=_fake(0x40), sc=0.1: L.basp_attn_fwd_sharded(
        *([t or tab(G)] * 4), lse, *a, f(sc), None)
    assert fwd(1, 1024, 8, 2, 128, 4, 4) == RANK
    assert fwd(1, 1002, 8, 2, 128, 4, 0) == SHAPE                  # S % G
    assert fwd(1, 1536, 8, 2, 128, 4, 0) == UNSUP                  # 384 rows per shard
    assert fwd(1, 128 * 256, 128, 128, 128, 128, 0, G=128) == UNSUP  # G > 64
    assert fwd(1, 1024, 8, 2, 72, 4, 0) == UNSUP                   # head dim
    assert fwd(1, 1024, 8, 2, 128, 4, 0, t=(vp * 4)(0x1000, 0, 0x3000, 0x4000)) == NULL
    assert fwd(1, 1024, 8, 2, 128, 4, 0, t=(vp * 4)(0x1000, 0x2008, 0x3000, 0x4000)) == ALIGN
    assert fwd(1, 1024, 8, 2, 128, 4, 0, lse=None) == NULL
    assert fwd(0, 1024, 8, 2, 128, 4, 0) == OK                     # empty
    bwd = lambda *a, G=4, ws=_fake(0x80), n=1 << 30: L.basp_attn_bwd_sharded(
        *([tab(G)] * 4), _fake(0x40), *([tab(G)] * 4), ws, n, *a, f(0.1), None)
    assert bwd(1, 1024, 8, 2, 128, 4, 1, n=16) == WS               # shared kv head (2 < 4)
    assert bwd(1, 1024, 8, 2, 128, 4, 1, ws=None) == NULL
    assert bwd(1, 1024, 8, 4, 128, 4, 1, n=16) == WS
    assert bwd(1, 1024, 8, 4, 128, 4, 1, ws=None) == NULL
    assert bwd(1, 1024, 8, 4, 128, 4, 9) == RANK
    assert bwd(0, 1024, 8, 4, 128, 4, 1) == OK


def test_batched_permutations_reject_before_any_hip_call():
    """basp_pack_qkv / basp_unpack_grads: any of the three tensors' errors
    stops the call before a launch (fake pointers; only invalid or empty)."""
    L = basp.lib()
    vp = ctypes.c_void_p
    tab = lambda base: (vp * 4)(*[base + 0x1000 * j for j in range(4)])
    a, b_, c = _fake(0x100000), _fake(0x200000), _fake(0x300000)
    pk = lambda *x, t=None: L.basp_pack_qkv(*(t or (tab(0x10000), tab(0x20000), tab(0x30000))),
                                           a, b_, c, *x, None)
    assert pk(1, 1024, 8, 3, 128, 4, 0, 0) == SHAPE          # 3 kv heads over 4 members
    assert pk(1, 1022, 8, 4, 128, 4, 0, 0) == SHAPE          # S % G
    assert pk(1, 1024, 8, 4, 128, 4, 4, 0) == RANK
    assert pk(1, 1024, 8, 4, 128, 4, 0, 7) == UNSUP          # dtype
    assert pk(1, 1024, 8, 4, 128, 4, 0, 0,
              t=(tab(0x10000), (vp * 4)(0x20000, 0, 0x22000, 0x23000), tab(0x30000))) == NULL
    assert pk(1, 1024, 8, 4, 128, 4, 0, 0,
              t=(tab(0x10000), tab(0x20000), (vp * 4)(0x30001, 0x31000, 0x32000, 0x33000))) == ALIGN
    assert pk(0, 1024, 8, 4, 128, 4, 0, 0) == OK             # empty
    ug = lambda *x, t=None: L.basp_unpack_grads(a, b_, c, *(t or (tab(0x10000), tab(0x20000),
                                                                   tab(0x30000))), *x, None)
    assert ug(1, 1024, 8, 3, 128, 4, 0) == SHAPE
    assert ug(1, 1024, 8, 4, 128, 4, -1) == RANK
    assert ug(1, 1024, 8, 4, 128, 4, 0, t=(None, tab(0x20000), tab(0x30000))) == NULL
    assert ug(0, 1024, 8, 2, 128, 4, 0) == OK


def test_attn_rejects_before_any_hip_call():
    L = basp.lib()
    p = [_fake(0x10000 * (i + 1)) for i in range(10)]
    fwd = lambda *a, ptrs=p[:5], scale=0.125: L.basp_attn_fwd(*ptrs, *a, ctypes.c_float(scale), None)
    assert fwd(1, 128, 8, 2, 72, 2) == UNSUP
    assert fwd(1, 128, 8, 2, 48, 2) == UNSUP
    assert fwd(1, 128, 8, 2, 128, 2, scale=0.0) == UNSUP
    assert fwd(1, 128, 8, 2, 128, 2, scale=float("nan")) == UNSUP
    assert fwd(1, 127, 8, 2, 128, 2) == SHAPE
    assert fwd(1, 128, 8, 2, 128, 2, ptrs=[None] + p[1:5]) == NULL
    assert fwd(1, 128, 8, 2, 128, 2, ptrs=[_fake(0x10008)] + p[1:5]) == ALIGN
    assert fwd(0, 128, 8, 2, 128, 2) == OK

    need = L.basp_attn_bwd_workspace_bytes(1, 128, 8, 2, 128, 2)
    assert need >= 1 * 4 * 128 * 4 and need % 256 == 0
    bwd = lambda ws, n, *a: L.basp_attn_bwd(*p[:9], ws, n, *a, ctypes.c_float(0.125), None)
    assert bwd(p[9], need - 1, 1, 128, 8, 2, 128, 2) == WS
    assert bwd(None, need, 1, 128, 8, 2, 128, 2) == NULL
    assert bwd(p[9], need, 1, 128, 8, 2, 64, 3) == SHAPE
    assert bwd(p[9], 0, 0, 128, 8, 2, 128, 2) == OK


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(basp, "_lib", None)
    monkeypatch.setattr(basp, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        basp.lib()


def test_noalloc_backward_rejects_before_any_hip_call():
    """basp_attn_bwd_noalloc: the shape checks of basp_attn_bwd, and a shape whose
    workspace exceeds the static buffer is refused (fake pointers: only invalid
    or empty calls here)."""
    L = basp.lib()
    p = [_fake(0x10000 * (i + 1)) for i in range(9)]
    f = ctypes.c_float(0.125)
    assert L.basp_attn_bwd_workspace_bytes(1, 131072, 64, 8, 128, 8) > basp.NOALLOC_SCRATCH_BYTES
    assert L.basp_attn_bwd_noalloc(*p, 1, 131072, 64, 8, 128, 8, f, None) == WS
    assert L.basp_attn_bwd_noalloc(*p[:5], None, *p[6:], 1, 4096, 8, 2, 128, 2, f, None) == NULL
    assert L.basp_attn_bwd_noalloc(*p, 1, 4096, 8, 2, 72, 2, f, None) == UNSUP
    assert L.basp_attn_bwd_noalloc(*p, 1, 4095, 8, 2, 128, 2, f, None) == SHAPE
    assert L.basp_attn_bwd_noalloc(*([None] * 9), 0, 4096, 8, 2, 128, 2, f, None) == OK


def test_a2a_pack_bf16_rejects_before_any_hip_call():
    """Only invalid (or empty) calls: the pointers are fake host values."""
    L = basp.lib()
    a, c = _fake(0x1000), _fake(0x2000)
    f = L.basp_a2a_pack_bf16
    assert f(a, c, 1, 63, 8, 64, 2, None) == SHAPE       # S % G
    assert f(a, c, 1, 64, 6, 64, 4, None) == SHAPE       # n neither multiple nor divisor of G
    assert f(a, c, 1, 64, 8, 64, 256, None) == SHAPE
    assert f(None, c, 1, 64, 8, 64, 2, None) == NULL
    assert f(a, None, 1, 64, 8, 64, 2, None) == NULL
    assert f(_fake(0x1002), c, 1, 64, 8, 64, 2, None) == ALIGN
    assert f(a, _fake(0x2001), 1, 64, 8, 64, 2, None) == ALIGN
    assert f(a, c, 1, 1 << 22, 32, 64, 2, None) == UNSUP
    assert f(None, None, 0, 64, 8, 64, 2, None) == OK    # empty


@pytest.mark.parametrize("S", [32768, 131072, 262144, 1 << 20])
def test_backward_workspace_grows_linearly_with_sequence(S):
    """The key pass's row-chunk partial sums take (chunks x S) rows; with at
    most 16 chunks the workspace stays linear in S: the two planes plus at
    most 16 fp32 dV and dK partials of the rank's kv heads."""
    L = basp.lib()
    b, H, H_kv, d, G = 1, 8, 8, 128, 8   # one local query and kv head
    planes = 2 * b * (H // G) * ((S + 63) // 64 * 64) * 4
    bound = planes + 256 + 2 * 16 * b * (H_kv // G) * S * d * 4
    need = L.basp_attn_bwd_workspace_bytes(b, S, H, H_kv, d, G)
    assert planes < need <= bound
