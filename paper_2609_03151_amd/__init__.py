"""Python binding of libbasp: one GPU's share of batch-aware Ulysses attention.

Argument marshalling only: every function checks tensor devices, dtypes and
contiguity, then passes raw device pointers, sizes and the current HIP stream
to the C ABI of ``include/basp.h``.  All work runs in the library's HIP
kernels; there is no fallback.  If ``libbasp.so`` has not been built, importing
the library raises.

Names follow the C ABI: ``pack``, ``unpack``, ``attn_fwd``, ``attn_bwd``,
``attn_bwd_workspace_bytes``, ``validate``, ``group_of``, ``status_str``.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbasp.so")

BASP_BF16, BASP_F32 = 0, 1
STATUS = {
    0: "BASP_OK", 1: "BASP_ERR_NULL", 2: "BASP_ERR_SHAPE", 3: "BASP_ERR_RANK",
    4: "BASP_ERR_UNSUPPORTED", 5: "BASP_ERR_ALIGN", 6: "BASP_ERR_WORKSPACE",
    7: "BASP_ERR_HIP", 8: "BASP_ERR_DP_FALLBACK",
}
# Every symbol include/basp.h declares.
EXPORTS = ("basp_status_str", "basp_group_of", "basp_validate", "basp_pack",
           "basp_unpack", "basp_unpack_add", "basp_pack_qkv", "basp_unpack_grads", "basp_a2a_pack", "basp_a2a_unpack",
           "basp_a2a_pack_bf16", "basp_attn_fwd",
           "basp_attn_fwd_sharded", "basp_attn_bwd_workspace_bytes", "basp_attn_bwd",
           "basp_attn_bwd_noalloc", "basp_attn_bwd_sharded_workspace_bytes",
           "basp_attn_bwd_sharded")
# Bytes of the static device buffer basp_attn_bwd_noalloc works in.
NOALLOC_SCRATCH_BYTES = 128 << 20


class BaspError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_str(status)}")


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libbasp.so; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built: run `python -c 'import __graft_entry__ as g; g.build()'` "
            "or `python paper_2609_03151_amd/build.py`")
    L = ctypes.CDLL(LIB_PATH)
    i, vp, sz, f = ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_float
    ip = ctypes.POINTER(ctypes.c_int)
    L.basp_status_str.argtypes = [i]
    L.basp_status_str.restype = ctypes.c_char_p
    L.basp_group_of.argtypes = [i, i, i, ip, ip, ip]
    L.basp_validate.argtypes = [i] * 7
    L.basp_pack.argtypes = [ctypes.POINTER(vp), vp] + [i] * 7 + [vp]
    L.basp_unpack.argtypes = [vp, ctypes.POINTER(vp)] + [i] * 7 + [vp]
    L.basp_unpack_add.argtypes = [vp, ctypes.POINTER(vp)] + [i] * 6 + [vp]
    L.basp_pack_qkv.argtypes = [ctypes.POINTER(vp)] * 3 + [vp] * 3 + [i] * 8 + [vp]
    L.basp_unpack_grads.argtypes = [vp] * 3 + [ctypes.POINTER(vp)] * 3 + [i] * 7 + [vp]
    L.basp_a2a_pack.argtypes = [vp, vp] + [i] * 6 + [vp]
    L.basp_a2a_unpack.argtypes = [vp, vp] + [i] * 6 + [vp]
    L.basp_a2a_pack_bf16.argtypes = [vp, vp] + [i] * 5 + [vp]
    L.basp_attn_fwd.argtypes = [vp] * 5 + [i] * 6 + [f, vp]
    L.basp_attn_bwd_workspace_bytes.argtypes = [i] * 6
    L.basp_attn_bwd_workspace_bytes.restype = sz
    L.basp_attn_bwd_sharded_workspace_bytes.argtypes = [i] * 6
    L.basp_attn_bwd_sharded_workspace_bytes.restype = sz
    L.basp_attn_bwd.argtypes = [vp] * 10 + [sz] + [i] * 6 + [f, vp]
    L.basp_attn_bwd_noalloc.argtypes = [vp] * 9 + [i] * 6 + [f, vp]
    tab = ctypes.POINTER(vp)
    L.basp_attn_fwd_sharded.argtypes = [tab] * 4 + [vp] + [i] * 7 + [f, vp]
    L.basp_attn_bwd_sharded.argtypes = ([tab] * 4 + [vp] + [tab] * 4 + [vp, sz] + [i] * 7
                                        + [f, vp])
    for name in ("basp_group_of", "basp_validate", "basp_pack", "basp_unpack",
                 "basp_a2a_pack", "basp_a2a_unpack", "basp_a2a_pack_bf16", "basp_attn_fwd",
                 "basp_attn_bwd",
                 "basp_attn_bwd_noalloc"):
        getattr(L, name).restype = i
    _lib = L
    return L


def status_str(status: int) -> str:
    return lib().basp_status_str(int(status)).decode()


def _check(rc: int, what: str):
    if rc != 0:
        raise BaspError(rc, what)


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BASP_BF16
    if t.dtype == torch.float32:
        return BASP_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


# ------------------------------------------------------------ host helpers
def group_of(world: int, micro_batch: int, global_rank: int):
    """(group, local_rank, group_size) of a global rank (Alg. 1 / Alg. 2)."""
    g, l, k = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(lib().basp_group_of(world, micro_batch, global_rank, ctypes.byref(g),
                               ctypes.byref(l), ctypes.byref(k)), "basp_group_of")
    return g.value, l.value, k.value


def validate(b, S, H, H_kv, d, G, rank) -> int:
    """Status code of a share's parameters (0 = valid); no GPU needed."""
    return lib().basp_validate(b, S, H, H_kv, d, G, rank)


# ------------------------------------------------------------ permutations
def heads_per_member(n: int, G: int) -> int:
    """Heads of an n-head tensor one member handles: n/G, or 1 for a head
    shared by G/n members (n < G, G divisible by n); 0 if neither holds."""
    if n % G == 0:
        return n // G
    return 1 if (n < G and G % n == 0) else 0


def pack(shards, rank: int, out: torch.Tensor | None = None) -> torch.Tensor:
    """G shards [b, S/G, n, d] -> the rank's head-sharded [b, S, nl, d]."""
    G = len(shards)
    b, Sg, n, d = shards[0].shape
    ptrs = (ctypes.c_void_p * G)(*[_dev(s, f"shards[{j}]", shards[0].dtype).value
                                   for j, s in enumerate(shards)])
    for s in shards:
        if s.shape != shards[0].shape or s.device != shards[0].device:
            raise ValueError("shards differ in shape or device")
    if out is None:
        out = torch.empty((b, Sg * G, heads_per_member(n, G), d), dtype=shards[0].dtype,
                          device=shards[0].device)
    _check(lib().basp_pack(ptrs, _dev(out, "out", shards[0].dtype), b, Sg * G, n, d, G, rank,
                           _dtype_code(out), _stream(out)), "basp_pack")
    return out


def unpack(local: torch.Tensor, shards, rank: int):
    """Write local [b, S, n/G, d] into the rank's head slice of every shard."""
    G = len(shards)
    b, Sg, n, d = shards[0].shape
    ptrs = (ctypes.c_void_p * G)(*[_dev(s, f"shards[{j}]", local.dtype).value
                                   for j, s in enumerate(shards)])
    _check(lib().basp_unpack(_dev(local, "local"), ptrs, b, Sg * G, n, d, G, rank,
                             _dtype_code(local), _stream(local)), "basp_unpack")
    return shards


def unpack_add(local: torch.Tensor, shards, rank: int):
    """fp32: add local [b, S, nl, d] into the rank's head slice of every shard
    (gradients of kv heads that several members share)."""
    G = len(shards)
    b, Sg, n, d = shards[0].shape
    ptrs = (ctypes.c_void_p * G)(*[_dev(s, f"shards[{j}]", torch.float32).value
                                   for j, s in enumerate(shards)])
    _check(lib().basp_unpack_add(_dev(local, "local", torch.float32), ptrs, b, Sg * G, n, d, G,
                                 rank, _stream(local)), "basp_unpack_add")
    return shards


def pack_qkv(q_shards, k_shards, v_shards, rank: int, q=None, k=None, v=None):
    """pack of Q, K and V in one call (one launch when G <= 16); returns (q, k, v)."""
    G = len(q_shards)
    b, Sg, H, d = q_shards[0].shape
    H_kv = k_shards[0].shape[2]
    dt = q_shards[0].dtype
    dev = q_shards[0].device
    if q is None:
        q = torch.empty((b, Sg * G, heads_per_member(H, G), d), dtype=dt, device=dev)
    if k is None:
        k = torch.empty((b, Sg * G, heads_per_member(H_kv, G), d), dtype=dt, device=dev)
    if v is None:
        v = torch.empty_like(k)
    tab = lambda xs, nm: (ctypes.c_void_p * G)(*[_dev(t, f"{nm}[{j}]", dt).value
                                                 for j, t in enumerate(xs)])
    _check(lib().basp_pack_qkv(tab(q_shards, "q_shards"), tab(k_shards, "k_shards"),
                               tab(v_shards, "v_shards"), _dev(q, "q", dt), _dev(k, "k", dt),
                               _dev(v, "v", dt), b, Sg * G, H, H_kv, d, G, rank, _dtype_code(q),
                               _stream(q)), "basp_pack_qkv")
    return q, k, v


def unpack_grads(dq, dk, dv, dq_shards, dk_shards, dv_shards, rank: int):
    """fp32 unpack of dQ, dK, dV in one call; dK, dV are added into the shards
    when the rank's kv head is shared (H_kv < G)."""
    G = len(dq_shards)
    b, Sg, H, d = dq_shards[0].shape
    H_kv = dk_shards[0].shape[2]
    f32 = torch.float32
    tab = lambda xs, nm: (ctypes.c_void_p * G)(*[_dev(t, f"{nm}[{j}]", f32).value
                                                 for j, t in enumerate(xs)])
    _check(lib().basp_unpack_grads(_dev(dq, "dq", f32), _dev(dk, "dk", f32), _dev(dv, "dv", f32),
                                   tab(dq_shards, "dq_shards"), tab(dk_shards, "dk_shards"),
                                   tab(dv_shards, "dv_shards"), b, Sg * G, H, H_kv, d, G, rank,
                                   _stream(dq)), "basp_unpack_grads")


def a2a_pack(own: torch.Tensor, G: int, out: torch.Tensor | None = None) -> torch.Tensor:
    """Own shard [b, S/G, n, d] -> send buffer [G, b, S/G, nl, d], one block per member."""
    b, Sg, n, d = own.shape
    if out is None:
        out = torch.empty((G, b, Sg, heads_per_member(n, G), d), dtype=own.dtype,
                          device=own.device)
    _check(lib().basp_a2a_pack(_dev(own, "own"), _dev(out, "out", own.dtype), b, Sg * G, n, d,
                               G, _dtype_code(own), _stream(own)), "basp_a2a_pack")
    return out


def a2a_pack_bf16(own: torch.Tensor, G: int, out: torch.Tensor | None = None) -> torch.Tensor:
    """fp32 own shard [b, S/G, n, d] -> bf16 send buffer [G, b, S/G, nl, d]
    (a2a_pack with the conversion to bf16, round to nearest even, fused)."""
    b, Sg, n, d = own.shape
    if out is None:
        out = torch.empty((G, b, Sg, heads_per_member(n, G), d), dtype=torch.bfloat16,
                          device=own.device)
    _check(lib().basp_a2a_pack_bf16(_dev(own, "own", torch.float32),
                                    _dev(out, "out", torch.bfloat16), b, Sg * G, n, d, G,
                                    _stream(own)), "basp_a2a_pack_bf16")
    return out


def a2a_unpack(recv: torch.Tensor, out: torch.Tensor | None = None,
               n_heads: int | None = None) -> torch.Tensor:
    """Received blocks [G, b, S/G, n/G, d] -> own shard [b, S/G, n, d].

    ``n_heads`` < G: fp32 gradients of shared heads, blocks [G, b, S/G, 1, d]
    summed per head in member order."""
    G, b, Sg, nl, d = recv.shape
    n = G * nl if n_heads is None else n_heads
    if out is None:
        out = torch.empty((b, Sg, n, d), dtype=recv.dtype, device=recv.device)
    _check(lib().basp_a2a_unpack(_dev(recv, "recv"), _dev(out, "out", recv.dtype), b, Sg * G,
                                 n, d, G, _dtype_code(recv), _stream(recv)),
           "basp_a2a_unpack")
    return out


# -------------------------------------------------------------- attention
def _attn_dims(q, k, G, H_kv):
    b, S, Hl, d = q.shape
    Hkl = k.shape[2]
    if k.shape[:2] != (b, S) or k.shape[3] != d:
        raise ValueError("q and k/v disagree in shape")
    if H_kv is None:
        H_kv = Hkl * G
    elif heads_per_member(H_kv, G) != Hkl:
        raise ValueError(f"k/v hold {Hkl} heads; a member of {G} handles "
                         f"{heads_per_member(H_kv, G)} of {H_kv}")
    return b, S, Hl * G, H_kv, d


def attn_fwd(q, k, v, G: int = 1, scale: float | None = None, out=None, lse=None,
             H_kv: int | None = None):
    """Causal GQA attention of the local heads: returns (o bf16, lse fp32 [b,Hl,S]).

    ``H_kv``: global kv heads (default: k's heads times G); give it when fewer
    kv heads than members share one head per member."""
    b, S, H, H_kv, d = _attn_dims(q, k, G, H_kv)
    scale = d ** -0.5 if scale is None else scale
    if v.shape != k.shape:
        raise ValueError("v must have k's shape")
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((b, q.shape[2], S), dtype=torch.float32, device=q.device)
    _check(lib().basp_attn_fwd(_dev(q, "q", torch.bfloat16), _dev(k, "k", torch.bfloat16),
                               _dev(v, "v", torch.bfloat16), _dev(out, "o", torch.bfloat16),
                               _dev(lse, "lse", torch.float32), b, S, H, H_kv, d, G,
                               float(scale), _stream(q)), "basp_attn_fwd")
    return out, lse


def attn_bwd_workspace_bytes(b, S, H, H_kv, d, G) -> int:
    return int(lib().basp_attn_bwd_workspace_bytes(b, S, H, H_kv, d, G))


def attn_bwd_sharded_workspace_bytes(b, S, H, H_kv, d, G) -> int:
    return int(lib().basp_attn_bwd_sharded_workspace_bytes(b, S, H, H_kv, d, G))


def attn_bwd(q, k, v, o, lse, do, G: int = 1, scale: float | None = None,
             dq=None, dk=None, dv=None, workspace=None, H_kv: int | None = None):
    """Backward of attn_fwd: returns (dq, dk, dv) in fp32."""
    b, S, H, H_kv, d = _attn_dims(q, k, G, H_kv)
    scale = d ** -0.5 if scale is None else scale
    if dq is None:
        dq = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if dk is None:
        dk = torch.empty(k.shape, dtype=torch.float32, device=q.device)
    if dv is None:
        dv = torch.empty(v.shape, dtype=torch.float32, device=q.device)
    need = attn_bwd_workspace_bytes(b, S, H, H_kv, d, G)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    _check(lib().basp_attn_bwd(
        _dev(q, "q", torch.bfloat16), _dev(k, "k", torch.bfloat16),
        _dev(v, "v", torch.bfloat16), _dev(o, "o", torch.bfloat16),
        _dev(lse, "lse", torch.float32), _dev(do, "do", torch.bfloat16),
        _dev(dq, "dq", torch.float32), _dev(dk, "dk", torch.float32),
        _dev(dv, "dv", torch.float32), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), b, S, H, H_kv, d, G, float(scale),
        _stream(q)), "basp_attn_bwd")
    return dq, dk, dv


def attn_bwd_noalloc(q, k, v, o, lse, do, dq, dk, dv, G: int = 1, scale: float | None = None,
                     H_kv: int | None = None):
    """attn_bwd into caller-given dq, dk, dv (fp32) with no workspace argument:
    the library's static device buffer serves instead (basp_attn_bwd_noalloc)."""
    b, S, H, H_kv, d = _attn_dims(q, k, G, H_kv)
    scale = d ** -0.5 if scale is None else scale
    _check(lib().basp_attn_bwd_noalloc(
        _dev(q, "q", torch.bfloat16), _dev(k, "k", torch.bfloat16),
        _dev(v, "v", torch.bfloat16), _dev(o, "o", torch.bfloat16),
        _dev(lse, "lse", torch.float32), _dev(do, "do", torch.bfloat16),
        _dev(dq, "dq", torch.float32), _dev(dk, "dk", torch.float32),
        _dev(dv, "dv", torch.float32), b, S, H, H_kv, d, G, float(scale),
        _stream(q)), "basp_attn_bwd_noalloc")
    return dq, dk, dv


# ------------------------------------------------- attention on the shards
def _table(shards, name, dtype):
    return (ctypes.c_void_p * len(shards))(*[_dev(t, f"{name}[{j}]", dtype).value
                                             for j, t in enumerate(shards)])


def attn_fwd_sharded(q_shards, k_shards, v_shards, o_shards, rank: int,
                     scale: float | None = None, lse=None):
    """Attention of the rank's heads read from the G sequence shards (each
    [b, S/G, H or H_kv, d] bf16) and written into the rank's head slice of
    o_shards; returns lse [b, H/G, S]."""
    G = len(q_shards)
    b, Sg, H, d = q_shards[0].shape
    H_kv = k_shards[0].shape[2]
    S = Sg * G
    scale = d ** -0.5 if scale is None else scale
    if lse is None:
        lse = torch.empty((b, H // G, S), dtype=torch.float32, device=q_shards[0].device)
    bf = torch.bfloat16
    _check(lib().basp_attn_fwd_sharded(
        _table(q_shards, "q", bf), _table(k_shards, "k", bf), _table(v_shards, "v", bf),
        _table(o_shards, "o", bf), _dev(lse, "lse", torch.float32), b, S, H, H_kv, d, G, rank,
        float(scale), _stream(lse)), "basp_attn_fwd_sharded")
    return lse


def attn_bwd_sharded(q_shards, k_shards, v_shards, o_shards, lse, do_shards, dq_shards,
                     dk_shards, dv_shards, rank: int, scale: float | None = None,
                     workspace=None):
    """Backward of attn_fwd_sharded: dQ, dK, dV (fp32) into the rank's head
    slices of their shard buffers.  With a shared kv head (H_kv < G),
    dk_shards / dv_shards are the G send blocks [b, S/G, 1, d] of this
    member's partial dK, dV instead."""
    G = len(q_shards)
    b, Sg, H, d = q_shards[0].shape
    H_kv = k_shards[0].shape[2]
    S = Sg * G
    scale = d ** -0.5 if scale is None else scale
    need = attn_bwd_sharded_workspace_bytes(b, S, H, H_kv, d, G)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=lse.device)
    bf, f32 = torch.bfloat16, torch.float32
    _check(lib().basp_attn_bwd_sharded(
        _table(q_shards, "q", bf), _table(k_shards, "k", bf), _table(v_shards, "v", bf),
        _table(o_shards, "o", bf), _dev(lse, "lse", f32), _table(do_shards, "do", bf),
        _table(dq_shards, "dq", f32), _table(dk_shards, "dk", f32), _table(dv_shards, "dv", f32),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        b, S, H, H_kv, d, G, rank, float(scale), _stream(lse)), "basp_attn_bwd_sharded")
