"""CPU oracle for one rank's share of batch-aware Ulysses attention.

TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the
benchmark's CPU-baseline leg are the only callers; the HIP library and its
Python binding never import this package, and this package never imports them.

The arithmetic lives in ``basp_oracle.c`` (plain C, fp64, OpenMP); this module
only builds it with gcc and marshals numpy/torch arrays through ctypes.
Attention functions take float64 arrays (bf16 inputs convert exactly).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "basp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# x86-64-v3 (AVX2 + FMA) so that a library built in one container also runs on
# another host; no fast-math, no contraction: plain IEEE fp64.
CFLAGS = ["-O3", "-march=x86-64-v3", "-ffp-contract=off", "-fopenmp", "-fPIC",
          "-shared", "-std=c11", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    """Compile liboracle.so with gcc (always recompiles)."""
    cmd = ["gcc", *CFLAGS, _SRC, "-o", _LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def lib():
    """Load liboracle.so, building it first only if nothing is built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    L = ctypes.CDLL(_LIB)
    c_long, c_int, c_double = ctypes.c_long, ctypes.c_int, ctypes.c_double
    vp, lp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_long)
    L.oracle_group_of.argtypes = [c_long, c_long, c_long, lp, lp, lp]
    L.oracle_seq_partition.argtypes = [c_long, c_long, c_long, lp, lp, lp, lp]
    L.oracle_pack.argtypes = [ctypes.POINTER(vp), vp] + [c_long] * 7
    L.oracle_unpack.argtypes = [vp, ctypes.POINTER(vp)] + [c_long] * 7
    L.oracle_unpack_add.argtypes = [vp, ctypes.POINTER(vp)] + [c_long] * 6
    L.oracle_a2a_pack.argtypes = [vp, vp] + [c_long] * 6
    L.oracle_a2a_unpack.argtypes = [vp, vp] + [c_long] * 6
    L.oracle_a2a_pack_bf16.argtypes = [vp, vp] + [c_long] * 5
    L.oracle_attn_fwd.argtypes = [vp] * 5 + [c_long] * 5 + [c_double, c_long, c_long]
    L.oracle_attn_bwd.argtypes = [vp] * 9 + [c_long] * 5 + [c_double, c_long]
    L.oracle_attn_rows.argtypes = ([vp] * 4 + [c_long] * 5 + [c_double, c_long]
                                   + [vp] * 6)
    L.oracle_set_threads.argtypes = [c_int]
    L.oracle_set_threads.restype = None
    L.oracle_attn_keys.argtypes = ([vp] * 6 + [c_long] * 5 + [c_double, c_long]
                                   + [vp] * 5)
    for f in ("oracle_group_of", "oracle_seq_partition", "oracle_pack",
              "oracle_unpack", "oracle_attn_fwd", "oracle_attn_bwd",
              "oracle_attn_rows", "oracle_attn_keys", "oracle_threads"):
        getattr(L, f).restype = c_int
    _lib = L
    return L


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} failed with code {rc}")


def threads() -> int:
    return lib().oracle_threads()


def set_threads(n: int) -> None:
    """Run the oracle's parallel loops on n threads (n < 1: all processors)."""
    lib().oracle_set_threads(int(n))


def _np(x) -> np.ndarray:
    """A C-contiguous numpy view (torch CPU tensors are converted)."""
    if hasattr(x, "detach"):
        x = x.detach().cpu()
        if str(x.dtype) == "torch.bfloat16":
            import torch
            x = x.view(torch.int16)
        x = x.numpy()
    return np.ascontiguousarray(x)


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):
        x = x.detach().cpu().double().numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


# ------------------------------------------------------------- index math
def group_of(world: int, micro_batch: int, global_rank: int):
    """Alg. 1 + Alg. 2: (group, local rank, group size K) of a global rank."""
    g, l, k = ctypes.c_long(), ctypes.c_long(), ctypes.c_long()
    rc = lib().oracle_group_of(world, micro_batch, global_rank,
                               ctypes.byref(g), ctypes.byref(l), ctypes.byref(k))
    _check(rc, "group_of")
    return g.value, l.value, k.value


def seq_partition(L: int, K: int, global_rank: int):
    """Alg. 2: (seq_start, seq_end, tok_start, tok_end) of a global rank."""
    out = [ctypes.c_long() for _ in range(4)]
    rc = lib().oracle_seq_partition(L, K, global_rank, *[ctypes.byref(o) for o in out])
    _check(rc, "seq_partition")
    return tuple(o.value for o in out)


# ------------------------------------------------------------ permutations
def pack(shards, rank: int, out: np.ndarray | None = None) -> np.ndarray:
    """G shards [b, S/G, n, d] -> head-sharded local [b, S, n/G, d] (raw bytes).

    ``out``: optional C-contiguous destination of that shape and dtype."""
    arrs = [_np(s) for s in shards]
    G = len(arrs)
    b, Sg, n, d = arrs[0].shape
    for a in arrs:
        if a.shape != arrs[0].shape or a.dtype != arrs[0].dtype:
            raise OracleError("shards differ in shape or dtype")
    nl = n // G if n % G == 0 else (1 if (n < G and G % n == 0) else 0)
    shape = (b, Sg * G, nl, d)
    if out is None:
        out = np.empty(shape, dtype=arrs[0].dtype)
    elif (out.shape != shape or out.dtype != arrs[0].dtype or not out.flags.c_contiguous):
        raise OracleError("out must be a C-contiguous array of the packed shape and dtype")
    ptrs = (ctypes.c_void_p * G)(*[a.ctypes.data for a in arrs])
    rc = lib().oracle_pack(ptrs, _ptr(out), b, Sg * G, n, d, G, rank,
                           arrs[0].dtype.itemsize)
    _check(rc, "pack")
    return out


def unpack(local, shards, rank: int):
    """Write local [b, S, n/G, d] into the rank's head slice of the G shards.

    ``shards`` are numpy arrays modified in place (other heads untouched)."""
    src = _np(local)
    G = len(shards)
    b, Sg, n, d = shards[0].shape
    for a in shards:
        if not (isinstance(a, np.ndarray) and a.flags.c_contiguous):
            raise OracleError("unpack targets must be C-contiguous numpy arrays")
        if a.dtype.itemsize != src.dtype.itemsize:
            raise OracleError("element size mismatch")
    ptrs = (ctypes.c_void_p * G)(*[a.ctypes.data for a in shards])
    rc = lib().oracle_unpack(_ptr(src), ptrs, b, Sg * G, n, d, G, rank,
                             src.dtype.itemsize)
    _check(rc, "unpack")
    return shards


def a2a_pack(own, G: int) -> np.ndarray:
    """Own shard [b, S/G, n, d] -> send buffer [G, b, S/G, n/G, d] (raw bytes)."""
    src = _np(own)
    b, Sg, n, d = src.shape
    nl = n // G if n % G == 0 else (1 if (n < G and G % n == 0) else 0)
    out = np.empty((G, b, Sg, nl, d), dtype=src.dtype)
    rc = lib().oracle_a2a_pack(_ptr(src), _ptr(out), b, Sg * G, n, d, G, src.dtype.itemsize)
    _check(rc, "a2a_pack")
    return out


def a2a_pack_bf16(own, G: int) -> np.ndarray:
    """fp32 own shard [b, S/G, n, d] -> bf16 bit patterns [G, b, S/G, n/G, d]
    (uint16), each element rounded to nearest even."""
    src = np.ascontiguousarray(own.detach().cpu().numpy() if hasattr(own, "detach") else own,
                               dtype=np.float32)
    b, Sg, n, d = src.shape
    nl = n // G if n % G == 0 else (1 if (n < G and G % n == 0) else 0)
    out = np.empty((G, b, Sg, nl, d), dtype=np.uint16)
    rc = lib().oracle_a2a_pack_bf16(_ptr(src), _ptr(out), b, Sg * G, n, d, G)
    _check(rc, "a2a_pack_bf16")
    return out


def a2a_unpack(recv, n_heads: int | None = None) -> np.ndarray:
    """Received blocks [G, b, S/G, n/G, d] -> own shard [b, S/G, n, d] (raw bytes).

    ``n_heads`` < G (shared heads, fp32): blocks [G, b, S/G, 1, d] are summed per head."""
    src = _np(recv)
    G, b, Sg, nl, d = src.shape
    n = G * nl if n_heads is None else n_heads
    out = np.empty((b, Sg, n, d), dtype=src.dtype)
    rc = lib().oracle_a2a_unpack(_ptr(src), _ptr(out), b, Sg * G, n, d, G,
                                 src.dtype.itemsize)
    _check(rc, "a2a_unpack")
    return out


def unpack_add(local, shards, rank: int):
    """fp32: add local [b, S, nl, d] into the rank's head slice of the G shards
    (numpy float32 arrays, modified in place); nl = n/G, or 1 for a shared head."""
    src = np.ascontiguousarray(_np(local), dtype=np.float32)
    G = len(shards)
    b, Sg, n, d = shards[0].shape
    for a in shards:
        if not (isinstance(a, np.ndarray) and a.flags.c_contiguous and a.dtype == np.float32):
            raise OracleError("unpack_add targets must be C-contiguous float32 numpy arrays")
    ptrs = (ctypes.c_void_p * G)(*[a.ctypes.data for a in shards])
    rc = lib().oracle_unpack_add(_ptr(src), ptrs, b, Sg * G, n, d, G, rank)
    _check(rc, "unpack_add")
    return shards


def heads_per_member(n: int, G: int) -> int:
    return n // G if n >= G else 1


# -------------------------------------------------------------- attention
def attn_fwd(q, k, v, scale: float, r0: int = 0, r1: int | None = None):
    """Causal GQA attention rows [r0, r1): returns (o [b,R,Hl,d], lse [b,Hl,R])."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    b, S, Hl, d = q.shape
    Hkl = k.shape[2]
    r1 = S if r1 is None else r1
    R = r1 - r0
    o = np.empty((b, R, Hl, d))
    lse = np.empty((b, Hl, R))
    rc = lib().oracle_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                               b, S, Hl, Hkl, d, scale, r0, r1)
    _check(rc, "attn_fwd")
    return o, lse


def attn_bwd(q, k, v, do, o, lse, scale: float, r0: int = 0):
    """Gradients of sum(O*dO) for query/key rows [r0, S): (dq, dk, dv), fp64."""
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    o, lse = _f64(o), _f64(lse)
    b, S, Hl, d = q.shape
    Hkl = k.shape[2]
    R = S - r0
    if o.shape != (b, R, Hl, d) or lse.shape != (b, Hl, R):
        raise OracleError("o/lse must cover rows [r0, S)")
    dq = np.empty((b, R, Hl, d))
    dk = np.empty((b, R, Hkl, d))
    dv = np.empty((b, R, Hkl, d))
    rc = lib().oracle_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(do), _ptr(o),
                               _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv),
                               b, S, Hl, Hkl, d, scale, r0)
    _check(rc, "attn_bwd")
    return dq, dk, dv


def attn_rows(q, k, v, do, scale: float, beta, head, row):
    """Row-local O, LSE and dQ at the sampled (beta, head, row) triples."""
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    b, S, Hl, d = q.shape
    Hkl = k.shape[2]
    beta = np.ascontiguousarray(beta, dtype=np.int64)
    head = np.ascontiguousarray(head, dtype=np.int64)
    row = np.ascontiguousarray(row, dtype=np.int64)
    n = len(row)
    o = np.empty((n, d))
    lse = np.empty((n,))
    dq = np.empty((n, d))
    rc = lib().oracle_attn_rows(_ptr(q), _ptr(k), _ptr(v), _ptr(do), b, S, Hl,
                                Hkl, d, scale, n, _ptr(beta), _ptr(head),
                                _ptr(row), _ptr(o), _ptr(lse), _ptr(dq))
    _check(rc, "attn_rows")
    return o, lse, dq


def attn_keys(q, k, v, do, o, lse, scale: float, beta, kvhead, key):
    """dK_j and dV_j (summed over the kv head's query heads) at the sampled
    (beta, kv head, key) triples; o [b,S,Hl,d] and lse [b,Hl,S] are every row
    of ``attn_fwd``."""
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    o, lse = _f64(o), _f64(lse)
    b, S, Hl, d = q.shape
    Hkl = k.shape[2]
    if o.shape != (b, S, Hl, d) or lse.shape != (b, Hl, S):
        raise OracleError("o/lse must cover every row")
    beta = np.ascontiguousarray(beta, dtype=np.int64)
    kvhead = np.ascontiguousarray(kvhead, dtype=np.int64)
    key = np.ascontiguousarray(key, dtype=np.int64)
    n = len(key)
    dk = np.empty((n, d))
    dv = np.empty((n, d))
    rc = lib().oracle_attn_keys(_ptr(q), _ptr(k), _ptr(v), _ptr(do), _ptr(o), _ptr(lse),
                                b, S, Hl, Hkl, d, scale, n, _ptr(beta), _ptr(kvhead),
                                _ptr(key), _ptr(dk), _ptr(dv))
    _check(rc, "attn_keys")
    return dk, dv
