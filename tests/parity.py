"""Helpers shared by the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import functools
import sys

import numpy as np
import torch

from synth_inputs import WORKLOADS, global_tensors, shards_of

# Attention parity bar against the fp64 oracle, per output tensor.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
LSE_MAX_ABS = 1e-3


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def check_close(name: str, got, ref, max_abs=MAX_ABS, mean_abs=MEAN_ABS):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    err = np.abs(got - ref)
    mx, mn = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    log(f"  {name}: max|d|={mx:.3e} mean|d|={mn:.3e} (ref max {np.abs(ref).max() if ref.size else 0:.3g})")
    assert mx <= max_abs, f"{name}: max abs error {mx} > {max_abs}"
    assert mn <= mean_abs, f"{name}: mean abs error {mn} > {mean_abs}"
    return mx, mn


@functools.lru_cache(maxsize=2)
def workload_inputs(name: str):
    """Global bf16 tensors of a named workload (CPU), drawn once per process."""
    w = WORKLOADS[name]
    log(f"  drawing inputs of {name} (seed {w.seed})")
    return global_tensors(w)


def local_heads(x: torch.Tensor, w, n: int):
    """The rank's head-sharded tensor, cut from the global batch on the CPU."""
    nl = n // w.G if n >= w.G else 1
    h0 = w.first_head(n)
    return x[w.seq_offset:w.seq_offset + w.b, :, h0:h0 + nl, :]


def device_shards(x: torch.Tensor, w, dev="cuda"):
    return [s.to(dev) for s in shards_of(x, w)]


def fp64_kv_head(ql, kl, vl, dl, n_rep, scale, block=2048, device="cuda"):
    """O, dQ of query heads 0 .. n_rep-1 and dK, dV of kv head 0 (sequence 0)
    in plain fp64 torch on ``device``: per block of query rows, the dense
    masked score block, its softmax, and the gradients of sum(O * dO) from
    the definition (D = rowsum(dO * O), dS = P (dP - D)).  A second
    reference for full-size shapes the CPU oracle cannot finish in a test;
    a CPU test ties it to the oracle on small shapes."""
    S, d = ql.shape[1], ql.shape[3]
    K, V = kl[0, :, 0].to(device).double(), vl[0, :, 0].to(device).double()
    rO = torch.empty(S, n_rep, d, dtype=torch.float64, device=device)
    rdQ = torch.empty_like(rO)
    rdK = torch.zeros(S, d, dtype=torch.float64, device=device)
    rdV = torch.zeros_like(rdK)
    for h in range(n_rep):
        Q, dO = ql[0, :, h].to(device).double(), dl[0, :, h].to(device).double()
        for r0 in range(0, S, block):
            r1 = min(S, r0 + block)
            s = (Q[r0:r1] @ K[:r1].T) * scale
            keys = torch.arange(r1, device=device)[None, :]
            rows = torch.arange(r0, r1, device=device)[:, None]
            s.masked_fill_(keys > rows, float("-inf"))
            p = torch.softmax(s, dim=1)
            del s
            ob = p @ V[:r1]
            rO[r0:r1, h] = ob
            ds = p * (dO[r0:r1] @ V[:r1].T - (dO[r0:r1] * ob).sum(1, keepdim=True))
            rdV[:r1] += p.T @ dO[r0:r1]
            del p
            rdQ[r0:r1, h] = scale * (ds @ K[:r1])
            rdK[:r1] += scale * (ds.T @ Q[r0:r1])
            del ds
    return rO, rdQ, rdK, rdV
