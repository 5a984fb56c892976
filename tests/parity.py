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
