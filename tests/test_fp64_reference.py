"""Ties the tests' second fp64 reference (``parity.fp64_kv_head``, plain torch,
used on the GPU at full sizes the oracle cannot finish in a test) to the CPU
oracle: on small shapes, run on the CPU, its O, dQ, dK and dV of one kv head
must equal the oracle's to fp64 rounding."""
import math

import numpy as np
import pytest
import torch

import oracle
from parity import fp64_kv_head
from synth_inputs import ramped_local


@pytest.mark.parametrize("S,n_rep,d,block", [(300, 2, 16, 64), (257, 4, 32, 100), (64, 1, 8, 64)])
def test_fp64_kv_head_equals_oracle(S, n_rep, d, block):
    g = torch.Generator().manual_seed(S + d)
    mk = lambda h: torch.randn(1, S, h, d, generator=g).to(torch.bfloat16)
    q, k, v, do = mk(n_rep), mk(1), mk(1), mk(n_rep)
    scale = 1.0 / math.sqrt(d)
    rO, rdQ, rdK, rdV = fp64_kv_head(q, k, v, do, n_rep, scale, block=block, device="cpu")
    o, lse = oracle.attn_fwd(q, k, v, scale)
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, scale)
    for name, a, b in (("O", rO.numpy(), o[0]), ("dQ", rdQ.numpy(), dq[0]),
                       ("dK", rdK.numpy(), dk[0, :, 0]), ("dV", rdV.numpy(), dv[0, :, 0])):
        assert np.allclose(a, b, rtol=1e-9, atol=1e-11), name


def test_fp64_kv_head_equals_oracle_on_growing_logits():
    """Same, on inputs whose logits rise along the sequence."""
    S, n_rep, d = 400, 2, 32
    q, k, v, do = ramped_local(1, S, n_rep, 1, d, seed=5)
    scale = 1.0 / math.sqrt(d)
    rO, rdQ, rdK, rdV = fp64_kv_head(q, k, v, do, n_rep, scale, block=128, device="cpu")
    o, lse = oracle.attn_fwd(q, k, v, scale)
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, scale)
    for name, a, b in (("O", rO.numpy(), o[0]), ("dQ", rdQ.numpy(), dq[0]),
                       ("dK", rdK.numpy(), dk[0, :, 0]), ("dV", rdV.numpy(), dv[0, :, 0])):
        assert np.allclose(a, b, rtol=1e-9, atol=1e-11), name
