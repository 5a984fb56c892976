"""basp_attn_bwd_noalloc (the backward without a workspace argument, for
callers that cannot allocate) against basp_attn_bwd on the same inputs: two
calls in a row on one GPU, the second with a smaller input, each bit for bit
equal to the workspace entry point's dQ, dK, dV (the same kernels in the same
order), with NaN-filled outputs so that every element must be written."""
import math

import pytest
import torch

import paper_2609_03151_amd as basp
from parity import log

pytestmark = pytest.mark.gpu

CALLS = [  # b, S, Hl, Hkl, d: key pass in two row chunks, then one chunk, ragged
    (1, 4096, 4, 1, 128),
    (2, 1000, 2, 2, 64),
]


def _inputs(b, S, Hl, Hkl, d, seed):
    g = torch.Generator().manual_seed(seed)
    mk = lambda h: torch.randn(b, S, h, d, generator=g).to(torch.bfloat16).cuda()
    return mk(Hl), mk(Hkl), mk(Hkl), mk(Hl)


def test_noalloc_backward_equals_workspace_backward():
    for i, (b, S, Hl, Hkl, d) in enumerate(CALLS):
        need = basp.attn_bwd_workspace_bytes(b, S, Hl, Hkl, d, 1)
        log(f"[noalloc] call {i}: b={b} S={S} Hl={Hl} Hkl={Hkl} d={d}, workspace {need} bytes")
        assert need <= basp.NOALLOC_SCRATCH_BYTES
        q, k, v, do = _inputs(b, S, Hl, Hkl, d, seed=11 + i)
        scale = 1.0 / math.sqrt(d)
        o, lse = basp.attn_fwd(q, k, v, scale=scale)
        ref = basp.attn_bwd(q, k, v, o, lse, do, scale=scale)
        torch.cuda.synchronize()
        got = tuple(torch.full_like(x, float("nan")) for x in ref)
        basp.attn_bwd_noalloc(q, k, v, o, lse, do, *got, scale=scale)
        torch.cuda.synchronize()
        for name, a, r in zip(("dQ", "dK", "dV"), got, ref):
            assert torch.equal(a, r), f"call {i}: {name} differs from basp_attn_bwd"


def test_noalloc_backward_refuses_shapes_beyond_its_buffer():
    b, S, Hl, Hkl, d = 1, 32768, 8, 2, 128
    assert basp.attn_bwd_workspace_bytes(b, S, Hl, Hkl, d, 1) > basp.NOALLOC_SCRATCH_BYTES
    q = torch.empty(b, S, Hl, d, dtype=torch.bfloat16, device="cuda")
    kv = torch.empty(b, S, Hkl, d, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(b, Hl, S, dtype=torch.float32, device="cuda")
    g = torch.empty(b, S, Hl, d, dtype=torch.float32, device="cuda")
    gk = torch.empty(b, S, Hkl, d, dtype=torch.float32, device="cuda")
    with pytest.raises(basp.BaspError) as e:
        basp.attn_bwd_noalloc(q, kv, kv, q, lse, q, g, gk, gk)
    assert e.value.status == 6  # BASP_ERR_WORKSPACE
