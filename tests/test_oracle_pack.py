"""Pins of the oracle's pack/unpack permutation (Sec. II-C, Sec. IV-C).

The head-parallel exchange hands a rank the full sequence for its heads, so
pack_r of the G sequence shards must equal the global tensor's head slice
[r*n/G, (r+1)*n/G) (computed here by torch slicing, not by the oracle's index
formula), and unpack must be its inverse on that slice only."""
import numpy as np
import pytest
import torch

import oracle
from synth_inputs import random_shards


def _np(t):
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.numpy()


CASES = [  # b, S, n, d, G
    (2, 512, 8, 64, 2),
    (1, 256, 32, 16, 4),
    (1, 96, 28, 8, 4),
    (3, 40, 8, 5, 8),     # odd d, one head per rank
    (1, 64, 4, 128, 1),   # G = 1: a plain copy
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("b,S,n,d,G", CASES)
def test_pack_is_head_slice_of_global(b, S, n, d, G, dtype):
    shards = random_shards(b, S, n, d, G, seed=S + n + d, dtype=dtype)
    glob = torch.cat(shards, dim=1)                     # [b, S, n, d]
    nl = n // G
    packed_all = []
    for r in range(G):
        out = oracle.pack(shards, r)
        ref = _np(glob[:, :, r * nl:(r + 1) * nl, :].contiguous())
        assert out.shape == ref.shape
        assert np.array_equal(out, ref)
        packed_all.append(out)
    # Concatenating every rank's share along heads rebuilds the global tensor.
    assert np.array_equal(np.concatenate(packed_all, axis=2), _np(glob))


@pytest.mark.parametrize("b,S,n,d,G", CASES)
def test_unpack_inverts_pack_and_touches_only_the_slice(b, S, n, d, G):
    shards = random_shards(b, S, n, d, G, seed=7 * S + d, dtype=torch.bfloat16)
    for r in range(G):
        local = oracle.pack(shards, r)
        # Sentinel-filled targets: only the rank's head slice may change.
        sentinel = np.int16(0x7F7B)
        tgt = [np.full(s.shape, sentinel, dtype=np.int16) for s in shards]
        oracle.unpack(local, tgt, r)
        nl = n // G
        for j in range(G):
            src = _np(shards[j])
            assert np.array_equal(tgt[j][:, :, r * nl:(r + 1) * nl], src[:, :, r * nl:(r + 1) * nl])
            rest = np.delete(tgt[j], np.s_[r * nl:(r + 1) * nl], axis=2)
            assert np.all(rest == sentinel)
        # pack(unpack(Y)) == Y
        assert np.array_equal(oracle.pack(tgt, r), local)
        # unpack(pack(X)) into X itself restores X byte for byte.
        own = [_np(s).copy() for s in shards]
        oracle.unpack(local, own, r)
        assert all(np.array_equal(a, _np(s)) for a, s in zip(own, shards))


def test_g1_is_plain_copy():
    (x,) = random_shards(2, 64, 4, 32, 1, seed=3)
    assert np.array_equal(oracle.pack([x], 0), _np(x))


def test_empty_and_errors():
    shards = random_shards(0, 8, 4, 8, 2, seed=1)
    assert oracle.pack(shards, 1).shape == (0, 8, 2, 8)
    shards = random_shards(1, 8, 4, 8, 2, seed=1)
    with pytest.raises(oracle.OracleError):
        oracle.pack(shards, 2)                     # rank >= G
    bad = random_shards(1, 8, 3, 8, 2, seed=1)     # 3 heads over G=2
    with pytest.raises(oracle.OracleError):
        oracle.pack(bad, 0)
