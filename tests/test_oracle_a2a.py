"""Pins of the oracle's all-to-all send/receive layouts (Sec. II-C).

The send-side pack and the receive-side unpack are checked through the whole
exchange of a simulated group, against the receive-side pack and send-side
unpack that test_oracle_pack.py pins to the global tensor:

* forward direction: every member r packs its own shard for sending; the
  exchange delivers block l of member j's send buffer to member l; member l
  lays its received blocks out along the sequence, and must hold exactly
  oracle.pack(shards, l);
* reverse direction: every member l splits its head-sharded output along the
  sequence into blocks for the owners; the exchange delivers them; owner r
  merges its received blocks with a2a_unpack and must hold exactly what
  oracle.unpack of every member's output into the shard buffers gives.
"""
import numpy as np
import pytest

import oracle


def _bits(rng, shape, elem):
    dt = np.uint16 if elem == 2 else np.uint32
    return rng.integers(0, np.iinfo(dt).max, size=shape, dtype=dt)


@pytest.mark.parametrize("b,S,n,d,G,elem", [
    (1, 8, 4, 3, 2, 2), (2, 12, 6, 5, 3, 2), (3, 16, 8, 2, 4, 4), (1, 4, 2, 7, 1, 4),
    (2, 6, 6, 1, 6, 2),
])
def test_forward_exchange_matches_receive_pack(b, S, n, d, G, elem):
    rng = np.random.default_rng(b * 100 + S + n + G)
    X = _bits(rng, (b, S, n, d), elem)            # global tensor
    Sg = S // G
    shards = [np.ascontiguousarray(X[:, r * Sg:(r + 1) * Sg]) for r in range(G)]
    send = [oracle.a2a_pack(shards[r], G) for r in range(G)]   # [G, b, Sg, n/G, d]
    for l in range(G):
        recv = [send[j][l] for j in range(G)]                  # block l of member j
        local = np.concatenate(recv, axis=1)                  # along the sequence
        assert np.array_equal(local, oracle.pack(shards, l))


@pytest.mark.parametrize("b,S,n,d,G,elem", [
    (1, 8, 4, 3, 2, 2), (2, 12, 6, 5, 3, 4), (3, 16, 8, 2, 4, 2), (2, 6, 6, 1, 6, 4),
])
def test_reverse_exchange_matches_send_unpack(b, S, n, d, G, elem):
    rng = np.random.default_rng(7 + b + S + n + G)
    Sg, nl = S // G, n // G
    outs = [_bits(rng, (b, S, nl, d), elem) for _ in range(G)]   # member l's output
    dt = outs[0].dtype
    ref = [np.zeros((b, Sg, n, d), dtype=dt) for _ in range(G)]
    for l in range(G):
        oracle.unpack(outs[l], ref, l)
    for r in range(G):
        recv = np.stack([outs[j][:, r * Sg:(r + 1) * Sg] for j in range(G)])  # [G, b, Sg, nl, d]
        assert np.array_equal(oracle.a2a_unpack(recv), ref[r])


def test_round_trip_and_single_member():
    rng = np.random.default_rng(3)
    own = _bits(rng, (2, 5, 6, 4), 2)
    for G in (1, 2, 3, 6):
        send = oracle.a2a_pack(own, G)
        assert send.shape == (G, 2, 5, 6 // G, 4)
        assert np.array_equal(oracle.a2a_unpack(send), own)
    assert np.array_equal(oracle.a2a_pack(own, 1)[0], own)   # G = 1 is a copy


def test_rejects_bad_shapes():
    own = np.zeros((1, 4, 6, 2), dtype=np.uint16)
    with pytest.raises(oracle.OracleError):
        oracle.a2a_pack(own, 4)        # n % G
    with pytest.raises(oracle.OracleError):
        oracle.a2a_pack(np.zeros((1, 4, 6, 2), dtype=np.uint8), 2)   # element size


def test_a2a_pack_bf16_rounds_like_torch_and_indexes_like_a2a_pack():
    """The cast variant: its bits equal torch's fp32 -> bfloat16 conversion
    (round to nearest even, a library routine) of a2a_pack's fp32 blocks, on
    normals of many magnitudes, exact ties, values that round to infinity,
    infinities, signed zeros and subnormals; shared heads (n < G) too."""
    import torch
    g = torch.Generator().manual_seed(3)
    for b, S, n, d, G in ((2, 16, 8, 8, 4), (1, 24, 2, 5, 4), (1, 8, 3, 4, 1)):
        own = torch.randn(b, S // G, n, d, generator=g) * torch.exp2(
            torch.randint(-20, 20, (b, S // G, n, d), generator=g).float())
        flat = own.view(-1)
        special = torch.tensor([1.00390625, 1.01171875, -1.00390625, 3.3961e38, -3.4e38,
                                float("inf"), float("-inf"), 0.0, -0.0, 1e-40, -3e-39,
                                65504.0, 2.0 ** -126], dtype=torch.float32)
        flat[:special.numel()] = special
        got = oracle.a2a_pack_bf16(own.numpy(), G)
        blocks = torch.from_numpy(oracle.a2a_pack(own.numpy(), G))
        ref = blocks.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(got, ref)


def test_a2a_pack_bf16_nan_stays_nan():
    own = np.full((1, 2, 2, 2), np.nan, dtype=np.float32)
    own[0, 0, 0, 0] = -np.nan
    got = oracle.a2a_pack_bf16(own, 2)
    assert np.all((got & 0x7F80) == 0x7F80) and np.all((got & 0x007F) != 0)
