"""GPU parity of attention run on the exchange's shard buffers in place
(basp_attn_fwd_sharded / basp_attn_bwd_sharded): no pack or unpack pass, Q,
K, V, O, dO read from the G sequence shards and O, dQ, dK, dV written into the
rank's head slices of the send buffers.

* bit for bit the same as the composed path (pack -> attention -> unpack) at
  shapes covering one and several row chunks of the backward, b > 1, group
  sizes 2 to 64 (shard row counts that are not powers of two included), head
  dims 64/80/96/128, and a kv head shared by several members, up to 8 (the
  partial dK, dV then go to one send block per member);
* other heads of the shard buffers untouched (sentinels);
* one shape against the oracle's composition directly;
* full size (the Llama-3-8B share, the batch-agnostic share with b = 2,
  G = 8, and the G = 16 share whose kv head two members share): every
  output bit for bit against the composed path."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_03151_amd as basp
from paper_2609_03151_amd.share import RankShare
from parity import check_close, device_shards, log, workload_inputs
from synth_inputs import WORKLOADS

pytestmark = pytest.mark.gpu


def _inputs(b, S, H, H_kv, d, G, seed):
    g = torch.Generator().manual_seed(seed)
    mk = lambda n: torch.randn(b, S, n, d, generator=g).to(torch.bfloat16)
    q, k, v, do = mk(H), mk(H_kv), mk(H_kv), mk(H)
    Sg = S // G
    sh = lambda x: [x[:, j * Sg:(j + 1) * Sg].contiguous().cuda() for j in range(G)]
    return q, k, v, do, sh(q), sh(k), sh(v), sh(do)


def _same(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def _compare_shares(ref: RankShare, got: RankShare, grads: bool = True):
    pairs = [("O", ref.o_shards, got.o_shards)]
    if grads:
        pairs += [("dQ", ref.dq_shards, got.dq_shards), ("dK", ref.dk_shards, got.dk_shards),
                  ("dV", ref.dv_shards, got.dv_shards)]
    for name, xs, ys in pairs:
        for j, (x, y) in enumerate(zip(xs, ys)):
            assert _same(x, y), f"{name} shard {j}"
    assert torch.equal(ref.lse, got.lse), "LSE"


CASES = [  # b, S, H, H_kv, d, G, rank
    (1, 1024, 8, 4, 128, 4, 1),     # one row chunk: dK/dV written by the key passes
    (2, 4096, 8, 4, 64, 2, 1),      # two row chunks: dK/dV written by the reduction
    (1, 2048, 12, 4, 96, 4, 3),     # d = 96, one kv head per member
    (1, 3072, 8, 8, 80, 4, 2),      # d = 80, 768 rows per shard
    (2, 1536, 6, 6, 128, 6, 5),     # G = 6
    (1, 4096, 16, 16, 64, 16, 9),   # G = 16
    (2, 8192, 32, 32, 128, 32, 17), # G = 32, b = 2, two row chunks
    (1, 16384, 64, 64, 64, 64, 63), # G = 64, the most the in-place path takes
]


@pytest.mark.parametrize("b,S,H,H_kv,d,G,rank", CASES)
def test_sharded_step_equals_composed_bitwise(b, S, H, H_kv, d, G, rank):
    log(f"[sharded] b={b} S={S} H={H} H_kv={H_kv} d={d} G={G} rank={rank}")
    _, _, _, _, qs, ks, vs, ds = _inputs(b, S, H, H_kv, d, G, seed=S + H + d + G)
    ref = RankShare(qs, ks, vs, ds, G=G, rank=rank)
    ref.step()
    got = RankShare(qs, ks, vs, ds, G=G, rank=rank)
    got.step_sharded()
    torch.cuda.synchronize()
    _compare_shares(ref, got)


SHARED = [  # b, S, H, H_kv, d, G, rank: a kv head shared by G / H_kv members
    (1, 2048, 16, 4, 128, 8, 3),    # one row chunk
    (2, 4096, 8, 2, 64, 4, 1),      # two row chunks, b = 2
    (1, 4096, 16, 8, 96, 16, 9),    # G = 16, 2 members per kv head
    (1, 16384, 64, 8, 128, 64, 37), # G = 64: Llama-3-70B heads, 8 members per kv head
]


@pytest.mark.parametrize("b,S,H,H_kv,d,G,rank", SHARED)
def test_shared_kv_head_in_place(b, S, H, H_kv, d, G, rank):
    """Forward in place as composed; the in-place backward writes the member's
    partial dK, dV into G send blocks, bit for bit the rows of the composed
    path's local dK, dV, and dQ into the shards as composed."""
    log(f"[sharded shared kv] b={b} S={S} H={H} H_kv={H_kv} d={d} G={G} rank={rank}")
    _, _, _, _, qs, ks, vs, ds = _inputs(b, S, H, H_kv, d, G, seed=5 + S + G)
    ref = RankShare(qs, ks, vs, ds, G=G, rank=rank)
    ref.step()
    got = RankShare(qs, ks, vs, ds, G=G, rank=rank)
    got.step_sharded()
    torch.cuda.synchronize()
    _compare_shares(ref, got, grads=False)
    for j, (x, y) in enumerate(zip(ref.dq_shards, got.dq_shards)):
        assert _same(x, y), f"dQ shard {j}"
    Sg = S // G
    for name, local, blocks in (("dK", ref.dk, got.dk_send), ("dV", ref.dv, got.dv_send)):
        for j in range(G):
            assert _same(blocks[j], local[:, j * Sg:(j + 1) * Sg].contiguous()), f"{name} block {j}"


def test_other_heads_untouched():
    b, S, H, H_kv, d, G, rank = 2, 1024, 8, 4, 64, 4, 2
    _, _, _, _, qs, ks, vs, ds = _inputs(b, S, H, H_kv, d, G, seed=9)
    sh = RankShare(qs, ks, vs, ds, G=G, rank=rank)
    for bufs in (sh.o_shards, sh.dq_shards, sh.dk_shards, sh.dv_shards):
        for t in bufs:
            t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).fill_(0x7F7B)
    sh.step_sharded()
    torch.cuda.synchronize()
    for bufs, n in ((sh.o_shards, H), (sh.dq_shards, H), (sh.dk_shards, H_kv), (sh.dv_shards, H_kv)):
        nl = n // G
        for t in bufs:
            bits = t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)
            rest = torch.cat([bits[:, :, :rank * nl], bits[:, :, (rank + 1) * nl:]], dim=2)
            assert bool((rest == 0x7F7B).all())
            assert not bool((bits[:, :, rank * nl:(rank + 1) * nl] == 0x7F7B).any())


def test_sharded_against_oracle():
    b, S, H, H_kv, d, G, rank = 1, 1024, 8, 4, 128, 4, 1
    q, k, v, do, qs, ks, vs, ds = _inputs(b, S, H, H_kv, d, G, seed=21)
    sh = RankShare(qs, ks, vs, ds, G=G, rank=rank)
    sh.step_sharded()
    torch.cuda.synchronize()
    c = 1.0 / math.sqrt(d)
    Sg = S // G
    cpu = lambda x: [x[:, j * Sg:(j + 1) * Sg].contiguous() for j in range(G)]
    bf = lambda a: torch.from_numpy(a).view(torch.bfloat16)
    ql, kl, vl, dl = (bf(oracle.pack(cpu(x), rank)) for x in (q, k, v, do))
    ro, rl = oracle.attn_fwd(ql, kl, vl, c)
    rdq, rdk, rdv = oracle.attn_bwd(ql, kl, vl, dl, ro, rl, c)
    for name, got_sh, ref_local, n in (("O", sh.o_shards, ro, H), ("dQ", sh.dq_shards, rdq, H),
                                       ("dK", sh.dk_shards, rdk, H_kv),
                                       ("dV", sh.dv_shards, rdv, H_kv)):
        nl = n // G
        ref_sh = [np.zeros((b, Sg, n, d), dtype=np.float32) for _ in range(G)]
        oracle.unpack(ref_local.astype(np.float32), ref_sh, rank)
        for j in range(G):
            got = got_sh[j].double().cpu().numpy()[:, :, rank * nl:(rank + 1) * nl]
            check_close(f"{name} shard {j}", got, ref_sh[j][:, :, rank * nl:(rank + 1) * nl])


@pytest.mark.parametrize("name", ["llama3_8b_s32k", "ulysses_g8_b2_s64k", "llama3_8b_g16_s64k"])
def test_sharded_full_size_equals_composed(name):
    w = WORKLOADS[name]
    log(f"[sharded full] {name}")
    q, k, v, do = workload_inputs(name)
    shards = [device_shards(x, w) for x in (q, k, v, do)]
    ref = RankShare(*shards, G=w.G, rank=w.rank, scale=w.scale)
    ref.step()
    got = RankShare(*shards, G=w.G, rank=w.rank, scale=w.scale)
    got.step_sharded()
    torch.cuda.synchronize()
    if w.H_kv >= w.G:
        _compare_shares(ref, got)
    else:
        _compare_shares(ref, got, grads=False)
        for j, (x, y) in enumerate(zip(ref.dq_shards, got.dq_shards)):
            assert _same(x, y), f"dQ shard {j}"
        Sg = w.S // w.G
        for name_, local, blocks in (("dK", ref.dk, got.dk_send), ("dV", ref.dv, got.dv_send)):
            for j in range(w.G):
                assert _same(blocks[j], local[:, j * Sg:(j + 1) * Sg].contiguous()), \
                    f"{name_} block {j}"
    del ref, got, shards
    torch.cuda.empty_cache()
