"""GPU parity of basp_pack / basp_unpack: bit-exact against the oracle at
small sizes (every rank, both element sizes, every vector width), with
sentinel guard bands; at the full workload sizes bit-exact against the head
slice of the global tensor and against the oracle on sampled token windows."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_03151_amd as basp
from synth_inputs import WORKLOADS, random_shards
from parity import device_shards, log, workload_inputs

pytestmark = pytest.mark.gpu

SENT16 = 0x7F7B  # a bf16 NaN pattern no input contains


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    return t.view(torch.int32).numpy()


def _guards_intact(buf, sent) -> bool:
    whole = buf.cpu().numpy()
    s = np.array(sent).astype(whole.dtype)
    return bool(np.all(whole[:64] == s) and np.all(whole[-64:] == s))


def _bits_t(t: torch.Tensor) -> torch.Tensor:
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _guarded(shape, dtype, pad=64, dev="cuda"):
    """A tensor of `shape` inside a sentinel-filled buffer with `pad` guard
    elements on each side; returns (view, whole buffer)."""
    n = int(np.prod(shape))
    itype = torch.int16 if dtype == torch.bfloat16 else torch.int32
    sent = SENT16 if dtype == torch.bfloat16 else 0x7FBADBAD
    buf = torch.full((pad + n + pad,), sent, dtype=itype, device=dev)
    return buf[pad:pad + n].view(dtype).view(shape), buf, sent


CASES = [  # b, S, n, d, G
    (2, 512, 8, 64, 2),
    (1, 256, 32, 128, 4),
    (1, 96, 28, 128, 4),      # 7 heads per rank
    (3, 40, 8, 5, 8),         # odd head dim: narrow accesses
    (1, 64, 4, 128, 1),       # G = 1: a copy
    (1, 24, 6, 6, 3),
    (2, 130, 2, 64, 2),       # one head per rank, odd token count per shard
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("b,S,n,d,G", CASES)
def test_pack_unpack_small_bitexact(b, S, n, d, G, dtype):
    host = random_shards(b, S, n, d, G, seed=S * 31 + n + d, dtype=dtype)
    dev = [s.cuda() for s in host]
    nl = n // G
    for r in range(G):
        out, buf, sent = _guarded((b, S, nl, d), dtype)
        basp.pack(dev, r, out=out)
        torch.cuda.synchronize()
        ref = oracle.pack(host, r)
        assert np.array_equal(_bits(out), ref.view(_bits(out).dtype)), f"pack rank {r}"
        whole = buf.cpu().numpy()
        assert np.all(whole[:64] == np.array(sent).astype(whole.dtype))
        assert np.all(whole[-64:] == np.array(sent).astype(whole.dtype))
        # unpack into sentinel-filled shards: only the rank's slice changes
        tgt = []
        bufs = []
        for _ in range(G):
            t, bb, _ = _guarded((b, S // G, n, d), dtype)
            tgt.append(t)
            bufs.append(bb)
        basp.unpack(out, tgt, r)
        torch.cuda.synchronize()
        ref_t = [np.full((b, S // G, n, d), sent, dtype=_bits(out).dtype) for _ in range(G)]
        oracle.unpack(ref, ref_t, r)
        for j in range(G):
            assert np.array_equal(_bits(tgt[j]), ref_t[j]), f"unpack rank {r} shard {j}"
            whole = bufs[j].cpu().numpy()
            assert np.all(whole[:64] == np.array(sent).astype(whole.dtype))
            assert np.all(whole[-64:] == np.array(sent).astype(whole.dtype))


def test_pack_misaligned_pointers_take_narrow_path():
    """Shard pointers offset by one element still pack exactly."""
    b, S, n, d, G = 1, 64, 8, 64, 2
    host = random_shards(b, S, n, d, G, seed=5)
    flat = [torch.empty(s.numel() + 1, dtype=torch.bfloat16, device="cuda") for s in host]
    dev = []
    for f, s in zip(flat, host):
        f[1:].copy_(s.reshape(-1).cuda())
        dev.append(f[1:].view(s.shape))
    for r in range(G):
        out = basp.pack(dev, r)
        torch.cuda.synchronize()
        assert np.array_equal(_bits(out), oracle.pack(host, r))


def test_empty_is_a_noop():
    host = random_shards(0, 8, 4, 8, 2, seed=1)
    dev = [s.cuda() for s in host]
    out = basp.pack(dev, 1)
    basp.unpack(out, dev, 1)
    torch.cuda.synchronize()
    assert out.shape == (0, 8, 2, 8)


FULL = ["llama3_8b_s32k", "qwen25_7b_s64k", "ulysses_g8_b2_s64k", "basp_g4_b1_s64k",
        "llama3_70b_s128k", "llama32_3b_s16k", "qwen25_3b_s16k", "llama32_1b_s16k",
        "llama3_8b_g16_s64k"]


@pytest.mark.parametrize("name", FULL)
def test_pack_unpack_full_size(name):
    """Full-size shards: every rank's pack equals the head slice of the
    concatenated shards (bit for bit, compared on the GPU); sampled token
    windows equal the oracle; unpack of the packed result restores the shards.
    A head shared by several members (n < G) is checked through unpack_add:
    every member adding its packed copy back gives (G/n) times the shards."""
    w = WORKLOADS[name]
    log(f"[pack full] {name}")
    q, k, v, _ = workload_inputs(name)
    for x, n in ((q, w.H), (k, w.H_kv)):
        shards = device_shards(x, w)
        glob = torch.cat(shards, dim=1)
        nl = basp.heads_per_member(n, w.G)
        ranks = sorted({0, w.rank, w.G - 1})
        for r in ranks:
            out = basp.pack(shards, r)
            torch.cuda.synchronize()
            h0 = r * n // w.G
            assert torch.equal(out.view(torch.int16),
                               glob[:, :, h0:h0 + nl].contiguous().view(torch.int16)), r
        # sampled token windows of every shard against the oracle
        r = w.rank
        out = basp.pack(shards, r).cpu()
        Sg = w.S // w.G
        for t0 in (0, Sg // 2 + 3, Sg - 17):
            win = [s[:, t0:t0 + 16].cpu().contiguous() for s in shards]
            ref = oracle.pack(win, r)               # [b, 16*G, nl, d]
            got = torch.cat([out[:, j * Sg + t0:j * Sg + t0 + 16] for j in range(w.G)], dim=1)
            assert np.array_equal(_bits(got), ref)
        if n >= w.G:
            # unpack restores the shards exactly (its slice rewritten, rest untouched)
            before = [s.clone() for s in shards]
            basp.unpack(basp.pack(shards, r), shards, r)
            torch.cuda.synchronize()
            assert all(torch.equal(a.view(torch.int16), b_.view(torch.int16))
                       for a, b_ in zip(shards, before))
        else:
            f32 = [s.float() for s in shards]
            acc = [torch.zeros_like(s) for s in f32]
            for r in range(w.G):
                basp.unpack_add(basp.pack(f32, r), acc, r)
            torch.cuda.synchronize()
            assert all(torch.equal(a, (w.G // n) * s) for a, s in zip(acc, f32))
            del f32, acc
        del shards, glob, out
    torch.cuda.empty_cache()


BATCH = [  # b, S, H, H_kv, d, G, rank, dtype
    (1, 2048, 32, 8, 128, 4, 1, torch.bfloat16),
    (2, 600, 12, 4, 64, 4, 3, torch.bfloat16),     # 150 tokens per shard
    (1, 384, 8, 2, 80, 8, 5, torch.bfloat16),      # shared kv head (2 < 8)
    (3, 96, 6, 3, 5, 3, 2, torch.bfloat16),        # odd head dim: 2-byte rows, separate launches
    (1, 512, 32, 32, 128, 32, 7, torch.bfloat16),  # G > 16: separate launches
    (1, 1024, 16, 8, 128, 8, 6, torch.float32),
]


@pytest.mark.parametrize("b,S,H,H_kv,d,G,rank,dtype", BATCH)
def test_pack_qkv_equals_three_packs(b, S, H, H_kv, d, G, rank, dtype):
    """basp_pack_qkv (one launch where it can) against three basp_pack calls
    and the oracle, bit for bit, with sentinel guard bands."""
    qs_h = random_shards(b, S, H, d, G, seed=S + H, dtype=dtype)
    ks_h = random_shards(b, S, H_kv, d, G, seed=S + H_kv + 1, dtype=dtype)
    vs_h = random_shards(b, S, H_kv, d, G, seed=S + H_kv + 2, dtype=dtype)
    qs, ks, vs = ([x.cuda() for x in xs] for xs in (qs_h, ks_h, vs_h))
    nq, nk = basp.heads_per_member(H, G), basp.heads_per_member(H_kv, G)
    q, qbuf, sent = _guarded((b, S, nq, d), dtype)
    k, kbuf, _ = _guarded((b, S, nk, d), dtype)
    v, vbuf, _ = _guarded((b, S, nk, d), dtype)
    basp.pack_qkv(qs, ks, vs, rank, q=q, k=k, v=v)
    torch.cuda.synchronize()
    for got, sh_h, sh, buf in ((q, qs_h, qs, qbuf), (k, ks_h, ks, kbuf), (v, vs_h, vs, vbuf)):
        assert np.array_equal(_bits(got), oracle.pack(sh_h, rank).view(_bits(got).dtype))
        assert torch.equal(_bits_t(got), _bits_t(basp.pack(sh, rank)))
        assert _guards_intact(buf, sent)


@pytest.mark.parametrize("b,S,H,H_kv,d,G,rank,dtype", BATCH)
def test_unpack_grads_equals_three_unpacks(b, S, H, H_kv, d, G, rank, dtype):
    """basp_unpack_grads against basp_unpack of dQ and basp_unpack (or
    basp_unpack_add, for a shared kv head) of dK and dV, bit for bit."""
    g = torch.Generator().manual_seed(b + S + G)
    nq, nk = basp.heads_per_member(H, G), basp.heads_per_member(H_kv, G)
    dq, dk, dv = (torch.randn(b, S, n, d, generator=g).cuda() for n in (nq, nk, nk))
    Sg = S // G
    base = [[torch.randn(b, Sg, n, d, generator=g).cuda() for _ in range(G)] for n in (H, H_kv, H_kv)]
    got = [[t.clone() for t in xs] for xs in base]
    ref = [[t.clone() for t in xs] for xs in base]
    basp.unpack_grads(dq, dk, dv, *got, rank)
    basp.unpack(dq, ref[0], rank)
    kv_op = basp.unpack_add if H_kv < G else basp.unpack
    kv_op(dk, ref[1], rank)
    kv_op(dv, ref[2], rank)
    torch.cuda.synchronize()
    for xs, ys in zip(got, ref):
        for x, y in zip(xs, ys):
            assert torch.equal(x.view(torch.int32), y.view(torch.int32))
