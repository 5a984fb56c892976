"""GPU parity of basp_a2a_pack / basp_a2a_unpack (the owner's side of the
head-parallel exchanges): bit-exact against the oracle at small sizes (both
element sizes, every vector width) with sentinel guard bands; at the full
workload sizes bit-exact against the oracle on the whole own shard; and,
through a simulated exchange of a whole group, consistent with basp_pack and
basp_unpack run on the same data."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_03151_amd as basp
from synth_inputs import WORKLOADS, random_shards
from parity import device_shards, log, workload_inputs

pytestmark = pytest.mark.gpu

SENT16 = 0x7F7B


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    return t.view(torch.int32).numpy()


def _guarded(shape, dtype, pad=64, dev="cuda"):
    n = int(np.prod(shape))
    itype = torch.int16 if dtype == torch.bfloat16 else torch.int32
    sent = SENT16 if dtype == torch.bfloat16 else 0x7FBADBAD
    buf = torch.full((pad + n + pad,), sent, dtype=itype, device=dev)
    return buf[pad:pad + n].view(dtype).view(shape), buf, sent


def _guards_intact(buf, sent):
    whole = buf.cpu().numpy()
    s = np.array(sent).astype(whole.dtype)
    return np.all(whole[:64] == s) and np.all(whole[-64:] == s)


CASES = [  # b, S, n, d, G
    (2, 512, 8, 64, 2),
    (1, 256, 32, 128, 4),
    (1, 96, 28, 128, 4),      # 7 heads per member
    (3, 40, 8, 5, 8),         # odd head dim: narrow accesses
    (1, 64, 4, 128, 1),       # G = 1: a copy
    (2, 130, 2, 64, 2),       # one head per member, odd token count per shard
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("b,S,n,d,G", CASES)
def test_a2a_small_bitexact(b, S, n, d, G, dtype):
    own_h = random_shards(b, S, n, d, G, seed=S * 7 + n + d + G, dtype=dtype)[0]  # [b, S/G, n, d]
    own = own_h.cuda()
    send, sbuf, sent = _guarded((G, b, S // G, n // G, d), dtype)
    basp.a2a_pack(own, G, out=send)
    torch.cuda.synchronize()
    ref = oracle.a2a_pack(own_h, G)
    assert np.array_equal(_bits(send), ref.view(_bits(send).dtype))
    assert _guards_intact(sbuf, sent)
    back, bbuf, sent = _guarded((b, S // G, n, d), dtype)
    basp.a2a_unpack(send, out=back)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(back), oracle.a2a_unpack(ref).view(_bits(back).dtype))
    assert _guards_intact(bbuf, sent)


def test_a2a_misaligned_pointers_take_narrow_path():
    b, S, n, d, G = 1, 64, 8, 64, 2
    own_h = random_shards(b, S, n, d, G, seed=3)[0]
    flat = torch.empty(own_h.numel() + 1, dtype=torch.bfloat16, device="cuda")
    flat[1:].copy_(own_h.reshape(-1).cuda())
    own = flat[1:].view(own_h.shape)
    send = basp.a2a_pack(own, G)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(send), oracle.a2a_pack(own_h, G))
    out_flat = torch.empty(own_h.numel() + 1, dtype=torch.bfloat16, device="cuda")
    basp.a2a_unpack(send, out=out_flat[1:].view(own_h.shape))
    torch.cuda.synchronize()
    assert np.array_equal(_bits(out_flat[1:].view(own_h.shape)), _bits(own_h))


def test_a2a_empty_is_a_noop():
    own = torch.empty((0, 4, 8, 8), dtype=torch.bfloat16, device="cuda")
    send = basp.a2a_pack(own, 2)
    back = basp.a2a_unpack(send)
    torch.cuda.synchronize()
    assert send.shape == (2, 0, 4, 4, 8) and back.shape == (0, 4, 8, 8)


@pytest.mark.parametrize("b,S,n,d,G", [(2, 96, 8, 64, 4), (1, 128, 32, 128, 4), (3, 30, 6, 4, 3)])
def test_group_exchange_consistent_with_pack_unpack(b, S, n, d, G):
    """Every member's send pack, exchanged, laid out along the sequence, is
    that member's basp_pack; the reverse way, basp_a2a_unpack of the returned
    blocks equals basp_unpack of every member's output into the shards."""
    shards = [s.cuda() for s in random_shards(b, S, n, d, G, seed=S + n + d + G)]
    Sg = S // G
    send = [basp.a2a_pack(shards[r], G) for r in range(G)]
    for l in range(G):
        got = torch.cat([send[j][l] for j in range(G)], dim=1)
        assert torch.equal(got.view(torch.int16), basp.pack(shards, l).view(torch.int16))
    outs = [basp.pack(shards, l) for l in range(G)]          # stand-in outputs
    ref = [torch.zeros_like(s) for s in shards]
    for l in range(G):
        basp.unpack(outs[l], ref, l)
    for r in range(G):
        recv = torch.stack([outs[j][:, r * Sg:(r + 1) * Sg] for j in range(G)]).contiguous()
        got = basp.a2a_unpack(recv)
        assert torch.equal(got.view(torch.int16), ref[r].view(torch.int16))
    torch.cuda.synchronize()


FULL = ["llama3_8b_s32k", "ulysses_g8_b2_s64k", "llama3_70b_s128k", "llama3_8b_g16_s64k"]


@pytest.mark.parametrize("name", FULL)
def test_a2a_full_size(name):
    """The full own shard of member `rank` (Q and K): send pack and its
    receive-side inverse, bit-exact against the oracle on the whole tensor."""
    w = WORKLOADS[name]
    log(f"[a2a full] {name}")
    q, k, _, _ = workload_inputs(name)
    for x, n in ((q, w.H), (k, w.H_kv)):
        own = device_shards(x, w)[w.rank]
        send = basp.a2a_pack(own, w.G)
        torch.cuda.synchronize()
        own_h = own.cpu()
        ref = oracle.a2a_pack(own_h, w.G)
        assert np.array_equal(_bits(send), ref)
        if n >= w.G:
            back = basp.a2a_unpack(send)
            torch.cuda.synchronize()
            assert torch.equal(back.view(torch.int16), own.view(torch.int16))
        else:
            # shared heads: the fp32 sum over a head's G/n copies is (G/n) x own
            own32 = own.float()
            back = basp.a2a_unpack(basp.a2a_pack(own32, w.G), n_heads=n)
            torch.cuda.synchronize()
            assert torch.equal(back, (w.G // n) * own32)
            del own32
        del own, send, back
    torch.cuda.empty_cache()


CAST_CASES = CASES + [(1, 64, 2, 64, 8), (2, 48, 4, 3, 8)]   # + shared heads (n < G)


def _cast_inputs(b, S, n, d, G, seed):
    """fp32 own shard: normals over many magnitudes, plus exact ties, values
    that round to infinity, infinities and signed zeros (no NaN, no
    subnormal: their handling is not part of the contract checked here)."""
    g = torch.Generator().manual_seed(seed)
    own = torch.randn(b, S // G, n, d, generator=g) * torch.exp2(
        torch.randint(-30, 30, (b, S // G, n, d), generator=g).float())
    flat = own.view(-1)
    special = torch.tensor([1.00390625, 1.01171875, -1.00390625, 3.3961e38, -3.4e38,
                            float("inf"), float("-inf"), 0.0, -0.0, 2.0 ** -126, 65504.0])
    k = min(special.numel(), flat.numel())
    flat[:k] = special[:k]
    return own


@pytest.mark.parametrize("b,S,n,d,G", CAST_CASES)
def test_a2a_pack_bf16_bitexact(b, S, n, d, G):
    own_h = _cast_inputs(b, S, n, d, G, seed=S + n + d + G)
    nl = basp.heads_per_member(n, G)
    send, sbuf, sent = _guarded((G, b, S // G, nl, d), torch.bfloat16)
    basp.a2a_pack_bf16(own_h.cuda(), G, out=send)
    torch.cuda.synchronize()
    ref = oracle.a2a_pack_bf16(own_h.numpy(), G)
    assert np.array_equal(_bits(send).view(np.uint16), ref)
    assert _guards_intact(sbuf, sent)


def test_a2a_pack_bf16_misaligned_takes_narrow_path():
    b, S, n, d, G = 1, 64, 8, 64, 4
    own_h = _cast_inputs(b, S, n, d, G, seed=77)
    flat = torch.zeros(own_h.numel() + 1, device="cuda")
    own = flat[1:].view(own_h.shape)            # 4-byte but not 16-byte aligned
    own.copy_(own_h.cuda())
    out_flat = torch.zeros(own_h.numel() + 1, dtype=torch.bfloat16, device="cuda")
    out = out_flat[1:].view(G, b, S // G, n // G, d)   # 2-byte aligned only
    lib = basp.lib()
    import ctypes
    rc = lib.basp_a2a_pack_bf16(ctypes.c_void_p(own.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                b, S, n, d, G, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    assert np.array_equal(_bits(out).view(np.uint16), oracle.a2a_pack_bf16(own_h.numpy(), G))


def test_a2a_pack_bf16_full_size_dout_shard():
    """The Llama-3-70B share's own dO shard [1, 16384, 64, 128] as fp32, sent as bf16."""
    w = WORKLOADS["llama3_70b_s128k"]
    g = torch.Generator().manual_seed(5)
    own_h = torch.randn(1, w.S // w.G, w.H, w.d, generator=g)
    send = basp.a2a_pack_bf16(own_h.cuda(), w.G)
    torch.cuda.synchronize()
    got = _bits(send).view(np.uint16)
    ref = oracle.a2a_pack_bf16(own_h.numpy(), w.G)
    assert np.array_equal(got, ref)
