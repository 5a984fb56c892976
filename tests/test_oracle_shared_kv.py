"""Pins of the oracle's permutations when a group has more members than the
tensor has heads (GQA kv heads under Ulysses' head split, Sec. II-A/II-C):
with n < G and n | G, member r handles the single head r*n/G, shared by G/n
members, and the gradients of a shared head are the sum of the members'
partial gradients.

* pack is the global head slice (torch slicing, not the index formula);
* unpack_add adds a member's part into exactly its head, checked against a
  NumPy construction on integers (exact in fp32);
* the all-to-all send pack / receive unpack agree with pack / unpack_add
  through a simulated exchange of the whole group;
* the whole per-member path -- pack Q/K/V/dO, local attention forward and
  backward with one kv head, unpack dQ, unpack_add dK/dV -- reproduces torch
  fp64 autograd of the global causal GQA attention; a dropped replica, an
  overwrite in place of a sum or a wrong head fails it.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _ints(rng, shape):
    return rng.integers(-64, 64, size=shape).astype(np.float32)


@pytest.mark.parametrize("b,S,n,d,G", [(2, 8, 2, 3, 4), (1, 12, 1, 5, 3), (3, 16, 2, 2, 8),
                                       (1, 6, 3, 4, 6)])
def test_pack_shared_head_is_global_slice(b, S, n, d, G):
    X = torch.randn(b, S, n, d, generator=torch.Generator().manual_seed(S + G))
    Sg = S // G
    shards = [X[:, r * Sg:(r + 1) * Sg].contiguous() for r in range(G)]
    for r in range(G):
        h = r * n // G
        out = oracle.pack(shards, r)
        assert out.shape == (b, S, 1, d)
        assert np.array_equal(out, X[:, :, h:h + 1].numpy())
    # members sharing a head receive identical copies
    for r in range(1, G):
        if r * n // G == (r - 1) * n // G:
            assert np.array_equal(oracle.pack(shards, r), oracle.pack(shards, r - 1))


@pytest.mark.parametrize("b,S,n,d,G", [(2, 8, 2, 3, 4), (1, 12, 1, 5, 3), (3, 16, 2, 2, 8),
                                       (2, 12, 4, 3, 4)])
def test_unpack_add_sums_every_member_into_its_head(b, S, n, d, G):
    rng = np.random.default_rng(b + S + n + G)
    Sg, nl = S // G, oracle.heads_per_member(n, G)
    outs = [_ints(rng, (b, S, nl, d)) for _ in range(G)]
    base = [_ints(rng, (b, Sg, n, d)) for _ in range(G)]
    got = [x.copy() for x in base]
    for l in range(G):
        oracle.unpack_add(outs[l], got, l)
    for j in range(G):
        ref = base[j].copy()
        for l in range(G):
            for h in range(nl):
                ref[:, :, l * n // G + h] += outs[l][:, j * Sg:(j + 1) * Sg, h]
        assert np.array_equal(got[j], ref)


@pytest.mark.parametrize("b,S,n,d,G,elem", [(1, 8, 2, 3, 4, 2), (2, 12, 1, 5, 3, 4),
                                            (3, 16, 2, 2, 8, 2), (1, 6, 3, 4, 6, 4)])
def test_forward_exchange_matches_pack_shared(b, S, n, d, G, elem):
    rng = np.random.default_rng(S * n + G)
    dt = np.uint16 if elem == 2 else np.uint32
    X = rng.integers(0, np.iinfo(dt).max, size=(b, S, n, d), dtype=dt)
    Sg = S // G
    shards = [np.ascontiguousarray(X[:, r * Sg:(r + 1) * Sg]) for r in range(G)]
    send = [oracle.a2a_pack(shards[r], G) for r in range(G)]
    assert send[0].shape == (G, b, Sg, 1, d)
    for l in range(G):
        local = np.concatenate([send[j][l] for j in range(G)], axis=1)
        assert np.array_equal(local, oracle.pack(shards, l))


@pytest.mark.parametrize("b,S,n,d,G", [(1, 8, 2, 3, 4), (2, 12, 1, 5, 3), (3, 16, 2, 2, 8),
                                       (1, 6, 3, 4, 6)])
def test_reverse_exchange_matches_unpack_add(b, S, n, d, G):
    rng = np.random.default_rng(11 + S + n + G)
    Sg = S // G
    outs = [rng.standard_normal((b, S, 1, d)).astype(np.float32) for _ in range(G)]
    ref = [np.zeros((b, Sg, n, d), dtype=np.float32) for _ in range(G)]
    for l in range(G):                       # members in order: the same sum order
        oracle.unpack_add(outs[l], ref, l)
    for r in range(G):
        recv = np.stack([outs[j][:, r * Sg:(r + 1) * Sg] for j in range(G)])   # [G, b, Sg, 1, d]
        got = oracle.a2a_unpack(recv, n_heads=n)
        assert got.shape == (b, Sg, n, d)
        assert np.array_equal(got, ref[r])


def _global_grads(q, k, v, do, c):
    """torch fp64 autograd of causal GQA attention on the global tensors."""
    Q = torch.tensor(q, requires_grad=True)
    K = torch.tensor(k, requires_grad=True)
    V = torch.tensor(v, requires_grad=True)
    rep = q.shape[2] // k.shape[2]
    S = q.shape[1]
    Qh = Q.permute(0, 2, 1, 3)
    Kh = K.permute(0, 2, 1, 3).repeat_interleave(rep, dim=1)
    Vh = V.permute(0, 2, 1, 3).repeat_interleave(rep, dim=1)
    s = c * Qh @ Kh.transpose(-1, -2)
    s = s.masked_fill(~torch.tril(torch.ones(S, S, dtype=torch.bool)), float("-inf"))
    O = (torch.softmax(s, dim=-1) @ Vh).permute(0, 2, 1, 3)
    (O * torch.tensor(do)).sum().backward()
    return O.detach().numpy(), Q.grad.numpy(), K.grad.numpy(), V.grad.numpy()


@pytest.mark.parametrize("b,S,H,Hkv,d,G", [(2, 24, 8, 2, 8, 4), (1, 30, 6, 3, 4, 6),
                                           (1, 32, 4, 1, 8, 4), (1, 16, 16, 4, 4, 8)])
def test_member_path_reproduces_global_gradients(b, S, H, Hkv, d, G):
    rng = np.random.default_rng(S + H + G)
    f32 = lambda shape: rng.standard_normal(shape).astype(np.float32)
    q, do = f32((b, S, H, d)), f32((b, S, H, d))
    k, v = f32((b, S, Hkv, d)), f32((b, S, Hkv, d))
    c = 1.0 / math.sqrt(d)
    O, dQ, dK, dV = _global_grads(q.astype(np.float64), k.astype(np.float64),
                                  v.astype(np.float64), do.astype(np.float64), c)
    Sg, Hl = S // G, H // G
    sh = lambda x: [np.ascontiguousarray(x[:, r * Sg:(r + 1) * Sg]) for r in range(G)]
    qs, ks, vs, dos = sh(q), sh(k), sh(v), sh(do)
    dq_sh = [np.zeros((b, Sg, H, d), np.float32) for _ in range(G)]
    dk_sh = [np.zeros((b, Sg, Hkv, d), np.float32) for _ in range(G)]
    dv_sh = [np.zeros((b, Sg, Hkv, d), np.float32) for _ in range(G)]
    for l in range(G):
        ql, kl, vl, dol = (oracle.pack(x, l) for x in (qs, ks, vs, dos))
        assert kl.shape == (b, S, 1, d)
        o, lse = oracle.attn_fwd(ql, kl, vl, c)
        np.testing.assert_allclose(o, O[:, :, l * Hl:(l + 1) * Hl], rtol=0, atol=1e-12)
        dq, dk, dv = oracle.attn_bwd(ql, kl, vl, dol, o, lse, c)
        oracle.unpack(dq.astype(np.float32), dq_sh, l)
        oracle.unpack_add(dk.astype(np.float32), dk_sh, l)
        oracle.unpack_add(dv.astype(np.float32), dv_sh, l)
    cat = lambda xs: np.concatenate(xs, axis=1)
    tol = dict(rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(cat(dq_sh), dQ, **tol)
    np.testing.assert_allclose(cat(dk_sh), dK, **tol)
    np.testing.assert_allclose(cat(dv_sh), dV, **tol)


def test_rejects_unshareable_shapes():
    with pytest.raises(oracle.OracleError):
        oracle.pack([np.zeros((1, 2, 3, 2), np.float32)] * 4, 0)       # 3 heads, 4 members
    with pytest.raises(oracle.OracleError):
        oracle.a2a_pack(np.zeros((1, 2, 3, 2), np.float32), 4)
    # a shared head cannot be overwritten by one member: unpack refuses it
    with pytest.raises(oracle.OracleError):
        oracle.unpack(np.zeros((1, 8, 1, 2), np.float32),
                      [np.zeros((1, 2, 2, 2), np.float32) for _ in range(4)], 0)
    # summing replicas on receipt is fp32 only
    with pytest.raises(oracle.OracleError):
        oracle.a2a_unpack(np.zeros((4, 1, 2, 1, 2), np.uint16), n_heads=2)
