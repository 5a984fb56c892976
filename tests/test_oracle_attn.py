"""Pins of the oracle's causal GQA attention (Sec. II-A) and its hand-derived
backward, against things other than the oracle itself:

* a NumPy brute force (dense masked score matrix) and torch's fp64
  scaled_dot_product_attention (a library routine);
* closed forms (K = 0 gives prefix means and LSE = ln(i+1); O_0 = V_0);
* invariants (convex combinations, shift invariance of K, sum_j dK_j = 0,
  sum_j dV_j = sum of dO over the group's heads, dQ_0 = 0);
* torch autograd in fp64 and central finite differences of sum(O * dO).
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _rand(shape, seed, scale=1.0):
    g = np.random.default_rng(seed)
    return g.standard_normal(shape) * scale


def _case(b=2, S=37, Hl=4, Hkl=2, d=16, seed=0):
    q = _rand((b, S, Hl, d), seed)
    k = _rand((b, S, Hkl, d), seed + 1)
    v = _rand((b, S, Hkl, d), seed + 2)
    do = _rand((b, S, Hl, d), seed + 3)
    return q, k, v, do


def _brute_numpy(q, k, v, c):
    """Dense masked softmax(c Q K^T) V per (beta, head), plain NumPy."""
    b, S, Hl, d = q.shape
    n_rep = Hl // k.shape[2]
    o = np.zeros_like(q)
    lse = np.zeros((b, Hl, S))
    mask = np.tril(np.ones((S, S), dtype=bool))
    for bt in range(b):
        for h in range(Hl):
            s = c * q[bt, :, h, :] @ k[bt, :, h // n_rep, :].T
            s = np.where(mask, s, -np.inf)
            mx = s.max(axis=1, keepdims=True)
            e = np.exp(s - mx)
            z = e.sum(axis=1, keepdims=True)
            o[bt, :, h, :] = (e / z) @ v[bt, :, h // n_rep, :]
            lse[bt, h, :] = (mx + np.log(z))[:, 0]
    return o, lse


def _torch_ref(q, k, v, c):
    """torch fp64 SDPA (library routine) with kv heads repeated per group."""
    Q = torch.tensor(q).permute(0, 2, 1, 3)
    n_rep = q.shape[2] // k.shape[2]
    K = torch.tensor(k).permute(0, 2, 1, 3).repeat_interleave(n_rep, dim=1)
    V = torch.tensor(v).permute(0, 2, 1, 3).repeat_interleave(n_rep, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(Q, K, V, is_causal=True, scale=c)
    return o.permute(0, 2, 1, 3).numpy()


@pytest.mark.parametrize("b,S,Hl,Hkl,d", [(2, 37, 4, 2, 16), (1, 64, 7, 1, 8), (1, 5, 2, 2, 3)])
def test_fwd_matches_brute_force_and_library(b, S, Hl, Hkl, d):
    q, k, v, _ = _case(b, S, Hl, Hkl, d, seed=S)
    c = 1.0 / math.sqrt(d)
    o, lse = oracle.attn_fwd(q, k, v, c)
    ob, lb = _brute_numpy(q, k, v, c)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lb, rtol=0, atol=1e-12)
    np.testing.assert_allclose(o, _torch_ref(q, k, v, c), rtol=0, atol=1e-12)


def test_first_row_is_v0_and_rows_are_convex():
    q, k, v, _ = _case(2, 50, 4, 2, 16, seed=5)
    o, lse = oracle.attn_fwd(q, k, v, 0.25)
    n_rep = 2
    for h in range(4):
        assert np.array_equal(o[:, 0, h, :], v[:, 0, h // n_rep, :])
        np.testing.assert_allclose(
            lse[:, h, 0], 0.25 * np.einsum("be,be->b", q[:, 0, h], k[:, 0, h // n_rep]),
            rtol=0, atol=1e-14)
        for i in range(50):
            lo = v[:, :i + 1, h // n_rep, :].min(axis=1)
            hi = v[:, :i + 1, h // n_rep, :].max(axis=1)
            assert np.all(o[:, i, h, :] >= lo - 1e-12) and np.all(o[:, i, h, :] <= hi + 1e-12)


def test_zero_keys_closed_form():
    """K = 0: every score is 0, so O_i is the prefix mean and LSE_i = ln(i+1)."""
    q, k, v, do = _case(1, 40, 4, 2, 8, seed=9)
    k[:] = 0.0
    o, lse = oracle.attn_fwd(q, k, v, 0.3)
    S = 40
    cnt = np.arange(1, S + 1)[None, :, None, None]
    pref = np.cumsum(v, axis=1) / cnt
    np.testing.assert_allclose(o, np.repeat(pref, 2, axis=2), rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, np.broadcast_to(np.log(cnt[0, :, 0, 0]), lse.shape),
                               rtol=0, atol=1e-13)
    # Backward closed forms: dQ = 0 (k = 0), dV_j = sum_h sum_{i>=j} dO_i / (i+1).
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, 0.3)
    assert np.abs(dq).max() < 1e-14
    w = do / cnt                                           # dO_i / (i+1)
    tail = np.flip(np.cumsum(np.flip(w, axis=1), axis=1), axis=1)   # sum_{i>=j}
    dv_ref = tail.reshape(1, S, 2, 2, 8).sum(axis=3)
    np.testing.assert_allclose(dv, dv_ref, rtol=0, atol=1e-12)


def test_shift_invariance_of_keys():
    """Adding one vector to every key shifts each score row by a constant."""
    q, k, v, _ = _case(1, 33, 4, 2, 16, seed=11)
    o1, _ = oracle.attn_fwd(q, k, v, 0.25)
    o2, _ = oracle.attn_fwd(q, k + _rand((1, 1, 2, 16), 99), v, 0.25)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-12)


def test_row_ranges_and_samples_agree_with_full():
    q, k, v, do = _case(2, 45, 4, 1, 8, seed=13)
    o, lse = oracle.attn_fwd(q, k, v, 0.35)
    o2, lse2 = oracle.attn_fwd(q, k, v, 0.35, 20, 31)
    assert np.array_equal(o2, o[:, 20:31]) and np.array_equal(lse2, lse[:, :, 20:31])
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, 0.35)
    ot, lt = oracle.attn_fwd(q, k, v, 0.35, 30, 45)
    dqt, dkt, dvt = oracle.attn_bwd(q, k, v, do, ot, lt, 0.35, r0=30)
    np.testing.assert_allclose(dqt, dq[:, 30:], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dkt, dk[:, 30:], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dvt, dv[:, 30:], rtol=0, atol=1e-13)
    beta = [0, 1, 1, 0]
    head = [3, 0, 2, 1]
    row = [0, 44, 17, 30]
    os_, ls, dqs = oracle.attn_rows(q, k, v, do, 0.35, beta, head, row)
    for n in range(4):
        np.testing.assert_allclose(os_[n], o[beta[n], row[n], head[n]], rtol=0, atol=1e-13)
        np.testing.assert_allclose(ls[n], lse[beta[n], head[n], row[n]], rtol=0, atol=1e-13)
        np.testing.assert_allclose(dqs[n], dq[beta[n], row[n], head[n]], rtol=0, atol=1e-13)


def _torch_grads(q, k, v, do, c):
    """Autograd of sum(O * dO) through a plain fp64 torch attention."""
    Q = torch.tensor(q, requires_grad=True)
    K = torch.tensor(k, requires_grad=True)
    V = torch.tensor(v, requires_grad=True)
    n_rep = q.shape[2] // k.shape[2]
    Qh = Q.permute(0, 2, 1, 3)
    Kh = K.permute(0, 2, 1, 3).repeat_interleave(n_rep, dim=1)
    Vh = V.permute(0, 2, 1, 3).repeat_interleave(n_rep, dim=1)
    S = q.shape[1]
    s = c * Qh @ Kh.transpose(-1, -2)
    s = s.masked_fill(~torch.tril(torch.ones(S, S, dtype=torch.bool)), float("-inf"))
    O = torch.softmax(s, dim=-1) @ Vh
    (O.permute(0, 2, 1, 3) * torch.tensor(do)).sum().backward()
    return Q.grad.numpy(), K.grad.numpy(), V.grad.numpy()


@pytest.mark.parametrize("b,S,Hl,Hkl,d", [(2, 29, 4, 2, 16), (1, 40, 7, 1, 8), (1, 17, 8, 8, 4)])
def test_bwd_matches_autograd(b, S, Hl, Hkl, d):
    q, k, v, do = _case(b, S, Hl, Hkl, d, seed=3 * S)
    c = 1.0 / math.sqrt(d)
    o, lse = oracle.attn_fwd(q, k, v, c)
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, c)
    tq, tk, tv = _torch_grads(q, k, v, do, c)
    np.testing.assert_allclose(dq, tq, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk, tk, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv, tv, rtol=0, atol=1e-12)


def test_bwd_central_finite_differences():
    """dL/dx for L = sum(O * dO) by central differences, every input entry."""
    b, S, Hl, Hkl, d = 1, 12, 4, 2, 8
    q, k, v, do = _case(b, S, Hl, Hkl, d, seed=21)
    c = 1.0 / math.sqrt(d)
    o, lse = oracle.attn_fwd(q, k, v, c)
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, c)

    def loss(q_, k_, v_):
        return float((oracle.attn_fwd(q_, k_, v_, c)[0] * do).sum())

    eps = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            args_p = {"q": q, "k": k, "v": v}
            args_m = dict(args_p)
            args_p[name], args_m[name] = xp, xm
            num[idx] = (loss(args_p["q"], args_p["k"], args_p["v"])
                        - loss(args_m["q"], args_m["k"], args_m["v"])) / (2 * eps)
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-7, err_msg=name)


def test_bwd_invariants():
    b, S, Hl, Hkl, d = 2, 64, 8, 2, 16
    q, k, v, do = _case(b, S, Hl, Hkl, d, seed=31)
    o, lse = oracle.attn_fwd(q, k, v, 0.25)
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, 0.25)
    assert np.abs(dq[:, 0]).max() < 1e-15                      # dS_00 = 0
    np.testing.assert_allclose(dk.sum(axis=1), 0.0, atol=1e-12)   # shift invariance
    dosum = do.reshape(b, S, Hkl, Hl // Hkl, d).sum(axis=(1, 3))
    np.testing.assert_allclose(dv.sum(axis=1), dosum, rtol=0, atol=1e-11)  # rows of P sum to 1


@pytest.mark.parametrize("b,S,Hl,Hkl,d", [(2, 29, 4, 2, 16), (1, 40, 7, 1, 8)])
def test_key_samples_match_autograd(b, S, Hl, Hkl, d):
    """The key-local dK_j, dV_j (summed over the kv head's query heads) equal
    torch fp64 autograd at every key, and the full backward's rows."""
    q, k, v, do = _case(b, S, Hl, Hkl, d, seed=7 * S)
    c = 1.0 / math.sqrt(d)
    o, lse = oracle.attn_fwd(q, k, v, c)
    _, tk, tv = _torch_grads(q, k, v, do, c)
    _, dk, dv = oracle.attn_bwd(q, k, v, do, o, lse, c)
    beta, kvh, key = zip(*[(bt, g, j) for bt in range(b) for g in range(Hkl) for j in range(S)])
    sk, sv = oracle.attn_keys(q, k, v, do, o, lse, c, beta, kvh, key)
    for n, (bt, g, j) in enumerate(zip(beta, kvh, key)):
        np.testing.assert_allclose(sk[n], tk[bt, j, g], rtol=0, atol=1e-12)
        np.testing.assert_allclose(sv[n], tv[bt, j, g], rtol=0, atol=1e-12)
        np.testing.assert_allclose(sk[n], dk[bt, j, g], rtol=0, atol=1e-13)
        np.testing.assert_allclose(sv[n], dv[bt, j, g], rtol=0, atol=1e-13)


def test_key_samples_closed_form_zero_keys():
    """K = 0: dV_j = sum_h sum_{i>=j} dO_i / (i+1) and dK_j = c sum_h sum_{i>=j}
    dS_ij q_i with P_ij = 1/(i+1), dS_ij = (dO_i.v_j - D_i)/(i+1)."""
    b, S, Hl, Hkl, d = 1, 33, 4, 2, 8
    q, k, v, do = _case(b, S, Hl, Hkl, d, seed=77)
    k[:] = 0.0
    c = 0.5
    o, lse = oracle.attn_fwd(q, k, v, c)
    n_rep = Hl // Hkl
    key = [0, 5, 32]
    for g in range(Hkl):
        sk, sv = oracle.attn_keys(q, k, v, do, o, lse, c, [0] * 3, [g] * 3, key)
        for n, j in enumerate(key):
            ev = np.zeros(d)
            ek = np.zeros(d)
            for h in range(g * n_rep, (g + 1) * n_rep):
                for i in range(j, S):
                    prefix = v[0, :i + 1, g].mean(axis=0)          # O_i: mean of v_0..v_i
                    Di = do[0, i, h] @ prefix
                    ev += do[0, i, h] / (i + 1)
                    ek += c * (do[0, i, h] @ v[0, j, g] - Di) / (i + 1) * q[0, i, h]
            np.testing.assert_allclose(sv[n], ev, rtol=0, atol=1e-12)
            np.testing.assert_allclose(sk[n], ek, rtol=0, atol=1e-12)


def test_key_samples_reject_bad_indices():
    q, k, v, do = _case(1, 8, 2, 1, 4, seed=1)
    o, lse = oracle.attn_fwd(q, k, v, 0.5)
    for bad in (([1], [0], [0]), ([0], [1], [0]), ([0], [0], [8]), ([0], [0], [-1])):
        with pytest.raises(oracle.OracleError):
            oracle.attn_keys(q, k, v, do, o, lse, 0.5, *bad)
