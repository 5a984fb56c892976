"""GPU parity of basp_attn_fwd / basp_attn_bwd against the fp64 oracle.

* small shapes (several tiles plus a ragged tail, GQA ratios 1, 4, 7): every
  output element, O and LSE, dQ, dK, dV; and sequence lengths that end inside
  and at the edges of the key pass's 32-row step halves;
* the whole share of the tiny workload (pack -> fwd -> unpack, pack dO ->
  bwd -> unpack) against the oracle's composition;
* exact cases: O_0 = V_0 bit for bit, K = 0 gives prefix means and
  LSE = ln(i+1), run-to-run bitwise determinism;
* full workload sizes, in the launch configuration the benchmark times:
  sampled rows of O, LSE, dQ, the last keys' dK and dV, and the invariants
  sum_j dK_j = 0 and sum_j dV_j = sum of dO over the group's heads; keys in
  every row chunk of the backward's key pass against the oracle; and, for
  one kv head, every row and key against a plain fp64 torch computation.
Bar: max |err| <= 2e-2 and mean |err| <= 2e-3 per tensor (LSE max 1e-3)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_03151_amd as basp
from paper_2609_03151_amd.share import RankShare
from parity import (LSE_MAX_ABS, check_close, device_shards, fp64_kv_head, local_heads, log,
                    workload_inputs)
from synth_inputs import WORKLOADS, Workload, global_tensors

pytestmark = pytest.mark.gpu


def _f64(t):
    return t.detach().cpu().double().numpy()


def _run(q, k, v, do, G=1, scale=None):
    o, lse = basp.attn_fwd(q, k, v, G=G, scale=scale)
    dq, dk, dv = basp.attn_bwd(q, k, v, o, lse, do, G=G, scale=scale)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


def _rand_local(b, S, Hl, Hkl, d, seed):
    g = torch.Generator().manual_seed(seed)
    mk = lambda h: torch.randn(b, S, h, d, generator=g).to(torch.bfloat16)
    return mk(Hl), mk(Hkl), mk(Hkl), mk(Hl)


SMALL = [  # b, S, Hl, Hkl, d
    (1, 128, 1, 1, 128),
    (2, 256, 4, 4, 64),
    (1, 384, 8, 2, 128),
    (1, 1000, 7, 1, 128),    # GQA 7, ragged tail (1000 = 7*128 + 104)
    (2, 200, 4, 1, 64),      # ragged, shorter than two row tiles
    (1, 77, 2, 2, 128),      # shorter than one tile
    (1, 1, 2, 1, 64),        # a single token
    (1, 2048, 4, 1, 128),    # 16 row tiles, 32 key tiles
    (1, 2500, 2, 1, 128),    # dK/dV rows split into 2 chunks, ragged tail
    (1, 4096, 4, 2, 64),     # 2 chunks, d = 64
    (1, 384, 8, 2, 96),      # d = 96 (Table II: 3072 / 32), GQA 4
    (1, 1000, 4, 1, 96),     # d = 96, ragged tail
    (2, 300, 3, 3, 80),      # d = 80 (Table II: 2560 / 32), computed at 96, ragged
    (1, 2500, 2, 1, 80),     # d = 80, 2 chunks, ragged tail
    (2, 2112, 4, 2, 128),    # 2 chunks, the second one 64-row step; GQA 2, b = 2
    (1, 4160, 7, 1, 64),     # 3 chunks (4160 = 2*2048 + 64), GQA 7, d = 64
]


# The key pass gives each of a workgroup's 8 waves 32 keys and one 32-row
# half of every 64-row step.  These lengths end the sequence inside the first
# half of a step, at its end, inside the second half and just past a step,
# and cut the 128-key tile's four key blocks at each such point.
HALVES = [(2, S, 2, 1, d) for S in (31, 32, 33, 63, 65, 95, 97, 129, 161, 191)
          for d in (64, 128)]


@pytest.mark.parametrize("b,S,Hl,Hkl,d", HALVES)
def test_key_pass_step_halves(b, S, Hl, Hkl, d):
    log(f"[attn halves] b={b} S={S} Hl={Hl} Hkl={Hkl} d={d}")
    q, k, v, do = _rand_local(b, S, Hl, Hkl, d, seed=7 * S + d)
    scale = 1.0 / math.sqrt(d)
    o, lse, dq, dk, dv = _run(q.cuda(), k.cuda(), v.cuda(), do.cuda())
    ro, rl = oracle.attn_fwd(q, k, v, scale)
    rdq, rdk, rdv = oracle.attn_bwd(q, k, v, do, ro, rl, scale)
    check_close("dQ", _f64(dq), rdq)
    check_close("dK", _f64(dk), rdk)
    check_close("dV", _f64(dv), rdv)


@pytest.mark.parametrize("b,S,Hl,Hkl,d", SMALL)
def test_attention_matches_oracle_small(b, S, Hl, Hkl, d):
    log(f"[attn small] b={b} S={S} Hl={Hl} Hkl={Hkl} d={d}")
    q, k, v, do = _rand_local(b, S, Hl, Hkl, d, seed=S + 13 * Hl + d)
    scale = 1.0 / math.sqrt(d)
    o, lse, dq, dk, dv = _run(q.cuda(), k.cuda(), v.cuda(), do.cuda())
    ro, rl = oracle.attn_fwd(q, k, v, scale)
    rdq, rdk, rdv = oracle.attn_bwd(q, k, v, do, ro, rl, scale)
    check_close("O", _f64(o), ro)
    check_close("LSE", _f64(lse), rl, max_abs=LSE_MAX_ABS, mean_abs=LSE_MAX_ABS)
    check_close("dQ", _f64(dq), rdq)
    check_close("dK", _f64(dk), rdk)
    check_close("dV", _f64(dv), rdv)


def test_tiny_workload_whole_share_matches_oracle():
    """The tiny workload end to end: pack, attention, unpack, and backward."""
    w = WORKLOADS["tiny"]
    q, k, v, do = global_tensors(w)
    sh = RankShare(device_shards(q, w), device_shards(k, w), device_shards(v, w),
                   device_shards(do, w), G=w.G, rank=w.rank, scale=w.scale)
    sh.step()
    torch.cuda.synchronize()
    # oracle composition: pack, fp64 attention, unpack
    qs, ks, vs, ds = (oracle.pack([s.cpu() for s in device_shards(x, w)], w.rank)
                      for x in (q, k, v, do))
    bf = lambda a: torch.from_numpy(a).view(torch.bfloat16)
    ql, kl, vl, dl = map(bf, (qs, ks, vs, ds))
    ro, rl = oracle.attn_fwd(ql, kl, vl, w.scale)
    rdq, rdk, rdv = oracle.attn_bwd(ql, kl, vl, dl, ro, rl, w.scale)
    Sg = w.S // w.G
    for name, got_sh, ref_local, n in (("O", sh.o_shards, ro, w.H), ("dQ", sh.dq_shards, rdq, w.H),
                                       ("dK", sh.dk_shards, rdk, w.H_kv),
                                       ("dV", sh.dv_shards, rdv, w.H_kv)):
        nl = n // w.G
        # oracle unpack (4-byte elements) of the fp64 result rounded to fp32
        ref_sh = [np.zeros((w.b, Sg, n, w.d), dtype=np.float32) for _ in range(w.G)]
        oracle.unpack(ref_local.astype(np.float32), ref_sh, w.rank)
        for j in range(w.G):
            got = _f64(got_sh[j])
            sl = np.s_[:, :, w.rank * nl:(w.rank + 1) * nl]
            check_close(f"{name} shard {j}", got[sl], ref_sh[j][sl])
            rest = np.delete(got, np.s_[w.rank * nl:(w.rank + 1) * nl], axis=2)
            assert np.all(rest == 0.0), f"{name} shard {j}: other heads written"
    check_close("LSE", _f64(sh.lse), rl, max_abs=LSE_MAX_ABS, mean_abs=LSE_MAX_ABS)


def test_first_row_is_exactly_v0():
    q, k, v, do = _rand_local(2, 300, 4, 2, 128, seed=3)
    o, lse, *_ = _run(q.cuda(), k.cuda(), v.cuda(), do.cuda())
    o = o.cpu()
    for h in range(4):
        assert torch.equal(o[:, 0, h].view(torch.int16), v[:, 0, h // 2].view(torch.int16))


def test_zero_keys_closed_form():
    b, S, Hl, Hkl, d = 1, 700, 4, 2, 128
    q, k, v, do = _rand_local(b, S, Hl, Hkl, d, seed=4)
    k.zero_()
    o, lse, dq, dk, dv = _run(q.cuda(), k.cuda(), v.cuda(), do.cuda())
    cnt = torch.arange(1, S + 1, dtype=torch.float64)
    pref = (v.double().cumsum(dim=1) / cnt[None, :, None, None]).repeat_interleave(2, dim=2)
    check_close("O (K=0)", _f64(o), pref.numpy())
    check_close("LSE (K=0)", _f64(lse), np.broadcast_to(np.log(cnt.numpy()), (b, Hl, S)),
                max_abs=1e-5, mean_abs=1e-5)
    assert float(dq.abs().max()) == 0.0  # every dS_ij multiplies k_j = 0


def test_bitwise_deterministic():
    q, k, v, do = (t.cuda() for t in _rand_local(1, 1536, 8, 2, 128, seed=6))
    a = _run(q, k, v, do)
    b_ = _run(q, k, v, do)
    for x, y, n in zip(a, b_, ("O", "LSE", "dQ", "dK", "dV")):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x, y.view(
            torch.int16) if y.dtype == torch.bfloat16 else y), n


FULL = ["llama3_8b_s32k", "qwen25_7b_s64k", "ulysses_g8_b2_s64k", "basp_g4_b1_s64k",
        "llama3_70b_s128k", "llama32_3b_s16k", "qwen25_3b_s16k", "llama32_1b_s16k",
        "llama3_8b_g16_s64k"]


def _sample_rows(S, rng, n=40):
    edge = [0, 1, 63, 64, 127, 128, 129, S // 2, S - 129, S - 128, S - 2, S - 1]
    rnd = rng.integers(0, S, size=n).tolist()
    return sorted({r for r in edge + rnd if 0 <= r < S})


@pytest.mark.parametrize("name", FULL)
def test_attention_full_size_sampled(name):
    w = WORKLOADS[name]
    log(f"[attn full] {name}: b={w.b} S={w.S} Hl={w.Hl} Hkl={w.Hkl}")
    q, k, v, do = workload_inputs(name)
    sh = RankShare(device_shards(q, w), device_shards(k, w), device_shards(v, w),
                   device_shards(do, w), G=w.G, rank=w.rank, scale=w.scale)
    sh.step()
    torch.cuda.synchronize()
    log("  GPU share done")
    ql, kl, vl, dl = (local_heads(x, w, n).contiguous()
                      for x, n in ((q, w.H), (k, w.H_kv), (v, w.H_kv), (do, w.H)))
    # the packed tensors on the GPU are exactly these head slices
    assert torch.equal(sh.q.cpu().view(torch.int16), ql.view(torch.int16))
    ql64, kl64, vl64, dl64 = (x.double().numpy() for x in (ql, kl, vl, dl))
    rng = np.random.default_rng(w.seed)
    rows = _sample_rows(w.S, rng)
    beta, head, row = [], [], []
    for bt in range(w.b):
        for h in range(w.Hl):
            for r in rows[(bt * w.Hl + h) % 3::3] + [0, w.S - 1]:
                beta.append(bt), head.append(h), row.append(r)
    ro, rl, rdq = oracle.attn_rows(ql64, kl64, vl64, dl64, w.scale, beta, head, row)
    log(f"  oracle rows: {len(row)}")
    bi, ri, hi = (torch.tensor(x, device="cuda") for x in (beta, row, head))
    pick = lambda t: t[bi, ri, hi].double().cpu().numpy()
    check_close("O rows", pick(sh.o), ro)
    check_close("LSE rows", sh.lse[bi, hi, ri].double().cpu().numpy(), rl,
                max_abs=LSE_MAX_ABS, mean_abs=LSE_MAX_ABS)
    check_close("dQ rows", pick(sh.dq), rdq)
    # last keys: dK, dV need every query row after them
    tail = 64
    r0 = w.S - tail
    to, tl = oracle.attn_fwd(ql64, kl64, vl64, w.scale, r0, w.S)
    tdq, tdk, tdv = oracle.attn_bwd(ql64, kl64, vl64, dl64, to, tl, w.scale, r0)
    log("  oracle tail done")
    check_close("dQ tail", _f64(sh.dq[:, r0:]), tdq)
    check_close("dK tail", _f64(sh.dk[:, r0:]), tdk)
    check_close("dV tail", _f64(sh.dv[:, r0:]), tdv)
    # invariants over every key
    dk_sum = sh.dk.double().sum(dim=1)
    scale_k = sh.dk.double().abs().sum(dim=1)
    assert float((dk_sum.abs() / scale_k.clamp_min(1e-30)).max()) < 1e-3
    dv_sum = sh.dv.double().sum(dim=1)
    do_sum = dl.double().reshape(w.b, w.S, w.Hkl, w.Hl // w.Hkl, w.d).sum(dim=(1, 3)).cuda()
    rel = ((dv_sum - do_sum).abs().max() / do_sum.abs().max()).item()
    log(f"  sum dV vs sum dO: rel {rel:.2e}")
    assert rel < 1e-3
    del sh
    torch.cuda.empty_cache()


KEY_WORKLOADS = ["llama3_8b_s32k", "llama32_3b_s16k", "qwen25_3b_s16k", "llama32_1b_s16k"]


def _keys_in_every_quarter(S, rng, per=6):
    """Keys spread over the four quarters of the sequence: every quarter's first
    and last key, keys at and beside 128-key tile edges, and random keys."""
    q4 = S // 4
    keys = {0, 1, 127, 128, S - 1}
    for c in range(4):
        lo = c * q4
        keys.update({lo, lo + 1, lo + q4 - 1, lo + 127, lo + 128})
        keys.update(rng.integers(lo, lo + q4, size=per).tolist())
    return sorted(k for k in keys if 0 <= k < S)


@pytest.mark.parametrize("name", KEY_WORKLOADS)
def test_attention_full_size_keys_every_chunk(name):
    """dK and dV at full size, in the benchmark's launch configuration, for keys
    in every quarter of the sequence -- the backward's key pass cuts the rows at
    a quarter of S (8192 rows at the Llama-3-8B share: 4 chunks), so key 0 sums
    the partials of every chunk and a key in the last quarter has one -- against
    the oracle's key-local gradients of kv head 0 (summed over its query heads;
    LSE and D from the oracle's own forward of every row)."""
    w = WORKLOADS[name]
    log(f"[attn full keys] {name}: b={w.b} S={w.S} Hl={w.Hl} Hkl={w.Hkl}")
    q, k, v, do = workload_inputs(name)
    sh = RankShare(device_shards(q, w), device_shards(k, w), device_shards(v, w),
                   device_shards(do, w), G=w.G, rank=w.rank, scale=w.scale)
    sh.step()
    torch.cuda.synchronize()
    n_rep = w.Hl // w.Hkl
    ql, kl, vl, dl = (local_heads(x, w, n)[:1, :, :nh].contiguous()
                      for x, n, nh in ((q, w.H, n_rep), (k, w.H_kv, 1), (v, w.H_kv, 1),
                                       (do, w.H, n_rep)))
    ql64, kl64, vl64, dl64 = (x.double().numpy() for x in (ql, kl, vl, dl))
    ro, rl = oracle.attn_fwd(ql64, kl64, vl64, w.scale)
    log("  oracle forward of every row done")
    keys = _keys_in_every_quarter(w.S, np.random.default_rng(w.seed + 100))
    rdk, rdv = oracle.attn_keys(ql64, kl64, vl64, dl64, ro, rl, w.scale,
                                [0] * len(keys), [0] * len(keys), keys)
    kt = torch.tensor(keys, device="cuda")
    check_close("dK keys", sh.dk[0, kt, 0].double().cpu().numpy(), rdk)
    check_close("dV keys", sh.dv[0, kt, 0].double().cpu().numpy(), rdv)
    check_close("O kv head 0", _f64(sh.o[:1, :, :n_rep]), ro)
    del sh
    torch.cuda.empty_cache()


def test_long_sequence_chunk_cap():
    """S = 131200 (just past 128K), one query and one kv head, d = 64: past
    S = 128K the key pass caps its row chunks at a sixteenth of S rounded up
    to the key tile (here 16 chunks of 8320 rows, the last 6400), so the
    workspace stays linear in S.  dK and dV of the keys in the last 6528 rows
    (the tail of chunk 14, summing the partials of two chunks, and all of
    chunk 15) and dQ, O, LSE of those rows against the oracle, and the
    invariants over every key."""
    b, S, Hl, Hkl, d = 1, 131200, 1, 1, 64
    log(f"[attn long] b={b} S={S} Hl={Hl} Hkl={Hkl} d={d}")
    q, k, v, do = _rand_local(b, S, Hl, Hkl, d, seed=2621)
    scale = 1.0 / math.sqrt(d)
    o, lse, dq, dk, dv = _run(q.cuda(), k.cuda(), v.cuda(), do.cuda())
    log("  GPU done")
    r0 = 15 * 8320 - 128
    q64, k64, v64, do64 = (x.double().numpy() for x in (q, k, v, do))
    to, tl = oracle.attn_fwd(q64, k64, v64, scale, r0, S)
    tdq, tdk, tdv = oracle.attn_bwd(q64, k64, v64, do64, to, tl, scale, r0)
    log("  oracle tail done")
    check_close("O tail", _f64(o[:, r0:]), to)
    check_close("LSE tail", _f64(lse[:, :, r0:]), tl, max_abs=LSE_MAX_ABS, mean_abs=LSE_MAX_ABS)
    check_close("dQ tail", _f64(dq[:, r0:]), tdq)
    check_close("dK tail", _f64(dk[:, r0:]), tdk)
    check_close("dV tail", _f64(dv[:, r0:]), tdv)
    dk_sum = dk.double().sum(dim=1)
    assert float((dk_sum.abs() / dk.double().abs().sum(dim=1).clamp_min(1e-30)).max()) < 1e-3
    do_sum = do.double().sum(dim=1).cuda()
    rel = ((dv.double().sum(dim=1) - do_sum).abs().max() / do_sum.abs().max()).item()
    assert rel < 1e-3


@pytest.mark.parametrize("name", ["llama3_8b_s32k", "qwen25_7b_s64k", "ulysses_g8_b2_s64k",
                                  "basp_g4_b1_s64k", "llama3_70b_s128k"])
def test_attention_full_size_kv_head_fp64(name):
    """Every row and key of one kv head at full size (sequence 0, kv head 0 and
    its query heads) against an independent fp64 computation in plain torch on
    the GPU (``fp64_kv_head``, tied to the oracle by a CPU test); the oracle's
    sampled rows and keys pin the same outputs."""
    w = WORKLOADS[name]
    log(f"[attn full fp64] {name}")
    q, k, v, do = workload_inputs(name)
    sh = RankShare(device_shards(q, w), device_shards(k, w), device_shards(v, w),
                   device_shards(do, w), G=w.G, rank=w.rank, scale=w.scale)
    sh.step()
    torch.cuda.synchronize()
    ql, kl, vl, dl = (local_heads(x, w, n).contiguous()
                      for x, n in ((q, w.H), (k, w.H_kv), (v, w.H_kv), (do, w.H)))
    n_rep = w.Hl // w.Hkl
    rO, rdQ, rdK, rdV = fp64_kv_head(ql, kl, vl, dl, n_rep, w.scale)
    torch.cuda.synchronize()
    log("  fp64 reference done")
    for nm, got, ref in (("O", sh.o[0, :, :n_rep], rO), ("dQ", sh.dq[0, :, :n_rep], rdQ),
                         ("dK", sh.dk[0, :, 0], rdK), ("dV", sh.dv[0, :, 0], rdV)):
        check_close(nm + " (fp64 torch)", got.double().cpu().numpy(), ref.cpu().numpy())
    del sh, rO, rdQ, rdK, rdV
    torch.cuda.empty_cache()


def test_batch_aware_and_batch_agnostic_shares_agree():
    """The Ulysses share (G=8, 2 sequences) and the BASP share (G=4, 1 sequence)
    of the same batch compute the same attention on what they share: sequence 0,
    query heads 0-3, kv head 0 -- bit for bit, forward and backward."""
    a, b_ = WORKLOADS["ulysses_g8_b2_s64k"], WORKLOADS["basp_g4_b1_s64k"]
    assert a.attn_fwd_flops() == b_.attn_fwd_flops()
    assert a.b * a.Hl * a.S == b_.b * b_.Hl * b_.S     # equal per-GPU tokens x heads
    q, k, v, do = workload_inputs(a.name)
    outs = []
    for w in (a, b_):
        log(f"[equivalence] {w.name}")
        sh = RankShare(device_shards(q, w), device_shards(k, w), device_shards(v, w),
                       device_shards(do, w), G=w.G, rank=w.rank, scale=w.scale)
        sh.step()
        torch.cuda.synchronize()
        outs.append((sh.o[0, :, 0:4].clone(), sh.lse[0, 0:4].clone(), sh.dq[0, :, 0:4].clone(),
                     sh.dk[0, :, 0:1].clone(), sh.dv[0, :, 0:1].clone()))
        del sh
        torch.cuda.empty_cache()
    for x, y, n in zip(outs[0], outs[1], ("O", "LSE", "dQ", "dK", "dV")):
        xb = x.view(torch.int16) if x.dtype == torch.bfloat16 else x
        yb = y.view(torch.int16) if y.dtype == torch.bfloat16 else y
        assert torch.equal(xb, yb), n
