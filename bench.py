"""Benchmark one GPU's share of batch-aware Ulysses attention on MI355X.

A step is one pass of the whole share over one batch of synthetic inputs
already resident in HBM:
  pack(Q, K, V) -> causal GQA attention fwd -> unpack(O)
  pack(dO) -> attention bwd -> unpack(dQ, dK, dV)
The default workload is the largest single-GPU share: Llama-3-70B shapes at
S = 128K (b = 1, 64 query / 8 kv heads, d = 128, G = 8, rank 5).
The reported value is attention FLOPs (fwd + bwd, causal half of S^2,
bwd = 2.5 x fwd) divided by the median step time, in TFLOP/s; the pack and
unpack permutations are inside the step and also reported as GB/s, both as
timed in the step and with cold caches (each call alone after a 1 GiB
scratch write).  Achievable peaks measured on the same GPU (back-to-back bf16
MFMAs, a 1 GiB streaming copy) are reported as second denominators next to
the published ones.  The CPU oracle is timed on a bounded sample of the
same workload: fp64 attention on all host cores, and the step's
permutations on one core and on all cores.

Prints one JSON line.  With --gpus N > 1 it exits: this build runs one rank's
share on one GPU (the exchange between ranks is not part of it).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "causal attn fwd+bwd TFLOP/s + pack/unpack GB/s, one rank's share, 1 GPU"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# Sources of the attention-backward kernels (the dominant call): the counter
# summary under profiles/ stays valid while these hash to what it records.
BWD_KERNEL_SOURCES = ("paper_2609_03151_amd/csrc/basp_attn_bwd.hip",
                      "paper_2609_03151_amd/csrc/basp_device.hpp",
                      "paper_2609_03151_amd/csrc/basp_internal.hpp")


def kernel_source_sha256() -> str:
    """Hash of the attention-backward kernel sources (matches profiles/traffic_*.txt)."""
    import hashlib
    h = hashlib.sha256()
    for p in BWD_KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(workload: str):
    """(bytes, source) of HBM traffic per attention-backward launch, from the
    committed rocprofv3 FETCH_SIZE/WRITE_SIZE summary of this workload, or
    (None, reason) when there is none or the kernels changed since."""
    rel = os.path.join("profiles", f"traffic_{workload}.txt")
    path = os.path.join(ROOT, rel)
    if not os.path.exists(path):
        return None, f"no counter summary {rel}"
    kv = {}
    with open(path) as f:
        for ln in f:
            if "=" in ln and not ln.startswith("#"):
                a, b = ln.split("=", 1)
                kv[a.strip()] = b.strip()
    if kv.get("source_sha256") != kernel_source_sha256():
        return None, f"{rel} was taken on other kernel sources"
    return int(kv["traffic_bytes"]), f"recorded: {rel} (rocprofv3 FETCH_SIZE + WRITE_SIZE)"


def cpu_info() -> dict:
    """Host CPU model and the cores this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"model": model, "cores_available": len(os.sched_getaffinity(0))}


def cpu_pack_unpack_baseline(w, q, k, v, do) -> dict:
    """The step's eight permutations (pack Q, K, V, unpack O, pack dO, unpack
    fp32 dQ, dK, dV) of the whole workload by the oracle's index loops, on one
    core and on all cores, in GB/s under the GPU's byte convention (each moved
    element read once and written once; an added gradient read twice)."""
    import numpy as np
    import oracle
    import torch
    from synth_inputs import shards_of

    bits = lambda x: [s.view(torch.int16).numpy() for s in shards_of(x, w)]
    qs, ks, vs, ds = bits(q), bits(k), bits(v), bits(do)
    b, Sg, G, r = w.b, w.S // w.G, w.G, w.rank
    shared = w.H_kv < w.G

    def shard_bufs(n, dtype):
        return [np.zeros((b, Sg, n, w.d), dtype=dtype) + 0 for _ in range(G)]

    o_sh = shard_bufs(w.H, np.int16)
    dq_sh, dk_sh, dv_sh = (shard_bufs(w.H, np.float32), shard_bufs(w.H_kv, np.float32),
                           shard_bufs(w.H_kv, np.float32))
    dq_l = np.ones((b, w.S, w.Hl, w.d), dtype=np.float32)
    dk_l = np.ones((b, w.S, w.Hkl, w.d), dtype=np.float32)

    # Destinations allocated and touched once, outside the timed calls.
    ql, dl = (np.zeros((b, w.S, w.Hl, w.d), dtype=np.int16) + 0 for _ in range(2))
    kl, vl = (np.zeros((b, w.S, w.Hkl, w.d), dtype=np.int16) + 0 for _ in range(2))

    def run():
        t0 = time.perf_counter()
        oracle.pack(qs, r, out=ql)
        oracle.pack(ks, r, out=kl)
        oracle.pack(vs, r, out=vl)
        oracle.unpack(ql, o_sh, r)          # O stand-in: a local tensor of O's shape
        oracle.pack(ds, r, out=dl)
        oracle.unpack(dq_l, dq_sh, r)
        if shared:
            oracle.unpack_add(dk_l, dk_sh, r)
            oracle.unpack_add(dk_l, dv_sh, r)
        else:
            oracle.unpack(dk_l, dk_sh, r)
            oracle.unpack(dk_l, dv_sh, r)
        nbytes = (2 * (ql.nbytes + kl.nbytes + vl.nbytes) + 2 * ql.nbytes + 2 * ql.nbytes
                  + 2 * dq_l.nbytes + (3 if shared else 2) * 2 * dk_l.nbytes)
        return nbytes, time.perf_counter() - t0

    oracle.set_threads(0)
    run()                                  # first touch of every buffer, untimed
    nb, t_all = run()
    cores = oracle.threads()
    oracle.set_threads(1)
    _, t_one = run()
    oracle.set_threads(0)
    return {"value": round(nb / t_all / 1e9, 3), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "value_1core": round(nb / t_one / 1e9, 3),
            "sample": f"the step's 8 permutations of the whole workload ({nb / 2**20:.0f} MiB "
                      f"moved): {t_all:.2f} s on {cores} cores, {t_one:.2f} s on 1 core",
            "seconds": round(t_all + t_one, 3)}


def cpu_baseline(w, target_s: float, q, k, v, do):
    """Time the oracle (fp64, OpenMP) on a bounded prefix of the workload.

    Sample: sequence 0 of the share, every local head, the first S' tokens,
    full forward and backward of causal attention restricted to them; S' is
    chosen from a short calibration run so the sample takes ~target_s."""
    import oracle

    oracle.set_threads(0)

    def loc(x, n):
        h0, nl = w.first_head(n), (n // w.G if n >= w.G else 1)
        return x[w.seq_offset:w.seq_offset + 1, :, h0:h0 + nl]

    ql, kl, vl, dl = loc(q, w.H), loc(k, w.H_kv), loc(v, w.H_kv), loc(do, w.H)

    def run(Sp):
        sl = lambda x: x[:, :Sp].double().contiguous().numpy()
        qq, kk, vv, dd = sl(ql), sl(kl), sl(vl), sl(dl)
        t0 = time.perf_counter()
        o, lse = oracle.attn_fwd(qq, kk, vv, w.scale)
        oracle.attn_bwd(qq, kk, vv, dd, o, lse, w.scale)
        return time.perf_counter() - t0

    # Work grows about as S'^2, a little faster once rows leave the caches:
    # time two prefixes, fit the exponent, and size the sample to the target.
    c1, c2 = min(2048, w.S), min(4096, w.S)
    t1 = run(c1)
    t2 = run(c2) if c2 > c1 else t1
    e = math.log(max(t2, 1e-6) / max(t1, 1e-6)) / math.log(c2 / c1) if c2 > c1 else 2.0
    e = min(max(e, 2.0), 3.0)
    Sp = int(c2 * (target_s / max(t2, 1e-6)) ** (1.0 / e))
    Sp = max(c2, min(w.S, (Sp // 64) * 64))
    secs = run(Sp) if Sp != c2 else t2
    flops = 3.5 * 2.0 * 1 * w.Hl * w.d * float(Sp) ** 2
    return {"value": flops / secs / 1e12, "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle",
            "sample": f"fp64 oracle fwd+bwd, sequence 0, all {w.Hl} local heads, first {Sp} "
                      f"of {w.S} tokens ({secs:.1f} s)",
            "seconds": secs}


def sharded_step_rate(sh, steps: int, flops: float) -> dict:
    """The same step with attention run on the shard buffers in place (no
    pack/unpack pass), timed like the main loop.  Skipped where the in-place
    path does not take the shape (it raises before launching anything)."""
    import torch
    import paper_2609_03151_amd as basp

    try:
        sh.step_sharded()
    except basp.BaspError as e:
        return {"sharded_step": f"not taken: {e}"}
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        sh.step_sharded()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    log(f"[bench] in-place step {ms:.3f} ms")
    return {"sharded_ms_per_step": round(ms, 4),
            "sharded_tflops": round(flops / (ms * 1e-3) / 1e12, 2)}


def cold_permutation_rates(sh, reps: int = 51):
    """Each pack/unpack call of the step (the batched Q/K/V pack and gradient
    unpack, and the O unpack and dO pack), and each single-tensor permutation,
    timed alone with cold caches: a 1 GiB scratch write (larger than L2 and
    the 256 MB MALL) precedes every timed call; the median of `reps` runs.
    Also the send/receive-side permutations of the owner's shard
    (basp_a2a_pack / basp_a2a_unpack) at the same shapes."""
    import statistics
    import torch
    scratch = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def cold(fn):
        ts = []
        for _ in range(reps):
            scratch.fill_(1.0)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts)

    per = {name: (cold(fn), nbytes) for name, fn, nbytes in sh.step_permutation_calls()}
    each = {name: (cold(fn), nbytes) for name, fn, nbytes in sh.permutation_calls()}
    # The owner's side of the same exchanges (send pack of the own Q and K
    # shards, receive unpack of O and of fp32 dQ), outside the step.
    import paper_2609_03151_amd as basp
    G, r = sh.G, sh.rank
    own_q, own_k = sh.q_shards[r], sh.k_shards[r]
    send_q = basp.a2a_pack(own_q, G)
    send_k = basp.a2a_pack(own_k, G)
    own_dq = torch.empty(sh.dq_shards[r].shape, dtype=torch.float32, device="cuda")
    recv_dq = basp.a2a_pack(own_dq.zero_(), G)
    # an fp32 dO shard sent as bf16 (the cast fused into the send-side split)
    own_do32 = sh.do_shards[r].float()
    send_do16 = basp.a2a_pack_bf16(own_do32, G)
    two = lambda t: 2 * t.numel() * t.element_size()
    a2a = {
        "a2a_pack_q": (cold(lambda: basp.a2a_pack(own_q, G, out=send_q)), two(own_q)),
        "a2a_pack_k": (cold(lambda: basp.a2a_pack(own_k, G, out=send_k)), two(own_k)),
        "a2a_unpack_o": (cold(lambda: basp.a2a_unpack(send_q, out=sh.o_shards[r])), two(own_q)),
        "a2a_unpack_dq": (cold(lambda: basp.a2a_unpack(recv_dq, out=own_dq)), two(own_dq)),
        "a2a_pack_bf16_do": (cold(lambda: basp.a2a_pack_bf16(own_do32, G, out=send_do16)),
                             6 * own_do32.numel()),
    }
    total_ms = sum(t for t, _ in per.values())
    total_bytes = sum(b for _, b in per.values())
    del scratch, send_q, send_k, own_dq, recv_dq, own_do32, send_do16
    return {
        "pack_unpack_cold_gbps": round(total_bytes / (total_ms * 1e-3) / 1e9, 1),
        "pack_unpack_cold_gbps_by_call": {n: round(b / (t * 1e-3) / 1e9, 1) for n, (t, b) in per.items()},
        "pack_unpack_cold_gbps_by_tensor": {n: round(b / (t * 1e-3) / 1e9, 1)
                                            for n, (t, b) in each.items()},
        "a2a_cold_gbps_by_call": {n: round(b / (t * 1e-3) / 1e9, 1) for n, (t, b) in a2a.items()},
    }


def measured_peaks() -> dict:
    """Achievable peaks of this GPU: bf16 MFMA issue rate and a 1 GiB copy."""
    from paper_2609_03151_amd import peak
    return {"mfma_bf16_tflops": round(peak.mfma_bf16_tflops(), 1),
            "hbm_copy_gbps": round(peak.copy_gbps(1 << 30), 1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3_70b_s128k")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one rank's share on one GPU; --gpus {args.gpus} is not "
              "supported (the inter-GPU exchange is outside this build)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_03151_amd as basp
    from paper_2609_03151_amd.share import RankShare
    from synth_inputs import WORKLOADS, global_tensors, shards_of

    basp.lib()
    w = WORKLOADS[args.workload]
    log(f"[bench] workload {w.name}: b={w.b} S={w.S} H={w.H} H_kv={w.H_kv} d={w.d} "
        f"G={w.G} rank={w.rank}")
    q, k, v, do = global_tensors(w)
    dev = lambda x: [s.cuda() for s in shards_of(x, w)]
    sh = RankShare(dev(q), dev(k), dev(v), dev(do), G=w.G, rank=w.rank, scale=w.scale)
    log("[bench] inputs on device")

    for _ in range(args.warmup):
        sh.step()
    torch.cuda.synchronize()
    log("[bench] warmup done")

    phases = ["pack_qkv", "attn_fwd", "unpack_o", "pack_do", "attn_bwd", "unpack_grads"]
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(phases) + 1)]
          for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for s in range(args.steps):
        e = ev[s]
        e[0].record()
        for i, ph in enumerate(phases):
            getattr(sh, ph)()
            e[i + 1].record()
    stop.record()
    torch.cuda.synchronize()
    import statistics
    total_ms = start.elapsed_time(stop)
    ms_mean = total_ms / args.steps
    ms_step = statistics.median(ev[s][0].elapsed_time(ev[s][-1]) for s in range(args.steps))
    phase_ms = {ph: sum(ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(args.steps)) / args.steps
                for i, ph in enumerate(phases)}
    log(f"[bench] {args.steps} steps, median {ms_step:.3f} ms/step (mean {ms_mean:.3f}); "
        f"phases {phase_ms}")

    fwd_f, bwd_f = sh.attn_fwd_flops(), sh.attn_bwd_flops()
    value = (fwd_f + bwd_f) / (ms_step * 1e-3) / 1e12
    nbytes = sh.pack_unpack_bytes()
    perm_ms = sum(phase_ms[p] for p in nbytes)
    perm_gbps = sum(nbytes.values()) / (perm_ms * 1e-3) / 1e9
    fwd_tf = fwd_f / (phase_ms["attn_fwd"] * 1e-3) / 1e12
    bwd_tf = bwd_f / (phase_ms["attn_bwd"] * 1e-3) / 1e12
    dom = "attn_bwd" if phase_ms["attn_bwd"] >= phase_ms["attn_fwd"] else "attn_fwd"
    achieved = bwd_tf if dom == "attn_bwd" else fwd_tf
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_mean": round(ms_mean, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "b": w.b, "S": w.S, "H": w.H, "H_kv": w.H_kv, "d": w.d,
                   "G": w.G, "rank": w.rank, "causal": True, "inputs": "bf16 N(0,1), seeded"},
        "roofline": {
            "kernel": ("basp_attn_bwd (bwd_pre, bwd_kv, 2 x bwd_reduce, bwd_dq)"
                       if dom == "attn_bwd" else "basp_attn_fwd"),
            "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": None,
        },
        "attn_fwd_tflops": round(fwd_tf, 2),
        "attn_bwd_tflops": round(bwd_tf, 2),
        "attn_fwd_frac": round(fwd_tf / PEAK_BF16_TFLOPS, 4),
        "pack_unpack_gbps": round(perm_gbps, 1),
        "pack_unpack_frac": round(perm_gbps / PEAK_HBM_GBPS, 4),
        "pack_unpack_gbps_by_call": {p: round(nbytes[p] / (phase_ms[p] * 1e-3) / 1e9, 1)
                                     for p in nbytes},
        "phase_ms": {p: round(t, 4) for p, t in phase_ms.items()},
        "cpu_baseline": None,
    }
    if dom == "attn_bwd":
        traffic, src = recorded_traffic(w.name)
        out["roofline"]["traffic"] = traffic
        out["roofline"]["traffic_source"] = src
    out.update(sharded_step_rate(sh, args.steps, fwd_f + bwd_f))
    out.update(cold_permutation_rates(sh))
    del sh
    torch.cuda.empty_cache()
    pk = measured_peaks()
    out["peak_measured"] = pk
    out["roofline"]["frac_of_measured_peak"] = round(achieved / pk["mfma_bf16_tflops"], 4)
    out["attn_fwd_frac_of_measured_peak"] = round(fwd_tf / pk["mfma_bf16_tflops"], 4)
    out["pack_unpack_cold_frac_of_measured_copy"] = round(
        out["pack_unpack_cold_gbps"] / pk["hbm_copy_gbps"], 4)
    log(f"[bench] cold permutations {out['pack_unpack_cold_gbps']} GB/s; measured peaks {pk}")
    if not args.no_cpu_baseline:
        out["cpu"] = cpu_info()
        log("[bench] timing the CPU oracle samples")
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, q, k, v, do)
        out["cpu_baseline_pack_unpack"] = cpu_pack_unpack_baseline(w, q, k, v, do)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
