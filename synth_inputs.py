"""Seeded synthetic inputs for one rank's share of batch-aware Ulysses attention.

This module only draws random tensors and names workload shapes.  It holds none
of the method's arithmetic: no permutation, no attention.  Both the CPU oracle
(under ``oracle/``) and the HIP path take their inputs from here, so they see
identical bytes.

Recipe (the paper trains Llama/Qwen models on an unnamed dataset and prints no
tensors, so these stand in for the attention activations of those models):

* one ``torch.Generator('cpu')`` seeded with the workload's seed;
* draw, in this order, the *global* (unsharded) tensors
  Q ``[B_tot, S, H, d]``, K ``[B_tot, S, H_kv, d]``, V (as K), dO (as Q),
  each as float32 standard normal, rounded to bfloat16 (round to nearest even);
* a rank's sequence shards are the G contiguous token chunks of the sequence(s)
  it holds (shard j = tokens ``[j*S/G, (j+1)*S/G)``, Alg. 2 of the paper).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class Workload:
    """Shape of one rank's share (paper notation, Sec. IV; G is the group size K)."""

    name: str
    b: int          # sequences held by the rank's group (micro-batch per group)
    S: int          # full sequence length
    H: int          # query heads of the model
    H_kv: int       # key/value heads of the model (GQA)
    d: int          # head dimension
    G: int          # all-to-all group size (paper's K = N/B)
    rank: int       # local rank inside the group, in [0, G)
    seed: int
    b_total: int = 0      # sequences in the global batch drawn from the seed
    seq_offset: int = 0   # first global sequence this group holds
    note: str = field(default="", compare=False)

    @property
    def Hl(self) -> int:
        return self.H // self.G

    @property
    def Hkl(self) -> int:
        """Local kv heads: H_kv/G, or one head shared by G/H_kv members."""
        return self.H_kv // self.G if self.H_kv >= self.G else 1

    def first_head(self, n: int) -> int:
        """First head of an n-head tensor that this rank handles."""
        return self.rank * n // self.G

    @property
    def n_rep(self) -> int:
        return self.H // self.H_kv

    @property
    def scale(self) -> float:
        return 1.0 / float(self.d) ** 0.5

    @property
    def B_draw(self) -> int:
        return self.b_total if self.b_total else self.b

    def attn_fwd_flops(self) -> float:
        """Causal half of the two S x S x d contractions, per local q head."""
        return 2.0 * self.b * self.Hl * self.d * float(self.S) * float(self.S)

    def attn_bwd_flops(self) -> float:
        return 2.5 * self.attn_fwd_flops()


# The workloads the library is measured and parity-tested on.  Shapes follow
# Llama-3-8B (32 q / 8 kv heads), Qwen2.5-7B (28 / 4), Llama-3-70B (64 / 8),
# all with head dim 128, at long-context lengths.
WORKLOADS = {
    "tiny": Workload("tiny", b=2, S=512, H=8, H_kv=8, d=64, G=2, rank=0, seed=1),
    "llama3_8b_s32k": Workload("llama3_8b_s32k", b=1, S=32768, H=32, H_kv=8, d=128,
                               G=4, rank=1, seed=2),
    "qwen25_7b_s64k": Workload("qwen25_7b_s64k", b=1, S=65536, H=28, H_kv=4, d=128,
                               G=4, rank=3, seed=3),
    # Batch-agnostic (Ulysses over all 8 ranks, 2 sequences per rank) versus
    # batch-aware (groups of 4, one sequence per group) shares of the same
    # global batch of 2 sequences; rank 0 in both, group 0 holds sequence 0.
    "ulysses_g8_b2_s64k": Workload("ulysses_g8_b2_s64k", b=2, S=65536, H=32, H_kv=8,
                                   d=128, G=8, rank=0, seed=4, b_total=2),
    "basp_g4_b1_s64k": Workload("basp_g4_b1_s64k", b=1, S=65536, H=32, H_kv=8, d=128,
                                G=4, rank=0, seed=4, b_total=2, seq_offset=0),
    "llama3_70b_s128k": Workload("llama3_70b_s128k", b=1, S=131072, H=64, H_kv=8,
                                 d=128, G=8, rank=5, seed=5),
    # Three Table II models whose hidden size / heads give the other head
    # dims, in the paper's training setup (sequence 16K, batch 2 on 8 GPUs:
    # groups of 4, one sequence each).  The paper gives no kv-head count; 8
    # is used.
    "llama32_3b_s16k": Workload("llama32_3b_s16k", b=1, S=16384, H=32, H_kv=8, d=96,
                                G=4, rank=1, seed=6),
    "qwen25_3b_s16k": Workload("qwen25_3b_s16k", b=1, S=16384, H=32, H_kv=8, d=80,
                               G=4, rank=2, seed=7),
    "llama32_1b_s16k": Workload("llama32_1b_s16k", b=1, S=16384, H=32, H_kv=8, d=64,
                                G=4, rank=3, seed=9),
    # Fewer kv heads than group members: Llama-3-8B under one group of 16
    # (two 8-GPU nodes, micro-batch 1); each kv head is shared by 2 members.
    "llama3_8b_g16_s64k": Workload("llama3_8b_g16_s64k", b=1, S=65536, H=32, H_kv=8,
                                   d=128, G=16, rank=5, seed=8),
}


def _randn_bf16(gen: torch.Generator, shape) -> torch.Tensor:
    return torch.randn(*shape, generator=gen, dtype=torch.float32).to(torch.bfloat16)


def global_tensors(w: Workload, with_grad: bool = True):
    """Draw the global Q, K, V (and dO) of the batch the workload's share is cut from.

    Returns bf16 CPU tensors ``q [B,S,H,d]``, ``k``/``v`` ``[B,S,H_kv,d]``,
    ``do`` ``[B,S,H,d]`` (or None), with ``B = w.B_draw``.
    """
    gen = torch.Generator(device="cpu")
    gen.manual_seed(w.seed)
    B = w.B_draw
    q = _randn_bf16(gen, (B, w.S, w.H, w.d))
    k = _randn_bf16(gen, (B, w.S, w.H_kv, w.d))
    v = _randn_bf16(gen, (B, w.S, w.H_kv, w.d))
    do = _randn_bf16(gen, (B, w.S, w.H, w.d)) if with_grad else None
    return q, k, v, do


def shards_of(x: torch.Tensor, w: Workload):
    """The G sequence shards ``[b, S/G, n, d]`` (contiguous copies) the rank's group holds."""
    seqs = x[w.seq_offset:w.seq_offset + w.b]
    return [c.contiguous() for c in torch.chunk(seqs, w.G, dim=1)]


def random_shards(shape_b, S, n, d, G, seed, dtype=torch.bfloat16):
    """G independent random shards ``[b, S/G, n, d]`` for permutation-only tests.

    float32 dtype draws normals; bfloat16 rounds them; int dtypes draw raw bits.
    """
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    out = []
    for _ in range(G):
        shp = (shape_b, S // G, n, d)
        if dtype in (torch.bfloat16, torch.float32):
            out.append(_randn_bf16(gen, shp).to(dtype) if dtype == torch.bfloat16
                       else torch.randn(*shp, generator=gen, dtype=torch.float32))
        else:
            out.append(torch.randint(-2**15, 2**15, shp, generator=gen,
                                     dtype=torch.int32).to(dtype))
    return out


def small_workload(b=1, S=384, H=8, H_kv=2, d=128, G=2, rank=1, seed=11, name=None):
    """A seeded workload small enough for the full fp64 oracle in seconds."""
    return Workload(name or f"small_b{b}_s{S}_h{H}_{H_kv}_d{d}_g{G}_r{rank}",
                    b=b, S=S, H=H, H_kv=H_kv, d=d, G=G, rank=rank, seed=seed)


def ramped_local(b, S, Hl, Hkl, d, seed, lift=12.0, ramp=12.0, do_std=0.25):
    """Local (head-sharded) Q, K, V, dO whose attention logits grow along the sequence.

    Q ``[b,S,Hl,d]``, K and V ``[b,S,Hkl,d]``, dO as Q, drawn in that order
    from one seeded generator as float32 standard normals; every element of Q
    is then shifted by ``lift/sqrt(d)`` and every element of K at position j
    by ``ramp*(j/S)/sqrt(d)``, dO is multiplied by ``do_std``, and all four
    are rounded to bfloat16 (round to nearest even).  The shifts add
    ``lift*ramp*j/S`` to the dot product of any query with key j, so a row's
    largest logit keeps rising over its later keys (a recency-biased
    attention pattern).  Such attention concentrates on few keys, which makes
    dK and dV larger than under N(0,1) inputs; the smaller incoming gradient
    keeps them in the same range (|dK|, |dV| up to about 2-3)."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    q = torch.randn(b, S, Hl, d, generator=gen, dtype=torch.float32)
    k = torch.randn(b, S, Hkl, d, generator=gen, dtype=torch.float32)
    v = torch.randn(b, S, Hkl, d, generator=gen, dtype=torch.float32)
    do = torch.randn(b, S, Hl, d, generator=gen, dtype=torch.float32)
    q += lift / d ** 0.5
    do *= do_std
    pos = torch.arange(S, dtype=torch.float32) / S
    k += (ramp / d ** 0.5) * pos[None, :, None, None]
    bf = torch.bfloat16
    return q.to(bf), k.to(bf), v.to(bf), do.to(bf)
