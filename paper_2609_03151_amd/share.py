"""One rank's share of a batch-aware Ulysses attention layer, on one GPU.

A rank of a BASP group (G members, Sec. IV of the paper) receives G sequence
shards of Q, K, V, runs attention on its H/G query heads over the full
sequence, and returns the output to the G shard owners; the backward mirrors
this with dO in and dQ, dK, dV out (the transposed exchanges of Ulysses,
Sec. II-C).  `RankShare` holds every device buffer of that share, allocated
once, and chains the library calls:

  forward:  pack(Q), pack(K), pack(V) -> attn_fwd -> unpack(O)
  backward: pack(dO) -> attn_bwd -> unpack(dQ), unpack(dK), unpack(dV)

(the three packs and the three gradient unpacks each as one call,
pack_qkv / unpack_grads).

With fewer kv heads than members (H_kv < G, G divisible by H_kv) the rank
holds one kv head shared by G/H_kv members, and its dK, dV are that head's
partial gradients: they are added into the shards (unpack_add), so the dK/dV
shard buffers accumulate over repeated backward calls.

The exchange itself (RCCL all-to-all) is outside this share: the shard
buffers stand for the receive and send buffers of that exchange.

`forward_sharded` / `backward_sharded` run the same step with no pack or
unpack pass: attention reads the shard buffers in place and writes O, dQ,
dK, dV straight into the send buffers (bit for bit the same results); with a
shared kv head, dK and dV go to one send block per member (`dk_send`,
`dv_send`), each the member's partial gradient for that member's tokens.
"""
from __future__ import annotations

import torch

from . import (attn_bwd, attn_bwd_sharded, attn_bwd_sharded_workspace_bytes,
               attn_bwd_workspace_bytes, attn_fwd,
               attn_fwd_sharded, heads_per_member, pack, pack_qkv, unpack, unpack_add,
               unpack_grads)


class RankShare:
    def __init__(self, q_shards, k_shards, v_shards, do_shards, G: int, rank: int,
                 scale: float | None = None):
        self.G, self.rank = G, rank
        self.q_shards, self.k_shards, self.v_shards = q_shards, k_shards, v_shards
        self.do_shards = do_shards
        b, Sg, H, d = q_shards[0].shape
        H_kv = k_shards[0].shape[2]
        self.b, self.S, self.H, self.H_kv, self.d = b, Sg * G, H, H_kv, d
        self.Hl, self.Hkl = H // G, heads_per_member(H_kv, G)
        self.shared_kv = H_kv < G
        self.scale = d ** -0.5 if scale is None else scale
        dev = q_shards[0].device
        bf, f32 = torch.bfloat16, torch.float32
        S = self.S
        # head-sharded local tensors
        self.q = torch.empty((b, S, self.Hl, d), dtype=bf, device=dev)
        self.k = torch.empty((b, S, self.Hkl, d), dtype=bf, device=dev)
        self.v = torch.empty_like(self.k)
        self.o = torch.empty_like(self.q)
        self.lse = torch.empty((b, self.Hl, S), dtype=f32, device=dev)
        self.do = torch.empty_like(self.q)
        self.dq = torch.empty((b, S, self.Hl, d), dtype=f32, device=dev)
        self.dk = torch.empty((b, S, self.Hkl, d), dtype=f32, device=dev)
        self.dv = torch.empty_like(self.dk)
        # send buffers of the output exchanges (shard layout)
        self.o_shards = [torch.zeros((b, Sg, H, d), dtype=bf, device=dev) for _ in range(G)]
        self.dq_shards = [torch.zeros((b, Sg, H, d), dtype=f32, device=dev) for _ in range(G)]
        self.dk_shards = [torch.zeros((b, Sg, H_kv, d), dtype=f32, device=dev) for _ in range(G)]
        self.dv_shards = [torch.zeros((b, Sg, H_kv, d), dtype=f32, device=dev) for _ in range(G)]
        # in-place backward with a shared kv head: the partial dK, dV go to
        # one send block per member (the reverse exchange sums them)
        if self.shared_kv:
            self.dk_send = [torch.zeros((b, Sg, 1, d), dtype=f32, device=dev) for _ in range(G)]
            self.dv_send = [torch.zeros((b, Sg, 1, d), dtype=f32, device=dev) for _ in range(G)]
        ws = max(attn_bwd_workspace_bytes(b, S, H, H_kv, d, G),
                 attn_bwd_sharded_workspace_bytes(b, S, H, H_kv, d, G))
        self.workspace = torch.empty(max(ws, 16), dtype=torch.uint8, device=dev)

    # individual steps, so that callers can time them
    def pack_qkv(self):
        pack_qkv(self.q_shards, self.k_shards, self.v_shards, self.rank, q=self.q, k=self.k,
                 v=self.v)

    def attn_fwd(self):
        attn_fwd(self.q, self.k, self.v, G=self.G, scale=self.scale, out=self.o, lse=self.lse,
                 H_kv=self.H_kv)

    def unpack_o(self):
        unpack(self.o, self.o_shards, self.rank)

    def pack_do(self):
        pack(self.do_shards, self.rank, out=self.do)

    def attn_bwd(self):
        attn_bwd(self.q, self.k, self.v, self.o, self.lse, self.do, G=self.G, scale=self.scale,
                 dq=self.dq, dk=self.dk, dv=self.dv, workspace=self.workspace, H_kv=self.H_kv)

    def _unpack_kv_grad(self, local, shards):
        (unpack_add if self.shared_kv else unpack)(local, shards, self.rank)

    def unpack_grads(self):
        unpack_grads(self.dq, self.dk, self.dv, self.dq_shards, self.dk_shards, self.dv_shards,
                     self.rank)

    def forward(self):
        self.pack_qkv()
        self.attn_fwd()
        self.unpack_o()

    def backward(self):
        self.pack_do()
        self.attn_bwd()
        self.unpack_grads()

    def step(self):
        self.forward()
        self.backward()

    # attention on the shard buffers in place
    def forward_sharded(self):
        attn_fwd_sharded(self.q_shards, self.k_shards, self.v_shards, self.o_shards, self.rank,
                         scale=self.scale, lse=self.lse)

    def backward_sharded(self):
        dk, dv = ((self.dk_send, self.dv_send) if self.shared_kv
                  else (self.dk_shards, self.dv_shards))
        attn_bwd_sharded(self.q_shards, self.k_shards, self.v_shards, self.o_shards, self.lse,
                         self.do_shards, self.dq_shards, dk, dv, self.rank, scale=self.scale,
                         workspace=self.workspace)

    def step_sharded(self):
        self.forward_sharded()
        self.backward_sharded()

    # work counts (FlashAttention convention: causal half of S^2)
    def attn_fwd_flops(self) -> float:
        return 2.0 * self.b * self.Hl * self.d * float(self.S) ** 2

    def attn_bwd_flops(self) -> float:
        return 2.5 * self.attn_fwd_flops()

    def step_permutation_calls(self) -> list:
        """(name, call, bytes read + written) of the four pack/unpack calls a step makes."""
        nb = self.pack_unpack_bytes()
        return [("pack_qkv", self.pack_qkv, nb["pack_qkv"]),
                ("unpack_o", self.unpack_o, nb["unpack_o"]),
                ("pack_do", self.pack_do, nb["pack_do"]),
                ("unpack_grads", self.unpack_grads, nb["unpack_grads"])]

    def permutation_calls(self) -> list:
        """(name, call, bytes read + written) of each of the eight single-tensor permutations."""
        two = lambda t: 2 * t.numel() * t.element_size()
        # an added gradient is read on both sides and written once
        kv_grad = (lambda t: 3 * t.numel() * t.element_size()) if self.shared_kv else two
        return [
            ("pack_q", lambda: pack(self.q_shards, self.rank, out=self.q), two(self.q)),
            ("pack_k", lambda: pack(self.k_shards, self.rank, out=self.k), two(self.k)),
            ("pack_v", lambda: pack(self.v_shards, self.rank, out=self.v), two(self.v)),
            ("unpack_o", lambda: unpack(self.o, self.o_shards, self.rank), two(self.o)),
            ("pack_do", lambda: pack(self.do_shards, self.rank, out=self.do), two(self.do)),
            ("unpack_dq", lambda: unpack(self.dq, self.dq_shards, self.rank), two(self.dq)),
            ("unpack_dk", lambda: self._unpack_kv_grad(self.dk, self.dk_shards), kv_grad(self.dk)),
            ("unpack_dv", lambda: self._unpack_kv_grad(self.dv, self.dv_shards), kv_grad(self.dv)),
        ]

    def pack_unpack_bytes(self) -> dict:
        """Bytes read + written by each permutation (each moved element twice)."""
        bq = self.q.numel() * 2
        bkv = self.k.numel() * 2
        return {
            "pack_qkv": 2 * (bq + 2 * bkv),
            "unpack_o": 2 * bq,
            "pack_do": 2 * bq,
            "unpack_grads": (2 * self.dq.numel() + (3 if self.shared_kv else 2) * 2 * self.dk.numel()) * 4,
        }
