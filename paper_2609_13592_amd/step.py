"""A full decode step of a pre-norm Llama-style model over tiered weights and a
tiered KV pool.

This module only sequences C-ABI calls and owns the activation buffers
(device tensors from torch); every operator runs in the library's kernels:

  embed_gather -> per layer [rmsnorm -> gemv(qkv) -> rope_qkv -> kv_append ->
  paged_attn_decode -> gemv(o) -> residual_add -> rmsnorm -> gemv(gate_up) ->
  silu_mul -> gemv(down) -> residual_add] -> rmsnorm -> gemv(lm_head) -> argmax

where every "residual_add -> rmsnorm" pair is one add_rmsnorm launch (the
down projection's residual is added by the next layer's first norm, or by
the final norm) and "rope_qkv -> kv_append" is one rope_kv_append launch.
Where the qkv, o and down projections split K over workgroups, their
partial slices go straight to the RoPE + KV append and to the residual
norms (down's to the next layer's first norm, or the final one), which sum
them in the order the GEMV's own reduction kernel does: the same bits, one
launch fewer per projection.

Weights are [out, in] bf16 matrices placed page by page (each tensor on its
own, so modulo placement restarts per tensor); norm weights are small bf16
vectors kept in plain device memory.
"""
from __future__ import annotations

from dataclasses import dataclass

from . import binding as bd

EPS = 1e-5
THETA = 500000.0


@dataclass
class Dims:
    layers: int
    d: int
    hq: int
    hkv: int
    hd: int
    ffn: int
    vocab: int

    def shapes(self):
        """[(name, N, K)] of the matrices of one layer."""
        return [("qkv", (self.hq + 2 * self.hkv) * self.hd, self.d),
                ("o", self.d, self.hq * self.hd),
                ("gate_up", 2 * self.ffn, self.d),
                ("down", self.d, self.ffn)]


class DecodeModel:
    def __init__(self, ctx: int, dims: Dims, batch: int, max_blocks: int, pool: int,
                 matrices: dict, norms: dict, fold_slices: bool = True):
        """matrices: name -> placed tensor handle for 'embed', 'lm_head' and
        '<kind>.<layer>'; norms: name -> device bf16 tensor for 'norm1.<l>',
        'norm2.<l>', 'norm_f'.  fold_slices: hand the split-K slices of qkv,
        o and down to their consumers (False: every projection reduces its
        own)."""
        import torch
        self.ctx, self.dims, self.B, self.mb, self.pool = ctx, dims, batch, max_blocks, pool
        self.mat, self.norms = matrices, norms
        D = dims
        dev = "cuda"
        f32, b16 = torch.float32, torch.bfloat16
        B = batch
        self.x = torch.zeros((B, D.d), dtype=f32, device=dev)
        self.h = torch.zeros((B, D.d), dtype=b16, device=dev)
        qkv_n = (D.hq + 2 * D.hkv) * D.hd
        self.fold = fold_slices

        def slices(N, K):
            n = bd.boost_gemv_slices_floats(N, K, B, bd.MAX_GEMV_SLICES)
            return torch.zeros((n,), dtype=f32, device=dev)
        if fold_slices:
            self.qkv = slices(qkv_n, D.d)
            self.o_sl = slices(D.d, D.hq * D.hd)
            self.down_sl = slices(D.d, D.ffn)
        else:
            self.qkv = torch.zeros((B, qkv_n), dtype=f32, device=dev)
        self.q = torch.zeros((B, D.hq, D.hd), dtype=b16, device=dev)
        self.o = torch.zeros((B, D.hq, D.hd), dtype=b16, device=dev)
        self.tmp = torch.zeros((B, D.d), dtype=f32, device=dev)
        self.gu = torch.zeros((B, 2 * D.ffn), dtype=f32, device=dev)
        self.act = torch.zeros((B, D.ffn), dtype=b16, device=dev)
        self.logits = torch.zeros((B, D.vocab), dtype=f32, device=dev)
        self.ids = torch.zeros((B,), dtype=torch.int32, device=dev)

    def step(self, tokens, positions, lens, tables, stream=None, hooks=None):
        """One decode step for the batch.  tokens, positions (= lens - 1),
        lens: device int32 [B]; tables: device int32 [B, max_blocks] holding
        the blocks of every request including the new token's.  Returns the
        device ids and logits buffers (valid once the stream reaches them).

        hooks (optional) gets before_layer(l), after_layer(l) and before_head()
        calls as the launches are issued (e.g. to order staging copies)."""
        c, D, B, s = self.ctx, self.dims, self.B, stream
        F32, BF16 = bd.DTYPE_F32, bd.DTYPE_BF16
        bd.boost_embed_gather(c, self.mat["embed"], D.vocab, D.d, tokens, B, self.x, s)
        qkv_n = (D.hq + 2 * D.hkv) * D.hd
        # a residual add waits (in tmp, or as down's slices) until the next
        # norm takes it (one launch)
        pending = False
        S_down = 1
        for l in range(D.layers):
            if hooks is not None:
                hooks.before_layer(l)
            if pending and self.fold:
                bd.boost_add_rmsnorm_slices(c, self.x, self.down_sl, S_down, D.ffn,
                                            self.norms[f"norm1.{l}"], B, D.d, EPS, self.h, s)
            elif pending:
                bd.boost_add_rmsnorm(c, self.x, self.tmp, self.norms[f"norm1.{l}"], B, D.d,
                                     EPS, self.h, s)
            else:
                bd.boost_rmsnorm(c, self.x, self.norms[f"norm1.{l}"], B, D.d, EPS, self.h, s)
            if self.fold:
                S = bd.boost_decode_gemv_slices(c, self.mat[f"qkv.{l}"], qkv_n, D.d, self.h, B,
                                                self.qkv, bd.MAX_GEMV_SLICES, s)
                bd.boost_rope_kv_append_slices(c, self.pool, l, self.qkv, S, D.d, positions, B,
                                               D.hq, THETA, tables, self.mb, self.q, s)
            else:
                bd.boost_decode_gemv(c, self.mat[f"qkv.{l}"], qkv_n, D.d, self.h, B, self.qkv,
                                     F32, s)
                bd.boost_rope_kv_append(c, self.pool, l, self.qkv, positions, B, D.hq, THETA,
                                        tables, self.mb, self.q, s)
            bd.boost_paged_attn_decode(c, self.pool, l, self.q, B, D.hq, tables, self.mb,
                                       lens, 0.0, self.o, BF16, s)
            if self.fold:
                S = bd.boost_decode_gemv_slices(c, self.mat[f"o.{l}"], D.d, D.hq * D.hd, self.o,
                                                B, self.o_sl, bd.MAX_GEMV_SLICES, s)
                bd.boost_add_rmsnorm_slices(c, self.x, self.o_sl, S, D.hq * D.hd,
                                            self.norms[f"norm2.{l}"], B, D.d, EPS, self.h, s)
            else:
                bd.boost_decode_gemv(c, self.mat[f"o.{l}"], D.d, D.hq * D.hd, self.o, B,
                                     self.tmp, F32, s)
                bd.boost_add_rmsnorm(c, self.x, self.tmp, self.norms[f"norm2.{l}"], B, D.d, EPS,
                                     self.h, s)
            bd.boost_decode_gemv(c, self.mat[f"gate_up.{l}"], 2 * D.ffn, D.d, self.h, B,
                                 self.gu, F32, s)
            bd.boost_silu_mul(c, self.gu, B, D.ffn, self.act, s)
            if self.fold:
                S_down = bd.boost_decode_gemv_slices(c, self.mat[f"down.{l}"], D.d, D.ffn,
                                                     self.act, B, self.down_sl,
                                                     bd.MAX_GEMV_SLICES, s)
            else:
                bd.boost_decode_gemv(c, self.mat[f"down.{l}"], D.d, D.ffn, self.act, B,
                                     self.tmp, F32, s)
            if hooks is not None:
                hooks.after_layer(l)
            pending = True
        if hooks is not None:
            hooks.before_head()
        if pending and self.fold:
            bd.boost_add_rmsnorm_slices(c, self.x, self.down_sl, S_down, D.ffn,
                                        self.norms["norm_f"], B, D.d, EPS, self.h, s)
        elif pending:
            bd.boost_add_rmsnorm(c, self.x, self.tmp, self.norms["norm_f"], B, D.d, EPS,
                                 self.h, s)
        else:
            bd.boost_rmsnorm(c, self.x, self.norms["norm_f"], B, D.d, EPS, self.h, s)
        bd.boost_decode_gemv(c, self.mat["lm_head"], D.vocab, D.d, self.h, B, self.logits,
                             F32, s)
        bd.boost_argmax(c, self.logits, B, D.vocab, self.ids, s)
        return self.ids, self.logits

    def bytes_per_step(self, lens) -> int:
        """Algorithmic bytes of one step: every weight matrix once, every
        layer's K and V of every context token, plus the embedding rows."""
        D = self.dims
        w = sum(N * K * 2 for _, N, K in D.shapes()) * D.layers + D.vocab * D.d * 2
        kv = sum(int(L) for L in lens) * D.hkv * D.hd * 2 * 2 * D.layers
        return w + kv + self.B * D.d * 2
