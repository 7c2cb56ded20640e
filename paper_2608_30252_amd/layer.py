"""One draft decoder layer around the compact-memory attention, on the GPU.

A decode step of the draft runs, per layer, for R rows: the raw token at
position p and, when p's pass materialises memory slots, those slot tokens
(Sec. 3.2: a slot is an extra position of the pass that runs through the same
transformer blocks; its normalised hidden state entering the layer feeds the
mirrored projections).  Per layer:
    xn, q, k, v = rmsnorm + Q/K/V projection + RoPE        (mad_rmsnorm_qkv_rope)
    slots only:  memory update of the new slots from xn     (mad_memory_update)
    o    = attention over the compact memory                (mad_draft_decode_attn,
                                                              or mad_draft_step_attn for R > 1)
    h    = x + o W_o^T                                       (mad_linear_residual)
    a    = silu(hn W_gate^T) * (hn W_up^T)                   (mad_rmsnorm_swiglu)
    y    = h + a W_down^T                                    (mad_linear_residual)
Every step runs in the library's kernels; this module only orders the calls
and owns the activation buffers.  Weights are random-init (no checkpoint).
"""
from dataclasses import dataclass

import torch

from . import (KV, draft_decode_attn, draft_step_attn, linear_residual, memory_update, rmsnorm_qkv_rope,
               rmsnorm_swiglu, synth)

MAX_ROWS = 8


@dataclass
class LayerWeights:
    gamma1: torch.Tensor      # [D]
    w_qkv: torch.Tensor       # [(Hq + 2 Hkv) d, D]
    w_kv_g: torch.Tensor      # [2 Hkv d, D]  mirrored K/V projections of slot tokens
    w_o: torch.Tensor         # [D, Hq d]
    gamma2: torch.Tensor      # [D]
    w_gate_up: torch.Tensor   # [2 F, D]
    w_down: torch.Tensor      # [D, F]

    @staticmethod
    def random(D, Hq, Hkv, d, F, seed, device="cuda", std=0.02):
        """N(0, std^2) projections, RMSNorm weights 1 + N(0, 0.1^2), bf16."""
        mk = lambda shape, i, s=std: synth.normal(shape, 1000 * seed + i, std=s).to(device)
        return LayerWeights(gamma1=(1 + synth.normal((D,), 1000 * seed + 1, std=0.1, dtype=torch.float32)).to(
                                torch.bfloat16).to(device),
                            w_qkv=mk(((Hq + 2 * Hkv) * d, D), 2), w_kv_g=mk((2 * Hkv * d, D), 3),
                            w_o=mk((D, Hq * d), 4),
                            gamma2=(1 + synth.normal((D,), 1000 * seed + 5, std=0.1, dtype=torch.float32)).to(
                                torch.bfloat16).to(device),
                            w_gate_up=mk((2 * F, D), 6), w_down=mk((D, F), 7))

    def weight_bytes(self, with_slot_projection=False):
        ts = [self.w_qkv, self.w_o, self.w_gate_up, self.w_down, self.gamma1, self.gamma2]
        if with_slot_projection:
            ts.append(self.w_kv_g)
        return sum(t.numel() * t.element_size() for t in ts)


class DraftLayer:
    """Activation buffers of one layer for up to MAX_ROWS rows, and its step."""

    def __init__(self, weights: LayerWeights, D, Hq, Hkv, d, F, rope_base=500000.0, eps=1e-5, device="cuda"):
        self.w, self.D, self.Hq, self.Hkv, self.d, self.F = weights, D, Hq, Hkv, d, F
        self.rope_base, self.eps = rope_base, eps
        bf = torch.bfloat16
        e = lambda *shape: torch.empty(shape, dtype=bf, device=device)
        self.xn, self.q, self.k, self.v = e(MAX_ROWS, D), e(MAX_ROWS, Hq, d), e(MAX_ROWS, Hkv, d), e(MAX_ROWS, Hkv, d)
        self.o, self.h, self.a, self.y = e(MAX_ROWS, Hq, d), e(MAX_ROWS, D), e(MAX_ROWS, F), e(MAX_ROWS, D)
        self.lse = torch.empty((MAX_ROWS, Hq), dtype=torch.float32, device=device)

    def step(self, x, p, lay, mem_k, mem_v, ring_k, ring_v, ws=None, full_kv=False):
        """x [R, D] rows entering the layer (row 0 the raw token at position p,
        rows 1.. the slots materialised in p's pass, in order).  mem_k/mem_v and
        ring_k/ring_v are [1, Hkv, cap, d] buffers described by `lay`.  Returns
        y [R, D] (a view of this layer's output buffer)."""
        R = x.shape[0]
        upd = None if full_kv else lay.update_in_pass_of(p)
        if (upd is None and R != 1) or (upd is not None and R != 1 + len(upd.positions)):
            raise ValueError("rows must be the raw token plus the slots materialised in its pass")
        pos = [p] + ([] if upd is None else list(upd.positions))
        w = self.w
        q, k, v, xn = self.q[:R], self.k[:R], self.v[:R], self.xn[:R]
        rmsnorm_qkv_rope(x, w.gamma1, w.w_qkv, pos, self.Hq, self.Hkv, self.d, q, k, v, xn, eps=self.eps,
                         rope_base=self.rope_base, kv_from_row0=R > 1)
        o = self.o[:R]
        if upd is None:
            view = lay.decode_view(p)
            mem = None if full_kv else KV(mem_k, mem_v, [view.mem_len])
            draft_decode_attn(q, mem, KV(ring_k, ring_v, [view.win_len], [view.win_start]), k, v, o,
                              self.lse[:R], ws=ws)
        else:
            memory_update(xn[1:].unsqueeze(0), w.w_kv_g, [upd.positions], KV(mem_k, mem_v, [upd.mem_row]),
                          rope_base=self.rope_base)
            views, modes = lay.step_views(p)
            draft_step_attn(q, KV(mem_k, mem_v, [vw.mem_len for vw in views]),
                            KV(ring_k, ring_v, [vw.win_len for vw in views], [vw.win_start for vw in views]),
                            k, v, modes, o, self.lse[:R], ws=ws)
        h = linear_residual(o.view(R, self.Hq * self.d), w.w_o, x, out=self.h[:R])
        a = rmsnorm_swiglu(h, w.gamma2, w.w_gate_up, out=self.a[:R], eps=self.eps)
        return linear_residual(a, w.w_down, h, out=self.y[:R])
