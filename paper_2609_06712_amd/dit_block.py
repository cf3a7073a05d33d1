"""A synthetic Wan-shaped video-DiT block around the attention module, with random weights.

It exists to relate the module's per-layer time to a denoising step: everything around the
self-attention is the usual video-DiT block (adaptive LayerNorm modulation, QKV projection with
RMSNorm on q and k, output projection, cross-attention to text tokens, GELU MLP), and the
self-attention is either the RoLA module (gate logits, backbone RoPE, block selection, low-rank
summary, sparse attention with the low-rank readout and gated combine in its epilogue -- all this
library's kernels) or this library's dense attention kernel. The projections and the MLP are plain
library GEMMs (torch.matmul); the cross-attention is a plain chunked softmax attention (torch). The
shapes follow the public Wan2.1 configurations; the weights are random, so only timing and plumbing
are meaningful.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import torch
import torch.nn.functional as F

from . import rola as R


@dataclass(frozen=True)
class DiTShape:
    name: str
    d_model: int
    heads: int
    ffn: int
    layers: int
    text_len: int
    grid: tuple
    split: tuple = (44, 42, 42)


WAN_1_3B_480P = DiTShape("wan2.1-1.3b-480p", 1536, 12, 8960, 30, 512, (21, 30, 52))
WAN_14B_720P = DiTShape("wan2.1-14b-720p", 5120, 40, 13824, 40, 512, (21, 45, 80))


def _rms(x, w, eps=1e-6):
    x32 = x.float()
    return (x32 * torch.rsqrt(x32.pow(2).mean(-1, keepdim=True) + eps) * w.float()).to(x.dtype)


def _ln(x, eps=1e-6):
    return F.layer_norm(x.float(), (x.shape[-1],), eps=eps)


class DiTBlock:
    """One block; `attn` is "rola" or "dense". Weights are drawn from a seeded generator."""

    def __init__(self, shape: DiTShape, attn="rola", block=64, sparsity=0.9, r=32, seed=0,
                 device="cuda"):
        self.s, self.attn, self.block, self.sparsity, self.r = shape, attn, block, sparsity, r
        d, H, dh = shape.d_model, shape.heads, shape.d_model // shape.heads
        assert dh == 128
        g = torch.Generator(device="cpu").manual_seed(seed)
        bf = torch.bfloat16

        def w(*sz, scale):
            return (torch.randn(sz, generator=g) * scale).to(bf).to(device)

        self.Wqkv, self.bqkv = w(3 * d, d, scale=d ** -0.5), w(3 * d, scale=0.02)
        self.Wo, self.bo = w(d, d, scale=d ** -0.5), w(d, scale=0.02)
        self.nq, self.nk = 1 + w(d, scale=0.1), 1 + w(d, scale=0.1)
        self.Wcq, self.Wck, self.Wcv = (w(d, d, scale=d ** -0.5) for _ in range(3))
        self.Wco = w(d, d, scale=d ** -0.5)
        self.ncq, self.nck = 1 + w(d, scale=0.1), 1 + w(d, scale=0.1)
        self.W1, self.b1 = w(shape.ffn, d, scale=d ** -0.5), w(shape.ffn, scale=0.02)
        self.W2, self.b2 = w(d, shape.ffn, scale=shape.ffn ** -0.5), w(d, scale=0.02)
        self.mod = w(6, d, scale=0.1)  # shift, scale, gate of the attention and of the MLP
        self.Pq, self.Pk = w(H, r, dh, scale=dh ** -0.5), w(H, r, dh, scale=dh ** -0.5)
        self.Wg, self.bg = torch.zeros(d, dtype=bf, device=device), -1.946  # the paper's init
        N = math.prod(shape.grid)
        prob = R.problem(1, H, N, dh, shape.grid, "bf16")
        self.cos, self.sin = R.rola_rope_tables(prob, shape.split)
        self.ws_sel = torch.empty(R.select_workspace_bytes(prob, block), dtype=torch.uint8,
                                  device=device)
        self.ws_sum = torch.empty(R.summary_workspace_bytes(prob, r), dtype=torch.uint8,
                                  device=device)
        self.ws_sp = torch.empty(R.sparse_combine_workspace_bytes(prob, block, sparsity, r),
                                 dtype=torch.uint8, device=device)

    def _heads(self, t):  # [N, d] -> [1, H, N, 128] contiguous
        N = t.shape[0]
        return t.view(N, self.s.heads, 128).transpose(0, 1).contiguous().unsqueeze(0)

    def self_attention(self, h, capture=None):
        """h: [N, d] modulated input -> [N, d] attention output before the output projection."""
        s, g = self.s, self.s.grid
        qkv = h @ self.Wqkv.t() + self.bqkv
        q, k, v = qkv.split(s.d_model, dim=-1)
        qn, kn, vh = self._heads(_rms(q, self.nq)), self._heads(_rms(k, self.nk)), self._heads(v)
        qr = R.rola_rope_apply(qn, self.cos, self.sin, g)
        kr = R.rola_rope_apply(kn, self.cos, self.sin, g)
        if self.attn == "dense":
            o = R.rola_dense_attn(qr, kr, vh, g, self.block)
            logits = None
        else:
            logits = R.rola_gate_logits(h.unsqueeze(0).contiguous(), self.Wg, self.bg, g,
                                        H=s.heads)
            idx = R.rola_block_select(qr, kr, g, self.block, self.sparsity, ws=self.ws_sel)
            C, _ = R.rola_lowrank_summary(kn, vh, self.Pk, self.r, self.cos, self.sin, g,
                                          ws=self.ws_sum, want_z=False)
            o = R.rola_sparse_attn_combine(qr, kr, vh, g, self.block, self.sparsity, idx, qn,
                                           self.Pq, self.r, self.cos, self.sin, C, logits,
                                           ws=self.ws_sp)
        if capture is not None:
            capture.update(h=h, qn=qn, kn=kn, v=vh, logits=logits, o=o)
        return o[0].transpose(0, 1).reshape(-1, s.d_model)

    def cross_attention(self, x, ctx, chunk=8192):
        s = self.s
        hc = _ln(x).to(x.dtype)
        q = _rms(hc @ self.Wcq.t(), self.ncq).view(-1, s.heads, 128).transpose(0, 1).contiguous()
        kc = _rms(ctx @ self.Wck.t(), self.nck).view(-1, s.heads, 128).transpose(0, 1)
        vc = (ctx @ self.Wcv.t()).view(-1, s.heads, 128).transpose(0, 1).contiguous()
        kt = kc.transpose(1, 2).contiguous()  # [H, 128, L]
        out = torch.empty_like(q)
        for n0 in range(0, q.shape[1], chunk):
            sc = torch.matmul(q[:, n0:n0 + chunk], kt).float() * (128 ** -0.5)
            out[:, n0:n0 + chunk] = torch.matmul(sc.softmax(-1).to(q.dtype), vc)
        return out.transpose(0, 1).reshape(-1, s.d_model) @ self.Wco.t()

    def forward(self, x, ctx, capture=None):
        """x: [N, d] hidden states, ctx: [L, d] text tokens (bf16) -> [N, d]."""
        sh1, sc1, g1, sh2, sc2, g2 = self.mod.float()
        h = (_ln(x) * (1 + sc1) + sh1).to(x.dtype)
        a = self.self_attention(h, capture)
        x = (x.float() + g1 * (a @ self.Wo.t() + self.bo).float()).to(x.dtype)
        x = (x.float() + self.cross_attention(x, ctx).float()).to(x.dtype)
        h2 = (_ln(x) * (1 + sc2) + sh2).to(x.dtype)
        f = F.gelu(h2 @ self.W1.t() + self.b1, approximate="tanh") @ self.W2.t() + self.b2
        return (x.float() + g2 * f.float()).to(x.dtype)


def inputs(shape: DiTShape, seed=1, device="cuda"):
    g = torch.Generator(device="cpu").manual_seed(seed)
    N = math.prod(shape.grid)
    x = torch.randn((N, shape.d_model), generator=g).to(torch.bfloat16).to(device)
    ctx = torch.randn((shape.text_len, shape.d_model), generator=g).to(torch.bfloat16).to(device)
    return x, ctx
