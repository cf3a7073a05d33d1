"""Forward and backward of the module for fine-tuning (Sec. 4.5: P_q, P_k, W_g, b_g are trained jointly
with the backbone), composed from the library's entry points.

forward() keeps what the backward needs: the rotated Q^r, K^r (Algorithm step 3), the block lists,
O^s with its per-query log-sum-exp, and the summary C. backward() runs the low-rank/fusion backward
(which also yields dO^s and the gate-logit gradient), the block-sparse attention backward, and maps
dQ^r, dK^r back through the backbone rotation (R(p)^T = R(-p)); the two branches' shares of dQ^n,
dK^n and dV are added. Every step, the additions included, runs in the library's kernels.
"""

from __future__ import annotations

import torch

from . import rola as R


def forward(Qn, Kn, V, Pq, Pk, logits, grid, split, block=64, sparsity=0.9, r=32, base=10000.0):
    prob = R.problem_of(Qn, grid)
    cos, sin = R.rola_rope_tables(prob, split, base)
    qr = R.rola_rope_apply(Qn, cos, sin, grid)
    kr = R.rola_rope_apply(Kn, cos, sin, grid)
    idx = R.rola_block_select(qr, kr, grid, block, sparsity)
    os_, lse = R.rola_sparse_attn_lse(qr, kr, V, grid, block, sparsity, idx)
    C, _ = R.rola_lowrank_summary(Kn, V, Pk, r, cos, sin, grid, want_z=False)
    out = R.rola_lowrank_readout_combine(Qn, Pq, r, cos, sin, C, os_, logits, grid)
    saved = dict(cos=cos, sin=sin, qr=qr, kr=kr, idx=idx, os=os_, lse=lse, C=C, grid=grid,
                 block=block, sparsity=sparsity, r=r)
    return out, saved


def backward(Qn, Kn, V, Pq, Pk, logits, saved, dO):
    """Gradients of <dO, O>: dict of dQn, dKn, dV (fp32 [B, H, N, d]), dPq, dPk (fp32 [H, r, d]) and
    dlogits (fp32 [B, N])."""
    g, r = saved["grid"], saved["r"]
    cos, sin = saved["cos"], saved["sin"]
    dOs, dQn, dKn, dV, dPq, dPk, dlog = R.rola_lowrank_backward(
        Qn, Kn, V, Pq, Pk, r, cos, sin, saved["C"], saved["os"], logits, dO, g)
    dQr, dKr, dVs = R.rola_sparse_attn_backward(saved["qr"], saved["kr"], V, g, saved["block"],
                                                saved["sparsity"], saved["idx"], saved["os"],
                                                saved["lse"], dOs)
    R.rola_rope_backward_accumulate(dQr, cos, sin, g, dQn)           # dQ^n += R(p)^T dQ^r
    R.rola_rope_backward_accumulate(dKr, cos, sin, g, dKn)           # dK^n += R(p)^T dK^r
    R.rola_rope_backward_accumulate(dVs, cos, sin, g, dV, rotate=False)
    return dict(dQn=dQn, dKn=dKn, dV=dV, dPq=dPq, dPk=dPk, dlogits=dlog)
