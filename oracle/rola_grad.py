"""Gradients of the RoLA module for fine-tuning (Sec. 4.5 "Implementation Details": the new
parameters P_q, P_k, W_g, b_g are trained jointly with the backbone, so the backward pass runs
through both branches and the gated fusion).

TEST INFRASTRUCTURE ONLY, like the rest of oracle/. The forward definitions of the numpy oracle
(Sec. 3 attention, eq. qklr, eq. ctx, eq. gate; Algorithm "RoLA attention forward pass") are
transcribed here into plain fp64 PyTorch CPU operations, written out densely (the block-sparse
softmax as a softmax over an explicit N x N block mask), and differentiated by torch.autograd. The
block selection is piecewise constant in its inputs and is held fixed (its index list is an input).
The transcription is pinned to the numpy oracle by finite differences in the tests.
"""

from __future__ import annotations

import math

import numpy as np
import torch

__all__ = ["sparse_attention_grads", "lowrank_combine_grads", "gate_grads", "module_grads"]

_T = torch.float64


def _t(x, grad=False):
    t = torch.as_tensor(np.asarray(x, np.float64), dtype=_T)
    return t.requires_grad_(grad)


def _rotate(x, cos, sin):
    """Pairs (2j, 2j+1) turned by +angle, table columns j < width/2 (the oracle's rotate)."""
    m = x.shape[-1] // 2
    c, s = cos[:, :m], sin[:, :m]
    a, b = x[..., 0::2], x[..., 1::2]
    return torch.stack((a * c - b * s, a * s + b * c), dim=-1).flatten(-2)


def _block_mask(idx, N, block):
    """M[p, q] = key q's block is among the blocks selected by query p's block."""
    nb = idx.shape[0]
    sel = torch.zeros((nb, nb), dtype=torch.bool)
    sel[torch.arange(nb)[:, None], torch.as_tensor(np.asarray(idx, np.int64))] = True
    blk = torch.arange(N) // block
    return sel[blk[:, None], blk[None, :]]


def _sparse(qr, kr, v, mask, scale):
    s = (qr @ kr.transpose(-1, -2)) * scale
    s = s.masked_fill(~mask, float("-inf"))
    return torch.softmax(s, dim=-1) @ v


def _features(x, P, cos, sin):
    y = x @ P.transpose(-1, -2)
    return _rotate(y * torch.sigmoid(y), cos, sin)


def _lowrank_u(qn, kn, v, Pq, Pk, cos, sin):
    C = _features(kn, Pk, cos, sin).transpose(-1, -2) @ v
    return _features(qn, Pq, cos, sin) @ C


def _combine(os_, u, logits, eps_lr, eps):
    olr = u / torch.sqrt((u * u).mean(-1, keepdim=True) + eps_lr)
    r = torch.sqrt((os_ * os_).mean(-1, keepdim=True) + eps)
    return (os_ / r + torch.sigmoid(logits)[..., None] * olr) * r


def sparse_attention_grads(qr, kr, v, idx, block, scale, dout):
    """d/d(Q^r, K^r, V) of <dout, O^s> for one head (idx: [n_b, keep], fixed)."""
    q, k, vv = _t(qr, True), _t(kr, True), _t(v, True)
    out = _sparse(q, k, vv, _block_mask(idx, q.shape[0], block), scale)
    g = torch.autograd.grad(out, (q, k, vv), _t(dout))
    return {n: x.numpy() for n, x in zip(("dqr", "dkr", "dv"), g)}


def lowrank_combine_grads(qn, kn, v, Pq, Pk, os_, logits, cos, sin, dout, eps_lr=1e-6, eps=1e-6):
    """d/d(Q^n, K^n, V, P_q, P_k, O^s, logits) of <dout, O> with O = combine(O^s, RMSNorm(q~^T C))
    for one head; the sparse output O^s enters as an input."""
    args = [_t(a, True) for a in (qn, kn, v, Pq, Pk, os_, logits)]
    qn_, kn_, v_, Pq_, Pk_, os_t, lg = args
    c, s = _t(cos), _t(sin)
    u = _lowrank_u(qn_, kn_, v_, Pq_, Pk_, c, s)
    out = _combine(os_t, u, lg, eps_lr, eps)
    g = torch.autograd.grad(out, args, _t(dout))
    return {n: x.numpy() for n, x in zip(("dqn", "dkn", "dv", "dPq", "dPk", "dos", "dlogits"), g)}


def gate_grads(X, Wg, dlogits):
    """d/d(X, W_g, b_g) of <dlogits, X W_g + b_g>."""
    X_, W_, b_ = _t(X, True), _t(Wg, True), _t(0.0, True)
    out = X_ @ W_ + b_
    g = torch.autograd.grad(out, (X_, W_, b_), _t(dlogits))
    return {"dX": g[0].numpy(), "dWg": g[1].numpy(), "dbg": float(g[2])}


def module_grads(qn, kn, v, Pq, Pk, logits, cos, sin, idx, block, dout, eps_lr=1e-6, eps=1e-6):
    """The whole module for one head with the backbone rotation Q^r = R(Q^n), K^r = R(K^n) inside:
    d/d(Q^n, K^n, V, P_q, P_k, logits) of <dout, O>."""
    args = [_t(a, True) for a in (qn, kn, v, Pq, Pk, logits)]
    qn_, kn_, v_, Pq_, Pk_, lg = args
    c, s = _t(cos), _t(sin)
    scale = 1.0 / math.sqrt(qn_.shape[-1])
    os_ = _sparse(_rotate(qn_, c, s), _rotate(kn_, c, s), v_,
                  _block_mask(idx, qn_.shape[0], block), scale)
    out = _combine(os_, _lowrank_u(qn_, kn_, v_, Pq_, Pk_, c, s), lg, eps_lr, eps)
    g = torch.autograd.grad(out, args, _t(dout))
    return {n: x.numpy() for n, x in zip(("dqn", "dkn", "dv", "dPq", "dPk", "dlogits"), g)}
