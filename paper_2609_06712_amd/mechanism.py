"""Positional metrics of the low-rank branch (Sec. 5.1, "RoPE placement"; Tab. mechanism).

On content-controlled inputs -- one query vector q^n at every token and one key vector k^n at every
token -- the pre-RMSNorm low-rank logit s(p, q) = q~_p . k~_q depends on the positions only. Along a
temporal line of the latent grid (y, x fixed), with s(t1, t2) the logit between the tokens at times t1
and t2:
  offset range    max - min over the offset D = t2 - t1 of the mean of s(t, t + D) over t;
  shift residual  max over D of the spread (max - min) of s(t, t + D) over t, i.e. the largest
                  |s(p + d, q + d) - s(p, q)| for a translation d along the line.
Both are divided by max |s| (the paper's normalisation is not stated). With the rotation outside the
activation the residual is zero up to rounding (Prop. exact); inside it, a nonlinear phi leaks the
absolute position (Prop. inside); without rotation the logit is constant.

The features come from rola_lowrank_features (the library's kernels); the T x T logits and the two
reductions over them are small host computations in fp64.
"""

from __future__ import annotations

import math

import numpy as np
import torch

from . import rola as R


def positional_metrics(phi="silu", rope_order="outside", grid=(21, 45, 80), split=(44, 42, 42), r=32,
                       seed=0, device="cuda"):
    T, Hs, Ws = grid
    N, d = T * Hs * Ws, sum(split)
    rng = np.random.default_rng(seed)
    f32 = lambda a: a.astype(np.float32).astype(np.float64)  # noqa: E731  values as the GPU sees them
    qv, kv = f32(rng.standard_normal(d)), f32(rng.standard_normal(d))
    Pq, Pk = (f32(rng.standard_normal((r, d)) / math.sqrt(d)) for _ in range(2))
    prob = R.problem(1, 1, N, d, grid, "f32")
    cos, sin = R.rola_rope_tables(prob, split)
    dev = torch.device(device)
    Xq = torch.tensor(qv, dtype=torch.float32, device=dev).expand(1, 1, N, d).contiguous()
    Xk = torch.tensor(kv, dtype=torch.float32, device=dev).expand(1, 1, N, d).contiguous()
    Pq_t = torch.tensor(Pq, dtype=torch.float32, device=dev)[None]
    Pk_t = torch.tensor(Pk, dtype=torch.float32, device=dev)[None]
    Fq = R.rola_lowrank_features(Xq, Pq_t, r, cos, sin, grid, phi, rope_order)
    Fk = R.rola_lowrank_features(Xk, Pk_t, r, cos, sin, grid, phi, rope_order)
    y, x = Hs // 2, Ws // 2
    line = torch.arange(T, device=dev) * (Hs * Ws) + y * Ws + x
    fq = Fq[0, 0, line].to("cpu", torch.float64).numpy()
    fk = Fk[0, 0, line].to("cpu", torch.float64).numpy()
    S = fq @ fk.T  # s(t1, t2)
    scale = float(np.abs(S).max())
    curve, spread = [], []
    for D in range(-(T - 1), T):
        diag = np.diagonal(S, offset=D)
        curve.append(diag.mean())
        spread.append(diag.max() - diag.min())
    norm = scale if scale > 0 else 1.0
    return dict(S=S, scale=scale, offset_range=float((max(curve) - min(curve)) / norm),
                shift_residual=float(max(spread) / norm), T=T, y=y, x=x, qv=qv, kv=kv, Pq=Pq, Pk=Pk,
                split=split, r=r)


def main():
    """Prints the metrics of every feature map and rotation order as a markdown table."""
    print("| phi | rotation | shift residual | offset range |\n|---|---|---|---|")
    for phi in R.PHI:
        for order in R.ROPE_ORDER:
            res = positional_metrics(phi=phi, rope_order=order, seed=3)
            print(f"| {phi} | {order} | {res['shift_residual']:.2e} | {res['offset_range']:.3f} |",
                  flush=True)


if __name__ == "__main__":
    main()
