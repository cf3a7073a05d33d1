"""Independent formulations used to pin the oracle (never used by the oracle itself).

The rotary matrix here is built as the matrix exponential of a skew-symmetric generator, with the
per-axis frequencies taken from numpy.logspace -- a different route to the same definition than the
oracle's table-and-pairs code, so a sign, index, axis-order or frequency mistake in either shows up.
"""

import math

import numpy as np
import scipy.linalg
import torch


def frequencies(split, base=10000.0):
    """RoFormer schedule per axis: theta_i = base^(-2i/d_a), i < d_a/2, via logspace."""
    out = []
    for d_a in split:
        n = d_a // 2
        out.append(np.logspace(0.0, -(n - 1) * 2.0 / d_a * math.log10(base), n))
    return out


def generator(split, pos, base=10000.0, r=None):
    """Skew-symmetric A(p) with R(p) = expm(A(p)): pair j turns by +pos_axis * theta_j.
    With r given, only the first r coordinates (r/2 pairs) are kept."""
    d = sum(split)
    A = np.zeros((d, d))
    j = 0
    for a, freqs in enumerate(frequencies(split, base)):
        for f in freqs:
            ang = pos[a] * f
            A[2 * j + 1, 2 * j] = ang
            A[2 * j, 2 * j + 1] = -ang
            j += 1
    if r is not None:
        A = A[:r, :r]
    return A


def rotation(split, pos, base=10000.0, r=None):
    return scipy.linalg.expm(generator(split, pos, base, r))


def positions(grid, offset=(0, 0, 0)):
    T, Hs, Ws = grid
    out = []
    for t in range(T):
        for y in range(Hs):
            for x in range(Ws):
                out.append((t + offset[0], y + offset[1], x + offset[2]))
    return np.asarray(out, dtype=np.float64)


def sdpa_f64(q, k, v):
    """torch's scaled_dot_product_attention in fp64 on the CPU (a library routine)."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None]
    return torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v))[0, 0].numpy()


def silu_ref(x):
    return x * (1.0 / (1.0 + np.exp(-x)))


def activation_ref(x, phi):
    """The ablation's feature maps written independently of the oracle: tanh through exponentials,
    ReLU as (x + |x|) / 2, GELU through scipy's normal CDF."""
    from scipy.stats import norm
    x = np.asarray(x, dtype=np.float64)
    if phi == "silu":
        return silu_ref(x)
    if phi == "identity":
        return x
    if phi == "tanh":
        e = np.exp(-2.0 * np.abs(x))
        return np.sign(x) * (1.0 - e) / (1.0 + e)
    if phi == "relu":
        return 0.5 * (x + np.abs(x))
    if phi == "gelu":
        return x * norm.cdf(x)
    raise ValueError(phi)
