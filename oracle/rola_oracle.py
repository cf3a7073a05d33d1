"""RoLA oracle: the sparse + rotary-low-rank attention module, written out plainly in fp64 numpy.

TEST INFRASTRUCTURE ONLY -- used by the tests, the smoke check and the benchmark's CPU-baseline leg,
never by the GPU library. Slow on purpose: every step is the paper's definition, in the paper's order,
with no blocking, fusion or reordering beyond what the definition states.

Paper: "RoLA: Rotary-Positioned Low-Rank Linear Attention for Efficient Diffusion Transformers".
Section / equation names below refer to it:
  * Sec. 3 (Preliminary): token grid, attention, 3D RoPE and the relative identity (eq. shiftinv).
  * Sec. 4.1 (Rotary-Positioned Low-Rank Linear Attention): eq. qklr and eq. ctx.
  * Sec. 4.2 (Dimensionality Truncation of the Rotary Schedule): R_r keeps the first r coordinates.
  * Sec. 4.3 (RoPE Outside the Activation): rotate after the nonlinearity.
  * Sec. 4.4 (Feature Alignment and Gated Fusion): gate and eq. gate.
  * Algorithm "RoLA attention forward pass" (appendix "Full Forward Pass"): order of all steps.
  * Appendix "Formal Sanity Checks": Prop. exact, Prop. truncation-bound, Prop. inside.

Points where the paper is silent are fixed by these readings (each also listed in the design notes):
  R1  sparse branch: 1-D contiguous blocks of `block` tokens in flattened (t, y, x) order; key blocks
      chosen per query block as the top-k of mean-pooled rotated Q/K scores q_bar . k_bar / sqrt(d_h);
      ties go to the lower key-block index; the chosen list is stored ascending.
  R2  keep = max(1, floor((1 - sparsity) * n_blocks + 1/2)), evaluated in fp64.
  R3  a partial last block pools over its valid tokens only; padded keys never enter a softmax.
  R4  rotary schedule: axes (t, y, x) each own a contiguous run of pairs (widths d_t, d_y, d_x);
      pair i of an axis of width d_a turns by pos_a * base^(-2i/d_a); pairs are interleaved
      (x_{2j}, x_{2j+1}) and turn by +angle; positions are integers from 0.
  R5  R_r keeps rotary pairs j < r/2 (the first r coordinates of the backbone ordering).
  R6  P_q, P_k have shape [r, d_h]; features are SiLU(P x) then R_r.
  R7  the readout has no linear-attention denominator; its normalisation is the RMSNorm over d_h,
      without a gain, eps_lr = 1e-6. The summary also returns z = sum_q k~_q (reported only).
  R8  the fused output uses eps = 1e-6 and one gate per token shared by all heads.
  R9  Q^r, K^r are the backbone's rotated tensors in the working precision: R(Q^n) rounded once
      (round-to-nearest-even) to the input dtype.
  R10 the activation ablation's GELU is the exact form x * Phi(x) (Phi the standard normal CDF);
      "rotation inside the activation" is phi(R_r(p) P x), as Prop. inside defines it; "no RoPE" is
      phi(P x). Everything else in the branch is unchanged by these variants.
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "token_positions", "pair_schedule", "rope_tables", "rotate", "round_to", "round_bf16",
    "num_blocks", "keep_blocks", "pool_blocks", "block_scores", "select_blocks",
    "sparse_attention", "sparse_attention_rows", "sparse_attention_blocks", "silu",
    "lowrank_features", "lowrank_summary", "lowrank_readout_u", "rms_normalize", "lowrank_readout",
    "gate", "combine", "forward_head", "forward", "lowrank_logit", "flop_counts", "activation",
    "features", "gate_logits",
]

# --------------------------------------------------------------------------------------------------
# Token grid and 3D RoPE  (Sec. 3, Notation and 3D RoPE; Sec. 4.2)
# --------------------------------------------------------------------------------------------------


def token_positions(T: int, Hs: int, Ws: int, offset=(0, 0, 0)) -> np.ndarray:
    """(t, y, x) of every flattened token, shape [N, 3], with token n = (t*Hs + y)*Ws + x.

    Sec. 3 flattens the video into L = T*Hs*Ws tokens p = (t, x, y); R4 fixes integer positions from 0.
    `offset` translates every position (used by the shift-invariance checks).
    """
    t, y, x = np.meshgrid(np.arange(T), np.arange(Hs), np.arange(Ws), indexing="ij")
    pos = np.stack([t.ravel(), y.ravel(), x.ravel()], axis=1).astype(np.float64)
    return pos + np.asarray(offset, dtype=np.float64)[None, :]


def pair_schedule(split, base: float = 10000.0):
    """Axis id and angular frequency of each rotary pair j in [0, d_h/2).

    3D RoPE partitions d_h = d_t + d_y + d_x (Sec. 3); each axis uses RoFormer's exponentially decaying
    schedule over its own width (reading R4): theta = base^(-2i/d_a) for local pair i.
    """
    axis, theta = [], []
    for a, d_a in enumerate(split):
        if d_a <= 0 or d_a % 2:
            raise ValueError(f"axis width {d_a} must be positive and even")
        for i in range(d_a // 2):
            axis.append(a)
            theta.append(base ** (-2.0 * i / d_a))
    return np.asarray(axis, dtype=np.int64), np.asarray(theta, dtype=np.float64)


def rope_tables(T: int, Hs: int, Ws: int, split, base: float = 10000.0, offset=(0, 0, 0)):
    """The backbone's (freqs_cos, freqs_sin): cos/sin of pos_axis(j) * theta_j, each [N, d_h/2]."""
    pos = token_positions(T, Hs, Ws, offset)
    axis, theta = pair_schedule(split, base)
    ang = pos[:, axis] * theta[None, :]
    return np.cos(ang), np.sin(ang)


def rotate(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Block-diagonal RoPE rotation of the interleaved pairs of the last axis of x ([..., N, m]).

    Uses table columns j < m/2, so m = d_h gives the full R(p) of Sec. 3 and m = r gives R_r(p) of
    Sec. 4.2 (the first r coordinates = r/2 complete pairs, reading R5). Pair j maps
    (a, b) -> (a cos - b sin, a sin + b cos), i.e. a turn by +angle (reading R4).
    """
    m = x.shape[-1]
    if m % 2:
        raise ValueError("rotated width must be even")
    c = cos[:, : m // 2]
    s = sin[:, : m // 2]
    a = x[..., 0::2]
    b = x[..., 1::2]
    out = np.empty(np.broadcast_shapes(x.shape), dtype=np.float64)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bfloat16 (8 significant bits), ties to even."""
    m, e = np.frexp(np.asarray(x, dtype=np.float64))
    return np.ldexp(np.rint(m * 256.0), e - 8)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round once to the working precision (reading R9); 'f64' leaves values untouched."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    raise ValueError(dtype)


# --------------------------------------------------------------------------------------------------
# Sparse branch  (Algorithm, steps 3-4; Sec. 4 opening: standard block-sparse attention, top-k ratio)
# --------------------------------------------------------------------------------------------------


def num_blocks(N: int, block: int) -> int:
    return -(-N // block)


def keep_blocks(n_blocks: int, sparsity: float) -> int:
    """Key blocks kept per query block (reading R2). Sparsity is the fraction of query-key
    interactions removed (Sec. 5.1 evaluation setting), so about (1 - S) * n_blocks blocks remain."""
    if not (0.0 <= sparsity < 1.0):
        raise ValueError("sparsity must lie in [0, 1)")
    k = int(math.floor((1.0 - sparsity) * float(n_blocks) + 0.5))
    return max(1, min(n_blocks, k))


def pool_blocks(x: np.ndarray, block: int) -> np.ndarray:
    """Mean of each contiguous block of tokens over its valid tokens only (readings R1, R3). x: [N, d]."""
    N = x.shape[0]
    nb = num_blocks(N, block)
    out = np.empty((nb, x.shape[1]), dtype=np.float64)
    for I in range(nb):
        out[I] = x[I * block: min(N, (I + 1) * block)].mean(axis=0)
    return out


def block_scores(qbar: np.ndarray, kbar: np.ndarray) -> np.ndarray:
    """Block score S_IJ = q_bar_I . k_bar_J / sqrt(d_h) (reading R1; scale of Sec. 3)."""
    return qbar @ kbar.T / math.sqrt(qbar.shape[1])


def select_blocks(scores: np.ndarray, keep: int) -> np.ndarray:
    """Indices of the `keep` largest scores of every row, ties to the lower index, stored ascending."""
    nb_q, nb_k = scores.shape
    idx = np.empty((nb_q, keep), dtype=np.int64)
    J = np.arange(nb_k)
    for I in range(nb_q):
        order = np.lexsort((J, -scores[I]))  # primary: score descending; secondary: index ascending
        idx[I] = np.sort(order[:keep])
    return idx


def _block_tokens(J: int, block: int, N: int) -> np.ndarray:
    return np.arange(J * block, min(N, (J + 1) * block))


def sparse_attention_rows(qr, kr, v, idx, block: int, scale: float, rows) -> np.ndarray:
    """O^s for the given query rows: softmax over the valid keys of the selected blocks of the row's
    query block (attention of Sec. 3 restricted to the block mask). Written as a direct softmax; the
    online form used on the GPU is an exact reformulation of it."""
    N = qr.shape[0]
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((rows.size, v.shape[1]), dtype=np.float64)
    for n, p in enumerate(rows):
        keys = np.concatenate([_block_tokens(J, block, N) for J in idx[p // block]])
        s = (kr[keys] @ qr[p]) * scale
        w = np.exp(s - s.max())
        out[n] = (w / w.sum()) @ v[keys]
    return out


def sparse_attention(qr, kr, v, idx, block: int, scale: float) -> np.ndarray:
    """O^s for every token, one query block at a time."""
    N = qr.shape[0]
    out = np.empty_like(v, dtype=np.float64)
    for I in range(idx.shape[0]):
        q_rows = _block_tokens(I, block, N)
        keys = np.concatenate([_block_tokens(J, block, N) for J in idx[I]])
        s = (qr[q_rows] @ kr[keys].T) * scale
        w = np.exp(s - s.max(axis=1, keepdims=True))
        out[q_rows] = (w / w.sum(axis=1, keepdims=True)) @ v[keys]
    return out


def sparse_attention_blocks(qr, kr, v, idx, block: int, scale: float, blocks) -> np.ndarray:
    """O^s for the tokens of the given query blocks (in the order given), the same direct softmax as
    sparse_attention; idx holds the lists of every query block [n_blocks, keep]."""
    N = qr.shape[0]
    out = []
    for I in blocks:
        q_rows = _block_tokens(int(I), block, N)
        keys = np.concatenate([_block_tokens(J, block, N) for J in idx[int(I)]])
        s = (qr[q_rows] @ kr[keys].T) * scale
        w = np.exp(s - s.max(axis=1, keepdims=True))
        out.append((w / w.sum(axis=1, keepdims=True)) @ v[keys])
    return np.concatenate(out, axis=0)


# --------------------------------------------------------------------------------------------------
# Low-rank branch  (eq. qklr, eq. ctx; Algorithm, steps 5-7)
# --------------------------------------------------------------------------------------------------


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU(x) = x / (1 + e^-x), evaluated without overflow for large |x|."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = x[pos] / (1.0 + np.exp(-x[pos]))
    e = np.exp(x[~pos])
    out[~pos] = x[~pos] * e / (1.0 + e)
    return out


_erf = np.vectorize(math.erf, otypes=[np.float64])


def activation(x: np.ndarray, phi: str = "silu") -> np.ndarray:
    """Feature map of the low-rank branch: SiLU (eq. qklr), or one of the alternatives of the
    activation ablation (Sec. 5.3, Tab. abl_activation): identity, tanh, ReLU, and GELU in its exact
    form x * Phi(x), Phi the standard normal CDF (reading R10)."""
    x = np.asarray(x, dtype=np.float64)
    if phi == "silu":
        return silu(x)
    if phi == "identity":
        return x.copy()
    if phi == "tanh":
        return np.tanh(x)
    if phi == "relu":
        return np.maximum(x, 0.0)
    if phi == "gelu":
        return x * 0.5 * (1.0 + _erf(x / math.sqrt(2.0)))
    raise ValueError(f"unknown feature map {phi!r}")


def features(x: np.ndarray, P: np.ndarray, cos, sin, phi: str = "silu",
             ordering: str = "outside") -> np.ndarray:
    """Low-rank features of every token under a feature map and a place of the rotation: outside,
    R_r(p) phi(P x_p) (eq. qklr, Sec. 4.3, the paper's design); inside, phi(R_r(p) P x_p) (Prop.
    inside); none, phi(P x_p) (position-blind). x: [N, d_h], P: [r, d_h] -> [N, r]."""
    y = x @ P.T
    if ordering == "outside":
        return rotate(activation(y, phi), cos, sin)
    if ordering == "inside":
        return activation(rotate(y, cos, sin), phi)
    if ordering == "none":
        return activation(y, phi)
    raise ValueError(f"unknown rotation order {ordering!r}")


def lowrank_features(x: np.ndarray, P: np.ndarray, cos, sin, phi: str = "silu",
                     ordering: str = "outside") -> np.ndarray:
    """Rotary low-rank features R_r(p) SiLU(P x_p) of every token (eq. qklr; RoPE outside the
    activation, Sec. 4.3), or a variant (see features). x: [N, d_h], P: [r, d_h] -> [N, r]."""
    return features(x, P, cos, sin, phi, ordering)


def lowrank_summary(kn, v, Pk, cos, sin, phi: str = "silu", ordering: str = "outside"):
    """Global context C = sum_q k~_q v_q^T in R^{r x d_h} (eq. ctx; computed once per head) and the
    feature sum z = sum_q k~_q (reading R7). v is not rotated."""
    kt = lowrank_features(kn, Pk, cos, sin, phi, ordering)
    return kt.T @ v, kt.sum(axis=0)


def lowrank_readout_u(qn, Pq, cos, sin, C, phi: str = "silu", ordering: str = "outside") -> np.ndarray:
    """Pre-normalisation readout u_p = q~_p^T C for every token (eq. ctx)."""
    return lowrank_features(qn, Pq, cos, sin, phi, ordering) @ C


def rms_normalize(u: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis without a gain (reading R7)."""
    return u / np.sqrt(np.mean(u * u, axis=-1, keepdims=True) + eps)


def lowrank_readout(qn, Pq, cos, sin, C, eps_lr: float = 1e-6, phi: str = "silu",
                    ordering: str = "outside") -> np.ndarray:
    """O^lr_p = RMSNorm(q~_p^T C) (eq. ctx)."""
    return rms_normalize(lowrank_readout_u(qn, Pq, cos, sin, C, phi, ordering), eps_lr)


# --------------------------------------------------------------------------------------------------
# Gated fusion  (Sec. 4.4, eq. gate; Algorithm, steps 8-10)
# --------------------------------------------------------------------------------------------------


def gate_logits(X: np.ndarray, Wg: np.ndarray, bg: float) -> np.ndarray:
    """The gate's pre-activation X W_g + b_g over the block's input hidden states (Sec. 4.4;
    Algorithm step 8). X: [..., d_model], W_g: [d_model] -> [...]."""
    return np.asarray(X, np.float64) @ np.asarray(Wg, np.float64) + float(bg)


def gate(logits: np.ndarray) -> np.ndarray:
    """g = sigma(X W_g + b_g); the ABI receives the logit X W_g + b_g (reading R8)."""
    x = np.asarray(logits, dtype=np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    e = np.exp(x[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def combine(os_, olr, logits, eps: float = 1e-6) -> np.ndarray:
    """O_p = (O^s_p / r_p + g_p O^lr_p) r_p with r_p = sqrt(mean_i (O^s_{p,i})^2 + eps) (eq. gate),
    in this literal form. os_, olr: [N, d_h]; logits: [N]."""
    r = np.sqrt(np.mean(os_ * os_, axis=-1, keepdims=True) + eps)
    return (os_ / r + gate(logits)[:, None] * olr) * r


# --------------------------------------------------------------------------------------------------
# Whole module
# --------------------------------------------------------------------------------------------------


def forward_head(qn, kn, v, Pq, Pk, logits, cos, sin, *, block, sparsity, dtype="f64",
                 eps_lr=1e-6, eps=1e-6):
    """One (batch, head) slice of the module, in the order of the Algorithm:
    step 3 Q^r, K^r = R(Q^n), R(K^n) (rounded to the working precision, reading R9); step 4 sparse
    branch (block selection + block-sparse softmax); steps 5-7 low-rank branch; steps 8-10 fusion.
    Returns every intermediate as a dict."""
    N, d_h = qn.shape
    qr = round_to(rotate(qn, cos, sin), dtype)
    kr = round_to(rotate(kn, cos, sin), dtype)
    block = int(block)
    nb = num_blocks(N, block)
    keep = keep_blocks(nb, sparsity)
    qbar, kbar = pool_blocks(qr, block), pool_blocks(kr, block)
    scores = block_scores(qbar, kbar)
    idx = select_blocks(scores, keep)
    scale = 1.0 / math.sqrt(d_h)
    o_s = sparse_attention(qr, kr, v, idx, block, scale)
    C, z = lowrank_summary(kn, v, Pk, cos, sin)
    u = lowrank_readout_u(qn, Pq, cos, sin, C)
    o_lr = rms_normalize(u, eps_lr)
    out = combine(o_s, o_lr, logits, eps)
    return dict(qr=qr, kr=kr, qbar=qbar, kbar=kbar, scores=scores, idx=idx, keep=keep, o_s=o_s,
                C=C, z=z, u=u, o_lr=o_lr, out=out)


def forward(Qn, Kn, V, Pq, Pk, logits, *, grid, split, block, sparsity, base=10000.0,
            dtype="f64", eps_lr=1e-6, eps=1e-6, offset=(0, 0, 0)):
    """The module over [B, H, N, d_h] inputs (P_q, P_k: [H, r, d_h]; logits: [B, N]).
    Returns a dict of stacked intermediates (idx: [B, H, n_b, keep])."""
    T, Hs, Ws = grid
    B, H, N, d_h = Qn.shape
    if N != T * Hs * Ws:
        raise ValueError("N must equal T*Hs*Ws")
    if sum(split) != d_h:
        raise ValueError("axis split must sum to d_h")
    cos, sin = rope_tables(T, Hs, Ws, split, base, offset)
    res = {}
    for b in range(B):
        for h in range(H):
            r = forward_head(Qn[b, h], Kn[b, h], V[b, h], Pq[h], Pk[h], logits[b], cos, sin,
                             block=block, sparsity=sparsity, dtype=dtype, eps_lr=eps_lr, eps=eps)
            for k, val in r.items():
                res.setdefault(k, []).append(val)
    out = {}
    for k, vals in res.items():
        if k == "keep":
            out[k] = vals[0]
            continue
        arr = np.stack(vals)
        out[k] = arr.reshape((B, H) + arr.shape[1:])
    out["cos"], out["sin"] = cos, sin
    return out


# --------------------------------------------------------------------------------------------------
# Negative controls and the mechanism metric  (Sec. 4.3; Prop. inside; Sec. 5.1 RoPE placement)
# --------------------------------------------------------------------------------------------------


def lowrank_logit(qn_p, kn_q, Pq, Pk, pos_p, pos_q, split, base=10000.0, ordering="outside",
                  phi="silu"):
    """Pre-RMSNorm low-rank logit s(p, q) = q~_p . k~_q of one query/key pair placed at explicit
    positions (the quantity whose shift residual |s(p+d, q+d) - s(p, q)| Sec. 5.1 measures)."""
    r = Pq.shape[0]
    axis, theta = pair_schedule(split, base)
    def table(pos):
        ang = np.asarray(pos, dtype=np.float64)[axis] * theta
        return np.cos(ang)[None, :], np.sin(ang)[None, :]
    cp, sp = table(pos_p)
    cq, sq = table(pos_q)
    a = features(qn_p[None, :], Pq, cp, sp, phi, ordering)[0]
    b = features(kn_q[None, :], Pk, cq, sq, phi, ordering)[0]
    assert a.shape == (r,)
    return float(a @ b)


# --------------------------------------------------------------------------------------------------
# FLOP accounting  (appendix "Computational Complexity Analysis")
# --------------------------------------------------------------------------------------------------


def flop_counts(B, H, L, d_h, r, S):
    """The paper's dominant-matmul FLOP counts: C_sparse, C_lowrank, C_fusion and eta."""
    c_sparse = 4.0 * B * H * L * L * (1.0 - S) * d_h
    c_lowrank = 8.0 * B * H * L * d_h * r
    c_fusion = 2.0 * B * H * L * d_h
    return dict(sparse=c_sparse, lowrank=c_lowrank, fusion=c_fusion,
                eta=(c_lowrank + c_fusion) / c_sparse)
