"""Pins of the oracle's sparse branch: block pooling, top-k block selection, mask density and the
block-sparse softmax (Algorithm steps 3-4; sparsity = fraction of query-key interactions removed)."""

import itertools
import math
import os

import numpy as np
import pytest

import oracle as O
from tests import _pins as P


def _golden_rows(name):
    rows = {}
    path = os.path.join(os.path.dirname(__file__), "golden", name)
    with open(path) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                sec, row, *vals = line.split()
                rows.setdefault(sec, {})[int(row)] = [float(v) for v in vals]
    return {sec: np.array([r[i] for i in sorted(r)]) for sec, r in rows.items()}


def test_block_scores_worked_example():
    """Hand-computed selection of tests/golden/block_scores.txt (d_h = 4, block 2, a partial last
    block): pooled means over valid tokens, scores with the 1/sqrt(d_h) factor, top-k with ties to
    the lower block. A score without the factor (x2), with 1/d_h (x1/2) or transposed fails."""
    g = _golden_rows("block_scores.txt")
    qbar, kbar = O.pool_blocks(g["q"], 2), O.pool_blocks(g["k"], 2)
    np.testing.assert_array_equal(qbar, g["qbar"])
    np.testing.assert_array_equal(kbar, g["kbar"])
    s = O.block_scores(qbar, kbar)
    np.testing.assert_allclose(s, g["score"], rtol=0, atol=1e-15)
    np.testing.assert_array_equal(O.select_blocks(s, 1), g["keep1"].astype(np.int64))
    np.testing.assert_array_equal(O.select_blocks(s, 2), g["keep2"].astype(np.int64))


def test_pool_uses_valid_tokens_only():
    """Each block holds a distinct constant; a partial last block (3 of 8 tokens) must pool to its own
    constant, which fails if padding were averaged in."""
    block, N, d = 8, 8 * 4 + 3, 5
    x = np.repeat(np.arange(1.0, 6.0)[:, None], block, axis=0)[:N] * np.ones((1, d))
    np.testing.assert_array_equal(O.pool_blocks(x, block), np.arange(1.0, 6.0)[:, None] * np.ones(d))


@pytest.mark.parametrize("n,s,want", [(8, 0.75, 2), (1182, 0.9, 118), (512, 0.9, 51),
                                      (1182, 0.8, 236), (1182, 0.95, 59), (591, 0.9, 59),
                                      (591, 0.8, 118), (591, 0.95, 30), (7, 0.0, 7),
                                      (10, 0.99, 1), (4, 0.5, 2)])
def test_keep_blocks(n, s, want):
    assert O.keep_blocks(n, s) == want


def _check_topk_property(scores, idx, keep):
    for I in range(scores.shape[0]):
        sel = idx[I]
        assert len(sel) == keep and np.all(np.diff(sel) > 0)
        mask = np.zeros(scores.shape[1], bool)
        mask[sel] = True
        if mask.all():
            continue
        lo, hi = scores[I, mask].min(), scores[I, ~mask].max()
        assert lo >= hi
        tied = np.flatnonzero(scores[I] == lo)
        # among blocks tied at the threshold, the chosen ones are the lowest indices
        chosen = tied[mask[tied]]
        assert np.array_equal(chosen, tied[: chosen.size])


def test_select_is_topk_with_lower_index_ties():
    rng = np.random.default_rng(0)
    scores = rng.integers(0, 5, size=(50, 37)).astype(np.float64)   # many exact ties
    for keep in (1, 3, 10, 36, 37):
        _check_topk_property(scores, O.select_blocks(scores, keep), keep)


def test_select_matches_exhaustive_search():
    """Brute force over all subsets: the kept set has the largest score sum and, among those, the
    lexicographically smallest index tuple (the lower-index tie rule)."""
    rng = np.random.default_rng(1)
    for _ in range(40):
        nb, keep = 7, int(rng.integers(1, 7))
        s = rng.integers(0, 4, size=nb).astype(np.float64)
        best = min(itertools.combinations(range(nb), keep), key=lambda c: (-sum(s[list(c)]), c))
        np.testing.assert_array_equal(O.select_blocks(s[None, :], keep)[0], best)


def test_exact_tie_from_duplicated_key_block_goes_to_lower_index():
    rng = np.random.default_rng(2)
    block, nb, d = 4, 6, 8
    q = rng.standard_normal((block * nb, d))
    k = rng.standard_normal((block * nb, d))
    k[4 * block:5 * block] = k[1 * block:2 * block]            # key block 4 duplicates block 1
    qbar, kbar = O.pool_blocks(q, block), O.pool_blocks(k, block)
    s = O.block_scores(qbar, kbar)
    for I in range(nb):
        rank = np.argsort(-s[I], kind="stable")
        keep = int(np.flatnonzero(rank == 1)[0]) + 1            # boundary falls on the tied pair
        sel = O.select_blocks(s[I:I + 1], keep)[0]
        assert 1 in sel and 4 not in sel


def test_keep_all_selects_every_block():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((9, 9))
    np.testing.assert_array_equal(O.select_blocks(s, 9), np.tile(np.arange(9), (9, 1)))


@pytest.mark.parametrize("N,block,s", [(256, 32, 0.75), (32760, 64, 0.9), (75600, 64, 0.9),
                                       (75600, 128, 0.95), (100, 32, 0.5)])
def test_mask_density_equals_sparsity(N, block, s):
    """Every row keeps exactly `keep` blocks, so the block-level density misses the stated sparsity
    by at most half a block; the tiny workload (8 blocks, keep 2) hits 75 % exactly."""
    nb = O.num_blocks(N, block)
    keep = O.keep_blocks(nb, s)
    rng = np.random.default_rng(4)
    idx = O.select_blocks(rng.standard_normal((min(nb, 16), nb)), keep)
    assert all(len(set(row)) == keep for row in idx)
    assert abs((1.0 - keep / nb) - s) <= 0.5 / nb + 1e-12
    if (N, block, s) == (256, 32, 0.75):
        assert 1.0 - keep / nb == 0.75


def _tiny(grid, split, seed):
    rng = np.random.default_rng(seed)
    N, d = int(np.prod(grid)), sum(split)
    return rng.standard_normal((N, d)), rng.standard_normal((N, d)), rng.standard_normal((N, d))


@pytest.mark.parametrize("grid,block", [((2, 4, 4), 8), ((3, 3, 5), 8), ((4, 8, 8), 32)])
def test_dense_limit_equals_library_sdpa(grid, block):
    """keep = n_blocks: the sparse branch is plain softmax attention (torch SDPA, fp64, CPU)."""
    split = (28, 18, 18)
    qn, kn, v = _tiny(grid, split, 5)
    cos, sin = O.rope_tables(*grid, split)
    qr, kr = O.rotate(qn, cos, sin), O.rotate(kn, cos, sin)
    nb = O.num_blocks(qr.shape[0], block)
    idx = np.tile(np.arange(nb), (nb, 1))
    got = O.sparse_attention(qr, kr, v, idx, block, 1.0 / math.sqrt(64))
    np.testing.assert_allclose(got, P.sdpa_f64(qr, kr, v), atol=1e-12)


@pytest.mark.parametrize("grid,block,s", [((2, 4, 4), 8, 0.5), ((3, 3, 5), 8, 0.6),
                                          ((4, 8, 8), 32, 0.75)])
def test_block_sparse_equals_bruteforce_masked_softmax(grid, block, s):
    """Full N x N rotary scores from explicit rotation matrices, a token mask expanded from the block
    list, masked softmax: equals the oracle's per-block gather, including a partial last block."""
    split = (28, 18, 18)
    qn, kn, v = _tiny(grid, split, 6)
    N = qn.shape[0]
    pos = P.positions(grid)
    R = [P.rotation(split, p) for p in pos]
    qr = np.stack([R[n] @ qn[n] for n in range(N)])
    kr = np.stack([R[n] @ kn[n] for n in range(N)])
    nb = O.num_blocks(N, block)
    keep = O.keep_blocks(nb, s)
    idx = O.select_blocks(O.block_scores(O.pool_blocks(qr, block), O.pool_blocks(kr, block)), keep)
    mask = np.zeros((N, N), bool)
    for p in range(N):
        for J in idx[p // block]:
            mask[p, J * block: min(N, (J + 1) * block)] = True
    S = np.where(mask, qr @ kr.T / 8.0, -np.inf)
    W = np.exp(S - S.max(axis=1, keepdims=True))
    want = (W / W.sum(axis=1, keepdims=True)) @ v
    got = O.sparse_attention(qr, kr, v, idx, block, 1.0 / 8.0)
    np.testing.assert_allclose(got, want, atol=1e-12)
    rows = np.array([0, N // 2, N - 1])
    np.testing.assert_allclose(O.sparse_attention_rows(qr, kr, v, idx, block, 1.0 / 8.0, rows),
                               want[rows], atol=1e-12)


def test_sparse_attention_blocks_is_the_restriction():
    """The block-wise form used for sampled parity rows equals the whole-head form on those blocks,
    a partial last block included."""
    rng = np.random.default_rng(9)
    block, N, d = 8, 8 * 5 + 3, 6
    qr, kr, v = (rng.standard_normal((N, d)) for _ in range(3))
    nb = O.num_blocks(N, block)
    idx = np.stack([np.sort(rng.choice(nb, 3, replace=False)) for _ in range(nb)])
    full = O.sparse_attention(qr, kr, v, idx, block, 0.4)
    blocks = [1, 3, 5]
    rows = np.concatenate([np.arange(I * block, min(N, (I + 1) * block)) for I in blocks])
    np.testing.assert_allclose(O.sparse_attention_blocks(qr, kr, v, idx, block, 0.4, blocks),
                               full[rows], rtol=0, atol=1e-14)
