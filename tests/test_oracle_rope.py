"""Pins of the oracle's rotary schedule against independent formulations (Sec. 3 3D RoPE and
eq. shiftinv; Sec. 4.2 truncation; appendix "Formal Sanity Checks": orthogonality and group property)."""

import numpy as np
import pytest
import torch

import oracle as O
from tests import _pins as P

SPLITS = [(28, 18, 18), (44, 42, 42), (24, 20, 20)]


def _matrix(split, pos, r=None):
    """R_r(pos) assembled from the oracle's rotate() applied to basis vectors."""
    d = sum(split) if r is None else r
    axis, theta = O.pair_schedule(split)
    ang = np.asarray(pos, dtype=np.float64)[axis] * theta
    cos, sin = np.cos(ang)[None, :], np.sin(ang)[None, :]
    cols = O.rotate(np.eye(d)[:, None, :], cos, sin)[:, 0, :]  # row k = R e_k
    return cols.T


@pytest.mark.parametrize("split", SPLITS)
def test_frequencies_match_logspace(split):
    _, theta = O.pair_schedule(split)
    np.testing.assert_allclose(theta, np.concatenate(P.frequencies(split)), rtol=1e-13)


@pytest.mark.parametrize("split", SPLITS)
def test_rotate_equals_matrix_exponential(split):
    rng = np.random.default_rng(0)
    grid, off = (2, 3, 4), (1, -2, 5)
    d = sum(split)
    cos, sin = O.rope_tables(*grid, split, offset=off)
    x = rng.standard_normal((np.prod(grid), d))
    got = O.rotate(x, cos, sin)
    for n, pos in enumerate(P.positions(grid, off)):
        np.testing.assert_allclose(got[n], P.rotation(split, pos) @ x[n], atol=1e-12)


@pytest.mark.parametrize("split,r", [((28, 18, 18), 16), ((44, 42, 42), 32), ((44, 42, 42), 64),
                                     ((44, 42, 42), 128), ((28, 18, 18), 64)])
def test_truncated_rotation_is_leading_block(split, r):
    """R_r keeps the first r coordinates of the backbone ordering (r/2 complete pairs)."""
    rng = np.random.default_rng(1)
    grid = (3, 2, 2)
    cos, sin = O.rope_tables(*grid, split)
    f = rng.standard_normal((np.prod(grid), r))
    got = O.rotate(f, cos, sin)
    for n, pos in enumerate(P.positions(grid)):
        np.testing.assert_allclose(got[n], P.rotation(split, pos, r=r) @ f[n], atol=1e-12)


@pytest.mark.parametrize("split", SPLITS)
def test_pair0_of_each_axis_turns_by_the_position(split):
    """theta_0 = 1 for every axis, so the first pair of axis a turns by exactly pos_a; pins the axis
    order (t, y, x) and the column offsets."""
    grid = (3, 4, 5)
    cos, sin = O.rope_tables(*grid, split)
    pos = P.positions(grid)
    off = 0
    for a, d_a in enumerate(split):
        np.testing.assert_allclose(cos[:, off], np.cos(pos[:, a]), atol=1e-15)
        np.testing.assert_allclose(sin[:, off], np.sin(pos[:, a]), atol=1e-15)
        off += d_a // 2


@pytest.mark.parametrize("split", SPLITS)
def test_orthogonal_and_group_property(split):
    rng = np.random.default_rng(2)
    for _ in range(5):
        p = rng.integers(-50, 50, size=3)
        q = rng.integers(-50, 50, size=3)
        Rp, Rq, Rqp = _matrix(split, p), _matrix(split, q), _matrix(split, q - p)
        np.testing.assert_allclose(Rp.T @ Rp, np.eye(sum(split)), atol=1e-12)
        np.testing.assert_allclose(Rp.T @ Rq, Rqp, atol=1e-11)
        for r in (16, 32):
            Rp_r, Rq_r, Rqp_r = (_matrix(split, x, r) for x in (p, q, q - p))
            np.testing.assert_allclose(Rp_r.T @ Rq_r, Rqp_r, atol=1e-11)


def test_relative_identity_eq_shiftinv():
    """<R(p) q, R(q) k> = <q, R(q - p) k> (eq. shiftinv)."""
    rng = np.random.default_rng(3)
    split = (44, 42, 42)
    for _ in range(5):
        p, q = rng.integers(0, 80, size=3), rng.integers(0, 80, size=3)
        a, b = rng.standard_normal(128), rng.standard_normal(128)
        lhs = (_matrix(split, p) @ a) @ (_matrix(split, q) @ b)
        rhs = a @ (P.rotation(split, q - p) @ b)
        assert abs(lhs - rhs) < 1e-10 * (1 + abs(rhs))


def test_round_bf16_matches_torch_rne():
    """Rounding to bfloat16 equals torch's fp32 -> bf16 conversion (round to nearest even), including
    exact halfway values."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal(100000).astype(np.float32) * np.float32(3.0)
    # exact midpoints between neighbouring bf16 values: both tie directions
    base = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    bits = base.view(np.uint32)
    mid = ((bits.astype(np.uint64) + 0x8000) & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    allx = np.concatenate([x, mid])
    want = torch.from_numpy(allx).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.round_bf16(allx.astype(np.float64)), want)
