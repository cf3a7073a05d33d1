"""Pins of the oracle's rotary low-rank branch and gated fusion (eq. qklr, eq. ctx, eq. gate; Prop.
exact, Prop. truncation-bound, Prop. inside; Table "mechanism"; appendix "Computational Complexity")."""

import math
import os

import numpy as np
import pytest

import oracle as O
from tests import _pins as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _content(N, d, r, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((N, d)), rng.standard_normal((N, d)), rng.standard_normal((N, d)),
            rng.standard_normal((r, d)) / math.sqrt(d), rng.standard_normal((r, d)) / math.sqrt(d))


@pytest.mark.parametrize("split,r", [((28, 18, 18), 16), ((28, 18, 18), 64), ((44, 42, 42), 32),
                                     ((44, 42, 42), 128)])
def test_readout_equals_relative_bruteforce(split, r):
    """Prop. exact: q~_p . k~_q = phi(q_p)^T R_r(q - p) psi(k_q). Summing that O(N^2) relative form
    against v (position-free features, explicit exp(generator) rotations) must equal the summary-then-
    readout path q~_p^T C."""
    grid = (2, 3, 4)
    N, d = int(np.prod(grid)), sum(split)
    qn, kn, v, Pq, Pk = _content(N, d, r, 0)
    cos, sin = O.rope_tables(*grid, split)
    C, z = O.lowrank_summary(kn, v, Pk, cos, sin)
    got = O.lowrank_readout_u(qn, Pq, cos, sin, C)
    phi, psi = P.silu_ref(qn @ Pq.T), P.silu_ref(kn @ Pk.T)
    pos = P.positions(grid)
    want = np.zeros((N, d))
    for p in range(N):
        for q in range(N):
            want[p] += (phi[p] @ P.rotation(split, pos[q] - pos[p], r=r) @ psi[q]) * v[q]
    np.testing.assert_allclose(got, want, atol=1e-10)
    # z is the summary of an all-ones value column
    np.testing.assert_allclose(z, O.lowrank_summary(kn, np.ones((N, 1)), Pk, cos, sin)[0][:, 0],
                               atol=1e-12)


def test_whole_module_is_shift_invariant():
    """Translating every position by delta leaves selection, both branches and the fused output
    unchanged (co-rotation of pooled Q/K; C' = R_r(delta) C). The inside-activation ordering is the
    negative control: its readout moves."""
    grid, split, r = (4, 8, 8), (28, 18, 18), 16
    N = 256
    rng = np.random.default_rng(1)
    Qn, Kn, V = (rng.standard_normal((1, 2, N, 64)) for _ in range(3))
    Pq, Pk = (rng.standard_normal((2, r, 64)) / 8.0 for _ in range(2))
    logits = -1.946 + 0.5 * rng.standard_normal((1, N))
    kw = dict(grid=grid, split=split, block=32, sparsity=0.75, dtype="f64")
    base = O.forward(Qn, Kn, V, Pq, Pk, logits, **kw)
    for delta in [(3, -5, 7), (1000, 1000, 1000)]:
        moved = O.forward(Qn, Kn, V, Pq, Pk, logits, offset=delta, **kw)
        np.testing.assert_array_equal(moved["idx"], base["idx"])
        for key in ("scores", "o_s", "u", "o_lr", "out"):
            np.testing.assert_allclose(moved[key], base[key], atol=1e-10, err_msg=key)
        Rd = P.rotation(split, np.asarray(delta, float), r=r)
        np.testing.assert_allclose(moved["C"][0, 0], Rd @ base["C"][0, 0], atol=1e-9)
    # negative control: inside-activation features give a different readout after the same shift
    cos0, sin0 = O.rope_tables(*grid, split)
    cos1, sin1 = O.rope_tables(*grid, split, offset=(3, -5, 7))
    def inside_u(cos, sin):
        C = O.features(Kn[0, 0], Pk[0], cos, sin, "silu", "inside").T @ V[0, 0]
        return O.features(Qn[0, 0], Pq[0], cos, sin, "silu", "inside") @ C
    assert np.abs(inside_u(cos0, sin0) - inside_u(cos1, sin1)).max() > 1e-3


def test_mechanism_table_qualitative():
    """Table "mechanism": no RoPE gives exactly zero shift residual and zero offset range; outside
    keeps a non-trivial offset dependence with a vanishing shift residual; inside leaks position."""
    rows = {r[0]: (float(r[1]), float(r[2])) for r in _golden("mechanism_table.txt")}
    rng = np.random.default_rng(2)
    split, r = (44, 42, 42), 64
    Pq, Pk = (rng.standard_normal((r, 128)) / math.sqrt(128) for _ in range(2))
    res = {}
    for ordering in ("none", "inside", "outside"):
        shift, rng_off = [], []
        for _ in range(8):
            qv, kv = rng.standard_normal(128), rng.standard_normal(128)
            p, q = np.array([2.0, 10, 20]), np.array([7.0, 10, 20])
            s0 = O.lowrank_logit(qv, kv, Pq, Pk, p, q, split, ordering=ordering)
            for delta in (np.array([5.0, 0, 0]), np.array([3.0, 7, -4])):
                s1 = O.lowrank_logit(qv, kv, Pq, Pk, p + delta, q + delta, split, ordering=ordering)
                shift.append(abs(s1 - s0))
            offs = [O.lowrank_logit(qv, kv, Pq, Pk, p, p + np.array([dt, 0, 0]), split,
                                    ordering=ordering) for dt in range(-10, 11)]
            rng_off.append(max(offs) - min(offs))
        res[ordering] = (max(shift), min(rng_off))
    assert res["none"] == (0.0, 0.0) == rows["none"]
    assert res["outside"][0] < 1e-10 and res["outside"][1] > 1e-3
    assert res["inside"][0] > 1e-3 and res["inside"][1] > 1e-3
    assert rows["outside"][0] < rows["inside"][0]


@pytest.mark.parametrize("dtype", ["f64"])
def test_full_rank_identity_projection_closed_form(dtype):
    """r = d_h, P_q = P_k = I and 0 % sparsity: O^s is dense softmax attention (torch SDPA) and
    O = SDPA + g r_s u / rms(u) with u_p = sum_q SiLU(q_p)^T R(q - p) SiLU(k_q) v_q. A gate logit of
    -800 (g = 0 in fp64) leaves exactly the dense attention."""
    grid, split = (2, 2, 4), (28, 18, 18)
    N, d = 16, 64
    rng = np.random.default_rng(3)
    Qn, Kn, V = (rng.standard_normal((1, 1, N, d)) for _ in range(3))
    I = np.eye(d)[None]
    logits = -1.946 + 0.5 * rng.standard_normal((1, N))
    res = O.forward(Qn, Kn, V, I, I, logits, grid=grid, split=split, block=4, sparsity=0.0,
                    dtype=dtype)
    pos = P.positions(grid)
    R = [P.rotation(split, p) for p in pos]
    qr = np.stack([R[n] @ Qn[0, 0, n] for n in range(N)])
    kr = np.stack([R[n] @ Kn[0, 0, n] for n in range(N)])
    dense = P.sdpa_f64(qr, kr, V[0, 0])
    phi, psi = P.silu_ref(Qn[0, 0]), P.silu_ref(Kn[0, 0])
    u = np.zeros((N, d))
    for p in range(N):
        for q in range(N):
            u[p] += (phi[p] @ P.rotation(split, pos[q] - pos[p]) @ psi[q]) * V[0, 0, q]
    g = 1.0 / (1.0 + np.exp(-logits[0]))
    rs = np.sqrt(np.mean(dense ** 2, axis=1) + 1e-6)
    want = dense + (g * rs)[:, None] * u / np.sqrt(np.mean(u ** 2, axis=1, keepdims=True) + 1e-6)
    np.testing.assert_allclose(res["o_s"][0, 0], dense, atol=1e-12)
    np.testing.assert_allclose(res["u"][0, 0], u, atol=1e-9)
    np.testing.assert_allclose(res["out"][0, 0], want, atol=1e-10)
    closed = O.forward(Qn, Kn, V, I, I, np.full((1, N), -800.0), grid=grid, split=split, block=4,
                       sparsity=0.0, dtype=dtype)
    np.testing.assert_allclose(closed["out"][0, 0], dense, atol=1e-12)


@pytest.mark.parametrize("r", [16, 32, 64])
def test_truncation_bound(r):
    """Prop. truncation-bound, nested setting: |s_full - s_r| <= ||Phi_{>r}|| ||Psi_{>r}|| for every
    pair, with s_r from the oracle's truncated rotation and s_full from explicit full rotations."""
    split, grid = (44, 42, 42), (3, 3, 3)
    N = 27
    rng = np.random.default_rng(4)
    Phi, Psi = rng.standard_normal((N, 128)), rng.standard_normal((N, 128))
    Phi[:, r:] *= 0.05
    Psi[:, r:] *= 0.05
    cos, sin = O.rope_tables(*grid, split)
    a, b = O.rotate(Phi[:, :r], cos, sin), O.rotate(Psi[:, :r], cos, sin)
    s_r = a @ b.T
    pos = P.positions(grid)
    for p in range(0, N, 4):
        for q in range(N):
            s_full = Phi[p] @ P.rotation(split, pos[q] - pos[p]) @ Psi[q]
            bound = np.linalg.norm(Phi[p, r:]) * np.linalg.norm(Psi[q, r:])
            assert abs(s_full - s_r[p, q]) <= bound + 1e-12


def test_readout_rms_and_value_scale_invariance():
    grid, split, r = (2, 4, 4), (28, 18, 18), 16
    N = 32
    qn, kn, v, Pq, Pk = _content(N, 64, r, 5)
    cos, sin = O.rope_tables(*grid, split)
    C, _ = O.lowrank_summary(kn, v, Pk, cos, sin)
    u = O.lowrank_readout_u(qn, Pq, cos, sin, C)
    olr = O.lowrank_readout(qn, Pq, cos, sin, C, 1e-6)
    ms = np.mean(u * u, axis=1)
    np.testing.assert_allclose(np.sqrt(np.mean(olr ** 2, axis=1)), np.sqrt(ms / (ms + 1e-6)),
                               rtol=1e-12)
    C3, _ = O.lowrank_summary(kn, 3.0 * v, Pk, cos, sin)
    np.testing.assert_allclose(O.lowrank_readout(qn, Pq, cos, sin, C3, 0.0),
                               O.lowrank_readout(qn, Pq, cos, sin, C, 0.0), atol=1e-12)


def test_silu_golden_derivatives():
    """SiLU(0) = 0, SiLU'(0) = 1/2, SiLU''(0) = 1/2 as printed in the proof of Prop. inside."""
    vals = {r[0]: float(r[1]) for r in _golden("silu_derivatives.txt")}
    h = 1e-4
    f = lambda x: float(O.silu(np.array([x]))[0])
    assert f(0.0) == vals["silu(0)"]
    assert abs((f(h) - f(-h)) / (2 * h) - vals["silu'(0)"]) < 1e-8
    assert abs((f(h) - 2 * f(0.0) + f(-h)) / h ** 2 - vals["silu''(0)"]) < 1e-6
    x = np.linspace(-800, 800, 4001)
    y = O.silu(x)
    assert np.all(np.isfinite(y)) and y[0] == 0.0 and y[-1] == 800.0
    assert np.all(y >= -0.2785) and np.all(np.diff(y[x > 0]) > 0)   # SiLU min is about -0.2785


def test_combine_special_cases():
    """eq. gate: a closed gate or a zero low-rank output leaves O^s; the literal form equals
    O^s + g r O^lr."""
    rng = np.random.default_rng(6)
    os_, olr = rng.standard_normal((20, 64)), rng.standard_normal((20, 64))
    logits = rng.standard_normal(20)
    np.testing.assert_allclose(O.combine(os_, olr, np.full(20, -800.0)), os_, rtol=1e-14)
    np.testing.assert_allclose(O.combine(os_, 0 * olr, logits), os_, rtol=1e-14)
    g = 1.0 / (1.0 + np.exp(-logits))
    r = np.sqrt(np.mean(os_ ** 2, axis=1) + 1e-6)
    np.testing.assert_allclose(O.combine(os_, olr, logits), os_ + (g * r)[:, None] * olr,
                               rtol=1e-13, atol=1e-14)
    assert O.gate(np.array([0.0]))[0] == 0.5
    np.testing.assert_allclose(O.gate(logits) + O.gate(-logits), 1.0, rtol=1e-15)


def test_flop_accounting_matches_simplified_forms():
    for row in _golden("complexity.txt"):
        B, H, L, d, r = (int(x) for x in row[:5])
        S = float(row[5])
        f = O.flop_counts(B, H, L, d, r, S)
        assert abs(f["eta"] - (2 * r + 0.5) / (L * (1 - S))) < 1e-12 * f["eta"]
        assert abs(f["lowrank"] / (4.0 * B * H * L * d * d) - 2.0 * r / d) < 1e-15


# ---- feature-map and rotation-order variants (Sec. 5.1 RoPE placement, Sec. 5.3 activation
# ablation, Prop. exact, Prop. inside) -------------------------------------------------------------

PHIS = ("silu", "identity", "tanh", "relu", "gelu")


def test_activation_golden_values():
    """Each feature map at points whose value is fixed by its definition (tests/golden)."""
    for phi, x, want in _golden("activations.txt"):
        got = O.activation(np.array([float(x)]), phi)[0]
        assert got == pytest.approx(float(want), abs=1e-14), (phi, x)


def test_activation_odd_parts():
    """sigma(x) + sigma(-x) = 1 and Phi(x) + Phi(-x) = 1 give f(x) - f(-x) = x for SiLU and GELU; ReLU
    also gives x; tanh is odd; identity gives 2x. Checks signs and dropped terms on a grid."""
    x = np.linspace(-6, 6, 241)
    odd = {"silu": x, "gelu": x, "relu": x, "identity": 2 * x, "tanh": 0 * x}
    for phi in PHIS:
        f = O.activation(x, phi)
        np.testing.assert_allclose(f - O.activation(-x, phi) if phi != "tanh" else f + O.activation(-x, phi),
                                   odd[phi], atol=1e-13, err_msg=phi)
        np.testing.assert_allclose(f, P.activation_ref(x, phi), atol=1e-13, err_msg=phi)


@pytest.mark.parametrize("phi", PHIS)
def test_variant_readout_equals_relative_bruteforce(phi):
    """Prop. exact holds for any position-free feature map: with the rotation outside, the
    summary-then-readout path equals the O(N^2) relative form sum_q phi(P_q q_p)^T R_r(q - p)
    phi(P_k k_q) v_q (explicit rotations, activation written independently)."""
    grid, split, r = (2, 3, 4), (28, 18, 18), 16
    N, d = int(np.prod(grid)), sum(split)
    qn, kn, v, Pq, Pk = _content(N, d, r, 5)
    cos, sin = O.rope_tables(*grid, split)
    C, _ = O.lowrank_summary(kn, v, Pk, cos, sin, phi=phi)
    got = O.lowrank_readout_u(qn, Pq, cos, sin, C, phi=phi)
    fq, fk = P.activation_ref(qn @ Pq.T, phi), P.activation_ref(kn @ Pk.T, phi)
    pos = P.positions(grid)
    want = np.zeros((N, d))
    for p in range(N):
        for q in range(N):
            want[p] += (fq[p] @ P.rotation(split, pos[q] - pos[p], r=r) @ fk[q]) * v[q]
    np.testing.assert_allclose(got, want, atol=1e-10)


def test_inside_and_none_orderings_closed_forms():
    """Inside: phi(R_r(p) P x) written with explicit rotation matrices. Identity commutes with the
    rotation, so inside and outside coincide for it. None: phi(P x) with no position at all."""
    grid, split, r = (2, 3, 4), (28, 18, 18), 16
    N, d = int(np.prod(grid)), sum(split)
    x, _, _, Pm, _ = _content(N, d, r, 6)
    cos, sin = O.rope_tables(*grid, split)
    pos = P.positions(grid)
    for phi in PHIS:
        want = np.stack([P.activation_ref(P.rotation(split, pos[n], r=r) @ (Pm @ x[n]), phi)
                         for n in range(N)])
        np.testing.assert_allclose(O.features(x, Pm, cos, sin, phi, "inside"), want, atol=1e-12)
        np.testing.assert_allclose(O.features(x, Pm, cos, sin, phi, "none"),
                                   P.activation_ref(x @ Pm.T, phi), atol=1e-12)
    np.testing.assert_allclose(O.features(x, Pm, cos, sin, "identity", "inside"),
                               O.features(x, Pm, cos, sin, "identity", "outside"), atol=1e-12)


def test_shift_residual_by_phi_and_ordering():
    """The Sec. 5.1 criterion for every feature map: with the rotation outside the logit depends on
    the offset only (shift residual ~ 0, offset range > 0, Prop. exact); inside, every nonlinear map
    leaks absolute position (Prop. inside) while the identity map does not; without rotation the
    logit is position-blind (both exactly 0)."""
    rng = np.random.default_rng(7)
    split, r = (44, 42, 42), 32
    Pq, Pk = (rng.standard_normal((r, 128)) / math.sqrt(128) for _ in range(2))
    qv, kv = rng.standard_normal(128), rng.standard_normal(128)
    p, q = np.array([2.0, 10, 20]), np.array([7.0, 10, 20])
    for phi in PHIS:
        for ordering in ("outside", "inside", "none"):
            s0 = O.lowrank_logit(qv, kv, Pq, Pk, p, q, split, ordering=ordering, phi=phi)
            res = max(abs(O.lowrank_logit(qv, kv, Pq, Pk, p + dl, q + dl, split, ordering=ordering,
                                          phi=phi) - s0)
                      for dl in (np.array([5.0, 0, 0]), np.array([11.0, 0, 0])))
            offs = [O.lowrank_logit(qv, kv, Pq, Pk, p, p + np.array([dt, 0, 0]), split,
                                    ordering=ordering, phi=phi) for dt in range(-8, 9)]
            span = max(offs) - min(offs)
            if ordering == "none":
                assert res == 0.0 and span == 0.0, phi
            elif ordering == "outside" or phi == "identity":
                assert res < 1e-10 and span > 1e-3, (phi, ordering, res, span)
            else:
                assert res > 1e-4 and span > 1e-3, (phi, ordering, res, span)


def test_gate_logits_closed_forms():
    """Sec. 4.4 / Algorithm step 8: X W_g + b_g. One-hot hidden states pick one weight; constant
    states give c * sum(W_g) + b_g; at the paper's initialisation (W_g = 0, b_g = b_0 = -1.946 of Tab.
    hyper) every logit is b_0 and the gate is sigma(b_0) = 0.125 (b_0 = -ln 7 to four digits)."""
    rng = np.random.default_rng(8)
    dm = 24
    Wg = rng.standard_normal(dm)
    eye = np.eye(dm)
    np.testing.assert_allclose(O.gate_logits(eye, Wg, 0.5), Wg + 0.5, atol=1e-15)
    np.testing.assert_allclose(O.gate_logits(np.full((3, dm), 2.0), Wg, -1.0), 2.0 * Wg.sum() - 1.0,
                               atol=1e-12)
    X = rng.standard_normal((5, 7, dm))
    b0 = -1.946
    np.testing.assert_array_equal(O.gate_logits(X, np.zeros(dm), b0), np.full((5, 7), b0))
    assert O.gate(np.array([b0]))[0] == pytest.approx(0.125, abs=1e-5)
