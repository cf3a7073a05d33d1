"""Pins of the gradient oracle (oracle/rola_grad.py, torch fp64 autograd of a transcription of the
forward): directional derivatives against central finite differences of the numpy oracle's own
forward functions (an independent implementation), plus identities the gradients must satisfy."""

import math

import numpy as np
import pytest

import oracle as O
from oracle import rola_grad as G

GRID, SPLIT, BLOCK, R = (2, 4, 6), (28, 18, 18), 16, 16  # N = 48, d = 64, three blocks


def _setup(seed):
    rng = np.random.default_rng(seed)
    N, d = int(np.prod(GRID)), sum(SPLIT)
    qn, kn, v = (rng.standard_normal((N, d)) for _ in range(3))
    Pq, Pk = (rng.standard_normal((R, d)) / math.sqrt(d) for _ in range(2))
    logits = -1.0 + 0.5 * rng.standard_normal(N)
    cos, sin = O.rope_tables(*GRID, SPLIT)
    idx = np.array([[0, 2], [1, 2], [0, 1]])  # a fixed selection, keep 2 of 3
    dout = rng.standard_normal((N, d))
    return dict(qn=qn, kn=kn, v=v, Pq=Pq, Pk=Pk, logits=logits, cos=cos, sin=sin, idx=idx,
                dout=dout, rng=rng)


def _numpy_module(s, qn, kn, v, Pq, Pk, logits):
    """The numpy oracle's forward steps composed with the fixed block list."""
    scale = 1.0 / math.sqrt(qn.shape[1])
    os_ = O.sparse_attention(O.rotate(qn, s["cos"], s["sin"]), O.rotate(kn, s["cos"], s["sin"]), v,
                             s["idx"], BLOCK, scale)
    C, _ = O.lowrank_summary(kn, v, Pk, s["cos"], s["sin"])
    u = O.lowrank_readout_u(qn, Pq, s["cos"], s["sin"], C)
    return O.combine(os_, O.rms_normalize(u, 1e-6), logits, 1e-6)


def _fd(f, args, name, delta, h=1e-5):
    plus, minus = dict(args), dict(args)
    plus[name] = args[name] + h * delta
    minus[name] = args[name] - h * delta
    return (f(**plus) - f(**minus)) / (2 * h)


@pytest.mark.parametrize("seed", [0, 1])
def test_module_grads_match_finite_differences(seed):
    s = _setup(seed)
    names = ("qn", "kn", "v", "Pq", "Pk", "logits")
    args = {n: s[n] for n in names}
    g = G.module_grads(*(s[n] for n in names), s["cos"], s["sin"], s["idx"], BLOCK, s["dout"])
    f = lambda **a: float((s["dout"] * _numpy_module(s, **a)).sum())  # noqa: E731
    for n in names:
        delta = s["rng"].standard_normal(args[n].shape)
        want = _fd(f, args, n, delta)
        got = float((g["d" + n] * delta).sum())
        assert got == pytest.approx(want, rel=1e-6, abs=1e-8), n


def test_sparse_grads_match_finite_differences_and_key_shift_identity():
    s = _setup(2)
    scale = 1.0 / math.sqrt(64)
    qr, kr = O.rotate(s["qn"], s["cos"], s["sin"]), O.rotate(s["kn"], s["cos"], s["sin"])
    g = G.sparse_attention_grads(qr, kr, s["v"], s["idx"], BLOCK, scale, s["dout"])
    f = lambda qr, kr, v: float((s["dout"] * O.sparse_attention(qr, kr, v, s["idx"], BLOCK, scale)).sum())  # noqa: E731,E501
    args = dict(qr=qr, kr=kr, v=s["v"])
    for n, gn in (("qr", "dqr"), ("kr", "dkr"), ("v", "dv")):
        delta = s["rng"].standard_normal(args[n].shape)
        assert float((g[gn] * delta).sum()) == pytest.approx(_fd(f, args, n, delta), rel=1e-6, abs=1e-8)
    # shifting every key by one vector shifts each row's scores by a constant: the output does not
    # move, so the key gradients sum to zero; V enters linearly: <dV, V> = <dout, O^s>
    np.testing.assert_allclose(g["dkr"].sum(axis=0), 0.0, atol=1e-10)
    os_ = O.sparse_attention(qr, kr, s["v"], s["idx"], BLOCK, scale)
    assert float((g["dv"] * s["v"]).sum()) == pytest.approx(float((s["dout"] * os_).sum()), rel=1e-10)


def test_lowrank_combine_grads_match_finite_differences():
    s = _setup(3)
    os_ = s["rng"].standard_normal(s["qn"].shape)
    names = ("qn", "kn", "v", "Pq", "Pk", "os_", "logits")
    args = {n: (os_ if n == "os_" else s[n]) for n in names}
    g = G.lowrank_combine_grads(*(args[n] for n in names), s["cos"], s["sin"], s["dout"])

    def f(qn, kn, v, Pq, Pk, os_, logits):
        C, _ = O.lowrank_summary(kn, v, Pk, s["cos"], s["sin"])
        u = O.lowrank_readout_u(qn, Pq, s["cos"], s["sin"], C)
        return float((s["dout"] * O.combine(os_, O.rms_normalize(u, 1e-6), logits, 1e-6)).sum())
    for n, gn in zip(names, ("dqn", "dkn", "dv", "dPq", "dPk", "dos", "dlogits")):
        delta = s["rng"].standard_normal(args[n].shape)
        assert float((g[gn] * delta).sum()) == pytest.approx(_fd(f, args, n, delta), rel=1e-6, abs=1e-8), n


def test_gate_grads_closed_form():
    rng = np.random.default_rng(4)
    X, Wg, dl = rng.standard_normal((7, 24)), rng.standard_normal(24), rng.standard_normal(7)
    g = G.gate_grads(X, Wg, dl)
    np.testing.assert_allclose(g["dX"], np.outer(dl, Wg), atol=1e-14)
    np.testing.assert_allclose(g["dWg"], X.T @ dl, atol=1e-13)
    assert g["dbg"] == pytest.approx(dl.sum(), abs=1e-13)
