"""GPU parity of the backward pass (fine-tuning, Sec. 4.5) against the gradient oracle (fp64 autograd
of the forward definitions, pinned by finite differences): the forward's log-sum-exp, and the
gradients of the block-sparse attention for fixed block lists."""

import math

import numpy as np
import pytest
import torch

import oracle as O
from oracle import rola_grad as G
from paper_2609_06712_amd import synth

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_06712_amd import rola as R  # noqa: E402
from tests import _parity as T  # noqa: E402


def _f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def _rel(got, want):
    return float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))


@pytest.mark.parametrize("grid,block,s,B", [((3, 10, 13), 64, 0.5, 1), ((3, 10, 13), 128, 0.5, 1),
                                            ((2, 9, 20), 64, 0.7, 2), ((4, 8, 16), 64, 0.0, 1)],
                         ids=["ragged-b64", "ragged-b128", "batch2", "keep-all"])
def test_sparse_backward(grid, block, s, B):
    w = synth.WAN_1_3B_480P.replace(grid=grid, H=2, B=B, block=block, sparsity=s)
    inp = synth.make_inputs(w, 7)
    d = {k: v.cuda() for k, v in inp.items()}
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(d["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(d["Kn"], cos, sin, g)
    idx = R.rola_block_select(qr, kr, g, block, s)
    os_, lse = R.rola_sparse_attn_lse(qr, kr, d["V"], g, block, s, idx)
    ref_os = R.rola_sparse_attn(qr, kr, d["V"], g, block, s, idx, share=False)
    gen = torch.Generator().manual_seed(3)
    dos = torch.randn(qr.shape, generator=gen).to(torch.bfloat16).cuda()
    dq, dk, dv = R.rola_sparse_attn_backward(qr, kr, d["V"], g, block, s, idx, os_, lse, dos)
    torch.cuda.synchronize()
    assert torch.equal(os_, ref_os)  # the lse variant computes the same O^s
    scale = 1.0 / math.sqrt(w.d_h)
    for b in range(w.B):
        for h in range(w.H):
            q, k, v = _f64(qr[b, h]), _f64(kr[b, h]), _f64(d["V"][b, h])
            ix = idx[b, h].cpu().numpy()
            # lse (log2 units) from its definition over the selected keys
            mask = np.zeros((w.N, w.N), bool)
            blk = np.arange(w.N) // block
            sel = np.zeros((ix.shape[0], ix.shape[0]), bool)
            sel[np.arange(ix.shape[0])[:, None], ix] = True
            mask = sel[blk[:, None], blk[None, :]]
            sc = np.where(mask, q @ k.T * scale, -np.inf)
            mx = sc.max(1, keepdims=True)
            lse_ref = (mx[:, 0] + np.log(np.exp(sc - mx).sum(1))) / math.log(2)
            # the forward's denominator sums the bf16-rounded probabilities that enter P V (relative
            # error <= 2^-9), so its log2 is within 2^-9 / ln 2 = 2.8e-3 of the exact one
            np.testing.assert_allclose(_f64(lse[b, h]), lse_ref, rtol=0, atol=2.9e-3)
            want = G.sparse_attention_grads(q, k, v, ix, block, scale, _f64(dos[b, h]))
            errs = {n: _rel(_f64(t[b, h]), want[n]) for n, t in (("dqr", dq), ("dkr", dk), ("dv", dv))}
            print(f"[parity] sparse backward grid {grid} block {block} s {s} b{b} h{h}: " +
                  ", ".join(f"{n} rel {e:.2e}" for n, e in errs.items()), flush=True)
            for n, e in errs.items():
                assert e <= 1e-2, (n, e)
            # shifting all keys leaves O^s unchanged: the key gradients sum to zero
            colsum = np.abs(_f64(dk[b, h]).sum(0)).max()
            assert colsum <= 1e-2 * np.abs(_f64(dk[b, h])).sum(0).max() + 1e-6
