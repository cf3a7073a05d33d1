"""The synthetic DiT block around the module (the context measurement of per-block time): its
plumbing against an fp64 reference, on a small Wan-like shape. Each stage is checked from the GPU's
own inputs to that stage, so bf16 rounding does not compound: the modulated input and the
normalised q, k; the module output against the oracle; the block output after the output
projection, the cross-attention and the MLP."""

import math

import numpy as np
import pytest
import torch

import oracle as O

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_06712_amd import dit_block as DB  # noqa: E402
from tests import _parity as T  # noqa: E402

TINY = DB.DiTShape("tiny", 256, 2, 512, 1, 16, (3, 10, 13))


def _f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def _ln(x, eps=1e-6):
    mu = x.mean(-1, keepdims=True)
    return (x - mu) / np.sqrt(((x - mu) ** 2).mean(-1, keepdims=True) + eps)


def _rms(x, w, eps=1e-6):
    return x / np.sqrt((x * x).mean(-1, keepdims=True) + eps) * w


def _gelu_tanh(x):
    return 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))


def _rel(got, want):
    return float(np.linalg.norm(got - want) / np.linalg.norm(want))


@pytest.mark.parametrize("attn", ["rola", "dense"])
def test_dit_block_plumbing(attn):
    blk = DB.DiTBlock(TINY, attn=attn, block=64, sparsity=0.5, r=32, seed=3)
    x, ctx = DB.inputs(TINY, seed=4)
    cap = {}
    out = blk.forward(x, ctx, capture=cap)
    torch.cuda.synchronize()
    W = {k: _f64(getattr(blk, k)) for k in ("Wqkv", "bqkv", "Wo", "bo", "nq", "nk", "Wcq", "Wck",
                                              "Wcv", "Wco", "ncq", "nck", "W1", "b1", "W2", "b2",
                                              "mod", "Pq", "Pk")}
    sh1, sc1, g1, sh2, sc2, g2 = W["mod"]
    d, H, N = TINY.d_model, TINY.heads, int(np.prod(TINY.grid))
    xf, cf = _f64(x), _f64(ctx)
    # modulated input, then q, k from the GPU's h
    h_ref = _ln(xf) * (1 + sc1) + sh1
    assert _rel(_f64(cap["h"]), h_ref) < 1e-2
    hq = _f64(cap["h"]) @ W["Wqkv"].T + W["bqkv"]
    heads = lambda t: t.reshape(N, H, 128).transpose(1, 0, 2)  # noqa: E731
    assert _rel(_f64(cap["qn"])[0], heads(_rms(hq[:, :d], W["nq"]))) < 1e-2
    assert _rel(_f64(cap["kn"])[0], heads(_rms(hq[:, d:2 * d], W["nk"]))) < 1e-2
    # the module from the GPU's own Q^n, K^n, V (and gate logits)
    qn, kn, v = _f64(cap["qn"]), _f64(cap["kn"]), _f64(cap["v"])
    if attn == "rola":
        lg = _f64(cap["logits"])
        assert np.all(lg == np.float32(-1.946))  # W_g = 0 (the paper's init): every logit is b_g
        ora = O.forward(qn, kn, v, W["Pq"], W["Pk"], lg, grid=TINY.grid, split=TINY.split,
                        block=64, sparsity=0.5, dtype="bf16")
        want = ora["out"]
    else:
        cos, sin = O.rope_tables(*TINY.grid, TINY.split)
        nb = O.num_blocks(N, 64)
        want = np.stack([O.sparse_attention(O.round_to(O.rotate(qn[0, h], cos, sin), "bf16"),
                                            O.round_to(O.rotate(kn[0, h], cos, sin), "bf16"),
                                            v[0, h], np.tile(np.arange(nb), (nb, 1)), 64,
                                            1 / math.sqrt(128)) for h in range(H)])[None]
    for h in range(H):
        T.assert_close(_f64(cap["o"])[0, h], want[0, h], "bf16", f"module output h{h}")
    # the rest of the block from the GPU's module output
    a = _f64(cap["o"])[0].transpose(1, 0, 2).reshape(N, d)
    x1 = xf + g1 * (a @ W["Wo"].T + W["bo"])
    hc = _ln(x1)
    qc = _rms(hc @ W["Wcq"].T, W["ncq"]).reshape(N, H, 128).transpose(1, 0, 2)
    kc = _rms(cf @ W["Wck"].T, W["nck"]).reshape(-1, H, 128).transpose(1, 0, 2)
    vc = (cf @ W["Wcv"].T).reshape(-1, H, 128).transpose(1, 0, 2)
    sc = qc @ kc.transpose(0, 2, 1) / math.sqrt(128)
    p = np.exp(sc - sc.max(-1, keepdims=True))
    p /= p.sum(-1, keepdims=True)
    x2 = x1 + (p @ vc).transpose(1, 0, 2).reshape(N, d) @ W["Wco"].T
    h2 = _ln(x2) * (1 + sc2) + sh2
    x3 = x2 + g2 * (_gelu_tanh(h2 @ W["W1"].T + W["b1"]) @ W["W2"].T + W["b2"])
    rel = _rel(_f64(out), x3)
    print(f"[parity] dit block ({attn}): block output relative error {rel:.3g}", flush=True)
    assert rel < 2e-2
