"""GPU parity of the steps either side of the module's path: the gate logits X W_g + b_g of the
token-wise gate (Sec. 4.4; Algorithm step 8) against the oracle."""

import numpy as np
import pytest
import torch

import oracle as O

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_06712_amd import rola as R  # noqa: E402


@pytest.mark.parametrize("dtype,B,N,dm", [("bf16", 1, 390, 5120), ("bf16", 2, 257, 1536),
                                          ("f32", 2, 131, 520), ("bf16", 1, 75600, 5120)],
                         ids=["wan14b-dmodel", "odd-rows", "f32", "wan14b-720p-tokens"])
def test_gate_logits(dtype, B, N, dm):
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    gen = torch.Generator().manual_seed(N + dm)
    X = torch.randn((B, N, dm), generator=gen).to(tdt)
    Wg = (torch.randn((dm,), generator=gen) / dm ** 0.5).to(tdt)
    bg = -1.946
    grid = (N, 1, 1)
    got = R.rola_gate_logits(X.cuda(), Wg.cuda(), bg, grid)
    zero = R.rola_gate_logits(X.cuda(), torch.zeros_like(Wg).cuda(), bg, grid)
    torch.cuda.synchronize()
    # at the paper's initialisation (W_g = 0) every logit is exactly b_g
    assert bool((zero.cpu() == torch.tensor(bg, dtype=torch.float32)).all())
    rows = np.arange(N) if N <= 4096 else np.sort(np.random.default_rng(0).choice(N, 4096, replace=False))
    Xf, Wf = X[:, torch.from_numpy(rows)].double().numpy(), Wg.double().numpy()
    want = O.gate_logits(Xf, Wf, bg)
    # fp32 accumulation of dm products: error <= dm * 2^-24 * sum |x w| (loose bound, in practice far less)
    bound = dm * 2.0 ** -24 * (np.abs(Xf) @ np.abs(Wf)) + 1e-6
    err = np.abs(got.cpu().double().numpy()[:, rows] - want)
    assert np.all(err <= bound), float((err / bound).max())
    print(f"[parity] gate logits {dtype} B{B} N{N} d_model {dm}: max-abs {err.max():.3g}", flush=True)
