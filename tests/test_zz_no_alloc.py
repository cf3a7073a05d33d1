"""The allocation-free attention + readout + combine (rola_sparse_attn_combine_noalloc, static
device scratch) against rola_sparse_attn_combine with a workspace, through the C ABI: bitwise equal
outputs on consecutive calls of decreasing size on the same device (the static scratch keeps the
previous call's contents), and a problem too large for the scratch rejected before any launch."""

import pytest
import torch

from paper_2609_06712_amd import synth

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_06712_amd import rola as R  # noqa: E402


def _layer(w, seed):
    inp = synth.make_inputs(w, seed, device="cuda")
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split, w.base)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    idx = R.rola_block_select(qr, kr, g, w.block, w.sparsity)
    C, _ = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g)
    args = (qr, kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"], inp["Pq"], w.r, cos, sin, C,
            inp["logits"])
    return args


def test_noalloc_matches_workspace_form():
    cases = [synth.WAN_14B_720P,                                   # about 23 MB of scratch
             synth.WAN_1_3B_480P.replace(name="small", grid=(3, 10, 13), H=2),
             synth.WAN_1_3B_480P.replace(name="small r64", grid=(2, 9, 20), H=3, B=2, r=64)]
    for seed, w in enumerate(cases):
        print(f"[noalloc] {w.name}", flush=True)
        args = _layer(w, seed)
        want = R.rola_sparse_attn_combine(*args)
        got = torch.full_like(want, float("nan"))
        R.rola_sparse_attn_combine_noalloc(*args, out=got)
        # with the key-block norms (the score-bound softmax reference) as well
        knorm = torch.empty((w.B, w.H, R.num_blocks(w.N, w.block)), dtype=torch.float32,
                            device="cuda")
        R.rola_rope_pool(args[1], None, None, w.grid, w.block, xnorm=knorm)
        want_b = R.rola_sparse_attn_combine(*args, key_norm=knorm)
        got_b = torch.full_like(want, float("nan"))
        R.rola_sparse_attn_combine_noalloc(*args, out=got_b, key_norm=knorm)
        torch.cuda.synchronize()
        assert torch.equal(got, want), w.name
        assert torch.equal(got_b, want_b), w.name
        del args, want, got, want_b, got_b


def test_noalloc_rejects_a_problem_beyond_the_scratch():
    w = synth.WAN_14B_720P.replace(name="keep-all 14B grid", H=8, sparsity=0.0)
    prob = R.problem(w.B, w.H, w.N, w.d_h, w.grid, w.dtype)
    assert R.sparse_combine_workspace_bytes(prob, 64, 0.0, 32) > (32 << 20)
    t = torch.zeros((1, w.H, w.N, 128), dtype=torch.bfloat16, device="cuda")
    nb = R.num_blocks(w.N, 64)
    idx = torch.zeros((1, w.H, nb, nb), dtype=torch.int32, device="cuda")
    cos = torch.zeros((w.N, 64), device="cuda")
    C = torch.zeros((1, w.H, 32, 128), device="cuda")
    lg = torch.zeros((1, w.N), device="cuda")
    with pytest.raises(R.RolaError) as e:
        R.rola_sparse_attn_combine_noalloc(t, t.clone(), t.clone(), w.grid, 64, 0.0, idx, t.clone(),
                                           torch.zeros((w.H, 32, 128), dtype=torch.bfloat16,
                                                       device="cuda"),
                                           32, cos, cos, C, lg, out=t.clone())
    assert e.value.status == R.ROLA_ERR_UNSUPPORTED
