"""Helpers of the GPU parity tests: run the HIP path through the C ABI, run the oracle on the same
seeded inputs (whole heads or sampled rows), and compare under the acceptance rules:
  * block lists bit-exact wherever the oracle's fp64 score gap between the keep-th and the next block
    exceeds 1e-4; elsewhere the lists may differ only by blocks within 1e-4 of the keep-th score;
  * bf16 outputs: max-abs <= 2e-2 and mean-abs <= 5e-3; fp32 outputs: max-abs <= 1e-5;
  * C and z: relative Frobenius error <= 1e-2 (bf16) or 1e-5 (fp32).
"""

import math

import numpy as np
import torch

import oracle as O
from paper_2609_06712_amd import rola as R
from paper_2609_06712_amd import synth

TIE_GAP = 1e-4
REPORTS = []  # one line per compared head, printed at the end of the run (tests/conftest.py)
TOL = {"bf16": dict(max_abs=2e-2, mean_abs=5e-3, frob=1e-2),
       "f32": dict(max_abs=1e-5, mean_abs=1e-5, frob=1e-5)}


def run_gpu(w: synth.Workload, inp: dict, fused_only=False):
    """All steps of the layer through the C ABI on the current device."""
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split, w.base)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    idx = R.rola_block_select(qr, kr, g, w.block, w.sparsity)
    o_s = R.rola_sparse_attn(qr, kr, inp["V"], g, w.block, w.sparsity, idx)
    C, z = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g)
    out_fused = R.rola_lowrank_readout_combine(inp["Qn"], inp["Pq"], w.r, cos, sin, C, o_s,
                                               inp["logits"], g)
    # the whole tail in one call: attention with the readout and combine in its epilogue
    out_epi = R.rola_sparse_attn_combine(qr, kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"],
                                         inp["Pq"], w.r, cos, sin, C, inp["logits"])
    # the benchmarked form: the planned call given each key block's largest norm (from the pooling
    # pass), so that the attention may use the score bound as its softmax reference
    knorm = torch.empty((w.B, w.H, R.num_blocks(w.N, w.block)), dtype=torch.float32, device=qr.device)
    R.rola_rope_pool(kr, None, None, g, w.block, xnorm=knorm)
    ws = torch.empty(max(16, R.sparse_combine_workspace_bytes(prob, w.block, w.sparsity, w.r)),
                     dtype=torch.uint8, device=qr.device)
    R.rola_sparse_plan(idx, qr, g, w.block, w.sparsity, w.r, ws)
    out_bound = R.rola_sparse_attn_combine_planned(qr, kr, inp["V"], g, w.block, w.sparsity, idx,
                                                   inp["Qn"], inp["Pq"], w.r, cos, sin, C,
                                                   inp["logits"], ws, key_norm=knorm)
    res = dict(cos=cos, sin=sin, qr=qr, kr=kr, idx=idx, o_s=o_s, C=C, z=z, out_fused=out_fused,
               out_epi=out_epi, out_bound=out_bound, knorm=knorm)
    if not fused_only:
        o_lr = R.rola_lowrank_readout(inp["Qn"], inp["Pq"], w.r, cos, sin, C, g)
        res["o_lr"] = o_lr
        res["out"] = R.rola_combine(o_s, o_lr, inp["logits"], g)
    torch.cuda.synchronize()
    return res


def oracle_head(w: synth.Workload, f64: dict, b: int, h: int, q_blocks=None):
    """Oracle results for one (b, h). Block scores and selections cover every query block. With
    q_blocks given, O^s / O^lr / O only for the rows of those query blocks (ascending); C, z always
    over the whole head."""
    cos, sin = O.rope_tables(*w.grid, w.split, w.base)
    qn, kn, v = f64["Qn"][b, h], f64["Kn"][b, h], f64["V"][b, h]
    qr = O.round_to(O.rotate(qn, cos, sin), w.dtype)
    kr = O.round_to(O.rotate(kn, cos, sin), w.dtype)
    nb = O.num_blocks(w.N, w.block)
    keep = O.keep_blocks(nb, w.sparsity)
    qbar, kbar = O.pool_blocks(qr, w.block), O.pool_blocks(kr, w.block)
    scores = O.block_scores(qbar, kbar)
    idx = O.select_blocks(scores, keep)
    qb = np.arange(nb) if q_blocks is None else np.asarray(sorted(set(int(i) for i in q_blocks)))
    rows = np.concatenate([np.arange(I * w.block, min(w.N, (I + 1) * w.block)) for I in qb])
    scale = 1.0 / math.sqrt(w.d_h)
    o_s = O.sparse_attention_blocks(qr, kr, v, idx, w.block, scale, qb)
    C, z = O.lowrank_summary(kn, v, f64["Pk"][h], cos, sin)
    u = O.lowrank_features(qn[rows], f64["Pq"][h], cos[rows], sin[rows]) @ C
    o_lr = O.rms_normalize(u, 1e-6)
    out = O.combine(o_s, o_lr, f64["logits"][b, rows], 1e-6)
    return dict(qb=qb, rows=rows, scores=scores, idx=idx, keep=keep, o_s=o_s, C=C, z=z,
                o_lr=o_lr, out=out, qr=qr, kr=kr, cos=cos, sin=sin)


def check_selection(scores: np.ndarray, gpu_idx: np.ndarray, ora_idx: np.ndarray, keep: int):
    """Returns (tie_rows, differing_rows); asserts the acceptance rule on every row."""
    tie_rows, differ = 0, []
    for i in range(scores.shape[0]):
        g = gpu_idx[i]
        assert len(g) == keep and np.all(np.diff(g) > 0), f"row {i}: not ascending/unique: {g}"
        s = scores[i]
        srt = np.sort(s)[::-1]
        kth = srt[keep - 1]
        gap = kth - srt[keep] if keep < len(s) else np.inf
        same = np.array_equal(g, ora_idx[i])
        if gap > TIE_GAP:
            assert same, f"row {i}: gap {gap:.3g} but lists differ"
        else:
            tie_rows += 1
            if not same:
                sym = np.setxor1d(g, ora_idx[i])
                assert np.all(np.abs(s[sym] - kth) <= TIE_GAP), f"row {i}: invalid tie swap {sym}"
                differ.append(i)
    return tie_rows, differ


def err_stats(got: np.ndarray, want: np.ndarray):
    d = np.abs(np.asarray(got, np.float64) - want)
    return float(d.max()), float(d.mean())


def assert_close(got, want, dtype, what):
    mx, mean = err_stats(got, want)
    tol = TOL[dtype]
    assert mx <= tol["max_abs"] and mean <= tol["mean_abs"], (
        f"{what}: max-abs {mx:.3g} (tol {tol['max_abs']}), mean-abs {mean:.3g} (tol {tol['mean_abs']})")
    return mx, mean


def assert_frob(got, want, dtype, what):
    got = np.asarray(got, np.float64)
    rel = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))
    assert rel <= TOL[dtype]["frob"], f"{what}: relative Frobenius error {rel:.3g}"
    return rel


def walked_lists(ws: torch.Tensor, B: int, H: int, nb: int, keep: int, paired: bool = True) -> torch.Tensor:
    """Each query block's selections in the order the work-queue attention walks them, read back
    from its workspace: [queue counters: 8 slots of 256 bytes][pair table I0 | I1 << 16 per group,
    padded to 256 bytes, when paired][per group: entry count E, then 2 keep entries J | members << 16].
    Checks on the way that every merged list is the union in walk order (by increasing
    bit-reversed key block index over the smallest power of two >= nb), rotated to some start, and that each member holds all keep of its entries. The one-block path walks a
    list in the order given, so on these lists both paths sum every query's keys alike."""
    heads, ng, stride = B * H, (nb + 1) // 2, 2 * keep + 1
    off = 8 * 256
    if paired:
        table = ws[off: off + heads * ng * 4].view(torch.int32).cpu().numpy().reshape(heads, ng)
        off += (heads * ng * 4 + 255) // 256 * 256
    else:
        g = np.arange(ng)
        table = np.broadcast_to(2 * g | (2 * g + 1) << 16, (heads, ng))
    table = table.astype(np.int64)
    lists = ws[off: off + heads * ng * stride * 4].view(torch.int32).cpu().numpy()
    lists = lists.reshape(heads, ng, stride).astype(np.int64)
    E, ent = lists[..., 0], lists[..., 1:]
    valid = np.arange(2 * keep)[None, None, :] < E[..., None]
    k = max(1, (nb - 1).bit_length())
    key = np.array([int(format(j, f"0{k}b")[::-1], 2) for j in range(1 << k)])
    pos = np.where(valid, key[np.clip(ent & 0xFFFF, 0, (1 << k) - 1)], -1)
    desc = np.sum(valid[..., 1:] & (pos[..., 1:] < pos[..., :-1]), axis=-1)
    last = np.take_along_axis(pos, np.maximum(E - 1, 0)[..., None], -1)[..., 0]
    assert np.all(desc <= 1) and np.all((desc == 0) | (last < pos[..., 0])), "not a rotated walk"
    out = np.full((heads, nb, keep), -1, np.int64)
    for b in range(2):
        I = table >> (16 * b) & 0xFFFF
        sel = valid & ((ent >> (16 + b)) & 1).astype(bool)
        hh, gg = np.nonzero(I < nb)
        assert np.all(sel.sum(-1)[hh, gg] == keep)
        order = np.argsort(~sel, axis=-1, kind="stable")[..., :keep]
        J = np.take_along_axis(ent & 0xFFFF, order, -1)
        out[hh, I[hh, gg]] = J[hh, gg]
    assert np.all(out >= 0)
    return torch.from_numpy(out.reshape(B, H, nb, keep).astype(np.int32)).to(ws.device)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()
