"""GPU parity: the HIP path, called through the C ABI, against the fp64 oracle on the same seeded
inputs. Small cases compare every element; the two Wan-shaped layers compare sampled heads and query
blocks (whole rows) plus the full low-rank summary of those heads."""

import math

import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_06712_amd import synth

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU hosts too; every test here is skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_06712_amd import rola as R  # noqa: E402
from tests import _parity as T  # noqa: E402


def _inputs(w, seed=0, device="cpu"):
    inp = synth.make_inputs(w, seed, device=device)
    return {k: v.cuda() for k, v in inp.items()}, synth.to_f64(inp)


def _report(name, **kv):
    line = f"[parity] {name}: " + ", ".join(f"{k}={v}" for k, v in kv.items())
    T.REPORTS.append(line)
    print(line, flush=True)


def _compare_head(w, gpu, ora, b, h, dtype, check_fused=True, check_unfused=True):
    """Selection on every query block (the acceptance rule, with the tie and swap counts), then
    O^s, C, z, O^lr and the outputs on the oracle's rows."""
    rows = ora["rows"]
    g_idx = gpu["idx"][b, h].cpu().numpy()
    ties, differ = T.check_selection(ora["scores"], g_idx, ora["idx"], ora["keep"])
    # rows whose (valid) tie swap changed the block list are excluded from the O^s / O comparison
    bad_blocks = set(int(i) for i in differ)
    keep_rows = np.array([r // w.block not in bad_blocks for r in rows])
    res = {"rows_selected": len(g_idx), "tie_rows": ties, "tie_fraction": round(ties / len(g_idx), 4),
           "swapped_rows": len(differ), "rows_compared": int(keep_rows.sum())}
    res["o_s"] = T.assert_close(T.to_np(gpu["o_s"][b, h])[rows][keep_rows], ora["o_s"][keep_rows],
                                dtype, "O^s")
    res["C"] = T.assert_frob(T.to_np(gpu["C"][b, h]), ora["C"], dtype, "C")
    res["z"] = T.assert_frob(T.to_np(gpu["z"][b, h]), ora["z"], dtype, "z")
    if check_unfused and "o_lr" in gpu:
        res["o_lr"] = T.assert_close(T.to_np(gpu["o_lr"][b, h])[rows], ora["o_lr"], dtype, "O^lr")
        res["out"] = T.assert_close(T.to_np(gpu["out"][b, h])[rows][keep_rows], ora["out"][keep_rows],
                                    dtype, "O")
    if check_fused and "out_fused" in gpu:
        res["out_fused"] = T.assert_close(T.to_np(gpu["out_fused"][b, h])[rows][keep_rows],
                                          ora["out"][keep_rows], dtype, "O fused")
    if "out_epi" in gpu:
        res["out_epi"] = T.assert_close(T.to_np(gpu["out_epi"][b, h])[rows][keep_rows],
                                        ora["out"][keep_rows], dtype, "O attention epilogue")
    if "out_bound" in gpu:
        res["out_bound"] = T.assert_close(T.to_np(gpu["out_bound"][b, h])[rows][keep_rows],
                                          ora["out"][keep_rows], dtype, "O with the score bound")
    if "knorm" in gpu:  # each key block's largest row norm, from the GPU's own K^r
        kr = T.to_np(gpu["kr"][b, h])
        nb = gpu["knorm"].shape[2]
        want = np.array([np.sqrt((kr[J * w.block:(J + 1) * w.block] ** 2).sum(1).max())
                         for J in range(nb)])
        np.testing.assert_allclose(T.to_np(gpu["knorm"][b, h]), want, rtol=1e-5, atol=0)
    return res


def test_tiny_fp32_module():
    """The tiny fp32 layer (B1 H2 d64, 4x8x8 grid, block 32, keep 2, r 16), every element."""
    w = synth.TINY
    inp, f64 = _inputs(w)
    gpu = T.run_gpu(w, inp)
    cos, sin = O.rope_tables(*w.grid, w.split, w.base)
    np.testing.assert_allclose(T.to_np(gpu["cos"]), cos, atol=1e-7)
    np.testing.assert_allclose(T.to_np(gpu["sin"]), sin, atol=1e-7)
    for h in range(w.H):
        ora = T.oracle_head(w, f64, 0, h)
        np.testing.assert_allclose(T.to_np(gpu["qr"][0, h]), ora["qr"], atol=1e-5)
        assert np.array_equal(gpu["idx"][0, h].cpu().numpy(), ora["idx"])
        res = _compare_head(w, gpu, ora, 0, h, "f32")
        _report(f"tiny h{h}", **res)


CASES = [
    # (name, grid, H, B, block, sparsity, r)
    ("ragged r32", (3, 10, 13), 2, 1, 64, 0.5, 32),
    ("ragged r16", (3, 10, 13), 2, 1, 64, 0.5, 16),
    ("ragged r64", (3, 10, 13), 2, 1, 64, 0.5, 64),
    ("ragged r128", (3, 10, 13), 1, 1, 64, 0.5, 128),
    ("block128", (3, 10, 13), 2, 1, 128, 0.5, 32),
    ("batch2", (2, 9, 20), 3, 2, 64, 0.6, 32),
    ("keep-all", (2, 8, 16), 2, 1, 64, 0.0, 32),
    ("keep-one", (4, 8, 16), 2, 1, 64, 0.95, 32),
    ("exact-multiple", (4, 8, 16), 2, 1, 64, 0.75, 32),
    ("single-block", (1, 4, 10), 1, 1, 64, 0.5, 32),
]


@pytest.mark.parametrize("name,grid,H,B,block,s,r", CASES, ids=[c[0] for c in CASES])
def test_bf16_small_every_element(name, grid, H, B, block, s, r):
    w = synth.WAN_1_3B_480P.replace(name=name, grid=grid, H=H, B=B, block=block, sparsity=s, r=r)
    inp, f64 = _inputs(w, seed=1)
    gpu = T.run_gpu(w, inp)
    for b in range(B):
        for h in range(H):
            ora = T.oracle_head(w, f64, b, h)
            res = _compare_head(w, gpu, ora, b, h, "bf16")
            _report(f"{name} b{b} h{h}", **res)


def _spread_blocks(nb, count, seed):
    """`count` query blocks spread over the sequence (so over the frames), seeded: the first and
    the last (possibly partial) block plus distinct random ones."""
    rng = np.random.default_rng(seed)
    rest = rng.choice(np.arange(1, nb - 1), size=count - 2, replace=False)
    return sorted({0, nb - 1, *(int(i) for i in rest)})


def _sampled(w, heads, count, unfused=False, ws_check=False):
    """Full-size layer on the GPU (the configuration the benchmark times). Per sampled head the
    oracle checks the selection of every query block (ties and swaps reported), O^s and O on the
    whole rows of `count` query blocks spread over the frames (the ragged last one included), the
    low-rank summary C, z over the whole head, and with `unfused` also the standalone readout O^lr
    and the separate combine."""
    print(f"[parity] {w.name}: generating inputs on the GPU", flush=True)
    inp = synth.make_inputs(w, 0, device="cuda")
    gpu = T.run_gpu(w, inp, fused_only=not unfused)
    nb = O.num_blocks(w.N, w.block)
    keep = O.keep_blocks(nb, w.sparsity)
    idx = gpu["idx"]
    assert idx.shape == (w.B, w.H, nb, keep)
    assert bool((idx[..., 1:] > idx[..., :-1]).all())
    assert int(idx.min()) >= 0 and int(idx.max()) < nb
    keys = ["idx", "o_s", "C", "z", "out_fused", "out_epi", "out_bound", "kr", "knorm"] + (
        ["o_lr", "out"] if unfused else [])
    for h in heads:
        head_in = {k: inp[k][:, h:h + 1] for k in ("Qn", "Kn", "V")}
        head_in.update(Pq=inp["Pq"][h:h + 1], Pk=inp["Pk"][h:h + 1], logits=inp["logits"])
        qb = _spread_blocks(nb, count, seed=1000 + h)
        ora = T.oracle_head(w, synth.to_f64(head_in), 0, 0, q_blocks=qb)
        sub = {k: gpu[k][:, h:h + 1] for k in keys}
        res = _compare_head(w, sub, ora, 0, 0, "bf16", check_unfused=unfused)
        _report(f"{w.name} h{h} blocks {len(qb)}", **res)
    return inp, gpu


def test_bf16_wan13b_480p_sampled():
    _sampled(synth.WAN_1_3B_480P, heads=[0, 11], count=16)


def test_bf16_wan14b_720p_sampled():
    """The benchmarked layer: selection of all 1182 query blocks of four heads on the smooth-field
    inputs (tie rows and swaps reported), 32 query blocks per head compared element by element,
    the unfused readout and combine too."""
    _sampled(synth.WAN_14B_720P, heads=[0, 13, 26, 39], count=32, unfused=True)


def test_bf16_wan14b_720p_block128_sampled():
    """The sparse sweep's 128-token blocks on the 14B grid (591 blocks, keep 59): sampled heads and
    query blocks, the ragged last block (80 tokens) included."""
    w = synth.WAN_14B_720P.replace(name="wan2.1-14b-720p block128", block=128)
    _sampled(w, heads=[0, 39], count=24)


def test_bf16_long_sequence_adjacent_pairs():
    """4200 query blocks (a 21x80x160 grid, 268800 tokens): beyond the 4064 blocks that pairing by
    overlap serves, so query blocks are paired with their neighbours. Sampled rows against the
    oracle, and the whole output bitwise against one query block per workgroup walking each list in
    the merged order."""
    w = synth.WAN_14B_720P.replace(name="21x80x160 H2 (adjacent pairs)", grid=(21, 80, 160), H=2)
    inp, gpu = _sampled(w, heads=[0, 1], count=8)
    nb = O.num_blocks(w.N, 64)
    keep = O.keep_blocks(nb, w.sparsity)
    assert nb == 4200
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    ws = torch.empty(R.sparse_workspace_bytes(prob, 64, w.sparsity), dtype=torch.uint8,
                     device="cuda")
    shared = R.rola_sparse_attn(gpu["qr"], gpu["kr"], inp["V"], g, 64, w.sparsity, gpu["idx"], ws=ws)
    single = R.rola_sparse_attn(gpu["qr"], gpu["kr"], inp["V"], g, 64, w.sparsity,
                                T.walked_lists(ws, w.B, w.H, nb, keep, paired=False), share=False)
    torch.cuda.synchronize()
    assert torch.equal(shared, single)


def test_bf16_long_merged_lists_sampled():
    """50 % sparsity on the 14B grid (keep 591 of 1182 blocks): the merged lists of a pair run past
    the 1024 entries the LDS table holds, so the attention reads them through scalar loads. Two
    heads, sampled query blocks against the oracle."""
    w = synth.WAN_14B_720P.replace(name="14B grid H2 s0.5 (lists past the LDS table)", H=2,
                                   sparsity=0.5)
    _sampled(w, heads=[0, 1], count=6)


@pytest.mark.parametrize("dtype,grid,block", [("bf16", (3, 10, 13), 64), ("bf16", (3, 10, 13), 128),
                                              ("f32", (4, 8, 8), 32)])
def test_dense_reference_kernel(dtype, grid, block):
    base = synth.WAN_1_3B_480P if dtype == "bf16" else synth.TINY
    w = base.replace(grid=grid, H=2, block=block)
    inp, f64 = _inputs(w, seed=2)
    prob = R.problem(w.B, w.H, w.N, w.d_h, grid, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, grid)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, grid)
    out = R.rola_dense_attn(qr, kr, inp["V"], grid, block)
    torch.cuda.synchronize()
    ocos, osin = O.rope_tables(*grid, w.split)
    for h in range(w.H):
        q = O.round_to(O.rotate(f64["Qn"][0, h], ocos, osin), w.dtype)
        k = O.round_to(O.rotate(f64["Kn"][0, h], ocos, osin), w.dtype)
        nb = O.num_blocks(w.N, block)
        want = O.sparse_attention(q, k, f64["V"][0, h], np.tile(np.arange(nb), (nb, 1)), block,
                                  1.0 / math.sqrt(w.d_h))
        T.assert_close(T.to_np(out[0, h]), want, w.dtype, "dense")


@pytest.mark.parametrize("grid,s", [((3, 10, 13), 0.5), ((2, 9, 20), 0.7), ((4, 8, 16), 0.0)],
                         ids=["odd-nb", "batchlike", "keep-all"])
def test_sparse_shared_loads(grid, s):
    """The path in which paired query blocks share K/V loads (merged block lists) against the
    one-block-per-workgroup path and the oracle, on random block lists: given each block's list in
    the order the merged lists walk it (read back from the workspace), the one-block path visits
    the same blocks in the same order (bitwise equal results); ascending and shuffled lists are
    valid input too (any order) and must still match the oracle."""
    w = synth.WAN_1_3B_480P.replace(grid=grid, H=2, sparsity=s)
    inp, f64 = _inputs(w, seed=6)
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    nb = O.num_blocks(w.N, 64)
    keep = O.keep_blocks(nb, s)
    rng = np.random.default_rng(7)
    lists = np.stack([np.stack([rng.choice(nb, keep, replace=False) for _ in range(nb)])
                      for _ in range(w.H)])[None]
    ocos, osin = O.rope_tables(*g, w.split)
    for order in ("ascending", "shuffled"):
        idx_np = np.sort(lists, axis=-1) if order == "ascending" else lists
        idx = torch.from_numpy(idx_np.astype(np.int32)).cuda()
        ws = torch.empty(R.sparse_workspace_bytes(prob, 64, s), dtype=torch.uint8, device="cuda")
        shared = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, s, idx, ws=ws, share=True)
        single = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, s, idx, share=False)
        walked = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, s,
                                    T.walked_lists(ws, w.B, w.H, nb, keep), share=False)
        torch.cuda.synchronize()
        assert torch.equal(shared, walked)
        for h in range(w.H):
            q = O.round_to(O.rotate(f64["Qn"][0, h], ocos, osin), w.dtype)
            k = O.round_to(O.rotate(f64["Kn"][0, h], ocos, osin), w.dtype)
            want = O.sparse_attention(q, k, f64["V"][0, h], idx_np[0, h], 64, 1.0 / math.sqrt(w.d_h))
            T.assert_close(T.to_np(shared[0, h]), want, w.dtype, f"shared {order} h{h}")
            T.assert_close(T.to_np(single[0, h]), want, w.dtype, f"single {order} h{h}")


def _greedy_pairs(lists, nb, window=64):
    """Pairing of query blocks by list overlap: blocks in ascending order; a block without a partner
    yet takes the free block among its next `window` that shares the most entries (the nearest on
    ties), or stays alone. Entries I | J << 16, J = nb for no partner."""
    sets = [set(int(j) for j in row if 0 <= j < nb) for row in lists]
    taken = np.zeros(nb, bool)
    out = []
    for i in range(nb):
        if taken[i]:
            continue
        best, bj = -1, nb
        for j in range(i + 1, min(nb, i + window + 1)):
            if not taken[j] and len(sets[i] & sets[j]) > best:
                best, bj = len(sets[i] & sets[j]), j
        if bj < nb:
            taken[bj] = True
        out.append(i | (bj << 16))
    return np.array(out, np.int64)


@pytest.mark.parametrize("lists_kind,s", [("selected", 0.8), ("far-partner", 0.85), ("keep-all", 0.0)])
def test_overlap_pairing(lists_kind, s):
    """Query blocks share a workgroup by list overlap: the pair table in the workspace equals the
    greedy matching computed here, covers every block once, and the attention output is bitwise
    that of one query block per workgroup walking the lists in the order the merged lists do. 135 query blocks
    (three 64-block chunks, ragged last block, odd count), two batch entries of two heads."""
    w = synth.WAN_1_3B_480P.replace(grid=(7, 30, 41), B=2, H=2, sparsity=s)
    inp, _ = _inputs(w, seed=8)
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    nb = O.num_blocks(w.N, 64)
    keep = O.keep_blocks(nb, s)
    assert nb == 135
    if lists_kind == "selected":
        idx = R.rola_block_select(qr, kr, g, 64, s)
    else:  # block I selects the keep blocks from (I * m) % nb on: its best partners sit far away
        def lists_for(m):
            start = (np.arange(nb) * m) % nb
            return np.sort((start[:, None] + np.arange(keep)[None, :]) % nb, axis=1)
        full = np.stack([np.stack([lists_for(37 + 16 * (b * w.H + h)) for h in range(w.H)])
                         for b in range(w.B)])
        idx = torch.from_numpy(full.astype(np.int32)).cuda()
    need = R.sparse_workspace_bytes(prob, 64, s)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    shared = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, s, idx, ws=ws)
    single = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, s, T.walked_lists(ws, w.B, w.H, nb, keep),
                                share=False)
    torch.cuda.synchronize()
    ngroups = (nb + 1) // 2
    # the workspace starts with the work-queue counters (8 slots of 256 bytes), then the pair table
    q = 8 * 256
    table = ws[q: q + w.B * w.H * ngroups * 4].view(torch.int32).cpu().numpy().reshape(w.B, w.H, ngroups)
    idx_np = idx.cpu().numpy()
    for b in range(w.B):
        for h in range(w.H):
            want = _greedy_pairs(idx_np[b, h], nb)
            got = table[b, h].astype(np.int64)
            assert np.array_equal(got, want), (b, h, np.nonzero(got != want)[0][:8])
            members = np.concatenate([got & 0xFFFF, got >> 16])
            assert np.array_equal(np.sort(members[members < nb]), np.arange(nb))
    _report("overlap pairing", kind=lists_kind, adjacent=int(sum(
        ((table[0, 0] >> 16) - (table[0, 0] & 0xFFFF)) == 1)), groups=ngroups)
    assert torch.equal(shared, single)


def test_work_queue_full_size():
    """At the 14B 720p size the attention kernel runs as resident workgroups that claim (head,
    pair) groups from per-XCD counters: 23640 groups, far more than the chip holds at once, so
    workgroups loop and XCDs that finish early take groups from the others. Every group must be
    done exactly once: starting from stale counters (the list-merge kernel clears them), all
    counters end past their ranges and the whole output is bitwise that of the path with one
    query block per workgroup (a static grid, each list in the order the merged lists walk it);
    a second call on the same workspace agrees."""
    w = synth.WAN_14B_720P
    inp = synth.make_inputs(w, 0, device="cuda")
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    idx = R.rola_block_select(qr, kr, g, 64, w.sparsity)
    ws = torch.empty(R.sparse_workspace_bytes(prob, 64, w.sparsity), dtype=torch.uint8, device="cuda")
    ws[:8 * 256].fill_(0x7F)
    shared = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, w.sparsity, idx, ws=ws)
    counters = ws[:8 * 256].view(torch.int32).cpu().numpy()[::64]  # one int per 256-byte slot
    again = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, w.sparsity, idx, ws=ws)
    nb = O.num_blocks(w.N, 64)
    keep = O.keep_blocks(nb, w.sparsity)
    single = R.rola_sparse_attn(qr, kr, inp["V"], g, 64, w.sparsity,
                                T.walked_lists(ws, w.B, w.H, nb, keep), share=False)
    torch.cuda.synchronize()
    total = w.B * w.H * ((nb + 1) // 2)
    q, rem = divmod(total, 8)
    _report("work queue", groups=total, counters=counters.tolist())
    assert all(counters[x] >= q + (x < rem) for x in range(8)), counters
    assert torch.equal(shared, single)
    assert torch.equal(again, single)


@pytest.mark.parametrize("grid", [(21, 45, 80), (21, 45, 104), (21, 45, 160)],
                         ids=["1182-blocks", "1536-blocks", "2363-blocks"])
def test_block_select_rows(grid):
    """Top-k over score rows of 1182 to 2363 key blocks (the radix select keeps a row's keys in
    LDS). One head, every row against the oracle (pooling, fp64 scores, top-k with ties to the
    lower block)."""
    w = synth.WAN_1_3B_480P.replace(grid=grid, H=1, B=1, sparsity=0.9)
    gen = torch.Generator().manual_seed(12)
    qr = torch.randn((1, 1, w.N, 128), generator=gen).to(torch.bfloat16)
    kr = torch.randn((1, 1, w.N, 128), generator=gen).to(torch.bfloat16)
    idx = R.rola_block_select(qr.cuda(), kr.cuda(), w.grid, 64, w.sparsity).cpu().numpy()[0, 0]
    nb = O.num_blocks(w.N, 64)
    keep = O.keep_blocks(nb, w.sparsity)
    scores = O.block_scores(O.pool_blocks(qr[0, 0].double().numpy(), 64),
                            O.pool_blocks(kr[0, 0].double().numpy(), 64))
    ties, differ = T.check_selection(scores, idx, O.select_blocks(scores, keep), keep)
    _report("block select", n_b=nb, keep=keep, tie_rows=ties, differing=len(differ))


@pytest.mark.parametrize("grid", [(21, 45, 80), (21, 45, 160), (21, 45, 180)],
                         ids=["1182-blocks", "2363-blocks", "2658-blocks"])
def test_topk_crafted_rows(grid):
    """Top-k on score rows built to reach every branch of the selection: means that are one-hot
    queries against key means holding a chosen value per block, so that row I's scores are exactly
    the values of pattern I mod 5 (products with 1.0, exact in fp32 and fp64). Patterns: distinct
    random values; values drawn from a few hundred levels (exact ties across the k-th score);
    300 distinct values within one part in 2^20 of each other across the k-th (more than 64
    candidates in the k-th key's upper-half bucket); 300 exactly equal values there; negative
    values only. Rows of 1182 and 2363 blocks take the register kernel, 2658 the LDS kernel.
    Every row against the oracle's top-k (ties to the lower block), bitwise."""
    w = synth.WAN_1_3B_480P.replace(grid=grid, H=1, B=1, sparsity=0.9)
    nb = O.num_blocks(w.N, 64)
    keep = O.keep_blocks(nb, w.sparsity)
    rng = np.random.default_rng(17)
    pats = np.zeros((5, nb))
    pats[0] = rng.standard_normal(nb)
    pats[1] = rng.integers(0, 300, nb) / 7.0
    mid = rng.permutation(nb)[:300]
    pats[2] = rng.standard_normal(nb) - 10.0
    pats[2][mid] = 1.0 + np.arange(300) * 2.0 ** -23
    pats[3] = rng.standard_normal(nb) - 10.0
    pats[3][mid] = 0.75
    pats[4] = -np.abs(rng.standard_normal(nb)) - 1.0
    pats = pats.astype(np.float32)
    qbar = np.zeros((nb, 128), np.float32)
    qbar[np.arange(nb), np.arange(nb) % 5] = 1.0
    kbar = np.zeros((nb, 128), np.float32)
    kbar[:, :5] = pats.T
    like = torch.zeros((1, 1, w.N, 128), dtype=torch.bfloat16, device="cuda")
    idx = R.rola_block_select_pooled(torch.from_numpy(qbar).view(1, 1, nb, 128).cuda(),
                                     torch.from_numpy(kbar).view(1, 1, nb, 128).cuda(), like,
                                     w.grid, 64, w.sparsity).cpu().numpy()[0, 0]
    scores = qbar.astype(np.float64) @ kbar.astype(np.float64).T
    want = O.select_blocks(scores, keep)
    _report("crafted top-k", n_b=nb, keep=keep)
    assert np.array_equal(idx, want)


def test_out_of_range_entries_skipped():
    """Block lists a caller hands in may hold entries outside [0, n_b): here n_b + 3 as the last
    entry of every other row and -1 as the first entry of every third. Every path skips them (the
    pairing and the list merge drop them; the one-block walk decodes them as no keys), so O^s is
    the oracle's attention over each row's valid entries, on the merged-list path and the
    one-block path alike. Ragged grid: 390 tokens, 7 blocks of 64, the last of 6 tokens."""
    w = synth.WAN_1_3B_480P.replace(grid=(3, 10, 13), H=2)
    gen = torch.Generator().manual_seed(21)
    qr = torch.randn((1, w.H, w.N, 128), generator=gen).to(torch.bfloat16)
    kr = torch.randn((1, w.H, w.N, 128), generator=gen).to(torch.bfloat16)
    v = torch.randn((1, w.H, w.N, 128), generator=gen).to(torch.bfloat16)
    nb = O.num_blocks(w.N, 64)
    idx = R.rola_block_select(qr.cuda(), kr.cuda(), w.grid, 64, 0.5)
    bad = idx.clone()
    bad[:, :, 0::2, -1] = nb + 3
    bad[:, :, 0::3, 0] = -1
    outs = {share: R.rola_sparse_attn(qr.cuda(), kr.cuda(), v.cuda(), w.grid, 64, 0.5, bad,
                                      share=share).double().cpu().numpy()
            for share in (True, False)}
    lists = bad.cpu().numpy()
    for h in range(w.H):
        valid = np.empty(nb, dtype=object)
        for I in range(nb):
            valid[I] = np.array([J for J in lists[0, h, I] if 0 <= J < nb], dtype=np.int64)
        want = O.sparse_attention(qr[0, h].double().numpy(), kr[0, h].double().numpy(),
                                  v[0, h].double().numpy(), valid, 64, 128 ** -0.5)
        for share, out in outs.items():
            d = np.abs(out[0, h] - want)
            _report("out-of-range entries", head=h, share=share, max_abs=float(d.max()),
                    mean_abs=float(d.mean()))
            assert d.max() <= T.TOL["bf16"]["max_abs"] and d.mean() <= T.TOL["bf16"]["mean_abs"]


def test_exact_ties_go_to_lower_block():
    """Identical key blocks tie exactly: every row must keep the lowest block indices."""
    w = synth.WAN_1_3B_480P.replace(grid=(2, 8, 16), H=2)
    g = w.grid
    rng = torch.Generator().manual_seed(5)
    qr = torch.randn((1, 2, w.N, 128), generator=rng).to(torch.bfloat16)
    blk = torch.randn((1, 2, 64, 128), generator=rng).to(torch.bfloat16)
    kr = blk.repeat(1, 1, w.N // 64, 1)
    idx = R.rola_block_select(qr.cuda(), kr.cuda(), g, 64, 0.5).cpu()
    keep = O.keep_blocks(w.N // 64, 0.5)
    assert torch.equal(idx, torch.arange(keep, dtype=torch.int32).expand_as(idx))


def test_bitwise_reproducible():
    w = synth.WAN_1_3B_480P.replace(grid=(3, 10, 13), H=2)
    inp, _ = _inputs(w, seed=3)
    a = T.run_gpu(w, inp)
    b = T.run_gpu(w, inp)
    for k in ("idx", "o_s", "C", "z", "o_lr", "out", "out_fused"):
        assert torch.equal(a[k], b[k]), k


def test_combine_in_place_matches_out_of_place():
    w = synth.WAN_1_3B_480P.replace(grid=(3, 10, 13), H=2)
    inp, _ = _inputs(w, seed=4)
    res = T.run_gpu(w, inp)
    os_copy = res["o_s"].clone()
    R.rola_combine(os_copy, res["o_lr"], inp["logits"], w.grid, out=os_copy)
    os_copy2 = res["o_s"].clone()
    prob = R.problem(w.B, w.H, w.N, w.d_h, w.grid, w.dtype)
    R.rola_lowrank_readout_combine(inp["Qn"], inp["Pq"], w.r, res["cos"], res["sin"], res["C"],
                                   os_copy2, inp["logits"], w.grid, out=os_copy2)
    torch.cuda.synchronize()
    assert torch.equal(os_copy, res["out"])
    assert torch.equal(os_copy2, res["out_fused"])


def test_plan_then_planned_attention_on_two_streams():
    """rola_sparse_plan + rola_sparse_attn_combine_planned, with the low-rank summary on a second
    stream between them (the benchmarked layer's schedule, on the 1.3B 480p layer), give bitwise the
    output of the single call rola_sparse_attn_combine."""
    w = synth.WAN_1_3B_480P
    inp = synth.make_inputs(w, 0, device="cuda")
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    idx = R.rola_block_select(qr, kr, g, w.block, w.sparsity)
    C, _ = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g)
    want = R.rola_sparse_attn_combine(qr, kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"],
                                      inp["Pq"], w.r, cos, sin, C, inp["logits"])
    ws = torch.empty(R.sparse_combine_workspace_bytes(prob, w.block, w.sparsity, w.r),
                     dtype=torch.uint8, device="cuda")
    C2 = torch.zeros_like(C)
    side = torch.cuda.Stream()
    fork, join = torch.cuda.Event(), torch.cuda.Event()
    torch.cuda.synchronize()
    fork.record()
    side.wait_event(fork)
    R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g, C=C2, stream=side)
    join.record(side)
    R.rola_sparse_plan(idx, qr, g, w.block, w.sparsity, w.r, ws)
    torch.cuda.current_stream().wait_event(join)
    got = R.rola_sparse_attn_combine_planned(qr, kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"],
                                             inp["Pq"], w.r, cos, sin, C2, inp["logits"], ws)
    torch.cuda.synchronize()
    assert torch.equal(C2, C)
    assert torch.equal(got, want)
    # block 128 has no plan: the planned call is the plain one
    w2 = w.replace(grid=(3, 10, 13), H=2, block=128, sparsity=0.5)
    inp2 = synth.make_inputs(w2, 1, device="cuda")
    p2 = R.problem(w2.B, w2.H, w2.N, w2.d_h, w2.grid, w2.dtype)
    c2, s2 = R.rola_rope_tables(p2, w2.split)
    q2 = R.rola_rope_apply(inp2["Qn"], c2, s2, w2.grid)
    k2 = R.rola_rope_apply(inp2["Kn"], c2, s2, w2.grid)
    i2 = R.rola_block_select(q2, k2, w2.grid, 128, 0.5)
    Cb, _ = R.rola_lowrank_summary(inp2["Kn"], inp2["V"], inp2["Pk"], w2.r, c2, s2, w2.grid)
    ws2 = torch.empty(max(16, R.sparse_combine_workspace_bytes(p2, 128, 0.5, w2.r)), dtype=torch.uint8,
                      device="cuda")
    a2 = (q2, k2, inp2["V"], w2.grid, 128, 0.5, i2, inp2["Qn"], inp2["Pq"], w2.r, c2, s2, Cb,
          inp2["logits"])
    R.rola_sparse_plan(i2, q2, w2.grid, 128, 0.5, w2.r, ws2)
    got2 = R.rola_sparse_attn_combine_planned(*a2, ws2)
    want2 = R.rola_sparse_attn_combine(*a2)
    torch.cuda.synchronize()
    assert torch.equal(got2, want2)


def test_score_bound_reference():
    """The planned call given each key block's largest norm takes B = |q| max|k| scale log2(e) as
    its softmax reference for every wave whose B are all at most 40, and the running maximum for
    the others. (a) On the 1.3B layer (B about 20 everywhere) it runs (not bitwise the call
    without norms) and differs from it by the rounding of the probabilities only. (b) With every
    query 8 times larger every wave falls back: bitwise the call without norms. (c) With the
    queries of every other 32-token wave 8 times larger (waves of both kinds in one workgroup),
    every element against the oracle."""
    w = synth.WAN_1_3B_480P
    inp = synth.make_inputs(w, 0, device="cuda")
    gpu = T.run_gpu(w, inp, fused_only=True)
    d = (gpu["out_bound"].float() - gpu["out_epi"].float()).abs()
    _report("score bound, 1.3B layer", max_diff=float(d.max()), mean_diff=float(d.mean()))
    assert not torch.equal(gpu["out_bound"], gpu["out_epi"])
    assert float(d.max()) <= 0.04 and float(d.mean()) <= 1e-3
    small = w.replace(name="score bound fallback", grid=(3, 10, 13), H=2)
    inp, f64 = _inputs(small, seed=3)
    big = dict(inp, Qn=inp["Qn"] * 8)  # exact in bf16, and the rotation commutes with it
    gpu = T.run_gpu(small, big, fused_only=True)
    assert torch.equal(gpu["out_bound"], gpu["out_epi"])
    mixed = inp["Qn"].clone()
    n = torch.arange(small.N, device="cuda")
    mixed[:, :, (n // 32) % 2 == 0] *= 8
    inp_m = dict(inp, Qn=mixed)
    gpu = T.run_gpu(small, inp_m, fused_only=True)
    f64_m = synth.to_f64({k: v.cpu() for k, v in inp_m.items()})
    for h in range(small.H):
        ora = T.oracle_head(small, f64_m, 0, h)
        res = _compare_head(small, gpu, ora, 0, h, "bf16", check_unfused=False)
        _report(f"score bound, mixed waves h{h}", **res)


@pytest.mark.parametrize("grid,H,block", [((21, 30, 52), 12, 64), ((3, 10, 13), 2, 64),
                                          ((3, 10, 13), 2, 128)],
                         ids=["1.3B-480p", "ragged-b64", "ragged-b128"])
def test_rope_pool_producer(grid, H, block):
    """The rotating pooling pass (rola_rope_pool): its K^r is bitwise rola_rope_apply's, its block
    means are the oracle's pool_blocks of the rounded rotation (fp32 sums of 64 or 128 rows), and the
    selection from them (rola_block_select_pooled) is bitwise rola_block_select's lists."""
    w = synth.WAN_1_3B_480P.replace(grid=grid, H=H, block=block)
    inp, f64 = _inputs(w, seed=9)
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    want_idx = R.rola_block_select(qr, kr, g, block, w.sparsity)
    nb = R.num_blocks(w.N, block)
    knorm = torch.empty((w.B, w.H, nb), dtype=torch.float32, device="cuda")
    knorm_r = torch.empty_like(knorm)
    kr2, kbar = R.rola_rope_pool(inp["Kn"], cos, sin, g, block, xnorm=knorm)
    none, qbar = R.rola_rope_pool(inp["Qn"], cos, sin, g, block, want_xr=False)
    idx = R.rola_block_select_pooled(qbar, kbar, qr, g, block, w.sparsity)
    _, qbar_r = R.rola_rope_pool(qr, None, None, g, block)   # pooling of the rotated tensor
    _, kbar_r = R.rola_rope_pool(kr, None, None, g, block, xnorm=knorm_r)
    torch.cuda.synchronize()
    assert none is None
    assert torch.equal(kr2, kr)
    assert torch.equal(idx, want_idx)
    assert torch.equal(qbar_r, qbar)
    assert torch.equal(kbar_r, kbar)
    # each block's largest row norm of the rounded rotation, both passes
    k64 = kr.double()
    rows = (k64 * k64).sum(-1).sqrt()
    pad = nb * block - w.N
    want = torch.nn.functional.pad(rows, (0, pad), value=0.0).view(w.B, w.H, nb, block).amax(-1)
    torch.testing.assert_close(knorm.double(), want, rtol=1e-5, atol=0)
    torch.testing.assert_close(knorm_r.double(), want, rtol=1e-5, atol=0)
    ocos, osin = O.rope_tables(*g, w.split)
    for h in range(w.H):
        # the pooling arithmetic: the oracle's pool_blocks of the GPU's own rounded rotation
        np.testing.assert_allclose(T.to_np(qbar[0, h]), O.pool_blocks(T.to_np(qr[0, h]), block),
                                   rtol=0, atol=2e-6)
        # against the oracle's fp64 rotation: the rounding of a few elements may differ by one bf16
        # ulp (2^-8 relative), diluted over the block
        q = O.round_to(O.rotate(f64["Qn"][0, h], ocos, osin), w.dtype)
        np.testing.assert_allclose(T.to_np(qbar[0, h]), O.pool_blocks(q, block), rtol=0, atol=1e-3)
    _report(f"rope_pool {grid} block {block}", heads=w.H, blocks=qbar.shape[2])


@pytest.mark.parametrize("grid,H,r", [((21, 30, 52), 12, 32), ((3, 10, 13), 2, 16),
                                      ((2, 9, 20), 3, 64)], ids=["1.3B-480p", "ragged-r16", "r64"])
def test_attention_rotates_queries_in_prologue(grid, H, r):
    """rola_sparse_attn_combine with Qr = None rotates Q^n in the attention's prologue: bitwise the
    output with Qr = rola_rope_apply(Qn), and the planned form agrees."""
    w = synth.WAN_1_3B_480P.replace(grid=grid, H=H, r=r)
    inp = synth.make_inputs(w, 4, device="cuda")
    g = w.grid
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    idx = R.rola_block_select(qr, kr, g, w.block, w.sparsity)
    C, _ = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g)
    rest = (kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"], inp["Pq"], w.r, cos, sin, C,
            inp["logits"])
    want = R.rola_sparse_attn_combine(qr, *rest)
    got = R.rola_sparse_attn_combine(None, *rest)
    ws = torch.empty(R.sparse_combine_workspace_bytes(prob, w.block, w.sparsity, w.r),
                     dtype=torch.uint8, device="cuda")
    R.rola_sparse_plan(idx, inp["Qn"], g, w.block, w.sparsity, w.r, ws)
    planned = R.rola_sparse_attn_combine_planned(None, *rest, ws)
    torch.cuda.synchronize()
    assert torch.equal(got, want)
    assert torch.equal(planned, want)
