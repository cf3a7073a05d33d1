"""Benchmark of one RoLA attention layer (sparse + rotary low-rank branches) on one MI355X.

One step = the whole hot path over one batch of synthetic input already resident in HBM, as C-ABI
calls on two HIP streams: on the main stream the block means of Q^r and K^r (with each key block's
largest key norm), the block scores and top-k, and the attention's pairing and list merge
(rola_sparse_plan); on a second stream, once the top-k is done, the low-rank summary; after the two
join, the block-sparse attention with the low-rank readout and the gated combine in its epilogue,
given the key norms so that it can take the score bound as its softmax reference. Workload: the
Wan2.1-14B-shaped 720p layer
(B1 H40 d128, 21x45x80 grid = 75600 tokens, block 64, 90 % sparsity -> 118 of 1182 key blocks, r 32,
bf16). The backbone's own steps (rotary tables, Q^r = R(Q^n), K^r = R(K^n)) are the step's input;
the same layer starting from Q^n, K^n (rotation fused into the pooling passes) is timed beside it.

Prints one JSON line: effective TFLOP/s of the layer (sparse FLOPs actually performed + the paper's
low-rank count 8 B H N d_h r, over the layer time), ms per layer (wall clock over the timed steps,
and the median / p10 / p90 of the per-step spans), the roofline of the dominant kernel (block-sparse
attention against the bf16 MFMA peak, timed with HIP events on its stream), the layer-level roofline
fraction, and the CPU oracle timed on a bounded sample of the same layer.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2609_06712_amd import synth  # noqa: E402

METRIC = "ms/attention layer + eff. TFLOP/s at Wan-14B 720p shape, 90% sparsity; % roofline"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sparse_attn_wan14b_720p_traffic.txt")
SPARSE_SRC = os.path.join(ROOT, "paper_2609_06712_amd", "csrc", "sparse_attn.hip")


def source_digest(path: str) -> str:
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic():
    """HBM bytes per launch of the sparse kernel from the committed counter summary (FETCH_SIZE and
    WRITE_SIZE, each calibrated on a plain copy of known size), or None when the kernel source has
    changed since the counters were taken."""
    try:
        rec = {}
        with open(TRAFFIC_FILE) as f:
            for line in f:
                if "=" in line and not line.startswith("#"):
                    k, v = line.split("=", 1)
                    rec[k.strip()] = v.strip()
        if rec.get("source_sha256") != source_digest(SPARSE_SRC):
            return None
        return float(rec["bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def sparse_flops_performed(idx: torch.Tensor, N: int, block: int, d: int) -> float:
    """4 d |I_valid| |K(I)_valid| summed over (b, h, query block): QK^T and PV on valid tokens."""
    nb = idx.shape[2]
    sizes = torch.full((nb,), block, dtype=torch.float64, device=idx.device)
    sizes[-1] = N - (nb - 1) * block
    keys = sizes[idx.long()].sum(dim=-1)            # [B, H, nb] valid keys per query block
    return float(4.0 * d * (keys * sizes).sum())


def summary_bytes(w) -> float:
    """HBM bytes the low-rank summary must move: K^n and V (2-byte elements) plus the rotary-table
    columns it uses."""
    return float(w.B * w.H * w.N * 2 * w.d_h * 2 + 2 * w.N * (w.r // 2) * 4)


CPU_HEADS = (0, 13, 26, 39)


def _oracle_head_worker(job):
    """One (b, h) of the layer through the oracle (every step of forward_head), BLAS on one thread."""
    import math
    from threadpoolctl import threadpool_limits
    import oracle as O
    path, h, grid, split, base, block, sparsity, dtype = job
    d = np.load(path)
    with threadpool_limits(1):
        t0 = time.perf_counter()
        cos, sin = O.rope_tables(*grid, split, base)
        r = O.forward_head(d["Qn"], d["Kn"], d["V"], d["Pq"], d["Pk"], d["logits"], cos, sin,
                           block=block, sparsity=sparsity, dtype=dtype)
        dt = time.perf_counter() - t0
    N, dh = d["Qn"].shape
    sizes = np.full(O.num_blocks(N, block), block, dtype=np.float64)
    sizes[-1] = N - (len(sizes) - 1) * block
    f_sparse = 4.0 * dh * float((sizes[r["idx"]].sum(axis=1) * sizes).sum())
    f_lowrank = 8.0 * N * dh * d["Pq"].shape[0]
    return h, dt, f_sparse + f_lowrank, math.isfinite(float(np.abs(r["out"]).max()))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, heads: dict, tmpdir: str) -> dict:
    """The fp64 oracle, as it stands, on the heads CPU_HEADS of the layer: one process per head
    (spawned, BLAS on one thread each), every step of the module over the whole sequence. Reports the
    oracle's throughput over the sample, the mean time per head and the layer time that implies
    (per head x H, labelled extrapolated)."""
    import multiprocessing as mp
    jobs = []
    for h, arrs in heads.items():
        path = os.path.join(tmpdir, f"oracle_head{h}.npz")
        np.savez(path, **arrs)
        jobs.append((path, h, w.grid, w.split, w.base, w.block, w.sparsity, w.dtype))
    t0 = time.perf_counter()
    with mp.get_context("spawn").Pool(len(jobs)) as pool:
        res = pool.map(_oracle_head_worker, jobs)
    wall = time.perf_counter() - t0
    assert all(ok for *_, ok in res)
    flops = sum(f for _, _, f, _ in res)
    per_head = float(np.mean([dt for _, dt, _, _ in res]))
    return {"value": flops / wall / 1e12, "unit": "TFLOP/s", "cores": len(jobs), "kind": "oracle",
            "sample": f"heads {list(heads)} of {w.H}, every step of the layer over all {w.N} tokens, "
                      f"one spawned process per head with BLAS on one thread; {wall:.1f} s wall",
            "cpu_model": cpu_model(), "host_cores_available": len(os.sched_getaffinity(0)),
            "s_per_head": round(per_head, 2),
            "layer_s_extrapolated": round(per_head * w.H * w.B, 1),
            "layer_s_extrapolated_note": "mean time per (b, h) on one core x B*H: extrapolated"}


def gemm_reference(dev, n: int = 16384, reps: int = 8) -> dict:
    """The dense bf16 rate this machine sustains for the plainest contraction: torch.matmul (the
    vendor GEMM library) on random n x n bf16 operands, HIP events like the layer. Context for the
    attention kernel's fraction of the published peak, not a bound on it."""
    g = torch.Generator(device=dev).manual_seed(0)
    a = torch.randn(n, n, dtype=torch.bfloat16, device=dev, generator=g)
    b = torch.randn(n, n, dtype=torch.bfloat16, device=dev, generator=g)
    c = torch.empty(n, n, dtype=torch.bfloat16, device=dev)
    for _ in range(2):
        torch.matmul(a, b, out=c)
    ms = time_call(lambda: torch.matmul(a, b, out=c), reps)[0]
    del a, b, c
    torch.cuda.empty_cache()
    tf = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    return {"what": f"torch.matmul, random bf16 {n}x{n} operands (vendor GEMM library), same box",
            "achieved": round(tf, 1), "unit": "TFLOP/s", "frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4)}


def time_call(fn, reps: int, cold=None):
    """Median, p10, p90 (ms) of fn() over reps runs, HIP events on the current stream; cold() runs
    between the timed intervals (e.g. a scratch write that evicts the caches)."""
    fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    out = []
    for _ in range(reps):
        if cold is not None:
            cold()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        fn()
        b.record(st)
        b.synchronize()
        out.append(a.elapsed_time(b))
    return float(np.median(out)), float(np.percentile(out, 10)), float(np.percentile(out, 90))


def sweep(reps: int) -> None:
    """Measurement sweeps besides the headline line, printed as markdown: the 1.3B 480p layer, the
    low-rank branch over N x r (summary and readout separately, warm and cold cache) and the sparse
    branch over sparsity x block size with the dense reference."""
    from paper_2609_06712_amd import rola as R
    dev = torch.device("cuda:0")
    scratch = torch.empty(1 << 30, dtype=torch.uint8, device=dev)   # 1 GiB: evicts L2 and MALL
    evict = lambda: scratch.fill_(1)  # noqa: E731

    # the 1.3B 480p layer: the headline's two-stream step
    w = synth.WAN_1_3B_480P
    L = LayerStep(R, w, dev)
    L.step()
    torch.cuda.synchronize()
    ms, lo, hi = time_call(L.step, reps)
    f = sparse_flops_performed(L.idx, w.N, w.block, w.d_h) + 8.0 * w.B * w.H * w.N * w.d_h * w.r
    print(f"## Layer, {w.name}\n\n| ms (median) | p10 | p90 | eff. TFLOP/s |\n|---|---|---|---|")
    print(f"| {ms:.3f} | {lo:.3f} | {hi:.3f} | {f / ms / 1e9:.1f} |\n", flush=True)
    del L

    # low-rank branch: N x r, summary and readout separately (warm / cold cache)
    print("## Low-rank branch, H40 d128 bf16 (HBM roofline 8 TB/s)\n")
    print("| N | r | kernel | bytes (MB) | warm ms | warm GB/s | cold ms | cold GB/s | cold % of 8 TB/s |")
    print("|---|---|---|---|---|---|---|---|---|", flush=True)
    for N in (8400, 32760, 75600):
        for r in (16, 32, 64):
            w = synth.lowrank_sweep(N, r)
            g = w.grid
            inp = synth.make_inputs(w, 0, device=dev)
            prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
            cos, sin = R.rola_rope_tables(prob, w.split, w.base)
            tensor = w.B * w.H * w.N * w.d_h * 2
            tables = 2 * w.N * (r // 2) * 4
            C, z = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], r, cos, sin, g)
            ws = torch.empty(R.summary_workspace_bytes(prob, r), dtype=torch.uint8, device=dev)
            olr = torch.empty_like(inp["Qn"])
            out = torch.empty_like(inp["Qn"])
            cases = [
                ("summary", 2 * tensor + tables,
                 lambda: R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], r, cos, sin, g, C=C,
                                                z=z, ws=ws)),
                ("readout", 2 * tensor + tables,
                 lambda: R.rola_lowrank_readout(inp["Qn"], inp["Pq"], r, cos, sin, C, g, out=olr)),
                ("readout+combine", 3 * tensor + tables,
                 lambda: R.rola_lowrank_readout_combine(inp["Qn"], inp["Pq"], r, cos, sin, C, inp["V"],
                                                        inp["logits"], g, out=out)),
            ]
            for name, nbytes, fn in cases:
                wm = time_call(fn, reps)[0]
                cm = time_call(fn, reps, cold=evict)[0]
                print(f"| {N} | {r} | {name} | {nbytes / 1e6:.0f} | {wm:.4f} | {nbytes / wm / 1e6:.0f} | "
                      f"{cm:.4f} | {nbytes / cm / 1e6:.0f} | {100 * nbytes / cm / 1e6 / PEAK_HBM_GBS:.1f} |",
                      flush=True)
            del inp, C, z, ws, olr, out
    print()

    # feature-map variants of the low-rank branch at the 14B shape (Sec. 5.1, Sec. 5.3)
    print("## Low-rank feature variants, H40 d128 N75600 r32 bf16 (warm cache)\n")
    print("| phi | rotation | summary ms | summary GB/s | readout+combine ms | readout+combine GB/s |")
    print("|---|---|---|---|---|---|", flush=True)
    w = synth.lowrank_sweep(75600, 32)
    g = w.grid
    inp = synth.make_inputs(w, 0, device=dev)
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split, w.base)
    tensor = w.B * w.H * w.N * w.d_h * 2
    tables = 2 * w.N * 16 * 4
    ws = torch.empty(R.summary_workspace_bytes(prob, 32), dtype=torch.uint8, device=dev)
    C, z = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], 32, cos, sin, g)
    out = torch.empty_like(inp["Qn"])
    for phi, order in (("silu", "outside"), ("identity", "outside"), ("tanh", "outside"),
                       ("relu", "outside"), ("gelu", "outside"), ("silu", "inside"), ("silu", "none")):
        sm = time_call(lambda: R.rola_lowrank_summary_ex(inp["Kn"], inp["V"], inp["Pk"], 32, cos, sin,
                                                         g, phi, order, C=C, z=z, ws=ws), reps)[0]
        rm = time_call(lambda: R.rola_lowrank_readout_combine_ex(
            inp["Qn"], inp["Pq"], 32, cos, sin, C, inp["V"], inp["logits"], g, phi, order, out=out),
            reps)[0]
        print(f"| {phi} | {order} | {sm:.4f} | {(2 * tensor + tables) / sm / 1e6:.0f} | {rm:.4f} | "
              f"{(3 * tensor + tables) / rm / 1e6:.0f} |", flush=True)
    del inp, C, z, ws, out
    print()

    # gate logits X W_g + b_g (Sec. 4.4; Algorithm step 8) at the 14B 720p shape
    print("## Gate logits X W_g + b_g, N 75600, d_model 5120 bf16 (HBM roofline 8 TB/s)\n")
    print("| bytes (MB) | warm ms | warm GB/s | cold ms | cold GB/s | cold % of 8 TB/s |")
    print("|---|---|---|---|---|---|", flush=True)
    gen = torch.Generator(device=dev).manual_seed(5)
    X = torch.randn((1, 75600, 5120), generator=gen, device=dev).to(torch.bfloat16)
    Wg = (torch.randn((5120,), generator=gen, device=dev) / 5120 ** 0.5).to(torch.bfloat16)
    lg = torch.empty((1, 75600), dtype=torch.float32, device=dev)
    nbytes = X.numel() * 2 + lg.numel() * 4
    fn = lambda: R.rola_gate_logits(X, Wg, -1.946, (21, 45, 80), out=lg)  # noqa: E731
    wm = time_call(fn, reps)[0]
    cm = time_call(fn, reps, cold=evict)[0]
    print(f"| {nbytes / 1e6:.0f} | {wm:.4f} | {nbytes / wm / 1e6:.0f} | {cm:.4f} | {nbytes / cm / 1e6:.0f} | "
          f"{100 * nbytes / cm / 1e6 / PEAK_HBM_GBS:.1f} |\n", flush=True)
    del X, Wg, lg

    # sparse branch: sparsity x block, dense reference
    print("## Sparse branch, H40 d128 N75600 bf16 (MFMA roofline 2.5 PFLOP/s)\n")
    print("| block | sparsity | keep | select ms | sparse ms | TFLOP/s performed | % of peak | "
          "sparse/dense time | keep/n_b |")
    print("|---|---|---|---|---|---|---|---|---|", flush=True)
    base = synth.sparse_sweep(0.9, 64)
    inp = synth.make_inputs(base, 0, device=dev)
    g = base.grid
    prob = R.problem(base.B, base.H, base.N, base.d_h, g, base.dtype)
    cos, sin = R.rola_rope_tables(prob, base.split, base.base)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    o_s = torch.empty_like(qr)
    for block in (64, 128):
        nb = R.num_blocks(base.N, block)
        dense_ms = time_call(lambda: R.rola_dense_attn(qr, kr, inp["V"], g, block, out=o_s), max(3, reps // 4))[0]
        f_dense = 4.0 * base.B * base.H * base.N * base.N * base.d_h
        for s in (0.8, 0.9, 0.95):
            keep = R.keep_blocks(nb, s)
            idx = R.rola_block_select(qr, kr, g, block, s)
            ws = torch.empty(max(R.sparse_workspace_bytes(prob, block, s), 16), dtype=torch.uint8,
                             device=dev)
            sel_ms = time_call(lambda: R.rola_block_select(qr, kr, g, block, s, out=idx), reps)[0]
            sp_ms = time_call(lambda: R.rola_sparse_attn(qr, kr, inp["V"], g, block, s, idx, out=o_s,
                                                         ws=ws), reps)[0]
            f = sparse_flops_performed(idx, base.N, block, base.d_h)
            print(f"| {block} | {s} | {keep} | {sel_ms:.3f} | {sp_ms:.3f} | {f / sp_ms / 1e9:.1f} | "
                  f"{100 * f / sp_ms / 1e9 / PEAK_BF16_TFLOPS:.1f} | {sp_ms / dense_ms:.4f} | "
                  f"{keep / nb:.4f} |", flush=True)
        print(f"| {block} | dense | {nb} | - | {dense_ms:.3f} | {f_dense / dense_ms / 1e9:.1f} | "
              f"{100 * f_dense / dense_ms / 1e9 / PEAK_BF16_TFLOPS:.1f} | 1 | 1 |", flush=True)


def train_bench(reps: int) -> None:
    """Forward (keeping what the backward needs) and backward of the module at the 14B 720p shape,
    per entry point, printed as markdown."""
    from paper_2609_06712_amd import rola as R
    w = synth.WAN_14B_720P
    g = w.grid
    dev = torch.device("cuda:0")
    inp = synth.make_inputs(w, 0, device=dev)
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split, w.base)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    idx = R.rola_block_select(qr, kr, g, w.block, w.sparsity)
    os_, lse = R.rola_sparse_attn_lse(qr, kr, inp["V"], g, w.block, w.sparsity, idx)
    C, _ = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g)
    dO = torch.randn_like(os_)
    f_fwd = sparse_flops_performed(idx, w.N, w.block, w.d_h)
    ws_sp = torch.empty(R.LIB.rola_sparse_backward_workspace_bytes(ctypes.byref(prob), w.block,
                                                                    w.sparsity), dtype=torch.uint8,
                        device=dev)
    ws_lr = torch.empty(R.LIB.rola_lowrank_backward_workspace_bytes(ctypes.byref(prob), w.r),
                        dtype=torch.uint8, device=dev)
    dOs = R.rola_lowrank_backward(inp["Qn"], inp["Kn"], inp["V"], inp["Pq"], inp["Pk"], w.r, cos, sin,
                                  C, os_, inp["logits"], dO, g, ws=ws_lr)[0]
    # the paper's default rank: projections of rank 64 drawn like the workload's own
    r64 = 64
    gen = torch.Generator(device=dev)
    gen.manual_seed(64)
    P64 = [(torch.randn((w.H, r64, w.d_h), generator=gen, device=dev) / w.d_h ** 0.5).to(torch.bfloat16)
           for _ in range(2)]
    C64, _ = R.rola_lowrank_summary(inp["Kn"], inp["V"], P64[1], r64, cos, sin, g)
    ws_lr64 = torch.empty(R.LIB.rola_lowrank_backward_workspace_bytes(ctypes.byref(prob), r64),
                          dtype=torch.uint8, device=dev)
    # HBM bytes the low-rank backward must move: Q^n, K^n, V, O^s, dO read and dO^s written (bf16),
    # dQ^n, dK^n, dV written (fp32)
    act = w.B * w.H * w.N * w.d_h
    lr_bytes = 6 * 2 * act + 3 * 4 * act
    rows = [
        ("sparse forward with lse", lambda: R.rola_sparse_attn_lse(qr, kr, inp["V"], g, w.block,
                                                                   w.sparsity, idx, out=os_, lse=lse),
         f_fwd, None),
        (f"low-rank + fusion backward, r {w.r}", lambda: R.rola_lowrank_backward(
            inp["Qn"], inp["Kn"], inp["V"], inp["Pq"], inp["Pk"], w.r, cos, sin, C, os_,
            inp["logits"], dO, g, ws=ws_lr), None, lr_bytes),
        (f"low-rank + fusion backward, r {r64}", lambda: R.rola_lowrank_backward(
            inp["Qn"], inp["Kn"], inp["V"], P64[0], P64[1], r64, cos, sin, C64, os_,
            inp["logits"], dO, g, ws=ws_lr64), None, lr_bytes),
        ("sparse attention backward", lambda: R.rola_sparse_attn_backward(
            qr, kr, inp["V"], g, w.block, w.sparsity, idx, os_, lse, dOs, ws=ws_sp), 2.5 * f_fwd, None),
    ]
    print("## Fine-tuning pass of the module, " + w.name + "\n")
    print("| step | ms (median) | TFLOP/s (algorithmic) | % of bf16 peak | TB/s (algorithmic bytes) | "
          "% of HBM peak |")
    print("|---|---|---|---|---|---|", flush=True)
    for name, fn, flops, nbytes in rows:
        ms = time_call(fn, reps)[0]
        tf = f"{flops / ms / 1e9:.1f}" if flops else "-"
        pc = f"{100 * flops / ms / 1e9 / PEAK_BF16_TFLOPS:.1f}" if flops else "-"
        tb = f"{nbytes / ms / 1e9:.2f}" if nbytes else "-"
        pb = f"{100 * nbytes / ms / 1e6 / PEAK_HBM_GBS:.1f}" if nbytes else "-"
        print(f"| {name} | {ms:.3f} | {tf} | {pc} | {tb} | {pb} |", flush=True)
    print()


def dit_bench(reps: int) -> None:
    """Per-block time of a synthetic Wan-shaped DiT block (random weights) with the RoLA module or
    the dense attention kernel as its self-attention, and the implied DiT time per denoising step
    (blocks x block time, one forward, no CFG). Printed as markdown."""
    from paper_2609_06712_amd import dit_block as DB
    print("## Synthetic Wan-shaped DiT block (random weights), bf16\n")
    print("| model | grid | attention | self-attention ms | block ms | blocks | DiT ms per step | "
          "dense / RoLA per step |")
    print("|---|---|---|---|---|---|---|---|", flush=True)
    for shape in (DB.WAN_1_3B_480P, DB.WAN_14B_720P):
        x, ctx = DB.inputs(shape)
        res = {}
        for attn in ("dense", "rola"):
            blk = DB.DiTBlock(shape, attn=attn)
            h = torch.randn_like(x)
            sa = time_call(lambda: blk.self_attention(h), max(2, reps // 2 if attn == "dense" else reps))[0]
            bm = time_call(lambda: blk.forward(x, ctx), max(2, reps // 2 if attn == "dense" else reps))[0]
            res[attn] = bm
            ratio = f"{res['dense'] / bm:.2f}" if attn == "rola" else "-"
            print(f"| {shape.name} | {'x'.join(map(str, shape.grid))} | {attn} | {sa:.2f} | {bm:.2f} | "
                  f"{shape.layers} | {bm * shape.layers:.0f} | {ratio} |", flush=True)
            del blk, h
            torch.cuda.empty_cache()
        del x, ctx
    print()


class LayerStep:
    """The timed layer (steps a1-a5 of the hot path; the backbone's rotation is the input) on two
    HIP streams, with its inputs and buffers for workload w. Main stream: the block means of Q^r and
    K^r (with each key block's largest key norm), the block scores and top-k, the attention's
    pairing and list merge; side stream, forked once the block lists exist: the low-rank summary,
    beside the pairing, whose passes are latency-bound (its greedy pass keeps one wave per head
    busy) and leave the chip's bandwidth to the summary. Forked after the pooling instead, the
    summary slows the score and top-k kernels beside it by more than it saves (0.1 ms per layer).
    After both: the block-sparse attention with the low-rank readout and the gated combine in its
    epilogue (O^s and O^lr never reach memory), given the key norms so that it can take the score
    bound as its softmax reference. step(rotate=True) starts from Q^n, K^n: the rotating pooling
    passes write Q^r and K^r (Algorithm step 3 fused with the pooling)."""
    NAMES = ["pool", "select", "plan", "attention_readout_combine"]

    def __init__(self, R, w, dev):
        self.R, self.w = R, w
        g = w.grid
        self.inp = inp = synth.make_inputs(w, 0, device=dev)
        self.prob = prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
        self.cos, self.sin = R.rola_rope_tables(prob, w.split, w.base)
        self.qr = R.rola_rope_apply(inp["Qn"], self.cos, self.sin, g)
        self.kr = R.rola_rope_apply(inp["Kn"], self.cos, self.sin, g)
        nb = R.num_blocks(w.N, w.block)
        self.keep = R.keep_blocks(nb, w.sparsity)
        self.idx = torch.empty((w.B, w.H, nb, self.keep), dtype=torch.int32, device=dev)
        u8 = dict(dtype=torch.uint8, device=dev)
        self.ws_sel = torch.empty(R.select_workspace_bytes(prob, w.block), **u8)
        self.ws_sum = torch.empty(R.summary_workspace_bytes(prob, w.r), **u8)
        self.ws_sp = torch.empty(R.sparse_combine_workspace_bytes(prob, w.block, w.sparsity, w.r), **u8)
        self.ws_pool = torch.empty(R.LIB.rola_select_pooled_workspace_bytes(ctypes.byref(prob),
                                                                            w.block), **u8)
        self.out = torch.empty_like(inp["Qn"])
        self.C = torch.empty((w.B, w.H, w.r, w.d_h), dtype=torch.float32, device=dev)
        self.z = torch.empty((w.B, w.H, w.r), dtype=torch.float32, device=dev)
        self.qbar = torch.empty((w.B, w.H, nb, w.d_h), dtype=torch.float32, device=dev)
        self.kbar = torch.empty_like(self.qbar)
        self.knorm = torch.empty((w.B, w.H, nb), dtype=torch.float32, device=dev)
        self.main_st = torch.cuda.current_stream()
        self.side_st = torch.cuda.Stream(device=dev)  # default priority

    def step(self, ev=None, sev=None, rotate=False):
        """One layer; ev: 5 timing events on the main stream around the NAMES spans, sev: 2 around
        the summary on the side stream."""
        R, w, inp, g = self.R, self.w, self.inp, self.w.grid
        main_st, side_st = self.main_st, self.side_st

        def mark(i):
            if ev is not None:
                ev[i].record(main_st)
        fork, join = torch.cuda.Event(), torch.cuda.Event()
        mark(0)
        if rotate:
            R.rola_rope_pool(inp["Qn"], self.cos, self.sin, g, w.block, xr=self.qr, xbar=self.qbar)
            R.rola_rope_pool(inp["Kn"], self.cos, self.sin, g, w.block, xr=self.kr, xbar=self.kbar,
                             xnorm=self.knorm)
        else:
            R.rola_rope_pool(self.qr, None, None, g, w.block, xbar=self.qbar)
            R.rola_rope_pool(self.kr, None, None, g, w.block, xbar=self.kbar, xnorm=self.knorm)
        mark(1)
        R.rola_block_select_pooled(self.qbar, self.kbar, self.kr, g, w.block, w.sparsity,
                                   out=self.idx, ws=self.ws_pool)
        mark(2)
        fork.record(main_st)
        side_st.wait_event(fork)
        if sev is not None:
            sev[0].record(side_st)
        R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, self.cos, self.sin, g, C=self.C,
                               z=self.z, ws=self.ws_sum, stream=side_st)
        if sev is not None:
            sev[1].record(side_st)
        join.record(side_st)
        R.rola_sparse_plan(self.idx, self.kr, g, w.block, w.sparsity, w.r, self.ws_sp)
        main_st.wait_event(join)
        mark(3)
        R.rola_sparse_attn_combine_planned(self.qr, self.kr, inp["V"], g, w.block, w.sparsity,
                                           self.idx, inp["Qn"], inp["Pq"], w.r, self.cos, self.sin,
                                           self.C, inp["logits"], self.ws_sp, out=self.out,
                                           key_norm=self.knorm)
        mark(4)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--quick", action="store_true",
                    help="only the timed steps (for profiler runs): no comparison timings")
    ap.add_argument("--sweep", action="store_true",
                    help="print the measurement sweeps (1.3B layer, low-rank N x r, sparse S x block) "
                         "as markdown instead of the JSON line")
    ap.add_argument("--sweep-reps", type=int, default=10)
    ap.add_argument("--train", action="store_true",
                    help="time the module's fine-tuning forward and backward at the 14B shape")
    ap.add_argument("--dit", action="store_true",
                    help="time a synthetic Wan-shaped DiT block with RoLA vs dense self-attention")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="one untimed device copy of one activation tensor (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}); the layer shards by "
              "(batch, head) with no communication, so N GPUs each run this single-GPU workload on "
              "their share of the heads", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(2)

    if args.sweep:
        sweep(args.sweep_reps)
        return
    if args.dit:
        dit_bench(args.sweep_reps)
        return
    if args.train:
        train_bench(args.sweep_reps)
        return
    from paper_2609_06712_amd import rola as R

    w = synth.WAN_14B_720P
    g = w.grid
    dev = torch.device("cuda:0")
    print(f"[bench] generating {w.name} inputs", file=sys.stderr, flush=True)
    L = LayerStep(R, w, dev)
    inp, cos, sin, qr, kr, idx, out, C, z = L.inp, L.cos, L.sin, L.qr, L.kr, L.idx, L.out, L.C, L.z
    ws_sel, ws_sum, ws_sp, prob, keep = L.ws_sel, L.ws_sum, L.ws_sp, L.prob, L.keep
    names, step = LayerStep.NAMES, L.step

    if args.calibration_copy:  # a plain copy of known size, for scaling FETCH_SIZE / WRITE_SIZE
        scratch = torch.empty_like(inp["V"])
        scratch.copy_(inp["V"])
        torch.cuda.synchronize()
        del scratch
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev_t = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    events = [[ev_t() for _ in range(len(names) + 1)] for _ in range(args.steps)]
    side_events = [[ev_t(), ev_t()] for _ in range(args.steps)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k], side_events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_kernel = {n: [] for n in names}
    spans = []
    for ev in events:
        for i, n in enumerate(names):
            per_kernel[n].append(ev[i].elapsed_time(ev[i + 1]))
        spans.append(ev[0].elapsed_time(ev[-1]))
    per_kernel["summary (side stream)"] = [a.elapsed_time(b) for a, b in side_events]
    kern_ms = {n: float(np.mean(v)) for n, v in per_kernel.items()}
    ms = wall * 1e3 / args.steps

    # the summary alone on one stream (its bandwidth without the selection running beside it)
    sum_ms = time_call(lambda: R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin,
                                                      g, C=C, z=z, ws=ws_sum), 20)[0] if not args.quick \
        else float("nan")
    # the layer as one stream of the three plain calls (selection, summary, attention with its
    # epilogue), and the same preceded by the backbone's rotation of Q^n and K^n; the two-stream
    # layer starting from Q^n, K^n (rotation fused with the pooling)
    def one_stream():
        R.rola_block_select(qr, kr, g, w.block, w.sparsity, out=idx, ws=ws_sel)
        R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g, C=C, z=z, ws=ws_sum)
        R.rola_sparse_attn_combine(qr, kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"],
                                   inp["Pq"], w.r, cos, sin, C, inp["logits"], out=out, ws=ws_sp)

    def one_stream_rotating():
        R.rola_rope_apply(inp["Qn"], cos, sin, g, out=qr)
        R.rola_rope_apply(inp["Kn"], cos, sin, g, out=kr)
        one_stream()
    nan3 = (float("nan"),) * 3
    one_ms = time_call(one_stream, 10) if not args.quick else nan3
    one_rot_ms = time_call(one_stream_rotating, 10) if not args.quick else nan3
    rot_ms = time_call(lambda: step(rotate=True), 10) if not args.quick else nan3

    f_sparse = sparse_flops_performed(idx, w.N, w.block, w.d_h)
    f_lowrank = 8.0 * w.B * w.H * w.N * w.d_h * w.r
    eff = (f_sparse + f_lowrank) / (ms * 1e-3) / 1e12
    attn_ms = kern_ms["attention_readout_combine"]
    achieved = f_sparse / (attn_ms * 1e-3) / 1e12
    sum_gbs = summary_bytes(w) / (sum_ms * 1e-3) / 1e9
    tensor = w.B * w.H * w.N * w.d_h * 2
    # HBM bytes the streaming steps must move: the pooling reads Q^r and K^r; the summary reads K^n
    # and V (+ its table columns); the epilogue reads Q^n and writes O
    layer_bytes = 2 * tensor + summary_bytes(w) + 2 * tensor
    layer_floor_ms = (f_sparse / (PEAK_BF16_TFLOPS * 1e12) + layer_bytes / (PEAK_HBM_GBS * 1e9)) * 1e3
    med, p10, p90 = (float(np.percentile(spans, q)) for q in (50, 10, 90))

    res = {
        "metric": METRIC, "value": round(eff, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded smooth-field-plus-noise Q/K/V, random P_q/P_k, gate logits)",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "grid": list(g), "d_h": w.d_h,
                   "block": w.block, "sparsity": w.sparsity, "keep": keep, "r": w.r,
                   "parallelism": "single GPU", "streams": 2,
                   "step": "block selection, sparse attention, low-rank summary and readout, gated "
                           "combine from Q^r, K^r, Q^n, K^n, V (the backbone's rotation untimed)"},
        "ms_per_step_spans": {"median": round(med, 4), "p10": round(p10, 4), "p90": round(p90, 4)},
        "ms_per_step_one_stream": {
            "median": round(one_ms[0], 4), "p10": round(one_ms[1], 4), "p90": round(one_ms[2], 4),
            "note": "rola_block_select, rola_lowrank_summary, rola_sparse_attn_combine on one stream"},
        "ms_per_step_from_qn_kn": {
            "two_streams_rotating_pooling": round(rot_ms[0], 4),
            "one_stream_rope_apply_then_layer": round(one_rot_ms[0], 4),
            "note": "medians; the layer including the backbone's rotation R(Q^n), R(K^n) (Algorithm "
                    "step 3): fused with the pooling passes, or as two rola_rope_apply calls"},
        "roofline": {"bound": "mfma", "kernel": "sparse_attn_kernel via "
                     "rola_sparse_attn_combine_planned (block-sparse attention with the low-rank "
                     "readout and gated combine in its epilogue; the call also runs the 4 us "
                     "C-fragment kernel)",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic()},
        "layer_roofline": {"frac": round(layer_floor_ms / ms, 4),
                           "floor_ms": round(layer_floor_ms, 4),
                           "definition": "(F_sparse / 2.5 PFLOP/s + streamed bytes / 8 TB/s) / "
                                         "ms_per_step",
                           "streamed_bytes": layer_bytes},
        "summary_roofline": {"bound": "hbm", "kernels": "rola_lowrank_summary (alone, one stream)",
                             "achieved": round(sum_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                             "frac": round(sum_gbs / PEAK_HBM_GBS, 4)},
        "kernels_ms": {k: round(v, 4) for k, v in kern_ms.items()},
        "flops": {"sparse_performed": f_sparse, "lowrank_paper": f_lowrank,
                  "sparse_paper_formula": 4.0 * w.B * w.H * w.N ** 2 * (1 - w.sparsity) * w.d_h},
    }
    if not args.quick:
        ref = gemm_reference(dev)
        ref["attention_vs_gemm"] = round(achieved / ref["achieved"], 4)
        res["gemm_reference"] = ref
    if not args.no_cpu_baseline:
        import tempfile
        print("[bench] timing the CPU oracle on 4 heads", file=sys.stderr, flush=True)
        heads = {}
        for h in CPU_HEADS:
            heads[h] = {k: inp[k][0, h].double().cpu().numpy() for k in ("Qn", "Kn", "V")}
            heads[h].update(Pq=inp["Pq"][h].double().cpu().numpy(),
                            Pk=inp["Pk"][h].double().cpu().numpy(),
                            logits=inp["logits"][0].double().cpu().numpy())
        with tempfile.TemporaryDirectory() as tmp:
            res["cpu_baseline"] = cpu_baseline(w, heads, tmp)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
