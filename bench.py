"""Benchmark of one RoLA attention layer (sparse + rotary low-rank branches) on one MI355X.

One step = the whole hot path over one batch of synthetic input already resident in HBM:
block selection -> block-sparse attention -> low-rank summary -> fused low-rank readout + gated combine,
each a call of the C ABI on one HIP stream. Workload: the Wan2.1-14B-shaped 720p layer
(B1 H40 d128, 21x45x80 grid = 75600 tokens, block 64, 90 % sparsity -> 118 of 1182 key blocks, r 32,
bf16). The backbone's own steps (rotary tables, Q^r = R(Q^n), K^r = R(K^n)) run once, untimed.

Prints one JSON line: effective TFLOP/s of the layer (sparse FLOPs actually performed + the paper's
low-rank count 8 B H N d_h r, over the layer time), ms per layer, the roofline of the dominant kernel
(block-sparse attention against the bf16 MFMA peak, timed with HIP events on its stream) and the CPU
oracle timed on a bounded sample of the same layer.
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


def cpu_baseline(w, inp_cpu_head0: dict, budget_s: float) -> dict:
    """The fp64 oracle, as it stands, on head 0: the whole low-rank branch (summary over every token)
    plus as many query blocks of selection + sparse attention + readout + combine as fit the budget."""
    import math
    import oracle as O
    from threadpoolctl import threadpool_info

    f64 = synth.to_f64(inp_cpu_head0)
    qn, kn, v = f64["Qn"][0, 0], f64["Kn"][0, 0], f64["V"][0, 0]
    t0 = time.perf_counter()
    cos, sin = O.rope_tables(*w.grid, w.split, w.base)
    qr = O.round_to(O.rotate(qn, cos, sin), w.dtype)
    kr = O.round_to(O.rotate(kn, cos, sin), w.dtype)
    nb = O.num_blocks(w.N, w.block)
    keep = O.keep_blocks(nb, w.sparsity)
    qbar, kbar = O.pool_blocks(qr, w.block), O.pool_blocks(kr, w.block)
    C, _ = O.lowrank_summary(kn, v, f64["Pk"][0], cos, sin)
    flops = 4.0 * w.N * w.d_h * w.r                       # summary: projection + k~ v^T
    scale = 1.0 / math.sqrt(w.d_h)
    n_blocks = 0
    for I in range(nb):
        if time.perf_counter() - t0 > budget_s:
            break
        idx = np.zeros((nb, keep), dtype=np.int64)
        idx[I] = O.select_blocks(O.block_scores(qbar[I:I + 1], kbar), keep)[0]
        rows = np.arange(I * w.block, min(w.N, (I + 1) * w.block))
        o_s = O.sparse_attention_rows(qr, kr, v, idx, w.block, scale, rows)
        u = O.lowrank_features(qn[rows], f64["Pq"][0], cos[rows], sin[rows]) @ C
        O.combine(o_s, O.rms_normalize(u, 1e-6), f64["logits"][0, rows], 1e-6)
        nkeys = sum(min(w.N, (J + 1) * w.block) - J * w.block for J in idx[I])
        flops += 4.0 * w.d_h * len(rows) * nkeys + 4.0 * len(rows) * w.d_h * w.r
        n_blocks += 1
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"head 0 of {w.H}: full low-rank summary over {w.N} tokens + selection, sparse "
                      f"attention, readout and combine for query blocks 0..{n_blocks - 1} of {nb}; "
                      f"{dt:.1f} s on {len(os.sched_getaffinity(0))} host cores"}


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

    # the 1.3B 480p layer (same step as the headline)
    w = synth.WAN_1_3B_480P
    g = w.grid
    inp = synth.make_inputs(w, 0, device=dev)
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split, w.base)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    ws_sp = torch.empty(R.sparse_combine_workspace_bytes(prob, w.block, w.sparsity, w.r),
                        dtype=torch.uint8, device=dev)
    idx = R.rola_block_select(qr, kr, g, w.block, w.sparsity)
    o_s = torch.empty_like(qr)

    def layer():
        R.rola_block_select(qr, kr, g, w.block, w.sparsity, out=idx)
        C, _ = R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g)
        R.rola_sparse_attn_combine(qr, kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"], inp["Pq"],
                                   w.r, cos, sin, C, inp["logits"], out=o_s, ws=ws_sp)
    ms, lo, hi = time_call(layer, reps)
    f = sparse_flops_performed(idx, w.N, w.block, w.d_h) + 8.0 * w.B * w.H * w.N * w.d_h * w.r
    print(f"## Layer, {w.name}\n\n| ms (median) | p10 | p90 | eff. TFLOP/s |\n|---|---|---|---|")
    print(f"| {ms:.3f} | {lo:.3f} | {hi:.3f} | {f / ms / 1e9:.1f} |\n", flush=True)
    del inp, qr, kr, idx, o_s

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
    rows = [
        ("sparse forward with lse", lambda: R.rola_sparse_attn_lse(qr, kr, inp["V"], g, w.block,
                                                                   w.sparsity, idx, out=os_, lse=lse),
         f_fwd),
        ("low-rank + fusion backward", lambda: R.rola_lowrank_backward(
            inp["Qn"], inp["Kn"], inp["V"], inp["Pq"], inp["Pk"], w.r, cos, sin, C, os_,
            inp["logits"], dO, g, ws=ws_lr), None),
        ("sparse attention backward", lambda: R.rola_sparse_attn_backward(
            qr, kr, inp["V"], g, w.block, w.sparsity, idx, os_, lse, dOs, ws=ws_sp), 2.5 * f_fwd),
    ]
    print("## Fine-tuning pass of the module, " + w.name + "\n")
    print("| step | ms (median) | TFLOP/s (algorithmic) | % of bf16 peak |")
    print("|---|---|---|---|", flush=True)
    for name, fn, flops in rows:
        ms = time_call(fn, reps)[0]
        tf = f"{flops / ms / 1e9:.1f}" if flops else "-"
        pc = f"{100 * flops / ms / 1e9 / PEAK_BF16_TFLOPS:.1f}" if flops else "-"
        print(f"| {name} | {ms:.3f} | {tf} | {pc} |", flush=True)
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle time")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    inp = synth.make_inputs(w, 0, device=dev)
    prob = R.problem(w.B, w.H, w.N, w.d_h, g, w.dtype)
    cos, sin = R.rola_rope_tables(prob, w.split, w.base)
    qr = R.rola_rope_apply(inp["Qn"], cos, sin, g)
    kr = R.rola_rope_apply(inp["Kn"], cos, sin, g)
    nb = R.num_blocks(w.N, w.block)
    keep = R.keep_blocks(nb, w.sparsity)
    idx = torch.empty((w.B, w.H, nb, keep), dtype=torch.int32, device=dev)
    ws_sel = torch.empty(R.select_workspace_bytes(prob, w.block), dtype=torch.uint8, device=dev)
    ws_sum = torch.empty(R.summary_workspace_bytes(prob, w.r), dtype=torch.uint8, device=dev)
    ws_sp = torch.empty(R.sparse_combine_workspace_bytes(prob, w.block, w.sparsity, w.r),
                        dtype=torch.uint8, device=dev)
    out = torch.empty_like(inp["Qn"])
    C = torch.empty((w.B, w.H, w.r, w.d_h), dtype=torch.float32, device=dev)
    z = torch.empty((w.B, w.H, w.r), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    # the layer: selection, low-rank summary, then the sparse attention with the low-rank readout
    # and the gated combine in its epilogue (O^s and O^lr never reach memory)
    names = ["select", "summary", "sparse_readout_combine"]

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record(stream)
        mark(0)
        R.rola_block_select(qr, kr, g, w.block, w.sparsity, out=idx, ws=ws_sel)
        mark(1)
        R.rola_lowrank_summary(inp["Kn"], inp["V"], inp["Pk"], w.r, cos, sin, g, C=C, z=z, ws=ws_sum)
        mark(2)
        R.rola_sparse_attn_combine(qr, kr, inp["V"], g, w.block, w.sparsity, idx, inp["Qn"],
                                   inp["Pq"], w.r, cos, sin, C, inp["logits"], out=out, ws=ws_sp)
        mark(3)

    if args.calibration_copy:  # a plain copy of known size, for scaling FETCH_SIZE / WRITE_SIZE
        scratch = torch.empty_like(inp["V"])
        scratch.copy_(inp["V"])
        torch.cuda.synchronize()
        del scratch
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
              for _ in range(args.steps)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_kernel = {n: [] for n in names}
    for ev in events:
        for i, n in enumerate(names):
            per_kernel[n].append(ev[i].elapsed_time(ev[i + 1]))
    kern_ms = {n: float(np.mean(v)) for n, v in per_kernel.items()}
    ms = wall * 1e3 / args.steps

    f_sparse = sparse_flops_performed(idx, w.N, w.block, w.d_h)
    f_lowrank = 8.0 * w.B * w.H * w.N * w.d_h * w.r
    eff = (f_sparse + f_lowrank) / (ms * 1e-3) / 1e12
    achieved = f_sparse / (kern_ms["sparse_readout_combine"] * 1e-3) / 1e12
    sum_gbs = summary_bytes(w) / (kern_ms["summary"] * 1e-3) / 1e9

    res = {
        "metric": METRIC, "value": round(eff, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded smooth-field-plus-noise Q/K/V, random P_q/P_k, gate logits)",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "grid": list(g), "d_h": w.d_h,
                   "block": w.block, "sparsity": w.sparsity, "keep": keep, "r": w.r,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "rola_sparse_attn_combine (block-sparse attention "
                     "with the low-rank readout and gated combine in its epilogue)",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic()},
        "summary_roofline": {"bound": "hbm", "kernels": "rola_lowrank_summary",
                             "achieved": round(sum_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                             "frac": round(sum_gbs / PEAK_HBM_GBS, 4)},
        "kernels_ms": {k: round(v, 4) for k, v in kern_ms.items()},
        "flops": {"sparse_performed": f_sparse, "lowrank_paper": f_lowrank,
                  "sparse_paper_formula": 4.0 * w.B * w.H * w.N ** 2 * (1 - w.sparsity) * w.d_h},
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        head0 = {k: inp[k][:, :1].cpu() for k in ("Qn", "Kn", "V")}
        head0.update(Pq=inp["Pq"][:1].cpu(), Pk=inp["Pk"][:1].cpu(), logits=inp["logits"].cpu())
        res["cpu_baseline"] = cpu_baseline(w, head0, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
