"""Seeded synthetic inputs shaped like Wan2.1 attention activations.

This module only draws inputs. It holds none of the attention module's arithmetic (no rotary tables,
no rotation, no projection), so both the GPU path and the CPU oracle can consume what it produces.

Recipe (one per tensor, seeded by (config id, tensor id)):
  * Q^n, K^n, V: for every (batch, head, channel) a smooth field over the T x Hs x Ws latent grid,
    field(t, y, x) = sum_{m<4} a_m sin(2 pi (f_t t/T + f_y y/Hs + f_x x/Ws) + phi_m),
    a_m ~ N(0, 1), f ~ U[0, 2) cycles per axis extent, phi_m ~ U[0, 2 pi), plus N(0, 1) noise.
    Optionally each (batch, head) slice is scaled to unit RMS. Values are rounded once
    (round-to-nearest-even) to the working dtype. The smooth part imitates the "sparse spikes on a
    smooth background" structure of video attention.
  * P_q, P_k: N(0, 1/d_h), shape [H, r, d_h] (the paper's Kaiming-style scale), in the working dtype.
  * gate logits: -1.946 + 0.5 N(0, 1) per (batch, token), fp32 (the paper's initial gate bias).
"""

from __future__ import annotations

import dataclasses
import math

import torch

TENSOR_IDS = {"Qn": 0, "Kn": 1, "V": 2, "Pq": 3, "Pk": 4, "logits": 5}
GATE_BIAS = -1.946


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic attention layer."""
    name: str
    B: int
    H: int
    d_h: int
    grid: tuple            # (T, Hs, Ws); N = T*Hs*Ws tokens in (t, y, x) row-major order
    block: int
    sparsity: float
    r: int
    dtype: str             # "f32" | "bf16"
    split: tuple           # rotary axis widths (d_t, d_y, d_x)
    unit_rms: bool = True
    cfg_id: int = 0
    base: float = 10000.0

    @property
    def N(self) -> int:
        T, Hs, Ws = self.grid
        return T * Hs * Ws

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads the module is specified on.
TINY = Workload("tiny-fp32 B1 H2 d64 grid4x8x8 block32 keep2 r16", 1, 2, 64, (4, 8, 8), 32, 0.75, 16,
                "f32", (28, 18, 18), unit_rms=False, cfg_id=0)
WAN_1_3B_480P = Workload("wan2.1-1.3b-480p H12 d128 grid21x30x52 block64 s0.9 r32", 1, 12, 128,
                         (21, 30, 52), 64, 0.9, 32, "bf16", (44, 42, 42), cfg_id=1)
WAN_14B_720P = Workload("wan2.1-14b-720p H40 d128 grid21x45x80 block64 s0.9 r32", 1, 40, 128,
                        (21, 45, 80), 64, 0.9, 32, "bf16", (44, 42, 42), cfg_id=2)
LOWRANK_GRIDS = {8400: (21, 20, 20), 32760: (21, 30, 52), 75600: (21, 45, 80)}


def lowrank_sweep(N: int, r: int) -> Workload:
    """Low-rank branch sweep point: H40 d128 bf16 on one of the three grids, rank r."""
    return WAN_14B_720P.replace(name=f"lowrank-sweep N{N} r{r}", grid=LOWRANK_GRIDS[N], r=r, cfg_id=3)


def sparse_sweep(sparsity: float, block: int) -> Workload:
    """Sparse branch sweep point at the 14B 720p shape."""
    return WAN_14B_720P.replace(name=f"sparse-sweep s{sparsity} block{block}", sparsity=sparsity,
                                block=block, cfg_id=4)


def torch_dtype(dtype: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def _gen(cfg_id: int, tensor: str, seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + cfg_id) * 16 + TENSOR_IDS[tensor])
    return g


def smooth_field(w: Workload, tensor: str, seed: int = 0, device="cpu") -> torch.Tensor:
    """[B, H, N, d_h] smooth-field-plus-noise activations in fp32 (before rounding)."""
    T, Hs, Ws = w.grid
    g = _gen(w.cfg_id, tensor, seed, device)
    dev = torch.device(device)
    t, y, x = torch.meshgrid(torch.arange(T, device=dev), torch.arange(Hs, device=dev),
                             torch.arange(Ws, device=dev), indexing="ij")
    u = torch.stack([t.reshape(-1) / T, y.reshape(-1) / Hs, x.reshape(-1) / Ws], dim=1).float()
    out = torch.empty((w.B, w.H, w.N, w.d_h), dtype=torch.float32, device=dev)
    for b in range(w.B):
        for h in range(w.H):
            amp = torch.randn((w.d_h, 4), generator=g, device=dev)
            freq = torch.rand((3, w.d_h * 4), generator=g, device=dev) * 2.0
            phase = torch.rand((w.d_h, 4), generator=g, device=dev) * (2.0 * math.pi)
            arg = (2.0 * math.pi) * (u @ freq)                       # [N, d_h*4]
            arg = arg.view(w.N, w.d_h, 4) + phase
            field = (torch.sin(arg) * amp).sum(dim=2)                # [N, d_h]
            field += torch.randn((w.N, w.d_h), generator=g, device=dev)
            if w.unit_rms:
                field /= field.square().mean().sqrt()
            out[b, h] = field
    return out


def make_inputs(w: Workload, seed: int = 0, device="cpu") -> dict:
    """All inputs of one layer, already rounded to the working dtype (logits stay fp32)."""
    dt = torch_dtype(w.dtype)
    res = {k: smooth_field(w, k, seed, device).to(dt) for k in ("Qn", "Kn", "V")}
    for k in ("Pq", "Pk"):
        g = _gen(w.cfg_id, k, seed, device)
        res[k] = (torch.randn((w.H, w.r, w.d_h), generator=g, device=device)
                  / math.sqrt(w.d_h)).to(dt)
    g = _gen(w.cfg_id, "logits", seed, device)
    res["logits"] = GATE_BIAS + 0.5 * torch.randn((w.B, w.N), generator=g, device=device)
    return res


def to_f64(inputs: dict) -> dict:
    """numpy fp64 copies of the (already rounded) inputs, for the CPU oracle."""
    return {k: v.detach().to("cpu", torch.float64).numpy() for k, v in inputs.items()}
