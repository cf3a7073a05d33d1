"""ctypes binding of librola.so (include/rola.h), with the same entry-point names.

Argument marshalling only: tensors are passed as raw device pointers together with the current HIP
stream, and every step runs in the library's kernels. Importing this module fails loudly when the
library has not been built; there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "librola.so")

ROLA_OK, ROLA_ERR_INVALID_ARGUMENT, ROLA_ERR_UNSUPPORTED, ROLA_ERR_WORKSPACE, ROLA_ERR_HIP = range(5)
DTYPE_F32, DTYPE_BF16 = 0, 1

# Every function include/rola.h declares, with (restype, argtypes).
_p, _i32, _f32, _f64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_double, ctypes.c_size_t


class Problem(ctypes.Structure):
    """rola_problem: [B, H, N, d_h] activations on a T x Hs x Ws grid."""
    _fields_ = [("B", _i32), ("H", _i32), ("N", _i32), ("d_h", _i32),
                ("T", _i32), ("Hs", _i32), ("Ws", _i32), ("dtype", _i32)]


_PP = ctypes.POINTER(Problem)
SIGNATURES = {
    "rola_num_blocks": (_i32, [_i32, _i32]),
    "rola_keep_blocks": (_i32, [_i32, _f64]),
    "rola_select_workspace_bytes": (_sz, [_PP, _i32]),
    "rola_summary_workspace_bytes": (_sz, [_PP, _i32]),
    "rola_status_string": (ctypes.c_char_p, [_i32]),
    "rola_last_error": (ctypes.c_char_p, []),
    "rola_rope_tables": (_i32, [_PP, _i32, _i32, _i32, _f64, _i32, _i32, _i32, _p, _p, _p]),
    "rola_rope_apply": (_i32, [_PP, _p, _p, _p, _i32, _p, _p]),
    "rola_rope_backward_accumulate": (_i32, [_PP, _p, _p, _p, _i32, _i32, _p, _p]),
    "rola_block_select": (_i32, [_PP, _p, _p, _i32, _f64, _p, _p, _sz, _p]),
    "rola_rope_pool": (_i32, [_PP, _p, _p, _p, _i32, _i32, _p, _p, _p, _p]),
    "rola_select_pooled_workspace_bytes": (_sz, [_PP, _i32]),
    "rola_block_select_pooled": (_i32, [_PP, _p, _p, _i32, _f64, _p, _p, _sz, _p]),
    "rola_sparse_workspace_bytes": (_sz, [_PP, _i32, _f64]),
    "rola_sparse_attn": (_i32, [_PP, _p, _p, _p, _i32, _f64, _p, _f32, _p, _p, _sz, _p]),
    "rola_dense_attn": (_i32, [_PP, _p, _p, _p, _i32, _f32, _p, _p]),
    "rola_lowrank_summary": (_i32, [_PP, _p, _p, _p, _i32, _p, _p, _i32, _p, _p, _p, _sz, _p]),
    "rola_lowrank_readout": (_i32, [_PP, _p, _p, _i32, _p, _p, _i32, _p, _f32, _p, _p]),
    "rola_combine": (_i32, [_PP, _p, _p, _p, _f32, _p, _p]),
    "rola_lowrank_readout_combine": (_i32, [_PP, _p, _p, _i32, _p, _p, _i32, _p, _f32, _p, _p, _f32,
                                            _p, _p]),
    "rola_lowrank_summary_ex": (_i32, [_PP, _p, _p, _p, _i32, _p, _p, _i32, _i32, _i32, _p, _p, _p,
                                       _sz, _p]),
    "rola_lowrank_readout_ex": (_i32, [_PP, _p, _p, _i32, _p, _p, _i32, _i32, _i32, _p, _f32, _p,
                                       _p]),
    "rola_lowrank_readout_combine_ex": (_i32, [_PP, _p, _p, _i32, _p, _p, _i32, _i32, _i32, _p, _f32,
                                               _p, _p, _f32, _p, _p]),
    "rola_lowrank_features": (_i32, [_PP, _p, _p, _i32, _p, _p, _i32, _i32, _i32, _p, _p]),
    "rola_gate_logits": (_i32, [_PP, _p, _i32, _p, _f32, _p, _p]),
    "rola_sparse_combine_workspace_bytes": (_sz, [_PP, _i32, _f64, _i32]),
    "rola_sparse_attn_lse": (_i32, [_PP, _p, _p, _p, _i32, _f64, _p, _f32, _p, _p, _p, _sz, _p]),
    "rola_lowrank_backward_workspace_bytes": (_sz, [_PP, _i32]),
    "rola_lowrank_backward": (_i32, [_PP, _p, _p, _p, _p, _p, _i32, _p, _p, _i32, _p, _p, _p, _f32,
                                     _f32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _sz, _p]),
    "rola_gate_backward_workspace_bytes": (_sz, [_PP, _i32]),
    "rola_gate_logits_backward": (_i32, [_PP, _p, _i32, _p, _p, _p, _p, _p, _p, _sz, _p]),
    "rola_sparse_backward_workspace_bytes": (_sz, [_PP, _i32, _f64]),
    "rola_sparse_attn_backward": (_i32, [_PP, _p, _p, _p, _i32, _f64, _p, _f32, _p, _p, _p, _p, _p,
                                         _p, _p, _sz, _p]),
    "rola_sparse_attn_combine": (_i32, [_PP, _p, _p, _p, _i32, _f64, _p, _f32, _p, _p, _i32, _p, _p,
                                        _i32, _p, _f32, _p, _f32, _p, _p, _p, _sz, _p]),
    "rola_sparse_plan": (_i32, [_PP, _i32, _f64, _p, _i32, _p, _sz, _p]),
    "rola_sparse_attn_combine_noalloc": (_i32, [_PP, _p, _p, _p, _i32, _f64, _p, _f32, _p, _p, _i32,
                                                _p, _p, _i32, _p, _f32, _p, _f32, _p, _p, _p]),
    "rola_sparse_attn_combine_planned": (_i32, [_PP, _p, _p, _p, _i32, _f64, _p, _f32, _p, _p, _i32,
                                                _p, _p, _i32, _p, _f32, _p, _f32, _p, _p, _p, _sz, _p]),
}

# Feature map and rotation order of the low-rank branch (rola_phi, rola_rope_order).
PHI = {"silu": 0, "identity": 1, "tanh": 2, "relu": 3, "gelu": 4}
ROPE_ORDER = {"outside": 0, "inside": 1, "none": 2}


def _code(table, v):
    return table[v] if isinstance(v, str) else int(v)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it first (python -m paper_2609_06712_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


LIB = _load()


class RolaError(RuntimeError):
    def __init__(self, status: int, fn: str):
        self.status = status
        msg = LIB.rola_last_error().decode()
        super().__init__(f"{fn}: {LIB.rola_status_string(status).decode()}: {msg}")


def _check(status: int, fn: str):
    if status != ROLA_OK:
        raise RolaError(status, fn)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def problem(B, H, N, d_h, grid, dtype) -> Problem:
    T, Hs, Ws = grid
    code = {"f32": DTYPE_F32, "bf16": DTYPE_BF16, torch.float32: DTYPE_F32,
            torch.bfloat16: DTYPE_BF16}[dtype]
    return Problem(B, H, N, d_h, T, Hs, Ws, code)


def problem_of(x: torch.Tensor, grid) -> Problem:
    """Problem descriptor of a [B, H, N, d_h] activation tensor."""
    B, H, N, d = x.shape
    return problem(B, H, N, d, grid, x.dtype)


# ---- argument checks ------------------------------------------------------------------------------
# Every tensor is checked before the ctypes call: first the element type and shape of every
# argument, then the memory layout (contiguous, or a unit inner stride for the rotary tables) and
# the device of every argument. A list or table of the wrong type or size would make the kernels
# read past a buffer, so nothing reaches the library unchecked.

_ACT_DTYPES = (torch.bfloat16, torch.float32)


class _Args:
    """Collects the tensors of one call: shapes and types are checked as they are added, the
    layout and device of all of them by done()."""

    def __init__(self):
        self.placed = []

    def tensor(self, x, name, shape, dtype, inner_only=False):
        if not isinstance(x, torch.Tensor):
            raise ValueError(f"{name} must be a tensor")
        if x.dtype != dtype:
            raise ValueError(f"{name} must be {dtype}, got {x.dtype}")
        if tuple(x.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(x.shape)}")
        self.placed.append((x, name, inner_only))
        return x

    def act(self, x, name, like=None):
        """A [B, H, N, d_h] activation (bf16 or fp32), of the same shape and type as `like`."""
        if like is not None:
            return self.tensor(x, name, like.shape, like.dtype)
        if not isinstance(x, torch.Tensor):
            raise ValueError(f"{name} must be a tensor")
        if x.dtype not in _ACT_DTYPES:
            raise ValueError(f"{name} must be bfloat16 or float32, got {x.dtype}")
        if x.dim() != 4:
            raise ValueError(f"{name} must be a [B, H, N, d_h] tensor, got shape {tuple(x.shape)}")
        self.placed.append((x, name, False))
        return x

    def proj(self, P, name, like, r):
        B, H, N, d = like.shape
        return self.tensor(P, name, (H, r, d), like.dtype)

    def tables(self, cos, sin, like, need):
        """Rotary tables fp32 [N, ld] sharing one row stride ld (returned) with >= need columns."""
        N = like.shape[2]
        for t, name in ((cos, "cos"), (sin, "sin")):
            if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or t.dim() != 2:
                raise ValueError(f"{name} must be a float32 [N, ld] table")
            if t.shape[0] != N or t.shape[1] < need:
                raise ValueError(f"{name} must have {N} rows and >= {need} columns, got "
                                 f"{tuple(t.shape)}")
            self.placed.append((t, name, True))
        if cos.stride(0) != sin.stride(0) or cos.stride(0) < need:
            raise ValueError("cos and sin must share one row stride of at least the columns used")
        return cos.stride(0)

    def blk_idx(self, idx, like, block, sparsity):
        B, H, N, _ = like.shape
        nb = num_blocks(N, block)
        keep = keep_blocks(nb, sparsity)
        if nb < 1 or keep < 1:
            raise ValueError(f"invalid block {block} or sparsity {sparsity}")
        return self.tensor(idx, "blk_idx", (B, H, nb, keep), torch.int32)

    def logits(self, lg, like):
        B, H, N, _ = like.shape
        return self.tensor(lg, "logits", (B, N), torch.float32)

    def context(self, C, like, r):
        B, H, N, d = like.shape
        return self.tensor(C, "C", (B, H, r, d), torch.float32)

    def workspace(self, ws):
        if ws is None:
            return None
        if not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8 or ws.dim() != 1:
            raise ValueError("ws must be a 1-D uint8 tensor")
        self.placed.append((ws, "ws", False))
        return ws

    def done(self):
        device = None
        for x, name, inner_only in self.placed:
            if inner_only:
                if x.stride(-1) != 1:
                    raise ValueError(f"{name} must have a unit inner stride")
            elif not x.is_contiguous():
                raise ValueError(f"{name} must be contiguous")
            if not x.is_cuda:
                raise ValueError(f"{name} must be a device tensor")
            if device is None:
                device = x.device
            elif x.device != device:
                raise ValueError(f"{name} is on {x.device}, the other arguments on {device}")


# ---- host helpers ---------------------------------------------------------------------------------

def num_blocks(N: int, block: int) -> int:
    return LIB.rola_num_blocks(N, block)


def keep_blocks(n_blocks: int, sparsity: float) -> int:
    return LIB.rola_keep_blocks(n_blocks, sparsity)


def select_workspace_bytes(prob: Problem, block: int) -> int:
    return LIB.rola_select_workspace_bytes(ctypes.byref(prob), block)


def sparse_workspace_bytes(prob: Problem, block: int, sparsity: float) -> int:
    return LIB.rola_sparse_workspace_bytes(ctypes.byref(prob), block, sparsity)


def summary_workspace_bytes(prob: Problem, r: int) -> int:
    return LIB.rola_summary_workspace_bytes(ctypes.byref(prob), r)


# ---- entry points (same names as the C ABI) -------------------------------------------------------

def rola_rope_tables(prob: Problem, split, base=10000.0, offset=(0, 0, 0), stream=None, device="cuda"):
    half = prob.d_h // 2
    cos = torch.empty((prob.N, half), dtype=torch.float32, device=device)
    sin = torch.empty_like(cos)
    _check(LIB.rola_rope_tables(ctypes.byref(prob), split[0], split[1], split[2], base, offset[0],
                                offset[1], offset[2], _ptr(cos), _ptr(sin), _stream(stream)),
           "rola_rope_tables")
    return cos, sin


def rola_rope_apply(X, cos, sin, grid, out=None, stream=None):
    a = _Args()
    a.act(X, "X")
    ld = a.tables(cos, sin, X, X.shape[3] // 2)
    out = torch.empty_like(X) if out is None else a.act(out, "out", X)
    a.done()
    prob = problem_of(X, grid)
    _check(LIB.rola_rope_apply(ctypes.byref(prob), _ptr(X), _ptr(cos), _ptr(sin), ld, _ptr(out),
                               _stream(stream)), "rola_rope_apply")
    return out


def rola_rope_backward_accumulate(dY, cos, sin, grid, dX, rotate=True, stream=None):
    """dX += R(p)^T dY (rotate) or dX += dY, fp32 [B, H, N, d_h], in place; returns dX."""
    a = _Args()
    a.act(dY, "dY")
    if dY.dtype != torch.float32:
        raise ValueError("dY must be float32")
    a.act(dX, "dX", dY)
    ld = a.tables(cos, sin, dY, dY.shape[3] // 2)
    a.done()
    prob = problem_of(dY, grid)
    _check(LIB.rola_rope_backward_accumulate(ctypes.byref(prob), _ptr(dY), _ptr(cos), _ptr(sin), ld,
                                             1 if rotate else 0, _ptr(dX), _stream(stream)),
           "rola_rope_backward_accumulate")
    return dX


def rola_block_select(Qr, Kr, grid, block, sparsity, out=None, ws=None, stream=None):
    a = _Args()
    a.act(Qr, "Qr")
    a.act(Kr, "Kr", Qr)
    prob = problem_of(Qr, grid)
    nb = num_blocks(prob.N, block)
    keep = keep_blocks(nb, sparsity)
    if out is None:
        out = torch.empty((prob.B, prob.H, nb, keep), dtype=torch.int32, device=Qr.device)
    a.blk_idx(out, Qr, block, sparsity)
    need = select_workspace_bytes(prob, block)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=Qr.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_block_select(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), block, sparsity, _ptr(out),
                                 _ptr(ws), ws.numel(), _stream(stream)), "rola_block_select")
    return out


def rola_rope_pool(X, cos, sin, grid, block, want_xr=True, xr=None, xbar=None, xnorm=None,
                   stream=None):
    """(R(X) or None, block means of R(X) fp32 [B, H, n_blocks, d_h]) in one pass. With cos and sin
    None, X is already rotated and only the means are computed. xnorm (optional, fp32
    [B, H, n_blocks]) receives each block's largest row norm."""
    a = _Args()
    a.act(X, "X")
    if cos is None and sin is None:
        ld, want_xr = 0, False
        if xr is not None:
            raise ValueError("xr needs the rotary tables")
    else:
        ld = a.tables(cos, sin, X, X.shape[3] // 2)
    B, H, N, d = X.shape
    if want_xr and xr is None:
        xr = torch.empty_like(X)
    if xr is not None:
        a.act(xr, "xr", X)
    shape = (B, H, num_blocks(N, block), d)
    if xbar is None:
        xbar = torch.empty(shape, dtype=torch.float32, device=X.device)
    a.tensor(xbar, "xbar", shape, torch.float32)
    if xnorm is not None:
        a.tensor(xnorm, "xnorm", shape[:3], torch.float32)
    a.done()
    prob = problem_of(X, grid)
    _check(LIB.rola_rope_pool(ctypes.byref(prob), _ptr(X), _ptr(cos), _ptr(sin), ld, block, _ptr(xr),
                              _ptr(xbar), _ptr(xnorm), _stream(stream)), "rola_rope_pool")
    return xr, xbar


def rola_block_select_pooled(Qbar, Kbar, like, grid, block, sparsity, out=None, ws=None,
                             stream=None):
    """Block lists from the means of rola_rope_pool; `like`: an activation of the layer (shape)."""
    a = _Args()
    a.act(like, "like")
    B, H, N, d = like.shape
    shape = (B, H, num_blocks(N, block), d)
    a.tensor(Qbar, "Qbar", shape, torch.float32)
    a.tensor(Kbar, "Kbar", shape, torch.float32)
    prob = problem_of(like, grid)
    if out is None:
        out = torch.empty((B, H, shape[2], keep_blocks(shape[2], sparsity)), dtype=torch.int32,
                          device=like.device)
    a.blk_idx(out, like, block, sparsity)
    need = LIB.rola_select_pooled_workspace_bytes(ctypes.byref(prob), block)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=like.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_block_select_pooled(ctypes.byref(prob), _ptr(Qbar), _ptr(Kbar), block, sparsity,
                                        _ptr(out), _ptr(ws), ws.numel(), _stream(stream)),
           "rola_block_select_pooled")
    return out


def rola_sparse_attn(Qr, Kr, V, grid, block, sparsity, blk_idx, scale=None, out=None, ws=None,
                     stream=None, share=True):
    """share=False passes no workspace: each workgroup then serves one query block."""
    a = _Args()
    a.act(Qr, "Qr")
    a.act(Kr, "Kr", Qr)
    a.act(V, "V", Qr)
    a.blk_idx(blk_idx, Qr, block, sparsity)
    prob = problem_of(Qr, grid)
    scale = prob.d_h ** -0.5 if scale is None else scale
    out = torch.empty_like(Qr) if out is None else a.act(out, "out", Qr)
    if ws is None and share:
        need = sparse_workspace_bytes(prob, block, sparsity)
        ws = torch.empty(need, dtype=torch.uint8, device=Qr.device) if need else None
    a.workspace(ws)
    a.done()
    _check(LIB.rola_sparse_attn(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), _ptr(V), block, sparsity,
                                _ptr(blk_idx), scale, _ptr(out), _ptr(ws) if ws is not None else None,
                                ws.numel() if ws is not None else 0, _stream(stream)),
           "rola_sparse_attn")
    return out


def rola_dense_attn(Qr, Kr, V, grid, block=64, scale=None, out=None, stream=None):
    a = _Args()
    a.act(Qr, "Qr")
    a.act(Kr, "Kr", Qr)
    a.act(V, "V", Qr)
    prob = problem_of(Qr, grid)
    scale = prob.d_h ** -0.5 if scale is None else scale
    out = torch.empty_like(Qr) if out is None else a.act(out, "out", Qr)
    a.done()
    _check(LIB.rola_dense_attn(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), _ptr(V), block, scale,
                               _ptr(out), _stream(stream)), "rola_dense_attn")
    return out


def _summary_args(a, Kn, V, Pk, r, cos, sin, C, z, want_z):
    a.act(Kn, "Kn")
    a.act(V, "V", Kn)
    a.proj(Pk, "Pk", Kn, r)
    ld = a.tables(cos, sin, Kn, r // 2)
    B, H, N, d = Kn.shape
    if C is None:
        C = torch.empty((B, H, r, d), dtype=torch.float32, device=Kn.device)
    a.context(C, Kn, r)
    if z is None and want_z:
        z = torch.empty((B, H, r), dtype=torch.float32, device=Kn.device)
    if z is not None:
        a.tensor(z, "z", (B, H, r), torch.float32)
    return ld, C, z


def rola_lowrank_summary(Kn, V, Pk, r, cos, sin, grid, C=None, z=None, ws=None, stream=None,
                         want_z=True):
    a = _Args()
    ld, C, z = _summary_args(a, Kn, V, Pk, r, cos, sin, C, z, want_z)
    prob = problem_of(Kn, grid)
    need = summary_workspace_bytes(prob, r)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=Kn.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_lowrank_summary(ctypes.byref(prob), _ptr(Kn), _ptr(V), _ptr(Pk), r, _ptr(cos),
                                    _ptr(sin), ld, _ptr(C), _ptr(z), _ptr(ws), ws.numel(),
                                    _stream(stream)), "rola_lowrank_summary")
    return C, z


def _readout_args(a, Qn, Pq, r, cos, sin, C):
    a.act(Qn, "Qn")
    a.proj(Pq, "Pq", Qn, r)
    a.context(C, Qn, r)
    return a.tables(cos, sin, Qn, r // 2)


def rola_lowrank_readout(Qn, Pq, r, cos, sin, C, grid, eps_lr=1e-6, out=None, stream=None):
    a = _Args()
    ld = _readout_args(a, Qn, Pq, r, cos, sin, C)
    out = torch.empty_like(Qn) if out is None else a.act(out, "out", Qn)
    a.done()
    prob = problem_of(Qn, grid)
    _check(LIB.rola_lowrank_readout(ctypes.byref(prob), _ptr(Qn), _ptr(Pq), r, _ptr(cos), _ptr(sin),
                                    ld, _ptr(C), eps_lr, _ptr(out), _stream(stream)),
           "rola_lowrank_readout")
    return out


def rola_combine(Os, Olr, logits, grid, eps=1e-6, out=None, stream=None):
    a = _Args()
    a.act(Os, "Os")
    a.act(Olr, "Olr", Os)
    a.logits(logits, Os)
    out = torch.empty_like(Os) if out is None else a.act(out, "out", Os)
    a.done()
    prob = problem_of(Os, grid)
    _check(LIB.rola_combine(ctypes.byref(prob), _ptr(Os), _ptr(Olr), _ptr(logits), eps, _ptr(out),
                            _stream(stream)), "rola_combine")
    return out


def rola_lowrank_readout_combine(Qn, Pq, r, cos, sin, C, Os, logits, grid, eps_lr=1e-6, eps=1e-6,
                                 out=None, stream=None):
    a = _Args()
    ld = _readout_args(a, Qn, Pq, r, cos, sin, C)
    a.act(Os, "Os", Qn)
    a.logits(logits, Qn)
    out = torch.empty_like(Os) if out is None else a.act(out, "out", Qn)
    a.done()
    prob = problem_of(Qn, grid)
    _check(LIB.rola_lowrank_readout_combine(ctypes.byref(prob), _ptr(Qn), _ptr(Pq), r, _ptr(cos),
                                            _ptr(sin), ld, _ptr(C), eps_lr, _ptr(Os),
                                            _ptr(logits), eps, _ptr(out), _stream(stream)),
           "rola_lowrank_readout_combine")
    return out


def rola_lowrank_summary_ex(Kn, V, Pk, r, cos, sin, grid, phi="silu", rope_order="outside", C=None,
                            z=None, ws=None, stream=None, want_z=True):
    a = _Args()
    ld, C, z = _summary_args(a, Kn, V, Pk, r, cos, sin, C, z, want_z)
    prob = problem_of(Kn, grid)
    need = summary_workspace_bytes(prob, r)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=Kn.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_lowrank_summary_ex(ctypes.byref(prob), _ptr(Kn), _ptr(V), _ptr(Pk), r, _ptr(cos),
                                       _ptr(sin), ld, _code(PHI, phi),
                                       _code(ROPE_ORDER, rope_order), _ptr(C), _ptr(z), _ptr(ws),
                                       ws.numel(), _stream(stream)), "rola_lowrank_summary_ex")
    return C, z


def rola_lowrank_readout_ex(Qn, Pq, r, cos, sin, C, grid, phi="silu", rope_order="outside",
                            eps_lr=1e-6, out=None, stream=None):
    a = _Args()
    ld = _readout_args(a, Qn, Pq, r, cos, sin, C)
    out = torch.empty_like(Qn) if out is None else a.act(out, "out", Qn)
    a.done()
    prob = problem_of(Qn, grid)
    _check(LIB.rola_lowrank_readout_ex(ctypes.byref(prob), _ptr(Qn), _ptr(Pq), r, _ptr(cos),
                                       _ptr(sin), ld, _code(PHI, phi),
                                       _code(ROPE_ORDER, rope_order), _ptr(C), eps_lr, _ptr(out),
                                       _stream(stream)), "rola_lowrank_readout_ex")
    return out


def rola_lowrank_readout_combine_ex(Qn, Pq, r, cos, sin, C, Os, logits, grid, phi="silu",
                                    rope_order="outside", eps_lr=1e-6, eps=1e-6, out=None,
                                    stream=None):
    a = _Args()
    ld = _readout_args(a, Qn, Pq, r, cos, sin, C)
    a.act(Os, "Os", Qn)
    a.logits(logits, Qn)
    out = torch.empty_like(Os) if out is None else a.act(out, "out", Qn)
    a.done()
    prob = problem_of(Qn, grid)
    _check(LIB.rola_lowrank_readout_combine_ex(ctypes.byref(prob), _ptr(Qn), _ptr(Pq), r, _ptr(cos),
                                               _ptr(sin), ld, _code(PHI, phi),
                                               _code(ROPE_ORDER, rope_order), _ptr(C), eps_lr,
                                               _ptr(Os), _ptr(logits), eps, _ptr(out),
                                               _stream(stream)), "rola_lowrank_readout_combine_ex")
    return out


def rola_lowrank_features(X, P, r, cos, sin, grid, phi="silu", rope_order="outside", out=None,
                          stream=None):
    """q~ (X = Q^n, P = P_q) or k~ (X = K^n, P = P_k) of every token: fp32 [B, H, N, r]."""
    a = _Args()
    a.act(X, "X")
    a.proj(P, "P", X, r)
    ld = a.tables(cos, sin, X, r // 2)
    prob = problem_of(X, grid)
    shape = (prob.B, prob.H, prob.N, r)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=X.device)
    a.tensor(out, "out", shape, torch.float32)
    a.done()
    _check(LIB.rola_lowrank_features(ctypes.byref(prob), _ptr(X), _ptr(P), r, _ptr(cos), _ptr(sin),
                                     ld, _code(PHI, phi), _code(ROPE_ORDER, rope_order),
                                     _ptr(out), _stream(stream)), "rola_lowrank_features")
    return out


def _hidden(a, X, Wg):
    if not isinstance(X, torch.Tensor) or X.dtype not in _ACT_DTYPES or X.dim() != 3:
        raise ValueError("X must be a [B, N, d_model] bfloat16 or float32 tensor")
    a.tensor(X, "X", X.shape, X.dtype)
    a.tensor(Wg, "Wg", (X.shape[2],), X.dtype)
    return X.shape


def rola_gate_logits(X, Wg, bg, grid, H=1, d_h=128, out=None, stream=None):
    """Gate logits X W_g + b_g of every token: X [B, N, d_model], W_g [d_model] -> fp32 [B, N]."""
    a = _Args()
    B, N, dm = _hidden(a, X, Wg)
    prob = problem(B, H, N, d_h, grid, X.dtype)
    if out is None:
        out = torch.empty((B, N), dtype=torch.float32, device=X.device)
    a.tensor(out, "out", (B, N), torch.float32)
    a.done()
    _check(LIB.rola_gate_logits(ctypes.byref(prob), _ptr(X), dm, _ptr(Wg), bg, _ptr(out),
                                _stream(stream)), "rola_gate_logits")
    return out


def sparse_combine_workspace_bytes(prob: Problem, block: int, sparsity: float, r: int) -> int:
    return LIB.rola_sparse_combine_workspace_bytes(ctypes.byref(prob), block, sparsity, r)


def _combine_args(a, Qr, Kr, V, block, sparsity, blk_idx, Qn, Pq, r, cos, sin, C, logits,
                  key_norm=None):
    """Qr may be None: the queries are then rotated from Qn in the attention's prologue. key_norm
    (optional): fp32 [B, H, n_blocks], per key block a bound on its keys' norms (rola_rope_pool's
    xnorm of K), which lets the attention use a fixed softmax reference."""
    a.act(Qn, "Qn")
    if key_norm is not None:
        B, H, N, _ = Qn.shape
        a.tensor(key_norm, "key_norm", (B, H, num_blocks(N, block)), torch.float32)
    for t, name in ((Qr, "Qr"), (Kr, "Kr"), (V, "V")):
        if t is not None or name != "Qr":
            a.act(t, name, Qn)
    a.blk_idx(blk_idx, Qn, block, sparsity)
    ld = _readout_args(a, Qn, Pq, r, cos, sin, C)
    a.logits(logits, Qn)
    if Qr is None and cos.shape[1] < Qn.shape[3] // 2:
        raise ValueError("Qr = None needs tables with d_h/2 columns")
    return ld


def rola_sparse_attn_combine(Qr, Kr, V, grid, block, sparsity, blk_idx, Qn, Pq, r, cos, sin, C,
                             logits, scale=None, eps_lr=1e-6, eps=1e-6, out=None, ws=None,
                             stream=None, key_norm=None):
    """O = combine(sparse attention, low-rank readout of C) in one call (fused epilogue)."""
    a = _Args()
    ld = _combine_args(a, Qr, Kr, V, block, sparsity, blk_idx, Qn, Pq, r, cos, sin, C, logits,
                       key_norm)
    prob = problem_of(Qn, grid)
    scale = prob.d_h ** -0.5 if scale is None else scale
    out = torch.empty_like(Qn) if out is None else a.act(out, "out", Qn)
    if ws is None:
        need = sparse_combine_workspace_bytes(prob, block, sparsity, r)
        ws = torch.empty(need, dtype=torch.uint8, device=Qn.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_sparse_attn_combine(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), _ptr(V), block,
                                        sparsity, _ptr(blk_idx), scale, _ptr(Qn), _ptr(Pq), r,
                                        _ptr(cos), _ptr(sin), ld, _ptr(C), eps_lr,
                                        _ptr(logits), eps, _ptr(key_norm), _ptr(out), _ptr(ws),
                                        ws.numel(), _stream(stream)), "rola_sparse_attn_combine")
    return out


def rola_sparse_plan(blk_idx, like, grid, block, sparsity, r, ws, stream=None):
    """Pairs and merged lists of rola_sparse_attn_combine_planned into ws (its workspace); `like` is
    any of the call's activations (for the shape)."""
    a = _Args()
    a.act(like, "like")
    a.blk_idx(blk_idx, like, block, sparsity)
    a.workspace(ws)
    a.done()
    prob = problem_of(like, grid)
    _check(LIB.rola_sparse_plan(ctypes.byref(prob), block, sparsity, _ptr(blk_idx), r, _ptr(ws),
                                ws.numel(), _stream(stream)), "rola_sparse_plan")
    return ws


def rola_sparse_attn_combine_planned(Qr, Kr, V, grid, block, sparsity, blk_idx, Qn, Pq, r, cos, sin,
                                     C, logits, ws, scale=None, eps_lr=1e-6, eps=1e-6, out=None,
                                     stream=None, key_norm=None):
    """rola_sparse_attn_combine on the plan rola_sparse_plan left in ws."""
    a = _Args()
    ld = _combine_args(a, Qr, Kr, V, block, sparsity, blk_idx, Qn, Pq, r, cos, sin, C, logits,
                       key_norm)
    prob = problem_of(Qn, grid)
    scale = prob.d_h ** -0.5 if scale is None else scale
    out = torch.empty_like(Qn) if out is None else a.act(out, "out", Qn)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_sparse_attn_combine_planned(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), _ptr(V),
                                                block, sparsity, _ptr(blk_idx), scale, _ptr(Qn),
                                                _ptr(Pq), r, _ptr(cos), _ptr(sin), ld, _ptr(C), eps_lr,
                                                _ptr(logits), eps, _ptr(key_norm), _ptr(out), _ptr(ws),
                                                ws.numel(), _stream(stream)),
           "rola_sparse_attn_combine_planned")
    return out


def rola_sparse_attn_combine_noalloc(Qr, Kr, V, grid, block, sparsity, blk_idx, Qn, Pq, r, cos, sin,
                                     C, logits, out, scale=None, eps_lr=1e-6, eps=1e-6,
                                     stream=None, key_norm=None):
    """rola_sparse_attn_combine with the library's static device scratch instead of a workspace:
    nothing is allocated (the output `out` is the caller's)."""
    a = _Args()
    ld = _combine_args(a, Qr, Kr, V, block, sparsity, blk_idx, Qn, Pq, r, cos, sin, C, logits,
                       key_norm)
    a.act(out, "out", Qn)
    a.done()
    prob = problem_of(Qn, grid)
    scale = prob.d_h ** -0.5 if scale is None else scale
    _check(LIB.rola_sparse_attn_combine_noalloc(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), _ptr(V),
                                                block, sparsity, _ptr(blk_idx), scale, _ptr(Qn),
                                                _ptr(Pq), r, _ptr(cos), _ptr(sin), ld, _ptr(C), eps_lr,
                                                _ptr(logits), eps, _ptr(key_norm), _ptr(out),
                                                _stream(stream)),
           "rola_sparse_attn_combine_noalloc")
    return out


def rola_sparse_attn_lse(Qr, Kr, V, grid, block, sparsity, blk_idx, scale=None, out=None, lse=None,
                         ws=None, stream=None, share=True):
    """Sparse attention that also returns the per-query log2-sum-exp2 (fp32 [B, H, N]); share=False
    passes no workspace (one query block per workgroup)."""
    a = _Args()
    a.act(Qr, "Qr")
    a.act(Kr, "Kr", Qr)
    a.act(V, "V", Qr)
    a.blk_idx(blk_idx, Qr, block, sparsity)
    prob = problem_of(Qr, grid)
    scale = prob.d_h ** -0.5 if scale is None else scale
    out = torch.empty_like(Qr) if out is None else a.act(out, "out", Qr)
    if lse is None:
        lse = torch.empty(Qr.shape[:3], dtype=torch.float32, device=Qr.device)
    a.tensor(lse, "lse", Qr.shape[:3], torch.float32)
    if ws is None and share:
        need = sparse_workspace_bytes(prob, block, sparsity)
        ws = torch.empty(need, dtype=torch.uint8, device=Qr.device) if need else None
    a.workspace(ws)
    a.done()
    _check(LIB.rola_sparse_attn_lse(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), _ptr(V), block, sparsity,
                                    _ptr(blk_idx), scale, _ptr(out), _ptr(lse),
                                    _ptr(ws) if ws is not None else None,
                                    ws.numel() if ws is not None else 0, _stream(stream)),
           "rola_sparse_attn_lse")
    return out, lse


def rola_sparse_attn_backward(Qr, Kr, V, grid, block, sparsity, blk_idx, Os, lse, dOs, scale=None,
                              ws=None, stream=None):
    """Gradients (dQ^r, dK^r, dV), fp32, of <dOs, O^s> for fixed block lists."""
    a = _Args()
    a.act(Qr, "Qr")
    for t, name in ((Kr, "Kr"), (V, "V"), (Os, "Os"), (dOs, "dOs")):
        a.act(t, name, Qr)
    a.blk_idx(blk_idx, Qr, block, sparsity)
    a.tensor(lse, "lse", Qr.shape[:3], torch.float32)
    prob = problem_of(Qr, grid)
    scale = prob.d_h ** -0.5 if scale is None else scale
    dQ = torch.empty(Qr.shape, dtype=torch.float32, device=Qr.device)
    dK, dV = torch.empty_like(dQ), torch.empty_like(dQ)
    if ws is None:
        need = LIB.rola_sparse_backward_workspace_bytes(ctypes.byref(prob), block, sparsity)
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=Qr.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_sparse_attn_backward(ctypes.byref(prob), _ptr(Qr), _ptr(Kr), _ptr(V), block,
                                         sparsity, _ptr(blk_idx), scale, _ptr(Os), _ptr(lse),
                                         _ptr(dOs), _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(ws),
                                         ws.numel(), _stream(stream)), "rola_sparse_attn_backward")
    return dQ, dK, dV


def rola_lowrank_backward(Qn, Kn, V, Pq, Pk, r, cos, sin, C, Os, logits, dO, grid, eps_lr=1e-6,
                          eps=1e-6, ws=None, stream=None):
    """(dOs bf16, dQn, dKn, dV fp32 [B, H, N, d], dPq, dPk fp32 [H, r, d], dlogits fp32 [B, N])."""
    a = _Args()
    ld = _readout_args(a, Qn, Pq, r, cos, sin, C)
    for t, name in ((Kn, "Kn"), (V, "V"), (Os, "Os"), (dO, "dO")):
        a.act(t, name, Qn)
    a.proj(Pk, "Pk", Qn, r)
    a.logits(logits, Qn)
    prob = problem_of(Qn, grid)
    dOs = torch.empty_like(Qn)
    f32 = dict(dtype=torch.float32, device=Qn.device)
    dQn, dKn, dV = (torch.empty(Qn.shape, **f32) for _ in range(3))
    dPq, dPk = torch.empty(Pq.shape, **f32), torch.empty(Pk.shape, **f32)
    dlog = torch.empty(logits.shape, **f32)
    if ws is None:
        need = LIB.rola_lowrank_backward_workspace_bytes(ctypes.byref(prob), r)
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=Qn.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_lowrank_backward(ctypes.byref(prob), _ptr(Qn), _ptr(Kn), _ptr(V), _ptr(Pq),
                                     _ptr(Pk), r, _ptr(cos), _ptr(sin), ld, _ptr(C),
                                     _ptr(Os), _ptr(logits), eps_lr, eps, _ptr(dO), _ptr(dOs),
                                     _ptr(dQn), _ptr(dKn), _ptr(dV), _ptr(dPq), _ptr(dPk),
                                     _ptr(dlog), _ptr(ws), ws.numel(), _stream(stream)),
           "rola_lowrank_backward")
    return dOs, dQn, dKn, dV, dPq, dPk, dlog


def rola_gate_logits_backward(X, Wg, dlogits, grid, H=1, d_h=128, want_dX=True, ws=None,
                              stream=None):
    """(dX fp32 [B, N, d_model] or None, dWg fp32 [d_model], dbg fp32 [1]) of X W_g + b_g."""
    a = _Args()
    B, N, dm = _hidden(a, X, Wg)
    a.tensor(dlogits, "dlogits", (B, N), torch.float32)
    prob = problem(B, H, N, d_h, grid, X.dtype)
    f32 = dict(dtype=torch.float32, device=X.device)
    dX = torch.empty(X.shape, **f32) if want_dX else None
    dWg, dbg = torch.empty(dm, **f32), torch.empty(4, **f32)
    if ws is None:
        need = LIB.rola_gate_backward_workspace_bytes(ctypes.byref(prob), dm)
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=X.device)
    a.workspace(ws)
    a.done()
    _check(LIB.rola_gate_logits_backward(ctypes.byref(prob), _ptr(X), dm, _ptr(Wg), _ptr(dlogits),
                                         _ptr(dX), _ptr(dWg), _ptr(dbg), _ptr(ws), ws.numel(),
                                         _stream(stream)), "rola_gate_logits_backward")
    return dX, dWg, dbg[:1]
