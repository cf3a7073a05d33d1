"""Host-side checks of the C ABI (no GPU work): every declared symbol is exported and bound, the
host helpers agree with the oracle's definitions, and invalid arguments are rejected before any
launch."""

import ctypes
import os
import re

import pytest
import torch

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rola.h")

R = pytest.importorskip("paper_2609_06712_amd.rola")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rola_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound():
    names = declared_functions()
    assert len(names) >= 15
    lib = ctypes.CDLL(R.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
        assert n in R.SIGNATURES, n
    assert set(R.SIGNATURES) == set(names)


@pytest.mark.parametrize("N,block", [(256, 32), (32760, 64), (75600, 64), (75600, 128), (1, 64),
                                     (8400, 64)])
def test_num_blocks(N, block):
    assert R.num_blocks(N, block) == O.num_blocks(N, block)


def test_keep_blocks_matches_oracle():
    for nb in list(range(1, 70)) + [512, 591, 1182, 4096]:
        for s in [0.0, 0.05, 0.1, 0.25, 0.5, 0.75, 0.8, 0.9, 0.95, 0.99, 0.999]:
            assert R.keep_blocks(nb, s) == O.keep_blocks(nb, s), (nb, s)
    assert R.keep_blocks(10, 1.0) == -1 and R.keep_blocks(0, 0.5) == -1


def test_workspace_helpers():
    p = R.problem(1, 40, 75600, 128, (21, 45, 80), "bf16")
    nb = 1182
    assert R.select_workspace_bytes(p, 64) >= 4 * (2 * 40 * nb * 128 + 40 * nb * nb)
    assert R.summary_workspace_bytes(p, 32) > 0
    assert R.select_workspace_bytes(p, 48) == 0          # unsupported block
    assert R.summary_workspace_bytes(p, 33) == 0         # odd rank
    bad = R.problem(1, 40, 75601, 128, (21, 45, 80), "bf16")
    assert R.select_workspace_bytes(bad, 64) == 0
    # the work-queue counters (8, each in a 256-byte slot), the pair table (one int32 per pair of
    # query blocks, padded to 256 B), then the pair-union lists: per (b, h, pair) a count and at most
    # 2 * keep entries; the region first holds the candidate ranks of every query block (64 bytes
    # each, whole chunks of 64)
    keep = O.keep_blocks(nb, 0.9)
    queue = 8 * 256
    table = -(-4 * 40 * ((nb + 1) // 2) // 256) * 256
    ranks = 40 * -(-nb // 64) * 64 * 64
    lists = max(4 * 40 * ((nb + 1) // 2) * (2 * keep + 1), ranks)
    assert R.sparse_workspace_bytes(p, 64, 0.9) == queue + table + lists
    keep1 = O.keep_blocks(nb, 0.99)  # short lists: the ranks set the size
    assert 4 * 40 * ((nb + 1) // 2) * (2 * keep1 + 1) < ranks
    assert R.sparse_workspace_bytes(p, 64, 0.99) == queue + table + ranks
    # more than 4064 query blocks: adjacent pairs, no table
    long = R.problem(1, 2, 64 * 4100, 128, (41, 80, 80), "bf16")
    assert R.sparse_workspace_bytes(long, 64, 0.9) == queue + 4 * 2 * 2050 * (2 * O.keep_blocks(4100, 0.9) + 1)
    assert R.sparse_workspace_bytes(p, 128, 0.9) == 0    # 128-token blocks share nothing
    assert R.sparse_workspace_bytes(R.problem(1, 2, 256, 64, (1, 16, 16), "f32"), 64, 0.5) == 0
    assert R.sparse_workspace_bytes(bad, 64, 0.9) == 0
    # attention + epilogue: the sparse workspace (rounded to 256 B) plus the C^T fragments,
    # 4 channel tiles x 2 k-steps per 16 rotary pairs x 64 lanes x 32 B per head
    sp = -(-R.sparse_workspace_bytes(p, 64, 0.9) // 256) * 256
    assert R.sparse_combine_workspace_bytes(p, 64, 0.9, 32) == sp + 40 * 4 * 2 * 64 * 32
    assert R.sparse_combine_workspace_bytes(p, 64, 0.9, 64) == sp + 40 * 4 * 4 * 64 * 32
    assert R.sparse_combine_workspace_bytes(p, 64, 0.9, 128) == sp + 16  # standalone readout path
    assert R.sparse_combine_workspace_bytes(p, 64, 0.9, 33) == 0


def test_status_strings():
    assert R.LIB.rola_status_string(0) == b"ROLA_OK"
    assert R.LIB.rola_status_string(3) == b"ROLA_ERR_WORKSPACE"


# Invalid-argument checks pass fake (aligned, never dereferenced) addresses. They are host logic and
# run where no GPU is present, so a validation bug can never turn into a launch on a real device.
no_gpu = pytest.mark.skipif(torch.cuda.device_count() > 0, reason="host-validation test: CPU only")
MIS = ctypes.c_void_p((1 << 20) + 4)
_fake_next = [1]


class _Fake:
    """Each use stands for a distinct aligned address (64 GiB apart), so that no two arguments of a
    case overlap unless a case says so."""

    @property
    def _as_parameter_(self):
        _fake_next[0] += 1
        return ctypes.c_void_p(_fake_next[0] << 36)


FAKE = _Fake()
SAME = ctypes.c_void_p(1 << 44)   # one address passed for two arguments: an overlap


def _call(name, *args):
    return getattr(R.LIB, name)(*args)


@no_gpu
def test_invalid_arguments_are_rejected_before_launch():
    g = (21, 45, 80)
    ok = R.problem(1, 2, 75600, 128, g, "bf16")
    big = R.problem(1, 1, 16385 * 64, 128, (1, 1, 16385 * 64), "bf16")  # 16385 blocks of 64
    P = ctypes.byref
    cases = [
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn", P(ok), None, FAKE, FAKE, 64, 0.9, FAKE, 0.1, FAKE, None, 0, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn", P(ok), MIS, FAKE, FAKE, 64, 0.9, FAKE, 0.1, FAKE, None, 0, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn", P(ok), FAKE, FAKE, FAKE, 64, 1.0, FAKE, 0.1, FAKE, None, 0, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn", P(ok), FAKE, FAKE, FAKE, 64, 0.9, FAKE, -1.0, FAKE, None, 0, None),
        (R.ROLA_ERR_UNSUPPORTED, "rola_sparse_attn", P(ok), FAKE, FAKE, FAKE, 32, 0.9, FAKE, 0.1, FAKE, None, 0, None),
        (R.ROLA_ERR_WORKSPACE, "rola_sparse_attn", P(ok), FAKE, FAKE, FAKE, 64, 0.9, FAKE, 0.1, FAKE, FAKE, 64, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn", P(ok), FAKE, FAKE, FAKE, 64, 0.9, FAKE, 0.1, FAKE, MIS, 1 << 40, None),
        (R.ROLA_ERR_UNSUPPORTED, "rola_dense_attn", P(ok), FAKE, FAKE, FAKE, 96, 0.1, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_block_select", P(R.problem(1, 2, 75601, 128, g, "bf16")),
         FAKE, FAKE, 64, 0.9, FAKE, FAKE, 1 << 40, None),
        (R.ROLA_ERR_WORKSPACE, "rola_block_select", P(ok), FAKE, FAKE, 64, 0.9, FAKE, FAKE, 16, None),
        (R.ROLA_ERR_UNSUPPORTED, "rola_block_select", P(R.problem(1, 2, 75600, 96, g, "f32")),
         FAKE, FAKE, 64, 0.9, FAKE, FAKE, 1 << 40, None),
        (R.ROLA_ERR_UNSUPPORTED, "rola_block_select", P(R.problem(1, 2, 75600, 64, g, "bf16")),
         FAKE, FAKE, 64, 0.9, FAKE, FAKE, 1 << 40, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_summary", P(ok), FAKE, FAKE, FAKE, 31, FAKE, FAKE,
         64, FAKE, None, FAKE, 1 << 40, None),
        (R.ROLA_ERR_UNSUPPORTED, "rola_lowrank_summary", P(ok), FAKE, FAKE, FAKE, 48, FAKE, FAKE,
         64, FAKE, None, FAKE, 1 << 40, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_summary", P(ok), FAKE, FAKE, FAKE, 32, FAKE, FAKE,
         6, FAKE, None, FAKE, 1 << 40, None),
        (R.ROLA_ERR_WORKSPACE, "rola_lowrank_summary", P(ok), FAKE, FAKE, FAKE, 32, FAKE, FAKE,
         64, FAKE, None, FAKE, 64, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_readout", P(ok), FAKE, FAKE, 32, FAKE, FAKE, 64,
         FAKE, -1.0, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_combine", P(ok), FAKE, FAKE, FAKE, -1.0, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_rope_tables", P(ok), 44, 42, 40, 10000.0, 0, 0, 0, FAKE,
         FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_rope_apply", P(ok), FAKE, FAKE, FAKE, 60, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_readout_combine", P(ok), FAKE, FAKE, 32, FAKE, FAKE,
         64, FAKE, 1e-6, None, FAKE, 1e-6, FAKE, None),
        # feature-map variants: unknown phi or rotation order
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_summary_ex", P(ok), FAKE, FAKE, FAKE, 32, FAKE,
         FAKE, 64, 5, 0, FAKE, None, FAKE, 1 << 40, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_summary_ex", P(ok), FAKE, FAKE, FAKE, 32, FAKE,
         FAKE, 64, 0, 3, FAKE, None, FAKE, 1 << 40, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_readout_ex", P(ok), FAKE, FAKE, 32, FAKE, FAKE, 64,
         -1, 0, FAKE, 1e-6, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_readout_combine_ex", P(ok), FAKE, FAKE, 32, FAKE,
         FAKE, 64, 0, 7, FAKE, 1e-6, FAKE, FAKE, 1e-6, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_features", P(ok), FAKE, FAKE, 32, FAKE, FAKE, 64,
         9, 0, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_features", P(ok), FAKE, FAKE, 32, FAKE, FAKE, 64,
         0, 0, None, None),
        (R.ROLA_ERR_UNSUPPORTED, "rola_lowrank_features", P(ok), FAKE, FAKE, 48, FAKE, FAKE, 64, 0, 0,
         FAKE, None),
        # gate logits: d_model not a multiple of 8, too large, non-finite bias, null output
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_gate_logits", P(ok), FAKE, 5124, FAKE, -1.9, FAKE, None),
        (R.ROLA_ERR_UNSUPPORTED, "rola_gate_logits", P(ok), FAKE, 16392, FAKE, -1.9, FAKE, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_gate_logits", P(ok), FAKE, 5120, FAKE, float("inf"), FAKE,
         None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_gate_logits", P(ok), FAKE, 5120, FAKE, -1.9, None, None),
        # attention + readout + combine: no workspace, too small a workspace, odd rank
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn_combine", P(ok), FAKE, FAKE, FAKE, 64, 0.9,
         FAKE, 0.1, FAKE, FAKE, 32, FAKE, FAKE, 64, FAKE, 1e-6, FAKE, 1e-6, None, FAKE, None, 0, None),
        (R.ROLA_ERR_WORKSPACE, "rola_sparse_attn_combine", P(ok), FAKE, FAKE, FAKE, 64, 0.9, FAKE,
         0.1, FAKE, FAKE, 32, FAKE, FAKE, 64, FAKE, 1e-6, FAKE, 1e-6, None, FAKE, FAKE, 64, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn_combine", P(ok), FAKE, FAKE, FAKE, 64, 0.9,
         FAKE, 0.1, FAKE, FAKE, 31, FAKE, FAKE, 64, FAKE, 1e-6, FAKE, 1e-6, None, FAKE, FAKE, 1 << 40,
         None),
        # sparse backward: more blocks per head than the transposed lists are built for
        (R.ROLA_ERR_UNSUPPORTED, "rola_sparse_attn_backward", P(big), FAKE, FAKE, FAKE, 64, 0.9, FAKE,
         0.1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40, None),
    ]
    assert R.LIB.rola_sparse_backward_workspace_bytes(P(big), 64, 0.9) == 0
    assert R.LIB.rola_sparse_backward_workspace_bytes(P(R.problem(1, 1, 8192 * 64, 128, (1, 1, 8192 * 64), "bf16")), 64, 0.9) > 0
    # outputs that overlap an input
    cases += [
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn", P(ok), FAKE, SAME, FAKE, 64, 0.9, FAKE, 0.1,
         SAME, None, 0, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_dense_attn", P(ok), FAKE, FAKE, SAME, 64, 0.1, SAME, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_sparse_attn_combine", P(ok), FAKE, FAKE, FAKE, 64, 0.9,
         FAKE, 0.1, SAME, FAKE, 32, FAKE, FAKE, 64, FAKE, 1e-6, FAKE, 1e-6, None, SAME, FAKE, 1 << 40,
         None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_combine", P(ok), FAKE, SAME, FAKE, 1e-6, SAME, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_combine", P(ok), SAME, FAKE, FAKE, 1e-6,
         ctypes.c_void_p((1 << 44) + 4096), None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_readout", P(ok), SAME, FAKE, 32, FAKE, FAKE, 64,
         FAKE, 1e-6, SAME, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_lowrank_readout_combine", P(ok), SAME, FAKE, 32, FAKE,
         FAKE, 64, FAKE, 1e-6, FAKE, FAKE, 1e-6, SAME, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_rope_apply", P(ok), SAME, FAKE, FAKE, 64, SAME, None),
        (R.ROLA_ERR_INVALID_ARGUMENT, "rola_rope_backward_accumulate",
         P(R.problem(1, 2, 75600, 128, g, "f32")), SAME, FAKE, FAKE, 64, 1, SAME, None),
    ]
    for want, name, *args in cases:
        got = _call(name, *args)
        assert got == want, (name, got, want, R.LIB.rola_last_error())
        assert R.LIB.rola_last_error()  # a message is always left behind


def _cpu(shape, dtype=torch.bfloat16):
    return torch.zeros(shape, dtype=dtype)


def test_binding_rejects_bad_tensors():
    """The binding checks type and shape of every tensor before anything reaches the library (and
    layout and device after that), so wrong block lists, tables or outputs raise ValueError."""
    g = (2, 4, 16)                                   # N = 128: 2 blocks of 64
    q = _cpu((1, 2, 128, 128))
    idx_ok = torch.zeros((1, 2, 2, 1), dtype=torch.int32)
    cos = torch.zeros((128, 64))
    bad = [
        ("blk_idx int64", lambda: R.rola_sparse_attn(q, q, q, g, 64, 0.5, idx_ok.long())),
        ("blk_idx keep", lambda: R.rola_sparse_attn(q, q, q, g, 64, 0.5,
                                                    torch.zeros((1, 2, 2, 2), dtype=torch.int32))),
        ("blk_idx other sparsity", lambda: R.rola_sparse_attn(q, q, q, g, 64, 0.0, idx_ok)),
        ("blk_idx other block", lambda: R.rola_sparse_attn(q, q, q, g, 128, 0.5, idx_ok)),
        ("V dtype", lambda: R.rola_sparse_attn(q, q, q.float(), g, 64, 0.5, idx_ok)),
        ("Kr shape", lambda: R.rola_sparse_attn(q, q[:, :1], q, g, 64, 0.5, idx_ok)),
        ("3-D activation", lambda: R.rola_dense_attn(q[0], q[0], q[0], g)),
        ("int activation", lambda: R.rola_dense_attn(q.int(), q.int(), q.int(), g)),
        ("table dtype", lambda: R.rola_rope_apply(q, cos.double(), cos.double(), g)),
        ("table rows", lambda: R.rola_rope_apply(q, cos[:100], cos[:100], g)),
        ("table columns", lambda: R.rola_rope_apply(q, cos[:, :32], cos[:, :32], g)),
        ("table strides differ", lambda: R.rola_rope_apply(q, cos, torch.zeros((128, 72))[:, :64], g)),
        ("Pk shape", lambda: R.rola_lowrank_summary(q, q, _cpu((2, 16, 128)), 32, cos, cos, g)),
        ("C dtype", lambda: R.rola_lowrank_readout(q, _cpu((2, 32, 128)), 32, cos, cos,
                                                   _cpu((1, 2, 32, 128)), g)),
        ("logits shape", lambda: R.rola_combine(q, q, torch.zeros((1, 127)), g)),
        ("logits dtype", lambda: R.rola_combine(q, q, torch.zeros((1, 128), dtype=torch.float64), g)),
        ("out shape", lambda: R.rola_combine(q, q, torch.zeros((1, 128)), g, out=q[:, :1])),
        ("ws dtype", lambda: R.rola_block_select(q, q, g, 64, 0.5, ws=torch.zeros(64))),
        ("lse shape", lambda: R.rola_sparse_attn_lse(q, q, q, g, 64, 0.5, idx_ok,
                                                     lse=torch.zeros((1, 2, 127)))),
        ("Wg shape", lambda: R.rola_gate_logits(_cpu((1, 128, 64)), _cpu((65,)), 0.0, g)),
        ("dY dtype", lambda: R.rola_rope_backward_accumulate(q, cos, cos, g, q.float())),
        # right types and shapes: the layout and device checks come last
        ("strided table", lambda: R.rola_rope_apply(q, torch.zeros((64, 128)).t(),
                                                    torch.zeros((64, 128)).t(), g)),
        ("non-contiguous", lambda: R.rola_dense_attn(q, q.transpose(2, 3).contiguous().transpose(2, 3),
                                                     q, g)),
        ("host tensors", lambda: R.rola_sparse_attn(q, q, q, g, 64, 0.5, idx_ok)),
    ]
    for what, fn in bad:
        with pytest.raises(ValueError):
            fn()
            pytest.fail(what)
