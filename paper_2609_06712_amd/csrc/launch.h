// Internal launcher interface between the C ABI (rola_api.cpp) and the kernels (*.hip).
// Launchers assume their arguments were validated by the ABI layer; they only enqueue work.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rola {

struct Shape {
  int B, H, N, d;      // activations [B, H, N, d]
  int T, Hs, Ws;       // latent grid, N == T*Hs*Ws
  bool bf16;           // element type: bf16 (true) or fp32
};

inline int num_blocks(int N, int block) { return (N + block - 1) / block; }

// rope.hip
hipError_t launch_rope_tables(const Shape& s, int dt, int dy, int dx, double base, int ot, int oy,
                              int ox, float* cos_tab, float* sin_tab, hipStream_t st);
hipError_t launch_rope_apply(const Shape& s, const void* X, const float* cos_tab,
                             const float* sin_tab, int ld, void* Xr, hipStream_t st);
// fp32 [B, H, N, d]: dX += R(p)^T dY (rotate) or dX += dY.
hipError_t launch_rope_grad(const Shape& s, const float* dY, const float* cos_tab,
                            const float* sin_tab, int ld, bool rotate, float* dX, hipStream_t st);

// select.hip
size_t select_workspace_bytes(const Shape& s, int block);
hipError_t launch_block_select(const Shape& s, const void* Qr, const void* Kr, int block, int keep,
                               int32_t* idx, void* ws, hipStream_t st);
// Means of the rotated rows per block from Q^n or K^n and the tables (fp32 [B, H, nb, d]); the
// rotated rows also go to Xr unless it is null. Built for d = 128 (rope_pool_supported). nmax, if
// not null: per block the largest fp32 norm of its (rotated, rounded) rows, [B, H, nb].
bool rope_pool_supported(const Shape& s, int block);
// Block means of an already rotated X (the pooling of launch_block_select alone).
hipError_t launch_block_pool(const Shape& s, const void* X, int block, float* means, float* nmax,
                             hipStream_t st);
hipError_t launch_rope_pool(const Shape& s, const void* X, const float* cos_tab,
                            const float* sin_tab, int ld, int block, void* Xr, float* means,
                            float* nmax, hipStream_t st);
// Scores and top-k from given means; ws: select_pooled_workspace_bytes(s, block).
size_t select_pooled_workspace_bytes(const Shape& s, int block);
hipError_t launch_select_pooled(const Shape& s, const float* qbar, const float* kbar, int block,
                                int keep, int32_t* idx, void* ws, hipStream_t st);

// sparse_attn.hip  (idx == nullptr: dense, every key block in order; keep must equal n_blocks)
// ws: sparse_workspace_bytes(s, block, keep) bytes, or nullptr (then no K/V loads are shared
// between query blocks).
size_t sparse_workspace_bytes(const Shape& s, int block, int keep);
// The low-rank readout and gated combine fused into the attention epilogue (bf16, d 128, r 16-64):
// Os then receives O = combine(O^s, RMSNorm(q~^T C), logits). fuse_ws: fuse_workspace_bytes(s, r).
struct LowrankFuse {
  const void* Qn;
  const void* Pq;
  int r;
  const float* cos_tab;
  const float* sin_tab;
  int ld;
  const float* C;
  float eps_lr;
  const float* logits;
  float eps;
  const float* knorm;  // optional: per key block the largest key norm, [B, H, nb] (score bound)
};
bool fuse_supported(const Shape& s, int r);
size_t fuse_workspace_bytes(const Shape& s, int r);
// lse (optional, bf16 path): [B, H, N] fp32, log2 of each query's softmax denominator of the
// log2e-scaled scores, i.e. P = exp2(S * scale * log2e - lse).
// planned: ws already holds the groups of these lists (launch_sparse_plan with the same r), so the
// pairing and list merge are not launched again.
hipError_t launch_sparse_attn(const Shape& s, const void* Qr, const void* Kr, const void* V,
                              int block, int keep, const int32_t* idx, float scale, void* Os,
                              void* ws, hipStream_t st, const LowrankFuse* lf = nullptr,
                              void* fuse_ws = nullptr, float* lse = nullptr, bool planned = false);
// Whether the path of (s, block) uses a plan (pairs, merged lists, queue counters in ws).
bool plan_used(const Shape& s, int block);
// The pairing and list merge of the 64-token bf16 path into ws (sparse_workspace_bytes), for the
// walk period of the kernel variant with fused rank r (0: plain attention). No-op elsewhere.
hipError_t launch_sparse_plan(const Shape& s, int keep, const int32_t* idx, int r, void* ws,
                              hipStream_t st);
// The per-device static scratch of the allocation-free entry point: its size, and its address on
// the current device (asked once per device, then cached).
size_t static_scratch_bytes();
hipError_t static_scratch(void** ptr);

// lowrank_bwd.hip: gradients of the low-rank branch and the gated fusion (bf16, d 128, r <= 64, SiLU
// with the rotation outside). dOs bf16; the other gradients fp32; dP_q, dP_k summed over the batch,
// dlogits over the heads. ws: lowrank_backward_workspace_bytes(s, r).
size_t lowrank_backward_workspace_bytes(const Shape& s, int r);
hipError_t launch_lowrank_backward(const Shape& s, const void* Qn, const void* Kn, const void* V,
                                   const void* Pq, const void* Pk, int r, const float* cos_tab,
                                   const float* sin_tab, int ld, const float* C, const void* Os,
                                   const float* logits, float eps_lr, float eps, const void* dO,
                                   void* dOs, float* dQn, float* dKn, float* dV, float* dPq,
                                   float* dPk, float* dlogits, void* ws, hipStream_t st);

// sparse_attn.hip: dQ^r of the block-sparse attention on the paired, queued attention kernel
// (bf16, d 128, block 64: dq_supported); lseD: per query {log-sum-exp (log2), D = dO^s . O^s};
// ws: sparse_workspace_bytes(s, 64, keep).
bool dq_supported(const Shape& s, int block);
hipError_t launch_sparse_dq(const Shape& s, const void* Qr, const void* Kr, const void* V, int keep,
                            const int32_t* idx, float scale, const void* dO, const void* lseD,
                            float* dQ, void* ws, hipStream_t st);

// sparse_bwd.hip: gradients of the block-sparse attention (bf16, d 128, block 64 or 128, at most
// kBwdMaxBlocks blocks per head: the transposed lists are built through one LDS word per block);
// fp32 outputs; ws: sparse_backward_workspace_bytes(s, block, keep), 0 when unsupported.
constexpr int kBwdMaxBlocks = 16384;
size_t sparse_backward_workspace_bytes(const Shape& s, int block, int keep);
hipError_t launch_sparse_backward(const Shape& s, const void* Qr, const void* Kr, const void* V,
                                  int block, int keep, const int32_t* idx, float scale,
                                  const void* Os, const float* lse, const void* dOs, float* dQ,
                                  float* dK, float* dV, void* ws, hipStream_t st);

// lowrank.hip
int summary_chunks(const Shape& s, int r);
size_t summary_workspace_bytes(const Shape& s, int r);
// feat: feature map phi | rotation order << 8 (the ROLA_PHI_* / ROLA_ROPE_* values; 0 = SiLU with
// the rotation outside, the paper's design).
hipError_t launch_lowrank_summary(const Shape& s, const void* Kn, const void* V, const void* Pk,
                                  int r, const float* cos_tab, const float* sin_tab, int ld,
                                  int feat, float* C, float* z, void* ws, hipStream_t st);
// Os == nullptr: plain readout into Out; otherwise readout fused with the gated combine.
hipError_t launch_lowrank_readout(const Shape& s, const void* Qn, const void* Pq, int r,
                                  const float* cos_tab, const float* sin_tab, int ld, int feat,
                                  const float* C, float eps_lr, const void* Os,
                                  const float* logits, float eps, void* Out, hipStream_t st);
// Features of every token, fp32 [B, H, N, r].
hipError_t launch_lowrank_features(const Shape& s, const void* X, const void* P, int r,
                                   const float* cos_tab, const float* sin_tab, int ld, int feat,
                                   float* F, hipStream_t st);
hipError_t launch_combine(const Shape& s, const void* Os, const void* Olr, const float* logits,
                          float eps, void* O, hipStream_t st);

// gate.hip: logits [B, N] = X [B, N, d_model] . Wg + bg (d_model % 8 == 0, <= gate_max_model()).
hipError_t launch_gate_logits(const Shape& s, const void* X, int d_model, const void* Wg, float bg,
                              float* logits, hipStream_t st);
int gate_max_model();
// Backward of the gate logits: dX (optional, fp32 [B, N, d_model]) = dlogits W_g; dWg (fp32 [d_model])
// = sum dlogits X; dbg (fp32 scalar) = sum dlogits. ws: gate_backward_workspace_bytes(d_model).
size_t gate_backward_workspace_bytes(int d_model);
hipError_t launch_gate_backward(const Shape& s, const void* X, int d_model, const void* Wg,
                                const float* dlogits, float* dX, float* dWg, float* dbg, void* ws,
                                hipStream_t st);

}  // namespace rola
