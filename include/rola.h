/*
 * rola.h -- C ABI of librola.so: the RoLA attention module (sparse + rotary low-rank branches) for
 * AMD Instinct MI355X (gfx950).
 *
 * Paper: "RoLA: Rotary-Positioned Low-Rank Linear Attention for Efficient Diffusion Transformers".
 * One attention layer, per (batch b, head h), is the Algorithm "RoLA attention forward pass":
 *   Q^r, K^r = R(Q^n), R(K^n)                         step 3   rola_rope_apply (backbone's job)
 *   blk_idx  = top-k key blocks per query block        step 4   rola_block_select
 *   O^s      = block-sparse softmax attention          step 4   rola_sparse_attn
 *   C, z     = sum_q R_r(q) SiLU(P_k k^n_q) v_q^T      steps 5-6 rola_lowrank_summary
 *   O^lr     = RMSNorm(R_r(p) SiLU(P_q q^n_p))^T C)    steps 5,7 rola_lowrank_readout
 *   O        = (O^s / r + sigma(logit) O^lr) r          steps 8-10 rola_combine
 * rola_lowrank_readout_combine fuses the last two; rola_dense_attn is the dense softmax reference.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tokens lie on a T x Hs x Ws latent grid (Sec. 3, Notation); token n = (t*Hs + y)*Ws + x and
 *    N = T*Hs*Ws.
 *  - Activations Q^n, K^n, Q^r, K^r, V, O^s, O^lr, O: [B, H, N, d_h], contiguous, row-major, element
 *    type `dtype` (fp32 or bf16). P_q, P_k: [H, r, d_h] in `dtype` (the paper's R^{r x d_h} per head).
 *  - Rotary tables cos/sin: fp32 [N, rope_ld], column j = pair j of the backbone ordering
 *    (interleaved pairs (x_{2j}, x_{2j+1}) turned by +angle). rope_ld >= d_h/2 for the full rotation,
 *    >= r/2 for the low-rank branch, which uses columns j < r/2 only (Sec. 4.2).
 *  - Gate logits (X W_g + b_g, one per token, shared by all heads; Sec. 4.4): fp32 [B, N].
 *  - C: fp32 [B, H, r, d_h]; z: fp32 [B, H, r]; block index list: int32 [B, H, n_blocks, keep].
 *  - Every pointer except the problem struct is a device pointer owned by the caller, 16-byte
 *    aligned. The library allocates nothing: scratch comes from the caller (see *_workspace_bytes).
 *    A workspace holds the state of the call it is passed to (lists, partial sums, work-queue
 *    counters) until that call's kernels finish: calls that may run at the same time, e.g. on
 *    different streams, need workspaces of their own.
 *    Inputs are never written; outputs are fully overwritten; outputs must not overlap inputs unless
 *    stated.
 *  - Every call validates all arguments first and launches nothing when one is invalid. It then
 *    enqueues its kernels on `stream` and returns without synchronising. A failed launch returns
 *    ROLA_ERR_HIP. rola_last_error() gives a per-thread message for the last non-OK status.
 *  - Process-wide state: besides the per-thread error message, the library caches, per device and
 *    per variant of the attention kernel, how many of its workgroups the device holds at once
 *    (hipOccupancyMaxActiveBlocksPerMultiprocessor times the compute units, asked on first use of
 *    the variant on that device). The cache is a set of atomics: calls from several threads are
 *    safe, and the value never changes once set.
 *  - Supported: d_h in {64, 128} for fp32, d_h == 128 for bf16; block in {32, 64, 128} (fp32) or
 *    {64, 128} (bf16); r even with 2 <= r <= d_h (fp32) or r in {16, 32, 64, 128} (bf16);
 *    N d_h < 2^31 and B H N < 2^31 (ROLA_ERR_UNSUPPORTED beyond); rope_ld <= 65536 and, in the
 *    attention calls with the epilogue, N rope_ld < 2^31 (per-query offsets are 32-bit).
 */
#ifndef ROLA_H_
#define ROLA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rola_status {
  ROLA_OK = 0,
  ROLA_ERR_INVALID_ARGUMENT = 1, /* null/misaligned pointer, inconsistent sizes, out-of-range value */
  ROLA_ERR_UNSUPPORTED = 2,      /* valid in principle, not built (d_h, block, r, dtype combination) */
  ROLA_ERR_WORKSPACE = 3,        /* workspace smaller than the *_workspace_bytes helper asks for */
  ROLA_ERR_HIP = 4               /* a HIP runtime call or kernel launch failed */
} rola_status;

typedef enum rola_dtype { ROLA_DTYPE_F32 = 0, ROLA_DTYPE_BF16 = 1 } rola_dtype;

/* Problem shape (Sec. 3): Q/K/V are [B, H, N, d_h] on a T x Hs x Ws grid, N == T*Hs*Ws. */
typedef struct rola_problem {
  int32_t B, H, N, d_h;
  int32_t T, Hs, Ws;
  int32_t dtype; /* rola_dtype */
} rola_problem;

/* ---- host-side helpers (no device work) ------------------------------------------------------ */

/* ceil(N / block): contiguous token blocks in flattened order; the last may be partial. -1 if an
 * argument is not positive. */
int32_t rola_num_blocks(int32_t N, int32_t block);

/* Key blocks kept per query block at the given sparsity (the fraction of query-key interactions
 * removed, Sec. 5.1): max(1, min(n_blocks, floor((1 - sparsity) * n_blocks + 0.5))) in double
 * precision. -1 if n_blocks < 1 or sparsity is outside [0, 1). */
int32_t rola_keep_blocks(int32_t n_blocks, double sparsity);

/* Bytes of device workspace rola_block_select needs (pooled block means); 0 if the shape is invalid. */
size_t rola_select_workspace_bytes(const rola_problem* p, int32_t block);

/* Bytes of device workspace rola_lowrank_summary needs (per-chunk partial sums); 0 if invalid. */
size_t rola_summary_workspace_bytes(const rola_problem* p, int32_t r);

const char* rola_status_string(rola_status s);
const char* rola_last_error(void);

/* ---- rotary schedule (Sec. 3 3D RoPE; Sec. 4.2) ---------------------------------------------- */

/* The backbone's rotary tables (freqs_cos, freqs_sin), each fp32 [N, d_h/2]. Axes t, y, x own
 * contiguous runs of d_t/2, d_y/2, d_x/2 pairs (d_t + d_y + d_x == d_h, each even); pair i of an
 * axis of width d_a turns by (pos_a + off_a) * base^(-2i/d_a). Evaluated in fp64, stored fp32. The
 * offsets translate every position (shift-invariance checks); use 0 for the backbone's tables. */
rola_status rola_rope_tables(const rola_problem* p, int32_t d_t, int32_t d_y, int32_t d_x,
                             double base, int32_t off_t, int32_t off_y, int32_t off_x,
                             float* cos_tab, float* sin_tab, hipStream_t stream);

/* Xr = R(X): full 3D RoPE of every [d_h] row of X ([B, H, N, d_h]) with pairs j < d_h/2 (Algorithm
 * step 3, the backbone's main-path rotation). fp32 arithmetic, result rounded to nearest even in
 * `dtype`. Xr must not overlap X. */
rola_status rola_rope_apply(const rola_problem* p, const void* X, const float* cos_tab,
                            const float* sin_tab, int32_t rope_ld, void* Xr, hipStream_t stream);

/* Backward of the main-path rotation, for fine-tuning (Algorithm step 3 transposed): dX += R(p)^T dY
 * for every [d_h] row, i.e. the rotation by -angle, when rotate is nonzero (the gradient of
 * Q^r = R(Q^n) reaching Q^n), else dX += dY (a plain accumulation, e.g. the two branches' shares
 * of dV). dY and dX are fp32 [B, H, N, d_h] whatever p->dtype; dX is read and written, and must
 * not overlap dY. Tables and rope_ld as in rola_rope_apply (read only when rotate is nonzero, but
 * always checked). */
rola_status rola_rope_backward_accumulate(const rola_problem* p, const float* dY,
                                          const float* cos_tab, const float* sin_tab,
                                          int32_t rope_ld, int32_t rotate, float* dX,
                                          hipStream_t stream);

/* The backbone rotation and the block pooling of the selection in one pass (Algorithm steps 3-4):
 * for every [d_h] row x_n of X (Q^n or K^n, [B, H, N, d_h]), R(p) x_n is rounded to dtype exactly
 * as rola_rope_apply rounds it and written to Xr unless Xr is NULL, and Xbar[b, h, I, :] (fp32
 * [B, H, n_blocks, d_h]) receives the mean of the rotated, rounded rows of block I over its valid
 * tokens: bitwise the means rola_block_select computes from Xr. Xr and Xbar must not overlap X or
 * each other. Tables as in rola_rope_apply (rope_ld >= d_h/2). Built for d_h = 128
 * (ROLA_ERR_UNSUPPORTED otherwise). With both tables NULL, X is taken as already rotated (Q^r or
 * K^r): only the means are computed (rope_ld is ignored, Xr must be NULL), on any supported d_h,
 * bitwise those of rola_block_select. Xnorm (optional, 16-byte aligned, fp32 [B, H, n_blocks]):
 * per block the largest norm |x| of its rows (rotated and rounded, fp32 sums of squares); for K
 * this is the key_norm the fused attention calls take to bound their scores. It must not overlap
 * the other buffers. */
rola_status rola_rope_pool(const rola_problem* p, const void* X, const float* cos_tab,
                           const float* sin_tab, int32_t rope_ld, int32_t block, void* Xr,
                           float* Xbar, float* Xnorm, hipStream_t stream);

/* ---- sparse branch (Algorithm step 4; Sec. 4 opening: standard block-sparse attention) -------- */

/* Top-k key blocks for every query block. For each (b, h): q_bar_I, k_bar_J = means of Q^r, K^r over
 * the valid tokens of block I, J (fp32); the block score of the definition is
 * q_bar_I . k_bar_J / sqrt(d_h); the kernels rank the dot products q_bar_I . k_bar_J themselves,
 * since the positive factor 1/sqrt(d_h) cannot change which blocks are largest (and leaving it out
 * adds no rounding). The dot products are fp32-accurate: each mean is split exactly into three
 * bf16 terms and the six significant cross products are summed in fp32 on the matrix cores. The keep = rola_keep_blocks(n_blocks, sparsity) largest scores are kept, equal
 * scores going to the lower J, and written ascending to blk_idx [B, H, n_blocks, keep]. ws: >=
 * rola_select_workspace_bytes(p, block) bytes of device scratch. */
rola_status rola_block_select(const rola_problem* p, const void* Qr, const void* Kr, int32_t block,
                              double sparsity, int32_t* blk_idx, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/* rola_block_select from the block means (rola_rope_pool of Q^n and K^n): the same scores, top-k
 * and lists, bitwise. ws: rola_select_pooled_workspace_bytes(p, block) bytes (the score matrix). */
size_t rola_select_pooled_workspace_bytes(const rola_problem* p, int32_t block);
rola_status rola_block_select_pooled(const rola_problem* p, const float* Qbar, const float* Kbar,
                                     int32_t block, double sparsity, int32_t* blk_idx, void* ws,
                                     size_t ws_bytes, hipStream_t stream);

/* Block-sparse attention: for a query token p in block I, O^s_p = sum softmax(q^r_p . k^r_q * scale)
 * v_q over the valid key tokens q of the blocks blk_idx[b, h, I, :] (keep = rola_keep_blocks(
 * n_blocks, sparsity) entries, each in [0, n_blocks); order irrelevant, duplicates not allowed).
 * Online softmax with fp32 statistics and accumulators; bf16 path on MFMA. scale is normally
 * 1/sqrt(d_h) (Sec. 3). Os: [B, H, N, d_h] in dtype.
 * ws: rola_sparse_workspace_bytes(p, block, sparsity) bytes of device scratch, in which the bf16
 * path with 64-token blocks pairs query blocks (each with the block among its next 64 whose list
 * it shares most, up to 4064 query blocks; adjacent blocks beyond), merges the lists of each pair
 * so that the two share their K/V loads, and keeps the counters of the per-XCD work queues the
 * attention kernel's resident workgroups take pairs from. The merged lists are walked by
 * increasing bit-reversed block index, each from a start phase set by the pair's place in its
 * work queue (a fixed function of the pair and the device's resident workgroup count), so
 * results are deterministic on a given device. ws may be NULL (ws_bytes 0): one query block per
 * workgroup, its list walked in the order given. The two agree up to the order in which each
 * query sums its keys (bitwise on lists given in the order the merged lists walk them). A
 * non-NULL ws smaller than needed is ROLA_ERR_WORKSPACE. */
size_t rola_sparse_workspace_bytes(const rola_problem* p, int32_t block, double sparsity);
rola_status rola_sparse_attn(const rola_problem* p, const void* Qr, const void* Kr, const void* V,
                             int32_t block, double sparsity, const int32_t* blk_idx,
                             float softmax_scale, void* Os, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/* The sparse branch, the low-rank readout and the gated combine in one call (Algorithm steps 4 and
 * 7-10): O = (O^s / r + g O^lr) r with O^s = rola_sparse_attn(...) and O^lr =
 * rola_lowrank_readout(...) of the summary C, without writing O^s or O^lr to memory. Arguments as in
 * those two calls and rola_combine; O: [B, H, N, d_h] in dtype, must not overlap Q^r, K^r, V or
 * Q^n (ROLA_ERR_INVALID_ARGUMENT: other workgroups still read them while O is written). ws:
 * rola_sparse_combine_workspace_bytes(p, block, sparsity, r) bytes, required (the pair lists of
 * rola_sparse_attn plus the C fragments of the epilogue). On the bf16 path with r in {16, 32, 64}
 * the readout and combine run in the attention kernel's epilogue; otherwise the attention and the
 * fused readout + combine run one after the other. Results agree with the separate calls to the
 * module's tolerance (the epilogue combines O^s before its bf16 rounding).
 * Qr may be NULL on the fused path (bf16, r 16-64): the queries are then R(Q^n), rotated from Qn
 * and the tables (rope_ld >= d_h/2 then) in the kernel's prologue and rounded exactly as
 * rola_rope_apply rounds them, so Q^r need not exist in memory; the results are bitwise those with
 * Qr = rola_rope_apply(Qn). Elsewhere Qr = NULL is ROLA_ERR_UNSUPPORTED.
 * key_norm (optional, 16-byte aligned, fp32 [B, H, n_blocks], must not overlap O): for every key
 * block an upper bound on the norms |k^r| of its keys, e.g. the Xnorm of rola_rope_pool on K. On
 * the fused bf16 path with 64-token blocks and a workspace, every pair of query blocks then takes
 * b, the largest bound among the key blocks it walks: each scaled score of a query q lies within
 * B = |q| b scale log2(e) of zero, and every wave of 32 queries whose B are all at most 40 uses B
 * as the fixed reference of its online softmax (no running maximum, no rescaling), which keeps
 * each probability in [2^-80, 1]; other waves track the running maximum as without key_norm. The
 * two references give the same softmax up to rounding (the bf16 rounding of the probabilities and
 * the order of the fp32 sums). With key_norm NULL, or on other paths, it is not read.
 * The same holds for the _planned and _noalloc forms below. */
size_t rola_sparse_combine_workspace_bytes(const rola_problem* p, int32_t block, double sparsity,
                                           int32_t r);
rola_status rola_sparse_attn_combine(const rola_problem* p, const void* Qr, const void* Kr,
                                     const void* V, int32_t block, double sparsity,
                                     const int32_t* blk_idx, float softmax_scale, const void* Qn,
                                     const void* Pq, int32_t r, const float* cos_tab,
                                     const float* sin_tab, int32_t rope_ld, const float* C,
                                     float eps_lr, const float* gate_logits, float eps,
                                     const float* key_norm, void* O, void* ws, size_t ws_bytes,
                                     hipStream_t stream);

/* The same call in two parts, so that other work can run between them (e.g. the low-rank summary,
 * which the epilogue needs, on a second stream while the pairs are planned). rola_sparse_plan
 * pairs the query blocks and merges their lists into ws (the workspace of
 * rola_sparse_attn_combine for the same p, block, sparsity and r, which it must also be given);
 * rola_sparse_attn_combine_planned then runs the attention with its epilogue on that plan. The two
 * must see the same blk_idx, and no other call may use ws in between. On paths without a plan
 * (128-token blocks, fp32) rola_sparse_plan launches nothing. Results are bitwise those of
 * rola_sparse_attn_combine. */
rola_status rola_sparse_plan(const rola_problem* p, int32_t block, double sparsity,
                             const int32_t* blk_idx, int32_t r, void* ws, size_t ws_bytes,
                             hipStream_t stream);
rola_status rola_sparse_attn_combine_planned(
    const rola_problem* p, const void* Qr, const void* Kr, const void* V, int32_t block,
    double sparsity, const int32_t* blk_idx, float softmax_scale, const void* Qn, const void* Pq,
    int32_t r, const float* cos_tab, const float* sin_tab, int32_t rope_ld, const float* C,
    float eps_lr, const float* gate_logits, float eps, const float* key_norm, void* O, void* ws,
    size_t ws_bytes, hipStream_t stream);

/* ---- allocation-free form ---------------------------------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc. rola_sparse_attn_combine_noalloc is rola_sparse_attn_combine
 * without a workspace argument: its scratch (the work-queue counters, pair table and merged lists,
 * the C^T fragments of the epilogue) lives in a static device array of ROLA_NOALLOC_SCRATCH_BYTES
 * bytes, which the library holds on every device it runs on until the process ends; the call
 * itself allocates nothing. A problem whose scratch (rola_sparse_combine_workspace_bytes) is larger
 * is ROLA_ERR_UNSUPPORTED (the Wan2.1-14B 720p layer needs about 23 MB). Every call on a device
 * shares that device's array and leaves its contents behind; each call writes everything it reads
 * (the queue counters are cleared by the call), but calls that overlap in time on one device, from
 * other streams or threads, race on the array and must be ordered by the caller. Results are
 * bitwise those of rola_sparse_attn_combine. */
#define ROLA_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
rola_status rola_sparse_attn_combine_noalloc(
    const rola_problem* p, const void* Qr, const void* Kr, const void* V, int32_t block,
    double sparsity, const int32_t* blk_idx, float softmax_scale, const void* Qn, const void* Pq,
    int32_t r, const float* cos_tab, const float* sin_tab, int32_t rope_ld, const float* C,
    float eps_lr, const float* gate_logits, float eps, const float* key_norm, void* O,
    hipStream_t stream);

/* ---- backward of the sparse branch (fine-tuning, Sec. 4.5; Algorithm step 4) ------------------
 * rola_sparse_attn_lse is rola_sparse_attn (same workspace rule: ws NULL or ws_bytes >=
 * rola_sparse_workspace_bytes) that also writes, per query,
 * lse[b, h, n] = log2 sum_k exp2(q^r_n . k^r_k * scale * log2 e) over its selected keys (fp32
 * [B, H, N]), which the backward needs. rola_sparse_attn_backward returns the gradients of
 * <dOs, O^s> with respect to Q^r, K^r and V (fp32 [B, H, N, d_h] each, fully overwritten) for the
 * given (fixed) block lists: dQ^r = scale dS K^r, dK^r = scale dS^T Q^r, dV = P^T dO^s with
 * P = softmax, dS = P (dO^s V^T - D), D_n = dO^s_n . O^s_n. Os and lse are the forward's outputs, dOs
 * is bf16 [B, H, N, d_h]. ws: rola_sparse_backward_workspace_bytes(p, block, sparsity) bytes (the
 * transposed block lists take 4 (n_b + 1) bytes per key block and head; with 64-token blocks the
 * dQ pass also keeps the pairs, merged lists and queue counters of rola_sparse_attn there). bf16
 * path only, block 64 or 128, at most 16384 blocks per head (ROLA_ERR_UNSUPPORTED otherwise; the
 * workspace size query returns 0 beyond that many blocks). */
rola_status rola_sparse_attn_lse(const rola_problem* p, const void* Qr, const void* Kr,
                                 const void* V, int32_t block, double sparsity,
                                 const int32_t* blk_idx, float softmax_scale, void* Os, float* lse,
                                 void* ws, size_t ws_bytes, hipStream_t stream);
size_t rola_sparse_backward_workspace_bytes(const rola_problem* p, int32_t block, double sparsity);
rola_status rola_sparse_attn_backward(const rola_problem* p, const void* Qr, const void* Kr,
                                      const void* V, int32_t block, double sparsity,
                                      const int32_t* blk_idx, float softmax_scale, const void* Os,
                                      const float* lse, const void* dOs, float* dQr, float* dKr,
                                      float* dV, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- backward of the low-rank branch, the fusion and the gate (fine-tuning, Sec. 4.5) ----------
 * rola_lowrank_backward: gradients of <dO, O> with O = (O^s / r_s + sigma(logit) RMSNorm(q~^T C)) r_s
 * (eq. gate, eq. ctx, eq. qklr; SiLU with the rotation outside) with respect to O^s (dOs, bf16
 * [B, H, N, d_h], the input of rola_sparse_attn_backward), Q^n, K^n and V through the low-rank branch
 * (dQn, dKn, dV: fp32 [B, H, N, d_h]; the sparse branch's shares come from rola_sparse_attn_backward),
 * P_q and P_k (dPq, dPk: fp32 [H, r, d_h], summed over the batch) and the gate logits (dlogits: fp32
 * [B, N], summed over the heads). C is the forward's summary, Os the forward's O^s. Reductions run in
 * a fixed order (reproducible). ws: rola_lowrank_backward_workspace_bytes(p, r). bf16 path with
 * r <= 64 (ROLA_ERR_UNSUPPORTED otherwise).
 * rola_gate_logits_backward: for logits = X W_g + b_g, dX = dlogits W_g^T (fp32 [B, N, d_model];
 * may be NULL), dWg = X^T dlogits (fp32 [d_model]) and dbg = sum dlogits (fp32, one device value).
 * ws: rola_gate_backward_workspace_bytes(p, d_model). */
size_t rola_lowrank_backward_workspace_bytes(const rola_problem* p, int32_t r);
rola_status rola_lowrank_backward(const rola_problem* p, const void* Qn, const void* Kn,
                                  const void* V, const void* Pq, const void* Pk, int32_t r,
                                  const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                  const float* C, const void* Os, const float* gate_logits,
                                  float eps_lr, float eps, const void* dO, void* dOs, float* dQn,
                                  float* dKn, float* dV, float* dPq, float* dPk, float* dlogits,
                                  void* ws, size_t ws_bytes, hipStream_t stream);
size_t rola_gate_backward_workspace_bytes(const rola_problem* p, int32_t d_model);
rola_status rola_gate_logits_backward(const rola_problem* p, const void* X, int32_t d_model,
                                      const void* Wg, const float* dlogits, float* dX, float* dWg,
                                      float* dbg, void* ws, size_t ws_bytes, hipStream_t stream);

/* Dense softmax attention O = softmax(Q^r K^r^T * scale) V (Sec. 3, "Full attention"): the 0 %
 * sparsity reference, same kernel as rola_sparse_attn walking every key block in order. */
rola_status rola_dense_attn(const rola_problem* p, const void* Qr, const void* Kr, const void* V,
                            int32_t block, float softmax_scale, void* O, hipStream_t stream);

/* ---- rotary low-rank branch (eq. qklr, eq. ctx; Algorithm steps 5-7) ------------------------- */

/* Global context C = sum_q k~_q v_q^T (fp32 [B, H, r, d_h]) and z = sum_q k~_q (fp32 [B, H, r];
 * may be NULL), with k~_q = R_r(q) SiLU(P_k k^n_q): projection to rank r, SiLU, then the rotation of
 * pairs j < r/2 (RoPE outside the activation, Sec. 4.3). V is not rotated. Reduced in a fixed order
 * (bitwise reproducible). ws: >= rola_summary_workspace_bytes(p, r) bytes. */
rola_status rola_lowrank_summary(const rola_problem* p, const void* Kn, const void* V,
                                 const void* Pk, int32_t r, const float* cos_tab,
                                 const float* sin_tab, int32_t rope_ld, float* C, float* z,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* O^lr_p = u_p / sqrt(mean_i u_{p,i}^2 + eps_lr) with u_p = q~_p^T C and q~_p = R_r(p) SiLU(P_q q^n_p)
 * (eq. ctx; RMSNorm without gain over d_h). Olr: [B, H, N, d_h] in dtype. */
rola_status rola_lowrank_readout(const rola_problem* p, const void* Qn, const void* Pq, int32_t r,
                                 const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                 const float* C, float eps_lr, void* Olr, hipStream_t stream);

/* ---- low-rank feature variants (Sec. 5.1 "Mechanism-Level Validation", Sec. 5.3 "Ablation
 * Study", Tab. abl_activation; Prop. inside) ----------------------------------------------------
 * The functions above use the paper's design, SiLU with the rotation outside it. The *_ex forms take
 * the feature map phi and the place of the rotation: outside (R_r(p) phi(P x), the paper's design),
 * inside (phi(R_r(p) P x), Prop. inside) or none (phi(P x), position-blind). Everything else is as in
 * the plain forms; phi = ROLA_PHI_SILU with ROLA_ROPE_OUTSIDE gives bitwise their results. An
 * unknown phi or order is ROLA_ERR_INVALID_ARGUMENT. */
typedef enum {
  ROLA_PHI_SILU = 0,      /* x / (1 + e^-x) */
  ROLA_PHI_IDENTITY = 1,  /* x */
  ROLA_PHI_TANH = 2,      /* tanh x */
  ROLA_PHI_RELU = 3,      /* max(x, 0) */
  ROLA_PHI_GELU = 4       /* x Phi(x), Phi the standard normal CDF (erf form) */
} rola_phi;
typedef enum { ROLA_ROPE_OUTSIDE = 0, ROLA_ROPE_INSIDE = 1, ROLA_ROPE_NONE = 2 } rola_rope_order;

rola_status rola_lowrank_summary_ex(const rola_problem* p, const void* Kn, const void* V,
                                    const void* Pk, int32_t r, const float* cos_tab,
                                    const float* sin_tab, int32_t rope_ld, int32_t phi,
                                    int32_t rope_order, float* C, float* z, void* ws,
                                    size_t ws_bytes, hipStream_t stream);
rola_status rola_lowrank_readout_ex(const rola_problem* p, const void* Qn, const void* Pq, int32_t r,
                                    const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                    int32_t phi, int32_t rope_order, const float* C, float eps_lr,
                                    void* Olr, hipStream_t stream);
rola_status rola_lowrank_readout_combine_ex(const rola_problem* p, const void* Qn, const void* Pq,
                                            int32_t r, const float* cos_tab, const float* sin_tab,
                                            int32_t rope_ld, int32_t phi, int32_t rope_order,
                                            const float* C, float eps_lr, const void* Os,
                                            const float* gate_logits, float eps, void* O,
                                            hipStream_t stream);

/* The low-rank features themselves, F[b, h, n, :] = the r-vector x~_n of X[b, h, n, :] under
 * projection P ([H, r, d_h], P_q or P_k), phi and rope_order, pairs (2j, 2j+1) interleaved; fp32
 * [B, H, N, r], fp32 projection. Not a step of the module: it exposes q~ and k~ so that the
 * pre-RMSNorm low-rank logit s(p, q) = q~_p . k~_q of Sec. 5.1 (its dependence on the offset p - q
 * and its shift residual |s(p + d, q + d) - s(p, q)|) can be measured. */
rola_status rola_lowrank_features(const rola_problem* p, const void* X, const void* P, int32_t r,
                                  const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                  int32_t phi, int32_t rope_order, float* F, hipStream_t stream);

/* ---- gated fusion (Sec. 4.4, eq. gate; Algorithm steps 8-10) --------------------------------- */

/* Gate logits of the token-wise gate g = sigmoid(X W_g + b_g) (Sec. 4.4; Algorithm step 8):
 * logits[b, n] = sum_i X[b, n, i] W_g[i] + b_g, fp32 accumulation, fp32 [B, N]; rola_combine and
 * rola_lowrank_readout_combine take these logits and apply the sigmoid. X: the attention block's
 * input hidden states [B, N, d_model] in p->dtype (p->H and p->d_h are not used); W_g: [d_model] in
 * p->dtype; d_model a multiple of 8, at most 16384 (else ROLA_ERR_UNSUPPORTED). */
rola_status rola_gate_logits(const rola_problem* p, const void* X, int32_t d_model, const void* Wg,
                             float bg, float* logits, hipStream_t stream);

/* O_p = (O^s_p / r_p + g_p O^lr_p) r_p, r_p = sqrt(mean_i (O^s_{p,i})^2 + eps), g_p =
 * 1/(1 + exp(-logit_{b,p})). O may alias Os (in place); it must not overlap Olr otherwise. */
rola_status rola_combine(const rola_problem* p, const void* Os, const void* Olr,
                         const float* gate_logits, float eps, void* O, hipStream_t stream);

/* rola_lowrank_readout followed by rola_combine in one pass, without materialising O^lr. O may
 * alias Os. */
rola_status rola_lowrank_readout_combine(const rola_problem* p, const void* Qn, const void* Pq,
                                         int32_t r, const float* cos_tab, const float* sin_tab,
                                         int32_t rope_ld, const float* C, float eps_lr,
                                         const void* Os, const float* gate_logits, float eps,
                                         void* O, hipStream_t stream);

#ifdef __cplusplus
} /* extern "C" */
#endif

#endif /* ROLA_H_ */
