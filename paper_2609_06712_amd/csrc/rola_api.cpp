// C ABI of librola.so (declared in include/rola.h): argument validation, workspace sizing, status
// reporting, then dispatch to the kernel launchers. Validation runs entirely on the host and touches
// no device, so every invalid call returns before anything is enqueued.
#include "rola.h"

#include <math.h>

#include <algorithm>
#include <initializer_list>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "launch.h"

namespace {

thread_local char g_last_error[512] = "";

rola_status fail(rola_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

rola_status hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return ROLA_OK;
  return fail(ROLA_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned(const void* p) { return p != nullptr && ((uintptr_t)p & 15u) == 0; }

#define REQUIRE_PTR(p)                                                                      \
  do {                                                                                      \
    if (!aligned(p))                                                                        \
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: pointer '%s' is null or not 16-byte aligned", \
                  __func__, #p);                                                            \
  } while (0)

rola_status check_problem(const rola_problem* p, const char* fn, rola::Shape* out) {
  if (!p) return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: problem is null", fn);
  if (p->B < 1 || p->H < 1 || p->N < 1 || p->T < 1 || p->Hs < 1 || p->Ws < 1)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: sizes must be positive (B=%d H=%d N=%d T=%d Hs=%d Ws=%d)",
                fn, p->B, p->H, p->N, p->T, p->Hs, p->Ws);
  // products of positive int32 values in 128 bits: no overflow for any input
  typedef unsigned __int128 u128;
  const u128 grid = (u128)p->T * (u128)p->Hs * (u128)p->Ws;
  if (grid != (u128)p->N)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: N=%d differs from T*Hs*Ws (T=%d Hs=%d Ws=%d)", fn,
                p->N, p->T, p->Hs, p->Ws);
  if (p->dtype != ROLA_DTYPE_F32 && p->dtype != ROLA_DTYPE_BF16)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: unknown dtype %d", fn, p->dtype);
  if (p->d_h != 64 && p->d_h != 128)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: d_h=%d (built: 64, 128)", fn, p->d_h);
  if (p->dtype == ROLA_DTYPE_BF16 && p->d_h != 128)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: bf16 path is built for d_h=128 only (got %d)", fn, p->d_h);
  if ((u128)p->B * (u128)p->H * (u128)p->N * (u128)p->d_h >= ((u128)1 << 40))
    return fail(ROLA_ERR_UNSUPPORTED, "%s: tensor too large", fn);
  if ((u128)p->N * (u128)p->d_h > (u128)((1ll << 31) - 1))
    return fail(ROLA_ERR_UNSUPPORTED, "%s: N*d_h must be below 2^31", fn);
  if ((u128)p->B * (u128)p->H * (u128)p->N > (u128)((1ll << 31) - 1))
    return fail(ROLA_ERR_UNSUPPORTED, "%s: B*H*N must fit in int32", fn);
  *out = rola::Shape{p->B, p->H, p->N, p->d_h, p->T, p->Hs, p->Ws, p->dtype == ROLA_DTYPE_BF16};
  return ROLA_OK;
}

rola_status check_block(const rola::Shape& s, int32_t block, const char* fn) {
  if (block != 32 && block != 64 && block != 128)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: block=%d (built: 32, 64, 128)", fn, block);
  if (s.bf16 && block == 32)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: bf16 path is built for block 64 and 128", fn);
  if (rola::num_blocks(s.N, block) > 8192)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: more than 8192 blocks", fn);
  if ((long long)rola::num_blocks(s.N, block) * s.H * s.B > 0x7fffffffll)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: too many blocks", fn);
  return ROLA_OK;
}

rola_status check_rank(const rola::Shape& s, int32_t r, const char* fn) {
  if (r < 2 || r > s.d || (r & 1))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: rank r=%d must be even with 2 <= r <= d_h=%d", fn, r, s.d);
  if (s.bf16 && r != 16 && r != 32 && r != 64 && r != 128)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: bf16 path is built for r in {16, 32, 64, 128} (got %d)", fn, r);
  return ROLA_OK;
}

rola_status check_feature(int32_t phi, int32_t order, const char* fn, int* feat) {
  if (phi < ROLA_PHI_SILU || phi > ROLA_PHI_GELU)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: unknown feature map phi = %d", fn, (int)phi);
  if (order < ROLA_ROPE_OUTSIDE || order > ROLA_ROPE_NONE)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: unknown rotation order %d", fn, (int)order);
  *feat = phi | order << 8;  // the kernels' encoding
  return ROLA_OK;
}

rola_status check_tables(const float* c, const float* s, int32_t ld, int32_t need, const char* fn) {
  if (!aligned(c) || !aligned(s))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: rotary tables null or not 16-byte aligned", fn);
  if (ld < need || (ld % 4) != 0 || ld > (1 << 16))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: rope_ld=%d must be a multiple of 4, >= %d and <= 65536",
                fn, ld, need);
  return ROLA_OK;
}

rola_status check_sparsity(double sparsity, const char* fn) {
  if (!(sparsity >= 0.0 && sparsity < 1.0))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: sparsity %g outside [0, 1)", fn, sparsity);
  return ROLA_OK;
}

// Whether the byte ranges [a, a + na) and [b, b + nb) overlap.
bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

// Bytes of one [B, H, N, d] activation tensor.
size_t act_bytes(const rola::Shape& s) {
  return (size_t)s.B * s.H * s.N * s.d * (s.bf16 ? 2 : 4);
}

// An output activation must not overlap the input activations `ins` (other workgroups still read
// them while it is written); `same` (nullable) is an input it may alias exactly (in-place forms).
struct Named {
  const void* p;
  const char* name;
};
rola_status check_out(const rola::Shape& s, const void* out, std::initializer_list<Named> ins,
                      const void* same, const char* fn) {
  const size_t n = act_bytes(s);
  for (const Named& in : ins) {
    if (in.p == nullptr || (in.p == same && out == same)) continue;
    if (overlap(out, n, in.p, n))
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: the output overlaps %s", fn, in.name);
  }
  return ROLA_OK;
}

#define TRY(expr)                     \
  do {                                \
    rola_status _s = (expr);          \
    if (_s != ROLA_OK) return _s;     \
  } while (0)

// Arguments of the attention + readout + combine calls other than the workspace, checked before
// anything is launched.
rola_status check_combine(const rola_problem* p, const void* Qr, const void* Kr, const void* V,
                          int32_t block, double sparsity, const int32_t* blk_idx,
                          float softmax_scale, const void* Qn, const void* Pq, int32_t r,
                          const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                          const float* C, float eps_lr, const float* gate_logits, float eps,
                          const float* key_norm, void* O, const char* fn, rola::Shape* s) {
  TRY(check_problem(p, fn, s));
  TRY(check_block(*s, block, fn));
  TRY(check_sparsity(sparsity, fn));
  TRY(check_rank(*s, r, fn));
  const void* ptrs[] = {Kr, V, blk_idx, Qn, Pq, C, gate_logits, O};
  const char* names[] = {"Kr", "V", "blk_idx", "Qn", "Pq", "C", "gate_logits", "O"};
  for (int i = 0; i < 8; ++i)
    if (!aligned(ptrs[i]))
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: pointer '%s' is null or not 16-byte aligned", fn,
                  names[i]);
  if (Qr == nullptr) {  // queries rotated from Q^n in the kernel's prologue
    if (!rola::fuse_supported(*s, r))
      return fail(ROLA_ERR_UNSUPPORTED, "%s: Qr = NULL needs the fused bf16 path (r 16-64)", fn);
    TRY(check_tables(cos_tab, sin_tab, rope_ld, s->d / 2, fn));
  } else if (!aligned(Qr)) {
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: pointer 'Qr' is not 16-byte aligned", fn);
  }
  TRY(check_tables(cos_tab, sin_tab, rope_ld, r / 2, fn));
  if ((unsigned __int128)s->N * (unsigned)rope_ld > (unsigned __int128)((1ll << 31) - 1))
    return fail(ROLA_ERR_UNSUPPORTED, "%s: N*rope_ld must be below 2^31", fn);
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: softmax_scale must be finite and positive", fn);
  if (!(eps_lr >= 0.f) || !isfinite(eps_lr) || !(eps >= 0.f) || !isfinite(eps))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: eps values must be finite and >= 0", fn);
  TRY(check_out(*s, O, {{Qr, "Qr"}, {Kr, "Kr"}, {V, "V"}, {Qn, "Qn"}}, nullptr, fn));
  if (key_norm != nullptr) {
    if (!aligned(key_norm))
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: key_norm not 16-byte aligned", fn);
    const size_t nk = (size_t)s->B * s->H * rola::num_blocks(s->N, block) * sizeof(float);
    if (overlap(key_norm, nk, O, act_bytes(*s)))
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: key_norm overlaps O", fn);
  }
  return ROLA_OK;
}

rola_status run_combine(const rola::Shape& s, const void* Qr, const void* Kr, const void* V,
                        int32_t block, int keep, const int32_t* blk_idx, float softmax_scale,
                        const void* Qn, const void* Pq, int32_t r, const float* cos_tab,
                        const float* sin_tab, int32_t rope_ld, const float* C, float eps_lr,
                        const float* gate_logits, float eps, const float* key_norm, void* O,
                        void* ws, bool planned, hipStream_t stream, const char* fn) {
  const size_t sp = rola::sparse_workspace_bytes(s, block, keep);
  void* fuse_ws = static_cast<char*>(ws) + ((sp + 255) & ~(size_t)255);
  if (rola::fuse_supported(s, r)) {
    const rola::LowrankFuse lf{Qn, Pq, r, cos_tab, sin_tab, rope_ld, C, eps_lr, gate_logits, eps,
                               key_norm};
    return hip_status(rola::launch_sparse_attn(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale, O,
                                               sp > 0 ? ws : nullptr, stream, &lf, fuse_ws, nullptr,
                                               planned),
                      fn);
  }
  // other shapes: the attention into O, then the readout and combine in place
  hipError_t e = rola::launch_sparse_attn(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale, O,
                                          sp > 0 ? ws : nullptr, stream, nullptr, nullptr, nullptr,
                                          planned);
  if (e == hipSuccess)
    e = rola::launch_lowrank_readout(s, Qn, Pq, r, cos_tab, sin_tab, rope_ld, 0, C, eps_lr, O,
                                     gate_logits, eps, O, stream);
  return hip_status(e, fn);
}


}  // namespace

extern "C" {

int32_t rola_num_blocks(int32_t N, int32_t block) {
  if (N < 1 || block < 1) return -1;
  return rola::num_blocks(N, block);
}

int32_t rola_keep_blocks(int32_t n_blocks, double sparsity) {
  if (n_blocks < 1 || !(sparsity >= 0.0 && sparsity < 1.0)) return -1;
  const double k = floor((1.0 - sparsity) * (double)n_blocks + 0.5);
  if (k < 1.0) return 1;
  if (k > (double)n_blocks) return n_blocks;
  return (int32_t)k;
}

size_t rola_select_workspace_bytes(const rola_problem* p, int32_t block) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || check_block(s, block, __func__) != ROLA_OK) return 0;
  return rola::select_workspace_bytes(s, block);
}

size_t rola_summary_workspace_bytes(const rola_problem* p, int32_t r) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || check_rank(s, r, __func__) != ROLA_OK) return 0;
  return rola::summary_workspace_bytes(s, r);
}

const char* rola_status_string(rola_status s) {
  switch (s) {
    case ROLA_OK: return "ROLA_OK";
    case ROLA_ERR_INVALID_ARGUMENT: return "ROLA_ERR_INVALID_ARGUMENT";
    case ROLA_ERR_UNSUPPORTED: return "ROLA_ERR_UNSUPPORTED";
    case ROLA_ERR_WORKSPACE: return "ROLA_ERR_WORKSPACE";
    case ROLA_ERR_HIP: return "ROLA_ERR_HIP";
  }
  return "ROLA_ERR_UNKNOWN";
}

const char* rola_last_error(void) { return g_last_error; }

rola_status rola_rope_tables(const rola_problem* p, int32_t d_t, int32_t d_y, int32_t d_x,
                             double base, int32_t off_t, int32_t off_y, int32_t off_x,
                             float* cos_tab, float* sin_tab, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  REQUIRE_PTR(cos_tab);
  REQUIRE_PTR(sin_tab);
  if (d_t < 2 || d_y < 2 || d_x < 2 || (d_t | d_y | d_x) & 1 || d_t + d_y + d_x != s.d)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: axis widths (%d, %d, %d) must be even, >= 2, and sum to d_h=%d",
                __func__, d_t, d_y, d_x, s.d);
  if (!(base > 1.0) || !isfinite(base))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: base %g must be finite and > 1", __func__, base);
  return hip_status(rola::launch_rope_tables(s, d_t, d_y, d_x, base, off_t, off_y, off_x, cos_tab,
                                             sin_tab, stream), __func__);
}

rola_status rola_rope_apply(const rola_problem* p, const void* X, const float* cos_tab,
                            const float* sin_tab, int32_t rope_ld, void* Xr, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  REQUIRE_PTR(X);
  REQUIRE_PTR(Xr);
  TRY(check_tables(cos_tab, sin_tab, rope_ld, s.d / 2, __func__));
  TRY(check_out(s, Xr, {{X, "X"}}, nullptr, __func__));
  return hip_status(rola::launch_rope_apply(s, X, cos_tab, sin_tab, rope_ld, Xr, stream), __func__);
}

rola_status rola_rope_backward_accumulate(const rola_problem* p, const float* dY,
                                          const float* cos_tab, const float* sin_tab,
                                          int32_t rope_ld, int32_t rotate, float* dX,
                                          hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  REQUIRE_PTR(dY);
  REQUIRE_PTR(dX);
  TRY(check_tables(cos_tab, sin_tab, rope_ld, s.d / 2, __func__));
  const size_t n = (size_t)s.B * s.H * s.N * s.d * sizeof(float);
  if (overlap(dX, n, dY, n))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: dX overlaps dY", __func__);
  return hip_status(rola::launch_rope_grad(s, dY, cos_tab, sin_tab, rope_ld, rotate != 0, dX, stream),
                    __func__);
}

rola_status rola_rope_pool(const rola_problem* p, const void* X, const float* cos_tab,
                           const float* sin_tab, int32_t rope_ld, int32_t block, void* Xr,
                           float* Xbar, float* Xnorm, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  REQUIRE_PTR(X);
  REQUIRE_PTR(Xbar);
  if (Xr != nullptr && !aligned(Xr))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: Xr not 16-byte aligned", __func__);
  if (Xnorm != nullptr && !aligned(Xnorm))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: Xnorm not 16-byte aligned", __func__);
  const size_t nblk = (size_t)s.B * s.H * rola::num_blocks(s.N, block);
  const size_t nbar = nblk * s.d * sizeof(float), nnorm = Xnorm ? nblk * sizeof(float) : 0;
  if (Xnorm && (overlap(Xnorm, nnorm, X, act_bytes(s)) || overlap(Xnorm, nnorm, Xbar, nbar) ||
                (Xr && overlap(Xnorm, nnorm, Xr, act_bytes(s)))))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: Xnorm overlaps X, Xr or Xbar", __func__);
  if (cos_tab == nullptr && sin_tab == nullptr) {  // X is already rotated: pooling only
    if (Xr != nullptr)
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: Xr must be NULL without tables", __func__);
    if (overlap(Xbar, nbar, X, act_bytes(s)))
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: Xbar overlaps X", __func__);
    return hip_status(rola::launch_block_pool(s, X, block, Xbar, Xnorm, stream), __func__);
  }
  TRY(check_tables(cos_tab, sin_tab, rope_ld, s.d / 2, __func__));
  if (!rola::rope_pool_supported(s, block))
    return fail(ROLA_ERR_UNSUPPORTED, "%s: built for d_h = 128", __func__);
  if (Xr) TRY(check_out(s, Xr, {{X, "X"}}, nullptr, __func__));
  if (overlap(Xbar, nbar, X, act_bytes(s)) || (Xr && overlap(Xbar, nbar, Xr, act_bytes(s))))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: Xbar overlaps X or Xr", __func__);
  return hip_status(rola::launch_rope_pool(s, X, cos_tab, sin_tab, rope_ld, block, Xr, Xbar, Xnorm,
                                           stream),
                    __func__);
}

size_t rola_select_pooled_workspace_bytes(const rola_problem* p, int32_t block) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || check_block(s, block, __func__) != ROLA_OK) return 0;
  return rola::select_pooled_workspace_bytes(s, block);
}

rola_status rola_block_select_pooled(const rola_problem* p, const float* Qbar, const float* Kbar,
                                     int32_t block, double sparsity, int32_t* blk_idx, void* ws,
                                     size_t ws_bytes, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  TRY(check_sparsity(sparsity, __func__));
  REQUIRE_PTR(Qbar);
  REQUIRE_PTR(Kbar);
  REQUIRE_PTR(blk_idx);
  REQUIRE_PTR(ws);
  const size_t need = rola::select_pooled_workspace_bytes(s, block);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  const int nb = rola::num_blocks(s.N, block);
  const int keep = rola_keep_blocks(nb, sparsity);
  return hip_status(rola::launch_select_pooled(s, Qbar, Kbar, block, keep, blk_idx, ws, stream),
                    __func__);
}

rola_status rola_block_select(const rola_problem* p, const void* Qr, const void* Kr, int32_t block,
                              double sparsity, int32_t* blk_idx, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  TRY(check_sparsity(sparsity, __func__));
  REQUIRE_PTR(Qr);
  REQUIRE_PTR(Kr);
  REQUIRE_PTR(blk_idx);
  REQUIRE_PTR(ws);
  const size_t need = rola::select_workspace_bytes(s, block);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  const int nb = rola::num_blocks(s.N, block);
  const int keep = rola_keep_blocks(nb, sparsity);
  return hip_status(rola::launch_block_select(s, Qr, Kr, block, keep, blk_idx, ws, stream), __func__);
}

size_t rola_sparse_workspace_bytes(const rola_problem* p, int32_t block, double sparsity) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || check_block(s, block, __func__) != ROLA_OK ||
      check_sparsity(sparsity, __func__) != ROLA_OK)
    return 0;
  return rola::sparse_workspace_bytes(s, block, rola_keep_blocks(rola::num_blocks(s.N, block), sparsity));
}

rola_status rola_sparse_attn(const rola_problem* p, const void* Qr, const void* Kr, const void* V,
                             int32_t block, double sparsity, const int32_t* blk_idx,
                             float softmax_scale, void* Os, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  TRY(check_sparsity(sparsity, __func__));
  REQUIRE_PTR(Qr);
  REQUIRE_PTR(Kr);
  REQUIRE_PTR(V);
  REQUIRE_PTR(blk_idx);
  REQUIRE_PTR(Os);
  TRY(check_out(s, Os, {{Qr, "Qr"}, {Kr, "Kr"}, {V, "V"}}, nullptr, __func__));
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: softmax_scale must be finite and positive", __func__);
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  const size_t need = rola::sparse_workspace_bytes(s, block, keep);
  if (ws && need > 0) {
    if (reinterpret_cast<uintptr_t>(ws) % 16)
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: ws must be 16-byte aligned", __func__);
    if (ws_bytes < need)
      return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  }
  return hip_status(rola::launch_sparse_attn(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale, Os,
                                             need > 0 ? ws : nullptr, stream), __func__);
}

rola_status rola_dense_attn(const rola_problem* p, const void* Qr, const void* Kr, const void* V,
                            int32_t block, float softmax_scale, void* O, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  REQUIRE_PTR(Qr);
  REQUIRE_PTR(Kr);
  REQUIRE_PTR(V);
  REQUIRE_PTR(O);
  TRY(check_out(s, O, {{Qr, "Qr"}, {Kr, "Kr"}, {V, "V"}}, nullptr, __func__));
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: softmax_scale must be finite and positive", __func__);
  const int nb = rola::num_blocks(s.N, block);
  return hip_status(rola::launch_sparse_attn(s, Qr, Kr, V, block, nb, nullptr, softmax_scale, O,
                                             nullptr, stream), __func__);
}

rola_status rola_sparse_attn_lse(const rola_problem* p, const void* Qr, const void* Kr,
                                 const void* V, int32_t block, double sparsity,
                                 const int32_t* blk_idx, float softmax_scale, void* Os, float* lse,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  TRY(check_sparsity(sparsity, __func__));
  if (!s.bf16) return fail(ROLA_ERR_UNSUPPORTED, "%s: built for the bf16 path", __func__);
  REQUIRE_PTR(Qr);
  REQUIRE_PTR(Kr);
  REQUIRE_PTR(V);
  REQUIRE_PTR(blk_idx);
  REQUIRE_PTR(Os);
  REQUIRE_PTR(lse);
  TRY(check_out(s, Os, {{Qr, "Qr"}, {Kr, "Kr"}, {V, "V"}}, nullptr, __func__));
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: softmax_scale must be finite and positive", __func__);
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  const size_t need = rola::sparse_workspace_bytes(s, block, keep);
  if (ws && need > 0) {
    if (reinterpret_cast<uintptr_t>(ws) % 16)
      return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: ws must be 16-byte aligned", __func__);
    if (ws_bytes < need)
      return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  }
  return hip_status(rola::launch_sparse_attn(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale, Os,
                                             need > 0 ? ws : nullptr, stream, nullptr, nullptr, lse),
                    __func__);
}

size_t rola_sparse_backward_workspace_bytes(const rola_problem* p, int32_t block, double sparsity) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || check_block(s, block, __func__) != ROLA_OK ||
      check_sparsity(sparsity, __func__) != ROLA_OK)
    return 0;
  return rola::sparse_backward_workspace_bytes(
      s, block, rola_keep_blocks(rola::num_blocks(s.N, block), sparsity));
}

rola_status rola_sparse_attn_backward(const rola_problem* p, const void* Qr, const void* Kr,
                                      const void* V, int32_t block, double sparsity,
                                      const int32_t* blk_idx, float softmax_scale, const void* Os,
                                      const float* lse, const void* dOs, float* dQr, float* dKr,
                                      float* dV, void* ws, size_t ws_bytes, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  TRY(check_sparsity(sparsity, __func__));
  if (!s.bf16) return fail(ROLA_ERR_UNSUPPORTED, "%s: built for the bf16 path", __func__);
  if (rola::num_blocks(s.N, block) > rola::kBwdMaxBlocks)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: %d blocks per head, at most %d", __func__,
                rola::num_blocks(s.N, block), rola::kBwdMaxBlocks);
  REQUIRE_PTR(Qr);
  REQUIRE_PTR(Kr);
  REQUIRE_PTR(V);
  REQUIRE_PTR(blk_idx);
  REQUIRE_PTR(Os);
  REQUIRE_PTR(lse);
  REQUIRE_PTR(dOs);
  REQUIRE_PTR(dQr);
  REQUIRE_PTR(dKr);
  REQUIRE_PTR(dV);
  REQUIRE_PTR(ws);
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: softmax_scale must be finite and positive", __func__);
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  const size_t need = rola::sparse_backward_workspace_bytes(s, block, keep);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  if (reinterpret_cast<uintptr_t>(ws) % 16)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: ws must be 16-byte aligned", __func__);
  return hip_status(rola::launch_sparse_backward(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale,
                                                 Os, lse, dOs, dQr, dKr, dV, ws, stream),
                    __func__);
}

size_t rola_sparse_combine_workspace_bytes(const rola_problem* p, int32_t block, double sparsity,
                                           int32_t r) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || check_block(s, block, __func__) != ROLA_OK ||
      check_sparsity(sparsity, __func__) != ROLA_OK || check_rank(s, r, __func__) != ROLA_OK)
    return 0;
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  const size_t sp = (rola::sparse_workspace_bytes(s, block, keep) + 255) & ~(size_t)255;
  return sp + std::max<size_t>(rola::fuse_workspace_bytes(s, r), 16);
}


rola_status rola_sparse_attn_combine(const rola_problem* p, const void* Qr, const void* Kr,
                                     const void* V, int32_t block, double sparsity,
                                     const int32_t* blk_idx, float softmax_scale, const void* Qn,
                                     const void* Pq, int32_t r, const float* cos_tab,
                                     const float* sin_tab, int32_t rope_ld, const float* C,
                                     float eps_lr, const float* gate_logits, float eps,
                                     const float* key_norm, void* O, void* ws, size_t ws_bytes,
                                     hipStream_t stream) {
  rola::Shape s;
  TRY(check_combine(p, Qr, Kr, V, block, sparsity, blk_idx, softmax_scale, Qn, Pq, r, cos_tab,
                    sin_tab, rope_ld, C, eps_lr, gate_logits, eps, key_norm, O, __func__, &s));
  REQUIRE_PTR(ws);
  const size_t need = rola_sparse_combine_workspace_bytes(p, block, sparsity, r);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  return run_combine(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale, Qn, Pq, r, cos_tab, sin_tab,
                     rope_ld, C, eps_lr, gate_logits, eps, key_norm, O, ws, false, stream, __func__);
}

rola_status rola_sparse_plan(const rola_problem* p, int32_t block, double sparsity,
                             const int32_t* blk_idx, int32_t r, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_block(s, block, __func__));
  TRY(check_sparsity(sparsity, __func__));
  TRY(check_rank(s, r, __func__));
  REQUIRE_PTR(blk_idx);
  REQUIRE_PTR(ws);
  const size_t need = rola_sparse_combine_workspace_bytes(p, block, sparsity, r);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  if (!rola::plan_used(s, block)) return ROLA_OK;
  return hip_status(rola::launch_sparse_plan(s, keep, blk_idx, rola::fuse_supported(s, r) ? r : 0,
                                             ws, stream),
                    __func__);
}

rola_status rola_sparse_attn_combine_planned(
    const rola_problem* p, const void* Qr, const void* Kr, const void* V, int32_t block,
    double sparsity, const int32_t* blk_idx, float softmax_scale, const void* Qn, const void* Pq,
    int32_t r, const float* cos_tab, const float* sin_tab, int32_t rope_ld, const float* C,
    float eps_lr, const float* gate_logits, float eps, const float* key_norm, void* O, void* ws,
    size_t ws_bytes, hipStream_t stream) {
  rola::Shape s;
  TRY(check_combine(p, Qr, Kr, V, block, sparsity, blk_idx, softmax_scale, Qn, Pq, r, cos_tab,
                    sin_tab, rope_ld, C, eps_lr, gate_logits, eps, key_norm, O, __func__, &s));
  REQUIRE_PTR(ws);
  const size_t need = rola_sparse_combine_workspace_bytes(p, block, sparsity, r);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  return run_combine(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale, Qn, Pq, r, cos_tab, sin_tab,
                     rope_ld, C, eps_lr, gate_logits, eps, key_norm, O, ws, true, stream, __func__);
}

rola_status rola_sparse_attn_combine_noalloc(
    const rola_problem* p, const void* Qr, const void* Kr, const void* V, int32_t block,
    double sparsity, const int32_t* blk_idx, float softmax_scale, const void* Qn, const void* Pq,
    int32_t r, const float* cos_tab, const float* sin_tab, int32_t rope_ld, const float* C,
    float eps_lr, const float* gate_logits, float eps, const float* key_norm, void* O,
    hipStream_t stream) {
  rola::Shape s;
  TRY(check_combine(p, Qr, Kr, V, block, sparsity, blk_idx, softmax_scale, Qn, Pq, r, cos_tab,
                    sin_tab, rope_ld, C, eps_lr, gate_logits, eps, key_norm, O, __func__, &s));
  const size_t need = rola_sparse_combine_workspace_bytes(p, block, sparsity, r);
  if (need > rola::static_scratch_bytes())
    return fail(ROLA_ERR_UNSUPPORTED,
                "%s: this problem needs %zu bytes of scratch; the static scratch holds %zu "
                "(use rola_sparse_attn_combine with a workspace)",
                __func__, need, rola::static_scratch_bytes());
  void* ws = nullptr;
  hipError_t e = rola::static_scratch(&ws);
  if (e != hipSuccess) return hip_status(e, __func__);
  const int keep = rola_keep_blocks(rola::num_blocks(s.N, block), sparsity);
  return run_combine(s, Qr, Kr, V, block, keep, blk_idx, softmax_scale, Qn, Pq, r, cos_tab, sin_tab,
                     rope_ld, C, eps_lr, gate_logits, eps, key_norm, O, ws, false, stream, __func__);
}

rola_status rola_lowrank_summary_ex(const rola_problem* p, const void* Kn, const void* V,
                                    const void* Pk, int32_t r, const float* cos_tab,
                                    const float* sin_tab, int32_t rope_ld, int32_t phi,
                                    int32_t rope_order, float* C, float* z, void* ws,
                                    size_t ws_bytes, hipStream_t stream) {
  rola::Shape s;
  int feat = 0;
  TRY(check_problem(p, __func__, &s));
  TRY(check_rank(s, r, __func__));
  TRY(check_feature(phi, rope_order, __func__, &feat));
  REQUIRE_PTR(Kn);
  REQUIRE_PTR(V);
  REQUIRE_PTR(Pk);
  REQUIRE_PTR(C);
  REQUIRE_PTR(ws);
  if (z != nullptr && !aligned(z))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: z not 16-byte aligned", __func__);
  TRY(check_tables(cos_tab, sin_tab, rope_ld, r / 2, __func__));
  const size_t need = rola::summary_workspace_bytes(s, r);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  return hip_status(rola::launch_lowrank_summary(s, Kn, V, Pk, r, cos_tab, sin_tab, rope_ld, feat,
                                                 C, z, ws, stream), __func__);
}

rola_status rola_lowrank_summary(const rola_problem* p, const void* Kn, const void* V,
                                 const void* Pk, int32_t r, const float* cos_tab,
                                 const float* sin_tab, int32_t rope_ld, float* C, float* z,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  return rola_lowrank_summary_ex(p, Kn, V, Pk, r, cos_tab, sin_tab, rope_ld, ROLA_PHI_SILU,
                                 ROLA_ROPE_OUTSIDE, C, z, ws, ws_bytes, stream);
}

rola_status rola_lowrank_readout_ex(const rola_problem* p, const void* Qn, const void* Pq, int32_t r,
                                    const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                    int32_t phi, int32_t rope_order, const float* C, float eps_lr,
                                    void* Olr, hipStream_t stream) {
  rola::Shape s;
  int feat = 0;
  TRY(check_problem(p, __func__, &s));
  TRY(check_rank(s, r, __func__));
  TRY(check_feature(phi, rope_order, __func__, &feat));
  REQUIRE_PTR(Qn);
  REQUIRE_PTR(Pq);
  REQUIRE_PTR(C);
  REQUIRE_PTR(Olr);
  TRY(check_out(s, Olr, {{Qn, "Qn"}}, nullptr, __func__));
  TRY(check_tables(cos_tab, sin_tab, rope_ld, r / 2, __func__));
  if (!(eps_lr >= 0.f) || !isfinite(eps_lr))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: eps_lr must be finite and >= 0", __func__);
  return hip_status(rola::launch_lowrank_readout(s, Qn, Pq, r, cos_tab, sin_tab, rope_ld, feat, C,
                                                 eps_lr, nullptr, nullptr, 0.f, Olr, stream),
                    __func__);
}

rola_status rola_lowrank_readout(const rola_problem* p, const void* Qn, const void* Pq, int32_t r,
                                 const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                 const float* C, float eps_lr, void* Olr, hipStream_t stream) {
  return rola_lowrank_readout_ex(p, Qn, Pq, r, cos_tab, sin_tab, rope_ld, ROLA_PHI_SILU,
                                 ROLA_ROPE_OUTSIDE, C, eps_lr, Olr, stream);
}

rola_status rola_lowrank_features(const rola_problem* p, const void* X, const void* P, int32_t r,
                                  const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                  int32_t phi, int32_t rope_order, float* F, hipStream_t stream) {
  rola::Shape s;
  int feat = 0;
  TRY(check_problem(p, __func__, &s));
  TRY(check_rank(s, r, __func__));
  TRY(check_feature(phi, rope_order, __func__, &feat));
  REQUIRE_PTR(X);
  REQUIRE_PTR(P);
  REQUIRE_PTR(F);
  TRY(check_tables(cos_tab, sin_tab, rope_ld, r / 2, __func__));
  return hip_status(rola::launch_lowrank_features(s, X, P, r, cos_tab, sin_tab, rope_ld, feat, F,
                                                  stream), __func__);
}

rola_status rola_gate_logits(const rola_problem* p, const void* X, int32_t d_model, const void* Wg,
                             float bg, float* logits, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  REQUIRE_PTR(X);
  REQUIRE_PTR(Wg);
  REQUIRE_PTR(logits);
  if (d_model <= 0 || (d_model % 8) != 0)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: d_model=%d must be a positive multiple of 8", __func__,
                (int)d_model);
  if (d_model > rola::gate_max_model())
    return fail(ROLA_ERR_UNSUPPORTED, "%s: d_model=%d above %d", __func__, (int)d_model,
                rola::gate_max_model());
  if (!isfinite(bg)) return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: b_g must be finite", __func__);
  return hip_status(rola::launch_gate_logits(s, X, d_model, Wg, bg, logits, stream), __func__);
}

size_t rola_gate_backward_workspace_bytes(const rola_problem* p, int32_t d_model) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || d_model <= 0 || (d_model % 8) != 0 ||
      d_model > rola::gate_max_model())
    return 0;
  return rola::gate_backward_workspace_bytes(d_model);
}

rola_status rola_gate_logits_backward(const rola_problem* p, const void* X, int32_t d_model,
                                      const void* Wg, const float* dlogits, float* dX, float* dWg,
                                      float* dbg, void* ws, size_t ws_bytes, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  REQUIRE_PTR(X);
  REQUIRE_PTR(Wg);
  REQUIRE_PTR(dlogits);
  REQUIRE_PTR(dWg);
  REQUIRE_PTR(dbg);
  REQUIRE_PTR(ws);
  if (dX != nullptr && !aligned(dX))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: dX not 16-byte aligned", __func__);
  if (d_model <= 0 || (d_model % 8) != 0)
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: d_model=%d must be a positive multiple of 8", __func__,
                (int)d_model);
  if (d_model > rola::gate_max_model())
    return fail(ROLA_ERR_UNSUPPORTED, "%s: d_model=%d above %d", __func__, (int)d_model,
                rola::gate_max_model());
  const size_t need = rola::gate_backward_workspace_bytes(d_model);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  return hip_status(rola::launch_gate_backward(s, X, d_model, Wg, dlogits, dX, dWg, dbg, ws, stream),
                    __func__);
}

size_t rola_lowrank_backward_workspace_bytes(const rola_problem* p, int32_t r) {
  rola::Shape s;
  if (check_problem(p, __func__, &s) != ROLA_OK || check_rank(s, r, __func__) != ROLA_OK) return 0;
  return rola::lowrank_backward_workspace_bytes(s, r);
}

rola_status rola_lowrank_backward(const rola_problem* p, const void* Qn, const void* Kn,
                                  const void* V, const void* Pq, const void* Pk, int32_t r,
                                  const float* cos_tab, const float* sin_tab, int32_t rope_ld,
                                  const float* C, const void* Os, const float* gate_logits,
                                  float eps_lr, float eps, const void* dO, void* dOs, float* dQn,
                                  float* dKn, float* dV, float* dPq, float* dPk, float* dlogits,
                                  void* ws, size_t ws_bytes, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  TRY(check_rank(s, r, __func__));
  if (!s.bf16 || r > 64)
    return fail(ROLA_ERR_UNSUPPORTED, "%s: built for the bf16 path with r <= 64", __func__);
  const void* ptrs[] = {Qn, Kn, V, Pq, Pk, C, Os, gate_logits, dO, dOs, dQn, dKn, dV, dPq, dPk,
                        dlogits, ws};
  for (const void* q : ptrs)
    if (!aligned(q)) return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: a pointer is null or not 16-byte aligned", __func__);
  TRY(check_tables(cos_tab, sin_tab, rope_ld, r / 2, __func__));
  if (!(eps_lr >= 0.f) || !isfinite(eps_lr) || !(eps >= 0.f) || !isfinite(eps))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: eps values must be finite and >= 0", __func__);
  const size_t need = rola::lowrank_backward_workspace_bytes(s, r);
  if (ws_bytes < need)
    return fail(ROLA_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", __func__, ws_bytes, need);
  return hip_status(rola::launch_lowrank_backward(s, Qn, Kn, V, Pq, Pk, r, cos_tab, sin_tab, rope_ld,
                                                  C, Os, gate_logits, eps_lr, eps, dO, dOs, dQn,
                                                  dKn, dV, dPq, dPk, dlogits, ws, stream),
                    __func__);
}

rola_status rola_combine(const rola_problem* p, const void* Os, const void* Olr,
                         const float* gate_logits, float eps, void* O, hipStream_t stream) {
  rola::Shape s;
  TRY(check_problem(p, __func__, &s));
  REQUIRE_PTR(Os);
  REQUIRE_PTR(Olr);
  REQUIRE_PTR(gate_logits);
  REQUIRE_PTR(O);
  TRY(check_out(s, O, {{Os, "Os"}, {Olr, "Olr"}}, Os, __func__));
  if (!(eps >= 0.f) || !isfinite(eps))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: eps must be finite and >= 0", __func__);
  return hip_status(rola::launch_combine(s, Os, Olr, gate_logits, eps, O, stream), __func__);
}

rola_status rola_lowrank_readout_combine_ex(const rola_problem* p, const void* Qn, const void* Pq,
                                            int32_t r, const float* cos_tab, const float* sin_tab,
                                            int32_t rope_ld, int32_t phi, int32_t rope_order,
                                            const float* C, float eps_lr, const void* Os,
                                            const float* gate_logits, float eps, void* O,
                                            hipStream_t stream) {
  rola::Shape s;
  int feat = 0;
  TRY(check_problem(p, __func__, &s));
  TRY(check_rank(s, r, __func__));
  TRY(check_feature(phi, rope_order, __func__, &feat));
  REQUIRE_PTR(Qn);
  REQUIRE_PTR(Pq);
  REQUIRE_PTR(C);
  REQUIRE_PTR(Os);
  REQUIRE_PTR(gate_logits);
  REQUIRE_PTR(O);
  TRY(check_out(s, O, {{Qn, "Qn"}, {Os, "Os"}}, Os, __func__));
  TRY(check_tables(cos_tab, sin_tab, rope_ld, r / 2, __func__));
  if (!(eps_lr >= 0.f) || !isfinite(eps_lr) || !(eps >= 0.f) || !isfinite(eps))
    return fail(ROLA_ERR_INVALID_ARGUMENT, "%s: eps values must be finite and >= 0", __func__);
  return hip_status(rola::launch_lowrank_readout(s, Qn, Pq, r, cos_tab, sin_tab, rope_ld, feat, C,
                                                 eps_lr, Os, gate_logits, eps, O, stream),
                    __func__);
}

rola_status rola_lowrank_readout_combine(const rola_problem* p, const void* Qn, const void* Pq,
                                         int32_t r, const float* cos_tab, const float* sin_tab,
                                         int32_t rope_ld, const float* C, float eps_lr,
                                         const void* Os, const float* gate_logits, float eps,
                                         void* O, hipStream_t stream) {
  return rola_lowrank_readout_combine_ex(p, Qn, Pq, r, cos_tab, sin_tab, rope_ld, ROLA_PHI_SILU,
                                         ROLA_ROPE_OUTSIDE, C, eps_lr, Os, gate_logits, eps, O,
                                         stream);
}

}  // extern "C"
