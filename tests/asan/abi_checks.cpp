// Host-only driver for an AddressSanitizer build of the C ABI's validation layer (rola_api.cpp):
// every call below is invalid and must be rejected before anything is enqueued, with the expected
// status and a message. Device pointers are fake, aligned addresses that are never dereferenced;
// nothing here touches a GPU. Built and run by tests/test_abi_asan.py.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "rola.h"

static int g_failed = 0, g_run = 0;

static void* fake(int k) { return (void*)((uintptr_t)k << 36); }  // distinct, 64 GiB apart
#define F(k) fake(k)
#define MIS ((void*)((uintptr_t)(1u << 20) + 4))

#define EXPECT(want, call)                                                                   \
  do {                                                                                       \
    ++g_run;                                                                                 \
    const rola_status got = (call);                                                          \
    const char* msg = rola_last_error();                                                     \
    if (got != (want) || msg == NULL || msg[0] == 0) {                                       \
      fprintf(stderr, "line %d: got %s, want %s (%s)\n", __LINE__, rola_status_string(got),  \
              rola_status_string(want), msg ? msg : "(null)");                               \
      ++g_failed;                                                                            \
    }                                                                                        \
  } while (0)

int main(void) {
  const rola_problem ok = {1, 2, 75600, 128, 21, 45, 80, ROLA_DTYPE_BF16};
  const rola_problem badN = {1, 2, 75601, 128, 21, 45, 80, ROLA_DTYPE_BF16};
  const rola_problem d96 = {1, 2, 75600, 96, 21, 45, 80, ROLA_DTYPE_F32};
  const rola_problem f32 = {1, 2, 75600, 128, 21, 45, 80, ROLA_DTYPE_F32};
  const rola_problem huge = {1 << 20, 1 << 20, 75600, 128, 21, 45, 80, ROLA_DTYPE_BF16};
  const rola_problem neg = {1, -2, 75600, 128, 21, 45, 80, ROLA_DTYPE_BF16};
  const rola_problem wide = {1, 2, 75600, 128, 1 << 30, 1 << 30, 1 << 30, ROLA_DTYPE_BF16};
  const size_t BIG = (size_t)1 << 40;
  const float* T = (const float*)F(40);

  // host helpers
  if (rola_num_blocks(75600, 64) != 1182 || rola_num_blocks(0, 64) != -1) ++g_failed;
  if (rola_keep_blocks(1182, 0.9) != 118 || rola_keep_blocks(10, 1.0) != -1) ++g_failed;
  if (rola_select_workspace_bytes(&badN, 64) != 0 || rola_select_workspace_bytes(NULL, 64) != 0)
    ++g_failed;
  if (rola_summary_workspace_bytes(&ok, 33) != 0) ++g_failed;
  if (rola_sparse_workspace_bytes(&huge, 64, 0.9) != 0) ++g_failed;
  g_run += 5;

  // problem descriptors
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_block_select(NULL, F(1), F(2), 64, 0.9, (int32_t*)F(3), F(4), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_block_select(&badN, F(1), F(2), 64, 0.9, (int32_t*)F(3), F(4), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_block_select(&neg, F(1), F(2), 64, 0.9, (int32_t*)F(3), F(4), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_block_select(&wide, F(1), F(2), 64, 0.9, (int32_t*)F(3), F(4), BIG, 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_block_select(&huge, F(1), F(2), 64, 0.9, (int32_t*)F(3), F(4), BIG, 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_block_select(&d96, F(1), F(2), 64, 0.9, (int32_t*)F(3), F(4), BIG, 0));
  EXPECT(ROLA_ERR_WORKSPACE, rola_block_select(&ok, F(1), F(2), 64, 0.9, (int32_t*)F(3), F(4), 16, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_block_select(&ok, MIS, F(2), 64, 0.9, (int32_t*)F(3), F(4), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_block_select(&ok, F(1), F(2), 64, NAN, (int32_t*)F(3), F(4), BIG, 0));

  // sparse attention
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn(&ok, NULL, F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), NULL, 0, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn(&ok, F(1), F(2), F(3), 64, 1.0, (int32_t*)F(4), 0.1f, F(5), NULL, 0, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), -1.f, F(5), NULL, 0, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), INFINITY, F(5), NULL, 0, 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_sparse_attn(&ok, F(1), F(2), F(3), 32, 0.9, (int32_t*)F(4), 0.1f, F(5), NULL, 0, 0));
  EXPECT(ROLA_ERR_WORKSPACE, rola_sparse_attn(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), F(6), 64, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(2), NULL, 0, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn_lse(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), NULL, NULL, 0, 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_sparse_attn_lse(&f32, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), (float*)F(6), NULL, 0, 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_dense_attn(&ok, F(1), F(2), F(3), 96, 0.1f, F(4), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_dense_attn(&ok, F(1), F(2), F(3), 64, 0.1f, F(1), 0));
  EXPECT(ROLA_ERR_WORKSPACE, rola_sparse_attn_backward(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), (float*)F(6), F(7), (float*)F(8), (float*)F(9), (float*)F(10), F(11), 16, 0));

  // attention + readout + combine
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn_combine(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), F(6), 31, T, T, 64, (float*)F(7), 1e-6f, (float*)F(8), 1e-6f, NULL, F(9), F(10), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn_combine(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), F(6), 32, T, T, 64, (float*)F(7), 1e-6f, (float*)F(8), 1e-6f, NULL, F(5), F(10), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_sparse_attn_combine(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), F(6), 32, T, T, 64, (float*)F(7), -1.f, (float*)F(8), 1e-6f, NULL, F(9), F(10), BIG, 0));
  EXPECT(ROLA_ERR_WORKSPACE, rola_sparse_attn_combine(&ok, F(1), F(2), F(3), 64, 0.9, (int32_t*)F(4), 0.1f, F(5), F(6), 32, T, T, 64, (float*)F(7), 1e-6f, (float*)F(8), 1e-6f, NULL, F(9), F(10), 64, 0));

  // low-rank branch and the combine
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_lowrank_summary(&ok, F(1), F(2), F(3), 31, T, T, 64, (float*)F(4), NULL, F(5), BIG, 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_lowrank_summary(&ok, F(1), F(2), F(3), 48, T, T, 64, (float*)F(4), NULL, F(5), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_lowrank_summary(&ok, F(1), F(2), F(3), 32, T, T, 6, (float*)F(4), NULL, F(5), BIG, 0));
  EXPECT(ROLA_ERR_WORKSPACE, rola_lowrank_summary(&ok, F(1), F(2), F(3), 32, T, T, 64, (float*)F(4), NULL, F(5), 64, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_lowrank_summary_ex(&ok, F(1), F(2), F(3), 32, T, T, 64, 9, 0, (float*)F(4), NULL, F(5), BIG, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_lowrank_readout(&ok, F(1), F(2), 32, T, T, 64, (float*)F(3), -1.f, F(4), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_lowrank_readout(&ok, F(1), F(2), 32, T, T, 64, (float*)F(3), 1e-6f, F(1), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_lowrank_readout_combine(&ok, F(1), F(2), 32, T, T, 64, (float*)F(3), 1e-6f, F(4), (float*)F(5), 1e-6f, F(1), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_combine(&ok, F(1), F(2), (float*)F(3), 1e-6f, F(2), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_combine(&ok, F(1), F(2), (float*)F(3), 1e-6f, (char*)F(1) + 4096, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_combine(&ok, F(1), F(2), (float*)F(3), NAN, F(4), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_lowrank_features(&ok, F(1), F(2), 32, T, T, 64, 0, 3, (float*)F(3), 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_lowrank_backward(&ok, F(1), F(2), F(3), F(4), F(5), 128, T, T, 64, (float*)F(6), F(7), (float*)F(8), 1e-6f, 1e-6f, F(9), F(10), (float*)F(11), (float*)F(12), (float*)F(13), (float*)F(14), (float*)F(15), (float*)F(16), F(17), BIG, 0));

  // rotary schedule, gate
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_rope_tables(&ok, 44, 42, 40, 10000.0, 0, 0, 0, (float*)F(1), (float*)F(2), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_rope_tables(&ok, 44, 42, 42, 1.0, 0, 0, 0, (float*)F(1), (float*)F(2), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_rope_apply(&ok, F(1), T, T, 60, F(2), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_rope_apply(&ok, F(1), T, T, 64, (char*)F(1) + 256, 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_rope_backward_accumulate(&f32, (float*)F(1), T, T, 64, 1, (float*)F(1), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_gate_logits(&ok, F(1), 5124, F(2), -1.9f, (float*)F(3), 0));
  EXPECT(ROLA_ERR_UNSUPPORTED, rola_gate_logits(&ok, F(1), 16392, F(2), -1.9f, (float*)F(3), 0));
  EXPECT(ROLA_ERR_INVALID_ARGUMENT, rola_gate_logits(&ok, F(1), 5120, F(2), INFINITY, (float*)F(3), 0));
  EXPECT(ROLA_ERR_WORKSPACE, rola_gate_logits_backward(&ok, F(1), 5120, F(2), (float*)F(3), NULL, (float*)F(4), (float*)F(5), F(6), 4, 0));

  // a very long message is truncated into the per-thread buffer, not written past it
  if (strlen(rola_last_error()) >= 512) ++g_failed;
  ++g_run;

  printf("%d checks, %d failed\n", g_run, g_failed);
  return g_failed ? 1 : 0;
}
