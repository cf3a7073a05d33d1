// Token gate logits of the gated fusion (Sec. 4.4; Algorithm step 8): logit[b, n] = X[b, n, :] . W_g
// + b_g over the attention block's input hidden states X [B, N, d_model]; the combine applies the
// sigmoid. A GEMV, bound by reading X once from HBM (d_model * elt bytes per token).
//
// One wave per token row (rows strided over the grid's waves), W_g staged once per workgroup in LDS
// as fp32; each lane reads 16-byte pieces of the row (8 bf16 or 4 fp32 values), accumulates in fp32,
// and the row sum is a cross-lane reduction. Two rows are in flight per wave so that each lane keeps
// two independent 16-byte loads outstanding per step.
#include "common.h"
#include "launch.h"

namespace rola {
namespace {

constexpr int kGateMaxModel = 16384;  // W_g in LDS as fp32: 64 KB

// One 16-byte piece of a row as fp32: 8 bf16 or 4 fp32 values.
__device__ __forceinline__ void load_piece(const bf16* p, float v[8]) { load8(p, v); }
__device__ __forceinline__ void load_piece(const float* p, float v[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}

__device__ __forceinline__ float wave_sum(float x) {
  x = rows_sum(x);  // lanes l, l^16, l^32, l^48
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

template <typename T>
__global__ __launch_bounds__(256) void gate_logits_kernel(long rows, int dm, const T* __restrict__ X,
                                                          const T* __restrict__ W, float bias,
                                                          float* __restrict__ logits) {
  extern __shared__ float w[];  // [dm]
  for (int i = threadIdx.x; i < dm; i += 256) w[i] = to_f32(W[i]);
  __syncthreads();
  constexpr int PER = 16 / sizeof(T);  // values per 16-byte piece
  const int lane = threadIdx.x % 64;
  const long wave = (long)blockIdx.x * 4 + threadIdx.x / 64, nwaves = (long)gridDim.x * 4;
  for (long r0 = 2 * wave; r0 < rows; r0 += 2 * nwaves) {
    const bool two = r0 + 1 < rows;
    const T* x0 = X + r0 * dm;
    const T* x1 = X + (two ? r0 + 1 : r0) * dm;
    float s0 = 0.f, s1 = 0.f;
    for (int c = lane * PER; c < dm; c += 64 * PER) {
      float a[8], b[8];
      load_piece(x0 + c, a);
      load_piece(x1 + c, b);
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        s0 = fmaf(a[k], w[c + k], s0);
        s1 = fmaf(b[k], w[c + k], s1);
      }
    }
    s0 = wave_sum(s0);
    s1 = wave_sum(s1);
    if (lane == 0) {
      logits[r0] = s0 + bias;
      if (two) logits[r0 + 1] = s1 + bias;
    }
  }
}

// Backward of the gate logits: dX[row] = dlogit[row] W_g (fp32), and per chunk of rows the partial
// sums of dW_g = sum_row dlogit[row] X[row] and db_g = sum_row dlogit[row] (slot dm of the partial).
template <typename T>
__global__ __launch_bounds__(256) void gate_bwd_kernel(long rows, int dm, long chunk,
                                                       const T* __restrict__ X,
                                                       const T* __restrict__ W,
                                                       const float* __restrict__ dlog,
                                                       float* __restrict__ dX,
                                                       float* __restrict__ part) {
  const long r0 = blockIdx.x * chunk, r1 = min(rows, r0 + chunk);
  for (int c = threadIdx.x; c <= dm; c += 256) {
    const float w = c < dm ? to_f32(W[c]) : 0.f;
    float acc = 0.f;
    for (long r = r0; r < r1; ++r) {
      const float g = dlog[r];
      if (c < dm) {
        acc = fmaf(g, to_f32(X[r * dm + c]), acc);
        if (dX) dX[r * dm + c] = g * w;
      } else {
        acc += g;
      }
    }
    part[blockIdx.x * (long)(dm + 1) + c] = acc;
  }
}

__global__ __launch_bounds__(256) void gate_bwd_reduce_kernel(int n, int dm,
                                                              const float* __restrict__ part,
                                                              float* __restrict__ dW,
                                                              float* __restrict__ db) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c > dm) return;
  float s = 0.f;
  for (int i = 0; i < n; ++i) s += part[(long)i * (dm + 1) + c];  // chunk order: reproducible
  if (c < dm) dW[c] = s;
  else *db = s;
}

constexpr int kGateBwdChunks = 1024;

}  // namespace

size_t gate_backward_workspace_bytes(int d_model) {
  return (size_t)kGateBwdChunks * (d_model + 1) * sizeof(float);
}

hipError_t launch_gate_backward(const Shape& s, const void* X, int d_model, const void* Wg,
                                const float* dlogits, float* dX, float* dWg, float* dbg, void* ws,
                                hipStream_t st) {
  const long rows = (long)s.B * s.N;
  const long chunk = (rows + kGateBwdChunks - 1) / kGateBwdChunks;
  const int n = (int)((rows + chunk - 1) / chunk);
  float* part = (float*)ws;
  if (s.bf16)
    hipLaunchKernelGGL(gate_bwd_kernel<bf16>, dim3(n), dim3(256), 0, st, rows, d_model, chunk,
                       (const bf16*)X, (const bf16*)Wg, dlogits, dX, part);
  else
    hipLaunchKernelGGL(gate_bwd_kernel<float>, dim3(n), dim3(256), 0, st, rows, d_model, chunk,
                       (const float*)X, (const float*)Wg, dlogits, dX, part);
  hipLaunchKernelGGL(gate_bwd_reduce_kernel, dim3((d_model + 1 + 255) / 256), dim3(256), 0, st, n,
                     d_model, (const float*)part, dWg, dbg);
  return hipGetLastError();
}

hipError_t launch_gate_logits(const Shape& s, const void* X, int d_model, const void* Wg, float bg,
                              float* logits, hipStream_t st) {
  const long rows = (long)s.B * s.N;
  const long want = (rows + 7) / 8;  // workgroups of 4 waves, 2 rows per wave per pass
  const dim3 grid((unsigned)(want < 2048 ? want : 2048));
  const size_t lds = (size_t)d_model * sizeof(float);
  if (s.bf16)
    hipLaunchKernelGGL(gate_logits_kernel<bf16>, grid, dim3(256), lds, st, rows, d_model,
                       (const bf16*)X, (const bf16*)Wg, bg, logits);
  else
    hipLaunchKernelGGL(gate_logits_kernel<float>, grid, dim3(256), lds, st, rows, d_model,
                       (const float*)X, (const float*)Wg, bg, logits);
  return hipGetLastError();
}

int gate_max_model() { return kGateMaxModel; }

}  // namespace rola
