// 3D rotary schedule (Sec. 3, 3D RoPE; Sec. 4.2): the backbone's cos/sin tables and the main-path
// rotation Q^r = R(Q^n) (Algorithm step 3). Both are memory-bound elementwise kernels.
#include "common.h"
#include "launch.h"

namespace rola {
namespace {

// One thread per (token, pair). Angles in fp64 so the fp32 tables are correctly rounded values of
// cos/sin of the exact angle.
__global__ void rope_tables_kernel(int N, int HsWs, int Ws, int half, int pt, int py, int dt,
                                   int dy, int dx, double base, int ot, int oy, int ox,
                                   float* __restrict__ cos_tab, float* __restrict__ sin_tab) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)N * half) return;
  const int n = (int)(i / half), j = (int)(i % half);
  const int t = n / HsWs, rem = n % HsWs, y = rem / Ws, x = rem % Ws;
  double pos;
  int loc, width;
  if (j < pt) { pos = t + ot; loc = j; width = dt; }
  else if (j < pt + py) { pos = y + oy; loc = j - pt; width = dy; }
  else { pos = x + ox; loc = j - pt - py; width = dx; }
  const double ang = pos * pow(base, -2.0 * loc / width);
  double s, c;
  sincos(ang, &s, &c);
  cos_tab[i] = (float)c;
  sin_tab[i] = (float)s;
}

// One thread per 4 pairs (8 elements) of one row; rows are [B*H*N] of d elements.
template <typename T>
__global__ void rope_apply_kernel(long rows, int N, int d, int ld, const T* __restrict__ X,
                                  const float* __restrict__ cos_tab,
                                  const float* __restrict__ sin_tab, T* __restrict__ Xr) {
  const int per_row = d / 8;
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * per_row) return;
  const long row = i / per_row;
  const int g = (int)(i % per_row);
  const int n = (int)(row % N);
  float v[8], o[8];
  load8(X + row * d + g * 8, v);
  const float4 c = *reinterpret_cast<const float4*>(cos_tab + (long)n * ld + g * 4);
  const float4 s = *reinterpret_cast<const float4*>(sin_tab + (long)n * ld + g * 4);
  const float cc[4] = {c.x, c.y, c.z, c.w}, ss[4] = {s.x, s.y, s.z, s.w};
#pragma unroll
  for (int p = 0; p < 4; ++p) rope_pair(v[2 * p], v[2 * p + 1], cc[p], ss[p], o[2 * p], o[2 * p + 1]);
  store8(Xr + row * d + g * 8, o);
}

// Backward of the rotation (fp32): dX += R(p)^T dY, pair (a, b) -> (a cos + b sin, b cos - a sin),
// or dX += dY without the rotation. One thread per 4 pairs of one row.
template <bool ROT>
__global__ void rope_grad_kernel(long rows, int N, int d, int ld, const float* __restrict__ dY,
                                 const float* __restrict__ cos_tab,
                                 const float* __restrict__ sin_tab, float* __restrict__ dX) {
  const int per_row = d / 8;
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * per_row) return;
  const long row = i / per_row;
  const int g = (int)(i % per_row);
  float v[8], o[8];
  load8(dY + row * d + g * 8, v);
  load8(dX + row * d + g * 8, o);
  if constexpr (ROT) {
    const int n = (int)(row % N);
    const float4 c = *reinterpret_cast<const float4*>(cos_tab + (long)n * ld + g * 4);
    const float4 sn = *reinterpret_cast<const float4*>(sin_tab + (long)n * ld + g * 4);
    const float cc[4] = {c.x, c.y, c.z, c.w}, ss[4] = {sn.x, sn.y, sn.z, sn.w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      o[2 * p] += v[2 * p] * cc[p] + v[2 * p + 1] * ss[p];
      o[2 * p + 1] += v[2 * p + 1] * cc[p] - v[2 * p] * ss[p];
    }
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] += v[k];
  }
  store8(dX + row * d + g * 8, o);
}

}  // namespace

hipError_t launch_rope_grad(const Shape& s, const float* dY, const float* cos_tab,
                            const float* sin_tab, int ld, bool rotate, float* dX, hipStream_t st) {
  const long rows = (long)s.B * s.H * s.N;
  const long total = rows * (s.d / 8);
  const int threads = 256;
  const dim3 grid((unsigned)((total + threads - 1) / threads));
  if (rotate)
    hipLaunchKernelGGL(rope_grad_kernel<true>, grid, dim3(threads), 0, st, rows, s.N, s.d, ld, dY,
                       cos_tab, sin_tab, dX);
  else
    hipLaunchKernelGGL(rope_grad_kernel<false>, grid, dim3(threads), 0, st, rows, s.N, s.d, ld, dY,
                       cos_tab, sin_tab, dX);
  return hipGetLastError();
}

hipError_t launch_rope_tables(const Shape& s, int dt, int dy, int dx, double base, int ot, int oy,
                              int ox, float* cos_tab, float* sin_tab, hipStream_t st) {
  const int half = s.d / 2;
  const long total = (long)s.N * half;
  const int threads = 256;
  hipLaunchKernelGGL(rope_tables_kernel, dim3((unsigned)((total + threads - 1) / threads)),
                     dim3(threads), 0, st, s.N, s.Hs * s.Ws, s.Ws, half, dt / 2, dy / 2, dt, dy,
                     dx, base, ot, oy, ox, cos_tab, sin_tab);
  return hipGetLastError();
}

hipError_t launch_rope_apply(const Shape& s, const void* X, const float* cos_tab,
                             const float* sin_tab, int ld, void* Xr, hipStream_t st) {
  const long rows = (long)s.B * s.H * s.N;
  const long total = rows * (s.d / 8);
  const int threads = 256;
  const dim3 grid((unsigned)((total + threads - 1) / threads));
  if (s.bf16)
    hipLaunchKernelGGL(rope_apply_kernel<bf16>, grid, dim3(threads), 0, st, rows, s.N, s.d, ld,
                       (const bf16*)X, cos_tab, sin_tab, (bf16*)Xr);
  else
    hipLaunchKernelGGL(rope_apply_kernel<float>, grid, dim3(threads), 0, st, rows, s.N, s.d, ld,
                       (const float*)X, cos_tab, sin_tab, (float*)Xr);
  return hipGetLastError();
}

}  // namespace rola
