// Backward of the rotary low-rank branch and the gated fusion (fine-tuning, Sec. 4.5; eq. qklr,
// eq. ctx, eq. gate; Algorithm steps 5-10). With u = q~^T C, rho = sqrt(mean u^2 + eps_lr),
// r_s = sqrt(mean (O^s)^2 + eps), g = sigmoid(logit), a = g r_s / rho and O = O^s + a u:
//   t = dO . u
//   dO^s = dO + (g t / rho) O^s / (d r_s)                    (through r_s)
//   dlogit = (r_s t / rho) g (1 - g)                          (summed over heads: one gate per token)
//   du = a dO - (a t / (d rho^2)) u                           (through the RMSNorm)
//   dq~ = C du,  dC = sum_p q~_p du_p^T,  dphi = R_r^T dq~,  dy = dphi * SiLU'(y),  y = P_q q^n
//   dq^n = P_q^T dy,  dP_q = sum_p dy_p q^n_p^T
// and on the key side, with C = sum_k k~_k v_k^T:
//   dk~ = dC v,  dv = dC^T k~,  dpsi = R_r^T dk~,  dy = dpsi * SiLU'(y),  dk^n = P_k^T dy,
//   dP_k = sum_k dy_k k^n_k^T.
// One workgroup per (b, h, chunk of tokens), four waves each on its own token: the per-token vectors
// use one lane per rotary coordinate (r <= 64) or channels l and l + 64; the outer products dC,
// dP_q, dP_k accumulate per thread over the chunk and are summed over chunks (and batch) in a fixed
// order afterwards, so every gradient is reproducible. fp32 arithmetic, bf16 inputs.
#include "common.h"
#include "launch.h"

namespace rola {
namespace {

constexpr int kD = 128, kMaxR = 64, kWaves = 4;
constexpr int kLd = kD + 1;  // LDS row pitch of P and C (floats): lane-strided row reads hit distinct banks
constexpr int kOuterPer = kMaxR * kD / 256;  // outer-product elements per thread (r <= 64)

__device__ __forceinline__ float wsum(float x) {  // sum over the 64 lanes
  x = rows_sum(x);
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ float silu_grad(float y) {  // d/dy y sigmoid(y)
  const float s = sigmoid(y);
  return s * (1.f + y * (1.f - s));
}

// Per-token work shared by both sides: y = P x (lane k < r), then the features x~ = R_r SiLU(y) of
// the lane's coordinate (pairs (2j, 2j+1) sit in lanes 2j, 2j+1).
struct Feat {
  float y, f;  // pre-activation and feature of this lane's coordinate (0 for lanes >= r)
};
__device__ __forceinline__ Feat features(const float* xs, const float* Ps, int r, int lane,
                                         float c, float s) {
  float y = 0.f;
  if (lane < r)
    for (int k = 0; k < kD; ++k) y = fmaf(Ps[lane * kLd + k], xs[k], y);
  const float a = silu(y);
  const float b = __shfl_xor(a, 1);  // the pair partner's activation
  const float f = (lane & 1) ? b * s + a * c : a * c - b * s;
  return {y, lane < r ? f : 0.f};
}

// R_r^T applied to a gradient of the features, then the SiLU derivative: dy of this lane.
__device__ __forceinline__ float feature_grad(float df, float y, int r, int lane, float c, float s) {
  const float p = __shfl_xor(df, 1);
  const float dphi = (lane & 1) ? p * (-s) + df * c : df * c + p * s;
  return lane < r ? dphi * silu_grad(y) : 0.f;
}

// Query side: dO^s, dlogit per head, dq^n (fp32) and the partial sums of dC and dP_q per chunk.
__global__ __launch_bounds__(256) void lr_bwd_q_kernel(
    int N, int H, int r, int chunk_len, int n_chunks, int ld, const bf16* __restrict__ Qn,
    const bf16* __restrict__ Pq, const float* __restrict__ cos_tab,
    const float* __restrict__ sin_tab, const float* __restrict__ C, const bf16* __restrict__ Os,
    const float* __restrict__ logits, float eps_lr, float eps, const bf16* __restrict__ dO,
    bf16* __restrict__ dOs, float* __restrict__ dQn, float* __restrict__ dlog_h,
    float* __restrict__ part_dC, float* __restrict__ part_dPq) {
  __shared__ float Cs[kMaxR * kLd], Ps[kMaxR * kLd];
  __shared__ float xq[kWaves][kD], vt[kWaves][kD];     // q^n and du of each wave's token
  __shared__ float ft[kWaves][kMaxR], dyt[kWaves][kMaxR];  // q~ and dy of each wave's token
  const long head = blockIdx.x / n_chunks;
  const int chunk = blockIdx.x % n_chunks, h = (int)(head % H);
  const long b = head / H;
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  for (int e = tid; e < r * kD; e += 256) {
    Cs[(e / kD) * kLd + e % kD] = C[head * r * kD + e];
    Ps[(e / kD) * kLd + e % kD] = to_f32(Pq[(long)h * r * kD + e]);
  }
  float accC[kOuterPer], accP[kOuterPer];
#pragma unroll
  for (int i = 0; i < kOuterPer; ++i) accC[i] = accP[i] = 0.f;
  const int t0 = chunk * chunk_len, t1 = min(N, t0 + chunk_len);
  for (int base = t0; base < t1; base += kWaves) {
    const int tok = base + wave;
    const bool valid = tok < t1;  // wave-uniform
    __syncthreads();  // the previous step's vectors are consumed
    if (valid) {
      const long row = (head * N + tok) * kD;
      float2 qv, ov, dv;
      qv = make_float2(to_f32(Qn[row + lane]), to_f32(Qn[row + lane + 64]));
      ov = make_float2(to_f32(Os[row + lane]), to_f32(Os[row + lane + 64]));
      dv = make_float2(to_f32(dO[row + lane]), to_f32(dO[row + lane + 64]));
      xq[wave][lane] = qv.x;
      xq[wave][lane + 64] = qv.y;
      const int j = lane / 2;
      const float c = lane < r ? cos_tab[(long)tok * ld + j] : 1.f;
      const float s = lane < r ? sin_tab[(long)tok * ld + j] : 0.f;
      __builtin_amdgcn_wave_barrier();
      const Feat fq = features(xq[wave], Ps, r, lane, c, s);
      ft[wave][lane] = lane < kMaxR ? fq.f : 0.f;
      __builtin_amdgcn_wave_barrier();
      // u = q~^T C for the lane's two channels
      float u0 = 0.f, u1 = 0.f;
      for (int k = 0; k < r; ++k) {
        const float fk = ft[wave][k];
        u0 = fmaf(fk, Cs[k * kLd + lane], u0);
        u1 = fmaf(fk, Cs[k * kLd + lane + 64], u1);
      }
      const float su = wsum(u0 * u0 + u1 * u1), so = wsum(ov.x * ov.x + ov.y * ov.y);
      const float t = wsum(dv.x * u0 + dv.y * u1);
      const float rho = sqrtf(su * (1.f / kD) + eps_lr), rs = sqrtf(so * (1.f / kD) + eps);
      const float g = sigmoid(logits[b * N + tok]);
      const float a = g * rs / rho;
      const float kos = g * t / (rho * kD * rs);
      dOs[row + lane] = (bf16)fmaf(kos, ov.x, dv.x);
      dOs[row + lane + 64] = (bf16)fmaf(kos, ov.y, dv.y);
      if (lane == 0) dlog_h[head * N + tok] = rs * t / rho * g * (1.f - g);
      const float kdu = a * t / (kD * rho * rho);
      const float du0 = a * dv.x - kdu * u0, du1 = a * dv.y - kdu * u1;
      vt[wave][lane] = du0;
      vt[wave][lane + 64] = du1;
      __builtin_amdgcn_wave_barrier();
      // dq~ = C du (lane k < r), then dy
      float dq = 0.f;
      if (lane < r)
        for (int cc = 0; cc < kD; ++cc) dq = fmaf(Cs[lane * kLd + cc], vt[wave][cc], dq);
      const float dy = feature_grad(dq, fq.y, r, lane, c, s);
      dyt[wave][lane] = dy;
      __builtin_amdgcn_wave_barrier();
      // dq^n = P_q^T dy for the lane's two channels
      float d0 = 0.f, d1 = 0.f;
      for (int k = 0; k < r; ++k) {
        const float dk = dyt[wave][k];
        d0 = fmaf(Ps[k * kLd + lane], dk, d0);
        d1 = fmaf(Ps[k * kLd + lane + 64], dk, d1);
      }
      dQn[row + lane] = d0;
      dQn[row + lane + 64] = d1;
    } else {
      for (int e = lane; e < kD; e += 64) xq[wave][e] = vt[wave][e] = 0.f;
      ft[wave][lane] = dyt[wave][lane] = 0.f;
    }
    __syncthreads();
    // outer products of the four tokens: thread owns elements e = tid + 256 i of the r x 128 matrix
#pragma unroll
    for (int i = 0; i < kOuterPer; ++i) {
      const int e = tid + 256 * i, k = e / kD, cc = e % kD;
      if (k < r) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
          accC[i] = fmaf(ft[w][k], vt[w][cc], accC[i]);
          accP[i] = fmaf(dyt[w][k], xq[w][cc], accP[i]);
        }
      }
    }
  }
  float* pc = part_dC + (head * n_chunks + chunk) * (long)(r * kD);
  float* pp = part_dPq + (head * n_chunks + chunk) * (long)(r * kD);
#pragma unroll
  for (int i = 0; i < kOuterPer; ++i) {
    const int e = tid + 256 * i;
    if (e < r * kD) {
      pc[e] = accC[i];
      pp[e] = accP[i];
    }
  }
}

// Partials part[(b * H + h) * n_chunks + c][e] summed in a fixed order (batch entries, then chunks):
// per_head = true: out[(b * H + h)][e] over c; per_head = false: out[h][e] over (b, c).
__global__ __launch_bounds__(256) void lr_bwd_reduce_kernel(int re, int B, int H, int n_chunks,
                                                            bool per_head,
                                                            const float* __restrict__ part,
                                                            float* __restrict__ out) {
  const long o = blockIdx.y;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= re) return;
  float s = 0.f;
  if (per_head) {
    const float* src = part + o * n_chunks * (long)re + e;
    for (int c = 0; c < n_chunks; ++c) s += src[(long)c * re];
  } else {
    for (int b = 0; b < B; ++b) {
      const float* src = part + ((long)b * H + o) * n_chunks * (long)re + e;
      for (int c = 0; c < n_chunks; ++c) s += src[(long)c * re];
    }
  }
  out[o * re + e] = s;
}

// Key side: dk^n, dv (fp32) and the partial sums of dP_k per chunk, from the reduced dC.
__global__ __launch_bounds__(256) void lr_bwd_k_kernel(
    int N, int H, int r, int chunk_len, int n_chunks, int ld, const bf16* __restrict__ Kn,
    const bf16* __restrict__ V, const bf16* __restrict__ Pk, const float* __restrict__ cos_tab,
    const float* __restrict__ sin_tab, const float* __restrict__ dC, float* __restrict__ dKn,
    float* __restrict__ dV, float* __restrict__ part_dPk) {
  __shared__ float Gs[kMaxR * kLd], Ps[kMaxR * kLd];
  __shared__ float xk[kWaves][kD], vv[kWaves][kD];
  __shared__ float ft[kWaves][kMaxR], dyt[kWaves][kMaxR];
  const long head = blockIdx.x / n_chunks;
  const int chunk = blockIdx.x % n_chunks, h = (int)(head % H);
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  for (int e = tid; e < r * kD; e += 256) {
    Gs[(e / kD) * kLd + e % kD] = dC[head * r * kD + e];
    Ps[(e / kD) * kLd + e % kD] = to_f32(Pk[(long)h * r * kD + e]);
  }
  float accP[kOuterPer];
#pragma unroll
  for (int i = 0; i < kOuterPer; ++i) accP[i] = 0.f;
  const int t0 = chunk * chunk_len, t1 = min(N, t0 + chunk_len);
  for (int base = t0; base < t1; base += kWaves) {
    const int tok = base + wave;
    const bool valid = tok < t1;
    __syncthreads();
    if (valid) {
      const long row = (head * N + tok) * kD;
      xk[wave][lane] = to_f32(Kn[row + lane]);
      xk[wave][lane + 64] = to_f32(Kn[row + lane + 64]);
      const float v0 = to_f32(V[row + lane]), v1 = to_f32(V[row + lane + 64]);
      vv[wave][lane] = v0;
      vv[wave][lane + 64] = v1;
      const int j = lane / 2;
      const float c = lane < r ? cos_tab[(long)tok * ld + j] : 1.f;
      const float s = lane < r ? sin_tab[(long)tok * ld + j] : 0.f;
      __builtin_amdgcn_wave_barrier();
      const Feat fk = features(xk[wave], Ps, r, lane, c, s);
      ft[wave][lane] = fk.f;
      __builtin_amdgcn_wave_barrier();
      // dk~ = dC v (lane k < r); dv = dC^T k~ (two channels per lane)
      float dk = 0.f;
      if (lane < r)
        for (int cc = 0; cc < kD; ++cc) dk = fmaf(Gs[lane * kLd + cc], vv[wave][cc], dk);
      float w0 = 0.f, w1 = 0.f;
      for (int k = 0; k < r; ++k) {
        const float fkk = ft[wave][k];
        w0 = fmaf(Gs[k * kLd + lane], fkk, w0);
        w1 = fmaf(Gs[k * kLd + lane + 64], fkk, w1);
      }
      dV[row + lane] = w0;
      dV[row + lane + 64] = w1;
      const float dy = feature_grad(dk, fk.y, r, lane, c, s);
      dyt[wave][lane] = dy;
      __builtin_amdgcn_wave_barrier();
      float d0 = 0.f, d1 = 0.f;
      for (int k = 0; k < r; ++k) {
        const float dyk = dyt[wave][k];
        d0 = fmaf(Ps[k * kLd + lane], dyk, d0);
        d1 = fmaf(Ps[k * kLd + lane + 64], dyk, d1);
      }
      dKn[row + lane] = d0;
      dKn[row + lane + 64] = d1;
    } else {
      for (int e = lane; e < kD; e += 64) xk[wave][e] = 0.f;
      dyt[wave][lane] = 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kOuterPer; ++i) {
      const int e = tid + 256 * i, k = e / kD, cc = e % kD;
      if (k < r) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) accP[i] = fmaf(dyt[w][k], xk[w][cc], accP[i]);
      }
    }
  }
  float* pp = part_dPk + (head * n_chunks + chunk) * (long)(r * kD);
#pragma unroll
  for (int i = 0; i < kOuterPer; ++i) {
    const int e = tid + 256 * i;
    if (e < r * kD) pp[e] = accP[i];
  }
}

// dlogit[b, n] = sum over heads of the per-head contributions, in head order.
__global__ __launch_bounds__(256) void lr_bwd_logit_kernel(long BN, int N, int H,
                                                           const float* __restrict__ dlog_h,
                                                           float* __restrict__ dlogits) {
  const long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= BN) return;
  const long b = e / N, n = e % N;
  float s = 0.f;
  for (int h = 0; h < H; ++h) s += dlog_h[(b * H + h) * (long)N + n];
  dlogits[e] = s;
}

int lr_bwd_chunk_len(const Shape& s) {
  const long heads = (long)s.B * s.H;
  const long want = (4096 + heads - 1) / heads;  // about 4096 workgroups
  long len = (s.N + want - 1) / want;
  len = (len + kWaves - 1) / kWaves * kWaves;
  return (int)(len < 64 ? 64 : len);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct LrBwdWs {
  size_t part, dlog, dC;
};
LrBwdWs lr_bwd_layout(const Shape& s, int r) {
  const size_t heads = (size_t)s.B * s.H;
  const size_t chunks = (s.N + lr_bwd_chunk_len(s) - 1) / lr_bwd_chunk_len(s);
  return {align256(heads * chunks * r * kD * 4), align256(heads * s.N * 4),
          align256(heads * r * kD * 4)};
}

}  // namespace

size_t lowrank_backward_workspace_bytes(const Shape& s, int r) {
  if (!s.bf16 || s.d != kD || r > kMaxR) return 0;
  const LrBwdWs w = lr_bwd_layout(s, r);
  return 3 * w.part + w.dlog + w.dC;  // partials of dC, dP_q, dP_k; per-head dlogit; dC
}

hipError_t launch_lowrank_backward(const Shape& s, const void* Qn, const void* Kn, const void* V,
                                   const void* Pq, const void* Pk, int r, const float* cos_tab,
                                   const float* sin_tab, int ld, const float* C, const void* Os,
                                   const float* logits, float eps_lr, float eps, const void* dO,
                                   void* dOs, float* dQn, float* dKn, float* dV, float* dPq,
                                   float* dPk, float* dlogits, void* ws, hipStream_t st) {
  const int chunk_len = lr_bwd_chunk_len(s);
  const int n_chunks = (s.N + chunk_len - 1) / chunk_len;
  const long heads = (long)s.B * s.H;
  const LrBwdWs lay = lr_bwd_layout(s, r);
  char* w = (char*)ws;
  float* part_dC = (float*)w;
  float* part_dPq = (float*)(w + lay.part);
  float* part_dPk = (float*)(w + 2 * lay.part);
  float* dlog_h = (float*)(w + 3 * lay.part);
  float* dC = (float*)(w + 3 * lay.part + lay.dlog);
  const int re = r * kD;
  const dim3 rgrid((re + 255) / 256, 1);
  hipLaunchKernelGGL(lr_bwd_q_kernel, dim3((unsigned)(heads * n_chunks)), dim3(256), 0, st, s.N,
                     s.H, r, chunk_len, n_chunks, ld, (const bf16*)Qn, (const bf16*)Pq, cos_tab,
                     sin_tab, C, (const bf16*)Os, logits, eps_lr, eps, (const bf16*)dO, (bf16*)dOs,
                     dQn, dlog_h, part_dC, part_dPq);
  // dC[b, h] = sum over chunks
  hipLaunchKernelGGL(lr_bwd_reduce_kernel, dim3(rgrid.x, (unsigned)heads), dim3(256), 0, st, re, s.B,
                     s.H, n_chunks, true, (const float*)part_dC, dC);
  hipLaunchKernelGGL(lr_bwd_k_kernel, dim3((unsigned)(heads * n_chunks)), dim3(256), 0, st, s.N,
                     s.H, r, chunk_len, n_chunks, ld, (const bf16*)Kn, (const bf16*)V,
                     (const bf16*)Pk, cos_tab, sin_tab, (const float*)dC, dKn, dV, part_dPk);
  // dP_q[h], dP_k[h] = sum over (b, chunk)
  hipLaunchKernelGGL(lr_bwd_reduce_kernel, dim3(rgrid.x, (unsigned)s.H), dim3(256), 0, st, re, s.B,
                     s.H, n_chunks, false, (const float*)part_dPq, dPq);
  hipLaunchKernelGGL(lr_bwd_reduce_kernel, dim3(rgrid.x, (unsigned)s.H), dim3(256), 0, st, re, s.B,
                     s.H, n_chunks, false, (const float*)part_dPk, dPk);
  hipLaunchKernelGGL(lr_bwd_logit_kernel, dim3((unsigned)(((long)s.B * s.N + 255) / 256)),
                     dim3(256), 0, st, (long)s.B * s.N, s.N, s.H, (const float*)dlog_h, dlogits);
  return hipGetLastError();
}

}  // namespace rola
