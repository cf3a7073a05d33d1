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

// ---- MFMA path (r <= 32) ---------------------------------------------------------------------
// One workgroup per (b, h, chunk of tokens); per step each of its four waves takes a 16-token tile
// (lane = token l%16, group g = l/16) through v_mfma_f32_16x16x32_bf16, in the layouts of the
// forward readout, where every product's output lands in the register layout the next one reads:
//   Y^T  = P X^T        A = even / odd rows of P (registers): rows = pairs 4g+v of lane (g, token)
//   f    = R_r SiLU(Y)  in registers, split into bf16 hi + lo
//   F^T  = M^T f^T      A = M^T fragments (LDS, hi + lo): query side u (M = C), key side dV (M = dC);
//                       lane (g, token) gets channels 32p + 8g .. +7 in F[2p], F[2p+1]
//   query side: RMSNorm and gate backward per token (in-lane sums + one four-lane reduction), du
//   G^T  = M vec^T      A = rows of M (LDS, hi + lo), B = du (hi + lo) or V: dq~ / dk~ per pair
//   dy   = SiLU'(Y) R_r^T G   in registers
//   dX^T = P^T dy^T     A = P^T fragments (LDS), B = dy (hi + lo): dQ^n / dK^n
// The outer products dC = sum f du^T and dP = sum dy x^T contract over tokens: the four waves write
// their tiles (token-major) to LDS and every wave contracts the step's 64 tokens for its own 32
// channels, reading the operands with ds_read_b64_tr_b16 (token-major rows -> one lane per column).
// fp32 operands enter as bf16 hi + lo pairs (three products, or two against exact bf16 data), which
// keeps them to about 2^-16 relative. Partials per chunk as in the plain kernels.
constexpr int kStep = 64;  // tokens per workgroup step
constexpr int kRp = 48;    // LDS row pitch (bf16) of coordinate tiles: conflict-free transposing reads
constexpr int kCp = 144;   // LDS row pitch (bf16) of channel tiles

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Channel held in row c of channel-fragment w (output lane (g, token) of fragments 2p and 2p + 1
// then holds the consecutive channels 32p + 8g .. +7).
__device__ __forceinline__ int frag_chan(int w, int c) {
  return 32 * (w >> 1) + 8 * (c >> 2) + 4 * (w & 1) + (c & 3);
}

// bf16 hi + lo parts of eight floats.
__device__ __forceinline__ void split8(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    hi[i] = (bf16)x[i];
    lo[i] = (bf16)(x[i] - (float)hi[i]);
  }
}

// Operand of a 16x16x32 MFMA that contracts over the rows of a row-major LDS tile: lane l gets
// column col0 + l%16 of rows row0 .. row0 + 7, row0 given per 16-lane group.
__device__ __forceinline__ bf16x8 tr_rows8(const bf16* tile, int pitch, int row0, int col0, int lane) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int i16 = lane % 16;
  const bf16* p = tile + (row0 + (i16 >> 2)) * pitch + col0 + 4 * (i16 & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 4 * pitch));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Pair-major (e0..e3, o0..o3) to coordinate order (e0, o0, e1, o1, ...).
__device__ __forceinline__ bf16x8 interleave(const bf16x8& x) {
  return __builtin_shufflevector(x, x, 0, 4, 1, 5, 2, 6, 3, 7);
}

struct LrBwdArgs {
  int N, H, r, chunk_len, n_chunks, ld;
  const bf16* X;        // Q^n (query side) or K^n (key side), [B, H, N, 128]
  const bf16* P;        // P_q or P_k, [H, r, 128]
  const float* cos_tab;
  const float* sin_tab;
  const float* M;       // C (query side) or dC (key side), [B, H, r, 128]
  const bf16* Os;       // query side: O^s
  const float* logits;  // query side: gate logits [B, N]
  float eps_lr, eps;
  const bf16* Y;        // query side: dO; key side: V
  bf16* dOs;            // query side
  float* dX;            // dQ^n or dK^n
  float* dV;            // key side
  float* dlog_h;        // query side: per-head gate-logit gradient [B, H, N]
  float* part_dM;       // query side: partial dC per chunk
  float* part_dP;       // partial dP_q or dP_k per chunk
};

template <bool KEY>
__global__ __launch_bounds__(256) void lr_bwd_mfma_kernel(const LrBwdArgs a) {
  constexpr int D = kD;
  __shared__ bf16x8 mt[2][8 * 64];      // A of F^T = M^T f^T, hi and lo
  __shared__ bf16x8 mr[2][2 * 4 * 64];  // A of G^T = M vec^T: (parity, channel chunk), hi and lo
  __shared__ bf16x8 pt[8 * 64];         // A of dX^T = P^T dy^T
  __shared__ __attribute__((aligned(16))) bf16 ty[2][kStep * kRp];  // dy hi, lo [token][coord]
  __shared__ __attribute__((aligned(16))) bf16 tx[kStep * kCp];     // x [token][channel]
  __shared__ __attribute__((aligned(16))) bf16 tf[KEY ? 1 : 2][KEY ? 8 : kStep * kRp];  // f hi, lo
  __shared__ __attribute__((aligned(16))) bf16 tu[KEY ? 1 : 2][KEY ? 8 : kStep * kCp];  // du hi, lo
  const long head = blockIdx.x / a.n_chunks;
  const int chunk = blockIdx.x % a.n_chunks, h = (int)(head % a.H);
  const long b = head / a.H;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, lr = lane % 16, g = lane / 16;
  const int r = a.r, half = r / 2, nrt = (r + 15) / 16;
  const bf16* Ph = a.P + (long)h * r * D;
  const float* Mh = a.M + head * r * D;

  // Fragments. mt, pt: row c = lane%16 of fragment w is channel frag_chan(w, c); k = 8g + s is
  // coordinate 2(4g + s%4) + s/4. mr: row = pair lane%16 (coordinate 2 pair + parity), k = channels
  // 32 kc + 8g + i. Coordinates >= r are zero.
  for (int e = tid; e < 8 * 64; e += 256) {
    const int ln = e % 64, w = e / 64, ch = frag_chan(w, ln % 16), gg = ln / 16;
    float m[8];
    bf16x8 pv;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int coord = 2 * (4 * gg + (s & 3)) + (s >> 2);
      m[s] = coord < r ? Mh[(long)coord * D + ch] : 0.f;
      pv[s] = coord < r ? Ph[(long)coord * D + ch] : (bf16)0.f;
    }
    bf16x8 hi, lo;
    split8(m, hi, lo);
    mt[0][e] = hi;
    mt[1][e] = lo;
    pt[e] = pv;
  }
  for (int e = tid; e < 2 * 4 * 64; e += 256) {
    const int ln = e % 64, kc = (e / 64) % 4, par = e / 256;
    const int coord = 2 * (ln % 16) + par, ch0 = 32 * kc + 8 * (ln / 16);
    float m[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) m[i] = coord < r ? Mh[(long)coord * D + ch0 + i] : 0.f;
    bf16x8 hi, lo;
    split8(m, hi, lo);
    mr[0][e] = hi;
    mr[1][e] = lo;
  }
  bf16x8 pe[4], po[4];  // A of Y^T: rows 2 lr and 2 lr + 1 of P, channels 32 kc + 8g .. +7
#pragma unroll
  for (int kc = 0; kc < 4; ++kc) {
    pe[kc] = lr < half ? *reinterpret_cast<const bf16x8*>(Ph + (long)(2 * lr) * D + 32 * kc + 8 * g)
                       : bf16x8{};
    po[kc] = lr < half ? *reinterpret_cast<const bf16x8*>(Ph + (long)(2 * lr + 1) * D + 32 * kc + 8 * g)
                       : bf16x8{};
  }
  f32x4 accm[2][2], accp[2][2];  // outer products: coordinate tile rt x channel tile ct
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) accm[rt][ct] = accp[rt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  __syncthreads();

  const int t0 = chunk * a.chunk_len, t1 = min(a.N, t0 + a.chunk_len);
  for (int base = t0; base < t1; base += kStep) {
    const int trow = 16 * wave + lr;  // this lane's token row in the step tiles
    const int tok = base + trow;
    const bool valid = tok < t1;
    const long row = (head * a.N + tok) * D;
    bf16x8 xf[4], yv[4], ov[4];
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      xf[kc] = valid ? *reinterpret_cast<const bf16x8*>(a.X + row + 32 * kc + 8 * g) : bf16x8{};
      yv[kc] = valid ? *reinterpret_cast<const bf16x8*>(a.Y + row + 32 * kc + 8 * g) : bf16x8{};
      if (!KEY)
        ov[kc] = valid ? *reinterpret_cast<const bf16x8*>(a.Os + row + 32 * kc + 8 * g) : bf16x8{};
    }
    float4 c4 = make_float4(1.f, 1.f, 1.f, 1.f), s4 = make_float4(0.f, 0.f, 0.f, 0.f);
    if (valid && 4 * g < half) {
      c4 = *reinterpret_cast<const float4*>(a.cos_tab + (long)tok * a.ld + 4 * g);
      s4 = *reinterpret_cast<const float4*>(a.sin_tab + (long)tok * a.ld + 4 * g);
    }
    const float lg = (!KEY && valid) ? a.logits[b * a.N + tok] : 0.f;
    const float cc[4] = {c4.x, c4.y, c4.z, c4.w}, ss[4] = {s4.x, s4.y, s4.z, s4.w};

    // Y^T and the features
    f32x4 ye = {0.f, 0.f, 0.f, 0.f}, yo = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      ye = mfma16(pe[kc], xf[kc], ye);
      yo = mfma16(po[kc], xf[kc], yo);
    }
    float fv[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float ae = silu(ye[v]), ao = silu(yo[v]);
      fv[v] = ae * cc[v] - ao * ss[v];
      fv[4 + v] = ae * ss[v] + ao * cc[v];
    }
    bf16x8 fh, fl;
    split8(fv, fh, fl);
    // F^T = M^T f^T
    f32x4 F[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const bf16x8 mh = mt[0][w * 64 + lane], ml = mt[1][w * 64 + lane];
      F[w] = mfma16(mh, fh, f32x4{0.f, 0.f, 0.f, 0.f});
      F[w] = mfma16(ml, fh, F[w]);
      F[w] = mfma16(mh, fl, F[w]);
    }
    bf16x8 vh[4], vl[4];  // B of G^T: du (query side, hi + lo) or V (key side)
    if constexpr (!KEY) {
      float su = 0.f, so = 0.f, tt = 0.f;
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float u = F[2 * p + (i >> 2)][i & 3], o = (float)ov[p][i], d = (float)yv[p][i];
          su = fmaf(u, u, su);
          so = fmaf(o, o, so);
          tt = fmaf(d, u, tt);
        }
      su = rows_sum(su);
      so = rows_sum(so);
      tt = rows_sum(tt);
      const float rho = sqrtf(su * (1.f / D) + a.eps_lr), rs = sqrtf(so * (1.f / D) + a.eps);
      const float gt = sigmoid(lg), coef = gt * rs / rho;
      const float kos = gt * tt / (rho * D * rs), kdu = coef * tt / (D * rho * rho);
      if (valid) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          bf16x8 o;
#pragma unroll
          for (int i = 0; i < 8; ++i) o[i] = (bf16)fmaf(kos, (float)ov[p][i], (float)yv[p][i]);
          *reinterpret_cast<bf16x8*>(a.dOs + row + 32 * p + 8 * g) = o;
        }
        if (g == 0) a.dlog_h[head * a.N + tok] = rs * tt / rho * gt * (1.f - gt);
      }
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        float du[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) du[i] = coef * (float)yv[p][i] - kdu * F[2 * p + (i >> 2)][i & 3];
        split8(du, vh[p], vl[p]);
      }
    } else {
      if (valid) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          *reinterpret_cast<float4*>(a.dV + row + 32 * p + 8 * g) =
              make_float4(F[2 * p][0], F[2 * p][1], F[2 * p][2], F[2 * p][3]);
          *reinterpret_cast<float4*>(a.dV + row + 32 * p + 8 * g + 4) =
              make_float4(F[2 * p + 1][0], F[2 * p + 1][1], F[2 * p + 1][2], F[2 * p + 1][3]);
        }
      }
#pragma unroll
      for (int p = 0; p < 4; ++p) vh[p] = yv[p];
    }
    // G^T = M vec^T, then dy
    f32x4 ge = {0.f, 0.f, 0.f, 0.f}, go = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      const bf16x8 eh = mr[0][kc * 64 + lane], el = mr[1][kc * 64 + lane];
      const bf16x8 oh = mr[0][(4 + kc) * 64 + lane], ol = mr[1][(4 + kc) * 64 + lane];
      ge = mfma16(eh, vh[kc], ge);
      ge = mfma16(el, vh[kc], ge);
      go = mfma16(oh, vh[kc], go);
      go = mfma16(ol, vh[kc], go);
      if constexpr (!KEY) {
        ge = mfma16(eh, vl[kc], ge);
        go = mfma16(oh, vl[kc], go);
      }
    }
    float dy[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float dae = ge[v] * cc[v] + go[v] * ss[v], dao = go[v] * cc[v] - ge[v] * ss[v];
      dy[v] = dae * silu_grad(ye[v]);
      dy[4 + v] = dao * silu_grad(yo[v]);
    }
    bf16x8 dh, dl;
    split8(dy, dh, dl);
    // dX^T = P^T dy^T
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      f32x4 d0 = mfma16(pt[(2 * p) * 64 + lane], dh, f32x4{0.f, 0.f, 0.f, 0.f});
      d0 = mfma16(pt[(2 * p) * 64 + lane], dl, d0);
      f32x4 d1 = mfma16(pt[(2 * p + 1) * 64 + lane], dh, f32x4{0.f, 0.f, 0.f, 0.f});
      d1 = mfma16(pt[(2 * p + 1) * 64 + lane], dl, d1);
      if (valid) {
        *reinterpret_cast<float4*>(a.dX + row + 32 * p + 8 * g) = make_float4(d0[0], d0[1], d0[2], d0[3]);
        *reinterpret_cast<float4*>(a.dX + row + 32 * p + 8 * g + 4) = make_float4(d1[0], d1[1], d1[2], d1[3]);
      }
    }

    // Outer products over the step's 64 tokens (invalid tokens hold zeros everywhere).
    __syncthreads();  // the previous step's tiles are consumed
    *reinterpret_cast<bf16x8*>(&ty[0][trow * kRp + 8 * g]) = interleave(dh);
    *reinterpret_cast<bf16x8*>(&ty[1][trow * kRp + 8 * g]) = interleave(dl);
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
      *reinterpret_cast<bf16x8*>(&tx[trow * kCp + 32 * kc + 8 * g]) = xf[kc];
    if constexpr (!KEY) {
      *reinterpret_cast<bf16x8*>(&tf[0][trow * kRp + 8 * g]) = interleave(fh);
      *reinterpret_cast<bf16x8*>(&tf[1][trow * kRp + 8 * g]) = interleave(fl);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        *reinterpret_cast<bf16x8*>(&tu[0][trow * kCp + 32 * p + 8 * g]) = vh[p];
        *reinterpret_cast<bf16x8*>(&tu[1][trow * kCp + 32 * p + 8 * g]) = vl[p];
      }
    }
    __syncthreads();
#pragma unroll
    for (int kt = 0; kt < kStep / 32; ++kt) {
      const int r0 = 32 * kt + 8 * g;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        if (rt >= nrt) break;
        const bf16x8 ah = tr_rows8(ty[0], kRp, r0, 16 * rt, lane);
        const bf16x8 al = tr_rows8(ty[1], kRp, r0, 16 * rt, lane);
        bf16x8 fh2, fl2;
        if constexpr (!KEY) {
          fh2 = tr_rows8(tf[0], kRp, r0, 16 * rt, lane);
          fl2 = tr_rows8(tf[1], kRp, r0, 16 * rt, lane);
        }
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) {
          const int c0 = 32 * wave + 16 * ct;
          const bf16x8 bx = tr_rows8(tx, kCp, r0, c0, lane);
          accp[rt][ct] = mfma16(ah, bx, accp[rt][ct]);
          accp[rt][ct] = mfma16(al, bx, accp[rt][ct]);
          if constexpr (!KEY) {
            const bf16x8 uh = tr_rows8(tu[0], kCp, r0, c0, lane);
            const bf16x8 ul = tr_rows8(tu[1], kCp, r0, c0, lane);
            accm[rt][ct] = mfma16(fh2, uh, accm[rt][ct]);
            accm[rt][ct] = mfma16(fh2, ul, accm[rt][ct]);
            accm[rt][ct] = mfma16(fl2, uh, accm[rt][ct]);
          }
        }
      }
    }
  }
  // Partials [coordinate][channel]: lane holds channel 32 wave + 16 ct + lr, coordinates
  // 16 rt + 4g + v.
  const long pbase = (head * a.n_chunks + chunk) * (long)(r * D);
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int coord = 16 * rt + 4 * g + v, ch = 32 * wave + 16 * ct + lr;
        if (coord < r) {
          a.part_dP[pbase + coord * D + ch] = accp[rt][ct][v];
          if constexpr (!KEY) a.part_dM[pbase + coord * D + ch] = accm[rt][ct][v];
        }
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
  len = (len + kStep - 1) / kStep * kStep;  // whole steps of the MFMA path
  return (int)(len < kStep ? kStep : len);
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
  const dim3 grid((unsigned)(heads * n_chunks));
  const bool mfma = r <= 32;
  if (mfma) {
    const LrBwdArgs q{s.N, s.H, r, chunk_len, n_chunks, ld, (const bf16*)Qn, (const bf16*)Pq,
                      cos_tab, sin_tab, C, (const bf16*)Os, logits, eps_lr, eps, (const bf16*)dO,
                      (bf16*)dOs, dQn, nullptr, dlog_h, part_dC, part_dPq};
    hipLaunchKernelGGL(lr_bwd_mfma_kernel<false>, grid, dim3(256), 0, st, q);
  } else {
    hipLaunchKernelGGL(lr_bwd_q_kernel, grid, dim3(256), 0, st, s.N, s.H, r, chunk_len, n_chunks,
                       ld, (const bf16*)Qn, (const bf16*)Pq, cos_tab, sin_tab, C, (const bf16*)Os,
                       logits, eps_lr, eps, (const bf16*)dO, (bf16*)dOs, dQn, dlog_h, part_dC,
                       part_dPq);
  }
  // dC[b, h] = sum over chunks
  hipLaunchKernelGGL(lr_bwd_reduce_kernel, dim3(rgrid.x, (unsigned)heads), dim3(256), 0, st, re, s.B,
                     s.H, n_chunks, true, (const float*)part_dC, dC);
  if (mfma) {
    const LrBwdArgs k{s.N, s.H, r, chunk_len, n_chunks, ld, (const bf16*)Kn, (const bf16*)Pk,
                      cos_tab, sin_tab, dC, nullptr, nullptr, 0.f, 0.f, (const bf16*)V, nullptr,
                      dKn, dV, nullptr, nullptr, part_dPk};
    hipLaunchKernelGGL(lr_bwd_mfma_kernel<true>, grid, dim3(256), 0, st, k);
  } else {
    hipLaunchKernelGGL(lr_bwd_k_kernel, grid, dim3(256), 0, st, s.N, s.H, r, chunk_len, n_chunks,
                       ld, (const bf16*)Kn, (const bf16*)V, (const bf16*)Pk, cos_tab, sin_tab,
                       (const float*)dC, dKn, dV, part_dPk);
  }
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
