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
// Two passes of one kernel (query side, then key side from the reduced dC), one workgroup per
// (b, h, chunk of tokens), on MFMA (below). The outer products dC, dP_q, dP_k accumulate per
// workgroup over its chunk and are summed over chunks (and batch) in a fixed order afterwards, so
// every gradient is reproducible. fp32 arithmetic from bf16 inputs, r <= 64.
#include "common.h"
#include "launch.h"

namespace rola {
namespace {

constexpr int kD = 128, kMaxR = 64;

__device__ __forceinline__ float silu_grad(float y) {  // d/dy y sigmoid(y)
  const float s = sigmoid(y);
  return s * (1.f + y * (1.f - s));
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

// ---- MFMA path (r <= 64) ---------------------------------------------------------------------
// One workgroup per (b, h, chunk of tokens); per step each of its four waves takes a 16-token tile
// (lane = token l%16, group g = l/16) through v_mfma_f32_16x16x32_bf16, in the layouts of the
// forward readout, where every product's output lands in the register layout the next one reads.
// The r coordinates form JT = ceil(r/32) tiles of 16 rotation pairs; lane (g, token) holds pairs
// 16 jt + 4g + v (v < 4) of tile jt:
//   Y^T  = P X^T        A = even / odd rows of P: rows = pairs, k = channels
//   f    = R_r SiLU(Y)  in registers, split into bf16 hi + lo
//   F^T  = M^T f^T      A = M^T (transposing reads), k = the 32 coordinates of one pair tile:
//                       query side u (M = C), key side dV (M = dC); lane (g, token) gets channels
//                       32p + 8g .. +7 in F[2p], F[2p+1]
//   query side: RMSNorm and gate backward per token (in-lane sums + one four-lane reduction), du
//   G^T  = M vec^T      A = rows of M (hi + lo), B = du (hi + lo) or V: dq~ / dk~ per pair
//   dy   = SiLU'(Y) R_r^T G   in registers
//   dX^T = P^T dy^T     A = P^T (transposing reads), B = dy (hi + lo): dQ^n / dK^n
// P and M (hi, lo) sit in LDS once per workgroup as row-major [coordinate][channel] tiles whose rows
// are held pair-major within each group of eight (coordinates 8a, 8a+2, 8a+4, 8a+6, 8a+1, ..):
// a transposing read of eight consecutive rows then yields the coordinates in the order the
// features are held, and a row read serves the even / odd rows of a pair tile.
// The outer products dC = sum f du^T and dP = sum dy x^T contract over tokens: the four waves write
// their tiles (token-major) to LDS and every wave contracts the step's 64 tokens for its own 32
// channels, reading the operands with ds_read_b64_tr_b16 (token-major rows -> one lane per column).
// fp32 operands enter as bf16 hi + lo pairs (three products, or two against exact bf16 data), which
// keeps them to about 2^-16 relative. Partials per chunk as in the plain kernels.
constexpr int kStep = 64;  // tokens per workgroup step
constexpr int kMp = 136;   // LDS row pitch (bf16) of the P and M tiles: conflict-free row reads
constexpr int kCp = 144;   // LDS row pitch (bf16) of token-major channel tiles

// LDS row pitch (bf16) of token-major coordinate tiles: conflict-free transposing reads.
template <int JT>
constexpr int coord_pitch() { return JT == 1 ? 48 : 72; }

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Row of the P / M tiles that holds coordinate c: pair-major within each group of eight.
__device__ __forceinline__ int tile_row(int c) { return (c & ~7) + 4 * (c & 1) + ((c & 7) >> 1); }

// bf16 hi + lo parts of eight floats.
__device__ __forceinline__ void split8(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    hi[i] = (bf16)x[i];
    lo[i] = (bf16)(x[i] - (float)hi[i]);
  }
}

// Transposing read of rows row0 .. row0 + 7 of a row-major LDS tile: lane 4q + e of each 16-lane
// group gets column col(q) + e of the eight rows (col(q) a multiple of 4).
template <typename Col>
__device__ __forceinline__ bf16x8 tr_read8(const bf16* tile, int pitch, int row0, Col col, int lane) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int i16 = lane % 16;
  const bf16* p = tile + (row0 + (i16 >> 2)) * pitch + col(i16 & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 4 * pitch));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Operand that contracts over the rows of a row-major LDS tile: lane l gets column col0 + l%16 of
// rows row0 .. row0 + 7, row0 given per 16-lane group.
__device__ __forceinline__ bf16x8 tr_rows8(const bf16* tile, int pitch, int row0, int col0, int lane) {
  return tr_read8(tile, pitch, row0, [=](int q) { return col0 + 4 * q; }, lane);
}

// A operand of a product whose output rows are channels (F^T, dX^T): fragment w, lane 4q + e of each
// 16-lane group, is channel 32(w/2) + 8q + 4(w%2) + e, so output lane (g, token) of fragments 2p and
// 2p + 1 holds the consecutive channels 32p + 8g .. +7. k = the coordinates of tile rows
// row0 .. row0 + 7.
__device__ __forceinline__ bf16x8 chan_frag(const bf16* tile, int w, int row0, int lane) {
  const int base = 32 * (w >> 1) + 4 * (w & 1);
  return tr_read8(tile, kMp, row0, [=](int q) { return base + 8 * q; }, lane);
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

template <bool KEY, int JT>
__global__ __launch_bounds__(256) void lr_bwd_mfma_kernel(const LrBwdArgs a) {
  constexpr int D = kD, RT = 32 * JT, kRp = coord_pitch<JT>();
  __shared__ __attribute__((aligned(16))) bf16 ps[RT * kMp];                // P
  __shared__ __attribute__((aligned(16))) bf16 ms[2][RT * kMp];             // M hi, lo
  __shared__ __attribute__((aligned(16))) bf16 ty[2][kStep * kRp];          // dy hi, lo [token][coord]
  __shared__ __attribute__((aligned(16))) bf16 tx[kStep * kCp];             // x [token][channel]
  __shared__ __attribute__((aligned(16))) bf16 tf[KEY ? 1 : 2][KEY ? 8 : kStep * kRp];  // f hi, lo
  __shared__ __attribute__((aligned(16))) bf16 tu[KEY ? 1 : 2][KEY ? 8 : kStep * kCp];  // du hi, lo
  const long head = blockIdx.x / a.n_chunks;
  const int chunk = blockIdx.x % a.n_chunks, h = (int)(head % a.H);
  const long b = head / a.H;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, lr = lane % 16, g = lane / 16;
  const int r = a.r, half = r / 2, nrt = (r + 15) / 16;
  const bf16* Ph = a.P + (long)h * r * D;
  const float* Mh = a.M + head * r * D;

  // The tiles; coordinates >= r are zero rows.
  for (int e = tid; e < RT * D / 4; e += 256) {
    const int c = e / (D / 4), ch = 4 * (e % (D / 4)), row = tile_row(c) * kMp + ch;
    float4 m = make_float4(0.f, 0.f, 0.f, 0.f);
    bf16x4 pv = {};
    if (c < r) {
      m = *reinterpret_cast<const float4*>(Mh + (long)c * D + ch);
      pv = *reinterpret_cast<const bf16x4*>(Ph + (long)c * D + ch);
    }
    const float mv[4] = {m.x, m.y, m.z, m.w};
    bf16x4 hi, lo;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      hi[i] = (bf16)mv[i];
      lo[i] = (bf16)(mv[i] - (float)hi[i]);
    }
    *reinterpret_cast<bf16x4*>(&ms[0][row]) = hi;
    *reinterpret_cast<bf16x4*>(&ms[1][row]) = lo;
    *reinterpret_cast<bf16x4*>(&ps[row]) = pv;
  }
  // Row operand of pair tile jt: row 16 jt + lr of the even (par 0) or odd coordinates, channels
  // 32 kc + 8g .. +7.
  auto row_op = [&](const bf16* tile, int jt, int par, int kc) {
    return *reinterpret_cast<const bf16x8*>(tile + tile_row(2 * (16 * jt + lr) + par) * kMp + 32 * kc + 8 * g);
  };
  f32x4 accm[2 * JT][2], accp[2 * JT][2];  // outer products: coordinate tile rt x channel tile ct
#pragma unroll
  for (int rt = 0; rt < 2 * JT; ++rt)
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
    float cc[JT][4], ss[JT][4];  // cos / sin of the lane's pairs 16 jt + 4g + v
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      float4 c4 = make_float4(1.f, 1.f, 1.f, 1.f), s4 = make_float4(0.f, 0.f, 0.f, 0.f);
      const int j0 = 16 * jt + 4 * g;
      if (valid && j0 < half) {  // j0 + 3 < ld: ld >= half and both are multiples of 4
        c4 = *reinterpret_cast<const float4*>(a.cos_tab + (long)tok * a.ld + j0);
        s4 = *reinterpret_cast<const float4*>(a.sin_tab + (long)tok * a.ld + j0);
      }
      cc[jt][0] = c4.x, cc[jt][1] = c4.y, cc[jt][2] = c4.z, cc[jt][3] = c4.w;
      ss[jt][0] = s4.x, ss[jt][1] = s4.y, ss[jt][2] = s4.z, ss[jt][3] = s4.w;
    }
    const float lg = (!KEY && valid) ? a.logits[b * a.N + tok] : 0.f;

    // Y^T and the features
    f32x4 ye[JT], yo[JT];
    bf16x8 fh[JT], fl[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      ye[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
      yo[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        ye[jt] = mfma16(row_op(ps, jt, 0, kc), xf[kc], ye[jt]);
        yo[jt] = mfma16(row_op(ps, jt, 1, kc), xf[kc], yo[jt]);
      }
      float fv[8];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float ae = silu(ye[jt][v]), ao = silu(yo[jt][v]);
        fv[v] = ae * cc[jt][v] - ao * ss[jt][v];
        fv[4 + v] = ae * ss[jt][v] + ao * cc[jt][v];
      }
      split8(fv, fh[jt], fl[jt]);
    }
    // F^T = M^T f^T
    f32x4 F[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      F[w] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        const bf16x8 mh = chan_frag(ms[0], w, 32 * jt + 8 * g, lane);
        const bf16x8 ml = chan_frag(ms[1], w, 32 * jt + 8 * g, lane);
        F[w] = mfma16(mh, fh[jt], F[w]);
        F[w] = mfma16(ml, fh[jt], F[w]);
        F[w] = mfma16(mh, fl[jt], F[w]);
      }
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
      // a padding token contributes nothing (with eps_lr = 0 its rho is 0 and coef not finite)
      const float cu = valid ? coef : 0.f, ku = valid ? kdu : 0.f;
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
        for (int i = 0; i < 8; ++i) du[i] = cu * (float)yv[p][i] - ku * F[2 * p + (i >> 2)][i & 3];
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
    // G^T = M vec^T per pair tile, then dy
    bf16x8 dh[JT], dl[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      f32x4 ge = {0.f, 0.f, 0.f, 0.f}, go = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        const bf16x8 eh = row_op(ms[0], jt, 0, kc), el = row_op(ms[1], jt, 0, kc);
        const bf16x8 oh = row_op(ms[0], jt, 1, kc), ol = row_op(ms[1], jt, 1, kc);
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
        const float c = cc[jt][v], s = ss[jt][v];
        const float dae = ge[v] * c + go[v] * s, dao = go[v] * c - ge[v] * s;
        dy[v] = dae * silu_grad(ye[jt][v]);
        dy[4 + v] = dao * silu_grad(yo[jt][v]);
      }
      split8(dy, dh[jt], dl[jt]);
    }
    // dX^T = P^T dy^T
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      f32x4 d0 = {0.f, 0.f, 0.f, 0.f}, d1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        const bf16x8 p0 = chan_frag(ps, 2 * p, 32 * jt + 8 * g, lane);
        const bf16x8 p1 = chan_frag(ps, 2 * p + 1, 32 * jt + 8 * g, lane);
        d0 = mfma16(p0, dh[jt], d0);
        d0 = mfma16(p0, dl[jt], d0);
        d1 = mfma16(p1, dh[jt], d1);
        d1 = mfma16(p1, dl[jt], d1);
      }
      if (valid) {
        *reinterpret_cast<float4*>(a.dX + row + 32 * p + 8 * g) = make_float4(d0[0], d0[1], d0[2], d0[3]);
        *reinterpret_cast<float4*>(a.dX + row + 32 * p + 8 * g + 4) = make_float4(d1[0], d1[1], d1[2], d1[3]);
      }
    }

    // Outer products over the step's 64 tokens (invalid tokens hold zeros everywhere).
    __syncthreads();  // the previous step's tiles are consumed
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      *reinterpret_cast<bf16x8*>(&ty[0][trow * kRp + 32 * jt + 8 * g]) = interleave(dh[jt]);
      *reinterpret_cast<bf16x8*>(&ty[1][trow * kRp + 32 * jt + 8 * g]) = interleave(dl[jt]);
      if constexpr (!KEY) {
        *reinterpret_cast<bf16x8*>(&tf[0][trow * kRp + 32 * jt + 8 * g]) = interleave(fh[jt]);
        *reinterpret_cast<bf16x8*>(&tf[1][trow * kRp + 32 * jt + 8 * g]) = interleave(fl[jt]);
      }
    }
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
      *reinterpret_cast<bf16x8*>(&tx[trow * kCp + 32 * kc + 8 * g]) = xf[kc];
    if constexpr (!KEY) {
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
      for (int rt = 0; rt < 2 * JT; ++rt) {
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
  for (int rt = 0; rt < 2 * JT; ++rt)
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
  const LrBwdArgs q{s.N, s.H, r, chunk_len, n_chunks, ld, (const bf16*)Qn, (const bf16*)Pq,
                    cos_tab, sin_tab, C, (const bf16*)Os, logits, eps_lr, eps, (const bf16*)dO,
                    (bf16*)dOs, dQn, nullptr, dlog_h, part_dC, part_dPq};
  if (r <= 32)
    hipLaunchKernelGGL((lr_bwd_mfma_kernel<false, 1>), grid, dim3(256), 0, st, q);
  else
    hipLaunchKernelGGL((lr_bwd_mfma_kernel<false, 2>), grid, dim3(256), 0, st, q);
  // dC[b, h] = sum over chunks
  hipLaunchKernelGGL(lr_bwd_reduce_kernel, dim3(rgrid.x, (unsigned)heads), dim3(256), 0, st, re, s.B,
                     s.H, n_chunks, true, (const float*)part_dC, dC);
  const LrBwdArgs k{s.N, s.H, r, chunk_len, n_chunks, ld, (const bf16*)Kn, (const bf16*)Pk,
                    cos_tab, sin_tab, dC, nullptr, nullptr, 0.f, 0.f, (const bf16*)V, nullptr,
                    dKn, dV, nullptr, nullptr, part_dPk};
  if (r <= 32)
    hipLaunchKernelGGL((lr_bwd_mfma_kernel<true, 1>), grid, dim3(256), 0, st, k);
  else
    hipLaunchKernelGGL((lr_bwd_mfma_kernel<true, 2>), grid, dim3(256), 0, st, k);
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
