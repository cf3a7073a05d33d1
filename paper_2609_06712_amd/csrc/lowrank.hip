// Rotary low-rank branch (eq. qklr, eq. ctx; Algorithm steps 5-7) and gated fusion (eq. gate,
// Algorithm steps 8-10).
//
// Features are the paper's even/odd split (Sec. 4.5, fused inference kernel): projecting with the
// even rows and the odd rows of P separately puts both members of every rotary pair in the same lane
// and register slot, so SiLU and the rotation R_r are in-register arithmetic between two MFMA
// results, no lane exchange.
//
// bf16 summary: per (b, h, token chunk) one workgroup of 4 waves, 32 tokens per wave per step.
//   Psi = K^n P^T      (even and odd P rows)  A = K^n rows straight from HBM (prefetched one step
//                      ahead), B = P fragments in registers; lane = pair j, 4 tokens per 16-token tile
//   k~ = R_r SiLU(Psi) in registers (fp32), rounded to bf16 as the B operand of
//   C^T += V^T k~      A = V^T from LDS (V transposed while staged), fp32 accumulators in registers.
// Waves are summed through LDS in a fixed order, chunks by a second kernel in a fixed order: C and z
// are bitwise reproducible (no float atomics).
//
// bf16 readout (+ combine): per wave 16-token tiles.
//   Phi = P Q^T        A = P fragments (registers), B = Q^n rows from HBM; lane = token, 4 pairs
//   q~ = R_r SiLU(Phi) in registers, rounded to bf16
//   u^T = C^T q~       A = C^T (bf16, registers, loaded once per workgroup)
//   RMSNorm over d_h (in-lane sums + 2 shuffles); fused: O = (O^s/r_s + g O^lr) r_s.
// Both kernels are HBM-bound; grids are ordered head-minor. The readout's is remapped so an XCD
// works on one token range for all heads, reading each rotary-table row once into its L2; the
// summary's is dealt round-robin (measured faster for it).
#include "common.h"
#include "launch.h"

namespace rola {
namespace {

constexpr int kSummaryStep = 128;  // tokens per workgroup step (4 waves x 32)

__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Feature map of the low-rank branch. The paper's design is SiLU with the rotation applied outside
// it (eq. qklr); its ablations replace SiLU by Identity, Tanh, ReLU or GELU and move the rotation
// inside the activation or drop it (Sec. 5.1 RoPE placement, Prop. inside). feat = phi | order << 8
// with the ROLA_PHI_* / ROLA_ROPE_* values of the ABI. Every phi maps 0 to 0, so zero rows (padding
// tokens, padding pairs) keep zero features under every variant.
constexpr int kPhiSilu = 0, kPhiIdentity = 1, kPhiTanh = 2, kPhiRelu = 3, kPhiGelu = 4;
constexpr int kRopeOutside = 0, kRopeInside = 1, kRopeNone = 2;

__device__ __forceinline__ float feature_act(float x, int phi) {
  switch (phi) {
    case kPhiIdentity: return x;
    case kPhiTanh: return tanhf(x);
    case kPhiRelu: return fmaxf(x, 0.f);
    case kPhiGelu: return 0.5f * x * (1.f + erff(x * 0.70710678118654752f));  // exact (erf) GELU
    default: return silu(x);
  }
}

// Features of one rotary pair from its two projections (e, o) = (P_2j x, P_2j+1 x) at a position
// with rotation (c, s). GENERIC = false is the paper's design, SiLU then the rotation; GENERIC =
// true applies feat at run time (the default feat gives the same arithmetic).
template <bool GENERIC>
__device__ __forceinline__ void feature_pair(float& e, float& o, float c, float s, int feat) {
  if (!GENERIC) {
    const float a = silu(e), b = silu(o);
    e = a * c - b * s;
    o = a * s + b * c;
    return;
  }
  const int phi = feat & 0xFF, order = feat >> 8;
  if (order == kRopeInside) {
    const float a = e * c - o * s, b = e * s + o * c;
    e = a;
    o = b;
  }
  const float a = feature_act(e, phi), b = feature_act(o, phi);
  if (order == kRopeOutside) {
    e = a * c - b * s;
    o = a * s + b * c;
  } else {
    e = a;
    o = b;
  }
}

int summary_chunk_len(const Shape& s) {
  const long heads = (long)s.B * s.H;
  // About 1024 workgroups, two rounds of the two per CU the chip holds. At the 14B shape, against
  // 2048: r = 32 314 -> 309 us, r = 64 420 -> 388 us (fewer partials to write and reduce); 512 and
  // 4096 were slower at r = 32.
  const long want = (1024 + heads - 1) / heads;
  long len = (s.N + want - 1) / want;
  len = (len + kSummaryStep - 1) / kSummaryStep * kSummaryStep;
  return (int)(len < kSummaryStep ? kSummaryStep : len);
}

// ------------------------------------------------------------------------------------------------
// bf16 summary
// ------------------------------------------------------------------------------------------------
// split = 2: each (b, h, chunk) is served by two workgroups, one per half of the pair tiles (r = 128
// as two r = 64 halves: one workgroup holding all four tiles spills). The two sit eight launch
// slots apart, i.e. on the same XCD at about the same time, so the second reads K^n and V from L2.
template <int JT, bool GENERIC>
__global__ __launch_bounds__(256, JT == 1 ? 2 : 1) void summary_mfma_kernel(
    int N, int H, int r, int chunk_len, int n_chunks, int total, int split, int ld, int feat,
    const bf16* __restrict__ Kn, const bf16* __restrict__ V, const bf16* __restrict__ Pk,
    const float* __restrict__ cos_tab, const float* __restrict__ sin_tab,
    float* __restrict__ part) {
  constexpr int D = 128, TOK = kSummaryStep;
  constexpr int TILE = TOK * D * 2;  // one step's V tile: 32 KB, row-major, chunks swizzled
  // Two V stages filled by direct global-to-LDS loads; the first stage is reused for the final
  // cross-wave reduction.
  __shared__ __attribute__((aligned(1024))) char lds[2 * TILE];

  const int BH = total / n_chunks;
  // heads minor in launch order, dealt round-robin to the XCDs: 2.7 % faster at the 14B shape than
  // giving each XCD a contiguous token range of all heads (which shared the table rows in L2)
  int L = blockIdx.x, jt0 = 0;  // jt0: first pair tile of this workgroup
  if (split == 2) {
    L = (int)(blockIdx.x / 16) * 8 + blockIdx.x % 8;
    jt0 = JT * ((blockIdx.x / 8) % 2);
    if (L >= total) return;  // the grid is rounded up to whole groups of 16
  }
  const int head = L % BH, chunk = L / BH;
  const int h = head % H;
  const int tid = threadIdx.x, lane = tid % 64, lr = lane % 16, g = lane / 16;
  const int wave = wave_uniform(tid / 64);
  const int half = r / 2;
  const bf16* Kh = Kn + (long)head * N * D;
  const char* Vh = reinterpret_cast<const char*>(V + (long)head * N * D);
  const bf16* Ph = Pk + (long)h * r * D;

  bf16x8 pe[JT][4], po[JT][4];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) {
    const int j = 16 * (jt0 + jt) + lr;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      if (j < half) {
        pe[jt][kc] = *reinterpret_cast<const bf16x8*>(Ph + (long)(2 * j) * D + 32 * kc + 8 * g);
        po[jt][kc] = *reinterpret_cast<const bf16x8*>(Ph + (long)(2 * j + 1) * D + 32 * kc + 8 * g);
      } else {
        pe[jt][kc] = bf16x8{};
        po[jt][kc] = bf16x8{};
      }
    }
  }
  f32x4 ce[JT][8], co[JT][8];
  float ze[JT], zo[JT];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) {
    ze[jt] = zo[jt] = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) ce[jt][w] = co[jt][w] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int t0 = chunk * chunk_len, t1 = min(N, t0 + chunk_len);
  // V tile DMA: lane l of 1-KB slot q (8 slots per wave) fills row 4q + l/16, position l%16 with
  // source chunk position ^ 2(row%8); rows past the chunk re-read its last row (V rows of tokens
  // beyond the chunk meet zero features, so they add nothing).
  typedef __attribute__((address_space(3))) void lds_void;
  // Slot i's row is row0 + 4i; its swizzle depends only on i's parity (rows advance by 4).
  const int row0 = 32 * wave + lane / 16, pos = lane % 16;
  int dvp[2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
    dvp[p] = (row0 + 4 * p) * D * 2 + ((pos ^ (((row0 + 4 * p) & 7) << 1)) << 4);
  auto issue_v = [&](int base, int buf) {
    char* dst = lds + buf * TILE;
    if (base + TOK <= t1) {
      const char* vb = Vh + (long)base * D * 2;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_global_load_lds((const void*)(vb + dvp[i & 1] + (i >> 1) * 2048),
                                         (lds_void*)(dst + (wave * 8 + i) * 1024), 16, 0, 0);
    } else {  // tail: rows past the chunk re-read its last row
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int row = row0 + 4 * i;
        const long shift = (long)(min(base + row, t1 - 1) - row) * D * 2;
        __builtin_amdgcn_global_load_lds((const void*)(Vh + shift + dvp[i & 1] + (i >> 1) * 2048),
                                         (lds_void*)(dst + (wave * 8 + i) * 1024), 16, 0, 0);
      }
    }
  };
  // Transposing-read offsets of the V^T operand: lane (g, 4 s' + m') reads token row
  // wave*32 + 4g + s' (+16), channels 16w + 4m'.
  const int sp = lr >> 2, mp = lr & 3, vr = wave * 32 + 4 * g + sp;
  int vo[8];
#pragma unroll
  for (int w = 0; w < 8; ++w)
    vo[w] = vr * 256 + (((2 * w + (mp >> 1)) ^ ((vr & 7) << 1)) << 4) + ((mp & 1) << 3);

  // A step reads K^n operand rows from registers and V from the wave's own rows of an LDS stage.
  // Each wave fills and reads only its own 32 rows of a stage, so the waves run their pipelines
  // independently, with no workgroup barrier: the K^n and V loads of step t+1 are issued before the
  // wave waits for those of step t, into registers and a stage that only this wave used at step
  // t-1. The rotary-table entries (L2-resident rows shared by all heads) are loaded at the start of
  // their own step: a second register set for them spills. At the 14B shape this loop is 1.5 %
  // faster than a workgroup-synchronous one at r = 32 and 12 % at r = 64; double-buffered tables
  // made it 19 % slower at r = 32.
  struct StepRegs {
    bf16x8 k[2][4];
  };
  float tcs[JT][2][4], tsn[JT][2][4];  // this step's table entries
  auto issue_step = [&](int base, int buf, StepRegs& R) {
    // the previous step's LDS reads of this stage are complete before the DMA may overwrite it
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    issue_v(base, buf);
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int tok = base + wave * 32 + tt * 16 + lr;
#pragma unroll
      for (int kc = 0; kc < 4; ++kc)
        R.k[tt][kc] = tok < t1 ? *reinterpret_cast<const bf16x8*>(Kh + (long)tok * D + 32 * kc + 8 * g)
                               : bf16x8{};
    }
  };
  auto load_tables = [&](int base) {
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int tok = base + wave * 32 + tt * 16 + 4 * g + v, j = 16 * (jt0 + jt) + lr;
          const bool ok = tok < t1 && j < half;
          tcs[jt][tt][v] = ok ? cos_tab[(long)tok * ld + j] : 1.f;
          tsn[jt][tt][v] = ok ? sin_tab[(long)tok * ld + j] : 0.f;
        }
  };
  // vector-memory instructions per wave of one issue_step
  constexpr int kStepLoads = 8 + 8;
  constexpr int kAhead = kStepLoads < 63 ? kStepLoads : 63;

  auto compute = [&](const StepRegs& R, int buf) {
    const char* Vs = lds + buf * TILE;
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      bf16x8 be, bo;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        f32x4 ye = {0.f, 0.f, 0.f, 0.f}, yo = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
          ye = mfma16x16x32(R.k[tt][kc], pe[jt][kc], ye);
          yo = mfma16x16x32(R.k[tt][kc], po[jt][kc], yo);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          float ke = ye[v], ko = yo[v];
          feature_pair<GENERIC>(ke, ko, tcs[jt][tt][v], tsn[jt][tt][v], feat);
          ze[jt] += ke;
          zo[jt] += ko;
          be[4 * tt + v] = (bf16)ke;
          bo[4 * tt + v] = (bf16)ko;
        }
      }
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + vo[w]));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(Vs + vo[w] + 16 * 256));
        const bf16x8 va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        ce[jt][w] = mfma16x16x32(va, be, ce[jt][w]);
        co[jt][w] = mfma16x16x32(va, bo, co[jt][w]);
      }
    }
  };
  // One step: start the next step's loads, wait for this step's (the next step's stay in flight),
  // compute.
  auto step = [&](int base, int buf, const StepRegs& cur, StepRegs& nxt) {
    load_tables(base);
    if (base + TOK < t1) {
      issue_step(base + TOK, buf ^ 1, nxt);
      __builtin_amdgcn_s_waitcnt((kAhead & 15) | ((kAhead >> 4) << 14) | (7 << 4) | (15 << 8));
    } else {
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    }
    compute(cur, buf);
  };

  StepRegs ra, rb;
  issue_step(t0, 0, ra);
  int base = t0;
  for (; base + TOK < t1; base += 2 * TOK) {
    step(base, 0, ra, rb);
    step(base + TOK, 1, rb, ra);
  }
  if (base < t1) step(base, 0, ra, rb);

  // z: the four lane groups hold different tokens of the same pair j
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) {
    ze[jt] = rows_sum(ze[jt]);
    zo[jt] = rows_sum(zo[jt]);
  }
  // Sum the four waves in a fixed order: wave 3 -> 2 -> 1 -> 0, one pair-tile at a time.
  constexpr int PER = 2 * 8 * 4 + 2;  // floats per lane per pair tile
  float* red = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) {
    for (int src = 3; src >= 1; --src) {
      __syncthreads();
      if (wave == src) {
#pragma unroll
        for (int w = 0; w < 8; ++w)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            red[((0 * 8 + w) * 4 + v) * 64 + lane] = ce[jt][w][v];
            red[((1 * 8 + w) * 4 + v) * 64 + lane] = co[jt][w][v];
          }
        red[(PER - 2) * 64 + lane] = ze[jt];
        red[(PER - 1) * 64 + lane] = zo[jt];
      }
      __syncthreads();
      if (wave == src - 1) {
#pragma unroll
        for (int w = 0; w < 8; ++w)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            ce[jt][w][v] += red[((0 * 8 + w) * 4 + v) * 64 + lane];
            co[jt][w][v] += red[((1 * 8 + w) * 4 + v) * 64 + lane];
          }
        ze[jt] += red[(PER - 2) * 64 + lane];
        zo[jt] += red[(PER - 1) * 64 + lane];
      }
    }
  }
  if (wave == 0) {
    float* P = part + ((long)head * n_chunks + chunk) * (long)(r * D + r);
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      const int j = 16 * (jt0 + jt) + lr;
      if (j >= half) continue;
#pragma unroll
      for (int w = 0; w < 8; ++w)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int dim = 16 * w + 4 * g + v;
          P[(long)(2 * j) * D + dim] = ce[jt][w][v];
          P[(long)(2 * j + 1) * D + dim] = co[jt][w][v];
        }
      if (g == 0) {
        P[(long)r * D + 2 * j] = ze[jt];
        P[(long)r * D + 2 * j + 1] = zo[jt];
      }
    }
  }
}

// ------------------------------------------------------------------------------------------------
// Plain summary for the fp32 path: 32-token sub-tiles through LDS, thread per (pair) then (r, c).
// ------------------------------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void summary_simple_kernel(
    int N, int H, int r, int chunk_len, int n_chunks, int ld, int feat, const T* __restrict__ Kn,
    const T* __restrict__ V, const T* __restrict__ Pk, const float* __restrict__ cos_tab,
    const float* __restrict__ sin_tab, float* __restrict__ part) {
  constexpr int TT = 32, MAXR = 128;
  __shared__ float Ks[TT][D];
  __shared__ float Vs[TT][D];
  __shared__ float kt[TT][MAXR];
  const int chunk = blockIdx.x;
  const long head = (long)blockIdx.z * gridDim.y + blockIdx.y;
  const int h = blockIdx.y;
  const T* Kh = Kn + head * (long)N * D;
  const T* Vh = V + head * (long)N * D;
  const T* Ph = Pk + (long)h * r * D;
  const int half = r / 2;
  const int t0 = chunk * chunk_len, t1 = min(N, t0 + chunk_len);
  constexpr int MAXE = MAXR * D / 256;
  float acc[MAXE];
  float zacc = 0.f;
#pragma unroll
  for (int i = 0; i < MAXE; ++i) acc[i] = 0.f;
  for (int b0 = t0; b0 < t1; b0 += TT) {
    __syncthreads();
    for (int e = threadIdx.x; e < TT * D; e += 256) {
      const int tr = e / D, c = e % D, tok = b0 + tr;
      Ks[tr][c] = tok < t1 ? to_f32(Kh[(long)tok * D + c]) : 0.f;
      Vs[tr][c] = tok < t1 ? to_f32(Vh[(long)tok * D + c]) : 0.f;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < TT * half; e += 256) {
      const int tr = e / half, j = e % half, tok = b0 + tr;
      float ae = 0.f, ao = 0.f;
      for (int c = 0; c < D; ++c) {
        ae = fmaf(to_f32(Ph[(long)(2 * j) * D + c]), Ks[tr][c], ae);
        ao = fmaf(to_f32(Ph[(long)(2 * j + 1) * D + c]), Ks[tr][c], ao);
      }
      float cs = 1.f, sn = 0.f;
      if (tok < t1) { cs = cos_tab[(long)tok * ld + j]; sn = sin_tab[(long)tok * ld + j]; }
      feature_pair<true>(ae, ao, cs, sn, feat);
      kt[tr][2 * j] = ae;
      kt[tr][2 * j + 1] = ao;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < MAXE; ++i) {
      const int e = threadIdx.x + 256 * i;
      if (e < r * D) {
        const int ri = e / D, c = e % D;
        float s = acc[i];
        for (int tr = 0; tr < TT; ++tr) s = fmaf(kt[tr][ri], Vs[tr][c], s);
        acc[i] = s;
      }
    }
    if (threadIdx.x < r)
      for (int tr = 0; tr < TT; ++tr) zacc += kt[tr][threadIdx.x];
  }
  float* P = part + (head * n_chunks + chunk) * (long)(r * D + r);
#pragma unroll
  for (int i = 0; i < MAXE; ++i) {
    const int e = threadIdx.x + 256 * i;
    if (e < r * D) P[e] = acc[i];
  }
  if (threadIdx.x < r) P[(long)r * D + threadIdx.x] = zacc;
}

// C, z = sum over chunks in chunk order (fixed order: reproducible).
__global__ __launch_bounds__(256) void summary_reduce_kernel(int rd, int r, int n_chunks,
                                                             const float* __restrict__ part,
                                                             float* __restrict__ C,
                                                             float* __restrict__ z) {
  const long head = blockIdx.y;
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int per = rd + r;
  if (e >= per) return;
  const float* P = part + head * n_chunks * (long)per + e;
  // chunk order kept; the loads of a batch are all issued before the first add
  constexpr int kBatch = 8;
  float s = 0.f;
  for (int c0 = 0; c0 < n_chunks; c0 += kBatch) {
    float v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) v[u] = P[(long)min(c0 + u, n_chunks - 1) * per];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) s = c0 + u < n_chunks ? s + v[u] : s;
  }
  if (e < rd) C[head * rd + e] = s;
  else if (z) z[head * r + (e - rd)] = s;
}

// ------------------------------------------------------------------------------------------------
// bf16 readout, optionally fused with the gated combine
// ------------------------------------------------------------------------------------------------
constexpr int kReadoutTilesPerWave = 4;  // 16-token tiles per wave per workgroup

template <int JT, bool COMBINE, bool GENERIC>
__global__ __launch_bounds__(256) void readout_mfma_kernel(
    int N, int H, int r, int n_groups, int total, int ld, int feat, const bf16* __restrict__ Qn,
    const bf16* __restrict__ Pq, const float* __restrict__ cos_tab,
    const float* __restrict__ sin_tab, const float* __restrict__ C, float eps_lr,
    const bf16* Os, const float* __restrict__ logits, float eps, bf16* Out) {
  constexpr int D = 128, TPW = kReadoutTilesPerWave;
  const int BH = total / n_groups;
  const int L = xcd_remap(blockIdx.x, total);
  const int head = L % BH, grp = L / BH;
  const int h = head % H, b = head / H;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, lr = lane % 16, g = lane / 16;
  const int half = r / 2;
  const bf16* Qh = Qn + (long)head * N * D;
  const bf16* Ph = Pq + (long)h * r * D;
  const float* Ch = C + (long)head * r * D;

  // A operand of Phi = P Q^T: even / odd rows of P for pair j = 16 jt + lr.
  bf16x8 pe[JT][4], po[JT][4];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt) {
    const int j = 16 * jt + lr;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      if (j < half) {
        pe[jt][kc] = *reinterpret_cast<const bf16x8*>(Ph + (long)(2 * j) * D + 32 * kc + 8 * g);
        po[jt][kc] = *reinterpret_cast<const bf16x8*>(Ph + (long)(2 * j + 1) * D + 32 * kc + 8 * g);
      } else {
        pe[jt][kc] = bf16x8{};
        po[jt][kc] = bf16x8{};
      }
    }
  }
  // A operand of u^T = C^T q~, staged once per workgroup in LDS in the order lanes read it.
  // Fragment (jt, w) row c holds channel 32(w/2) + 8(c/4) + 4(w%2) + c%4, so the output lane
  // (g, token) of tiles 2p and 2p+1 ends up with the 8 consecutive channels 32p + 8g .. +7 (16-byte
  // O^s loads and O stores). Slots 0-3 = even rows 2(16jt+4g+s), slots 4-7 = odd rows. C = hi + lo
  // (two bf16 terms) keeps the contraction accurate to ~2^-16 relative with fp32 accumulation.
  __shared__ bf16x8 cfrag[2][JT * 8 * 64];
  for (int e = tid; e < JT * 8 * 64; e += 256) {
    const int ln = e % 64, w = (e / 64) % 8, jt = e / 512;
    const int c = ln % 16, ch = 32 * (w >> 1) + 8 * (c >> 2) + 4 * (w & 1) + (c & 3), gg = ln / 16;
    bf16x8 hi, lo;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int jj = 16 * jt + 4 * gg + (s & 3);
      const float c = jj < half ? Ch[(long)(2 * jj + (s >> 2)) * D + ch] : 0.f;
      hi[s] = (bf16)c;
      lo[s] = (bf16)(c - (float)hi[s]);
    }
    cfrag[0][e] = hi;
    cfrag[1][e] = lo;
  }
  __syncthreads();

  // Two 16-token tiles per wave at a time: every load of both tiles (Q^n rows, table entries, O^s,
  // gate logits) is issued before either is computed, so HBM sees both tiles' traffic in flight.
  constexpr int TG = 2;
  for (int it0 = 0; it0 < TPW; it0 += TG) {
    bf16x8 qf[TG][4];
    float4 c4[TG][JT], s4[TG][JT];
    bf16x8 osr[TG][4];
    float lg[TG];
    int tokv[TG];
#pragma unroll
    for (int tg = 0; tg < TG; ++tg) {
      const int tok = (grp * 4 * TPW + (it0 + tg) * 4 + wave) * 16 + lr;
      const bool valid = tok < N;
      tokv[tg] = tok;
#pragma unroll
      for (int kc = 0; kc < 4; ++kc)
        qf[tg][kc] = valid ? *reinterpret_cast<const bf16x8*>(Qh + (long)tok * D + 32 * kc + 8 * g)
                           : bf16x8{};
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        const int jb = 16 * jt + 4 * g;  // pairs jb..jb+3 of token `tok`
        c4[tg][jt] = make_float4(1.f, 1.f, 1.f, 1.f);
        s4[tg][jt] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (valid && jb < half) {
          c4[tg][jt] = *reinterpret_cast<const float4*>(cos_tab + (long)tok * ld + jb);
          s4[tg][jt] = *reinterpret_cast<const float4*>(sin_tab + (long)tok * ld + jb);
        }
      }
      if constexpr (COMBINE) {
        const bf16* srow = Os + (long)head * N * D + (long)tok * D;
#pragma unroll
        for (int p = 0; p < 4; ++p)
          osr[tg][p] = valid ? *reinterpret_cast<const bf16x8*>(srow + 32 * p + 8 * g) : bf16x8{};
        lg[tg] = valid ? logits[(long)b * N + tok] : 0.f;
      }
    }
#pragma unroll
    for (int tg = 0; tg < TG; ++tg) {
      const int tok = tokv[tg];
      if (tok - lr >= N) continue;  // whole tile past the end (uniform)
      const bool valid = tok < N;
      f32x4 u[8];
#pragma unroll
      for (int w = 0; w < 8; ++w) u[w] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        f32x4 ye = {0.f, 0.f, 0.f, 0.f}, yo = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
          ye = mfma16x16x32(pe[jt][kc], qf[tg][kc], ye);
          yo = mfma16x16x32(po[jt][kc], qf[tg][kc], yo);
        }
        const float cc[4] = {c4[tg][jt].x, c4[tg][jt].y, c4[tg][jt].z, c4[tg][jt].w};
        const float ss[4] = {s4[tg][jt].x, s4[tg][jt].y, s4[tg][jt].z, s4[tg][jt].w};
        bf16x8 bq, bl;  // q~ = hi + lo
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          float qe = ye[v], qo = yo[v];
          feature_pair<GENERIC>(qe, qo, cc[v], ss[v], feat);
          bq[v] = (bf16)qe;
          bq[4 + v] = (bf16)qo;
          bl[v] = (bf16)(qe - (float)bq[v]);
          bl[4 + v] = (bf16)(qo - (float)bq[4 + v]);
        }
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          const bf16x8 ch = cfrag[0][(jt * 8 + w) * 64 + lane];
          const bf16x8 cl = cfrag[1][(jt * 8 + w) * 64 + lane];
          u[w] = mfma16x16x32(ch, bq, u[w]);
          u[w] = mfma16x16x32(cl, bq, u[w]);
          u[w] = mfma16x16x32(ch, bl, u[w]);
        }
      }
      float ss_u = 0.f;
#pragma unroll
      for (int w = 0; w < 8; ++w)
#pragma unroll
        for (int v = 0; v < 4; ++v) ss_u = fmaf(u[w][v], u[w][v], ss_u);
      const float inv_u = rsqrtf(rows_sum(ss_u) * (1.0f / D) + eps_lr);
      bf16* orow = Out + (long)head * N * D + (long)tok * D;
      // Lane holds channels 32p + 8g + 4h + v in u[2p + h][v].
      if constexpr (COMBINE) {
        float ss_s = 0.f;
#pragma unroll
        for (int p = 0; p < 4; ++p)
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const float x = (float)osr[tg][p][i];
            ss_s = fmaf(x, x, ss_s);
          }
        const float rs = sqrtf(rows_sum(ss_s) * (1.0f / D) + eps);
        // (O^s / r + g O^lr) r  ==  O^s + (g r / rms(u)) u
        const float coef = sigmoid(lg[tg]) * rs * inv_u;
        if (valid) {
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            bf16x8 o;
#pragma unroll
            for (int i = 0; i < 8; ++i)
              o[i] = (bf16)fmaf(coef, u[2 * p + (i >> 2)][i & 3], (float)osr[tg][p][i]);
            *reinterpret_cast<bf16x8*>(orow + 32 * p + 8 * g) = o;
          }
        }
      } else {
        if (valid) {
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            bf16x8 o;
#pragma unroll
            for (int i = 0; i < 8; ++i) o[i] = (bf16)(u[2 * p + (i >> 2)][i & 3] * inv_u);
            *reinterpret_cast<bf16x8*>(orow + 32 * p + 8 * g) = o;
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------------------
// Plain readout (+ combine) for the fp32 path: 32 tokens per workgroup, 8 threads per token.
// ------------------------------------------------------------------------------------------------
template <typename T, int D, bool COMBINE>
__global__ __launch_bounds__(256) void readout_simple_kernel(
    int N, int H, int r, int ld, int feat, const T* __restrict__ Qn, const T* __restrict__ Pq,
    const float* __restrict__ cos_tab, const float* __restrict__ sin_tab,
    const float* __restrict__ C, float eps_lr, const T* Os, const float* __restrict__ logits,
    float eps, T* Out) {
  constexpr int TT = 32, MAXR = 128;
  __shared__ float Cs[MAXR * D];
  __shared__ float Qs[TT][D];
  __shared__ float ft[TT][MAXR];
  const long head = (long)blockIdx.z * gridDim.y + blockIdx.y;
  const int h = blockIdx.y, b = blockIdx.z;
  const int tok0 = blockIdx.x * TT;
  const T* Qh = Qn + head * (long)N * D;
  const T* Ph = Pq + (long)h * r * D;
  const int half = r / 2;
  for (int e = threadIdx.x; e < r * D; e += 256) Cs[e] = C[head * r * D + e];
  for (int e = threadIdx.x; e < TT * D; e += 256) {
    const int tr = e / D, c = e % D, tok = tok0 + tr;
    Qs[tr][c] = tok < N ? to_f32(Qh[(long)tok * D + c]) : 0.f;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < TT * half; e += 256) {
    const int tr = e / half, j = e % half, tok = tok0 + tr;
    float ae = 0.f, ao = 0.f;
    for (int c = 0; c < D; ++c) {
      ae = fmaf(to_f32(Ph[(long)(2 * j) * D + c]), Qs[tr][c], ae);
      ao = fmaf(to_f32(Ph[(long)(2 * j + 1) * D + c]), Qs[tr][c], ao);
    }
    float cs = 1.f, sn = 0.f;
    if (tok < N) { cs = cos_tab[(long)tok * ld + j]; sn = sin_tab[(long)tok * ld + j]; }
    feature_pair<true>(ae, ao, cs, sn, feat);
    ft[tr][2 * j] = ae;
    ft[tr][2 * j + 1] = ao;
  }
  __syncthreads();
  const int tr = threadIdx.x / 8, sub = threadIdx.x % 8, tok = tok0 + tr;
  constexpr int PER = D / 8;
  float u[PER];
  float ss_u = 0.f;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = sub + 8 * k;
    float s = 0.f;
    for (int ri = 0; ri < r; ++ri) s = fmaf(ft[tr][ri], Cs[ri * D + c], s);
    u[k] = s;
    ss_u = fmaf(s, s, ss_u);
  }
  ss_u += __shfl_xor(ss_u, 1);
  ss_u += __shfl_xor(ss_u, 2);
  ss_u += __shfl_xor(ss_u, 4);
  const float inv_u = 1.0f / sqrtf(ss_u / D + eps_lr);
  T* orow = Out + head * (long)N * D + (long)tok * D;
  if constexpr (COMBINE) {
    const T* srow = Os + head * (long)N * D + (long)tok * D;
    float os[PER];
    float ss_s = 0.f;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      os[k] = tok < N ? to_f32(srow[sub + 8 * k]) : 0.f;
      ss_s = fmaf(os[k], os[k], ss_s);
    }
    ss_s += __shfl_xor(ss_s, 1);
    ss_s += __shfl_xor(ss_s, 2);
    ss_s += __shfl_xor(ss_s, 4);
    const float rs = sqrtf(ss_s / D + eps);
    if (tok < N) {
      const float gate = 1.0f / (1.0f + expf(-logits[(long)b * N + tok]));
#pragma unroll
      for (int k = 0; k < PER; ++k)
        orow[sub + 8 * k] = from_f32<T>((os[k] / rs + gate * (u[k] * inv_u)) * rs);
    }
  } else {
    if (tok < N) {
#pragma unroll
      for (int k = 0; k < PER; ++k) orow[sub + 8 * k] = from_f32<T>(u[k] * inv_u);
    }
  }
}

// ------------------------------------------------------------------------------------------------
// Gated combine alone: one row of d_h elements per d_h/8 lanes, 8 elements per lane.
// ------------------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(long rows, int N, int H, int d,
                                                      const T* Os, const T* __restrict__ Olr,
                                                      const float* __restrict__ logits, float eps,
                                                      T* O) {
  const int G = d / 8;
  const long gidx = (long)blockIdx.x * 256 + threadIdx.x;
  const long row = gidx / G;
  const int sub = (int)(gidx % G);
  const bool valid = row < rows;
  float os[8] = {}, ol[8] = {};
  if (valid) {
    load8(Os + row * d + sub * 8, os);
    load8(Olr + row * d + sub * 8, ol);
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) ss = fmaf(os[i], os[i], ss);
  for (int m = 1; m < G; m <<= 1) ss += __shfl_xor(ss, m);
  if (!valid) return;
  const float rs = sqrtf(ss / d + eps);
  const long b = row / ((long)H * N);
  const int n = (int)(row % N);
  const float gate = 1.0f / (1.0f + expf(-logits[b * N + n]));
  float o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = (os[i] / rs + gate * ol[i]) * rs;
  store8(O + row * d + sub * 8, o);
}

// ------------------------------------------------------------------------------------------------
// Features q~ (or k~) of every token, fp32 [B, H, N, r], pairs interleaved: one thread per (token,
// pair), fp32 projection, then feature_pair. Not on the module's path: it exposes the features for
// checks and for the positional metrics of the RoPE-placement study (Sec. 5.1).
// ------------------------------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void features_kernel(long total, int N, int H, int r, int ld,
                                                       int feat, const T* __restrict__ X,
                                                       const T* __restrict__ P,
                                                       const float* __restrict__ cos_tab,
                                                       const float* __restrict__ sin_tab,
                                                       float* __restrict__ F) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int half = r / 2;
  const int j = (int)(i % half);
  const long row = i / half;  // (b, h, token)
  const int tok = (int)(row % N), h = (int)((row / N) % H);
  const T* x = X + row * D;
  const T* pe = P + ((long)h * r + 2 * j) * D;
  const T* po = pe + D;
  float e = 0.f, o = 0.f;
  for (int c = 0; c < D; ++c) {
    const float xc = to_f32(x[c]);
    e = fmaf(to_f32(pe[c]), xc, e);
    o = fmaf(to_f32(po[c]), xc, o);
  }
  feature_pair<true>(e, o, cos_tab[(long)tok * ld + j], sin_tab[(long)tok * ld + j], feat);
  F[row * r + 2 * j] = e;
  F[row * r + 2 * j + 1] = o;
}

template <int JT, bool GENERIC>
hipError_t summary_mfma(const Shape& s, const void* Kn, const void* V, const void* Pk, int r,
                        const float* ct, const float* st_, int ld, int feat, float* part,
                        int chunk_len, int n_chunks, hipStream_t st) {
  const int total = s.B * s.H * n_chunks;
  const int split = r > 32 * JT ? 2 : 1;  // r = 128 on the two-tile kernel
  const unsigned grid = split == 2 ? (unsigned)((total + 7) / 8 * 16) : (unsigned)total;
  hipLaunchKernelGGL((summary_mfma_kernel<JT, GENERIC>), dim3(grid), dim3(256), 0, st, s.N, s.H,
                     r, chunk_len, n_chunks, total, split, ld, feat, (const bf16*)Kn,
                     (const bf16*)V, (const bf16*)Pk, ct, st_, part);
  return hipGetLastError();
}

template <int JT>
hipError_t summary_mfma_feat(const Shape& s, const void* Kn, const void* V, const void* Pk, int r,
                             const float* ct, const float* st_, int ld, int feat, float* part,
                             int chunk_len, int n_chunks, hipStream_t st) {
  if (feat == 0)
    return summary_mfma<JT, false>(s, Kn, V, Pk, r, ct, st_, ld, feat, part, chunk_len, n_chunks, st);
  return summary_mfma<JT, true>(s, Kn, V, Pk, r, ct, st_, ld, feat, part, chunk_len, n_chunks, st);
}

template <int JT, bool COMBINE, bool GENERIC>
hipError_t readout_mfma(const Shape& s, const void* Qn, const void* Pq, int r, const float* ct,
                        const float* st_, int ld, int feat, const float* C, float eps_lr,
                        const void* Os, const float* logits, float eps, void* Out, hipStream_t st) {
  const int per_group = 4 * kReadoutTilesPerWave * 16;
  const int n_groups = (s.N + per_group - 1) / per_group;
  const int total = s.B * s.H * n_groups;
  hipLaunchKernelGGL((readout_mfma_kernel<JT, COMBINE, GENERIC>), dim3(total), dim3(256), 0, st,
                     s.N, s.H, r, n_groups, total, ld, feat, (const bf16*)Qn, (const bf16*)Pq, ct,
                     st_, C, eps_lr, (const bf16*)Os, logits, eps, (bf16*)Out);
  return hipGetLastError();
}

template <int JT, bool COMBINE>
hipError_t readout_mfma_feat(const Shape& s, const void* Qn, const void* Pq, int r,
                             const float* ct, const float* st_, int ld, int feat, const float* C,
                             float eps_lr, const void* Os, const float* logits, float eps,
                             void* Out, hipStream_t st) {
  if (feat == 0)
    return readout_mfma<JT, COMBINE, false>(s, Qn, Pq, r, ct, st_, ld, feat, C, eps_lr, Os, logits,
                                            eps, Out, st);
  return readout_mfma<JT, COMBINE, true>(s, Qn, Pq, r, ct, st_, ld, feat, C, eps_lr, Os, logits,
                                         eps, Out, st);
}

template <bool COMBINE>
hipError_t readout_dispatch(const Shape& s, const void* Qn, const void* Pq, int r, const float* ct,
                            const float* st_, int ld, int feat, const float* C, float eps_lr,
                            const void* Os, const float* logits, float eps, void* Out,
                            hipStream_t st) {
  if (s.bf16) {
    if (r <= 32)
      return readout_mfma_feat<1, COMBINE>(s, Qn, Pq, r, ct, st_, ld, feat, C, eps_lr, Os, logits,
                                           eps, Out, st);
    if (r <= 64)
      return readout_mfma_feat<2, COMBINE>(s, Qn, Pq, r, ct, st_, ld, feat, C, eps_lr, Os, logits,
                                           eps, Out, st);
    return readout_mfma_feat<4, COMBINE>(s, Qn, Pq, r, ct, st_, ld, feat, C, eps_lr, Os, logits,
                                         eps, Out, st);
  }
  const dim3 grid((s.N + 31) / 32, s.H, s.B);
  if (s.d == 64)
    hipLaunchKernelGGL((readout_simple_kernel<float, 64, COMBINE>), grid, dim3(256), 0, st, s.N,
                       s.H, r, ld, feat, (const float*)Qn, (const float*)Pq, ct, st_, C, eps_lr,
                       (const float*)Os, logits, eps, (float*)Out);
  else
    hipLaunchKernelGGL((readout_simple_kernel<float, 128, COMBINE>), grid, dim3(256), 0, st, s.N,
                       s.H, r, ld, feat, (const float*)Qn, (const float*)Pq, ct, st_, C, eps_lr,
                       (const float*)Os, logits, eps, (float*)Out);
  return hipGetLastError();
}

}  // namespace

int summary_chunks(const Shape& s, int r) {
  (void)r;
  const int len = summary_chunk_len(s);
  return (s.N + len - 1) / len;
}

size_t summary_workspace_bytes(const Shape& s, int r) {
  return (size_t)s.B * s.H * summary_chunks(s, r) * (size_t)(r * s.d + r) * sizeof(float);
}

hipError_t launch_lowrank_summary(const Shape& s, const void* Kn, const void* V, const void* Pk,
                                  int r, const float* cos_tab, const float* sin_tab, int ld,
                                  int feat, float* C, float* z, void* ws, hipStream_t st) {
  const int chunk_len = summary_chunk_len(s);
  const int n_chunks = (s.N + chunk_len - 1) / chunk_len;
  float* part = (float*)ws;
  hipError_t e;
  if (s.bf16) {
    if (r <= 32)
      e = summary_mfma_feat<1>(s, Kn, V, Pk, r, cos_tab, sin_tab, ld, feat, part, chunk_len,
                               n_chunks, st);
    else if (r <= 64)
      e = summary_mfma_feat<2>(s, Kn, V, Pk, r, cos_tab, sin_tab, ld, feat, part, chunk_len,
                               n_chunks, st);
    else  // r = 128: two workgroups of two pair tiles each per chunk
      e = summary_mfma_feat<2>(s, Kn, V, Pk, r, cos_tab, sin_tab, ld, feat, part, chunk_len,
                               n_chunks, st);
  } else {
    const dim3 grid(n_chunks, s.H, s.B);
    if (s.d == 64)
      hipLaunchKernelGGL((summary_simple_kernel<float, 64>), grid, dim3(256), 0, st, s.N, s.H, r,
                         chunk_len, n_chunks, ld, feat, (const float*)Kn, (const float*)V,
                         (const float*)Pk, cos_tab, sin_tab, part);
    else
      hipLaunchKernelGGL((summary_simple_kernel<float, 128>), grid, dim3(256), 0, st, s.N, s.H, r,
                         chunk_len, n_chunks, ld, feat, (const float*)Kn, (const float*)V,
                         (const float*)Pk, cos_tab, sin_tab, part);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  const int per = r * s.d + r;
  hipLaunchKernelGGL(summary_reduce_kernel, dim3((per + 255) / 256, s.B * s.H), dim3(256), 0, st,
                     r * s.d, r, n_chunks, part, C, z);
  return hipGetLastError();
}

hipError_t launch_lowrank_readout(const Shape& s, const void* Qn, const void* Pq, int r,
                                  const float* cos_tab, const float* sin_tab, int ld, int feat,
                                  const float* C, float eps_lr, const void* Os,
                                  const float* logits, float eps, void* Out, hipStream_t st) {
  if (Os)
    return readout_dispatch<true>(s, Qn, Pq, r, cos_tab, sin_tab, ld, feat, C, eps_lr, Os, logits,
                                  eps, Out, st);
  return readout_dispatch<false>(s, Qn, Pq, r, cos_tab, sin_tab, ld, feat, C, eps_lr, nullptr,
                                 nullptr, 0.f, Out, st);
}

hipError_t launch_lowrank_features(const Shape& s, const void* X, const void* P, int r,
                                   const float* cos_tab, const float* sin_tab, int ld, int feat,
                                   float* F, hipStream_t st) {
  const long total = (long)s.B * s.H * s.N * (r / 2);
  const dim3 grid((unsigned)((total + 255) / 256));
  if (s.bf16) {
    if (s.d == 64)
      hipLaunchKernelGGL((features_kernel<bf16, 64>), grid, dim3(256), 0, st, total, s.N, s.H, r,
                         ld, feat, (const bf16*)X, (const bf16*)P, cos_tab, sin_tab, F);
    else
      hipLaunchKernelGGL((features_kernel<bf16, 128>), grid, dim3(256), 0, st, total, s.N, s.H, r,
                         ld, feat, (const bf16*)X, (const bf16*)P, cos_tab, sin_tab, F);
  } else {
    if (s.d == 64)
      hipLaunchKernelGGL((features_kernel<float, 64>), grid, dim3(256), 0, st, total, s.N, s.H, r,
                         ld, feat, (const float*)X, (const float*)P, cos_tab, sin_tab, F);
    else
      hipLaunchKernelGGL((features_kernel<float, 128>), grid, dim3(256), 0, st, total, s.N, s.H, r,
                         ld, feat, (const float*)X, (const float*)P, cos_tab, sin_tab, F);
  }
  return hipGetLastError();
}

hipError_t launch_combine(const Shape& s, const void* Os, const void* Olr, const float* logits,
                          float eps, void* O, hipStream_t st) {
  const long rows = (long)s.B * s.H * s.N;
  const long threads = rows * (s.d / 8);
  const dim3 grid((unsigned)((threads + 255) / 256));
  if (s.bf16)
    hipLaunchKernelGGL(combine_kernel<bf16>, grid, dim3(256), 0, st, rows, s.N, s.H, s.d,
                       (const bf16*)Os, (const bf16*)Olr, logits, eps, (bf16*)O);
  else
    hipLaunchKernelGGL(combine_kernel<float>, grid, dim3(256), 0, st, rows, s.N, s.H, s.d,
                       (const float*)Os, (const float*)Olr, logits, eps, (float*)O);
  return hipGetLastError();
}

}  // namespace rola
