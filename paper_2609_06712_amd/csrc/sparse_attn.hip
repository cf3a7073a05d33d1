// Block-sparse softmax attention of the sparse branch (Algorithm step 4; attention as in Sec. 3):
// every query block attends to the valid tokens of its `keep` selected key blocks, by online
// softmax with fp32 running max / sum / accumulators. With no index list every key block is walked
// in order, which is dense softmax attention (the 0 % sparsity reference).
//
// bf16 path (d_h = 128): one workgroup per (b, h, query block of BLK tokens), BLK/32 waves of 32
// queries (two 16-query MFMA tiles) each, Q fragments in registers. Keys stream in 32-key sub-tiles:
//   S^T = K Q^T     v_mfma_f32_16x16x32_bf16, A = K sub-tile from LDS, B = Q fragments; lane
//                   (g = lane/16, c = lane%16) receives keys 4g+v of each 16-key tile for query c,
//                   so softmax statistics stay per lane (row max: two permlane swaps).
//   P = exp2(S^T * scale*log2e - m), rounded to bf16 in registers: directly the B operand of
//   O^T = V^T P^T   A = V^T: V stays row-major in LDS and is read with the gfx950 transposing LDS read
//                   ds_read_b64_tr_b16, which hands lane i of each 16-lane group channel i of 4
//                   consecutive keys -- exactly the MFMA operand layout.
// Row sums come from one more MFMA against a ones operand. Sub-tiles are double-buffered in LDS and
// filled by direct global-to-LDS loads (global_load_lds_dwordx4): no staging registers. The 16-byte
// chunks of every row are XOR-swizzled (K: chunk ^ row%16, V: chunk ^ 2(row%8)) so that the K
// operand reads (16 rows per cycle) and the transposing V reads (8 rows per cycle) are free of
// bank conflicts. O is rescaled only when a sub-tile raises a row max by more than 2^8: the softmax
// ratio does not depend on the reference max, so this is exact. The grid is remapped so that
// consecutive query blocks of one head run on the same XCD (sharing its L2).
#include "common.h"
#include "launch.h"

#ifndef ROLA_B128_NBUF
#define ROLA_B128_NBUF 2  // LDS stages of the 128-token-block kernel with a block list
#endif
#ifndef ROLA_SPARSE_REMAP
#define ROLA_SPARSE_REMAP 1  // 1: XCD-contiguous logical ranges; 2: interleaved chunks; 0: none
#endif

namespace rola {
namespace {

__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// bf16 kernel, pipelined: one workgroup per (b, h, query block of BLK tokens) with BLK/32 waves of
// 32 queries each; keys stream in 32-key sub-tiles (two or four per selected block) that are
// double-buffered in LDS and filled by direct global-to-LDS loads (global_load_lds_dwordx4), so no
// registers stage them. Rows are stored with their 16-byte chunks XOR-swizzled (K: chunk ^ row%16,
// V: chunk ^ 2(row%8)), which makes both the K operand reads (ds_read_b128, 16 rows per cycle) and
// the transposing V reads (ds_read_b64_tr_b16, 8 rows per cycle) bank-conflict free.
// Online softmax keeps a per-query reference max and rescales O only when a new tile raises the max
// by more than 2^8: the softmax ratio is independent of the reference, so this is exact.
constexpr int kSub = 32;          // keys per sub-tile
constexpr float kRescaleTau = 8.f;  // log2 headroom before O is rescaled

template <int BLK, int NBUF>
__global__ __launch_bounds__(BLK * 2, 2) void sparse_pipe_kernel(
    int N, int nb, int keep, int total, const int32_t* __restrict__ idx, float scale_log2,
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    bf16* __restrict__ O) {
  constexpr int D = 128, NW = BLK / 32, QT = 2;
  constexpr int TILE_BYTES = kSub * D * 2;              // 8 KB
  constexpr int DMA_PER_WAVE = TILE_BYTES / 1024 / NW;  // 1 KB instructions per wave per tensor
  constexpr int SUBS = BLK / kSub;                     // sub-tiles per selected block
  constexpr int BUF_BYTES = 2 * TILE_BYTES;            // K then V
  __shared__ __attribute__((aligned(1024))) char lds[NBUF * BUF_BYTES];

  const int L = ROLA_SPARSE_REMAP == 2 ? xcd_chunk_remap(blockIdx.x, total, (nb + kNumXcd - 1) / kNumXcd)
              : ROLA_SPARSE_REMAP ? xcd_remap(blockIdx.x, total) : (int)blockIdx.x;
  const int I = L % nb;
  const long head = L / nb;
  const int tid = threadIdx.x, lane = tid % 64, lr = lane % 16, g = lane / 16;
  const int wave = wave_uniform(tid / 64);  // wave-uniform: LDS DMA bases in SGPRs
  const bf16* Qh = Q + head * (long)N * D;
  const char* Kh = reinterpret_cast<const char*>(K + head * (long)N * D);
  const char* Vh = reinterpret_cast<const char*>(V + head * (long)N * D);
  bf16* Oh = O + head * (long)N * D;
  const int32_t* sel = idx ? idx + (head * nb + I) * (long)keep : nullptr;
  const int steps = keep * SUBS;

  bf16x8 qf[QT][4];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int q = I * BLK + (wave * QT + qt) * 16 + lr;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
      qf[qt][kc] = q < N ? *reinterpret_cast<const bf16x8*>(Qh + (long)q * D + 32 * kc + 8 * g)
                         : bf16x8{};
  }
  f32x4 acc[QT][8], accl[QT];  // O^T tiles and the row sums (all four rows of accl are equal)
  float m[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m[qt] = -INFINITY;
    accl[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 8; ++w) acc[qt][w] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (bf16)1.0f;

  // Per-lane constant offsets. DMA: lane l of 1-KB slot q fills row 4q + l/16, position l%16 with
  // source chunk (position ^ swizzle(row)). Reads: K operand of (kt, kc) and V^T operand of w.
  int dk[DMA_PER_WAVE], dv[DMA_PER_WAVE], drow[DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < DMA_PER_WAVE; ++i) {
    const int q = wave * DMA_PER_WAVE + i, row = 4 * q + lane / 16, pos = lane % 16;
    drow[i] = row;
    dk[i] = row * D * 2 + ((pos ^ (row & 15)) << 4);
    dv[i] = row * D * 2 + ((pos ^ ((row & 7) << 1)) << 4);
  }
  int ko[2][4];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      const int row = 16 * kt + lr;
      ko[kt][kc] = row * 256 + (((4 * kc + g) ^ (row & 15)) << 4);
    }
  const int sp = lr >> 2, mp = lr & 3, vr = 4 * g + sp;
  int vo[8];
#pragma unroll
  for (int w = 0; w < 8; ++w)
    vo[w] = TILE_BYTES + vr * 256 + (((2 * w + (mp >> 1)) ^ ((vr & 7) << 1)) << 4) + ((mp & 1) << 3);

  // The block list is read through the constant address space: uniform scalar loads, counted by
  // lgkmcnt, so reading an index never drains the DMA loads in flight (vmcnt).
  typedef const __attribute__((address_space(4))) int32_t* const_i32;
  const const_i32 sel_s = (const_i32)sel;
  auto step_key0 = [&](int t) {  // first key of step t; -1 if its block index is out of range
    const int J = sel ? sel_s[t / SUBS] : t / SUBS;
    return (unsigned)J < (unsigned)nb ? J * BLK + (t % SUBS) * kSub : -1;
  };
  typedef __attribute__((address_space(3))) void lds_void;
  auto issue = [&](int t, int buf) {  // always DMA_PER_WAVE * 2 instructions (fixed vmcnt per step)
    const int k0 = max(step_key0(t), 0);
    char* dst = lds + buf * BUF_BYTES;
    if (k0 + kSub <= N) {
      const char* kb = Kh + (long)k0 * D * 2;
      const char* vb = Vh + (long)k0 * D * 2;
#pragma unroll
      for (int i = 0; i < DMA_PER_WAVE; ++i) {
        const int q = wave * DMA_PER_WAVE + i;
        __builtin_amdgcn_global_load_lds((const void*)(kb + dk[i]), (lds_void*)(dst + q * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds((const void*)(vb + dv[i]), (lds_void*)(dst + TILE_BYTES + q * 1024), 16, 0, 0);
      }
    } else {  // tail: rows past N re-read row N-1 (finite data, masked out of the softmax)
#pragma unroll
      for (int i = 0; i < DMA_PER_WAVE; ++i) {
        const int q = wave * DMA_PER_WAVE + i;
        const long shift = (long)(min(k0 + drow[i], N - 1) - drow[i]) * D * 2;
        __builtin_amdgcn_global_load_lds((const void*)(Kh + shift + dk[i]), (lds_void*)(dst + q * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds((const void*)(Vh + shift + dv[i]), (lds_void*)(dst + TILE_BYTES + q * 1024), 16, 0, 0);
      }
    }
  };

  auto compute = [&](const char* base, int k0) {
    f32x4 s[QT][2];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) s[qt][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
    bf16x8 kfr[4][2];  // all K operands of the step first, then four independent MFMA chains
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) kfr[kc][kt] = *reinterpret_cast<const bf16x8*>(base + ko[kt][kc]);
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        s[qt][0] = mfma16x16x32(kfr[kc][0], qf[qt][kc], s[qt][0]);
        s[qt][1] = mfma16x16x32(kfr[kc][1], qf[qt][kc], s[qt][1]);
      }
    if (k0 + kSub > N) {
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (k0 + 16 * kt + 4 * g + v >= N) s[qt][kt][v] = -INFINITY;
    }
    bf16x8 pb[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float mx = fmaxf(fmaxf(fmaxf(s[qt][0][0], s[qt][0][1]), fmaxf(s[qt][0][2], s[qt][0][3])),
                       fmaxf(fmaxf(s[qt][1][0], s[qt][1][1]), fmaxf(s[qt][1][2], s[qt][1][3])));
      const float mt = rows_max(mx) * scale_log2;
      if (__any(mt > m[qt] + kRescaleTau)) {
        const float mnew = fmaxf(m[qt], mt);
        const float alpha = __builtin_amdgcn_exp2f(m[qt] - mnew);
        m[qt] = mnew;
        accl[qt] *= alpha;
#pragma unroll
        for (int w = 0; w < 8; ++w) acc[qt][w] *= alpha;
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          pb[qt][4 * kt + v] = (bf16)__builtin_amdgcn_exp2f(fmaf(s[qt][kt][v], scale_log2, -m[qt]));
      accl[qt] = mfma16x16x32(ones, pb[qt], accl[qt]);
    }
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    bf16x8 vfr[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + vo[w]));
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(base + vo[w] + 16 * 256));
      vfr[w] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
#pragma unroll
    for (int w = 0; w < 8; ++w)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) acc[qt][w] = mfma16x16x32(vfr[w], pb[qt], acc[qt][w]);
  };

  // Step t computes buffer t % NBUF while the loads of the next NBUF-1 steps fill the others. The
  // loop is unrolled by NBUF so each buffer's base is a compile-time offset.
  constexpr int PER_STEP = 2 * DMA_PER_WAVE;  // vector-memory instructions this wave issues per step
  auto run_step = [&](int t, int buf) {
    if (t + NBUF - 1 <= steps) {  // loads of steps t+1 .. t+NBUF-2 may stay in flight
      constexpr int allowed = PER_STEP * (NBUF - 2);
      __builtin_amdgcn_s_waitcnt((allowed & 15) | ((allowed >> 4) << 14) | (7 << 4) | (15 << 8));
    } else {
      __builtin_amdgcn_s_waitcnt(0);
    }
    __syncthreads();  // everyone's loads of step t landed; step t-1 is done with its buffer
    if (t + NBUF - 1 < steps) issue(t + NBUF - 1, (buf + NBUF - 1) % NBUF);
    const int k0 = step_key0(t);
    if (k0 >= 0 && k0 < N) compute(lds + buf * BUF_BYTES, k0);
  };
#pragma unroll
  for (int j = 0; j < NBUF - 1; ++j)
    if (j < steps) issue(j, j);
  for (int t = 0; t < steps; t += NBUF) {
#pragma unroll
    for (int j = 0; j < NBUF; ++j)
      if (t + j < steps) run_step(t + j, j);
  }

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float inv = 1.0f / accl[qt][0];
    const int q = I * BLK + (wave * QT + qt) * 16 + lr;
    if (q < N) {
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        bf16x4 o;
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = (bf16)(acc[qt][w][v] * inv);
        *reinterpret_cast<bf16x4*>(Oh + (long)q * D + 16 * w + 4 * g) = o;
      }
    }
  }
}

// Plain kernel for the fp32 path: one thread per query, keys streamed through LDS 32 at a time.
template <typename T, int D>
__global__ __launch_bounds__(128) void sparse_simple_kernel(int N, int block, int nb, int keep,
                                                            const int32_t* __restrict__ idx,
                                                            float scale, const T* __restrict__ Q,
                                                            const T* __restrict__ K,
                                                            const T* __restrict__ V,
                                                            T* __restrict__ O) {
  constexpr int KC = 32;
  __shared__ float Ks[KC][D];
  __shared__ float Vs[KC][D];
  const int I = blockIdx.x;
  const long head = (long)blockIdx.z * gridDim.y + blockIdx.y;
  const T* Qh = Q + head * (long)N * D;
  const T* Kh = K + head * (long)N * D;
  const T* Vh = V + head * (long)N * D;
  const int32_t* sel = idx ? idx + (head * nb + I) * (long)keep : nullptr;
  const int p = I * block + threadIdx.x;
  const bool valid = threadIdx.x < block && p < N;
  float q[D], o[D];
#pragma unroll
  for (int c = 0; c < D; ++c) { q[c] = valid ? to_f32(Qh[(long)p * D + c]) : 0.f; o[c] = 0.f; }
  float m = -INFINITY, l = 0.f;
  for (int t = 0; t < keep; ++t) {
    const int J = sel ? sel[t] : t;
    if ((unsigned)J >= (unsigned)nb) continue;  // out-of-range entry: skipped
    const int k0 = J * block, k1 = min(N, k0 + block);
    for (int c0 = k0; c0 < k1; c0 += KC) {
      const int cn = min(KC, k1 - c0);
      __syncthreads();
      for (int e = threadIdx.x; e < KC * D; e += blockDim.x) {
        const int r = e / D, c = e % D;
        Ks[r][c] = r < cn ? to_f32(Kh[(long)(c0 + r) * D + c]) : 0.f;
        Vs[r][c] = r < cn ? to_f32(Vh[(long)(c0 + r) * D + c]) : 0.f;
      }
      __syncthreads();
      float s[KC];
      float mx = m;
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        float a = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) a = fmaf(q[c], Ks[j][c], a);
        s[j] = j < cn ? a * scale : -INFINITY;
        mx = fmaxf(mx, s[j]);
      }
      const float alpha = expf(m - mx);
      l *= alpha;
#pragma unroll
      for (int c = 0; c < D; ++c) o[c] *= alpha;
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        const float w = expf(s[j] - mx);
        l += w;
#pragma unroll
        for (int c = 0; c < D; ++c) o[c] = fmaf(w, Vs[j][c], o[c]);
      }
      m = mx;
    }
  }
  if (valid) {
    const float inv = 1.0f / l;
#pragma unroll
    for (int c = 0; c < D; ++c) O[head * (long)N * D + (long)p * D + c] = from_f32<T>(o[c] * inv);
  }
}

template <int BLK, int NBUF>
hipError_t launch_pipe(const Shape& s, const void* Qr, const void* Kr, const void* V, int keep,
                       const int32_t* idx, float scale, void* Os, hipStream_t st) {
  const int nb = num_blocks(s.N, BLK);
  const int total = nb * s.H * s.B;
  hipLaunchKernelGGL((sparse_pipe_kernel<BLK, NBUF>), dim3(total), dim3(BLK * 2), 0, st, s.N, nb, keep,
                     total, idx, scale * 1.4426950408889634f, (const bf16*)Qr, (const bf16*)Kr,
                     (const bf16*)V, (bf16*)Os);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_simple(const Shape& s, const void* Qr, const void* Kr, const void* V, int block,
                         int keep, const int32_t* idx, float scale, void* Os, hipStream_t st) {
  const int nb = num_blocks(s.N, block);
  hipLaunchKernelGGL((sparse_simple_kernel<T, D>), dim3(nb, s.H, s.B), dim3(block), 0, st, s.N,
                     block, nb, keep, idx, scale, (const T*)Qr, (const T*)Kr, (const T*)V, (T*)Os);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_attn(const Shape& s, const void* Qr, const void* Kr, const void* V,
                              int block, int keep, const int32_t* idx, float scale, void* Os,
                              hipStream_t st) {
  if (s.bf16) {
    // Three LDS stages for gathered blocks (latency of scattered K/V reads); the dense walk, whose
    // reads are L2-friendly, keeps two stages and the higher occupancy.
    if (block == 64)
      return idx ? launch_pipe<64, 3>(s, Qr, Kr, V, keep, idx, scale, Os, st)
                 : launch_pipe<64, 2>(s, Qr, Kr, V, keep, idx, scale, Os, st);
    return idx ? launch_pipe<128, ROLA_B128_NBUF>(s, Qr, Kr, V, keep, idx, scale, Os, st)
               : launch_pipe<128, 2>(s, Qr, Kr, V, keep, idx, scale, Os, st);
  }
  if (s.d == 64) return launch_simple<float, 64>(s, Qr, Kr, V, block, keep, idx, scale, Os, st);
  return launch_simple<float, 128>(s, Qr, Kr, V, block, keep, idx, scale, Os, st);
}

}  // namespace rola
