// Block selection of the sparse branch (Algorithm step 4): mean-pool rotated Q/K per block of
// tokens, score every (query block, key block) pair with an fp32 dot product, keep the top-k key
// blocks of every query block (ties to the lower index), written ascending.
//
//   pool_kernel   HBM-bound: reads Q^r and K^r once (coalesced 16-byte loads), writes means (fp32);
//                 its rotating form reads Q^n or K^n instead, rotates each row (writing K^r) and
//                 pools the rotated values: the backbone rotation and the pooling in one pass.
//   score_kernel  per (b, h): S = q_bar k_bar^T, a small GEMM tiled 128 x 128 through LDS, fp32-accurate
//                 from bf16 MFMA with each operand split into three bf16 terms. The positive
//                 factor 1/sqrt(d_h) is left out: it cannot change the ranking.
//   topk_reg_kernel  one wave per score row, the row's order-preserving uint32 keys in registers:
//                 the k-th largest key found bit by bit from the top with ballot/popcount counts,
//                 then an ascending ballot/popcount compaction. Integer work, bit-reproducible.
//                 Rows of more than 2560 blocks take topk_kernel (4-pass 8-bit radix select with
//                 the keys and histograms in LDS).
#include "common.h"
#include "launch.h"

namespace rola {
namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Block means of Q^r or K^r, one workgroup per (b, h, block), 16 threads of 8 channels per token
// row. Summation order: per thread over its tokens in order, then over the 16 threads in order.
// Sum of x over the G consecutive lanes that share one row (G = 8 or 16, lanes aligned to G).
__device__ __forceinline__ float row_group_sum(float x, int G) {
  for (int off = G / 2; off >= 1; off >>= 1) x += __shfl_xor(x, off, G);
  return x;
}

// *out = sqrt of the largest sq over the workgroup's 256 threads (every thread calls it).
__device__ __forceinline__ void block_norm_max(float sq, float* out) {
  __shared__ float wmax[4];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) sq = fmaxf(sq, __shfl_xor(sq, off));
  if (threadIdx.x % 64 == 0) wmax[threadIdx.x / 64] = sq;
  __syncthreads();
  if (threadIdx.x == 0)
    *out = sqrtf(fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3])));
}

template <typename T>
__global__ __launch_bounds__(256) void pool_kernel(int N, int d, int block, const T* __restrict__ X,
                                                   float* __restrict__ out, float* __restrict__ nmax) {
  const int I = blockIdx.x, nb = gridDim.x;
  const long head = (long)blockIdx.z * gridDim.y + blockIdx.y;
  const T* xh = X + head * (long)N * d;
  const int G = d / 8, L = 256 / G;
  const int g = threadIdx.x % G, lane = threadIdx.x / G;
  const int n0 = I * block, n1 = min(N, n0 + block);
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  float sq = 0.f;  // largest squared row norm among this thread's rows (its G-lane share)
  // Rows in batches of kPoolRows per thread, every load of a batch issued before the first is
  // used (one row at a time, each load waited for before the next is issued, made every
  // workgroup four serial memory round trips). Rows past n1 re-read row n1 - 1 and are left out
  // by selects, so the batch has no branch between its loads and the sums are the row-by-row ones.
  constexpr int kPoolRows = 4;
  for (int nb0 = n0 + lane; nb0 < n1; nb0 += kPoolRows * L) {
    float v[kPoolRows][8];
#pragma unroll
    for (int r = 0; r < kPoolRows; ++r) load8(xh + (long)min(nb0 + r * L, n1 - 1) * d + g * 8, v[r]);
#pragma unroll
    for (int r = 0; r < kPoolRows; ++r) {
      const bool ok = nb0 + r * L < n1;  // the same for the G lanes of a row
      float part = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        acc[i] = ok ? acc[i] + v[r][i] : acc[i];
        part = fmaf(v[r][i], v[r][i], part);
      }
      if (nmax) {
        const float rs = row_group_sum(part, G);
        sq = ok ? fmaxf(sq, rs) : sq;
      }
    }
  }
  __shared__ float red[256 * 8];
#pragma unroll
  for (int i = 0; i < 8; ++i) red[threadIdx.x * 8 + i] = acc[i];
  __syncthreads();
  if (threadIdx.x < d) {
    const int c = threadIdx.x, gc = c / 8, ic = c % 8;
    float s = 0.f;
    for (int l = 0; l < L; ++l) s += red[(l * G + gc) * 8 + ic];
    out[(head * nb + I) * d + c] = s / (float)(n1 - n0);
  }
  if (nmax) block_norm_max(sq, nmax + head * nb + I);
}

// The rotating form (d_h = 128): X is Q^n or K^n. One workgroup per (block, group of HG heads): the
// block's rotary-table entries are loaded into registers once and serve every head of the group
// (the tables are twice the bytes of an activation row, so reading them per head would triple the
// traffic). Each row is rotated (rope_pair, as rola_rope_apply), rounded to T, written to Xr unless
// Xr is null, and pooled as rounded, in pool_kernel's thread layout and order: the means are
// bitwise pool_kernel's over Xr. TPT = block / 16 tokens per thread.
constexpr int kRopePoolHeads = 8;
template <typename T, int TPT>
__global__ __launch_bounds__(256) void rope_pool_kernel(int N, int block, int heads, int ld,
                                                        const T* __restrict__ X,
                                                        const float* __restrict__ cos_tab,
                                                        const float* __restrict__ sin_tab,
                                                        T* __restrict__ Xr, float* __restrict__ out,
                                                        float* __restrict__ nmax) {
  constexpr int D = 128, G = D / 8, L = 256 / G;
  const int I = blockIdx.x, nb = gridDim.x;
  const int h0 = blockIdx.y * kRopePoolHeads, h1 = min(heads, h0 + kRopePoolHeads);
  const int g = threadIdx.x % G, lane = threadIdx.x / G;
  const int n0 = I * block, n1 = min(N, n0 + block);
  float cc[TPT][4], ss[TPT][4];
#pragma unroll
  for (int k = 0; k < TPT; ++k) {
    const int n = min(n0 + lane + L * k, n1 - 1);  // rows past the block are not pooled
    const float4 c = *reinterpret_cast<const float4*>(cos_tab + (long)n * ld + g * 4);
    const float4 sn = *reinterpret_cast<const float4*>(sin_tab + (long)n * ld + g * 4);
    cc[k][0] = c.x; cc[k][1] = c.y; cc[k][2] = c.z; cc[k][3] = c.w;
    ss[k][0] = sn.x; ss[k][1] = sn.y; ss[k][2] = sn.z; ss[k][3] = sn.w;
  }
  __shared__ float red[256 * 8];
  for (int head = h0; head < h1; ++head) {
    const T* xh = X + (long)head * N * D;
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    float sq = 0.f;  // largest squared norm of a rotated, rounded row (this thread's share of it)
    float v[TPT][8];
#pragma unroll
    for (int k = 0; k < TPT; ++k)  // loads first, none under a branch: one memory latency per head
      load8(xh + (long)min(n0 + lane + L * k, n1 - 1) * D + g * 8, v[k]);  // rows past n1 unused
#pragma unroll
    for (int k = 0; k < TPT; ++k) {
      const int n = n0 + lane + L * k;
      if (n < n1) {
        T r[8];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          float x, y;
          rope_pair(v[k][2 * p], v[k][2 * p + 1], cc[k][p], ss[k][p], x, y);
          r[2 * p] = from_f32<T>(x);
          r[2 * p + 1] = from_f32<T>(y);
        }
        float o[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = to_f32(r[i]);
        if (Xr) store8(Xr + (long)head * N * D + (long)n * D + g * 8, o);
        float part = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          acc[i] += o[i];
          part = fmaf(o[i], o[i], part);
        }
        if (nmax) sq = fmaxf(sq, row_group_sum(part, G));
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) red[threadIdx.x * 8 + i] = acc[i];
    __syncthreads();
    if (threadIdx.x < D) {
      const int c = threadIdx.x, gc = c / 8, ic = c % 8;
      float s = 0.f;
      for (int l = 0; l < L; ++l) s += red[(l * G + gc) * 8 + ic];
      out[((long)head * nb + I) * D + c] = s / (float)(n1 - n0);
    }
    if (nmax) block_norm_max(sq, nmax + (long)head * nb + I);
    __syncthreads();
  }
}

// S[I][J] = sum_c qbar[I][c] * kbar[J][c] for one (b, h) per blockIdx.z, with fp32 accuracy (the
// 1e-4 tie gap of the selection rules out plain bf16 operands) from bf16 MFMA products:
// x = hi + mid + lo exactly: each term is the remainder of the ones before, rounded to bf16 (eight
// significant bits each, and each remainder is exact in fp32). Dropping the three products of two
// lower terms (mid lo, lo mid, lo lo: about 2^-24 of hi hi) leaves six bf16 MFMA products whose fp32
// sum is as accurate as an fp32 dot product, at 16x the fp32 MFMA rate per product.
__device__ __forceinline__ void split3(const float (&x)[8], bf16x8& hi, bf16x8& mid, bf16x8& lo) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    hi[i] = (bf16)x[i];
    const float r1 = x[i] - (float)hi[i];
    mid[i] = (bf16)r1;
    lo[i] = (bf16)(r1 - (float)mid[i]);
  }
}

// 128 x 128 tile of S per workgroup, four waves of 64 x 64. Each chunk of 32 channels is split
// into the three bf16 terms once, in LDS (the split costs a workgroup about half as much vector
// work per product as a 64 x 64 tile would, and each mean crosses L2 half as often); the next
// chunk's loads are in flight while this one is multiplied. Every 16 x 16 product takes the six
// significant products, smallest terms first, chunks in order. Rows past nb re-read row nb-1;
// their scores are not stored. Two workgroups per CU (60 KB of LDS each).
template <int D>
__global__ __launch_bounds__(256, 2) void score_kernel(int nb, const float* __restrict__ qbar,
                                                    const float* __restrict__ kbar,
                                                    float* __restrict__ S) {
  constexpr int TS = 128, KC = 32, NCH = D / KC;
  constexpr int RS = KC + 8;  // row stride in bf16: 80 bytes, so 16 rows' 16-byte reads spread
  __shared__ __attribute__((aligned(16))) bf16 As[3][TS][RS];
  __shared__ __attribute__((aligned(16))) bf16 Bs[3][TS][RS];
  const long head = blockIdx.z;
  const float* q = qbar + head * (long)nb * D;
  const float* k = kbar + head * (long)nb * D;
  const int I0 = blockIdx.y * TS, J0 = blockIdx.x * TS;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, lr = lane % 16, g = lane / 16;
  const int wi = (wave >> 1) * 64, wj = (wave & 1) * 64;  // this wave's 64 x 64 sub-tile
  const int lrow = tid / 2, lcol = (tid % 2) * 16;         // 16 channels of one row per thread
  const float* qrow = q + (long)min(I0 + lrow, nb - 1) * D + lcol;
  const float* krow = k + (long)min(J0 + lrow, nb - 1) * D + lcol;
  float a[16], b[16];  // this thread's 16 channels of the chunk being split
  load8(qrow, a);
  load8(qrow + 8, a + 8);
  load8(krow, b);
  load8(krow + 8, b + 8);
  f32x4 acc[4][4];
#pragma unroll
  for (int a4 = 0; a4 < 4; ++a4)
#pragma unroll
    for (int b4 = 0; b4 < 4; ++b4) acc[a4][b4] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (c) __syncthreads();  // the previous chunk's reads are done
#pragma unroll
    for (int h8 = 0; h8 < 2; ++h8) {
      bf16x8 h, m, l;
      split3(*reinterpret_cast<const float(*)[8]>(a + 8 * h8), h, m, l);
      *reinterpret_cast<bf16x8*>(&As[0][lrow][lcol + 8 * h8]) = h;
      *reinterpret_cast<bf16x8*>(&As[1][lrow][lcol + 8 * h8]) = m;
      *reinterpret_cast<bf16x8*>(&As[2][lrow][lcol + 8 * h8]) = l;
      split3(*reinterpret_cast<const float(*)[8]>(b + 8 * h8), h, m, l);
      *reinterpret_cast<bf16x8*>(&Bs[0][lrow][lcol + 8 * h8]) = h;
      *reinterpret_cast<bf16x8*>(&Bs[1][lrow][lcol + 8 * h8]) = m;
      *reinterpret_cast<bf16x8*>(&Bs[2][lrow][lcol + 8 * h8]) = l;
    }
    if (c + 1 < NCH) {  // the next chunk loads while this one is multiplied
      load8(qrow + (c + 1) * KC, a);
      load8(qrow + (c + 1) * KC + 8, a + 8);
      load8(krow + (c + 1) * KC, b);
      load8(krow + (c + 1) * KC + 8, b + 8);
    }
    __syncthreads();
    // lane holds A[row lr][k 8g..8g+7] and B[k 8g..8g+7][col lr] of each 16 x 16 tile
    bf16x8 bv[4][3];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int p = 0; p < 3; ++p)
        bv[t][p] = *reinterpret_cast<const bf16x8*>(&Bs[p][wj + 16 * t + lr][8 * g]);
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      bf16x8 av[3];
#pragma unroll
      for (int p = 0; p < 3; ++p)
        av[p] = *reinterpret_cast<const bf16x8*>(&As[p][wi + 16 * a4 + lr][8 * g]);
#pragma unroll
      for (int b4 = 0; b4 < 4; ++b4) {
        f32x4 x = acc[a4][b4];  // smallest terms first
        x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[2], bv[b4][0], x, 0, 0, 0);
        x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[1], bv[b4][1], x, 0, 0, 0);
        x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[0], bv[b4][2], x, 0, 0, 0);
        x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[1], bv[b4][0], x, 0, 0, 0);
        x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[0], bv[b4][1], x, 0, 0, 0);
        acc[a4][b4] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[0], bv[b4][0], x, 0, 0, 0);
      }
    }
  }
  float* Sh = S + head * (long)nb * nb;
#pragma unroll
  for (int a4 = 0; a4 < 4; ++a4)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int I = I0 + wi + 16 * a4 + 4 * g + v;
      if (I < nb) {
#pragma unroll
        for (int b4 = 0; b4 < 4; ++b4) {
          const int J = J0 + wj + 16 * b4 + lr;
          if (J < nb) Sh[(long)I * nb + J] = acc[a4][b4][v];
        }
      }
    }
}

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // larger float -> larger key
}

// Rows too long for the register kernel: one 64-lane workgroup per score row; dynamic LDS holds the
// row's nb keys. Every loop over the row takes kBatch elements per lane at a time, loads first: one
// memory (or LDS) latency per batch instead of one per element.
constexpr int kBatch = 8;
__global__ __launch_bounds__(64) void topk_kernel(int nb, int keep, const float* __restrict__ S,
                                                  int32_t* __restrict__ idx) {
  extern __shared__ uint32_t keys[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t found[2];
  const long row = ((long)blockIdx.z * gridDim.y + blockIdx.y) * nb + blockIdx.x;
  const float* s = S + row * nb;
  int32_t* out = idx + row * keep;
  const int lane = threadIdx.x;
  if (keep >= nb) {
    for (int j = lane; j < nb; j += 64) out[j] = j;
    return;
  }
  for (int base = 0; base < nb; base += 64 * kBatch) {
    float v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int j = base + 64 * u + lane;
      v[u] = j < nb ? s[j] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int j = base + 64 * u + lane;
      if (j < nb) keys[j] = order_key(v[u]);
    }
  }
  uint32_t prefix = 0, mask = 0;
  uint32_t remaining = (uint32_t)keep;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = lane; i < 256; i += 64) hist[i] = 0;
    __syncthreads();
    for (int base = 0; base < nb; base += 64 * kBatch) {
      uint32_t k[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int j = base + 64 * u + lane;
        k[u] = j < nb ? keys[j] : 0u;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int j = base + 64 * u + lane;
        if (j < nb && (k[u] & mask) == prefix) atomicAdd(&hist[(k[u] >> shift) & 255u], 1u);
      }
    }
    __syncthreads();
    uint32_t c[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) c[b] = hist[4 * lane + b];
    // elements whose digit lies in higher lanes' bins: exclusive suffix sum across the wave
    const uint32_t mine = c[0] + c[1] + c[2] + c[3];
    uint32_t incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t o = __shfl_down(incl, off);
      if (lane + off < 64) incl += o;
    }
    uint32_t g = incl - mine;
#pragma unroll
    for (int b = 3; b >= 0; --b) {
      if (g < remaining && remaining <= g + c[b]) { found[0] = 4 * lane + b; found[1] = g; }
      g += c[b];
    }
    __syncthreads();
    const uint32_t D = found[0], gt = found[1];
    __syncthreads();
    remaining -= gt;
    prefix |= D << shift;
    mask |= 255u << shift;
  }
  // Keys > prefix are all kept; of the keys == prefix, the `remaining` lowest indices are kept.
  uint32_t written = 0, eq_seen = 0;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int base0 = 0; base0 < nb; base0 += 64 * kBatch) {
    uint32_t kk[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int j = base0 + 64 * u + lane;
      kk[u] = j < nb ? keys[j] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int j = base0 + 64 * u + lane;
      const uint32_t k = kk[u];
      const bool gt = j < nb && k > prefix;
      const bool eq = j < nb && k == prefix;
      const uint64_t eqm = __ballot(eq);
      const uint32_t eq_rank = eq_seen + (uint32_t)__popcll(eqm & below);
      const bool sel = gt || (eq && eq_rank < remaining);
      const uint64_t selm = __ballot(sel);
      const uint32_t pos = written + (uint32_t)__popcll(selm & below);
      if (sel && pos < (uint32_t)keep) out[pos] = j;
      written += (uint32_t)__popcll(selm);
      eq_seen += (uint32_t)__popcll(eqm);
    }
  }
}

// Top-k of one score row per wave with the row in registers: lane l holds keys 64u + l, u < U
// (padding key 0 lies below every finite score's key and is never counted). The k-th largest key T
// is built from the top bit down: T | bit is kept when at least `keep` keys are >= it, a wave's
// count being the popcounts of one ballot per slot. Once the upper 16 bits are fixed, only keys
// whose upper half equals T's can decide the lower half; when at most 64 of them exist they are
// gathered one per lane through LDS and the lower 16 bits are searched over that one slot (keys in
// higher buckets are counted once). Otherwise (heavy exact ties) the search goes on over every slot.
// Kept: every key > T, and of the keys == T the lowest indices (when exactly `keep` keys are >= T,
// that is every key >= T), written ascending. Four rows per workgroup, no workgroup barrier.
constexpr int kTopkMaxSlots = 40;
template <int U>
__global__ __launch_bounds__(256) void topk_reg_kernel(int nb, int keep, long rows,
                                                       const float* __restrict__ S,
                                                       int32_t* __restrict__ idx) {
  __shared__ uint32_t cand[4][64];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const long row = (long)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  const float* s = S + row * nb;
  int32_t* out = idx + row * keep;
  uint32_t key[U];
  {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = s[min(64 * u + lane, nb - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u) key[u] = 64 * u + lane < nb ? order_key(v[u]) : 0u;
  }
  const uint32_t ukeep = (uint32_t)keep;
  uint32_t T = 0, nT = (uint32_t)nb;  // nT = number of (valid) keys >= T
  for (int b = 31; b >= 16; --b) {
    const uint32_t c = T | (1u << b);
    uint32_t n = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) n += (uint32_t)__popcll(__ballot(key[u] >= c));
    if (n >= ukeep) { T = c; nT = n; }
  }
  const uint32_t hiT = T >> 16;
  uint32_t above = 0, ncand = 0;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    above += (uint32_t)__popcll(__ballot((key[u] >> 16) > hiT));
    ncand += (uint32_t)__popcll(__ballot((key[u] >> 16) == hiT));
  }
  if (ncand <= 64) {
    uint32_t base = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool c = (key[u] >> 16) == hiT;
      const uint64_t m = __ballot(c);
      const uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                       __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (c) cand[wave][base + below] = key[u];
      base += (uint32_t)__popcll(m);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint32_t ck = (uint32_t)lane < ncand ? cand[wave][lane] : 0u;
    for (int b = 15; b >= 0; --b) {
      const uint32_t c = T | (1u << b);
      const uint32_t n = above + (uint32_t)__popcll(__ballot(ck >= c));
      if (n >= ukeep) { T = c; nT = n; }
    }
  } else {
    for (int b = 15; b >= 0; --b) {
      const uint32_t c = T | (1u << b);
      uint32_t n = 0;
#pragma unroll
      for (int u = 0; u < U; ++u) n += (uint32_t)__popcll(__ballot(key[u] >= c));
      if (n >= ukeep) { T = c; nT = n; }
    }
  }
  if (nT == ukeep && T != 0) {  // no surplus ties at the boundary: keep every key >= T
    uint32_t written = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool sel = key[u] >= T;
      const uint64_t m = __ballot(sel);
      const uint32_t pos = written + __builtin_amdgcn_mbcnt_hi(
                                         (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (sel && pos < ukeep) out[pos] = 64 * u + lane;
      written += (uint32_t)__popcll(m);
    }
    return;
  }
  uint32_t gt_total = 0;
#pragma unroll
  for (int u = 0; u < U; ++u)
    gt_total += (uint32_t)__popcll(__ballot(64 * u + lane < nb && key[u] > T));
  const uint32_t remaining = ukeep - gt_total;
  uint32_t written = 0, eq_seen = 0;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const bool valid = 64 * u + lane < nb;
    const bool gt = valid && key[u] > T, eq = valid && key[u] == T;
    const uint64_t eqm = __ballot(eq);
    const uint32_t eq_rank = eq_seen + __builtin_amdgcn_mbcnt_hi(
                                           (uint32_t)(eqm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)eqm, 0u));
    const bool sel = gt || (eq && eq_rank < remaining);
    const uint64_t selm = __ballot(sel);
    const uint32_t pos = written + __builtin_amdgcn_mbcnt_hi(
                                       (uint32_t)(selm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)selm, 0u));
    if (sel && pos < ukeep) out[pos] = 64 * u + lane;
    written += (uint32_t)__popcll(selm);
    eq_seen += (uint32_t)__popcll(eqm);
  }
}

template <int U>
void launch_topk_reg(int nb, int keep, long rows, const float* S, int32_t* idx, hipStream_t st) {
  hipLaunchKernelGGL(topk_reg_kernel<U>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, nb,
                     keep, rows, S, idx);
}

// Row top-k over the score matrix: the register kernel with the fewest slots that hold a row.
void launch_topk(int nb, int keep, int B, int H, const float* S, int32_t* idx, hipStream_t st) {
  const long rows = (long)B * H * nb;
  const int need = (nb + 63) / 64;
  if (keep >= nb || need > kTopkMaxSlots) {
    hipLaunchKernelGGL(topk_kernel, dim3(nb, H, B), dim3(64), (size_t)nb * sizeof(uint32_t), st,
                       nb, keep, S, idx);
    return;
  }
  if (need <= 1) return launch_topk_reg<1>(nb, keep, rows, S, idx, st);
  if (need <= 2) return launch_topk_reg<2>(nb, keep, rows, S, idx, st);
  if (need <= 4) return launch_topk_reg<4>(nb, keep, rows, S, idx, st);
  if (need <= 6) return launch_topk_reg<6>(nb, keep, rows, S, idx, st);
  if (need <= 8) return launch_topk_reg<8>(nb, keep, rows, S, idx, st);
  if (need <= 10) return launch_topk_reg<10>(nb, keep, rows, S, idx, st);
  if (need <= 12) return launch_topk_reg<12>(nb, keep, rows, S, idx, st);
  if (need <= 16) return launch_topk_reg<16>(nb, keep, rows, S, idx, st);
  if (need <= 19) return launch_topk_reg<19>(nb, keep, rows, S, idx, st);
  if (need <= 24) return launch_topk_reg<24>(nb, keep, rows, S, idx, st);
  if (need <= 32) return launch_topk_reg<32>(nb, keep, rows, S, idx, st);
  return launch_topk_reg<kTopkMaxSlots>(nb, keep, rows, S, idx, st);
}

hipError_t launch_pool(const Shape& s, const void* X, int block, float* means, hipStream_t st,
                       float* nmax = nullptr) {
  const dim3 grid(num_blocks(s.N, block), s.H, s.B);
  if (s.bf16)
    hipLaunchKernelGGL(pool_kernel<bf16>, grid, dim3(256), 0, st, s.N, s.d, block, (const bf16*)X,
                       means, nmax);
  else
    hipLaunchKernelGGL(pool_kernel<float>, grid, dim3(256), 0, st, s.N, s.d, block, (const float*)X,
                       means, nmax);
  return hipGetLastError();
}

template <typename T, int TPT>
hipError_t launch_rope_pool_t(const Shape& s, const void* X, const float* cos_tab,
                              const float* sin_tab, int ld, int block, void* Xr, float* means,
                              float* nmax, hipStream_t st) {
  const int heads = s.B * s.H;
  const dim3 grid(num_blocks(s.N, block), (heads + kRopePoolHeads - 1) / kRopePoolHeads);
  hipLaunchKernelGGL((rope_pool_kernel<T, TPT>), grid, dim3(256), 0, st, s.N, block, heads, ld,
                     (const T*)X, cos_tab, sin_tab, (T*)Xr, means, nmax);
  return hipGetLastError();
}

}  // namespace

size_t select_pooled_workspace_bytes(const Shape& s, int block) {
  const size_t nb = (size_t)num_blocks(s.N, block);
  return align_up((size_t)s.B * s.H * nb * nb * sizeof(float));
}

hipError_t launch_select_pooled(const Shape& s, const float* qbar, const float* kbar, int block,
                                int keep, int32_t* idx, void* ws, hipStream_t st) {
  const int nb = num_blocks(s.N, block);
  const size_t heads = (size_t)s.B * s.H;
  float* S = (float*)ws;
  const int tiles = (nb + 127) / 128;
  if (s.d == 128)
    hipLaunchKernelGGL(score_kernel<128>, dim3(tiles, tiles, (unsigned)heads), dim3(256), 0, st, nb,
                       qbar, kbar, S);
  else
    hipLaunchKernelGGL(score_kernel<64>, dim3(tiles, tiles, (unsigned)heads), dim3(256), 0, st, nb,
                       qbar, kbar, S);
  launch_topk(nb, keep, s.B, s.H, S, idx, st);
  return hipGetLastError();
}

hipError_t launch_block_pool(const Shape& s, const void* X, int block, float* means, float* nmax,
                             hipStream_t st) {
  return launch_pool(s, X, block, means, st, nmax);
}

bool rope_pool_supported(const Shape& s, int block) { return s.d == 128 && block >= 32; }

hipError_t launch_rope_pool(const Shape& s, const void* X, const float* cos_tab,
                            const float* sin_tab, int ld, int block, void* Xr, float* means,
                            float* nmax, hipStream_t st) {
  switch ((s.bf16 ? 1000 : 0) + block) {
    case 1064: return launch_rope_pool_t<bf16, 4>(s, X, cos_tab, sin_tab, ld, block, Xr, means, nmax, st);
    case 1128: return launch_rope_pool_t<bf16, 8>(s, X, cos_tab, sin_tab, ld, block, Xr, means, nmax, st);
    case 32: return launch_rope_pool_t<float, 2>(s, X, cos_tab, sin_tab, ld, block, Xr, means, nmax, st);
    case 64: return launch_rope_pool_t<float, 4>(s, X, cos_tab, sin_tab, ld, block, Xr, means, nmax, st);
    case 128: return launch_rope_pool_t<float, 8>(s, X, cos_tab, sin_tab, ld, block, Xr, means, nmax, st);
  }
  return hipErrorInvalidValue;
}

size_t select_workspace_bytes(const Shape& s, int block) {
  const size_t nb = (size_t)num_blocks(s.N, block);
  const size_t heads = (size_t)s.B * s.H;
  return 2 * align_up(heads * nb * s.d * sizeof(float)) + align_up(heads * nb * nb * sizeof(float));
}

hipError_t launch_block_select(const Shape& s, const void* Qr, const void* Kr, int block, int keep,
                               int32_t* idx, void* ws, hipStream_t st) {
  const int nb = num_blocks(s.N, block);
  const size_t heads = (size_t)s.B * s.H;
  char* w = (char*)ws;
  float* qbar = (float*)w;
  float* kbar = (float*)(w + align_up(heads * nb * s.d * sizeof(float)));
  float* S = (float*)(w + 2 * align_up(heads * nb * s.d * sizeof(float)));
  hipError_t e = launch_pool(s, Qr, block, qbar, st);
  if (e == hipSuccess) e = launch_pool(s, Kr, block, kbar, st);
  if (e == hipSuccess) e = launch_select_pooled(s, qbar, kbar, block, keep, idx, S, st);
  return e;
}

}  // namespace rola
