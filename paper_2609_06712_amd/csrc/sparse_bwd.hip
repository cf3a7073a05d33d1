// Backward pass of the block-sparse attention (the sparse branch's part of fine-tuning, Sec. 4.5):
// from dO^s, the saved O^s and the forward's log-sum-exp, the gradients dQ^r, dK^r, dV of
// O^s = softmax(Q^r K^r^T * scale) V restricted to the selected key blocks (Algorithm step 4). The
// block lists are constant (the selection is piecewise constant in Q^r, K^r).
//
// With P = exp(S*scale - lse) and D_q = sum_c dO^s_qc O^s_qc:  dP = dO V^T,  dS = P (dP - D),
// dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO.  Two kernels, each recomputing S and P:
//   sparse_dq_kernel   per query block, walking its own list (as the forward): Q and dO of the wave's
//                      32 queries in registers, K and V sub-tiles through three LDS stages;
//   sparse_dkv_kernel  per key block, walking the query blocks that selected it (lists transposed by
//                      bwd_reverse_kernel) in 32-query steps: one role of waves holds the keys' K
//                      (S, P, dV), the other their V (dP, dS, dK) and takes P from the first one
//                      step later; Q and dO rows (and the queries' lse and D) through four LDS
//                      stages.
// Products on v_mfma_f32_32x32x16_bf16. S and dP come out with one lane per key and the 32 queries
// in its registers; the products that contract over keys (dQ) or queries (dK, dV) take their other
// operand through the transposing LDS read ds_read_b64_tr_b16, in the order the registers hold the
// contracted index (as the forward's P V). dQ needs dS with one lane per query: each wave passes its
// dS tile through 2 KB of LDS. Tiles are stored with a swizzle that keeps both the row reads and the
// transposing reads free of bank conflicts. Gradients are fp32.
#include "common.h"
#include "launch.h"

namespace rola {
namespace {

constexpr int kBSub = 32;      // keys (dQ) or queries (dK, dV) per sub-tile
constexpr int kLsePad = 128;  // zero entries after the packed lse/D array: a sub-tile of the last
                              // query block reads up to block - 1 entries past the last query
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}


// D_q = sum_c dO_qc O_qc and the forward's lse, packed per query: lseD[q] = {lse_q, D_q}. 16 lanes
// per query row, 8 channels each. The array is padded by kLsePad zero entries (read past the end).
__global__ __launch_bounds__(256) void bwd_rowdot_kernel(long rows, const bf16* __restrict__ O,
                                                         const bf16* __restrict__ dO,
                                                         const float* __restrict__ lse,
                                                         float2* __restrict__ lseD) {
  const long row = ((long)blockIdx.x * 256 + threadIdx.x) / 16;
  const int part = threadIdx.x % 16;
  float s = 0.f;
  if (row < rows) {
    float a[8], b[8];
    load8(O + row * 128 + part * 8, a);
    load8(dO + row * 128 + part * 8, b);
#pragma unroll
    for (int i = 0; i < 8; ++i) s = fmaf(a[i], b[i], s);
  }
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) s += __shfl_xor(s, off, 16);
  if (part == 0) {
    if (row < rows) lseD[row] = make_float2(lse[row], s);
    else if (row < rows + kLsePad) lseD[row] = make_float2(0.f, 0.f);
  }
}

// Membership bitmaps of the block lists: bits[head][I][J / 32] bit J % 32. Each row is built in
// LDS (words * 4 bytes of dynamic shared memory) and written whole, so no clearing pass is needed.
__global__ __launch_bounds__(64) void bwd_bits_kernel(int nb, int keep, int words,
                                                      const int32_t* __restrict__ idx,
                                                      uint32_t* __restrict__ bits) {
  extern __shared__ uint32_t row_bits[];
  const long row = blockIdx.x;  // head * nb + I
  for (int w = threadIdx.x; w < words; w += 64) row_bits[w] = 0u;
  __syncthreads();
  for (int k = threadIdx.x; k < keep; k += 64) {
    const int J = idx[row * keep + k];
    if ((unsigned)J < (unsigned)nb) atomicOr(&row_bits[J >> 5], 1u << (J & 31));
  }
  __syncthreads();
  for (int w = threadIdx.x; w < words; w += 64) bits[row * words + w] = row_bits[w];
}

// Walk order of the transposed lists: query blocks by increasing bit-reversed index over the smallest
// power of two >= nb, a low-discrepancy order in which every list's entries spread evenly. Key
// blocks whose lists are about equally long then sit on about the same query blocks after the same
// number of steps, and bwd_order_kernel has the dK/dV workgroups that run at once take key blocks
// of about equal list length: concurrent workgroups share Q and dO rows in L2.
__host__ __device__ inline int rev_walk_bits(int nb) {
  int k = 1;
  while ((1 << k) < nb) ++k;
  return k;
}

// Transposed lists: rev[head][J] = count, then the query blocks I that selected J in walk order.
// One wave per (head, 32 key blocks): the bitmap column of the 32 key blocks over every query block
// goes to LDS (nb words), then lane j < 32 collects key block 32w + j's list.
__global__ __launch_bounds__(64) void bwd_reverse_kernel(int nb, int words, int kb,
                                                         const uint32_t* __restrict__ bits,
                                                         int32_t* __restrict__ rev) {
  extern __shared__ uint32_t col[];  // [nb]: bit j of col[I] = query block I selected J = 32w + j
  const long head = blockIdx.x / words;
  const int w = (int)(blockIdx.x % words), lane = threadIdx.x;
  for (int I = lane; I < nb; I += 64) col[I] = bits[(head * nb + I) * words + w];
  __syncthreads();
  const int J = 32 * w + lane;
  if (lane >= 32 || J >= nb) return;
  int32_t* out = rev + (head * nb + J) * (long)(nb + 1);
  int cnt = 0;
  for (int p = 0; p < (1 << kb); ++p) {
    const int I = (int)(__brev((unsigned)p) >> (32 - kb));
    if (I < nb && ((col[I] >> lane) & 1u)) out[1 + cnt++] = I;
  }
  out[0] = cnt;
}

// Order of the key blocks for the dK/dV workgroups: longer lists first (equal lengths by ascending
// J), order[head][rank] = J. One workgroup per (head, 256 key blocks): every list length of the
// head goes to LDS, and each thread ranks one key block against all of them.
__global__ __launch_bounds__(256) void bwd_order_kernel(int nb, int chunks,
                                                        const int32_t* __restrict__ rev,
                                                        int32_t* __restrict__ order) {
  extern __shared__ int32_t len[];  // [nb]
  const long head = blockIdx.x / chunks;
  const int J = (int)(blockIdx.x % chunks) * 256 + threadIdx.x;
  for (int K = threadIdx.x; K < nb; K += 256) len[K] = rev[(head * nb + K) * (long)(nb + 1)];
  __syncthreads();
  if (J >= nb) return;
  const int e = len[J];
  int rank = 0;
  for (int K = 0; K < nb; ++K) rank += len[K] > e || (len[K] == e && K < J);
  order[head * nb + rank] = J;
}

// ---- dQ: one workgroup per (b, h, query block), BLK/32 waves of 32 queries -------------------------
template <int BLK, int NBUF>
__global__ __launch_bounds__(BLK * 2, 2) void sparse_dq_kernel(
    int N, int nb, int total, const int32_t* __restrict__ lists, int keep, float scale_log2,
    float scale, const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const bf16* __restrict__ dO, const float2* __restrict__ lseD, float* __restrict__ dQ) {
  constexpr int D = 128, NW = BLK / 32;
  constexpr int TILE = kBSub * D * 2, STAGE = 2 * TILE;
  constexpr int DMA_PER_WAVE = TILE / 1024 / NW, SUBS = BLK / kBSub;
  constexpr int SPITCH = 72;  // bytes per row of the dS^T scratch tile (32 queries + 4 pad)
  __shared__ __attribute__((aligned(1024))) char lds[NBUF * STAGE];
  __shared__ __attribute__((aligned(16))) char scr[NW][kBSub * SPITCH];

  const int L = xcd_remap(blockIdx.x, total);
  const int I = L % nb;
  const long head = L / nb;
  const int tid = threadIdx.x, lane = tid % 64, hh = lane / 32;
  const int wave = wave_uniform(tid / 64);
  const int qrow0 = I * BLK + wave * 32;  // the wave's first query
  const int q = qrow0 + lane % 32;        // A-operand row of this lane (and column of dQ^T)
  const bool qvalid = q < N;
  const long hoff = head * (long)N * D;
  const char* Kh = reinterpret_cast<const char*>(K + hoff);
  const char* Vh = reinterpret_cast<const char*>(V + hoff);
  typedef const __attribute__((address_space(4))) int32_t* const_i32;
  const const_i32 slist = (const_i32)(lists + (head * nb + I) * (long)keep);
  const int T = keep * SUBS;

  bf16x8 qf[8], df[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    qf[s] = qvalid ? *reinterpret_cast<const bf16x8*>(Q + hoff + (long)q * D + 16 * s + 8 * hh) : bf16x8{};
    df[s] = qvalid ? *reinterpret_cast<const bf16x8*>(dO + hoff + (long)q * D + 16 * s + 8 * hh) : bf16x8{};
  }
  // lse and D of the rows 8j + 4(l/32) + i the S tiles hand this lane; +inf lse for rows past N
  float lse[16], dsum[16];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = qrow0 + 8 * j + 4 * hh + i;
      const float2 v = r < N ? lseD[head * (long)N + r] : make_float2(INFINITY, 0.f);
      lse[4 * j + i] = v.x;
      dsum[4 * j + i] = v.y;
    }
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0): nothing of this waits in the loop

  f32x16 acc[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) acc[w] = f32x16{};

  uint32_t dsrc[DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < DMA_PER_WAVE; ++i) {
    const int row = 4 * (wave * DMA_PER_WAVE + i) + lane / 16, pos = lane % 16;
    dsrc[i] = row * D * 2 + ((pos ^ bw_swizzle(row)) << 4);
  }
  const uint32_t lds0 = lds_address(lds);
  auto key0 = [&](int t) {
    const int J = slist[t / SUBS];
    return (unsigned)J < (unsigned)nb ? J * BLK + (t % SUBS) * kBSub : -1;
  };
  auto issue = [&](int k0, int buf) {  // 2 * DMA_PER_WAVE loads per wave, always
    k0 = max(k0, 0);
    const uint32_t dst = lds0 + buf * STAGE;
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) {
      const uint32_t slot = (wave * DMA_PER_WAVE + i) * 1024;
      const int r = 4 * (wave * DMA_PER_WAVE + i) + lane / 16;
      const uint32_t rowoff = (uint32_t)(min(k0 + r, N - 1) - r) * (D * 2);  // rows past N: N-1
      dma16(Kh, rowoff + dsrc[i], dst + slot);
      dma16(Vh, rowoff + dsrc[i], dst + TILE + slot);
    }
  };
  char* sc = scr[wave];

  constexpr int PER_STEP = 2 * DMA_PER_WAVE;
  int issued = 0;
#pragma unroll
  for (int j = 0; j < NBUF - 1; ++j)
    if (j < T) issue(key0(j), j), ++issued;
  for (int t = 0; t < T;) {
#pragma unroll
    for (int b = 0; b < NBUF; ++b) {
      if (t >= T) break;
      if (issued == t + NBUF - 1) {
        constexpr int allowed = PER_STEP * (NBUF - 2);
        __builtin_amdgcn_s_waitcnt((allowed & 15) | ((allowed >> 4) << 14) | (7 << 4) | (15 << 8));
      } else {
        __builtin_amdgcn_s_waitcnt(0);
      }
      __syncthreads();
      if (issued < T) issue(key0(issued), (b + NBUF - 1) % NBUF), ++issued;
      const int k0 = key0(t);
      if (k0 >= 0 && k0 < N) {
        const char* Kt = lds + b * STAGE;
        const char* Vt = Kt + TILE;
        f32x16 S = f32x16{}, dP = f32x16{};
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          S = mfma32(qf[s], row_frag(Kt, lane % 32, s, hh), S);
          dP = mfma32(df[s], row_frag(Vt, lane % 32, s, hh), dP);
        }
        // dS with one lane per key (column l%32); rows 8j + 4(l/32) + i are queries
        const bool kvalid = k0 + lane % 32 < N;
        bf16x4 ds4[4];
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const float e = __builtin_amdgcn_exp2f(fmaf(S[k], scale_log2, -lse[k]));
          const float p = kvalid ? e : 0.f;
          ds4[k / 4][k % 4] = (bf16)(p * (dP[k] - dsum[k]));
        }
        // dS^T row-major [key][query] in the wave's scratch, then read back transposed
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<bf16x4*>(sc + (lane % 32) * SPITCH + 2 * (8 * j + 4 * hh)) = ds4[j];
        asm volatile("" ::: "memory");  // the reads below follow the writes (one wave, in order)
        bf16x8 dsf[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int i16 = lane % 16, g1 = (lane / 16) & 1;
          bf16x4 part[2];
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const int row = 16 * u + 8 * half + 4 * hh + i16 / 4;
            part[half] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (lds_bf16x4*)(sc + row * SPITCH + 2 * (16 * g1 + 4 * (i16 & 3))));
          }
          dsf[u] = __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7);
        }
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
          for (int u = 0; u < 2; ++u) acc[w] = mfma32(tr_frag(Kt, w, u, lane), dsf[u], acc[w]);
      }
      ++t;
    }
  }
  if (qvalid) {  // dQ^T: lane = query, rows = channels 32w + 8j + 4(l/32) + i
    float* dq = dQ + hoff + (long)q * D;
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<float4*>(dq + 32 * w + 8 * j + 4 * hh) =
            make_float4(acc[w][4 * j] * scale, acc[w][4 * j + 1] * scale, acc[w][4 * j + 2] * scale,
                        acc[w][4 * j + 3] * scale);
  }
}

// ---- dK, dV: one workgroup per (b, h, key block) ------------------------------------------------
// Two roles of BLK/32 waves each over the same 32-key column tiles. Role 0 holds the keys' K and
// computes S, P = exp2(S scale log2e - lse) and dV += dO^T P; role 1 holds their V and computes
// dP = dO V^T, dS = P (dP - D) and dK += Q^T dS, taking P from role 0 through LDS one step later
// (double-buffered, so one barrier per step serves the tile stages and the hand-over). A wave then
// needs one B operand set and one accumulator set (a wave doing both needs twice that, more than
// half the register file, and the compiler then moves accumulators between the two register files
// every step), so two waves run per SIMD. A step takes 32 queries. P goes over as fp16: it lies
// in [0, 1], where fp16's relative error (2^-11; absolute 2^-25 below 2^-14) is an eighth of the
// bf16 rounding dS takes next. Workgroups take a head's key blocks longest list first
// (bwd_order_kernel) and walk each list in the bit-reversed order, so that workgroups running at
// the same time sit on about the same query blocks and share their Q and dO rows in L2.
constexpr int kDkvNbuf = 4;  // LDS stages of sparse_dkv_kernel: 32 Q rows, 32 dO rows, lse/D (17 KB)
template <int BLK, int NBUF>
__global__ __launch_bounds__(BLK * 4) __attribute__((amdgpu_waves_per_eu(2, 2)))
void sparse_dkv_kernel(
    int N, int nb, int total, const int32_t* __restrict__ rev, float scale_log2, float scale,
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const bf16* __restrict__ dO, const float2* __restrict__ lseD, const int32_t* __restrict__ order,
    float* __restrict__ dK, float* __restrict__ dV) {
  constexpr int D = 128, NKW = BLK / 32, NW = 2 * NKW;
  constexpr int TILE = kBSub * D * 2;          // 32 rows of 256 bytes
  constexpr int STAGE = 2 * TILE + 1024;       // Q, dO, then lse/D of the 32 queries (256 B used)
  constexpr int DPW = 2 * (TILE / 1024) / NW;  // 1 KB tile loads per wave and step
  constexpr int SUBS = BLK / kBSub;            // steps per query block
  constexpr int PBUF = NKW * 2048;             // P of a step, fp16: per key tile 16 values a lane
  constexpr int AHEAD = NBUF - 2;              // stages loaded ahead (role 1 still reads one back)
  static_assert(DPW >= 1 && 2 * (TILE / 1024) % NW == 0 && AHEAD >= 1, "64- or 128-key blocks");
  __shared__ __attribute__((aligned(1024))) char lds[NBUF * STAGE + 2 * PBUF];

  typedef const __attribute__((address_space(4))) int32_t* const_i32;
  const int L = xcd_remap(blockIdx.x, total);
  const long head = L / nb;
  const int J = ((const_i32)order)[L];  // key blocks of one head, longer lists first
  const int tid = threadIdx.x, lane = tid % 64, hh = lane / 32;
  const int wave = wave_uniform(tid / 64);
  const int role = wave / NKW, kw = wave % NKW;
  const int key = J * BLK + kw * 32 + lane % 32;  // B-operand column of this lane
  const bool kvalid = key < N;
  const long hoff = head * (long)N * D;
  const char* Qh = reinterpret_cast<const char*>(Q + hoff);
  const char* dOh = reinterpret_cast<const char*>(dO + hoff);
  const const_i32 rl = (const_i32)(rev + (head * nb + J) * (long)(nb + 1));
  const int E = rl[0];
  const int T = E * SUBS;

  const bf16* bsrc = (role ? V : K) + hoff + (long)key * D + 8 * hh;
  bf16x8 bf[8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
    bf[s] = kvalid ? *reinterpret_cast<const bf16x8*>(bsrc + 16 * s) : bf16x8{};
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)

  f32x16 acc[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) acc[w] = f32x16{};

  // Tile loads: load g = wave * DPW + i moves rows 4(g % 8) .. +3 of Q (g < 8) or dO (g >= 8).
  uint32_t dsrc[DPW];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int g = wave * DPW + i, row = 4 * (g % 8) + lane / 16, pos = lane % 16;
    dsrc[i] = row * D * 2 + ((pos ^ bw_swizzle(row)) << 4);
  }
  const uint32_t lds0 = lds_address(lds);
  const char* lsebase = reinterpret_cast<const char*>(lseD + head * (long)N);
  auto query0 = [&](int t) {  // t >= 0
    return rl[1 + (unsigned)t / SUBS] * BLK + (int)((unsigned)t % SUBS) * kBSub;
  };
  auto issue = [&](int q0, int buf) {  // DPW loads per wave, and wave 0 one more (lse/D)
    const uint32_t dst = lds0 + buf * STAGE;
    if (q0 + kBSub <= N) {  // every row of the tile exists: one scalar base per tensor
      const uint32_t base = (uint32_t)q0 * (D * 2);
#pragma unroll
      for (int i = 0; i < DPW; ++i) {
        const int g = wave * DPW + i;
        dma16((g < 8 ? Qh : dOh) + base, dsrc[i], dst + (g / 8) * TILE + (g % 8) * 1024);
      }
    } else {
#pragma unroll
      for (int i = 0; i < DPW; ++i) {
        const int g = wave * DPW + i, r = 4 * (g % 8) + lane / 16;
        const uint32_t rowoff = (uint32_t)(min(q0 + r, N - 1) - r) * (D * 2);  // rows past N: N-1
        dma16(g < 8 ? Qh : dOh, rowoff + dsrc[i], dst + (g / 8) * TILE + (g % 8) * 1024);
      }
    }
    // lse, D of the 32 queries (256 bytes; lanes 16-63 repeat lanes 0-15): the array is padded by
    // kLsePad entries, and rows past N are masked below
    if (wave == 0) dma16(lsebase, (uint32_t)(q0 * 8 + (lane % 16) * 16), dst + 2 * TILE);
  };

  int issued = 0;
#pragma unroll
  for (int j = 0; j < AHEAD; ++j)
    if (j < T) issue(query0(j), j), ++issued;
  char* pbase = lds + NBUF * STAGE + kw * 2048 + lane * 16;  // + buffer * PBUF + u * 1024
  // Iteration t: role 0 takes step t (t < T), role 1 step t - 1 (t >= 1).
  for (int t = 0; t <= T;) {
#pragma unroll
    for (int b = 0; b < NBUF; ++b) {
      if (t > T) break;
      // The first query of this step's tile and of the tile whose loads it issues, read from the
      // list before the wait and the barrier (indices clamped into the list; pinned in SGPRs, or
      // the compiler sinks the scalar loads behind the barrier).
      int qcur = query0(max(0, min(t, T - 1))), qiss = query0(max(0, min(issued, T - 1)));
      asm volatile("" : "+s"(qcur), "+s"(qiss));
      if (t < T && issued == t + AHEAD) {
        constexpr int a0 = (DPW + 1) * (AHEAD - 1), a1 = DPW * (AHEAD - 1);
        if (wave == 0)
          __builtin_amdgcn_s_waitcnt((a0 & 15) | ((a0 >> 4) << 14) | (7 << 4) | (15 << 8));
        else
          __builtin_amdgcn_s_waitcnt((a1 & 15) | ((a1 >> 4) << 14) | (7 << 4) | (15 << 8));
      } else {
        __builtin_amdgcn_s_waitcnt(0);
      }
      __syncthreads();
      if (issued < T) issue(qiss, (b + AHEAD) % NBUF), ++issued;
      if (role ? t >= 1 : t < T) {
        const char* Qt = lds + (role ? (b + NBUF - 1) % NBUF : b) * STAGE;
        const char* dOt = Qt + TILE;
        const float2* lt = reinterpret_cast<const float2*>(Qt + 2 * TILE);
        char* pb = pbase + ((b + role) % 2) * PBUF;  // role 0 writes step t's, role 1 reads t - 1's
        // S (role 0) or dP (role 1): one lane per key; rows 8j + 4(l/32) + i are the step's queries
        // All operand fragments of the step are read up front (the transposed ones do not wait
        // for P), so that the products do not wait on LDS one fragment at a time.
        const char* A1 = role ? dOt : Qt;
        const char* A2 = role ? Qt : dOt;
        bf16x8 fa[8], fb[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) fa[s] = row_frag(A1, lane % 32, s, hh);
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
          for (int u = 0; u < 2; ++u) fb[2 * w + u] = tr_frag(A2, w, u, lane);
        __builtin_amdgcn_sched_barrier(0);
        f32x16 X = f32x16{};
#pragma unroll
        for (int s = 0; s < 8; ++s) X = mfma32(fa[s], bf[s], X);
        float p[16];
        bf16x8 b2[2];
        if (role == 0) {
          const int q0 = qcur;
          // The exponentials are computed unconditionally and rows past N zeroed in one uniform
          // branch: a per-element condition around them splits the step into a basic block per
          // element, across which no matrix instruction can be scheduled.
#pragma unroll
          for (int k = 0; k < 16; ++k)
            p[k] = __builtin_amdgcn_exp2f(fmaf(X[k], scale_log2, -lt[8 * (k / 4) + 4 * hh + k % 4].x));
          if (q0 + kBSub > N) {  // ragged last query block (uniform)
#pragma unroll
            for (int k = 0; k < 16; ++k) p[k] = q0 + 8 * (k / 4) + 4 * hh + k % 4 < N ? p[k] : 0.f;
          }
          f16x8 ph[2];
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            b2[k / 8][k % 8] = (bf16)p[k];
            ph[k / 8][k % 8] = (_Float16)p[k];
          }
          *reinterpret_cast<f16x8*>(pb) = ph[0];
          *reinterpret_cast<f16x8*>(pb + 1024) = ph[1];
        } else {
          const f16x8 ph0 = *reinterpret_cast<const f16x8*>(pb);
          const f16x8 ph1 = *reinterpret_cast<const f16x8*>(pb + 1024);
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            const float pk = (float)(k < 8 ? ph0[k] : ph1[k - 8]);
            b2[k / 8][k % 8] = (bf16)(pk * (X[k] - lt[8 * (k / 4) + 4 * hh + k % 4].y));
          }
        }
        // dV^T += dO^T P (role 0) or dK^T += Q^T dS (role 1), the transposed operand in the order
        // the registers hold the queries
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
          for (int u = 0; u < 2; ++u) acc[w] = mfma32(fb[2 * w + u], b2[u], acc[w]);
      }
      ++t;
    }
  }
  if (kvalid) {  // dV^T (role 0), dK^T (role 1): lane = key, rows = channels 32w + 8j + 4(l/32) + i
    float* out = (role ? dK : dV) + hoff + (long)key * D;
    const float f = role ? scale : 1.f;
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = 32 * w + 8 * j + 4 * hh;
        *reinterpret_cast<float4*>(out + c) = make_float4(acc[w][4 * j] * f, acc[w][4 * j + 1] * f,
                                                          acc[w][4 * j + 2] * f, acc[w][4 * j + 3] * f);
      }
  }
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace: [lse, D per query][bitmaps][transposed lists][key-block order][with dq_supported: the
// attention workspace of the dQ pass (pairs, merged lists, queue counters)].
struct BwdWs {
  size_t lsed, bits, rev, order, dq;
};
BwdWs bwd_layout(const Shape& s, int block, int keep) {
  const size_t heads = (size_t)s.B * s.H, nb = num_blocks(s.N, block), words = (nb + 31) / 32;
  return {align256((heads * s.N + kLsePad) * sizeof(float2)), align256(heads * nb * words * 4),
          align256(heads * nb * (nb + 1) * 4), align256(heads * nb * 4),
          dq_supported(s, block) ? align256(sparse_workspace_bytes(s, block, keep)) : 0};
}

template <int BLK>
hipError_t launch_bwd(const Shape& s, const void* Qr, const void* Kr, const void* V, int keep,
                      const int32_t* idx, float scale, const void* Os, const float* lse,
                      const void* dOs, float* dQ, float* dK, float* dV, void* ws, hipStream_t st) {
  const int nb = num_blocks(s.N, BLK), words = (nb + 31) / 32;
  const long heads = (long)s.B * s.H, rows = heads * s.N;
  const BwdWs lay = bwd_layout(s, BLK, keep);
  float2* lseD = (float2*)ws;
  uint32_t* bits = (uint32_t*)((char*)ws + lay.lsed);
  int32_t* rev = (int32_t*)((char*)ws + lay.lsed + lay.bits);
  int32_t* order = (int32_t*)((char*)ws + lay.lsed + lay.bits + lay.rev);
  const long rd_threads = (rows + kLsePad) * 16;
  hipLaunchKernelGGL(bwd_rowdot_kernel, dim3((unsigned)((rd_threads + 255) / 256)), dim3(256), 0,
                     st, rows, (const bf16*)Os, (const bf16*)dOs, lse, lseD);
  hipLaunchKernelGGL(bwd_bits_kernel, dim3((unsigned)(heads * nb)), dim3(64), words * sizeof(uint32_t),
                     st, nb, keep, words, idx, bits);
  hipLaunchKernelGGL(bwd_reverse_kernel, dim3((unsigned)(heads * words)), dim3(64),
                     nb * sizeof(uint32_t), st, nb, words, rev_walk_bits(nb), (const uint32_t*)bits,
                     rev);
  const int ochunks = (nb + 255) / 256;
  hipLaunchKernelGGL(bwd_order_kernel, dim3((unsigned)(heads * ochunks)), dim3(256),
                     nb * sizeof(int32_t), st, nb, ochunks, (const int32_t*)rev, order);
  const int total = (int)(heads * nb);
  const float sl = scale * 1.4426950408889634f;
  if (dq_supported(s, BLK)) {  // dQ on the paired, queued attention kernel
    const hipError_t e2 = launch_sparse_dq(s, Qr, Kr, V, keep, idx, scale, dOs, lseD, dQ,
                                           (char*)ws + lay.lsed + lay.bits + lay.rev + lay.order, st);
    if (e2 != hipSuccess) return e2;
  } else {
    hipLaunchKernelGGL((sparse_dq_kernel<BLK, 3>), dim3(total), dim3(BLK * 2), 0, st, s.N, nb, total,
                       idx, keep, sl, scale, (const bf16*)Qr, (const bf16*)Kr, (const bf16*)V,
                       (const bf16*)dOs, (const float2*)lseD, dQ);
  }
  hipLaunchKernelGGL((sparse_dkv_kernel<BLK, kDkvNbuf>), dim3(total), dim3(BLK * 4), 0, st, s.N, nb, total,
                     (const int32_t*)rev, sl, scale, (const bf16*)Qr, (const bf16*)Kr,
                     (const bf16*)V, (const bf16*)dOs, (const float2*)lseD, (const int32_t*)order,
                     dK, dV);
  return hipGetLastError();
}

}  // namespace

size_t sparse_backward_workspace_bytes(const Shape& s, int block, int keep) {
  if (!s.bf16 || s.d != 128 || (block != 64 && block != 128) ||
      num_blocks(s.N, block) > kBwdMaxBlocks)
    return 0;
  const BwdWs w = bwd_layout(s, block, keep);
  return w.lsed + w.bits + w.rev + w.order + w.dq;
}

hipError_t launch_sparse_backward(const Shape& s, const void* Qr, const void* Kr, const void* V,
                                  int block, int keep, const int32_t* idx, float scale,
                                  const void* Os, const float* lse, const void* dOs, float* dQ,
                                  float* dK, float* dV, void* ws, hipStream_t st) {
  if (block == 64)
    return launch_bwd<64>(s, Qr, Kr, V, keep, idx, scale, Os, lse, dOs, dQ, dK, dV, ws, st);
  return launch_bwd<128>(s, Qr, Kr, V, keep, idx, scale, Os, lse, dOs, dQ, dK, dV, ws, st);
}

}  // namespace rola
