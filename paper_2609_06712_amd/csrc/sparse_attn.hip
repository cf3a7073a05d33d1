// Block-sparse softmax attention of the sparse branch (Algorithm step 4; attention as in Sec. 3):
// every query block attends to the valid tokens of its `keep` selected key blocks, by online
// softmax with fp32 running max / sum / accumulators. With no index list every key block is walked
// in order, which is dense softmax attention (the 0 % sparsity reference).
//
// bf16 path (d_h = 128). A workgroup serves G = 1 or 2 query blocks of BLK tokens, with BLK/32
// waves of 32 queries per query block. With G = 2 (a pair: neighbours, or matched by list overlap)
// it walks the union of the two blocks' lists (built by group_union_kernel, in the walk order and
// from the start phase described there): a key block both hold is fetched into LDS once, and
// each wave computes only on the blocks its own query block selected. Adjacent query blocks share
// about half of their selections, so this cuts the K/V bytes that cross L2 by about a quarter.
// Keys stream in 32-key sub-tiles through NBUF LDS stages filled by direct global-to-LDS loads.
// Per wave and sub-tile, on v_mfma_f32_32x32x16_bf16:
//   S^T = K Q^T   A = K rows from LDS (ds_read_b128), B = Q fragments held in registers; lane l gets
//                 query l%32 and keys 8j + 4(l/32) + i, so a row max needs one permlane32 swap.
//   P = exp2(S^T * scale*log2e - m) rounded to bf16 in registers: directly the B operand of
//   O^T = V^T P^T A = V^T through the transposing LDS read ds_read_b64_tr_b16 of row-major V; the
//                 sum over keys runs in the order the S^T layout hands them out (two reads of four
//                 keys per operand), which leaves the result unchanged.
// Row sums accumulate per lane with v_dot2 on the bf16 probabilities. A step holds few registers
// (about 160), so three workgroups of four waves share a CU and the matrix and vector work of one
// wave overlaps that of the others. O is rescaled only when a sub-tile raises a row max by more
// than 2^8: the softmax ratio does not depend on the reference max, so this is exact.
#include <algorithm>
#include <atomic>
#include <climits>
#include <mutex>

#include "common.h"
#include "launch.h"
#include "rola.h"

namespace rola {
namespace {

constexpr int kSub = 32;            // keys per sub-tile: one LDS stage holds its K and V (8 KB each)
constexpr int kB64Group = 2;        // query blocks per workgroup of the 64-token path with a list
constexpr int kB64Nbuf = 3;         // its LDS stages (16 KB each)
constexpr float kRescaleTau = 8.f;  // log2 headroom before O is rescaled
// Largest score bound (log2 units) that serves as the softmax reference of the BOUND variant:
// probabilities then stay in [2^-80, 1], clear of fp32 and bf16 underflow for any V.
constexpr float kBoundMax = 40.f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// LDS layouts of a sub-tile: rows of 256 bytes (128 channels), the 16-byte chunks of each row
// XOR-swizzled. K: chunk ^ row%16, so the 16 rows of an operand read (ds_read_b128) hit distinct
// banks. V: chunk ^ 2*{0,3,5,6}[row%4], so the four rows x 64 bytes of each half of a transposing
// read land in distinct banks whether the LDS serves 128 or 256 bytes per pass.
__device__ __forceinline__ int k_swizzle(int row) { return row & 15; }
__device__ __forceinline__ int v_swizzle(int row) { return 2 * ((0x6530 >> (4 * (row & 3))) & 15); }

// Data-adaptive pairing of query blocks (G = 2). Query blocks whose lists overlap most are put in
// one workgroup; neighbours share about half of their selections, the best partner among the
// following 64 blocks often shares more. The pairing changes which query blocks share K/V loads
// and where each group's walk starts (walk_start); each query block sums its own selections only,
// bitwise as the one-block path does when given them in the same order.
constexpr int kPairWindow = 64;  // candidate partners of a query block: the next 64 blocks
constexpr int kPairRows = 128;   // bitmap rows one overlap workgroup holds (64 blocks + window)

// Row stride (words) of the membership bitmaps in LDS: odd, so a wave reading one word of 64
// consecutive rows hits 64 distinct banks.
__host__ __device__ inline int pair_row_stride(int nb) { return ((nb + 31) >> 5) | 1; }

// Candidate preference of every query block, one workgroup per (head, chunk of 64 query blocks).
// The membership bitmaps of the chunk's blocks and of the 64 after them are built in LDS from the
// lists (out-of-range entries dropped); lane d of a wave then intersects row I with row I+1+d and
// ranks the 64 candidates by overlap, larger first, the nearer first on equal overlap, candidates
// past the last block after all others. pref[head][chunk][k][r] = offset d of the k-th choice of
// query block chunk*64 + r: k-major, so that the greedy pass reads its column per lane.
__global__ __launch_bounds__(256) void pair_rank_kernel(int nb, int keep, int nchunks,
                                                        const int32_t* __restrict__ idx,
                                                        uint8_t* __restrict__ pref) {
  extern __shared__ uint32_t bits[];  // [kPairRows][rs]
  const int words = (nb + 31) >> 5, rs = pair_row_stride(nb);
  const long head = blockIdx.x / nchunks;
  const int chunk = (int)(blockIdx.x % nchunks), I0 = chunk * kPairWindow;
  const int rows = min(kPairRows, nb - I0);
  const int tid = threadIdx.x;
  for (int w = tid; w < kPairRows * rs; w += 256) bits[w] = 0u;
  __syncthreads();
  const int32_t* sel = idx + (head * nb + I0) * (long)keep;  // rows I0 .. I0+rows-1, contiguous
  for (int e = tid; e < rows * keep; e += 256) {
    const int J = sel[e];
    if ((unsigned)J < (unsigned)nb) atomicOr(&bits[(e / keep) * rs + (J >> 5)], 1u << (J & 31));
  }
  __syncthreads();
  const int d = tid % 64;
  uint8_t* out = pref + (head * nchunks + chunk) * (long)(kPairWindow * kPairWindow);
  for (int i = tid / 64; i < kPairWindow && I0 + i < nb; i += 4) {  // wave-uniform bounds
    int key = 63 - d - 64;  // past the last block: below every valid candidate
    if (I0 + i + 1 + d < nb) {  // then row i+1+d < rows
      const uint32_t* a = bits + i * rs;
      const uint32_t* b = bits + (i + 1 + d) * rs;
      int c = 0;
      for (int w = 0; w < words; ++w) c += __popc(a[w] & b[w]);
      key = (c << 6) | (63 - d);
    }
    int rank = 0;  // keys are distinct: the ranks are a permutation of 0..63
#pragma unroll
    for (int o = 0; o < 64; ++o) rank += __builtin_amdgcn_readlane(key, o) > key;
    out[rank * kPairWindow + i] = (uint8_t)d;
  }
}

// Greedy pairing, one wave per head: query blocks are visited in ascending order; a block not yet
// taken is paired with the untaken block among its next 64 that it ranks first, or stays alone
// when none is left. A block is only ever taken by one of the 63 blocks before it, so block I+64
// is always free when I is visited: every block but possibly the last gets a partner, which makes
// exactly ceil(nb / 2) groups. pairs[head][g] = I | J << 16 (J = nb: no partner), in the order the
// groups are formed. Lane k holds the k-th choices of a chunk's 64 blocks (64 bytes in registers,
// the next chunk loading meanwhile); a step is a ballot over the lanes whose choice is still free
// and a find-first-set. The table is gathered in LDS and written out at the end, so no store
// shares the memory counter with the chunk loads.
constexpr int kMaxPairGroups = 2032;  // ceil(4064 / 2): the most query blocks pairing serves
__global__ __launch_bounds__(64) void pair_greedy_kernel(int nb, int ngroups, int nchunks,
                                                         const uint8_t* __restrict__ pref,
                                                         int32_t* __restrict__ pairs) {
  __shared__ int32_t tbl[kMaxPairGroups];
  const long head = blockIdx.x;
  const int lane = threadIdx.x;
  const uint4* src = reinterpret_cast<const uint4*>(pref + head * nchunks * (long)(kPairWindow * kPairWindow));
  int32_t* out = pairs + head * ngroups;
  uint4 cur[4], nxt[4];
  auto fetch = [&](int c, uint4 (&r)[4]) {  // lane k: the 64 bytes of choice k, chunk c
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = src[(long)c * 256 + lane * 4 + j];
  };
  fetch(0, cur);
  uint64_t taken = 0;  // bit k: block I+k already has a partner
  int g = 0;
  for (int c = 0; c < nchunks; ++c) {
    fetch(min(c + 1, nchunks - 1), nxt);  // unconditional: a fixed count of loads in flight
    const uint32_t w[16] = {cur[0].x, cur[0].y, cur[0].z, cur[0].w, cur[1].x, cur[1].y,
                            cur[1].z, cur[1].w, cur[2].x, cur[2].y, cur[2].z, cur[2].w,
                            cur[3].x, cur[3].y, cur[3].z, cur[3].w};
#pragma unroll
    for (int r = 0; r < kPairWindow; ++r) {
      const int I = c * kPairWindow + r;
      if (I < nb) {
        if (taken & 1) {
          taken >>= 1;
        } else {
          const int d = (w[r / 4] >> (8 * (r % 4))) & 0xFF;  // this lane's choice
          const bool free_d = I + 1 + d < nb && !(((taken >> d) >> 1) & 1);
          const uint64_t m = __ballot(free_d);
          taken >>= 1;
          int partner = nb;
          if (m) {
            const int dd = __builtin_amdgcn_readlane(d, (int)__builtin_ctzll(m));
            partner = I + 1 + dd;
            taken |= 1ull << dd;
          }
          if (g < ngroups) tbl[g] = I | (partner << 16);  // every lane stores the same value
          ++g;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) cur[j] = nxt[j];
  }
  __syncthreads();
  for (int i = lane; i < ngroups; i += 64) out[i] = tbl[i];
}

// Walk order of the merged lists: key blocks by increasing bit-reversed index, over the smallest
// power of two >= nb. Any one list's entries spread evenly over this order (a low-discrepancy
// sequence), so workgroups that have walked the same fraction of their lists sit on nearly the
// same key blocks at the same time, whatever part of the sequence they selected; concurrent
// workgroups then share K/V in L2 more than in ascending order, where each list's dense regions
// (its own neighbourhood) put them at different key blocks (14B layer: about 4 % less kernel
// time, 7 % less for the bare K/V gather).
__host__ __device__ inline int walk_bits(int nb) {
  int k = 1;
  while ((1 << k) < nb) ++k;
  return k;
}
__host__ __device__ inline int walk_words(int nb) {
  return ((1 << walk_bits(nb)) + 31) >> 5;
}
__device__ __forceinline__ int walk_pos(int J, int kb) {
  return (int)(__brev((unsigned)J) >> (32 - kb));
}

// Start phase of a merged list (period > 0): the work queue hands group L out as entry i of its
// XCD's range (xcd_queue_claim), and in the steady state the XCD's `period` resident workgroups
// claim about `period` groups per group duration, so i / period tracks the time at which L
// starts. Walking L's list cyclically from the fraction (i mod period) / period of it puts all
// groups that run at once at about the same fraction of their walks, i.e. (walk order above) on
// about the same key blocks: the XCD's working set shrinks to a window of the head's K/V (14B
// layer: 22 % fewer bytes fetched beyond L2, about 2 % less time). Returns the first entry of a
// list of E entries.
__host__ __device__ inline int walk_start(int L, int total, int period, int E) {
  if (period <= 0 || E <= 0) return 0;
  const int q = total / kNumXcd, rem = total % kNumXcd;
  const int i = L < rem * (q + 1) ? L % (q + 1) : (L - rem * (q + 1)) % q;
  return (int)((long long)(i % period) * E / period);
}

// G query blocks share a workgroup of the attention kernel: G consecutive ones, or with G = 2 and
// a pair table the two that pair_greedy_kernel matched. For each (b, h, group) this writes the
// entry count and then the union of the G block lists in walk order (above), rotated to start at
// walk_start, each entry J | (bit i: query block i of the group selected J) << 16. Built through
// bitmaps indexed by walk position, so the lists may come in any order; out-of-range entries are
// dropped, as the attention skips them.
template <int G>
__global__ __launch_bounds__(256) void group_union_kernel(int nb, int keep, int ngroups, int stride,
                                                          const int32_t* __restrict__ idx,
                                                          const int32_t* __restrict__ pairs,
                                                          int32_t* __restrict__ out,
                                                          int* __restrict__ queue, int period) {
  extern __shared__ uint32_t sh[];
  const int kb = walk_bits(nb);
  const int words = walk_words(nb);
  uint32_t* bits = sh;                                 // [G][words]: membership of each list
  int* scan = reinterpret_cast<int*>(sh + G * words);  // [256]
  const long gp = blockIdx.x;
  const long head = gp / ngroups;
  const int I0 = G * (int)(gp % ngroups);
  const int tid = threadIdx.x;
  if (queue && gp == 0 && tid < kNumXcd) queue[tid * kQueueStride] = 0;  // the attention kernel's queue
  for (int w = tid; w < G * words; w += 256) bits[w] = 0u;
  __syncthreads();
  const int pr = G == 2 && pairs ? pairs[gp] : 0;
  for (int b = 0; b < G; ++b) {
    const int Ib = G == 2 && pairs ? (b ? pr >> 16 : pr & 0xFFFF) : I0 + b;
    if (Ib >= nb) break;
    const int32_t* sel = idx + (head * nb + Ib) * (long)keep;
    for (int i = tid; i < keep; i += 256) {
      const int J = sel[i];
      if ((unsigned)J < (unsigned)nb) {
        const int p = walk_pos(J, kb);
        atomicOr(&bits[b * words + (p >> 5)], 1u << (p & 31));
      }
    }
  }
  __syncthreads();
  const int per = (words + 255) / 256, w0 = min(words, tid * per), w1 = min(words, w0 + per);
  int cnt = 0;
  for (int w = w0; w < w1; ++w) {
    uint32_t u = 0;
#pragma unroll
    for (int b = 0; b < G; ++b) u |= bits[b * words + w];
    cnt += __popc(u);
  }
  scan[tid] = cnt;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {  // inclusive scan of the per-thread counts
    const int v = tid >= off ? scan[tid - off] : 0;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  int32_t* o = out + gp * (long)stride;
  const int E = scan[255];
  if (tid == 255) o[0] = E;
  const int e0 = walk_start((int)gp, (int)gridDim.x, period, E);
  int pos = scan[tid] - cnt - e0;  // rotated position of this thread's first entry
  if (pos < 0) pos += E;
  for (int w = w0; w < w1; ++w) {
    uint32_t m[G], u = 0;
#pragma unroll
    for (int b = 0; b < G; ++b) u |= (m[b] = bits[b * words + w]);
    for (; u; u &= u - 1) {
      const int bit = __ffs(u) - 1;
      uint32_t mask = 0;
#pragma unroll
      for (int b = 0; b < G; ++b) mask |= ((m[b] >> bit) & 1u) << b;
      o[1 + pos] = walk_pos(w * 32 + bit, kb) | (int)(mask << 16);  // the reversal is its own inverse
      if (++pos == E) pos = 0;
    }
  }
}

// ---- fused low-rank readout + gated combine in the attention epilogue ------------------------------
// (eq. ctx readout, eq. gate; Algorithm steps 7-10) for the 32 queries of a wave, whose O^s sits in
// the accumulators: lane l holds query l%32 and channels 32w + 8j + 4(l/32) + i in acc[w][4j + i].
//   Phi = P_q Q^n    on v_mfma_f32_32x32x16_bf16 per tile of 16 rotary pairs: A rows 0-15 = even
//                    rows of P_q, rows 16-31 = odd rows, B = Q^n in the layout Q^r has in the main
//                    loop, so both members of a pair land in one lane (c[4j+i] and c[4j+8+i]);
//   q~ = R_r SiLU(Phi) in registers, split into bf16 hi + lo;
//   u^T = C^T q~     A = C^T fragments prepared per head by cfrag_kernel (hi + lo), k ordered as the
//                    lanes hold q~; three MFMAs per k-step (hi.hi, lo.hi, hi.lo) as in the standalone
//                    readout, so the contraction is accurate to ~2^-16;
//   O = O^s + (sigma(logit) r_s / rms(u)) u  with r_s, rms(u) over the 128 channels (in-lane sums
//                    plus one permlane32 swap); O lands in the accumulators' layout.
struct FuseArgs {
  const bf16* Qn;        // [B, H, N, 128]
  const bf16* Pq;        // [H, r, 128]
  const float* cos_tab;  // [N, ld]
  const float* sin_tab;
  const uint4* cfrag;    // cfrag_kernel output
  const float* logits;   // [B, N]
  int H, r, ld;
  float eps_lr, eps;
  float* lse_out;        // optional [B, H, N]: log2 of the softmax denominator of the scaled scores
  int rot_q;             // the attention's Q is Q^n, rotated in the prologue with these tables
};

// C^T fragments: entry (head, w, t, s, lane) = {hi, lo} of the 8 values C[2J + s][32w + l%32],
// J = 16t + 8(m/4) + 4(l/32) + m%4 for m = 0..7 (zero for J >= r/2).
__global__ __launch_bounds__(256) void cfrag_kernel(long total, int r, int RJ,
                                                    const float* __restrict__ C,
                                                    uint4* __restrict__ out) {
  const long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= total) return;
  const int lane = (int)(e % 64);
  const int ts = (int)((e / 64) % (2 * RJ)), w = (int)((e / (64 * 2 * RJ)) % 4);
  const long head = e / (64L * 2 * RJ * 4);
  const int t = ts / 2, sd = ts % 2, half = r / 2;
  const int c = 32 * w + lane % 32, h = lane / 32;
  const float* Ch = C + head * (long)r * 128;
  bf16x8 hi, lo;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const int J = 16 * t + 8 * (m / 4) + 4 * h + m % 4;
    const float v = J < half ? Ch[(long)(2 * J + sd) * 128 + c] : 0.f;
    hi[m] = (bf16)v;
    lo[m] = (bf16)(v - (float)hi[m]);
  }
  out[2 * e] = *reinterpret_cast<const uint4*>(&hi);
  out[2 * e + 1] = *reinterpret_cast<const uint4*>(&lo);
}

template <int RJ>
__device__ __forceinline__ void fuse_epilogue(const FuseArgs& fz, f32x16 (&acc)[4], float l,
                                              bool qvalid, long head, int N, int q, int lane,
                                              bf16* __restrict__ O) {
  constexpr int D = 128;
  // the query index through an empty asm: the epilogue's address arithmetic is not hoisted in front
  // of the main loop, where it held registers across it (and spilled); the per-query offsets are
  // 32-bit (the ABI bounds N d_h and N rope_ld below 2^31)
  asm volatile("" : "+v"(q));
  const int hh = lane / 32, half = fz.r / 2;
  const int h = (int)(head % fz.H);
  const long bidx = head / fz.H;
  // O^s and its RMS
  const float inv = qvalid ? 1.0f / l : 0.f;
  float ss = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      acc[w][k] *= inv;
      ss = fmaf(acc[w][k], acc[w][k], ss);
    }
  {
    const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(ss), __float_as_uint(ss), false, false);
    ss = __uint_as_float(x[0]) + __uint_as_float(x[1]);
  }
  const float rs = sqrtf(ss * (1.0f / D) + fz.eps);
  // Q^n operand (query q, d = 16s + 8(l/32) .. +7) and the token's gate logit
  const bf16* Qq = fz.Qn + head * (long)N * D + (uint32_t)q * (uint32_t)D;
  bf16x8 qn[8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
    qn[s] = qvalid ? *reinterpret_cast<const bf16x8*>(Qq + 16 * s + 8 * hh) : bf16x8{};
  const float lg = qvalid ? fz.logits[bidx * N + q] : 0.f;
  f32x16 u[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) u[w] = f32x16{};
#pragma unroll
  for (int t = 0; t < RJ; ++t) {
    const int rho = lane % 32, pair = 16 * t + (rho & 15);
    const bool pok = pair < half;
    const bf16* Pr = fz.Pq + ((long)h * fz.r + 2 * pair + (rho >> 4)) * D + 8 * hh;
    f32x16 ph = f32x16{};
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const bf16x8 pa = pok ? *reinterpret_cast<const bf16x8*>(Pr + 16 * s) : bf16x8{};
      ph = mfma32(pa, qn[s], ph);
    }
    // features of this lane's pairs J = 16t + 8jp + 4(l/32) + i: e in ph[4jp+i], o in ph[4jp+8+i]
    bf16x8 beh, bel, boh, bol;
#pragma unroll
    for (int jp = 0; jp < 2; ++jp) {
      const int J0 = 16 * t + 8 * jp + 4 * hh;  // half is a multiple of 8: 4 pairs valid or none
      float4 c4 = {1.f, 1.f, 1.f, 1.f}, s4 = {0.f, 0.f, 0.f, 0.f};
      if (qvalid && J0 < half) {
        c4 = *reinterpret_cast<const float4*>(fz.cos_tab + (uint32_t)q * (uint32_t)fz.ld + J0);
        s4 = *reinterpret_cast<const float4*>(fz.sin_tab + (uint32_t)q * (uint32_t)fz.ld + J0);
      }
      const float cc[4] = {c4.x, c4.y, c4.z, c4.w}, sn[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float a = silu(ph[4 * jp + i]), b = silu(ph[4 * jp + 8 + i]);
        const float qe = a * cc[i] - b * sn[i], qo = a * sn[i] + b * cc[i];
        beh[4 * jp + i] = (bf16)qe;
        bel[4 * jp + i] = (bf16)(qe - (float)beh[4 * jp + i]);
        boh[4 * jp + i] = (bf16)qo;
        bol[4 * jp + i] = (bf16)(qo - (float)boh[4 * jp + i]);
      }
    }
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int sd = 0; sd < 2; ++sd) {
        const uint4* fr = fz.cfrag + ((((head * 4 + w) * (2 * RJ) + 2 * t + sd) * 64) + lane) * 2;
        const uint4 fh = fr[0], fl = fr[1];
        const bf16x8 ah = *reinterpret_cast<const bf16x8*>(&fh);
        const bf16x8 al = *reinterpret_cast<const bf16x8*>(&fl);
        const bf16x8& bh = sd ? boh : beh;
        const bf16x8& bl = sd ? bol : bel;
        u[w] = mfma32(ah, bh, u[w]);
        u[w] = mfma32(al, bh, u[w]);
        u[w] = mfma32(ah, bl, u[w]);
      }
  }
  float su = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int k = 0; k < 16; ++k) su = fmaf(u[w][k], u[w][k], su);
  {
    const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(su), __float_as_uint(su), false, false);
    su = __uint_as_float(x[0]) + __uint_as_float(x[1]);
  }
  const float inv_u = rsqrtf(su * (1.0f / D) + fz.eps_lr);
  // (O^s / r_s + g O^lr) r_s  ==  O^s + (g r_s / rms(u)) u
  const float coef = sigmoid(lg) * rs * inv_u;
  if (qvalid) {
    bf16* Oq = O + head * (long)N * D + (uint32_t)q * (uint32_t)D;
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (bf16)fmaf(coef, u[w][4 * j + i], acc[w][4 * j + i]);
        *reinterpret_cast<bf16x4*>(Oq + 32 * w + 8 * j + 4 * hh) = o;
      }
  }
}

// Query block qb of group grp: from the pair table when there is one (G = 2), else grp*G + qb.
template <int G>
__device__ __forceinline__ int group_block(const int32_t* pairs, long entry, int grp, int qb) {
  if (G != 2 || !pairs) return grp * G + qb;
  typedef const __attribute__((address_space(4))) int32_t* const_i32;
  const int pr = ((const_i32)pairs)[entry];
  return qb ? pr >> 16 : pr & 0xFFFF;
}

// bf16 attention kernel: one workgroup per (b, h, G query blocks); see the file comment.
// lists: G = 1: the block lists [B, H, nb, list_stride] (list_len entries used); G > 1:
//        group_union_kernel output, list_stride ints per (b, h, group); nullptr: every key block in
//        order for all query blocks of the group (list_len = nb).
// RJ > 0: the epilogue also computes the low-rank readout (r <= 32 RJ) and the gated combine
// (fuse_epilogue) and writes O instead of O^s.
struct AttnArgs {
  int N, nb, ngroups, total;  // total = B * H * ngroups groups
  const int32_t* lists;
  int list_len, list_stride;
  const int32_t* pairs;
  float scale_log2;
  const bf16* Q;
  const bf16* K;
  const bf16* V;
  bf16* O;
  FuseArgs fz;
  int* queue;  // QUEUE: kNumXcd counters, zero at launch
  // dQ mode: dO^s, the per-query {lse, D = dO^s . O^s} and the output dQ^r (fp32), scale
  const bf16* dO;
  const float2* lseD;
  float* dQ;
  float scale;
  int rot_q;  // Q holds Q^n: the prologue rotates it with fz's tables (rounded as rola_rope_apply)
  const float* knorm;  // BOUND: per key block the largest norm of its keys, [B, H, nb]
};

// DQ: the backward's dQ^r = scale dS K^r over the same groups and lists (fine-tuning, Sec. 4.5):
// per sub-tile S^T = K Q^T and dP^T = V dO^T (keys as rows, one lane per query, as the forward's
// S^T), P = exp2(S^T scale log2e - lse) with the forward's log-sum-exp, dS^T = P (dP^T - D), and
// dQ^T += K^T dS^T with K^T through transposing reads in the order the registers hold the keys. K
// and V tiles use the swizzle that serves both row and transposing reads (bw_swizzle).
// BOUND (merged lists, G > 1): the softmax reference of each wave is the bound on its scores that
// the key-block norms give, where that bound is small enough (see the prologue).
template <int BLK, int G, int NBUF, int TAB, int RJ, bool QUEUE, bool DQ = false, bool BOUND = false>
__global__ __launch_bounds__(G * BLK * 2, QUEUE && RJ < 2 && !DQ ? 3 : 2) void sparse_attn_kernel(
    const AttnArgs args) {
  static_assert(G == 1 || G == 2 || G == 4, "one, two or four query blocks per workgroup");
  static_assert(NBUF >= 3, "loads of later sub-tiles stay in flight during a step");
  constexpr int D = 128, WPB = BLK / 32, NW = G * WPB;
  constexpr int TILE = kSub * D * 2;              // 8 KB: K (or V) of one sub-tile
  constexpr int STAGE = 2 * TILE;                 // K then V
  constexpr int DMA_PER_WAVE = TILE / 1024 / NW;  // 1 KB loads per wave per tensor and sub-tile
  constexpr int SUBS = BLK / kSub;                // sub-tiles per key block
  static_assert(DMA_PER_WAVE >= 1, "at most 8 waves");
  __shared__ __attribute__((aligned(1024))) char lds[NBUF * STAGE];
  __shared__ int tab[TAB > 0 ? TAB : 1];  // the workgroup's block list (TAB > 0)

  const int wave = wave_uniform(threadIdx.x / 64);  // wave-uniform: LDS DMA bases in SGPRs

  // One group (b, h, G query blocks), logical id L in [0, total). With the work queue the
  // arguments and the lane index are re-derived per group through opaque values: otherwise the
  // compiler hoists everything derived from them out of the group loop, and the kernel, already at
  // the SGPR limit, spills them into VGPRs and loses a workgroup per CU.
  auto run = [&](const int L) {
    typedef const __attribute__((address_space(4))) AttnArgs* args_ptr;
    // the only explicit argument, at offset 0 of the kernel-argument segment
    args_ptr ap = (args_ptr)__builtin_amdgcn_kernarg_segment_ptr();
    int lane;
    if constexpr (QUEUE) {
      asm volatile("" : "+s"(ap));
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
    } else {
      lane = threadIdx.x % 64;
    }
    const int tid = wave * 64 + lane;
    const int N = ap->N, nb = ap->nb, ngroups = ap->ngroups;
    const int list_len = ap->list_len, list_stride = ap->list_stride;
    const int32_t* __restrict__ lists = ap->lists;
    const int32_t* __restrict__ pairs = ap->pairs;
    const float scale_log2 = ap->scale_log2;
    const bf16* __restrict__ Q = ap->Q;
    const bf16* __restrict__ K = ap->K;
    const bf16* __restrict__ V = ap->V;
    bf16* __restrict__ O = ap->O;
    const FuseArgs& fz = *(const FuseArgs*)&ap->fz;
    const int hh = lane / 32;
    const int qb = wave / WPB;  // which of the group's query blocks this wave serves
    // Per-lane LDS offsets. DMA: lane l of 1-KB slot s fills row 4s + l/16 at chunk position l%16
    // with source chunk (position ^ swizzle(row)). K operand of k-step s: row l%32, chunk 2s + l/32.
    // V^T operand of channel tile w: the lane supplies row 4(l/32) + (l%16)/4 (plus 16u + 8 for the
    // second four keys of k-step u) and channels 32w + 16((l/16)%2) + 4(l%4) .. +3.
    uint32_t dk[DMA_PER_WAVE], dv[DMA_PER_WAVE];
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) {
      const int row = 4 * (wave * DMA_PER_WAVE + i) + lane / 16, pos = lane % 16;
      dk[i] = row * D * 2 + ((pos ^ (DQ ? bw_swizzle(row) : k_swizzle(row))) << 4);
      dv[i] = row * D * 2 + ((pos ^ (DQ ? bw_swizzle(row) : v_swizzle(row))) << 4);
    }
    int ko[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int row = lane % 32;
      ko[s] = row * 256 + (((2 * s + hh) ^ k_swizzle(row)) << 4);
    }
    int vo[4];
    {
      const int i16 = lane % 16, row = 4 * hh + i16 / 4;
      const int c = 2 * ((lane / 16) & 1) + ((i16 & 3) >> 1);
#pragma unroll
      for (int w = 0; w < 4; ++w)
        vo[w] = TILE + row * 256 + (((4 * w + c) ^ v_swizzle(row)) << 4) + 8 * (i16 & 1);
    }
    const uint32_t lds0 = lds_address(lds);
    const int grp = L % ngroups;
    const long head = L / ngroups;
    const int I = group_block<G>(pairs, head * ngroups + grp, grp, qb);  // nb: missing second block
    const int q = I * BLK + (wave % WPB) * 32 + lane % 32;  // this lane's query (column of S^T, O^T)
    const bool qvalid = I < nb && q < N;
    const int mybit = 1 << qb;
    const bf16* Qh = Q + head * (long)N * D;
    const char* Kh = reinterpret_cast<const char*>(K + head * (long)N * D);
    const char* Vh = reinterpret_cast<const char*>(V + head * (long)N * D);

    // The workgroup's block list: with TAB > 0 it is copied into LDS once (E <= TAB) and each step
    // reads the entries of the next step, which the barrier of that step finds complete, so list reads
    // never stall a step; otherwise entries come through uniform scalar loads.
    typedef const __attribute__((address_space(4))) int32_t* const_i32;
    const int32_t* glist = nullptr;
    int E = list_len;
    if (lists && G > 1) {
      glist = lists + (head * ngroups + grp) * (long)list_stride;
      E = ((const_i32)glist)[0];
      glist += 1;
    } else if (lists) {
      glist = lists + (head * nb + grp) * (long)list_stride;
    }
    const const_i32 slist = (const_i32)glist;
    const int T = E * SUBS;  // sub-tiles the workgroup walks
    float kmax = 0.f;        // BOUND: the largest key-block norm among the group's entries
    if (TAB > 0 && glist) {
      for (int i = tid; i < E; i += NW * 64) {
        const int v = glist[i];
        tab[i] = v;
        if (BOUND && (v & 0xFFFF) < nb) kmax = fmaxf(kmax, ap->knorm[head * nb + (v & 0xFFFF)]);
      }
    } else if (BOUND && glist) {
      for (int i = tid; i < E; i += NW * 64) {
        const int v = glist[i];
        if ((v & 0xFFFF) < nb) kmax = fmaxf(kmax, ap->knorm[head * nb + (v & 0xFFFF)]);
      }
    }
    struct Step {
      int k0;    // first key, -1 if the block index is out of range
      int mask;  // query blocks of the group that selected the block
    };
    // raw(e): entry e of the list (in a VGPR when it comes from the LDS table); step_of decodes the
    // entry of sub-tile t.
    auto raw = [&](int e) -> int {
      // the table is only used with a list (TAB > 0: never the dense walk), which saves a branch
      // per lookup (about 2 % of the kernel)
      if (TAB == 0 && !glist) return G > 1 ? (e | (((1 << G) - 1) << 16)) : e;  // dense: every block
      const int i = min(e, max(E - 1, 0));
      return TAB > 0 ? tab[i] : (int)slist[i];
    };
    auto step_of = [&](int v, int t) {
      v = TAB > 0 ? wave_uniform(v) : v;
      const int J = G > 1 ? (v & 0xFFFF) : v;
      const int mask = G > 1 ? (v >> 16) : 1;
      return Step{(unsigned)J < (unsigned)nb ? J * BLK + (int)((unsigned)t % SUBS) * kSub : -1, mask};
    };

    // Q^T fragments of the 8 k-steps (d = 16s + 8(l/32) .. +7) stay in registers. They are complete
    // before the first K/V load is issued: a wait for them inside the loop would also drain the
    // K/V loads in flight.
    bf16x8 qf[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
      qf[s] = qvalid ? *reinterpret_cast<const bf16x8*>(Qh + (uint32_t)q * (uint32_t)D + 16 * s + 8 * hh) : bf16x8{};
    if (ap->rot_q && qvalid) {  // Q^r = R(Q^n): pairs 8s + 4(l/32) .. +3 of this lane's query
      const float* ct = fz.cos_tab + (uint32_t)q * (uint32_t)fz.ld + 4 * hh;
      const float* st = fz.sin_tab + (uint32_t)q * (uint32_t)fz.ld + 4 * hh;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const float4 c = *reinterpret_cast<const float4*>(ct + 8 * s);
        const float4 sn = *reinterpret_cast<const float4*>(st + 8 * s);
        const float cc[4] = {c.x, c.y, c.z, c.w}, ss[4] = {sn.x, sn.y, sn.z, sn.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          float x, y;
          rope_pair((float)qf[s][2 * p], (float)qf[s][2 * p + 1], cc[p], ss[p], x, y);
          qf[s][2 * p] = (bf16)x;
          qf[s][2 * p + 1] = (bf16)y;
        }
      }
    }
    bf16x8 df[DQ ? 8 : 1];  // dQ mode: dO^T fragments, same layout as qf
    float lse_q = 0.f, dsum_q = 0.f;
    if constexpr (DQ) {
      const bf16* dOq = ap->dO + head * (long)N * D + (uint32_t)q * (uint32_t)D;
#pragma unroll
      for (int s = 0; s < 8; ++s)
        df[s] = qvalid ? *reinterpret_cast<const bf16x8*>(dOq + 16 * s + 8 * hh) : bf16x8{};
      const float2 v = qvalid ? ap->lseD[head * (long)N + q] : make_float2(INFINITY, 0.f);
      lse_q = v.x;
      dsum_q = v.y;
    }
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    __shared__ float kmax_w[BOUND ? NW : 1];
    if constexpr (BOUND) {
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) kmax = fmaxf(kmax, __shfl_xor(kmax, off));
      if (lane == 0) kmax_w[wave] = kmax;
    }
    if (TAB > 0 || BOUND) __syncthreads();  // the list table and the per-wave maxima are complete

    f32x16 acc[4];        // O^T channel tiles 32w .. 32w+31
    float m = -INFINITY;  // reference max (log2 units) of this lane's query
    // BOUND: with b the largest norm of the keys the group selected, each scaled score of query q
    // lies in [-B, B], B = scale_log2 |q| b, so m = B keeps every probability in [2^-2B, 1] and the
    // walk needs no running max and no rescale. A wave where some B exceeds kBoundMax (or is not
    // finite) tracks the running max instead. fixed_m is wave-uniform.
    int fixed_m = 0;
    if constexpr (BOUND) {
      float b = kmax_w[0];
#pragma unroll
      for (int i = 1; i < NW; ++i) b = fmaxf(b, kmax_w[i]);
      typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
      float q2 = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const bf16x2_t v = {qf[s][e], qf[s][e + 1]};
          q2 = __builtin_amdgcn_fdot2_f32_bf16(v, v, q2, false);
        }
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(q2), __float_as_uint(q2), false, false);
      q2 = __uint_as_float(x[0]) + __uint_as_float(x[1]);
      const float bound = scale_log2 * sqrtf(q2) * b;
      fixed_m = __any(!(bound <= kBoundMax)) ? 0 : 1;
      if (fixed_m) m = bound;
    }
    float l = 0.f;        // running sum of this lane's 16 keys per sub-tile (the other 16: lane l^32)
#pragma unroll
    for (int w = 0; w < 4; ++w) acc[w] = f32x16{};

    auto issue = [&](const Step& s, int buf) {  // always 2 * DMA_PER_WAVE loads (fixed vmcnt per step)
      const int k0 = max(s.k0, 0);
      const uint32_t dst = lds0 + buf * STAGE;
      if (k0 + kSub <= N) {
        const char* kb = Kh + (long)k0 * D * 2;
        const char* vb = Vh + (long)k0 * D * 2;
#pragma unroll
        for (int i = 0; i < DMA_PER_WAVE; ++i) {
          const uint32_t slot = (wave * DMA_PER_WAVE + i) * 1024;
          dma16(kb, dk[i], dst + slot);
          dma16(vb, dv[i], dst + TILE + slot);
        }
      } else {  // ragged tail: rows past N re-read row N-1 (a valid key, see mask_tail)
#pragma unroll
        for (int i = 0; i < DMA_PER_WAVE; ++i) {
          const uint32_t slot = (wave * DMA_PER_WAVE + i) * 1024;
          const int r = 4 * (wave * DMA_PER_WAVE + i) + lane / 16;
          const uint32_t row = (uint32_t)(min(k0 + r, N - 1) - r) * (D * 2);
          dma16(Kh, row + dk[i], dst + slot);
          dma16(Vh, row + dv[i], dst + TILE + slot);
        }
      }
    };

    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    auto load_k = [&](int buf, int s0, bf16x8 (&kf)[4]) {  // K operands of k-steps s0 .. s0+3
#pragma unroll
      for (int s = 0; s < 4; ++s)
        kf[s] = *reinterpret_cast<const bf16x8*>(lds + buf * STAGE + ko[s0 + s]);
    };
    auto v_operand = [&](int buf, int u, int w) {  // V^T operand of channel tile w, key k-step u
      const char* p = lds + buf * STAGE + vo[w] + 16 * u * 256;
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 8 * 256));
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    };
    auto load_v = [&](int buf, int u, bf16x8 (&vf)[4]) {  // V^T operands of key k-step u
#pragma unroll
      for (int w = 0; w < 4; ++w) vf[w] = v_operand(buf, u, w);
    };
    // Softmax pieces on S^T of one sub-tile (16 keys of this lane's query; the other 16 in lane l^32).
    auto row_max = [&](const f32x16& s) {
      float mx = s[0];
#pragma unroll
      for (int k = 1; k < 16; ++k) mx = fmaxf(mx, s[k]);
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      return fmaxf(__uint_as_float(x[0]), __uint_as_float(x[1])) * scale_log2;
    };
    auto rescale = [&](float mt) {  // lazy: only when the max grew by more than 2^tau
      if (__any(mt > m + kRescaleTau)) {
        const float mnew = fmaxf(m, mt);
        const float alpha = __builtin_amdgcn_exp2f(m - mnew);
        m = mnew;
        l *= alpha;
#pragma unroll
        for (int w = 0; w < 4; ++w) acc[w] *= alpha;
      }
    };
    // Rows of a ragged last sub-tile repeat key N-1, whose score is a valid one: they leave the row
    // max unchanged and only their probabilities are zeroed. The row sum adds exactly the bf16
    // probabilities that enter P V (v_dot2 against (1, 1), fp32 accumulation).
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    auto probs = [&](const f32x16& s, int k0, int tail, bf16x8 (&pb)[2]) {
#pragma unroll
      for (int k = 0; k < 16; ++k)
        pb[k / 8][k % 8] = (bf16)__builtin_amdgcn_exp2f(fmaf(s[k], scale_log2, -m));
      if (tail) {  // value k holds key k0 + 8(k/4) + 4(l/32) + k%4
        const int lim = N - k0 - 4 * hh;
#pragma unroll
        for (int k = 0; k < 16; ++k)
          if (8 * (k / 4) + k % 4 >= lim) pb[k / 8][k % 8] = (bf16)0.f;
      }
      const bf16x2 one2 = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
      for (int k = 0; k < 16; k += 2)
        l = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[k / 8][k % 8], pb[k / 8][k % 8 + 1]}, one2, l, false);
    };
    auto qk = [&](int s0, const bf16x8* kf, f32x16& sacc, int n) {  // k-steps s0 .. s0+n-1
#pragma unroll
      for (int s = 0; s < n; ++s) sacc = mfma32(kf[s], qf[s0 + s], sacc);
    };

    // Pipeline: step t waits for the loads of sub-tile t and a barrier, issues the loads of sub-tile
    // t+NBUF-1 into the buffer sub-tile t-1 has released, then S = QK(t), softmax, O += P V(t). The
    // second wave on each SIMD overlaps its matrix and vector work with this one's. Unrolled by NBUF
    // so each buffer is a compile-time offset.
    constexpr int PER_STEP = 2 * DMA_PER_WAVE;  // vector-memory instructions per wave per sub-tile
    int issued = 0;
#pragma unroll
    for (int j = 0; j < NBUF - 1; ++j)
      if (j < T) {
        issue(step_of(raw(j / SUBS), j), j);
        ++issued;
      }
    int pi = raw((unsigned)issued / SUBS), pc = raw(0);  // entries the next step decodes
    for (int t = 0; t < T;) {
#pragma unroll
      for (int j = 0; j < NBUF; ++j) {
        if (t >= T) break;
        // This step's entry and the one whose loads it issues are decoded before the wait and the
        // barrier: only the loads themselves must follow the barrier, so the scalar decoding no
        // longer sits between the barrier and the step's first LDS reads and products.
        Step cur = step_of(pc, t), nxt = step_of(pi, issued);
        cur.k0 = wave_uniform(cur.k0);
        nxt.k0 = wave_uniform(nxt.k0);
        const int cmask = wave_uniform(cur.mask);
        // whether this wave computes the step, in scalar arithmetic: k0 >= 0 && k0 < N as one
        // unsigned compare
        int act = wave_uniform(((cmask & mybit) != 0) & ((unsigned)cur.k0 < (unsigned)N));
        int ctail = wave_uniform(cur.k0 + kSub > N);  // ragged last sub-tile
        const bool more = issued < T;
        // (pinned here: the compiler would otherwise sink the decoding to its uses)
        asm volatile("" : "+s"(cur.k0), "+s"(nxt.k0), "+s"(act), "+s"(ctail));
        if (issued == t + NBUF - 1) {  // loads of t+1 .. t+NBUF-2 may stay in flight
          constexpr int allowed = PER_STEP * (NBUF - 2);
          __builtin_amdgcn_s_waitcnt((allowed & 15) | ((allowed >> 4) << 14) | (7 << 4) | (15 << 8));
        } else {
          __builtin_amdgcn_s_waitcnt(0);
        }
        __syncthreads();  // sub-tile t landed for every wave; every wave is done with sub-tile t-1
        if (more) {
          issue(nxt, (j + NBUF - 1) % NBUF);
          ++issued;
        }
        pi = raw((unsigned)issued / SUBS);
        pc = raw((unsigned)(t + 1) / SUBS);
        if (DQ && act) {
          const char* Kt = lds + j * STAGE;
          const char* Vt = Kt + TILE;
          f32x16 sc = f32x16{}, dp = f32x16{};
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            sc = mfma32(row_frag(Kt, lane % 32, s, hh), qf[s], sc);
            dp = mfma32(row_frag(Vt, lane % 32, s, hh), df[s], dp);
          }
          // value k: key k0 + 8(k/4) + 4(l/32) + k%4 of this lane's query
          float pr[16];
#pragma unroll
          for (int k = 0; k < 16; ++k) pr[k] = __builtin_amdgcn_exp2f(fmaf(sc[k], scale_log2, -lse_q));
          if (cur.k0 + kSub > N) {  // ragged last block: keys past N
            const int lim = N - cur.k0 - 4 * hh;
#pragma unroll
            for (int k = 0; k < 16; ++k) pr[k] = 8 * (k / 4) + k % 4 < lim ? pr[k] : 0.f;
          }
          bf16x8 ds[2];
#pragma unroll
          for (int k = 0; k < 16; ++k) ds[k / 8][k % 8] = (bf16)(pr[k] * (dp[k] - dsum_q));
          __builtin_amdgcn_s_setprio(1);  // as the forward's P V products (sparse backward -0.8 %)
#pragma unroll
          for (int w = 0; w < 4; ++w)
#pragma unroll
            for (int u = 0; u < 2; ++u) acc[w] = mfma32(tr_frag(Kt, w, u, lane), ds[u], acc[w]);
          __builtin_amdgcn_s_setprio(0);
        } else if (!DQ && act) {
          bf16x8 kf[4], kg[4], vf[4], pb[2];
          load_k(j, 0, kf);
          load_k(j, 4, kg);
          f32x16 sc = mfma32(kf[0], qf[0], f32x16{});
          qk(1, kf + 1, sc, 3);
          qk(4, kg, sc, 4);
          // four K operand reads ahead of the chain of eight dependent products, then one read per
          // product (the default schedule kept two in flight: 12.95 -> 12.82 ms for the fused call
          // on the 14B layer, bitwise identical)
          __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // DS reads
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
          load_v(j, 0, vf);
          // (BOUND re-reads the flag as uniform: taken as a per-lane value, the branch keeps the
          // step's registers live on both sides and the kernel spills)
          if (!BOUND || !wave_uniform(fixed_m)) rescale(row_max(sc));
          probs(sc, cur.k0, ctail, pb);
          // the P V products at raised wave priority: a wave that has its probabilities issues its
          // MFMAs ahead of the other waves' score and softmax work (plain attention on the 14B
          // layer: 12.80 -> 12.58 ms; the same priority around Q K^T costs a third more time).
          // The V^T operands of the second key step are read into each channel tile's registers
          // right behind that tile's first product, so their LDS latency hides under the other
          // three (fused call 12.90 -> 12.66 ms on one box, bitwise identical).
          __builtin_amdgcn_s_setprio(1);
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            acc[w] = mfma32(vf[w], pb[0], acc[w]);
            vf[w] = v_operand(j, 1, w);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // its tile's two DS reads
          }
#pragma unroll
          for (int w = 0; w < 4; ++w) acc[w] = mfma32(vf[w], pb[1], acc[w]);
          __builtin_amdgcn_s_setprio(0);
        }
        ++t;
      }
    }

    if constexpr (DQ) {  // dQ^T: lane = query, rows = channels 32w + 8j + 4(l/32) + i
      if (qvalid) {
        float* dq = ap->dQ + head * (long)N * D + (uint32_t)q * (uint32_t)D;
        const float sc = ap->scale;
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            *reinterpret_cast<float4*>(dq + 32 * w + 8 * jj + 4 * hh) =
                make_float4(acc[w][4 * jj] * sc, acc[w][4 * jj + 1] * sc, acc[w][4 * jj + 2] * sc,
                            acc[w][4 * jj + 3] * sc);
      }
      return;
    }
    {
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l), false, false);
      l = __uint_as_float(x[0]) + __uint_as_float(x[1]);
    }
    if (fz.lse_out && qvalid && hh == 0)  // sum_k exp2(x_k - m) = l: log2 sum exp2 x = m + log2 l
      fz.lse_out[head * (long)N + q] = m + __log2f(l);
    if constexpr (RJ > 0) {
      fuse_epilogue<RJ>(fz, acc, l, qvalid, head, N, q, lane, O);
      return;
    }
    if (qvalid) {
      const float inv = 1.0f / l;
      bf16* Oq = O + head * (long)N * D + (uint32_t)q * (uint32_t)D;
#pragma unroll
      for (int w = 0; w < 4; ++w)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bf16x4 o;
#pragma unroll
          for (int i = 0; i < 4; ++i) o[i] = (bf16)(acc[w][4 * j + i] * inv);
          *reinterpret_cast<bf16x4*>(Oq + 32 * w + 8 * j + 4 * hh) = o;
        }
    }
  };

  if constexpr (!QUEUE) {  // static grid: one group per workgroup, XCD-ordered
    run(xcd_remap(blockIdx.x, args.total));
  } else {  // a grid of resident workgroups claims groups until none are left (xcd_queue_claim)
    __shared__ int next_group;
    const int xcd = xcd_id();
    for (;;) {
      __syncthreads();  // every wave is done with the previous group's LDS stages, table and id
      if (threadIdx.x == 0) next_group = xcd_queue_claim(args.queue, xcd, args.total);
      __syncthreads();
      const int L = wave_uniform(next_group);
      if (L < 0) break;
      run(L);
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

// Workgroups of `kernel` (threads each) that the current device holds at once, cached per device
// in `cache` (one per kernel: every variant has the same function type).
constexpr int kMaxDevices = 64;
template <typename Kernel>
int resident_workgroups(Kernel kernel, int threads, std::atomic<int> (&cache)[kMaxDevices]) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = -1;
  if (dev >= 0) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev < 0 ? 0 : dev) != hipSuccess)
    cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess)
    per_cu = 0;
  (void)hipGetLastError();
  const int n = std::max(1, cus) * std::max(1, per_cu);
  if (dev >= 0) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

// The dQ mode's extra operands (sparse_attn_kernel<.., DQ = true>).
struct DqArgs {
  const bf16* dO;
  const float2* lseD;
  float* dQ;
};

// Resident workgroups of the work-queue variant of sparse_attn_kernel (a cache per variant).
template <int BLK, int G, int NBUF, int TAB, int RJ, bool DQ, bool BOUND = false>
int queue_resident() {
  static std::atomic<int> cache[kMaxDevices];
  return resident_workgroups(sparse_attn_kernel<BLK, G, NBUF, TAB, RJ, true, DQ, BOUND>, G * BLK * 2,
                             cache);
}

// queue: kNumXcd zeroed counters, or nullptr for the static grid of one workgroup per group.
template <int BLK, int G, int NBUF, int TAB, int RJ, bool DQ = false, bool BOUND = false>
hipError_t launch_bf16_tab(const Shape& s, const void* Qr, const void* Kr, const void* V,
                           const int32_t* lists, int list_len, int list_stride,
                           const int32_t* pairs, float scale, void* Os, const FuseArgs& fz,
                           int* queue, hipStream_t st, const DqArgs& dq = DqArgs{},
                           const float* knorm = nullptr) {
  const int nb = num_blocks(s.N, BLK);
  const int ngroups = (nb + G - 1) / G;
  const int total = ngroups * s.H * s.B;
  const float sl = scale * 1.4426950408889634f;
  const int threads = G * BLK * 2;
  const AttnArgs a{s.N, nb, ngroups, total, lists, list_len, list_stride, pairs, sl,
                   (const bf16*)Qr, (const bf16*)Kr, (const bf16*)V, (bf16*)Os, fz, queue,
                   dq.dO, dq.lseD, dq.dQ, scale, fz.rot_q, knorm};
  if (queue) {
    const int grid = std::min(total, queue_resident<BLK, G, NBUF, TAB, RJ, DQ, BOUND>());
    hipLaunchKernelGGL((sparse_attn_kernel<BLK, G, NBUF, TAB, RJ, true, DQ, BOUND>), dim3(grid),
                       dim3(threads), 0, st, a);
  } else {
    hipLaunchKernelGGL((sparse_attn_kernel<BLK, G, NBUF, TAB, RJ, false, DQ>), dim3(total),
                       dim3(threads), 0, st, a);
  }
  return hipGetLastError();
}

// Lists of up to kTable entries go through the LDS table; longer ones through scalar loads.
constexpr int kTable = 1024;
// knorm (merged lists with a work queue and a fused epilogue only): the BOUND variant.
template <int BLK, int G, int NBUF, int RJ>
hipError_t launch_bf16_rj(const Shape& s, const void* Qr, const void* Kr, const void* V,
                          const int32_t* lists, int list_len, int list_stride, float scale,
                          void* Os, const int32_t* pairs, const FuseArgs& fz, int* queue,
                          hipStream_t st, const float* knorm) {
  const int max_len = G > 1 ? list_stride - 1 : list_len;
  if constexpr (G > 1 && RJ > 0) {
    if (knorm && lists && queue) {
      if (max_len <= kTable)
        return launch_bf16_tab<BLK, G, NBUF, kTable, RJ, false, true>(
            s, Qr, Kr, V, lists, list_len, list_stride, pairs, scale, Os, fz, queue, st, DqArgs{},
            knorm);
      return launch_bf16_tab<BLK, G, NBUF, 0, RJ, false, true>(
          s, Qr, Kr, V, lists, list_len, list_stride, pairs, scale, Os, fz, queue, st, DqArgs{},
          knorm);
    }
  }
  if (lists && max_len <= kTable)
    return launch_bf16_tab<BLK, G, NBUF, kTable, RJ>(s, Qr, Kr, V, lists, list_len, list_stride,
                                                     pairs, scale, Os, fz, queue, st);
  return launch_bf16_tab<BLK, G, NBUF, 0, RJ>(s, Qr, Kr, V, lists, list_len, list_stride, pairs,
                                              scale, Os, fz, queue, st);
}

// fz.r == 0: plain attention (O^s); otherwise the fused epilogue with RJ = r / 32 tiles (r 16 -> 1).
template <int BLK, int G, int NBUF>
hipError_t launch_bf16(const Shape& s, const void* Qr, const void* Kr, const void* V,
                       const int32_t* lists, int list_len, int list_stride, float scale, void* Os,
                       hipStream_t st, const int32_t* pairs = nullptr, const FuseArgs* fz = nullptr,
                       int* queue = nullptr, const float* knorm = nullptr) {
  static const FuseArgs none{};
  if (!fz || fz->r == 0)
    return launch_bf16_rj<BLK, G, NBUF, 0>(s, Qr, Kr, V, lists, list_len, list_stride, scale, Os,
                                           pairs, fz ? *fz : none, queue, st, knorm);
  if (fz->r <= 32)
    return launch_bf16_rj<BLK, G, NBUF, 1>(s, Qr, Kr, V, lists, list_len, list_stride, scale, Os,
                                           pairs, *fz, queue, st, knorm);
  return launch_bf16_rj<BLK, G, NBUF, 2>(s, Qr, Kr, V, lists, list_len, list_stride, scale, Os,
                                         pairs, *fz, queue, st, knorm);
}

template <typename T, int D>
hipError_t launch_simple(const Shape& s, const void* Qr, const void* Kr, const void* V, int block,
                         int keep, const int32_t* idx, float scale, void* Os, hipStream_t st) {
  const int nb = num_blocks(s.N, block);
  hipLaunchKernelGGL((sparse_simple_kernel<T, D>), dim3(nb, s.H, s.B), dim3(block), 0, st, s.N,
                     block, nb, keep, idx, scale, (const T*)Qr, (const T*)Kr, (const T*)V, (T*)Os);
  return hipGetLastError();
}

// Query blocks per workgroup when a workspace for the merged lists is given.
int group_of(const Shape& s, int block) { return s.bf16 && block == 64 ? kB64Group : 1; }

// Pairs are matched by overlap when G = 2 and one overlap workgroup's bitmaps fit in 64 KB of LDS
// (up to 4064 query blocks); otherwise the pairs are adjacent blocks.
bool pairing_on(int G, int nb) {
  return G == 2 && kPairRows * pair_row_stride(nb) * 4 <= 65536 &&
         (nb + 1) / 2 <= kMaxPairGroups;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace: [work-queue counters: kNumXcd ints, 256 bytes apart][pair table: int32 per group, when
// pairing][union lists, which the candidate ranks (kPairWindow bytes per query block, whole
// chunks) occupy before the lists are written].
constexpr size_t kQueueBytes = kNumXcd * kQueueStride * sizeof(int);  // a 256-byte slot per counter
struct SparseWs {
  size_t queue_bytes, pair_bytes, list_bytes;
};
SparseWs sparse_ws_layout(const Shape& s, int block, int keep) {
  const int G = group_of(s, block);
  if (G == 1) return {0, 0, 0};
  const int nb = num_blocks(s.N, block);
  const size_t heads = (size_t)s.B * s.H, ngroups = (nb + G - 1) / G;
  size_t lists = heads * ngroups * ((size_t)G * keep + 1) * sizeof(int32_t);
  if (!pairing_on(G, nb)) return {kQueueBytes, 0, lists};
  const size_t nchunks = (nb + kPairWindow - 1) / kPairWindow;
  lists = std::max(lists, heads * nchunks * kPairWindow * kPairWindow);
  return {kQueueBytes, align256(heads * ngroups * sizeof(int32_t)), lists};
}

// Period of walk_start for the merged lists of the 64-token path: resident workgroups per XCD of
// the work-queue variant that will walk them (the table and epilogue variant launch_bf16_rj picks
// for lists of stride - 1 entries and rank r; the dQ mode has no epilogue).
template <int NBUF, bool DQ>
int walk_period(int stride, int r) {
  constexpr int G = kB64Group;
  int n;
  if constexpr (DQ) {
    n = stride - 1 <= kTable ? queue_resident<64, G, NBUF, kTable, 0, true>()
                             : queue_resident<64, G, NBUF, 0, 0, true>();
  } else if (stride - 1 <= kTable) {
    n = r == 0    ? queue_resident<64, G, NBUF, kTable, 0, false>()
        : r <= 32 ? queue_resident<64, G, NBUF, kTable, 1, false>()
                  : queue_resident<64, G, NBUF, kTable, 2, false>();
  } else {
    n = r == 0    ? queue_resident<64, G, NBUF, 0, 0, false>()
        : r <= 32 ? queue_resident<64, G, NBUF, 0, 1, false>()
                  : queue_resident<64, G, NBUF, 0, 2, false>();
  }
  return n / kNumXcd;
}

// Groups of the 64-token path in the workspace: pairs matched by overlap (or adjacent), their
// merged lists in walk order rotated to their start phases (walk_start), the work-queue counters
// cleared. r: rank of the fused epilogue (0: none); DQ: the lists are for the dQ mode.
struct Groups {
  int* queue;
  int32_t* pairs;
  int32_t* lists;
  int stride;
};
// Pointers of the groups inside the workspace (no device work).
Groups groups_in(const Shape& s, int keep, void* ws) {
  constexpr int G = kB64Group;
  const SparseWs lay = sparse_ws_layout(s, 64, keep);
  Groups gr;
  gr.stride = G * keep + 1;
  gr.queue = (int*)ws;
  gr.pairs = lay.pair_bytes ? (int32_t*)((char*)ws + lay.queue_bytes) : nullptr;
  gr.lists = (int32_t*)((char*)ws + lay.queue_bytes + lay.pair_bytes);
  return gr;
}

template <bool DQ>
hipError_t prepare_groups(const Shape& s, int keep, const int32_t* idx, void* ws, int r,
                          hipStream_t st, Groups& gr) {
  constexpr int G = kB64Group;
  const int nb = num_blocks(s.N, 64);
  const int ngroups = (nb + G - 1) / G, heads = s.B * s.H;
  gr = groups_in(s, keep, ws);
  if (gr.pairs) {
    const int nchunks = (nb + kPairWindow - 1) / kPairWindow;
    hipLaunchKernelGGL(pair_rank_kernel, dim3(nchunks * heads), dim3(256),
                       kPairRows * pair_row_stride(nb) * sizeof(uint32_t), st, nb, keep, nchunks,
                       idx, (uint8_t*)gr.lists);
    hipLaunchKernelGGL(pair_greedy_kernel, dim3(heads), dim3(64), 0, st, nb, ngroups, nchunks,
                       (const uint8_t*)gr.lists, gr.pairs);
  }
  const int period = walk_period<DQ ? 3 : kB64Nbuf, DQ>(gr.stride, r);
  hipLaunchKernelGGL(group_union_kernel<G>, dim3(ngroups * heads), dim3(256),
                     (G * walk_words(nb) + 256) * sizeof(uint32_t), st, nb, keep, ngroups, gr.stride,
                     idx, (const int32_t*)gr.pairs, gr.lists, gr.queue, period);
  return hipGetLastError();
}

// Device scratch of the allocation-free entry point: one copy per device, alive until the process
// ends. Host code never names the array itself (its host-side name is no device address): the
// address each device gives for it is asked once per device, with that device current, and kept.
constexpr size_t kStaticScratchBytes = ROLA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mutex;

}  // namespace

size_t sparse_workspace_bytes(const Shape& s, int block, int keep) {
  const SparseWs w = sparse_ws_layout(s, block, keep);
  return w.queue_bytes + w.pair_bytes + w.list_bytes;
}

size_t fuse_workspace_bytes(const Shape& s, int r) {
  if (!fuse_supported(s, r)) return 0;
  const size_t RJ = r <= 32 ? 1 : 2;
  return (size_t)s.B * s.H * 4 * 2 * RJ * 64 * 2 * sizeof(uint4);
}

bool fuse_supported(const Shape& s, int r) { return s.bf16 && s.d == 128 && r >= 16 && r <= 64; }

bool dq_supported(const Shape& s, int block) {
  return s.bf16 && s.d == 128 && block == 64;
}

hipError_t launch_sparse_dq(const Shape& s, const void* Qr, const void* Kr, const void* V, int keep,
                            const int32_t* idx, float scale, const void* dO, const void* lseD,
                            float* dQ, void* ws, hipStream_t st) {
  Groups gr;
  const hipError_t e = prepare_groups<true>(s, keep, idx, ws, 0, st, gr);
  if (e != hipSuccess) return e;
  const DqArgs dq{(const bf16*)dO, (const float2*)lseD, dQ};
  const FuseArgs none{};
  if (gr.stride - 1 <= kTable)
    return launch_bf16_tab<64, 2, 3, kTable, 0, true>(s, Qr, Kr, V, gr.lists, 0, gr.stride, gr.pairs,
                                                      scale, nullptr, none, gr.queue, st, dq);
  return launch_bf16_tab<64, 2, 3, 0, 0, true>(s, Qr, Kr, V, gr.lists, 0, gr.stride, gr.pairs, scale,
                                               nullptr, none, gr.queue, st, dq);
}

bool plan_used(const Shape& s, int block) { return s.bf16 && block == 64 && kB64Group > 1; }

hipError_t launch_sparse_plan(const Shape& s, int keep, const int32_t* idx, int r, void* ws,
                              hipStream_t st) {
  if (!plan_used(s, 64)) return hipSuccess;
  Groups gr;
  return prepare_groups<false>(s, keep, idx, ws, r, st, gr);
}

size_t static_scratch_bytes() { return kStaticScratchBytes; }

hipError_t static_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return hipSuccess;
}

hipError_t launch_sparse_attn(const Shape& s, const void* Qr, const void* Kr, const void* V,
                              int block, int keep, const int32_t* idx, float scale, void* Os,
                              void* ws, hipStream_t st, const LowrankFuse* lf, void* fuse_ws,
                              float* lse, bool planned) {
  FuseArgs fz{};
  fz.lse_out = lse;
  if (lf) {  // fused epilogue: C^T fragments first (fuse_ws: fuse_workspace_bytes)
    const int RJ = lf->r <= 32 ? 1 : 2;
    const long total = (long)s.B * s.H * 4 * 2 * RJ * 64;
    hipLaunchKernelGGL(cfrag_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, total,
                       lf->r, RJ, lf->C, (uint4*)fuse_ws);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    fz = FuseArgs{(const bf16*)lf->Qn, (const bf16*)lf->Pq, lf->cos_tab, lf->sin_tab,
                  (const uint4*)fuse_ws, lf->logits, s.H, lf->r, lf->ld, lf->eps_lr, lf->eps, lse,
                  Qr == nullptr ? 1 : 0};
    if (Qr == nullptr) Qr = lf->Qn;  // queries rotated from Q^n in the prologue
  }
  const FuseArgs* fp = (lf || lse) ? &fz : nullptr;
  if (s.bf16) {
    const int nb = num_blocks(s.N, block);
    if (block == 64) {
      constexpr int G = kB64Group;
      if (!idx) return launch_bf16<64, 2, 3>(s, Qr, Kr, V, nullptr, nb, 0, scale, Os, st, nullptr, fp);
      if (ws && G > 1) {
        Groups gr = groups_in(s, keep, ws);
        if (!planned) {
          const hipError_t e = prepare_groups<false>(s, keep, idx, ws, lf ? lf->r : 0, st, gr);
          if (e != hipSuccess) return e;
        }
        return launch_bf16<64, G, kB64Nbuf>(s, Qr, Kr, V, gr.lists, 0, gr.stride, scale, Os, st,
                                                 gr.pairs, fp, gr.queue, lf ? lf->knorm : nullptr);
      }
      return launch_bf16<64, 1, 3>(s, Qr, Kr, V, idx, keep, keep, scale, Os, st, nullptr, fp);
    }
    if (!idx) return launch_bf16<128, 1, 3>(s, Qr, Kr, V, nullptr, nb, 0, scale, Os, st, nullptr, fp);
    return launch_bf16<128, 1, 3>(s, Qr, Kr, V, idx, keep, keep, scale, Os, st, nullptr, fp);
  }
  if (s.d == 64) return launch_simple<float, 64>(s, Qr, Kr, V, block, keep, idx, scale, Os, st);
  return launch_simple<float, 128>(s, Qr, Kr, V, block, keep, idx, scale, Os, st);
}

}  // namespace rola
