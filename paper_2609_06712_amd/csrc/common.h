// Device-side helpers shared by the RoLA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rola {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;  // MI355X: 8 accelerator complex dies, workgroups dealt round-robin

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }  // RNE (v_cvt_pk_bf16_f32)

// Load 8 consecutive elements (16-byte aligned for bf16, 32-byte for fp32) as fp32.
__device__ __forceinline__ void load8(const float* p, float v[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void load8(const bf16* p, float v[8]) {
  const bf16x8 a = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
}
__device__ __forceinline__ void store8(float* p, const float v[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void store8(bf16* p, const float v[8]) {
  bf16x8 a;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = (bf16)v[i];
  *reinterpret_cast<bf16x8*>(p) = a;
}

// Direct global-to-LDS load of 16 bytes per lane (global_load_lds_dwordx4, scalar-base form): lane l
// reads base + voff(l) and the wave's 64 x 16 bytes land at LDS byte address lds_addr + 16 l
// (base and lds_addr wave-uniform). Issued as inline assembly on purpose: the compiler then does
// not track these LDS writes and adds no drains of its own (s_waitcnt vmcnt(0)) before later LDS
// reads, which would empty the prefetch pipeline; callers wait for completion themselves with
// s_waitcnt vmcnt(n) and a workgroup barrier.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_addr)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

// Marks a value as wave-uniform (moves it to a scalar register).
__device__ __forceinline__ int wave_uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Max over the lanes {l, l^16, l^32, l^48} (the four 16-lane rows) with two gfx950 permlane swaps:
// a 32-lane swap then a 16-lane swap, both plain VALU ops (no LDS round trip).
__device__ __forceinline__ float rows_max(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
// Sum over the same four lanes.
__device__ __forceinline__ float rows_sum(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float m = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Rotation of one interleaved pair (a, b) by the angle with cosine c and sine s (3D RoPE, turn by
// +angle): x = a c - b s, y = a s + b c, with explicit fused multiply-adds so that every kernel that
// rotates (the backbone rotation, the rotating pooling, the attention's query prologue) rounds alike.
__device__ __forceinline__ void rope_pair(float a, float b, float c, float s, float& x, float& y) {
  x = fmaf(a, c, -(b * s));
  y = fmaf(a, s, b * c);
}

// SiLU and the logistic gate with a hardware reciprocal (1 ulp) instead of an IEEE divide.
__device__ __forceinline__ float sigmoid(float x) { return __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }
__device__ __forceinline__ float silu(float x) { return x * sigmoid(x); }

// Bijective remap of a linear workgroup id so that consecutive logical ids run on the same XCD:
// hardware deals workgroup w to XCD w % 8, so XCD x gets the logical range [x*q(+rem), ...).
__device__ __forceinline__ int xcd_remap(int wg, int total) {
  const int q = total / kNumXcd, rem = total % kNumXcd;
  const int xcd = wg % kNumXcd, local = wg / kNumXcd;
  return (xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q) + local;
}

// 16-byte chunk swizzle of a 256-byte tile row: a bijection on row%16 (16 consecutive rows of a
// row read hit distinct chunks) whose bits 1-3 differ across every aligned group of four rows (the
// four rows of a transposing read hit distinct 32-byte chunk pairs).
__device__ __forceinline__ int bw_swizzle(int row) {
  return ((row & 3) << 1) | ((row >> 2) & 1) | (row & 8);
}

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// A operand from a row-major [row][128] tile: the lane's row l%32 (+ row0), channels 16s + 8(l/32).
__device__ __forceinline__ bf16x8 row_frag(const char* tile, int row, int s, int hh) {
  return *reinterpret_cast<const bf16x8*>(tile + row * 256 + (((2 * s + hh) ^ bw_swizzle(row)) << 4));
}

// Transposed operand of a row-major [row][128] tile for channel tile w and the 16 rows of k-step u:
// lane (channel 32w + 16((l/16)%2) + l%16) receives rows 16u + 4(l/32) + s and 16u + 8 + 4(l/32) + s,
// s = 0..3 -- the order in which an MFMA output hands its rows to a lane.
__device__ __forceinline__ bf16x8 tr_frag(const char* tile, int w, int u, int lane) {
  const int i16 = lane % 16, hh = lane / 32, g1 = (lane / 16) & 1;
  const int c = 2 * g1 + ((i16 & 3) >> 1);
  bf16x4 part[2];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    const int row = 16 * u + 8 * half + 4 * hh + i16 / 4;
    const char* p = tile + row * 256 + (((4 * w + c) ^ bw_swizzle(row)) << 4) + 8 * (i16 & 1);
    part[half] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
  }
  return __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7);
}

// The XCD the calling wave runs on (hardware register XCC_ID).
__device__ __forceinline__ int xcd_id() {
  unsigned v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return (int)(v % kNumXcd);
}

// Work queue over the same XCD ranges as xcd_remap, for a grid of resident workgroups: XCD x
// hands out its range [begin(x), begin(x) + len(x)) in ascending order through counter[x] (zero
// at launch), and a workgroup whose XCD's range is used up takes ids from the other ranges. The
// dies of one chip do not run equally fast (their finishing times under a static split differ by
// up to a fifth, and which die is slow changes from chip to chip), so the kernel then ends when
// the work ends, not when the slowest die's share does. Returns -1 once all ranges are used up;
// every call ends after at most kNumXcd atomics, as the counters only grow.
// Counter x sits at counter[x * kQueueStride]: each in a 256-byte slot of its own, because
// atomics on one cache line serialise (with the eight counters in one line, the claims of the
// whole chip queued behind each other: about 1 ms per launch at 23640 claims).
constexpr int kQueueStride = 64;
__device__ inline int xcd_queue_claim(int* counter, int xcd, int total) {
  const int q = total / kNumXcd, rem = total % kNumXcd;
  for (int k = 0; k < kNumXcd; ++k) {
    const int y = (xcd + k) % kNumXcd;
    const int len = q + (y < rem);
    int* c = counter + y * kQueueStride;
    if (__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= len) continue;
    const int i = atomicAdd(c, 1);
    if (i < len) return (y < rem ? y * (q + 1) : rem * (q + 1) + (y - rem) * q) + i;
  }
  return -1;
}

}  // namespace rola
