// Shared device helpers for the SegPagedAttention kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace segpa {

typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// Matrix-core steps. Lane layouts (gfx950, checked on hardware):
//   16x16x32 bf16: A[i = l%16][k = 8*(l/16) + e], B[k = 8*(l/16) + e][j = l%16]
//   16x16x16 bf16: A[i = l%16][k = 4*(l/16) + e], B[k = 4*(l/16) + e][j = l%16]
//   result (both): C[i = 4*(l/16) + r][j = l%16], r = 0..3
__device__ __forceinline__ f32x4 mfma16x16x32(s16x8 a, s16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16x16x16(s16x4 a, s16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Four floats -> four bf16 (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ s16x4 pack_bf16x4(float a, float b, float c, float d) {
  bf16x4 v;
  v.x = (__bf16)a;
  v.y = (__bf16)b;
  v.z = (__bf16)c;
  v.w = (__bf16)d;
  return __builtin_bit_cast(s16x4, v);
}

__device__ __forceinline__ float bf16_bits_to_float(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// Buffer resource (V#) for raw buffer loads on gfx9-family parts: base
// address, no stride, `bytes` of range (reads past it return 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}

// Make a wave-uniform 64-bit value provably uniform (scalar registers).
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <typename T>
__device__ __forceinline__ T clampv(T x, T lo, T hi) {
  return x < lo ? lo : (x > hi ? hi : x);
}

// Algorithm 2, Translate: logical page j of one head stream -> physical page.
// Returns -1 for anything out of range (the page is then skipped).
__device__ __forceinline__ int translate_page(const int32_t* __restrict__ seg_row,
                                              const int32_t* __restrict__ page_table, int j,
                                              int pps, int max_segs, int64_t n_virtual,
                                              int64_t n_phys) {
  if (j < 0) return -1;
  const int s = j / pps;
  const int o = j - s * pps;
  if (s >= max_segs) return -1;
  const int v0 = seg_row[s];
  if (v0 < 0) return -1;
  const int64_t v = (int64_t)v0 + o;
  if (v >= n_virtual) return -1;
  const int ph = page_table[v];
  if (ph < 0 || (int64_t)ph >= n_phys) return -1;
  return ph;
}

// SplitMix64 (Steele, Lea, Flood, OOPSLA 2014): output function, and one
// generator output from a state (advance by the golden gamma, then mix).
__device__ __forceinline__ uint64_t splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
__device__ __forceinline__ uint64_t splitmix64(uint64_t state) {
  return splitmix64_mix(state + 0x9E3779B97F4A7C15ull);
}

typedef int v4i __attribute__((ext_vector_type(4)));

// HBM -> LDS copy of 16 bytes per lane: bytes [voff, voff + 16) of the buffer
// at `base` (range `bytes`; zero-range reads nothing) land at LDS byte address
// lds_byte + 16 * lane. Inline assembly, so that the compiler does not wait
// for the copy before each LDS read (it cannot tell the stages apart); the
// pipeline's own waits order it. `base` and `lds_byte` are wave-uniform (a
// caller that computes the address with scalar arithmetic keeps the chain off
// the vector unit). The compiler's hazard checks do not see into the
// assembly, so it keeps the wait states GFX9 asks for itself: 5 between a
// vector instruction writing an SGPR (the descriptor comes out of
// v_readfirstlane) and a memory instruction reading it, and 1 between the M0
// write and the LDS-destination load (s_mov + s_nop 4 = 6).
__device__ __forceinline__ void copy_to_lds_at(const void* base, int bytes, uint32_t lds_byte, int voff) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const v4i rs = {(int)__builtin_amdgcn_readfirstlane((uint32_t)b),
                  (int)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32) & 0xffffu),
                  __builtin_amdgcn_readfirstlane(bytes), 0x00020000};
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_byte);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(m0v), "v"(voff), "s"(rs) : "m0");
}

// bf16 quiet NaN x 8: what the LDS-poison debug build writes into key and
// value slots before their copies
constexpr s16x8 kLdsPoison8 = {0x7FC0, 0x7FC0, 0x7FC0, 0x7FC0, 0x7FC0, 0x7FC0, 0x7FC0, 0x7FC0};

// LDS byte address of a pointer into LDS
__device__ __forceinline__ uint32_t lds_address(const void* lds) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)lds;
}

__device__ __forceinline__ void copy_to_lds(const void* base, int bytes, const void* lds, int voff) {
  copy_to_lds_at(base, bytes, lds_address(lds), voff);
}

// Inclusive prefix sum of an int over the 64 lanes of a wave with DPP moves
// (no LDS round trip): running sums within each row of 16 lanes (shifts by 1,
// 2, 4, 8; lanes whose source lies before the row's start add 0), then lane
// 15's sum added to rows 1 and 3 and lane 31's to rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Block-wide exclusive prefix sum of one value per thread, in thread order,
// and the block total (a scan in each wave, then the wave totals in wave
// order: a fixed order of additions). `scratch` holds BS / 64 values. Ints
// scan each wave with DPP moves (exact in any order); other types with
// shuffles, keeping the sequential order within the wave and no subtraction.
template <int BS, typename T>
__device__ void block_scan(T x, T& ex, T& tot, T* scratch) {
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  T incl = x;
  if constexpr (__is_same(T, int)) {
    incl = wave_incl_scan(x);
  } else {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const T y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
  }
  if (lane == 63) scratch[w] = incl;
  __syncthreads();
  T pre = 0;
  tot = 0;
#pragma unroll
  for (int i = 0; i < BS / 64; ++i) {
    const T c = scratch[i];
    if (i < w) pre += c;
    tot += c;
  }
  if constexpr (__is_same(T, int)) {
    ex = pre + (incl - x);
  } else {
    const T below = __shfl_up(incl, 1);   // in-wave exclusive sum (no subtraction)
    ex = lane == 0 ? pre : pre + below;
  }
  __syncthreads();
}

}  // namespace segpa
