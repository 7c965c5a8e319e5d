// Device helpers shared by the CateKV kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace catekv {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

// ---- bf16 <-> fp32 (bf16 kept as raw 16-bit patterns) -------------------
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// ---- DPP lane exchange within a row of 16 lanes --------------------------
// quad_perm [1,0,3,2] = lane ^ 1 ; [2,3,0,1] = lane ^ 2 ; row_half_mirror
// pairs lane i with 7 - i inside each group of 8 ; row_mirror pairs i with
// 15 - i inside each row of 16.
constexpr int kDppXor1 = 0xB1;
constexpr int kDppXor2 = 0x4E;
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over the 8 lanes of each aligned group of 8 (every lane gets the sum).
__device__ __forceinline__ float sum8(float x) {
  x += dpp<kDppXor1>(x);
  x += dpp<kDppXor2>(x);
  x += dpp<kDppHalfMirror>(x);
  return x;
}
// Sum / max over the 16 lanes of each row of 16.
__device__ __forceinline__ float sum16(float x) {
  x = sum8(x);
  x += dpp<kDppMirror>(x);
  return x;
}
__device__ __forceinline__ float max16(float x) {
  x = fmaxf(x, dpp<kDppXor1>(x));
  x = fmaxf(x, dpp<kDppXor2>(x));
  x = fmaxf(x, dpp<kDppHalfMirror>(x));
  x = fmaxf(x, dpp<kDppMirror>(x));
  return x;
}

// x combined with x of lane ^ 16 (or ^ 32) on every lane, through the gfx950
// row-swap instructions (VALU; no LDS traffic).  Swapping a register with
// itself leaves one half of each lane pair in each result, so the two results
// of the swap hold x[lane] and x[lane ^ 16] in some order.
__device__ __forceinline__ float add_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Maximum over each aligned group of g lanes (g a power of two up to 64, the
// same on every lane); every lane of a group gets the group's maximum.
__device__ __forceinline__ float max_in_group(float x, int g) {
  if (g >= 2) x = fmaxf(x, dpp<kDppXor1>(x));
  if (g >= 4) x = fmaxf(x, dpp<kDppXor2>(x));
  if (g >= 8) x = fmaxf(x, dpp<kDppHalfMirror>(x));
  if (g >= 16) x = fmaxf(x, dpp<kDppMirror>(x));
  if (g >= 32) x = max_xor16(x);
  if (g >= 64) x = max_xor32(x);
  return x;
}

// Cross-row exchange through the LDS crossbar (no LDS storage used).
__device__ __forceinline__ float shfl_xor(float x, int mask) {
  int lane = __lane_id();
  return __int_as_float(__builtin_amdgcn_ds_bpermute((lane ^ mask) << 2, __float_as_int(x)));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Compiler-only memory barrier: keeps LDS accesses on their side of a
// hand-placed s_waitcnt / s_barrier pair.
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// Workgroup barrier that waits only for this wave's LDS operations, so that
// global-to-LDS loads still in flight keep flowing across it.
// s_waitcnt immediate: lgkmcnt(0), vmcnt and expcnt not waited on.
__device__ __forceinline__ void barrier_lds_only() {
  compiler_fence();
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  compiler_fence();
}

// 16-byte load that the compiler keeps as one dwordx4.
__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// 16-byte load through the global address space (a global_load_dwordx4, not a
// flat load), for pointers the compiler cannot prove global by itself.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16(const void* p) {
  const u32x4_t v = *(const __attribute__((address_space(1))) u32x4_t*)(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

}  // namespace catekv
