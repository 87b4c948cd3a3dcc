// Device helpers shared by the gfx950 kernels: wave64 reductions through DPP
// and ds_swizzle, and the 2-bit code unpacking of the packed weight format.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mmf {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// wave64 all-reductions.  Steps: DPP quad_perm xor 1, xor 2, row_half_mirror,
// row_mirror (each row of 16 lanes then holds its total), ds_swizzle xor 16
// (each half-wave holds its total), and a readlane of lanes 0 and 32.  The
// combination order is fixed, so every call returns the same bits.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}

constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // row_half_mirror
constexpr int kDppMirror = 0x140;     // row_mirror
constexpr int kSwizzleXor16 = 0x401F; // ds_swizzle bit mode: and 0x1F, xor 0x10

struct I32Parts {
  int lo, hi;
};

__device__ __forceinline__ I32Parts split(double v) {
  uint64_t b = __builtin_bit_cast(uint64_t, v);
  return {static_cast<int>(static_cast<uint32_t>(b)), static_cast<int>(static_cast<uint32_t>(b >> 32))};
}
__device__ __forceinline__ double join(I32Parts p) {
  uint64_t b = (static_cast<uint64_t>(static_cast<uint32_t>(p.hi)) << 32) | static_cast<uint32_t>(p.lo);
  return __builtin_bit_cast(double, b);
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  I32Parts p = split(v);
  p.lo = dpp_i32<CTRL>(p.lo);
  p.hi = dpp_i32<CTRL>(p.hi);
  return join(p);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(dpp_i32<CTRL>(__float_as_int(v)));
}

__device__ __forceinline__ int swz_xor16_i32(int v) {
  return __builtin_amdgcn_ds_swizzle(v, kSwizzleXor16);
}
__device__ __forceinline__ double swz_xor16_f64(double v) {
  I32Parts p = split(v);
  p.lo = swz_xor16_i32(p.lo);
  p.hi = swz_xor16_i32(p.hi);
  return join(p);
}

__device__ __forceinline__ double readlane_f64(double v, int lane) {
  I32Parts p = split(v);
  p.lo = __builtin_amdgcn_readlane(p.lo, lane);
  p.hi = __builtin_amdgcn_readlane(p.hi, lane);
  return join(p);
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  v += dpp_f64<kDppHalfMirror>(v);
  v += dpp_f64<kDppMirror>(v);
  v += swz_xor16_f64(v);
  return readlane_f64(v, 0) + readlane_f64(v, 32);
}

__device__ __forceinline__ float wave_max_f32(float v) {
  v = fmaxf(v, dpp_f32<kDppXor1>(v));
  v = fmaxf(v, dpp_f32<kDppXor2>(v));
  v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppMirror>(v));
  v = fmaxf(v, __int_as_float(swz_xor16_i32(__float_as_int(v))));
  return fmaxf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)),
               __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32)));
}

__device__ __forceinline__ int wave_sum_i32(int v) {
  v += dpp_i32<kDppXor1>(v);
  v += dpp_i32<kDppXor2>(v);
  v += dpp_i32<kDppHalfMirror>(v);
  v += dpp_i32<kDppMirror>(v);
  v += swz_xor16_i32(v);
  return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 32);
}

// ---------------------------------------------------------------------------
// Packed ternary weights: code c = t + 1 of k = 16j + 4i + b sits at bits
// 8b + 2i of word j, so (w >> 2i) & 0x03030303 gives the four codes of
// k = 16j + 4i .. 16j + 4i + 3 as bytes in k order.
// ---------------------------------------------------------------------------
constexpr uint32_t kCodeMask = 0x03030303u;

__device__ __forceinline__ uint32_t codes4(uint32_t w, int i) {
  return (w >> (2 * i)) & kCodeMask;
}

// int8 dot product of four byte pairs, accumulated into c (v_dot4_i32_i8).
__device__ __forceinline__ int dot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4(static_cast<int>(a), static_cast<int>(b), c, false);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

}  // namespace mmf
