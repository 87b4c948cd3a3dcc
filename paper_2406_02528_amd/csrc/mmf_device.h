// Device helpers shared by the gfx950 kernels: wave64 reductions through DPP
// and readlane, the RMSNorm root, the 2-bit code unpacking of the packed
// weight format and the affine (bias + activation) epilogue.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mmf_launch.h"

namespace mmf {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// wave64 all-reductions.  Steps: DPP quad_perm xor 1, xor 2, row_half_mirror,
// row_mirror (each row of 16 lanes then holds its total), then readlane of
// lanes 0, 16, 32 and 48 and the combination (r0 + r1) + (r2 + r3) on
// wave-uniform values.  The combination order is fixed, so every call
// returns the same bits; no LDS round trip is involved.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}

constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // row_half_mirror
constexpr int kDppMirror = 0x140;     // row_mirror

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

__device__ __forceinline__ double readlane_f64(double v, int lane) {
  I32Parts p = split(v);
  p.lo = __builtin_amdgcn_readlane(p.lo, lane);
  p.hi = __builtin_amdgcn_readlane(p.hi, lane);
  return join(p);
}
__device__ __forceinline__ float readlane_f32(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  v += dpp_f64<kDppHalfMirror>(v);
  v += dpp_f64<kDppMirror>(v);
  return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

__device__ __forceinline__ float wave_max_f32(float v) {
  v = fmaxf(v, dpp_f32<kDppXor1>(v));
  v = fmaxf(v, dpp_f32<kDppXor2>(v));
  v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppMirror>(v));
  return fmaxf(fmaxf(readlane_f32(v, 0), readlane_f32(v, 16)), fmaxf(readlane_f32(v, 32), readlane_f32(v, 48)));
}

__device__ __forceinline__ int wave_sum_i32(int v) {
  v += dpp_i32<kDppXor1>(v);
  v += dpp_i32<kDppXor2>(v);
  v += dpp_i32<kDppHalfMirror>(v);
  v += dpp_i32<kDppMirror>(v);
  return (__builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16)) +
         (__builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48));
}

// ---------------------------------------------------------------------------
// RMSNorm reciprocal scale r = 1 / sqrt(sum_k x_k^2 / K + eps), eps = 1e-6,
// returned in fp32 and equal to the fp32 rounding of the fp64 sequence
// mean = ss / K, v = mean + eps, s = sqrt(v), r = 1 / s with every step
// correctly rounded.
//
// The division by K is a multiplication when K is a power of two (exact).
// 1/sqrt(v) is first evaluated as a hardware reciprocal-square-root estimate
// refined by two Newton steps in fp64 (within a few fp64 ulps of the exact
// value).  The fp64 sequence above is within 2^-52 (relative) of the exact
// value too, so both round to the same fp32 number unless the exact value
// lies within about 2^-49 of a midpoint between two fp32 numbers; when the
// refined value is within 2^-44 of one (or fp32 r would not be a normal
// number) the sequence itself is evaluated.  All inputs are wave-uniform, so
// the branch does not diverge.
// ---------------------------------------------------------------------------
constexpr double kRmsEps = 1e-6;

__device__ __forceinline__ float rms_rstd(double ss, int K) {
  const double mean = (K & (K - 1)) == 0 ? ss * (1.0 / static_cast<double>(K)) : ss / static_cast<double>(K);
  const double v = mean + kRmsEps;
  const double h = 0.5 * v;
  double y = __builtin_amdgcn_rsq(v);
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const double e = __builtin_fma(-(h * y), y, 0.5);  // 1/2 - v y^2 / 2
    y = __builtin_fma(y, e, y);
  }
  const float r = static_cast<float>(y);
  const uint32_t bits = __float_as_uint(r);
  const int ex = static_cast<int>((bits >> 23) & 0xFFu);
  const double d = y - static_cast<double>(r);
  // half the spacing of fp32 numbers on the side of r where y lies
  double half = __builtin_ldexp(1.0, ex - 127 - 24);
  if ((bits & 0x7FFFFFu) == 0 && d < 0.0) half *= 0.5;
  const bool safe = ex > 0 && ex < 0xFE && __builtin_fabs(d) < half * (1.0 - 0x1p-20);
  if (safe) return r;
  return static_cast<float>(1.0 / __builtin_sqrt(v));
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

// ---------------------------------------------------------------------------
// Activation quantisation steps (Sec. on the BitLinear layer: per-token
// absmax int8 quantisation).
//
// sum_sq(ss, f): ss + f^2 in fp64 with one fused multiply-add -- the square
// of an fp32 value is exact in fp64, so this is the same bits as a separate
// multiply and add.
//
// quantise4(y, s): q_e = round-half-even(fl(y_e s)) for four values, packed
// little-endian into one word.  Adding 1.5 2^23 (an even integer, where the
// fp32 spacing is 1) rounds fl(y s) to an integer with ties to even, as rint
// does, and leaves it in two's complement in the low byte of the sum's bits.
// With s = 127 / a and a >= max |y| the product stays within 127 (1 + 2u), so
// q lies in [-127, 127] without a clamp.  The product and the sum are rounded
// separately (__fmul_rn / __fadd_rn are never fused).  Inputs must be finite.
//
// byte_sum4(w, acc): acc + the four signed bytes of w.
// ---------------------------------------------------------------------------
__device__ __forceinline__ double sum_sq(double ss, float f) {
  const double d = static_cast<double>(f);
  return __builtin_fma(d, d, ss);
}

__device__ __forceinline__ uint32_t quantise4(const float* y, float s) {
  constexpr float kRound = 12582912.0f;  // 1.5 * 2^23
  uint32_t b[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) b[e] = __float_as_uint(__fadd_rn(__fmul_rn(y[e], s), kRound));
  // v_perm_b32: selector bytes 0-3 take bytes of the second operand, 4-7 of
  // the first, 0x0c gives zero
  const uint32_t lo = __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u);  // q0, q1 in bytes 0, 1
  const uint32_t hi = __builtin_amdgcn_perm(b[3], b[2], 0x04000c0cu);  // q2, q3 in bytes 2, 3
  return lo | hi;
}

__device__ __forceinline__ int byte_sum4(uint32_t w, int acc) { return dot4(w, 0x01010101u, acc); }

// ---------------------------------------------------------------------------
// Logistic sigmoid 1 / (1 + e^-v) from the hardware base-2 exponential and
// reciprocal (v_exp_f32, v_rcp_f32, 1 ulp each): e^-v = 2^(-v log2 e) with
// the argument rounded once in fp32, so the result carries a relative error
// of about (1 - sigmoid) (|v| + 2) u + 3u (u = 2^-24).  Saturates cleanly:
// 2^x overflows to inf for v << 0 (sigmoid 0) and underflows to 0 for
// v >> 0 (sigmoid 1).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float sigmoid_hw(float v) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(v * -1.44269504088896341f));
}

// ---------------------------------------------------------------------------
// MLGRU recurrence step and output gate on one channel, fp32, one rounding
// per operation (the recurrence kernels and the fused decode prologue share
// them, so both give the same bits):
//   h' = f h + (1 - f) c,   o' = g sigmoid(h')
// ---------------------------------------------------------------------------
__device__ __forceinline__ float mlgru_step(float h, float f, float c) { return f * h + (1.0f - f) * c; }
__device__ __forceinline__ float mlgru_out_gate(float g, float h) { return g * sigmoid_hw(h); }

// ---------------------------------------------------------------------------
// Affine epilogue.  z = (float)acc * (a_scale * w_scale[s]) + bias[n] in
// fp32, one rounding per operation, then the activation of segment s:
// identity, (1 - lb) sigmoid(z) + lb (sigmoid with a lower bound) or
// z sigmoid(z) (SiLU).  The column factors go through buffer resources of
// size 0 when an array is absent, which read as 0 with no memory access.
// ---------------------------------------------------------------------------
constexpr int kBufferWord3 = 0x00020000;  // gfx9 buffer descriptor word 3

__device__ __forceinline__ float affine_act(float z, uint32_t act, float lb) {
  if (act == kActIdentity) return z;
  const float s = sigmoid_hw(z);
  if (act == kActSilu) return z * s;
  return (1.0f - lb) * s + lb;
}

struct ColAffine {
  float ws, bias, lb;
  uint32_t act;
};

// Factors of column n (< N, a multiple of seg) of an affine epilogue.
__device__ __forceinline__ ColAffine load_col_affine(const Affine& a, const float* w_scale,
                                                     uint32_t N, uint32_t n) {
  const uint32_t seg = static_cast<uint32_t>(a.seg);
  const uint32_t s = n / seg;
  const __amdgpu_buffer_rsrc_t ws_r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(w_scale), 0, static_cast<int>((N / seg) * 4u), kBufferWord3);
  const __amdgpu_buffer_rsrc_t b_r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.bias), 0, a.bias != nullptr ? static_cast<int>(N * 4u) : 0, kBufferWord3);
  const __amdgpu_buffer_rsrc_t l_r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.lb), 0, a.lb != nullptr ? static_cast<int>(seg * 4u) : 0, kBufferWord3);
  ColAffine c;
  c.ws = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ws_r, 4u * s, 0, 0));
  c.bias = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(b_r, 4u * n, 0, 0));
  c.lb = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(l_r, 4u * (n - s * seg), 0, 0));
  c.act = (a.acts >> (2u * s)) & 3u;
  return c;
}

// Four consecutive columns n .. n + 3 (n % 4 == 0, seg % 16 == 0: one segment).
typedef float v4f __attribute__((ext_vector_type(4)));
struct ColAffine4 {
  float ws;
  v4f bias, lb;
  uint32_t act;
};

__device__ __forceinline__ ColAffine4 load_col_affine4(const Affine& a, const float* w_scale,
                                                       uint32_t N, uint32_t n) {
  const uint32_t seg = static_cast<uint32_t>(a.seg);
  const uint32_t s = n / seg;
  const __amdgpu_buffer_rsrc_t ws_r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(w_scale), 0, static_cast<int>((N / seg) * 4u), kBufferWord3);
  const __amdgpu_buffer_rsrc_t b_r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.bias), 0, a.bias != nullptr ? static_cast<int>(N * 4u) : 0, kBufferWord3);
  const __amdgpu_buffer_rsrc_t l_r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.lb), 0, a.lb != nullptr ? static_cast<int>(seg * 4u) : 0, kBufferWord3);
  ColAffine4 c;
  c.ws = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ws_r, 4u * s, 0, 0));
  c.bias = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(b_r, 4u * n, 0, 0));
  c.lb = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(l_r, 4u * (n - s * seg), 0, 0));
  c.act = (a.acts >> (2u * s)) & 3u;
  return c;
}

}  // namespace mmf
