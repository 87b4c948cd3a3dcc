// Fused RMSNorm + per-token absmax int8 quantisation (Algorithm 1,
// rms_norm_fwd + activation_quant; RMSNorm with the mean of squares and
// eps = 1e-6, learned scale gamma), optionally keeping rstd for the backward.
// One, two or four wave64s per token row; the row is read from HBM once and
// kept in registers while the two row statistics (sum of squares, then
// absmax of the normalised values) are reduced across the row's lanes.
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kRowsPerBlock = 4;  // waves per 256-thread block
constexpr int kBufferFlags = 0x00020000;  // gfx9 buffer descriptor word 3

// 16-byte vector of activations: 8 bf16 or 4 fp32.
template <typename XT> struct Vec;
template <> struct Vec<uint16_t> {
  static constexpr int kElems = 8;
  using Raw = uint4;
  __device__ static void to_f32(const Raw& r, float* f) {
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
};
template <> struct Vec<float> {
  static constexpr int kElems = 4;
  using Raw = float4;
  __device__ static void to_f32(const Raw& r, float* f) {
    f[0] = r.x; f[1] = r.y; f[2] = r.z; f[3] = r.w;
  }
};

// q of one 16-byte vector (E values) into its row: E / 4 packed words, and
// their byte sum added to rs
template <int E>
__device__ __forceinline__ void quantise_store(int8_t* dst, const float* y, float s, int& rs) {
  uint32_t w[E / 4];
#pragma unroll
  for (int g = 0; g < E / 4; ++g) {
    w[g] = quantise4(y + 4 * g, s);
    rs = byte_sum4(w[g], rs);
  }
  if constexpr (E == 8)
    *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
  else
    *reinterpret_cast<uint32_t*>(dst) = w[0];
}

__device__ __forceinline__ float row_rstd(double ss, int K) { return rms_rstd(ss, K); }

// One row per W waves (W = 1, 2 or 4; 256-thread blocks hold 4 / W rows).
// VPL > 0: each lane keeps VPL 16-byte vectors of its row in registers (rows
// of at most 64 W VPL vectors), so the row is read from HBM once; with W > 1
// the row's statistics are combined across its waves through LDS, in a fixed
// order (the fp64 sum of squares is therefore deterministic).  VPL == 0: any
// K; the row is re-read from memory (L2) for each of the three passes.
template <typename XT, int W, int VPL>
__global__ __launch_bounds__(256) void act_quant_kernel(
    const XT* __restrict__ x, const float* __restrict__ gamma,
    int8_t* __restrict__ q, float* __restrict__ a_scale,
    int32_t* __restrict__ q_rowsum, float* __restrict__ rstd, int64_t M, int K) {
  using V = Vec<XT>;
  constexpr int E = V::kElems;
  constexpr int kRows = kRowsPerBlock / W;  // rows per block
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int rw = wave % W;                   // wave within the row
  const int rl = rw * kWave + lane;          // lane within the row
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kRows + wave / W;
  const bool live = row < M;                 // uniform per wave (and per row)
  // per-row statistics of the W waves: [row in block][wave in row]
  __shared__ double s_ss[kRowsPerBlock];
  __shared__ float s_amax[kRowsPerBlock];
  __shared__ int s_rs[kRowsPerBlock];
  const int slot0 = (wave / W) * W;
  auto combine_f64 = [&](double v) -> double {
    if constexpr (W == 1) {
      return v;
    } else {
      if (lane == 0) s_ss[wave] = v;
      __syncthreads();
      double t = 0.0;
#pragma unroll
      for (int w = 0; w < W; ++w) t += s_ss[slot0 + w];
      return t;
    }
  };
  auto combine_max = [&](float v) -> float {
    if constexpr (W == 1) {
      return v;
    } else {
      if (lane == 0) s_amax[wave] = v;
      __syncthreads();
      float t = 0.0f;
#pragma unroll
      for (int w = 0; w < W; ++w) t = fmaxf(t, s_amax[slot0 + w]);
      return t;
    }
  };
  auto combine_i32 = [&](int v) -> int {
    if constexpr (W == 1) {
      return v;
    } else {
      if (lane == 0) s_rs[wave] = v;
      __syncthreads();
      int t = 0;
#pragma unroll
      for (int w = 0; w < W; ++w) t += s_rs[slot0 + w];
      return t;
    }
  };
  if constexpr (W == 1) {
    if (!live) return;  // whole wave leaves together
  }
  // a block's rows past M read nothing (a resource of size 0) and store nothing;
  // their waves still take part in the block's barriers
  const int64_t srow = live ? row : 0;
  const int nvec = K / E;
  const typename V::Raw* xr = reinterpret_cast<const typename V::Raw*>(x + srow * K);
  int8_t* qr = q + srow * K;

  if constexpr (VPL > 0) {
    // Every load of the row and of gamma is issued at once, without branches:
    // both go through buffer resources of the row's (gamma's) size, so the
    // vectors past the row's end read as zero (and gamma == NULL as a
    // resource of size 0).  Guarded loads would each wait for the last.
    const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<XT*>(x + srow * K), 0, live ? static_cast<int>(K * sizeof(XT)) : 0, kBufferFlags);
    const __amdgpu_buffer_rsrc_t grsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(gamma), 0, gamma != nullptr ? K * 4 : 0, kBufferFlags);
    typename V::Raw raw[VPL];
    float4 gv[VPL][E / 4];
#pragma unroll
    for (int i = 0; i < VPL; ++i)
      raw[i] = __builtin_bit_cast(typename V::Raw, __builtin_amdgcn_raw_buffer_load_b128(
                                                       xrsrc, static_cast<uint32_t>((rl + W * kWave * i) * 16), 0, 0));
#pragma unroll
    for (int i = 0; i < VPL; ++i)
#pragma unroll
      for (int e4 = 0; e4 < E / 4; ++e4)
        gv[i][e4] = __builtin_bit_cast(
            float4, __builtin_amdgcn_raw_buffer_load_b128(
                        grsrc, static_cast<uint32_t>(((rl + W * kWave * i) * E + 4 * e4) * 4), 0, 0));
    __builtin_amdgcn_sched_barrier(0);  // all loads before the first wait
    float xf[VPL][E];
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      V::to_f32(raw[i], xf[i]);  // zero past the row's end
#pragma unroll
      for (int e = 0; e < E; ++e) ss = sum_sq(ss, xf[i][e]);
    }
    ss = combine_f64(wave_sum_f64(ss));
    const float r = row_rstd(ss, K);

    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      if (gamma != nullptr) {  // uniform
#pragma unroll
        for (int e4 = 0; e4 < E / 4; ++e4) {
          xf[i][4 * e4 + 0] = (xf[i][4 * e4 + 0] * r) * gv[i][e4].x;
          xf[i][4 * e4 + 1] = (xf[i][4 * e4 + 1] * r) * gv[i][e4].y;
          xf[i][4 * e4 + 2] = (xf[i][4 * e4 + 2] * r) * gv[i][e4].z;
          xf[i][4 * e4 + 3] = (xf[i][4 * e4 + 3] * r) * gv[i][e4].w;
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) xf[i][e] = xf[i][e] * r;
      }
#pragma unroll
      for (int e = 0; e < E; ++e) amax = fmaxf(amax, fabsf(xf[i][e]));
    }
    amax = fmaxf(combine_max(wave_max_f32(amax)), 1e-5f);
    const float s = 127.0f / amax;

    int rs = 0;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int v = rl + W * kWave * i;
      if (live && v < nvec) quantise_store<E>(qr + v * E, xf[i], s, rs);
    }
    rs = combine_i32(wave_sum_i32(rs));
    if (live && rl == 0) {
      a_scale[row] = amax / 127.0f;
      if (q_rowsum != nullptr) q_rowsum[row] = rs;
      if (rstd != nullptr) rstd[row] = r;
    }
  } else {
    // pass 1: sum of squares
    double ss = 0.0;
    if (live) {
      for (int v = rl; v < nvec; v += W * kWave) {
        float f[E];
        V::to_f32(xr[v], f);
#pragma unroll
        for (int e = 0; e < E; ++e) ss = sum_sq(ss, f[e]);
      }
    }
    ss = combine_f64(wave_sum_f64(ss));
    const float r = row_rstd(ss, K);
    // pass 2: absmax of the normalised row
    float amax = 0.0f;
    if (live) {
      for (int v = rl; v < nvec; v += W * kWave) {
        float f[E];
        V::to_f32(xr[v], f);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          float y = f[e] * r;
          if (gamma != nullptr) y = y * gamma[v * E + e];
          amax = fmaxf(amax, fabsf(y));
        }
      }
    }
    amax = fmaxf(combine_max(wave_max_f32(amax)), 1e-5f);
    const float s = 127.0f / amax;
    // pass 3: quantise
    int rs = 0;
    if (live) {
      for (int v = rl; v < nvec; v += W * kWave) {
        float f[E];
        V::to_f32(xr[v], f);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          f[e] = f[e] * r;
          if (gamma != nullptr) f[e] = f[e] * gamma[v * E + e];
        }
        quantise_store<E>(qr + v * E, f, s, rs);
      }
    }
    rs = combine_i32(wave_sum_i32(rs));
    if (live && rl == 0) {
      a_scale[row] = amax / 127.0f;
      if (q_rowsum != nullptr) q_rowsum[row] = rs;
      if (rstd != nullptr) rstd[row] = r;
    }
  }
}

// Waves per row and vectors per lane: one wave while a lane holds at most 4
// vectors of the row, else 2 or 4 waves, so that rows up to 64 x 4 x 8
// vectors stay in registers (bf16 K <= 16384, fp32 K <= 8192); the number of
// vectors per lane is the smallest compiled value that holds the row (loads
// past the row's end return zeros but cost nearly a real load each).
template <typename XT, int W>
hipError_t launch_w(const XT* x, const float* gamma, int8_t* q, float* a_scale, int32_t* q_rowsum,
                    float* rstd, int64_t M, int K, int vpl, hipStream_t stream) {
  constexpr int kRows = kRowsPerBlock / W;
  const dim3 grid(static_cast<unsigned>((M + kRows - 1) / kRows));
  const dim3 block(kWave * kRowsPerBlock);
#define MMF_AQ_LAUNCH(V)                                                             \
  hipLaunchKernelGGL((act_quant_kernel<XT, W, V>), grid, block, 0, stream, x, gamma, \
                     q, a_scale, q_rowsum, rstd, M, K)
  switch (vpl) {
    case 1: MMF_AQ_LAUNCH(1); break;
    case 2: MMF_AQ_LAUNCH(2); break;
    case 3: MMF_AQ_LAUNCH(3); break;
    case 4: MMF_AQ_LAUNCH(4); break;
    case 5: case 6: MMF_AQ_LAUNCH(6); break;
    case 7: case 8: MMF_AQ_LAUNCH(8); break;
    default: MMF_AQ_LAUNCH(0); break;
  }
#undef MMF_AQ_LAUNCH
  return hipGetLastError();
}

template <typename XT>
hipError_t launch_typed(const XT* x, const float* gamma, int8_t* q, float* a_scale,
                        int32_t* q_rowsum, float* rstd, int64_t M, int K, hipStream_t stream) {
  constexpr int E = Vec<XT>::kElems;
  const int nvec = K / E;
  if (nvec <= kWave * 4)
    return launch_w<XT, 1>(x, gamma, q, a_scale, q_rowsum, rstd, M, K, (nvec + kWave - 1) / kWave, stream);
  if (nvec <= 2 * kWave * 4)
    return launch_w<XT, 2>(x, gamma, q, a_scale, q_rowsum, rstd, M, K, (nvec + 2 * kWave - 1) / (2 * kWave),
                           stream);
  const int vpl = (nvec + 4 * kWave - 1) / (4 * kWave);
  return launch_w<XT, 4>(x, gamma, q, a_scale, q_rowsum, rstd, M, K, vpl <= 8 ? vpl : 0, stream);
}

}  // namespace

hipError_t launch_act_quant(const void* x, bool x_is_f32, const float* gamma, int8_t* q,
                            float* a_scale, int32_t* q_rowsum, int64_t M, int K,
                            hipStream_t stream, float* rstd) {
  if (M == 0) return hipSuccess;
  if (x_is_f32)
    return launch_typed(static_cast<const float*>(x), gamma, q, a_scale, q_rowsum, rstd, M, K, stream);
  return launch_typed(static_cast<const uint16_t*>(x), gamma, q, a_scale, q_rowsum, rstd, M, K, stream);
}

}  // namespace mmf
