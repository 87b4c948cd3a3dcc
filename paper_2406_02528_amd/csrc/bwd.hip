// Backward of the BitLinear (Algorithm 1, backward_pass and rms_norm_bwd; the
// straight-through estimator of Sec. "Surrogate Gradient" passes the
// gradient through both quantisers unchanged), in the RMSNorm reading with
// the learned scale after the normalisation, y = (x r) gamma:
//   dY  = dO Wt^T  (Wt = t w_scale, the weights the forward used)
//   dx  = r g - (r^3 / K) x s,   g = gamma dY,  s = sum_k g_k x_k
//   dW  = dO^T Yq  (Yq = q a_scale, stored as bfloat16)
//   db  = sum_m dO,  dgamma = sum_m dY x r
// The two products are dense contractions over floating-point gradients, so
// they run as plain bf16 GEMMs on the matrix cores (rocBLAS, fp32
// accumulation); the kernels here prepare their operands (the ternary codes
// as exact bf16 -1/0/+1, Yq) and do the row-wise RMSNorm backward and the
// column sums, all streaming and HBM-bound.
#include <rocblas/rocblas.h>

#include <mutex>
#include <type_traits>

#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kBlock = 256;
constexpr int kRowsPerBlock = kBlock / kWave;  // one wave per row
constexpr uint16_t kBf16One = 0x3F80, kBf16MinusOne = 0xBF80;

unsigned blocks_for(int64_t threads) { return static_cast<unsigned>((threads + kBlock - 1) / kBlock); }

// Word (j, n) of the packed weights holds t[n][16j .. 16j+15]; the code of
// k = 16j + 4i + b sits at bits 8b + 2i.  Thread (j, n) writes column n of
// rows 16j .. 16j+15 of T [K][N], so a wave's stores are contiguous.
__global__ __launch_bounds__(kBlock) void expand_ternary_kernel(const uint32_t* __restrict__ Wp, int64_t J,
                                                                int64_t N, uint16_t* __restrict__ T) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= J * N) return;
  const int64_t j = idx / N, n = idx % N;
  const uint32_t w = Wp[idx];
#pragma unroll
  for (int kk = 0; kk < 16; ++kk) {
    const uint32_t c = (w >> (8 * (kk & 3) + 2 * (kk >> 2))) & 3u;
    T[(16 * j + kk) * N + n] = c == 0 ? kBf16MinusOne : (c == 2 ? kBf16One : uint16_t(0));
  }
}

__device__ __forceinline__ uint32_t bf16_bits_rne(float v) {
  const uint32_t b = __float_as_uint(v);
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// Yq = q a_scale[m] in fp32, rounded to nearest-even bf16; 8 elements per
// thread (K % 16 == 0, so a group never crosses a row).
__global__ __launch_bounds__(kBlock) void dequant_bf16_kernel(const int8_t* __restrict__ q,
                                                              const float* __restrict__ a_scale, int64_t M,
                                                              int K, uint16_t* __restrict__ yq) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int64_t e0 = idx * 8;
  if (e0 >= M * K) return;
  const float a = a_scale[e0 / K];
  const uint2 qv = *reinterpret_cast<const uint2*>(q + e0);
  const uint32_t words[2] = {qv.x, qv.y};
  uint32_t out[4];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int8_t lo = static_cast<int8_t>((words[h] >> (16 * p)) & 0xFF);
      const int8_t hi = static_cast<int8_t>((words[h] >> (16 * p + 8)) & 0xFF);
      out[2 * h + p] = bf16_bits_rne(static_cast<float>(lo) * a) | (bf16_bits_rne(static_cast<float>(hi) * a) << 16);
    }
  }
  *reinterpret_cast<uint4*>(yq + e0) = make_uint4(out[0], out[1], out[2], out[3]);
}

// four activations of a row as fp32
__device__ __forceinline__ void load_x4(const uint16_t* x, float* f) {
  const uint2 v = *reinterpret_cast<const uint2*>(x);
  f[0] = __uint_as_float(v.x << 16);
  f[1] = __uint_as_float(v.x & 0xFFFF0000u);
  f[2] = __uint_as_float(v.y << 16);
  f[3] = __uint_as_float(v.y & 0xFFFF0000u);
}
__device__ __forceinline__ void load_x4(const float* x, float* f) {
  const float4 v = *reinterpret_cast<const float4*>(x);
  f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
}

// four activations from a buffer resource (zero past its range): the raw
// words, then their fp32 values
constexpr int kBufFlags = 0x00020000;  // gfx9 buffer descriptor word 3
template <typename XT> struct Raw4;
template <> struct Raw4<uint16_t> {
  uint2 v;
  __device__ void load(__amdgpu_buffer_rsrc_t rs, uint32_t k) {
    v = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rs, 2u * k, 0, 0));
  }
  __device__ void to_f32(float* f) const {
    f[0] = __uint_as_float(v.x << 16);
    f[1] = __uint_as_float(v.x & 0xFFFF0000u);
    f[2] = __uint_as_float(v.y << 16);
    f[3] = __uint_as_float(v.y & 0xFFFF0000u);
  }
};
template <> struct Raw4<float> {
  float4 v;
  __device__ void load(__amdgpu_buffer_rsrc_t rs, uint32_t k) {
    v = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, 4u * k, 0, 0));
  }
  __device__ void to_f32(float* f) const { f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w; }
};

// One wave per row: s = sum_k g_k x_k in fp64 over the row, then
// dx = r g - coef x with coef = r^3 s / K (rounded from fp64 once).  VPL > 0:
// the lane keeps its VPL groups of 4 (g and x) in registers between the two
// passes (rows of K <= 256 VPL); VPL == 0 re-reads the row.
template <typename XT, int VPL>
__global__ __launch_bounds__(kBlock) void rms_norm_bwd_kernel(const float* __restrict__ dYs,
                                                              const float* __restrict__ w_scale,
                                                              const XT* __restrict__ x,
                                                              const float* __restrict__ gamma,
                                                              const float* __restrict__ rstd, int64_t M, int K,
                                                              float* __restrict__ dx) {
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= M) return;  // whole wave
  const float w = w_scale[0];
  const float r = rstd[row];
  const float* dr = dYs + row * K;
  const XT* xr = x + row * K;
  auto load_gx = [&](int k, float* g, float* xf) {
    const float4 d = *reinterpret_cast<const float4*>(dr + k);
    const float dv[4] = {d.x, d.y, d.z, d.w};
    load_x4(xr + k, xf);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float dy = w * dv[e];
      g[e] = gamma != nullptr ? gamma[k + e] * dy : dy;
    }
  };
  auto store_dx = [&](int k, const float* g, const float* xf, float coef) {
    float o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = r * g[e] - coef * xf[e];
    *reinterpret_cast<float4*>(dx + row * K + k) = make_float4(o[0], o[1], o[2], o[3]);
  };
  double s = 0.0;
  if constexpr (VPL > 0) {
    // every load of the lane issued at entry, without a branch: dY, x and
    // gamma through buffer resources of the row's size (gamma's: 0 when it
    // is NULL), which read as zero past their ends
    const __amdgpu_buffer_rsrc_t drs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(dr), 0, K * 4, kBufFlags);
    const __amdgpu_buffer_rsrc_t xrs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<XT*>(xr), 0, K * static_cast<int>(sizeof(XT)), kBufFlags);
    const __amdgpu_buffer_rsrc_t grs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(gamma), 0, gamma != nullptr ? K * 4 : 0, kBufFlags);
    float4 dv[VPL], gv[VPL];
    Raw4<XT> xv[VPL];
    float g[VPL][4], xf[VPL][4];
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const uint32_t k = 4u * static_cast<uint32_t>(lane + kWave * i);
      dv[i] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(drs, 4u * k, 0, 0));
      xv[i].load(xrs, k);
      gv[i] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(grs, 4u * k, 0, 0));
    }
    __builtin_amdgcn_sched_barrier(0);  // all loads before the first wait
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      xv[i].to_f32(xf[i]);
      const float d4[4] = {dv[i].x, dv[i].y, dv[i].z, dv[i].w};
      const float g4[4] = {gv[i].x, gv[i].y, gv[i].z, gv[i].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float dy = w * d4[e];
        g[i][e] = gamma != nullptr ? g4[e] * dy : dy;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) s += static_cast<double>(g[i][e]) * static_cast<double>(xf[i][e]);
    }
    s = wave_sum_f64(s);
    const double rd = static_cast<double>(r);
    const float coef = static_cast<float>(rd * rd * rd * s / static_cast<double>(K));
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int k = 4 * (lane + kWave * i);
      if (k < K) store_dx(k, g[i], xf[i], coef);
    }
  } else {
    for (int k = 4 * lane; k < K; k += 4 * kWave) {
      float g[4], xf[4];
      load_gx(k, g, xf);
#pragma unroll
      for (int e = 0; e < 4; ++e) s += static_cast<double>(g[e]) * static_cast<double>(xf[e]);
    }
    s = wave_sum_f64(s);
    const double rd = static_cast<double>(r);
    const float coef = static_cast<float>(rd * rd * rd * s / static_cast<double>(K));
    for (int k = 4 * lane; k < K; k += 4 * kWave) {
      float g[4], xf[4];
      load_gx(k, g, xf);
      store_dx(k, g, xf, coef);
    }
  }
}

// Column sums: partial p of a column is the fp64 sum over the rows
// [p R, (p+1) R), R = max(ceil(M / kMaxParts), kMinRowsPerPart); a final
// pass adds the partials.  Every sum runs in a fixed order, so the results
// are reproducible; 16-byte loads where a row's group of 8 is aligned.
constexpr int64_t kMaxParts = 64;
constexpr int64_t kMinRowsPerPart = 256;

struct SumBf16 {
  const uint16_t* a;
  int64_t cols;
  __device__ void add8(int64_t m, int64_t c0, double* acc) const {
    const uint16_t* p = a + m * cols + c0;
    if ((cols & 7) == 0) {
      const uint4 v = *reinterpret_cast<const uint4*>(p);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += static_cast<double>(__uint_as_float(w[i] << 16));
        acc[2 * i + 1] += static_cast<double>(__uint_as_float(w[i] & 0xFFFF0000u));
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (c0 + e < cols) acc[e] += static_cast<double>(__uint_as_float(static_cast<uint32_t>(p[e]) << 16));
    }
  }
};
template <typename XT>
struct SumDgamma {  // cols = K, a multiple of 16
  const float* dYs;
  const float* w_scale;
  const XT* x;
  const float* rstd;
  int64_t cols;
  __device__ void add8(int64_t m, int64_t c0, double* acc) const {
    const float w = w_scale[0];
    const double r = static_cast<double>(rstd[m]);
    const float4 d0 = *reinterpret_cast<const float4*>(dYs + m * cols + c0);
    const float4 d1 = *reinterpret_cast<const float4*>(dYs + m * cols + c0 + 4);
    const float dv[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
    float xv[8];
    load_x4(x + m * cols + c0, xv);
    load_x4(x + m * cols + c0 + 4, xv + 4);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      acc[e] += static_cast<double>(w * dv[e]) * static_cast<double>(xv[e]) * r;
  }
};

// Partial pass: a workgroup owns 64 columns (8 groups of 8) and the rows
// [p R, (p+1) R); thread (row lane rl, group cg) adds rows m0 + rl + 32 i,
// so a wave reads 8 rows of 64 contiguous columns at a time; the 32 row
// lanes are then added in LDS in a fixed order.
constexpr int kColGroups = 8, kRowLanes = kBlock / kColGroups;  // 8 x 32

template <typename F>
__global__ __launch_bounds__(kBlock) void col_partial_kernel(F f, int64_t M, int64_t cols, int64_t rows_per_part,
                                                             double* partials) {
  __shared__ double red[kRowLanes][kColGroups * 8 + 1];
  const int cg = threadIdx.x % kColGroups, rl = threadIdx.x / kColGroups;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * (kColGroups * 8) + 8 * cg;
  const int64_t p = blockIdx.y;
  const int64_t m0 = p * rows_per_part;
  const int64_t m1 = m0 + rows_per_part < M ? m0 + rows_per_part : M;
  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (c0 < cols) {
#pragma unroll 2
    for (int64_t m = m0 + rl; m < m1; m += kRowLanes) f.add8(m, c0, acc);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rl][8 * cg + e] = acc[e];
  __syncthreads();
  if (threadIdx.x < kColGroups * 8) {
    const int c = threadIdx.x;
    double s = 0.0;
    for (int l = 0; l < kRowLanes; ++l) s += red[l][c];
    const int64_t col = static_cast<int64_t>(blockIdx.x) * (kColGroups * 8) + c;
    if (col < cols) partials[p * cols + col] = s;
  }
}

// Final pass: 32 columns per workgroup, 8 lanes per column over the partials,
// then the lanes in a fixed order.
__global__ __launch_bounds__(kBlock) void col_final_kernel(const double* partials, int64_t nparts, int64_t cols,
                                                           float* out) {
  constexpr int kCols = 32, kLanes = kBlock / kCols;
  __shared__ double red[kLanes][kCols];
  const int c = threadIdx.x % kCols, l = threadIdx.x / kCols;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * kCols + c;
  double acc = 0.0;
  if (col < cols)
    for (int64_t p = l; p < nparts; p += kLanes) acc += partials[p * cols + col];
  red[l][c] = acc;
  __syncthreads();
  if (l == 0 && col < cols) {
    double s = 0.0;
    for (int i = 0; i < kLanes; ++i) s += red[i][c];
    out[col] = static_cast<float>(s);
  }
}

int64_t rows_per_part(int64_t M) {
  int64_t R = (M + kMaxParts - 1) / kMaxParts;
  return R < kMinRowsPerPart ? kMinRowsPerPart : R;
}

template <typename F>
hipError_t col_sum(F f, int64_t M, int64_t cols, double* partials, float* out, hipStream_t stream) {
  const int64_t R = rows_per_part(M);
  const int64_t nparts = (M + R - 1) / R;
  hipLaunchKernelGGL(col_partial_kernel<F>,
                     dim3(static_cast<unsigned>((cols + kColGroups * 8 - 1) / (kColGroups * 8)),
                          static_cast<unsigned>(nparts)),
                     dim3(kBlock), 0, stream, f, M, cols, R, partials);
  hipLaunchKernelGGL(col_final_kernel, dim3(static_cast<unsigned>((cols + 31) / 32)), dim3(kBlock), 0, stream,
                     partials, nparts, cols, out);
  return hipGetLastError();
}

// Sum of S partial products [S][n] into out [n], in order, in fp64.
__global__ __launch_bounds__(kBlock) void sum_parts_kernel(const float* parts, int64_t S, int64_t n, float* out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n) return;
  double acc = 0.0;
  for (int64_t s = 0; s < S; ++s) acc += static_cast<double>(parts[s * n + i]);
  out[i] = static_cast<float>(acc);
}

// One rocBLAS handle per device, created on first use; the stream is set
// under the lock for each call.
struct BlasHandles {
  std::mutex mu;
  rocblas_handle h[64] = {};
};
BlasHandles& blas() {
  static BlasHandles b;
  return b;
}

}  // namespace

hipError_t launch_expand_ternary(const uint32_t* Wpacked, int K, int64_t N, uint16_t* T, hipStream_t stream) {
  const int64_t J = K / 16;
  if (J * N == 0) return hipSuccess;
  hipLaunchKernelGGL(expand_ternary_kernel, dim3(blocks_for(J * N)), dim3(kBlock), 0, stream, Wpacked, J, N, T);
  return hipGetLastError();
}

hipError_t launch_dequant_bf16(const int8_t* q, const float* a_scale, int64_t M, int K, uint16_t* yq,
                               hipStream_t stream) {
  if (M * K == 0) return hipSuccess;
  hipLaunchKernelGGL(dequant_bf16_kernel, dim3(blocks_for(M * K / 8)), dim3(kBlock), 0, stream, q, a_scale, M, K,
                     yq);
  return hipGetLastError();
}

hipError_t launch_rms_norm_bwd(const float* dYs, const float* w_scale, const void* x, bool x_is_f32,
                               const float* gamma, const float* rstd, int64_t M, int K, float* dx,
                               hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((M + kRowsPerBlock - 1) / kRowsPerBlock));
  const int vpl = (K + 4 * kWave - 1) / (4 * kWave);
  auto go = [&](auto xt, auto v) {
    using XT = decltype(xt);
    constexpr int V = decltype(v)::value;
    hipLaunchKernelGGL((rms_norm_bwd_kernel<XT, V>), grid, dim3(kBlock), 0, stream, dYs, w_scale,
                       static_cast<const XT*>(x), gamma, rstd, M, K, dx);
  };
  auto by_vpl = [&](auto xt) {
    if (vpl <= 1) go(xt, std::integral_constant<int, 1>{});
    else if (vpl <= 2) go(xt, std::integral_constant<int, 2>{});
    else if (vpl <= 4) go(xt, std::integral_constant<int, 4>{});
    else if (vpl <= 8) go(xt, std::integral_constant<int, 8>{});
    else go(xt, std::integral_constant<int, 0>{});
  };
  if (x_is_f32)
    by_vpl(float{});
  else
    by_vpl(uint16_t{});
  return hipGetLastError();
}

int64_t col_sum_partials(int64_t M) {
  if (M <= 0) return 1;
  const int64_t R = rows_per_part(M);
  return (M + R - 1) / R;
}

hipError_t launch_col_sum_bf16(const uint16_t* dO, int64_t M, int64_t N, double* partials, float* db,
                               hipStream_t stream) {
  return col_sum(SumBf16{dO, N}, M, N, partials, db, stream);
}

hipError_t launch_dgamma(const float* dYs, const float* w_scale, const void* x, bool x_is_f32,
                         const float* rstd, int64_t M, int K, double* partials, float* dgamma,
                         hipStream_t stream) {
  if (x_is_f32)
    return col_sum(SumDgamma<float>{dYs, w_scale, static_cast<const float*>(x), rstd, K}, M, K, partials, dgamma,
                   stream);
  return col_sum(SumDgamma<uint16_t>{dYs, w_scale, static_cast<const uint16_t*>(x), rstd, K}, M, K, partials,
                 dgamma, stream);
}

int64_t dw_split(int64_t M, int64_t N, int64_t K) {
  // Split the contraction over tokens into S equal parts (S a power of two
  // dividing M, parts of at least 1024 tokens) while the output has fewer than
  // 128 tiles of 256 x 256: a long, narrow product otherwise leaves most of
  // the matrix cores idle.
  const int64_t tiles = ((N + 255) / 256) * ((K + 255) / 256);
  int64_t S = 1;
  while (S < 8 && tiles * S < 128 && M % (2 * S) == 0 && M / (2 * S) >= 1024) S *= 2;
  return S;
}

hipError_t gemm_bf16_dw(int64_t M, int64_t N, int64_t K, const uint16_t* dO, const uint16_t* yq, float* dW,
                        float* parts, hipStream_t stream) {
  const int64_t S = dw_split(M, N, K);
  if (S == 1) return gemm_bf16(true, false, N, K, M, dO, N, yq, K, dW, K, stream, 1, 0, 0, 0);
  const int64_t Ms = M / S;
  const hipError_t e = gemm_bf16(true, false, N, K, Ms, dO, N, yq, K, parts, K, stream, S, Ms * N, Ms * K, N * K);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sum_parts_kernel, dim3(blocks_for(N * K)), dim3(kBlock), 0, stream, parts, S, N * K, dW);
  return hipGetLastError();
}

hipError_t gemm_bf16(bool transA, bool transB, int64_t Mr, int64_t Nc, int64_t Kc, const uint16_t* A,
                     int64_t lda, const uint16_t* B, int64_t ldb, float* C, int64_t ldc, hipStream_t stream,
                     int64_t batch, int64_t strideA, int64_t strideB, int64_t strideC) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  BlasHandles& bh = blas();
  std::lock_guard<std::mutex> lock(bh.mu);
  if (bh.h[dev] == nullptr && rocblas_create_handle(&bh.h[dev]) != rocblas_status_success) {
    bh.h[dev] = nullptr;
    return hipErrorUnknown;
  }
  rocblas_handle h = bh.h[dev];
  if (rocblas_set_stream(h, stream) != rocblas_status_success) return hipErrorUnknown;
  const float alpha = 1.0f, beta = 0.0f;
  // row-major C = op(A) op(B) is column-major C^T = op(B)^T op(A)^T
  const rocblas_operation opB = transB ? rocblas_operation_transpose : rocblas_operation_none;
  const rocblas_operation opA = transA ? rocblas_operation_transpose : rocblas_operation_none;
  rocblas_status st;
  if (batch == 1)
    st = rocblas_gemm_ex(h, opB, opA, static_cast<rocblas_int>(Nc), static_cast<rocblas_int>(Mr),
                         static_cast<rocblas_int>(Kc), &alpha, B, rocblas_datatype_bf16_r,
                         static_cast<rocblas_int>(ldb), A, rocblas_datatype_bf16_r, static_cast<rocblas_int>(lda),
                         &beta, C, rocblas_datatype_f32_r, static_cast<rocblas_int>(ldc), C,
                         rocblas_datatype_f32_r, static_cast<rocblas_int>(ldc), rocblas_datatype_f32_r,
                         rocblas_gemm_algo_standard, 0, 0);
  else
    st = rocblas_gemm_strided_batched_ex(
        h, opB, opA, static_cast<rocblas_int>(Nc), static_cast<rocblas_int>(Mr), static_cast<rocblas_int>(Kc),
        &alpha, B, rocblas_datatype_bf16_r, static_cast<rocblas_int>(ldb), strideB, A, rocblas_datatype_bf16_r,
        static_cast<rocblas_int>(lda), strideA, &beta, C, rocblas_datatype_f32_r, static_cast<rocblas_int>(ldc),
        strideC, C, rocblas_datatype_f32_r, static_cast<rocblas_int>(ldc), strideC,
        static_cast<rocblas_int>(batch), rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  return st == rocblas_status_success ? hipSuccess : hipErrorUnknown;
}

}  // namespace mmf
