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

#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kBlock = 256;
constexpr int kRowsPerBlock = kBlock / kWave;  // one wave per row
constexpr int64_t kChunkRows = 64;            // rows per partial of a column sum
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

// One wave per row: s = sum_k g_k x_k in fp64 over the row, then
// dx = r g - coef x with coef = r^3 s / K (rounded from fp64 once).
template <typename XT>
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
  double s = 0.0;
  for (int k = 4 * lane; k < K; k += 4 * kWave) {
    const float4 d = *reinterpret_cast<const float4*>(dr + k);
    const float dv[4] = {d.x, d.y, d.z, d.w};
    float xf[4];
    load_x4(xr + k, xf);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float dy = w * dv[e];
      const float g = gamma != nullptr ? gamma[k + e] * dy : dy;
      s += static_cast<double>(g) * static_cast<double>(xf[e]);
    }
  }
  s = wave_sum_f64(s);
  const double rd = static_cast<double>(r);
  const float coef = static_cast<float>(rd * rd * rd * s / static_cast<double>(K));
  for (int k = 4 * lane; k < K; k += 4 * kWave) {
    const float4 d = *reinterpret_cast<const float4*>(dr + k);
    const float dv[4] = {d.x, d.y, d.z, d.w};
    float xf[4];
    load_x4(xr + k, xf);
    float o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float dy = w * dv[e];
      const float g = gamma != nullptr ? gamma[k + e] * dy : dy;
      o[e] = r * g - coef * xf[e];
    }
    *reinterpret_cast<float4*>(dx + row * K + k) = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// Column sums: partial p of column c is the fp64 sum over rows
// [p kChunkRows, (p+1) kChunkRows); the final pass adds the partials in order.
struct SumBf16 {
  const uint16_t* a;
  int64_t cols;
  __device__ double operator()(int64_t m, int64_t c) const {
    return static_cast<double>(__uint_as_float(static_cast<uint32_t>(a[m * cols + c]) << 16));
  }
};
template <typename XT>
struct SumDgamma {
  const float* dYs;
  const float* w_scale;
  const XT* x;
  const float* rstd;
  int64_t cols;
  __device__ double operator()(int64_t m, int64_t c) const {
    float xv;
    if constexpr (sizeof(XT) == 2)
      xv = __uint_as_float(static_cast<uint32_t>(x[m * cols + c]) << 16);
    else
      xv = x[m * cols + c];
    const float dy = w_scale[0] * dYs[m * cols + c];
    return static_cast<double>(dy) * static_cast<double>(xv) * static_cast<double>(rstd[m]);
  }
};

template <typename F>
__global__ __launch_bounds__(kBlock) void col_partial_kernel(F f, int64_t M, int64_t cols, double* partials) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (c >= cols) return;
  const int64_t p = blockIdx.y;
  const int64_t m0 = p * kChunkRows;
  const int64_t m1 = m0 + kChunkRows < M ? m0 + kChunkRows : M;
  double acc = 0.0;
  for (int64_t m = m0; m < m1; ++m) acc += f(m, c);
  partials[p * cols + c] = acc;
}

__global__ __launch_bounds__(kBlock) void col_final_kernel(const double* partials, int64_t nparts, int64_t cols,
                                                           float* out) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (c >= cols) return;
  double acc = 0.0;
  for (int64_t p = 0; p < nparts; ++p) acc += partials[p * cols + c];
  out[c] = static_cast<float>(acc);
}

template <typename F>
hipError_t col_sum(F f, int64_t M, int64_t cols, double* partials, float* out, hipStream_t stream) {
  const int64_t nparts = col_sum_partials(M);
  if (nparts > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(col_partial_kernel<F>, dim3(blocks_for(cols), static_cast<unsigned>(nparts)), dim3(kBlock), 0,
                     stream, f, M, cols, partials);
  hipLaunchKernelGGL(col_final_kernel, dim3(blocks_for(cols)), dim3(kBlock), 0, stream, partials, nparts, cols, out);
  return hipGetLastError();
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
  if (x_is_f32)
    hipLaunchKernelGGL(rms_norm_bwd_kernel<float>, grid, dim3(kBlock), 0, stream, dYs, w_scale,
                       static_cast<const float*>(x), gamma, rstd, M, K, dx);
  else
    hipLaunchKernelGGL(rms_norm_bwd_kernel<uint16_t>, grid, dim3(kBlock), 0, stream, dYs, w_scale,
                       static_cast<const uint16_t*>(x), gamma, rstd, M, K, dx);
  return hipGetLastError();
}

int64_t col_sum_partials(int64_t M) { return M > 0 ? (M + kChunkRows - 1) / kChunkRows : 1; }

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

hipError_t gemm_bf16(bool transA, bool transB, int64_t Mr, int64_t Nc, int64_t Kc, const uint16_t* A,
                     int64_t lda, const uint16_t* B, int64_t ldb, float* C, int64_t ldc, hipStream_t stream) {
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
  const rocblas_status st = rocblas_gemm_ex(
      h, transB ? rocblas_operation_transpose : rocblas_operation_none,
      transA ? rocblas_operation_transpose : rocblas_operation_none, static_cast<rocblas_int>(Nc),
      static_cast<rocblas_int>(Mr), static_cast<rocblas_int>(Kc), &alpha, B, rocblas_datatype_bf16_r,
      static_cast<rocblas_int>(ldb), A, rocblas_datatype_bf16_r, static_cast<rocblas_int>(lda), &beta, C,
      rocblas_datatype_f32_r, static_cast<rocblas_int>(ldc), C, rocblas_datatype_f32_r,
      static_cast<rocblas_int>(ldc), rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  return st == rocblas_status_success ? hipSuccess : hipErrorUnknown;
}

}  // namespace mmf
