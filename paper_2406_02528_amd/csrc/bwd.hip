// Final sums of the BitLinear backward (Algorithm 1, backward_pass): the
// fp64 partials of column sums (db from the dY kernel's row tiles, dgamma's)
// added in a fixed order, and the fixed-order fp64 sum of the token-range
// parts of dW when its contraction is split (the two products and the
// partials themselves are in bwd_gemm.hip).
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kBlock = 256;

unsigned blocks_for(int64_t threads) { return static_cast<unsigned>((threads + kBlock - 1) / kBlock); }

// out[c] = sum of partials [nparts][cols] over p: 8 columns per workgroup,
// 32 lanes per column, lane l taking the partials l, l + 32, ... (their loads
// issued together), then the 32 lane sums of a column added in lane order.
// Both orders are fixed, so the result is the same bits on every call.
__global__ __launch_bounds__(kBlock) void col_final_kernel(const double* partials, int64_t nparts, int64_t cols,
                                                           float* out) {
  constexpr int kCols = 8, kLanes = kBlock / kCols;
  __shared__ double red[kCols][kLanes + 1];
  const int c = threadIdx.x % kCols, l = threadIdx.x / kCols;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * kCols + c;
  double acc = 0.0;
  if (col < cols) {
#pragma unroll 4
    for (int64_t p = l; p < nparts; p += kLanes) acc += partials[p * cols + col];
  }
  red[c][l] = acc;
  __syncthreads();
  if (l == 0 && col < cols) {
    double s = 0.0;
    for (int i = 0; i < kLanes; ++i) s += red[c][i];
    out[col] = static_cast<float>(s);
  }
}

// Sum of S partial products [S][n] into out [n], in order, in fp64.
__global__ __launch_bounds__(kBlock) void sum_parts_kernel(const float* parts, int64_t S, int64_t n, float* out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (i >= n) return;
  double acc = 0.0;
  for (int64_t s = 0; s < S; ++s) acc += static_cast<double>(parts[s * n + i]);
  out[i] = static_cast<float>(acc);
}

}  // namespace

hipError_t launch_col_final(const double* partials, int64_t nparts, int64_t cols, float* out, hipStream_t stream) {
  if (cols == 0) return hipSuccess;
  hipLaunchKernelGGL(col_final_kernel, dim3(static_cast<unsigned>((cols + 7) / 8)), dim3(kBlock), 0, stream,
                     partials, nparts, cols, out);
  return hipGetLastError();
}

hipError_t launch_sum_parts(const float* parts, int64_t S, int64_t n, float* out, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(sum_parts_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, parts, S, n, out);
  return hipGetLastError();
}

}  // namespace mmf
