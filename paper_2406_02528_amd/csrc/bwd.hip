// Column sums of the BitLinear backward (Algorithm 1, backward_pass): the
// bias gradient db[n] = sum over tokens of dO[m][n], in fp64 and in a fixed
// order, and the fixed-order fp64 sum of the token-range parts of dW when its
// contraction is split (the two products themselves are in bwd_gemm.hip).
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kBlock = 256;

unsigned blocks_for(int64_t threads) { return static_cast<unsigned>((threads + kBlock - 1) / kBlock); }

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

}  // namespace

int64_t col_sum_partials(int64_t M) {
  if (M <= 0) return 1;
  const int64_t R = rows_per_part(M);
  return (M + R - 1) / R;
}

hipError_t launch_col_sum_bf16(const uint16_t* dO, int64_t M, int64_t N, double* partials, float* db,
                               hipStream_t stream) {
  return col_sum(SumBf16{dO, N}, M, N, partials, db, stream);
}

hipError_t launch_col_final(const double* partials, int64_t nparts, int64_t cols, float* out, hipStream_t stream) {
  if (cols == 0) return hipSuccess;
  hipLaunchKernelGGL(col_final_kernel, dim3(static_cast<unsigned>((cols + 31) / 32)), dim3(kBlock), 0, stream,
                     partials, nparts, cols, out);
  return hipGetLastError();
}

hipError_t launch_sum_parts(const float* parts, int64_t S, int64_t n, float* out, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(sum_parts_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, parts, S, n, out);
  return hipGetLastError();
}

}  // namespace mmf
