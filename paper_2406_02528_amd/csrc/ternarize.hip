// Weight ternarisation and 2-bit packing (Algorithm 1, weight_quant):
//   w_scale = max(mean |W|, 1e-5) over the whole tensor (fp64 sum -> fp32),
//   t = clamp(round_half_even(W * (1 / w_scale)), -1, 1),
// packed as code t + 1 into the [K/16][N] uint32 layout.  Offline: runs once
// per weight tensor.  Three launches: per-block fp64 partial sums of |W| in a
// fixed assignment, a one-block finalise, and a tiled pack that reads W rows
// coalesced and writes packed rows coalesced through an LDS transpose.  The
// reduction order is fixed, so repeated calls give identical bits.
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kSumThreads = 256;
constexpr int kMaxPartials = 1024;

__device__ double block_sum_f64(double v, double* red) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
#pragma unroll
  for (int s = kSumThreads / 2; s > 0; s >>= 1) {
    if (tid < s) red[tid] += red[tid + s];
    __syncthreads();
  }
  return red[0];
}

// Block b sums |W| over elements [b * chunk, min((b + 1) * chunk, count)).
__global__ __launch_bounds__(kSumThreads) void sum_abs_kernel(
    const float* __restrict__ W, int64_t count, int64_t chunk, double* __restrict__ partials) {
  __shared__ double red[kSumThreads];
  const int64_t begin = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t end = min(begin + chunk, count);
  // count and chunk are multiples of 4, W is 16-byte aligned.  Four loads
  // per thread go out together and feed four independent fp64 sums (one
  // chain of dependent adds per load would hold each thread to one load in
  // flight).
  constexpr int64_t kStride = 4 * kSumThreads;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  int64_t i = begin + 4 * threadIdx.x;
  for (; i + 3 * kStride < end; i += 4 * kStride) {
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const float4*>(W + i + u * kStride);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      acc[u] += static_cast<double>(fabsf(v[u].x));
      acc[u] += static_cast<double>(fabsf(v[u].y));
      acc[u] += static_cast<double>(fabsf(v[u].z));
      acc[u] += static_cast<double>(fabsf(v[u].w));
    }
  }
  for (; i < end; i += kStride) {
    const float4 v = *reinterpret_cast<const float4*>(W + i);
    acc[0] += static_cast<double>(fabsf(v.x));
    acc[0] += static_cast<double>(fabsf(v.y));
    acc[0] += static_cast<double>(fabsf(v.z));
    acc[0] += static_cast<double>(fabsf(v.w));
  }
  const double total = block_sum_f64((acc[0] + acc[1]) + (acc[2] + acc[3]), red);
  if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

__global__ __launch_bounds__(kSumThreads) void finalize_scale_kernel(
    const double* __restrict__ partials, int n_partials, int64_t count, float* __restrict__ w_scale) {
  __shared__ double red[kSumThreads];
  double acc = 0.0;
  for (int i = threadIdx.x; i < n_partials; i += kSumThreads) acc += partials[i];
  const double total = block_sum_f64(acc, red);
  if (threadIdx.x == 0) {
    const double mean = total / static_cast<double>(count);
    w_scale[0] = fmaxf(static_cast<float>(mean), 1e-5f);
  }
}

// Tile: 64 output rows n x 16 packed words j (256 k).  Each wave packs 16 rows:
// lane l reads W[n][16 j0 + 4 l .. + 3] (one 1 KB coalesced read per row),
// forms the bits of its four codes, and a quad OR merges the four lanes that
// share a word.  Words go through LDS so that the [K/16][N] output is written
// as 256-byte rows.
constexpr int kPackRows = 64;
constexpr int kPackWords = 16;

__global__ __launch_bounds__(256) void pack_kernel(
    const float* __restrict__ W, const float* __restrict__ w_scale, uint32_t* __restrict__ Wp,
    int64_t N, int K) {
  __shared__ uint32_t tile[kPackWords][kPackRows];
  const int J = K / 16;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * kPackRows;
  const int j0 = blockIdx.y * kPackWords;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const float s = 1.0f / w_scale[0];
  const int jl = lane >> 2;   // word within the tile
  const int i = lane & 3;     // which group of four k inside the word
  const bool word_ok = (j0 + jl) < J;

  for (int r = 0; r < kPackRows / 4; ++r) {
    const int nl = wave * (kPackRows / 4) + r;
    const int64_t n = n0 + nl;
    uint32_t bits = 0;
    if (n < N && word_ok) {
      const float4 v = *reinterpret_cast<const float4*>(W + n * K + 16 * (j0 + jl) + 4 * i);
      const float w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        float t = __builtin_rintf(w4[b] * s);
        t = fminf(fmaxf(t, -1.0f), 1.0f);
        const uint32_t code = static_cast<uint32_t>(static_cast<int>(t) + 1);
        bits |= code << (8 * b + 2 * i);
      }
    }
    bits |= static_cast<uint32_t>(dpp_i32<kDppXor1>(static_cast<int>(bits)));
    bits |= static_cast<uint32_t>(dpp_i32<kDppXor2>(static_cast<int>(bits)));
    if (i == 0) tile[jl][nl] = bits;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < (kPackWords * kPackRows) / 256; ++r) {
    const int jl2 = r * 4 + wave;
    const int64_t n = n0 + lane;
    if (j0 + jl2 < J && n < N) Wp[static_cast<int64_t>(j0 + jl2) * N + n] = tile[jl2][lane];
  }
}

__global__ __launch_bounds__(256) void row_sum_kernel(const int8_t* __restrict__ q,
                                                      int32_t* __restrict__ rowsum, int64_t M, int K) {
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int8_t* qr = q + row * K;
  int acc = 0;
  for (int v = lane; v < K / 4; v += kWave) {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(qr + 4 * v);
    acc = dot4(w, 0x01010101u, acc);
  }
  acc = wave_sum_i32(acc);
  if (lane == 0) rowsum[row] = acc;
}

int64_t sum_chunk(int64_t count, int blocks) {
  int64_t chunk = (count + blocks - 1) / blocks;
  return (chunk + 3) & ~static_cast<int64_t>(3);
}

}  // namespace

int ternarize_partials_count(int64_t count) {
  int64_t b = (count + 256 * 64 - 1) / (256 * 64);
  if (b < 1) b = 1;
  if (b > kMaxPartials) b = kMaxPartials;
  return static_cast<int>(b);
}

hipError_t launch_ternarize(const float* W, int64_t N, int K, uint32_t* Wpacked,
                            float* w_scale, double* partials, hipStream_t stream) {
  const int64_t count = N * static_cast<int64_t>(K);
  const int blocks = ternarize_partials_count(count);
  const int64_t chunk = sum_chunk(count, blocks);
  hipLaunchKernelGGL(sum_abs_kernel, dim3(blocks), dim3(kSumThreads), 0, stream, W, count, chunk,
                     partials);
  hipLaunchKernelGGL(finalize_scale_kernel, dim3(1), dim3(kSumThreads), 0, stream, partials,
                     blocks, count, w_scale);
  const int J = K / 16;
  const dim3 grid(static_cast<unsigned>((N + kPackRows - 1) / kPackRows),
                  static_cast<unsigned>((J + kPackWords - 1) / kPackWords));
  hipLaunchKernelGGL(pack_kernel, grid, dim3(256), 0, stream, W, w_scale, Wpacked, N, K);
  return hipGetLastError();
}

hipError_t launch_row_sum(const int8_t* q, int32_t* q_rowsum, int64_t M, int K,
                          hipStream_t stream) {
  if (M == 0) return hipSuccess;
  hipLaunchKernelGGL(row_sum_kernel, dim3(static_cast<unsigned>((M + 3) / 4)), dim3(256), 0, stream,
                     q, q_rowsum, M, K);
  return hipGetLastError();
}

}  // namespace mmf
