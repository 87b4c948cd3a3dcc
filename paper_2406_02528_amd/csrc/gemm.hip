// Prefill contraction (any M, built for M in the thousands): the ternary sum
// as a dense int8 contraction on the gfx950 matrix cores.
//
// At thousands of tokens the ternary accumulation is a dense contraction of
// int8 activations against {-1,0,1} weights, so it runs on
// v_mfma_i32_32x32x32_i8 with exact int32 accumulation.  The weight operand is
// the code c = t + 1 in {0,1,2}; the epilogue subtracts sum_k q (sum q*t =
// sum q*c - sum q) and dequantises.
//
// Operand staging:
//  - A (q, int8 [M][K]) is staged through LDS per 128 x 64 tile.
//  - B needs no LDS: for a 32x32x32 MFMA, lane l supplies column l % 32 and the
//    16 k-values of group l / 32, which is exactly one packed word
//    Wpacked[j][n]; lanes 0-31 read 32 consecutive words.  The word is
//    expanded in registers into four dwords of code bytes.
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BK = 64;              // k per stage (bytes of q per row)
constexpr int kThreads = 256;       // 4 waves, 2 x 2, 64 x 64 each
constexpr int kLdsStride = BK + 16; // padded row stride of the A tile (bytes)

template <Epilogue EP>
__global__ __launch_bounds__(kThreads) void gemm_kernel(
    const int8_t* __restrict__ q, const float* __restrict__ a_scale,
    const int32_t* __restrict__ q_rowsum, const uint32_t* __restrict__ Wp,
    const float* __restrict__ w_scale, void* __restrict__ out, int64_t M, int K, int64_t N,
    int64_t tiles_n) {
  __shared__ __attribute__((aligned(16))) int8_t As[BM * kLdsStride];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t tile = blockIdx.x;
  const int64_t m0 = (tile / tiles_n) * BM;
  const int64_t n0 = (tile % tiles_n) * BN;
  const int J = K / 16;
  const int l32 = lane & 31;
  const int g = lane >> 5;  // k group of this lane inside one MFMA

  v16i acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

  // B columns of this lane for its two 32-column fragments
  int64_t ncol[2];
  bool nok[2];
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) {
    ncol[ni] = n0 + wn * 64 + ni * 32 + l32;
    nok[ni] = ncol[ni] < N;
  }

  for (int k0 = 0; k0 < K; k0 += BK) {
    // ---- A tile: 128 rows x 64 bytes, 512 chunks of 16 bytes ----
    uint4 av[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int chunk = tid + c * kThreads;
      const int row = chunk >> 2;
      const int col = (chunk & 3) * 16;
      const int64_t m = m0 + row;
      if (m < M && k0 + col < K)
        av[c] = *reinterpret_cast<const uint4*>(q + m * K + k0 + col);
      else
        av[c] = make_uint4(0, 0, 0, 0);
    }
    // ---- B words for this stage: 2 k32 steps x 2 column fragments ----
    uint32_t bw[2][2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int j = k0 / 16 + 2 * ks + g;
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bw[ks][ni] = (j < J && nok[ni]) ? Wp[static_cast<int64_t>(j) * N + ncol[ni]] : 0x55555555u;
    }
    __syncthreads();  // previous stage's reads of As are done
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int chunk = tid + c * kThreads;
      const int row = chunk >> 2;
      const int col = (chunk & 3) * 16;
      *reinterpret_cast<uint4*>(As + row * kLdsStride + col) = av[c];
    }
    __syncthreads();

#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      v4i bf[2];
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const uint32_t w = bw[ks][ni];
        bf[ni] = v4i{static_cast<int>(codes4(w, 0)), static_cast<int>(codes4(w, 1)),
                     static_cast<int>(codes4(w, 2)), static_cast<int>(codes4(w, 3))};
      }
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        const int row = wm * 64 + mi * 32 + l32;
        const v4i af = *reinterpret_cast<const v4i*>(As + row * kLdsStride + ks * 32 + g * 16);
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af, bf[ni], acc[mi][ni], 0, 0, 0);
      }
    }
  }

  // ---- epilogue: lane holds column l32, rows 8*(r/4) + 4*g + r%4 ----
  const float ws = (EP == Epilogue::kDequantF32) ? w_scale[0] : 0.0f;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t m = m0 + wm * 64 + mi * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
      if (m >= M) continue;
      const int rs = q_rowsum[m];
      float sc = 0.0f;
      if constexpr (EP == Epilogue::kDequantF32) sc = a_scale[m] * ws;
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        if (!nok[ni]) continue;
        const int v = acc[mi][ni][r] - rs;
        if constexpr (EP == Epilogue::kDequantF32)
          static_cast<float*>(out)[m * N + ncol[ni]] = static_cast<float>(v) * sc;
        else
          static_cast<int32_t*>(out)[m * N + ncol[ni]] = v;
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm(const ContractArgs& a, hipStream_t stream) {
  const int64_t gm = (a.M + BM - 1) / BM;
  const int64_t gn = (a.N + BN - 1) / BN;
  if (gm * gn > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<unsigned>(gm * gn));
  if (a.epilogue == Epilogue::kDequantF32)
    hipLaunchKernelGGL(gemm_kernel<Epilogue::kDequantF32>, grid, dim3(kThreads), 0, stream, a.q,
                       a.a_scale, a.q_rowsum, a.Wpacked, a.w_scale, a.out, a.M, a.K, a.N, gn);
  else
    hipLaunchKernelGGL(gemm_kernel<Epilogue::kRawI32>, grid, dim3(kThreads), 0, stream, a.q,
                       a.a_scale, a.q_rowsum, a.Wpacked, a.w_scale, a.out, a.M, a.K, a.N, gn);
  return hipGetLastError();
}

}  // namespace mmf
