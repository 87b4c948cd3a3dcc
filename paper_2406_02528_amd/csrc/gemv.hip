// Decode contraction (M <= 8 tokens): ternary accumulation on the VALU.
//
// The packed weights are [K/16][N] words, so for a fixed word row j the 64
// lanes of a wave read 64 consecutive columns n (a 256-byte coalesced load)
// and each lane owns one output column: no cross-lane reduction is needed.
// The quantised activations q[m][16j .. 16j+15] are the same for every lane
// and are read with scalar loads.  A workgroup of 16 waves covers 64 columns;
// its waves split the K dimension and their int32 partial sums are added in
// LDS (exact, so the order does not matter).
//
// Per word of 16 weights and per token the work is four v_dot4_i32_i8 of the
// codes c = t + 1 in {0, 1, 2} against q; the epilogue subtracts sum_k q
// (sum q*t = sum q*c - sum q), which turns the code sum into the ternary sum
// of the paper: +q where t = 1, nothing where t = 0, -q where t = -1.
#include "mmf_device.h"
#include "mmf_launch.h"

namespace mmf {
namespace {

constexpr int kGemvWaves = 16;
constexpr int kGemvThreads = kGemvWaves * kWave;
constexpr int kGemvMaxTokens = 8;

template <int MT, Epilogue EP>
__global__ __launch_bounds__(kGemvThreads) void gemv_kernel(
    const int8_t* __restrict__ q, const float* __restrict__ a_scale,
    const int32_t* __restrict__ q_rowsum, const uint32_t* __restrict__ Wp,
    const float* __restrict__ w_scale, void* __restrict__ out, int K, int64_t N) {
  __shared__ int red[kGemvWaves][MT][kWave];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t n = static_cast<int64_t>(blockIdx.x) * kWave + lane;
  const bool col_ok = n < N;
  const int J = K / 16;
  const int per_wave = (J + kGemvWaves - 1) / kGemvWaves;
  const int j_begin = wave * per_wave;
  const int j_end = min(j_begin + per_wave, J);
  const uint32_t* __restrict__ qw = reinterpret_cast<const uint32_t*>(q);
  const int kw = K / 4;  // q words per token row

  int acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = 0;

  const uint32_t* wp = Wp + (col_ok ? n : 0);
#pragma unroll 4
  for (int j = j_begin; j < j_end; ++j) {
    const uint32_t w = col_ok ? wp[static_cast<int64_t>(j) * N] : 0x55555555u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t c = codes4(w, i);
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m] = dot4(c, qw[m * kw + 4 * j + i], acc[m]);
    }
  }

#pragma unroll
  for (int m = 0; m < MT; ++m) red[wave][m][lane] = acc[m];
  __syncthreads();
  if (threadIdx.x < MT * kWave) {
    const int m = threadIdx.x >> 6;
    int s = 0;
#pragma unroll
    for (int w = 0; w < kGemvWaves; ++w) s += red[w][m][lane];
    if (col_ok) {
      const int v = s - q_rowsum[m];
      if constexpr (EP == Epilogue::kDequantF32) {
        static_cast<float*>(out)[m * N + n] = static_cast<float>(v) * (a_scale[m] * w_scale[0]);
      } else {
        static_cast<int32_t*>(out)[m * N + n] = v;
      }
    }
  }
}

template <Epilogue EP>
void launch_tokens(int mt, const ContractArgs& a, int64_t m0, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>((a.N + kWave - 1) / kWave));
  const dim3 block(kGemvThreads);
  const int8_t* q = a.q + m0 * a.K;
  const float* as = a.a_scale ? a.a_scale + m0 : nullptr;
  const int32_t* rs = a.q_rowsum + m0;
  void* out = EP == Epilogue::kDequantF32
                  ? static_cast<void*>(static_cast<float*>(a.out) + m0 * a.N)
                  : static_cast<void*>(static_cast<int32_t*>(a.out) + m0 * a.N);
#define MMF_GEMV(MT)                                                                          \
  case MT:                                                                                    \
    hipLaunchKernelGGL((gemv_kernel<MT, EP>), grid, block, 0, stream, q, as, rs, a.Wpacked, \
                       a.w_scale, out, a.K, a.N);                                            \
    break
  switch (mt) {
    MMF_GEMV(1); MMF_GEMV(2); MMF_GEMV(3); MMF_GEMV(4);
    MMF_GEMV(5); MMF_GEMV(6); MMF_GEMV(7); MMF_GEMV(8);
    default: break;
  }
#undef MMF_GEMV
}

}  // namespace

hipError_t launch_gemv(const ContractArgs& a, hipStream_t stream) {
  for (int64_t m0 = 0; m0 < a.M; m0 += kGemvMaxTokens) {
    const int mt = static_cast<int>(a.M - m0 < kGemvMaxTokens ? a.M - m0 : kGemvMaxTokens);
    if (a.epilogue == Epilogue::kDequantF32)
      launch_tokens<Epilogue::kDequantF32>(mt, a, m0, stream);
    else
      launch_tokens<Epilogue::kRawI32>(mt, a, m0, stream);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace mmf
