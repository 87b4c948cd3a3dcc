// Weight order for the fused GLU up-projection (Sec. "MatMul-free Channel
// Mixer": g = x (*) W_g, u = x (*) W_u, p = SiLU(g) * u).
//
// The two packed projections, [K/16][L] words each, are interleaved into one
// [K/16][2L] array in blocks of 16 columns: gate channels 16b .. 16b + 15,
// then the up channels with the same indices, then the next gate block.  A
// 16-column MFMA block of the prefill kernel then holds 16 gate channels and
// the next block the matching up channels, so the gate is formed in the
// contraction's epilogue without another pass over g and u.
#include "mmf_launch.h"

namespace mmf {
namespace {

__global__ void glu_pack_kernel(const uint32_t* __restrict__ Wg, const uint32_t* __restrict__ Wu,
                                int64_t L, int64_t total, uint32_t* __restrict__ Wgu) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int64_t row = i / (2 * L), c = i % (2 * L);
  const int64_t block = c / 16, within = c % 16;
  const int64_t ch = (block / 2) * 16 + within;
  Wgu[i] = (block % 2 == 0) ? Wg[row * L + ch] : Wu[row * L + ch];
}

}  // namespace

hipError_t launch_glu_pack(const uint32_t* Wg, const uint32_t* Wu, int64_t L, int K, uint32_t* Wgu,
                           hipStream_t stream) {
  const int64_t total = static_cast<int64_t>(K / 16) * 2 * L;
  constexpr int kThreads = 256;
  const int64_t blocks = (total + kThreads - 1) / kThreads;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(glu_pack_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream,
                     Wg, Wu, L, total, Wgu);
  return hipGetLastError();
}

}  // namespace mmf
