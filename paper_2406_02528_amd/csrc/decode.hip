// Fused decode forward: dispatch over the activation source and epilogue,
// and the shape limits of the decode kernel (the kernel is in decode_impl.h,
// instantiated per activation source in decode_<src>.hip).
#include "decode_impl.h"

namespace mmf {

bool decode_fits(int64_t mt, int K, int64_t N, bool from_x, bool x_is_f32) {
  if (mt < 1 || mt > kDecodeMaxTokens || K <= 0) return false;
  // q of every token row in LDS (padded rows for the matrix-core contraction)
  if (dec::q_region(static_cast<int>(mt), K + 16) > kDecodeMaxLdsQ) return false;
  // 32-bit offsets: the packed array below 2^31 bytes
  if (static_cast<int64_t>(K / 16) * N * 4 >= (int64_t(1) << 31)) return false;
  if (!from_x) return true;
  return dec::needed_vp(static_cast<int>(mt), K, x_is_f32) <= 4;
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  if (a.M < 1 || a.M > kDecodeMaxTokens) return hipErrorInvalidValue;  // the caller slices larger M
  if (a.q != nullptr) return launch_decode_q(a, stream);
  if (a.mlgru_in) return launch_decode_mlgru(a, stream);
  if (a.x_is_f32) return launch_decode_f32(a, stream);
  return launch_decode_bf16(a, stream);
}

}  // namespace mmf
