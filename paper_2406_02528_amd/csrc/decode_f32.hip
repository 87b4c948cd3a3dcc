// Fused decode forward from f32 activations x: the dequant, affine (bias and
// per-segment activation) and GLU (SiLU(g) * u) epilogues.
#include "decode_impl.h"

namespace mmf {

hipError_t launch_decode_f32(const DecodeArgs& a, hipStream_t stream) {
  using dec::Src;
  if (a.epilogue == Epilogue::kGluF32) {
    if (a.N % 32 != 0) return hipErrorInvalidValue;
    return dec::dispatch<Src::kF32, Epilogue::kGluF32>(a, stream);
  }
  if (a.epilogue == Epilogue::kAffineF32) return dec::dispatch<Src::kF32, Epilogue::kAffineF32>(a, stream);
  if (a.epilogue == Epilogue::kDequantF32) return dec::dispatch<Src::kF32, Epilogue::kDequantF32>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace mmf
