// Decode contraction from pre-quantised activations (q, a_scale, q_rowsum):
// the dequant and raw int32 epilogues.
#include "decode_impl.h"

namespace mmf {

hipError_t launch_decode_q(const DecodeArgs& a, hipStream_t stream) {
  using dec::Src;
  if (a.epilogue == Epilogue::kDequantF32) return dec::dispatch<Src::kQuantised, Epilogue::kDequantF32>(a, stream);
  if (a.epilogue == Epilogue::kRawI32) return dec::dispatch<Src::kQuantised, Epilogue::kRawI32>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace mmf
