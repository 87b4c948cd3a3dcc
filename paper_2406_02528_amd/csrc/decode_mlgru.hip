// Decode step of the MLGRU output projection: the recurrence and output gate
// o' = g sigmoid(f h + (1 - f) c) formed on load from the gates and the state,
// then the affine (bias) epilogue.
#include "decode_impl.h"

namespace mmf {

hipError_t launch_decode_mlgru(const DecodeArgs& a, hipStream_t stream) {
  if (a.epilogue != Epilogue::kAffineF32) return hipErrorInvalidValue;
  return dec::dispatch<dec::Src::kMlgru, Epilogue::kAffineF32>(a, stream);
}

}  // namespace mmf
