// fp32 (validation mode) instantiations of the attention kernels.  This unit
// is compiled at -O1: at -O2 and above the ROCm 7.2 compiler crashes (in
// machine copy propagation) on the fp32 forward kernel.
#include "attention_kernels.h"

namespace atom {

hipError_t attn_fwd_f32(const void* qkv, void* o, float* lse, int B, int T, int H, int dh, hipStream_t s) {
  if (dh == 64) return attn::fwd_t<float, 64>(qkv, o, lse, B, T, H, s);
  if (dh == 128) return attn::fwd_t<float, 128>(qkv, o, lse, B, T, H, s);
  return hipErrorInvalidValue;
}

hipError_t attn_bwd_f32(const void* qkv, const void* o, const void* dout, const float* lse, float* delta, void* dqkv,
                        int B, int T, int H, int dh, hipStream_t s) {
  if (dh == 64) return attn::bwd_t<float, 64>(qkv, o, dout, lse, delta, dqkv, B, T, H, s);
  if (dh == 128) return attn::bwd_t<float, 128>(qkv, o, dout, lse, delta, dqkv, B, T, H, s);
  return hipErrorInvalidValue;
}

}  // namespace atom
