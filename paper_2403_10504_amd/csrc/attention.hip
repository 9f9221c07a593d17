// Causal self-attention: bf16 instantiations and the dtype/head-size
// dispatch.  The kernels are in attention_kernels.h; the fp32 validation-mode
// instantiations live in attention_f32.hip.
#include "attention_kernels.h"

namespace atom {

// fp32 instantiations (attention_f32.hip).
hipError_t attn_fwd_f32(const void* qkv, void* o, float* lse, int B, int T, int H, int dh, hipStream_t s);
hipError_t attn_bwd_f32(const void* qkv, const void* o, const void* dout, const float* lse, float* delta, void* dqkv,
                        int B, int T, int H, int dh, hipStream_t s);

hipError_t attn_fwd(int dtype, const void* qkv, void* o, float* lse, int B, int T, int H, int dh, hipStream_t s) {
  if (B <= 0 || T <= 0 || H <= 0) return hipErrorInvalidValue;
  if (dtype != DT_BF16) return attn_fwd_f32(qkv, o, lse, B, T, H, dh, s);
  if (dh == 64) return attn::fwd_t<bf16_t, 64>(qkv, o, lse, B, T, H, s);
  if (dh == 128) return attn::fwd_t<bf16_t, 128>(qkv, o, lse, B, T, H, s);
  return hipErrorInvalidValue;
}

hipError_t attn_bwd(int dtype, const void* qkv, const void* o, const void* dout, const float* lse, float* delta,
                    void* dqkv, int B, int T, int H, int dh, hipStream_t s) {
  if (B <= 0 || T <= 0 || H <= 0) return hipErrorInvalidValue;
  if (dtype != DT_BF16) return attn_bwd_f32(qkv, o, dout, lse, delta, dqkv, B, T, H, dh, s);
  if (dh == 64) return attn::bwd_t<bf16_t, 64>(qkv, o, dout, lse, delta, dqkv, B, T, H, s);
  if (dh == 128) return attn::bwd_t<bf16_t, 128>(qkv, o, dout, lse, delta, dqkv, B, T, H, s);
  return hipErrorInvalidValue;
}

}  // namespace atom
