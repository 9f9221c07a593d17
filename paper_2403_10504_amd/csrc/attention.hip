// Causal self-attention: bf16 instantiations and the dtype/head-size
// dispatch.  The kernels are in attention_kernels.h; the fp32 validation-mode
// instantiations live in attention_f32.hip.
#include <mutex>
#include <vector>

#include "../../include/atom.h"
#include "../../include/atom_kernels.h"
#include "attention_kernels.h"

// Scratch of atom_k_attn_bwd_noalloc: D = rowsum(dO * O), one fp32 per
// (batch, head, query row), which atom_k_attn_bwd takes as a caller-supplied
// argument.  One copy per GPU, kept until the process ends.  In host code the
// name is only a handle: the device address comes from hipGetSymbolAddress.
static __device__ __align__(256) float scratch[ATOM_ATTN_NOALLOC_MAX_ROWS];

namespace {

std::mutex g_scratch_mu;
std::vector<float*> g_scratch;  // device address of `scratch`, per device (null: not resolved yet)

// Device address of `scratch` on the current device, resolved on the first
// call on that device (with it current) and kept.
hipError_t scratch_on_current_device(float** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> l(g_scratch_mu);
  if (static_cast<int>(g_scratch.size()) <= dev) g_scratch.resize(dev + 1, nullptr);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = static_cast<float*>(p);
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

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

extern "C" int atom_k_attn_bwd_noalloc(int dtype, const void* qkv, const void* o, const void* dout, const float* lse,
                                       void* dqkv, int B, int T, int H, int dh, void* stream) {
  using namespace atom;
  if ((dtype != ATOM_F32 && dtype != ATOM_BF16) || !qkv || !o || !dout || !lse || !dqkv) return ATOM_EINVAL;
  if (B <= 0 || T <= 0 || H <= 0) return ATOM_EINVAL;
  if (static_cast<int64_t>(B) * H * T > ATOM_ATTN_NOALLOC_MAX_ROWS) return ATOM_EINVAL;
  float* delta = nullptr;
  if (scratch_on_current_device(&delta) != hipSuccess) return ATOM_EHIP;
  // every D value is written by the backward before it is read: nothing to clear
  const hipError_t e = attn_bwd(dtype == ATOM_BF16 ? DT_BF16 : DT_F32, qkv, o, dout, lse, delta, dqkv, B, T, H, dh,
                                static_cast<hipStream_t>(stream));
  if (e == hipSuccess) return ATOM_OK;
  return e == hipErrorInvalidValue ? ATOM_EINVAL : ATOM_EHIP;
}
