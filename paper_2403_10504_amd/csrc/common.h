// Device-side helpers shared by the CDNA4 (gfx950) kernels of libatom.
//
// Element types: activations and weights are either fp32 (validation mode) or
// bfloat16 stored as raw uint16 bit patterns.  Accumulation is always fp32.
//
// MFMA convention used by every kernel.  A 16x16 output tile is produced by
// __builtin_amdgcn_mfma_f32_16x16x32_bf16 (bf16) or by eight
// __builtin_amdgcn_mfma_f32_16x16x4f32 (fp32) over a 32-wide slice of the
// contraction index k.  Lane l supplies operand row (or column) l % 16 and the
// eight k values 8*(l/16) .. 8*(l/16)+7 of the slice, as one "fragment".  The
// same (lane group, element) -> k map is used for both operands, so any
// permutation of k inside a slice leaves the contraction unchanged.  That
// freedom lets a kernel feed the fp32 accumulators of one MFMA straight into
// the next one (attention's P tile) by choosing which k each element holds.
// Output: lane l holds D[4*(l/16) + r][l % 16] in accumulator r (r = 0..3).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

#define ATOM_DEV __device__ __forceinline__

ATOM_DEV float bf2f(bf16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// fp32 -> bf16, round to nearest even, NaN stays NaN: the gfx950 hardware
// conversion (pairs of calls fuse into one v_cvt_pk_bf16_f32).
ATOM_DEV bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f)); }

// Two fp32 -> one dword of two bf16 (a low, b high), round to nearest even:
// one v_cvt_pk_bf16_f32 (converting separately and packing with shifts cost
// three instructions per pair).
ATOM_DEV uint32_t pack_bf16(float a, float b) {
  typedef float f2v __attribute__((ext_vector_type(2)));
  typedef __bf16 b2v __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2v{a, b}), b2v));
}

template <typename T> ATOM_DEV float to_f(T v);
template <> ATOM_DEV float to_f<float>(float v) { return v; }
template <> ATOM_DEV float to_f<bf16_t>(bf16_t v) { return bf2f(v); }

template <typename T> ATOM_DEV T from_f(float v);
template <> ATOM_DEV float from_f<float>(float v) { return v; }
template <> ATOM_DEV bf16_t from_f<bf16_t>(float v) { return f2bf(v); }

// A fragment: eight consecutive-k elements of one operand row for one lane.
template <typename T> struct Frag;
template <> struct Frag<bf16_t> { uint4 v; };
template <> struct Frag<float> { float4 lo, hi; };

// Load a fragment from 8 contiguous elements (16-byte aligned for bf16,
// 32-byte aligned for fp32), from LDS or global memory.
ATOM_DEV void frag_load(Frag<bf16_t>& f, const bf16_t* p) { f.v = *reinterpret_cast<const uint4*>(p); }
ATOM_DEV void frag_load(Frag<float>& f, const float* p) {
  f.lo = *reinterpret_cast<const float4*>(p);
  f.hi = *reinterpret_cast<const float4*>(p + 4);
}
// Load a fragment from two runs of four contiguous elements (elements 0..3
// from p0, 4..7 from p1).
ATOM_DEV void frag_load2(Frag<bf16_t>& f, const bf16_t* p0, const bf16_t* p1) {
  uint2 a = *reinterpret_cast<const uint2*>(p0);
  uint2 b = *reinterpret_cast<const uint2*>(p1);
  f.v = make_uint4(a.x, a.y, b.x, b.y);
}
ATOM_DEV void frag_load2(Frag<float>& f, const float* p0, const float* p1) {
  f.lo = *reinterpret_cast<const float4*>(p0);
  f.hi = *reinterpret_cast<const float4*>(p1);
}
ATOM_DEV void frag_zero(Frag<bf16_t>& f) { f.v = make_uint4(0, 0, 0, 0); }
ATOM_DEV void frag_zero(Frag<float>& f) {
  f.lo = make_float4(0.f, 0.f, 0.f, 0.f);
  f.hi = f.lo;
}
// Build a fragment from eight fp32 values (rounded to the element type).
ATOM_DEV void frag_from_f32(Frag<bf16_t>& f, const float* x) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = pack_bf16(x[2 * i], x[2 * i + 1]);
  f.v = make_uint4(w[0], w[1], w[2], w[3]);
}
ATOM_DEV void frag_from_f32(Frag<float>& f, const float* x) {
  f.lo = make_float4(x[0], x[1], x[2], x[3]);
  f.hi = make_float4(x[4], x[5], x[6], x[7]);
}

// LDS byte address of a __shared__ object.
ATOM_DEV uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)(p)));
}

// One 16-byte direct global-to-LDS load per lane: lane i of the wave writes
// LDS bytes lds + 16 i (lds wave-uniform).  Issued as inline assembly so
// that the compiler does not track these LDS writes (its conservative
// tracking drains every load in flight before LDS reads it cannot attribute
// to a stage); kernels order them with explicit vmcnt waits and barriers.
ATOM_DEV void lds_dma16(const void* gptr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(gptr), "s"(lds) : "memory", "m0");
}

// ds_read_b64_tr_b16: each lane of a 16-lane group names 8 bytes (4 bf16 of
// one row r = lane >> 2 of a 4-row block, columns 4 (lane & 3) .. +3); lane l
// receives column l of the block's 4 rows, in row order.
ATOM_DEV uint2 ds_read_tr8(const void* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  const v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(const_cast<void*>(p)));
  return make_uint2(static_cast<uint32_t>(static_cast<uint16_t>(v[0])) | (static_cast<uint32_t>(static_cast<uint16_t>(v[1])) << 16),
                    static_cast<uint32_t>(static_cast<uint16_t>(v[2])) | (static_cast<uint32_t>(static_cast<uint16_t>(v[3])) << 16));
}

// acc += A_frag x B_frag over one 32-wide k slice (16x16 output tile).
ATOM_DEV void mfma16(f32x4_t& acc, const Frag<bf16_t>& a, const Frag<bf16_t>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                 __builtin_bit_cast(bf16x8_t, b.v), acc, 0, 0, 0);
}
ATOM_DEV void mfma16(f32x4_t& acc, const Frag<float>& a, const Frag<float>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.x, b.lo.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.y, b.lo.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.z, b.lo.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.w, b.lo.w, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.x, b.hi.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.y, b.hi.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.z, b.hi.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.w, b.hi.w, acc, 0, 0, 0);
}

// Wavefront (64 lanes) reductions.
ATOM_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
ATOM_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Reductions over the lane pairs (l, l ^ 16) and (l, l ^ 32) on the VALU:
// v_permlane16_swap / v_permlane32_swap exchange rows of 16 (32) lanes
// between two registers, so with both operands = v a lane ends up holding
// the even-row and the odd-row value of its pair in that order (the same
// order in both lanes of the pair, so both get the same bits).  A
// __shfl_xor goes through the LDS crossbar (ds_bpermute) with its latency.
ATOM_DEV void pair16(float v, float& lo, float& hi) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
ATOM_DEV void pair32(float v, float& lo, float& hi) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
// max and sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48, as
// (v0 op v1) op (v2 op v3) with v_k the value of row k of the wave.
ATOM_DEV float rows4_max(float v) {
  float a, b;
  pair16(v, a, b);
  pair32(fmaxf(a, b), a, b);
  return fmaxf(a, b);
}
ATOM_DEV float rows4_sum(float v) {
  float a, b;
  pair16(v, a, b);
  pair32(a + b, a, b);
  return a + b;
}

// GELU, tanh form, and its derivative.
// GELU, tanh form, through 0.5 (1 + tanh y) = s = 1 / (1 + exp(-2y)) with
// y = c (u + a u^3): one hardware exp2 and one reciprocal (each within a few
// units in the last place) instead of a library tanh.  s saturates cleanly:
// exp2 overflows to inf for y << 0 (s = 0), and goes to 0 for y >> 0 (s = 1).
ATOM_DEV float gelu_s(float u) {
  const float c = 0.7978845608028654f, a = 0.044715f, m2log2e = -2.8853900817779268f;  // -2 log2(e)
  const float y = c * (u + a * u * u * u);
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(m2log2e * y));
}
ATOM_DEV float gelu_f(float u) { return u * gelu_s(u); }
// d/du [u s] = s + u * 2 s (1 - s) * c (1 + 3 a u^2), since 1 - tanh^2 = 4 s (1 - s).
ATOM_DEV float gelu_grad_f(float u) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  const float s = gelu_s(u);
  return s + 2.f * u * s * (1.f - s) * c * (1.f + 3.f * a * u * u);
}
