// Causal self-attention kernel templates; instantiated by attention.hip
// (bf16) and attention_f32.hip (fp32 validation mode).
// Fused causal self-attention on CDNA4 matrix cores (tiled, online softmax;
// the [T, T] score matrix never leaves registers).
//
// Layout: qkv [B*T][3*d] with q, k, v at column offsets 0, d, 2d and head h at
// h*dh inside each; o [B*T][d]; lse [B][H][T] (natural log of the row sum of
// exp(scale * q.k) over the unmasked keys).  scale = 1/sqrt(dh); key j is
// visible to query i iff j <= i.
//
// Workgroup = (64-row tile, batch*head), four waves of 16 rows each.
//   forward : S^T = K Q^T per 64-key tile (lanes hold one query, so the
//             accumulators feed the P V^T product as B operands directly);
//   dK, dV  : one workgroup per 64-key tile loops over the query tiles at or
//             below the diagonal; S = Q K^T, dP = dO V^T, dS = P (dP - D);
//             dV += P^T dO, dK += dS^T Q;
//   dQ      : one workgroup per 64-query tile loops over key tiles; dQ += dS K.
// Splitting dQ from dK/dV makes every output owned by one workgroup, so the
// backward needs no atomics and is bitwise reproducible.
#pragma once
#include "common.h"
#include "launch.h"

namespace atom {
namespace attn {

constexpr int BT = 64;  // rows per tile (queries or keys)
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

template <typename T, int DH>
struct ALay {
  static constexpr int KV = 16 / sizeof(T);  // elements per 16 bytes
  static constexpr int PAD = KV;
  static constexpr int RP = DH + PAD;        // pitch of a [64][DH] tile
  static constexpr int TP = BT + PAD;        // pitch of a transposed [DH][64] tile
  static constexpr int NS = DH / 32;         // 32-wide k slices over dh
  static constexpr int NCT = DH / 16;        // 16-wide column tiles over dh
};

// Stage rows [r0, r0+64) of a head slice (row stride ld) into S[64][RP].
template <typename T, int DH>
__device__ __forceinline__ void stage_rows(T* S, const T* __restrict__ base, int64_t ld, int r0, int nrows,
                                           int tid) {
  using L = ALay<T, DH>;
  constexpr int CPR = DH / L::KV;  // 16-byte chunks per row
  for (int c = tid; c < BT * CPR; c += 256) {
    const int r = c / CPR, k = (c % CPR) * L::KV;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r0 + r < nrows) v = *reinterpret_cast<const uint4*>(base + static_cast<int64_t>(r0 + r) * ld + k);
    *reinterpret_cast<uint4*>(S + r * L::RP + k) = v;
  }
}

// Stage the same rows transposed into S[DH][TP] (S[c][r] = x[r0 + r][c]).
template <typename T, int DH>
__device__ __forceinline__ void stage_rows_t(T* S, const T* __restrict__ base, int64_t ld, int r0, int nrows,
                                             int tid) {
  using L = ALay<T, DH>;
  constexpr int PAIR = 4 / sizeof(T);
  constexpr int UC = DH / PAIR;            // dword columns
  constexpr int UNITS = (BT / L::KV) * UC; // (KV rows x PAIR cols) units
  for (int u = tid; u < UNITS; u += 256) {
    const int rb = u / UC, cc = (u % UC) * PAIR;
    uint32_t d[L::KV];
#pragma unroll
    for (int j = 0; j < L::KV; ++j) {
      const int r = r0 + rb * L::KV + j;
      d[j] = r < nrows ? *reinterpret_cast<const uint32_t*>(base + static_cast<int64_t>(r) * ld + cc) : 0u;
    }
    if constexpr (sizeof(T) == 2) {
      uint4 lo, hi;
      lo.x = (d[0] & 0xffffu) | (d[1] << 16); hi.x = (d[0] >> 16) | (d[1] & 0xffff0000u);
      lo.y = (d[2] & 0xffffu) | (d[3] << 16); hi.y = (d[2] >> 16) | (d[3] & 0xffff0000u);
      lo.z = (d[4] & 0xffffu) | (d[5] << 16); hi.z = (d[4] >> 16) | (d[5] & 0xffff0000u);
      lo.w = (d[6] & 0xffffu) | (d[7] << 16); hi.w = (d[6] >> 16) | (d[7] & 0xffff0000u);
      *reinterpret_cast<uint4*>(S + cc * L::TP + rb * 8) = lo;
      *reinterpret_cast<uint4*>(S + (cc + 1) * L::TP + rb * 8) = hi;
    } else {
      *reinterpret_cast<uint4*>(S + cc * L::TP + rb * 4) = make_uint4(d[0], d[1], d[2], d[3]);
    }
  }
}

// Fragment of a head row (for a register-resident operand): row r, k slice s.
template <typename T>
__device__ __forceinline__ void frag_global(Frag<T>& f, const T* __restrict__ base, int64_t ld, int r, int nrows,
                                            int col) {
  if (r < nrows) frag_load(f, base + static_cast<int64_t>(r) * ld + col);
  else frag_zero(f);
}

// Build the B-operand fragment for a 32-wide slice from two 16-row tiles of
// per-lane accumulator values x[t][r] (t = 2s, 2s+1): element e < 4 takes
// x[2s][e], e >= 4 takes x[2s+1][e-4].  The matching A operand reads rows
// 32s + 4g + e and 32s + 16 + 4g + (e-4) (see frag_pair_rows).
template <typename T>
__device__ __forceinline__ void frag_from_pair(Frag<T>& f, const float (*x)[4], int s) {
  float v[8] = {x[2 * s][0], x[2 * s][1], x[2 * s][2], x[2 * s][3],
                x[2 * s + 1][0], x[2 * s + 1][1], x[2 * s + 1][2], x[2 * s + 1][3]};
  frag_from_f32(f, v);
}
// A-operand fragment from a transposed tile S[c][TP]: row c, slice s.
template <typename T, int DH>
__device__ __forceinline__ void frag_pair_rows(Frag<T>& f, const T* S, int c, int s, int lg) {
  using L = ALay<T, DH>;
  const T* p = S + c * L::TP + 32 * s + 4 * lg;
  frag_load2(f, p, p + 16);
}

template <typename T>
__device__ __forceinline__ void store_row4(T* p, const float* v, int nvalid) {
  if (nvalid == 4) {
    if constexpr (sizeof(T) == 2) {
      uint2 w;
      w.x = static_cast<uint32_t>(f2bf(v[0])) | (static_cast<uint32_t>(f2bf(v[1])) << 16);
      w.y = static_cast<uint32_t>(f2bf(v[2])) | (static_cast<uint32_t>(f2bf(v[3])) << 16);
      *reinterpret_cast<uint2*>(p) = w;
    } else {
      *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    }
  } else {
    for (int r = 0; r < nvalid; ++r) p[r] = from_f<T>(v[r]);
  }
}

// ------------------------------------------------------------------ forward
template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_fwd_kernel(const T* __restrict__ qkv, T* __restrict__ o,
                                                       float* __restrict__ lse, int B, int Tn, int H) {
  using L = ALay<T, DH>;
  __shared__ __attribute__((aligned(16))) T Ks[BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Vt[DH * L::TP];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const T* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const T* kb = qb + d;
  const T* vb = qb + 2 * d;
  const int q0 = blockIdx.x * BT;
  const int qi = q0 + w * 16 + lr;  // this lane's query
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));

  Frag<T> qf[L::NS];
#pragma unroll
  for (int s = 0; s < L::NS; ++s) frag_global(qf[s], qb, ld, qi, Tn, 32 * s + 8 * lg);

  f32x4_t acc_o[L::NCT];
#pragma unroll
  for (int c = 0; c < L::NCT; ++c) acc_o[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_i = -1e30f, l_i = 0.f;

  const int n_kt = min((Tn + BT - 1) / BT, (q0 + BT - 1) / BT + 1);
  for (int kt = 0; kt < n_kt; ++kt) {
    const int j0 = kt * BT;
    __syncthreads();
    stage_rows<T, DH>(Ks, kb, ld, j0, Tn, tid);
    stage_rows_t<T, DH>(Vt, vb, ld, j0, Tn, tid);
    __syncthreads();

    float p[4][4];
    float mloc = -INFINITY;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
      f32x4_t a = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < L::NS; ++s) {
        Frag<T> kf;
        frag_load(kf, Ks + (jt * 16 + lr) * L::RP + 32 * s + 8 * lg);
        mfma16(a, kf, qf[s]);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = j0 + jt * 16 + 4 * lg + r;
        const float x = (j <= qi && j < Tn) ? a[r] * sc : -INFINITY;
        p[jt][r] = x;
        mloc = fmaxf(mloc, x);
      }
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_i, mloc);
    const float alpha = exp2f(m_i - m_new);
    float lsum = 0.f;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p[jt][r] = exp2f(p[jt][r] - m_new);
        lsum += p[jt][r];
      }
    l_i = l_i * alpha + lsum;
    m_i = m_new;
#pragma unroll
    for (int c = 0; c < L::NCT; ++c) acc_o[c] *= alpha;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      Frag<T> pf;
      frag_from_pair(pf, p, s2);
#pragma unroll
      for (int c = 0; c < L::NCT; ++c) {
        Frag<T> vf;
        frag_pair_rows<T, DH>(vf, Vt, c * 16 + lr, s2, lg);
        mfma16(acc_o[c], vf, pf);
      }
    }
  }

  float l_tot = l_i + __shfl_xor(l_i, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  if (qi < Tn) {
    const float inv = 1.f / l_tot;
    T* orow = o + (static_cast<int64_t>(b) * Tn + qi) * d + h * DH;
#pragma unroll
    for (int c = 0; c < L::NCT; ++c) {
      float v[4] = {acc_o[c][0] * inv, acc_o[c][1] * inv, acc_o[c][2] * inv, acc_o[c][3] * inv};
      store_row4<T>(orow + c * 16 + 4 * lg, v, 4);
    }
    if (lg == 0) lse[(static_cast<int64_t>(b) * H + h) * Tn + qi] = (m_i + log2f(l_tot)) * LN2;
  }
}

// ------------------------------------------------------- backward: delta
template <typename T>
__global__ void __launch_bounds__(256) attn_delta_kernel(const T* __restrict__ o, const T* __restrict__ dout,
                                                         float* __restrict__ delta, int64_t n_rows, int Tn, int H,
                                                         int dh) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 4 + w;  // (row, head)
  if (idx >= n_rows * H) return;
  const int64_t row = idx / H;
  const int h = static_cast<int>(idx % H);
  const int64_t off = row * static_cast<int64_t>(H) * dh + static_cast<int64_t>(h) * dh;
  float s = 0.f;
  for (int c = lane; c < dh; c += 64) s += to_f<T>(o[off + c]) * to_f<T>(dout[off + c]);
  s = wave_sum(s);
  if (lane == 0) {
    const int64_t b = row / Tn, t = row % Tn;
    delta[(b * H + h) * Tn + t] = s;
  }
}

// ------------------------------------------------------ backward: dK, dV
template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_bwd_dkdv_kernel(const T* __restrict__ qkv, const T* __restrict__ dout,
                                                            const float* __restrict__ lse,
                                                            const float* __restrict__ delta, T* __restrict__ dqkv,
                                                            int B, int Tn, int H) {
  using L = ALay<T, DH>;
  __shared__ __attribute__((aligned(16))) T Qs[BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Qt[DH * L::TP];
  __shared__ __attribute__((aligned(16))) T Os[BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Ot[DH * L::TP];
  __shared__ float lse_s[BT], del_s[BT];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const T* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const T* kb = qb + d;
  const T* vb = qb + 2 * d;
  const T* ob = dout + static_cast<int64_t>(b) * Tn * d + h * DH;  // dO, row stride d
  const float* lse_b = lse + (static_cast<int64_t>(b) * H + h) * Tn;
  const float* del_b = delta + (static_cast<int64_t>(b) * H + h) * Tn;
  const int j0 = blockIdx.x * BT;
  const int kj = j0 + w * 16 + lr;  // this lane's key
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));

  Frag<T> kf[L::NS], vf[L::NS];
#pragma unroll
  for (int s = 0; s < L::NS; ++s) {
    frag_global(kf[s], kb, ld, kj, Tn, 32 * s + 8 * lg);
    frag_global(vf[s], vb, ld, kj, Tn, 32 * s + 8 * lg);
  }
  f32x4_t acc_dk[L::NCT], acc_dv[L::NCT];
#pragma unroll
  for (int c = 0; c < L::NCT; ++c) {
    acc_dk[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc_dv[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  const int n_qt = (Tn + BT - 1) / BT;
  for (int qt = j0 / BT; qt < n_qt; ++qt) {
    const int i0 = qt * BT;
    __syncthreads();
    stage_rows<T, DH>(Qs, qb, ld, i0, Tn, tid);
    stage_rows_t<T, DH>(Qt, qb, ld, i0, Tn, tid);
    stage_rows<T, DH>(Os, ob, d, i0, Tn, tid);
    stage_rows_t<T, DH>(Ot, ob, d, i0, Tn, tid);
    if (tid < BT) {
      const int i = i0 + tid;
      lse_s[tid] = i < Tn ? lse_b[i] * LOG2E : INFINITY;
      del_s[tid] = i < Tn ? del_b[i] : 0.f;
    }
    __syncthreads();

    float p[4][4], ds[4][4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      f32x4_t sa = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < L::NS; ++s) {
        Frag<T> qf, of;
        frag_load(qf, Qs + (it * 16 + lr) * L::RP + 32 * s + 8 * lg);
        frag_load(of, Os + (it * 16 + lr) * L::RP + 32 * s + 8 * lg);
        mfma16(sa, qf, kf[s]);  // S[i][j]: lane holds key kj, queries 4lg + r
        mfma16(dp, of, vf[s]);  // dP[i][j]
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int il = it * 16 + 4 * lg + r;
        const int i = i0 + il;
        const float pv = (kj <= i && kj < Tn) ? exp2f(sa[r] * sc - lse_s[il]) : 0.f;
        p[it][r] = pv;
        ds[it][r] = pv * (dp[r] - del_s[il]);
      }
    }
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      Frag<T> pf, dsf;
      frag_from_pair(pf, p, s2);
      frag_from_pair(dsf, ds, s2);
#pragma unroll
      for (int c = 0; c < L::NCT; ++c) {
        Frag<T> of, qf;
        frag_pair_rows<T, DH>(of, Ot, c * 16 + lr, s2, lg);
        frag_pair_rows<T, DH>(qf, Qt, c * 16 + lr, s2, lg);
        mfma16(acc_dv[c], of, pf);   // dV^T[c][j]
        mfma16(acc_dk[c], qf, dsf);  // dK^T[c][j]
      }
    }
  }

  if (kj < Tn) {
    const float scale = 1.f / sqrtf(static_cast<float>(DH));
    T* row = dqkv + (static_cast<int64_t>(b) * Tn + kj) * ld + h * DH;
#pragma unroll
    for (int c = 0; c < L::NCT; ++c) {
      float vk[4] = {acc_dk[c][0] * scale, acc_dk[c][1] * scale, acc_dk[c][2] * scale, acc_dk[c][3] * scale};
      float vv[4] = {acc_dv[c][0], acc_dv[c][1], acc_dv[c][2], acc_dv[c][3]};
      store_row4<T>(row + d + c * 16 + 4 * lg, vk, 4);
      store_row4<T>(row + 2 * d + c * 16 + 4 * lg, vv, 4);
    }
  }
}

// ----------------------------------------------------------- backward: dQ
template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_bwd_dq_kernel(const T* __restrict__ qkv, const T* __restrict__ dout,
                                                          const float* __restrict__ lse,
                                                          const float* __restrict__ delta, T* __restrict__ dqkv,
                                                          int B, int Tn, int H) {
  using L = ALay<T, DH>;
  __shared__ __attribute__((aligned(16))) T Ks[BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Kt[DH * L::TP];
  __shared__ __attribute__((aligned(16))) T Vs[BT * L::RP];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const T* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const T* kb = qb + d;
  const T* vb = qb + 2 * d;
  const T* ob = dout + static_cast<int64_t>(b) * Tn * d + h * DH;
  const int q0 = blockIdx.x * BT;
  const int qi = q0 + w * 16 + lr;
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));
  const float lse_i = qi < Tn ? lse[(static_cast<int64_t>(b) * H + h) * Tn + qi] * LOG2E : INFINITY;
  const float del_i = qi < Tn ? delta[(static_cast<int64_t>(b) * H + h) * Tn + qi] : 0.f;

  Frag<T> qf[L::NS], of[L::NS];
#pragma unroll
  for (int s = 0; s < L::NS; ++s) {
    frag_global(qf[s], qb, ld, qi, Tn, 32 * s + 8 * lg);
    frag_global(of[s], ob, d, qi, Tn, 32 * s + 8 * lg);
  }
  f32x4_t acc_dq[L::NCT];
#pragma unroll
  for (int c = 0; c < L::NCT; ++c) acc_dq[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int n_kt = min((Tn + BT - 1) / BT, (q0 + BT - 1) / BT + 1);
  for (int kt = 0; kt < n_kt; ++kt) {
    const int j0 = kt * BT;
    __syncthreads();
    stage_rows<T, DH>(Ks, kb, ld, j0, Tn, tid);
    stage_rows_t<T, DH>(Kt, kb, ld, j0, Tn, tid);
    stage_rows<T, DH>(Vs, vb, ld, j0, Tn, tid);
    __syncthreads();

    float ds[4][4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
      f32x4_t sa = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < L::NS; ++s) {
        Frag<T> kf, vf;
        frag_load(kf, Ks + (jt * 16 + lr) * L::RP + 32 * s + 8 * lg);
        frag_load(vf, Vs + (jt * 16 + lr) * L::RP + 32 * s + 8 * lg);
        mfma16(sa, kf, qf[s]);  // S^T[j][i]: lane holds query qi, keys 4lg + r
        mfma16(dp, vf, of[s]);  // dP^T[j][i]
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = j0 + jt * 16 + 4 * lg + r;
        const float pv = (j <= qi && j < Tn) ? exp2f(sa[r] * sc - lse_i) : 0.f;
        ds[jt][r] = pv * (dp[r] - del_i);
      }
    }
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      Frag<T> dsf;
      frag_from_pair(dsf, ds, s2);
#pragma unroll
      for (int c = 0; c < L::NCT; ++c) {
        Frag<T> kf;
        frag_pair_rows<T, DH>(kf, Kt, c * 16 + lr, s2, lg);
        mfma16(acc_dq[c], kf, dsf);  // dQ^T[c][i]
      }
    }
  }

  if (qi < Tn) {
    const float scale = 1.f / sqrtf(static_cast<float>(DH));
    T* row = dqkv + (static_cast<int64_t>(b) * Tn + qi) * ld + h * DH;
#pragma unroll
    for (int c = 0; c < L::NCT; ++c) {
      float v[4] = {acc_dq[c][0] * scale, acc_dq[c][1] * scale, acc_dq[c][2] * scale, acc_dq[c][3] * scale};
      store_row4<T>(row + c * 16 + 4 * lg, v, 4);
    }
  }
}

template <typename T, int DH>
hipError_t fwd_t(const void* qkv, void* o, float* lse, int B, int Tn, int H, hipStream_t s) {
  dim3 grid((Tn + BT - 1) / BT, B * H), block(256);
  hipLaunchKernelGGL((attn_fwd_kernel<T, DH>), grid, block, 0, s, static_cast<const T*>(qkv), static_cast<T*>(o),
                     lse, B, Tn, H);
  return hipGetLastError();
}

template <typename T, int DH>
hipError_t bwd_t(const void* qkv, const void* o, const void* dout, const float* lse, float* delta, void* dqkv, int B,
                 int Tn, int H, hipStream_t s) {
  const int64_t n_rows = static_cast<int64_t>(B) * Tn;
  hipLaunchKernelGGL(attn_delta_kernel<T>, dim3(static_cast<unsigned>((n_rows * H + 3) / 4)), dim3(256), 0, s,
                     static_cast<const T*>(o), static_cast<const T*>(dout), delta, n_rows, Tn, H, DH);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((Tn + BT - 1) / BT, B * H), block(256);
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, DH>), grid, block, 0, s, static_cast<const T*>(qkv),
                     static_cast<const T*>(dout), lse, delta, static_cast<T*>(dqkv), B, Tn, H);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<T, DH>), grid, block, 0, s, static_cast<const T*>(qkv),
                     static_cast<const T*>(dout), lse, delta, static_cast<T*>(dqkv), B, Tn, H);
  return hipGetLastError();
}

}  // namespace attn
}  // namespace atom
