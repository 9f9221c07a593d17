// Row- and column-wise kernels of the GPT step: LayerNorm forward and
// backward, deterministic column sums (bias and LayerNorm-parameter grads),
// token/position embedding forward and backward, softmax cross-entropy, and
// small helpers.  All are HBM-bound: each reads its inputs once with
// coalesced accesses and reduces inside a wavefront or a workgroup in a fixed
// order, so every result is bitwise reproducible.
#include "common.h"
#include "launch.h"

namespace atom {
namespace {

constexpr float LN_EPS = 1e-5f;

// ---------------------------------------------------------------- LayerNorm
// Workgroup reductions: wavefront shuffles, then the four wave sums in order,
// so results do not depend on scheduling.
__device__ __forceinline__ float block_sum4(float v, float* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_sum(v);
  if (lane == 0) sh[w] = v;
  __syncthreads();
  const float r = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  __syncthreads();
  return r;
}

// Backward: LNB_ROWS consecutive rows per workgroup; per-thread partial
// column sums of dy*xhat and dy go to part[block][2][d].
constexpr int LNB_ROWS = 16;

template <typename T, int MAXE>
__global__ void __launch_bounds__(256) ln_bwd_kernel(const T* __restrict__ dy, const float* __restrict__ x,
                                                     const float* __restrict__ mean, const float* __restrict__ rstd,
                                                     const T* __restrict__ gamma, float* __restrict__ dres,
                                                     T* __restrict__ dres_lp, int accumulate,
                                                     float* __restrict__ part, int64_t rows, int d) {
  // colacc[0][c] / colacc[1][c]: this workgroup's running sums of dy*xhat and
  // dy for column c (each column is owned by one thread).
  extern __shared__ float colacc[];
  __shared__ float sh[4];
  const int tid = threadIdx.x;
  for (int c = tid; c < 2 * d; c += 256) colacc[c] = 0.f;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * LNB_ROWS;
#pragma unroll 1
  for (int rr = 0; rr < LNB_ROWS; ++rr) {
    const int64_t row = r0 + rr;
    if (row >= rows) break;
    const float mu = mean[row], r = rstd[row];
    const T* dyr = dy + row * d;
    const float* xr = x + row * d;
    float* dr = dres + row * d;
    float dyv[MAXE], xh[MAXE];
    float sa = 0.f, sb = 0.f;
#pragma unroll
    for (int i = 0; i < MAXE; ++i) {
      const int c = tid + 256 * i;
      dyv[i] = 0.f;
      xh[i] = 0.f;
      if (c < d) {
        dyv[i] = to_f<T>(dyr[c]);
        xh[i] = (xr[c] - mu) * r;
        const float gp = dyv[i] * to_f<T>(gamma[c]);
        sa += gp;
        sb += gp * xh[i];
        colacc[c] += dyv[i] * xh[i];
        colacc[d + c] += dyv[i];
      }
    }
    const float a = block_sum4(sa, sh) / static_cast<float>(d);
    const float b = block_sum4(sb, sh) / static_cast<float>(d);
#pragma unroll
    for (int i = 0; i < MAXE; ++i) {
      const int c = tid + 256 * i;
      if (c < d) {
        const float dx = r * (dyv[i] * to_f<T>(gamma[c]) - a - xh[i] * b);
        const float o = accumulate ? dr[c] + dx : dx;
        dr[c] = o;
        if (dres_lp) dres_lp[row * d + c] = from_f<T>(o);
      }
    }
  }
  float* p = part + static_cast<int64_t>(blockIdx.x) * 2 * d;
  for (int c = tid; c < 2 * d; c += 256) p[c] = colacc[c];
}

// Backward, one wavefront per row (d a multiple of 256, at most 64*4*LNW_MAXCH).
// Lane l owns columns 4l + 256j (j < nch = d/256), read as 4-element vectors
// (8 bytes bf16, 16 bytes fp32), so every load of a wave is one contiguous
// 512- or 1024-byte run and row sums need only wavefront shuffles.  Each wave
// takes rpw consecutive rows and keeps its column sums of dy*xhat and dy in
// registers; the four waves' sums are added in LDS in wave order into one
// partial per workgroup (part[block][2][d]).
constexpr int LNW_MAXCH = 20;

// Rows per wave: 4 when there are enough rows to give every compute unit a
// workgroup, else 2.
inline int lnw_rows_per_wave(int64_t rows) { return rows >= 4096 ? 4 : 2; }

template <typename T> struct Vec4;
template <> struct Vec4<bf16_t> {
  uint2 v;
  ATOM_DEV void load(const bf16_t* p) { v = *reinterpret_cast<const uint2*>(p); }
  ATOM_DEV float get(int i) const {
    const uint32_t w = i < 2 ? v.x : v.y;
    return __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  ATOM_DEV static void store(bf16_t* p, const float* f) {
    uint2 o;
    o.x = pack_bf16(f[0], f[1]);
    o.y = pack_bf16(f[2], f[3]);
    *reinterpret_cast<uint2*>(p) = o;
  }
};
template <> struct Vec4<float> {
  float4 v;
  ATOM_DEV void load(const float* p) { v = *reinterpret_cast<const float4*>(p); }
  ATOM_DEV float get(int i) const { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }
  ATOM_DEV static void store(float* p, const float* f) {
    *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
  }
};

// Forward, one workgroup per row: four consecutive columns per thread and
// pass (16-byte loads of x, 8-byte bf16 stores), NV passes cover d.
template <typename T, int NV>
__global__ void __launch_bounds__(256) ln_fwd_kernel(const float* __restrict__ x, const T* __restrict__ gamma,
                                                     const T* __restrict__ beta, T* __restrict__ y,
                                                     float* __restrict__ mean, float* __restrict__ rstd, int d) {
  __shared__ float sh[4];
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;
  const float* xr = x + row * d;
  float v[NV][4];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = 4 * tid + 1024 * i;
    const float4 t = c < d ? *reinterpret_cast<const float4*>(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    v[i][0] = t.x;
    v[i][1] = t.y;
    v[i][2] = t.z;
    v[i][3] = t.w;
    s += (t.x + t.y) + (t.z + t.w);
  }
  const float mu = block_sum4(s, sh) / static_cast<float>(d);
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (4 * tid + 1024 * i < d) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t = v[i][e] - mu;
        q += t * t;
      }
    }
  const float var = block_sum4(q, sh) / static_cast<float>(d);
  const float r = 1.f / sqrtf(var + LN_EPS);
  T* yr = y + row * d;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = 4 * tid + 1024 * i;
    if (c < d) {
      Vec4<T> g, b;
      g.load(gamma + c);
      b.load(beta + c);
      float o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = (v[i][e] - mu) * r * g.get(e) + b.get(e);
      Vec4<T>::store(yr + c, o);
    }
  }
  if (tid == 0) {
    mean[row] = mu;
    rstd[row] = r;
  }
}

template <typename T, int MAXCH>
__global__ void __launch_bounds__(256) ln_bwd_wave_kernel(const T* __restrict__ dy, const float* __restrict__ x,
                                                          const float* __restrict__ mean,
                                                          const float* __restrict__ rstd, const T* __restrict__ gamma,
                                                          float* __restrict__ dres, T* __restrict__ dres_lp,
                                                          int accumulate, float* __restrict__ part, int64_t rows,
                                                          int d, int rpw) {
  extern __shared__ float red[];  // [4][d]
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nch = d >> 8;
  float ca[MAXCH * 4], cb[MAXCH * 4];
#pragma unroll
  for (int i = 0; i < MAXCH * 4; ++i) {
    ca[i] = 0.f;
    cb[i] = 0.f;
  }
  const float inv_d = 1.f / static_cast<float>(d);
  const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * 4 + w) * rpw;
  for (int rr = 0; rr < rpw; ++rr) {
    const int64_t row = row0 + rr;
    if (row >= rows) break;  // uniform over the wave
    const float mu = mean[row], r = rstd[row];
    float dyv[MAXCH * 4], xh[MAXCH * 4];
    float sa = 0.f, sb = 0.f;
#pragma unroll
    for (int j = 0; j < MAXCH; ++j) {
      if (j < nch) {
        const int c = 4 * lane + 256 * j;
        Vec4<T> vy, vg;
        vy.load(dy + row * d + c);
        vg.load(gamma + c);
        const float4 xv = *reinterpret_cast<const float4*>(x + row * d + c);
        const float xs[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float g = vy.get(i), h = (xs[i] - mu) * r;
          dyv[4 * j + i] = g;
          xh[4 * j + i] = h;
          const float gp = g * vg.get(i);
          sa += gp;
          sb += gp * h;
          ca[4 * j + i] += g * h;
          cb[4 * j + i] += g;
        }
      }
    }
    const float a = wave_sum(sa) * inv_d, b = wave_sum(sb) * inv_d;
#pragma unroll
    for (int j = 0; j < MAXCH; ++j) {
      if (j < nch) {
        const int c = 4 * lane + 256 * j;
        Vec4<T> vg;
        vg.load(gamma + c);
        float* dr = dres + row * d + c;
        float o[4];
        if (accumulate) {
          const float4 prev = *reinterpret_cast<const float4*>(dr);
          o[0] = prev.x;
          o[1] = prev.y;
          o[2] = prev.z;
          o[3] = prev.w;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float dx = r * (dyv[4 * j + i] * vg.get(i) - a - xh[4 * j + i] * b);
          o[i] = accumulate ? o[i] + dx : dx;
        }
        *reinterpret_cast<float4*>(dr) = make_float4(o[0], o[1], o[2], o[3]);
        if (dres_lp) Vec4<T>::store(dres_lp + row * d + c, o);
      }
    }
  }
  // workgroup partial: the four waves' column sums, added in wave order
  float* p = part + static_cast<int64_t>(blockIdx.x) * 2 * d;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const float* src = q == 0 ? ca : cb;
#pragma unroll
    for (int j = 0; j < MAXCH; ++j)
      if (j < nch)
        *reinterpret_cast<float4*>(red + w * d + 4 * lane + 256 * j) =
            make_float4(src[4 * j], src[4 * j + 1], src[4 * j + 2], src[4 * j + 3]);
    __syncthreads();
    for (int c = threadIdx.x; c < d; c += 256) p[q * d + c] = ((red[c] + red[d + c]) + red[2 * d + c]) + red[3 * d + c];
    __syncthreads();
  }
}

// Backward for d >= 1024: one workgroup (four waves) per block of LNT_ROWS
// consecutive rows.  Thread t owns columns 4t + 1024j (j < NCH, 4-vector
// loads), so each wave reads contiguous 512-byte (bf16) or 1 KB (fp32) runs;
// every thread keeps gamma and its columns' running sums of dy*xhat and dy
// in registers over the block's rows and writes them as the block's partial
// (part[block][2][d]), no LDS pass.  The row sums meet in LDS (one barrier
// per row, double-buffered), and the next row's dy and x are requested
// before the current row's reduction (up to d = 4096), so a workgroup keeps
// two rows of loads in flight.  (One wave per row with 64 columns per lane held 256 registers
// of column sums and row values: one wave per SIMD, 2.5 TB/s in the step.)
constexpr int LNT_ROWS = 8;

template <typename T, int NCH>
__global__ void __launch_bounds__(256) ln_bwd_team_kernel(const T* __restrict__ dy, const float* __restrict__ x,
                                                          const float* __restrict__ mean,
                                                          const float* __restrict__ rstd, const T* __restrict__ gamma,
                                                          float* __restrict__ dres, T* __restrict__ dres_lp,
                                                          int accumulate, float* __restrict__ part, int64_t rows,
                                                          int d) {
  constexpr bool PF = NCH <= 4;
  __shared__ float red[2][4][2];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * LNT_ROWS;
  const int nrow = static_cast<int>(min(static_cast<int64_t>(LNT_ROWS), rows - r0));
  const float inv_d = 1.f / static_cast<float>(d);
  bool on[NCH];
  float gam[NCH * 4], ca[NCH * 4], cb[NCH * 4];
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const int c = 4 * tid + 1024 * j;
    on[j] = c < d;
    Vec4<T> vg;
    if (on[j]) vg.load(gamma + c);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      gam[4 * j + i] = on[j] ? vg.get(i) : 0.f;
      ca[4 * j + i] = 0.f;
      cb[4 * j + i] = 0.f;
    }
  }
  float gv[NCH * 4], xv[NCH * 4];
  auto load_row = [&](int64_t row, float* g, float* xx) {
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      if (on[j]) {
        const int c = 4 * tid + 1024 * j;
        Vec4<T> vy;
        vy.load(dy + row * d + c);
        const float4 v = *reinterpret_cast<const float4*>(x + row * d + c);
        const float xs[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          g[4 * j + i] = vy.get(i);
          xx[4 * j + i] = xs[i];
        }
      }
    }
  };
  load_row(r0, gv, xv);
  for (int k = 0; k < nrow; ++k) {
    const int64_t row = r0 + k;
    const float mu = mean[row], r = rstd[row];
    float* h = xv;  // xhat replaces x in place
    float sa = 0.f, sb = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      if (on[j]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = 4 * j + i;
          h[e] = (xv[e] - mu) * r;
          const float gp = gv[e] * gam[e];
          sa += gp;
          sb += gp * h[e];
          ca[e] += gv[e] * h[e];
          cb[e] += gv[e];
        }
      }
    }
    // the next row's loads go out now when the registers allow (PF)
    float ng[PF ? NCH * 4 : 1], nx[PF ? NCH * 4 : 1];
    if constexpr (PF) {
      if (k + 1 < nrow) load_row(row + 1, ng, nx);
    }
    float prev[NCH * 4];
    if (accumulate) {
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        if (on[j]) {
          const float4 v = *reinterpret_cast<const float4*>(dres + row * d + 4 * tid + 1024 * j);
          prev[4 * j] = v.x;
          prev[4 * j + 1] = v.y;
          prev[4 * j + 2] = v.z;
          prev[4 * j + 3] = v.w;
        }
      }
    }
    sa = wave_sum(sa);
    sb = wave_sum(sb);
    const int buf = k & 1;
    if (lane == 0) {
      red[buf][w][0] = sa;
      red[buf][w][1] = sb;
    }
    __syncthreads();
    const float a = (((red[buf][0][0] + red[buf][1][0]) + red[buf][2][0]) + red[buf][3][0]) * inv_d;
    const float b = (((red[buf][0][1] + red[buf][1][1]) + red[buf][2][1]) + red[buf][3][1]) * inv_d;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      if (on[j]) {
        const int c = 4 * tid + 1024 * j;
        float o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = 4 * j + i;
          const float dx = r * (gv[e] * gam[e] - a - h[e] * b);
          o[i] = accumulate ? prev[e] + dx : dx;
        }
        *reinterpret_cast<float4*>(dres + row * d + c) = make_float4(o[0], o[1], o[2], o[3]);
        if (dres_lp) Vec4<T>::store(dres_lp + row * d + c, o);
      }
    }
    if constexpr (PF) {
#pragma unroll
      for (int e = 0; e < NCH * 4; ++e) {
        gv[e] = ng[e];
        xv[e] = nx[e];
      }
    } else {
      if (k + 1 < nrow) load_row(row + 1, gv, xv);
    }
  }
  float* p = part + static_cast<int64_t>(blockIdx.x) * 2 * d;
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    if (on[j]) {
      const int c = 4 * tid + 1024 * j;
      *reinterpret_cast<float4*>(p + c) = make_float4(ca[4 * j], ca[4 * j + 1], ca[4 * j + 2], ca[4 * j + 3]);
      *reinterpret_cast<float4*>(p + d + c) = make_float4(cb[4 * j], cb[4 * j + 1], cb[4 * j + 2], cb[4 * j + 3]);
    }
  }
}

// ------------------------------------------------------------- column sums
// Rows per partial sum: 16, so that a [4096][4096] input gives 1024
// workgroups (four per CU) whose loads are all issued before the first add
// (64 rows per block left one workgroup per CU and 2 TB/s).
constexpr int CS_ROWS = 16;

// Column sums over CS_ROWS-row blocks, four consecutive columns per thread
// (vector loads); cols and ld multiples of 4.  Each column is summed over its
// rows in order, as in colsum_partial_kernel.
template <typename T>
__global__ void __launch_bounds__(256) colsum_partial4_kernel(const T* __restrict__ x, int64_t rows, int cols,
                                                              int64_t ld, float* __restrict__ part) {
  const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (c >= cols) return;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * CS_ROWS;
  const int64_t r1 = min(rows, r0 + CS_ROWS);
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  if (r1 - r0 == CS_ROWS) {
    Vec4<T> v[CS_ROWS];
#pragma unroll
    for (int i = 0; i < CS_ROWS; ++i) v[i].load(x + (r0 + i) * ld + c);
#pragma unroll
    for (int i = 0; i < CS_ROWS; ++i) {
      s0 += v[i].get(0);
      s1 += v[i].get(1);
      s2 += v[i].get(2);
      s3 += v[i].get(3);
    }
  } else {
    for (int64_t r = r0; r < r1; ++r) {
      Vec4<T> v;
      v.load(x + r * ld + c);
      s0 += v.get(0);
      s1 += v.get(1);
      s2 += v.get(2);
      s3 += v.get(3);
    }
  }
  *reinterpret_cast<float4*>(part + static_cast<int64_t>(blockIdx.y) * cols + c) = make_float4(s0, s1, s2, s3);
}

template <typename T>
__global__ void __launch_bounds__(256) colsum_partial_kernel(const T* __restrict__ x, int64_t rows, int cols,
                                                             int64_t ld, float* __restrict__ part) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * CS_ROWS;
  const int64_t r1 = min(rows, r0 + CS_ROWS);
  float s = 0.f;
  for (int64_t r = r0; r < r1; ++r) s += to_f<T>(x[r * ld + c]);
  part[static_cast<int64_t>(blockIdx.y) * cols + c] = s;
}

// out[c] (+)= sum over p of part[p * stride + c].  A workgroup owns 16
// columns; its 16 slices each add parts slice, slice + 16, ... in order, and
// the slice sums are added in slice order, so the result is independent of
// scheduling.
constexpr int SP_COLS = 16, SP_SLICES = 16;

// Column c of the partials goes to out[c] below split and to out2[c - split]
// from there on (two targets in one launch: a LayerNorm's gamma and beta).
template <typename TO>
__global__ void __launch_bounds__(256) sum_parts_kernel(const float* __restrict__ part, int64_t nparts, int cols,
                                                        int64_t stride, TO* __restrict__ out, TO* __restrict__ out2,
                                                        int split, int accumulate) {
  __shared__ float sh[SP_SLICES][SP_COLS];
  const int cl = threadIdx.x % SP_COLS, sl = threadIdx.x / SP_COLS;
  const int c = blockIdx.x * SP_COLS + cl;
  float s = 0.f;
  if (c < cols) {
    // eight parts requested at a time, added in the same order as one by one
    int64_t p = sl;
    for (; p + 7 * SP_SLICES < nparts; p += 8 * SP_SLICES) {
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = part[(p + i * SP_SLICES) * stride + c];
#pragma unroll
      for (int i = 0; i < 8; ++i) s += v[i];
    }
    for (; p < nparts; p += SP_SLICES) s += part[p * stride + c];
  }
  sh[sl][cl] = s;
  __syncthreads();
  if (sl == 0 && c < cols) {
    float t = sh[0][cl];
#pragma unroll
    for (int i = 1; i < SP_SLICES; ++i) t += sh[i][cl];
    TO* dst = c < split ? out + c : out2 + (c - split);
    if (accumulate) t += to_f<TO>(*dst);
    *dst = from_f<TO>(t);
  }
}

// --------------------------------------------------------------- embedding
// A token id outside [0, V) gives a NaN row instead of an out-of-range read.
template <typename T>
__global__ void __launch_bounds__(256) embed_fwd_kernel(const int32_t* __restrict__ tok, const T* __restrict__ wte,
                                                        const T* __restrict__ wpe, float* __restrict__ x, int T_,
                                                        int V, int d) {
  const int64_t n = blockIdx.x;
  const int64_t v = tok[n];
  const int64_t t = n % T_;
  const bool ok = v >= 0 && v < V;
  for (int c = threadIdx.x; c < d; c += 256)
    x[n * d + c] = ok ? to_f<T>(wte[v * d + c]) + to_f<T>(wpe[t * d + c]) : __builtin_nanf("");
}

template <typename TO>
__global__ void __launch_bounds__(256) embed_bwd_wte_kernel(const float* __restrict__ dx,
                                                            const int32_t* __restrict__ perm,
                                                            const int32_t* __restrict__ seg,
                                                            const int32_t* __restrict__ uniq, TO* __restrict__ dwte,
                                                            int V, int d, int accumulate) {
  const int u = blockIdx.x;
  const int p0 = seg[u], p1 = seg[u + 1];
  const int64_t v = uniq[u];
  if (v < 0 || v >= V) return;
  for (int c = threadIdx.x; c < d; c += 256) {
    float s = 0.f;
    for (int p = p0; p < p1; ++p) s += dx[static_cast<int64_t>(perm[p]) * d + c];
    if (accumulate) s += to_f<TO>(dwte[v * d + c]);
    dwte[v * d + c] = from_f<TO>(s);
  }
}

template <typename TO>
__global__ void __launch_bounds__(256) embed_bwd_wpe_kernel(const float* __restrict__ dx, TO* __restrict__ dwpe,
                                                            int T_, int B, int d, int accumulate) {
  const int64_t t = blockIdx.x;
  for (int c = threadIdx.x; c < d; c += 256) {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += dx[(static_cast<int64_t>(b) * T_ + t) * d + c];
    if (accumulate) s += to_f<TO>(dwpe[t * d + c]);
    dwpe[t * d + c] = from_f<TO>(s);
  }
}

// ------------------------------------------------------------ cross-entropy
// Merge two (max, sum of exp(x - max)) pairs; an empty pair is (-inf, 0).
__device__ __forceinline__ void merge_ms(float& m, float& s, float m2, float s2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) {
    m = m2;
    s = s2;
    return;
  }
  const float mm = fmaxf(m, m2);
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

template <typename T>
__global__ void __launch_bounds__(256) xent_kernel(const float* __restrict__ z, int64_t ldz,
                                                   const int32_t* __restrict__ tgt, T* __restrict__ dz, int64_t lddz,
                                                   float* __restrict__ loss_rows, int V, float scale) {
  __shared__ float sm[8], ss[8];
  const int64_t row = blockIdx.x;
  const float* zr = z + row * ldz;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  float m = -INFINITY, s = 0.f;
  for (int v = tid; v < V; v += 256) {
    const float x = zr[v];
    if (x > m) {
      s = s * __expf(m - x) + 1.f;
      m = x;
    } else {
      s += __expf(x - m);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, 64), s2 = __shfl_xor(s, o, 64);
    merge_ms(m, s, m2, s2);
  }
  if (lane == 0) {
    sm[w] = m;
    ss[w] = s;
  }
  __syncthreads();
  m = sm[0];
  s = ss[0];
  for (int i = 1; i < 4; ++i) merge_ms(m, s, sm[i], ss[i]);
  const float lse = m + logf(s);
  const int y = tgt[row];
  T* dr = dz + row * lddz;
  for (int v = tid; v < lddz; v += 256) {
    float g = 0.f;
    if (v < V) g = (__expf(zr[v] - lse) - (v == y ? 1.f : 0.f)) * scale;
    dr[v] = from_f<T>(g);
  }
  // a target outside [0, V) gives a NaN loss instead of an out-of-range read
  if (tid == 0) loss_rows[row] = (y >= 0 && y < V) ? lse - zr[y] : __builtin_nanf("");
}

// Cross-entropy with the row in registers: 1024 threads per row, thread t
// owns the 16-byte chunks t + 1024 i (i < NV) of the fp32 logits, so the row
// is read from HBM once (the two-pass kernel above reads it twice, with
// 4-byte loads).  Max, then the sum of 2^((z - max) log2 e) kept in the same
// registers, then dz = (p - onehot) scale from them: two block reductions,
// each wave's shuffles then the 16 waves in a fixed order.  Columns V..lddz-1
// of dz are zeroed; the loss row is lse - z[y] (NaN for y outside [0, V)).
// Needs ldz and lddz multiples of 4 and 16-byte aligned rows (dispatch).
template <typename T, int NV>
__global__ void __launch_bounds__(1024) xent_reg_kernel(const float* __restrict__ z, int64_t ldz,
                                                        const int32_t* __restrict__ tgt, T* __restrict__ dz,
                                                        int64_t lddz, float* __restrict__ loss_rows, int V,
                                                        float scale) {
  __shared__ float red[2][16];
  const int64_t row = blockIdx.x;
  const float* zr = z + row * ldz;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  constexpr float L2E = 1.4426950408889634f;
  float x[NV][4];
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = 4 * (tid + 1024 * i);
    if (c + 4 <= V) {
      const float4 v = *reinterpret_cast<const float4*>(zr + c);
      x[i][0] = v.x;
      x[i][1] = v.y;
      x[i][2] = v.z;
      x[i][3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) x[i][e] = c + e < V ? zr[c + e] : -INFINITY;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) m = fmaxf(m, x[i][e]);
  }
  m = wave_max(m);
  if (lane == 0) red[0][w] = m;
  __syncthreads();
  m = red[0][0];
#pragma unroll
  for (int i = 1; i < 16; ++i) m = fmaxf(m, red[0][i]);
  const float mb = m * L2E;
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[i][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[i][e], L2E, -mb));  // 0 for the -inf fill
      sum += x[i][e];
    }
  sum = wave_sum(sum);
  if (lane == 0) red[1][w] = sum;
  __syncthreads();
  sum = red[1][0];
#pragma unroll
  for (int i = 1; i < 16; ++i) sum += red[1][i];
  const float inv = 1.f / sum;
  const int y = tgt[row];
  T* dr = dz + row * lddz;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = 4 * (tid + 1024 * i);
    if (c >= lddz) break;
    float g[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) g[e] = c + e < V ? (x[i][e] * inv - (c + e == y ? 1.f : 0.f)) * scale : 0.f;
    Vec4<T>::store(dr + c, g);  // lddz is a multiple of 4: the chunk is inside the row
  }
  // a target outside [0, V) gives a NaN loss instead of an out-of-range read
  if (tid == 0) loss_rows[row] = (y >= 0 && y < V) ? m + logf(sum) - zr[y] : __builtin_nanf("");
}

// ---------------------------------------------------------------- helpers
__global__ void __launch_bounds__(256) sum_fixed_kernel(const float* __restrict__ x, int64_t n,
                                                        float* __restrict__ out) {
  __shared__ double sh[256];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) s += static_cast<double>(x[i]);
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = static_cast<float>(sh[0]);
}

template <typename T>
__global__ void __launch_bounds__(256) convert_kernel(const float* __restrict__ x, T* __restrict__ y, int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256)
    y[i] = from_f<T>(x[i]);
}

__global__ void __launch_bounds__(256) fill_zero_kernel(uint4* __restrict__ p, int64_t n16, uint8_t* tail,
                                                        int ntail) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n16;
       i += static_cast<int64_t>(gridDim.x) * 256)
    p[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < ntail) tail[threadIdx.x] = 0;
}

__global__ void __launch_bounds__(256) fill_word_kernel(uint4* __restrict__ p, int64_t n16, uint32_t w) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n16;
       i += static_cast<int64_t>(gridDim.x) * 256)
    p[i] = make_uint4(w, w, w, w);
}

// *out = max(*out, 1 + index of the last 16-byte unit of p[0..n16) that
// holds a word other than w); *out is left alone if every unit still holds w.
__global__ void __launch_bounds__(256) high_water_kernel(const uint4* __restrict__ p, int64_t n16, uint32_t w,
                                                         unsigned long long* __restrict__ out) {
  unsigned long long hi = 0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n16;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const uint4 v = p[i];
    if (v.x != w || v.y != w || v.z != w || v.w != w) hi = static_cast<unsigned long long>(i) + 1;
  }
  __shared__ unsigned long long red[256];
  red[threadIdx.x] = hi;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if (static_cast<int>(threadIdx.x) < k) red[threadIdx.x] = red[threadIdx.x + k] > red[threadIdx.x] ? red[threadIdx.x + k] : red[threadIdx.x];
    __syncthreads();
  }
  if (threadIdx.x == 0 && red[0] > 0) atomicMax(out, red[0]);
}

// Streaming copy, 16 bytes per thread and iteration.
__global__ void __launch_bounds__(256) copy16_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                     int64_t n16) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n16;
       i += static_cast<int64_t>(gridDim.x) * 256)
    dst[i] = src[i];
}

// Word copy whose source may be mapped pinned host memory (read over the host
// link by the kernel itself).
__global__ void __launch_bounds__(256) copy_words_kernel(const uint32_t* __restrict__ src,
                                                         uint32_t* __restrict__ dst, int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256)
    dst[i] = src[i];
}

// System-scope acquire on every compute unit and L2: lines cached before a
// DMA engine rewrote device memory are dropped, so later kernels read the new
// contents.  256 workgroups reach every XCD's L2 (workgroups are spread over
// the XCDs round-robin).
__global__ void __launch_bounds__(64) dma_acquire_kernel() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, ""); }

inline unsigned grid_for(int64_t n) {
  int64_t g = (n + 255) / 256;
  return static_cast<unsigned>(g < 1 ? 1 : (g > 65536 ? 65536 : g));
}

template <typename T>
hipError_t ln_fwd_t(const float* x, const void* gamma, const void* beta, void* y, float* mean, float* rstd,
                    int64_t rows, int d, hipStream_t s) {
  const int ne = (d + 255) / 256;
  dim3 grid(static_cast<unsigned>(rows)), block(256);
  auto g = static_cast<const T*>(gamma);
  auto b = static_cast<const T*>(beta);
  auto yy = static_cast<T*>(y);
#define ATOM_LNF(E) hipLaunchKernelGGL((ln_fwd_kernel<T, E>), grid, block, 0, s, x, g, b, yy, mean, rstd, d)
  if (ne <= 4) ATOM_LNF(1);
  else if (ne <= 8) ATOM_LNF(2);
  else if (ne <= 16) ATOM_LNF(4);
  else ATOM_LNF(8);
#undef ATOM_LNF
  return hipGetLastError();
}

bool lnw_usable(int d) { return d % 256 == 0 && d / 256 <= LNW_MAXCH; }
#ifndef ATOM_LN_TEAM
#define ATOM_LN_TEAM 1
#endif
bool lnt_usable(int d) { return ATOM_LN_TEAM && d >= 1024 && d % 4 == 0 && d <= 8192; }

template <typename T>
hipError_t ln_bwd_t(const void* dy, const float* x, const float* mean, const float* rstd, const void* gamma,
                    float* dres, void* dres_lp, bool acc, float* part, int64_t rows, int d, hipStream_t s) {
  const int ne = (d + 255) / 256;
  auto a0 = static_cast<const T*>(dy);
  auto g = static_cast<const T*>(gamma);
  auto lp = static_cast<T*>(dres_lp);
  const int ac = acc ? 1 : 0;
  if (lnt_usable(d)) {
    dim3 grid(static_cast<unsigned>((rows + LNT_ROWS - 1) / LNT_ROWS)), block(256);
#define ATOM_LNT(CH)                                                                                             \
  hipLaunchKernelGGL((ln_bwd_team_kernel<T, CH>), grid, block, 0, s, a0, x, mean, rstd, g, dres, lp, ac, part, rows, \
                     d)
    if (ne <= 4) ATOM_LNT(1);
    else if (ne <= 8) ATOM_LNT(2);
    else if (ne <= 12) ATOM_LNT(3);
    else if (ne <= 16) ATOM_LNT(4);
    else if (ne <= 20) ATOM_LNT(5);
    else ATOM_LNT(8);
#undef ATOM_LNT
    return hipGetLastError();
  }
  if (lnw_usable(d)) {
    const int rpw = lnw_rows_per_wave(rows);
    dim3 wgrid(static_cast<unsigned>((rows + 4 * rpw - 1) / (4 * rpw))), wblock(256);
    const size_t lds = 4 * static_cast<size_t>(d) * sizeof(float);
#define ATOM_LNW(CH)                                                                                            \
  hipLaunchKernelGGL((ln_bwd_wave_kernel<T, CH>), wgrid, wblock, lds, s, a0, x, mean, rstd, g, dres, lp, ac, part, \
                     rows, d, rpw)
    if (ne <= 1) ATOM_LNW(1);
    else if (ne <= 4) ATOM_LNW(4);
    else if (ne <= 8) ATOM_LNW(8);
    else if (ne <= 16) ATOM_LNW(16);
    else ATOM_LNW(LNW_MAXCH);
#undef ATOM_LNW
    return hipGetLastError();
  }
  dim3 grid(static_cast<unsigned>((rows + LNB_ROWS - 1) / LNB_ROWS)), block(256);
#define ATOM_LNB(E) \
  hipLaunchKernelGGL((ln_bwd_kernel<T, E>), grid, block, 2 * d * sizeof(float), s, a0, x, mean, rstd, g, dres, lp, \
                     ac, part, rows, d)
  if (ne <= 1) ATOM_LNB(1);
  else if (ne <= 2) ATOM_LNB(2);
  else if (ne <= 4) ATOM_LNB(4);
  else if (ne <= 8) ATOM_LNB(8);
  else if (ne <= 16) ATOM_LNB(16);
  else ATOM_LNB(32);
#undef ATOM_LNB
  return hipGetLastError();
}

}  // namespace

hipError_t layernorm_fwd(int dtype, const float* x, const void* gamma, const void* beta, void* y, float* mean,
                         float* rstd, int64_t rows, int d, hipStream_t s) {
  if (d <= 0 || d % 64 || d > 8192 || rows < 0) return hipErrorInvalidValue;
  if (rows == 0) return hipSuccess;
  return dtype == DT_BF16 ? ln_fwd_t<bf16_t>(x, gamma, beta, y, mean, rstd, rows, d, s)
                          : ln_fwd_t<float>(x, gamma, beta, y, mean, rstd, rows, d, s);
}

int64_t layernorm_bwd_blocks(int64_t rows, int d) {
  if (lnt_usable(d)) return (rows + LNT_ROWS - 1) / LNT_ROWS;
  if (lnw_usable(d)) {
    const int rpw = lnw_rows_per_wave(rows);
    return (rows + 4 * rpw - 1) / (4 * rpw);
  }
  return (rows + LNB_ROWS - 1) / LNB_ROWS;
}

hipError_t layernorm_bwd(int dtype, const void* dy, const float* x, const float* mean, const float* rstd,
                         const void* gamma, float* dres, void* dres_lp, bool accumulate, float* part, int64_t rows,
                         int d, hipStream_t s) {
  if (d <= 0 || d % 64 || d > 8192 || rows < 0) return hipErrorInvalidValue;
  if (rows == 0) return hipSuccess;
  return dtype == DT_BF16 ? ln_bwd_t<bf16_t>(dy, x, mean, rstd, gamma, dres, dres_lp, accumulate, part, rows, d, s)
                          : ln_bwd_t<float>(dy, x, mean, rstd, gamma, dres, dres_lp, accumulate, part, rows, d, s);
}

int64_t colsum_blocks(int64_t rows) { return (rows + CS_ROWS - 1) / CS_ROWS; }

hipError_t colsum_partial(int in_dtype, const void* x, int64_t rows, int cols, int64_t ld, float* part,
                          hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipErrorInvalidValue;
  const bool vec = cols % 4 == 0 && ld % 4 == 0 &&
                   reinterpret_cast<uintptr_t>(x) % (in_dtype == DT_BF16 ? 8 : 16) == 0;
  if (vec) {
    dim3 g4(static_cast<unsigned>((cols / 4 + 255) / 256), static_cast<unsigned>(colsum_blocks(rows))), b4(256);
    if (in_dtype == DT_BF16)
      hipLaunchKernelGGL(colsum_partial4_kernel<bf16_t>, g4, b4, 0, s, static_cast<const bf16_t*>(x), rows, cols,
                         ld, part);
    else
      hipLaunchKernelGGL(colsum_partial4_kernel<float>, g4, b4, 0, s, static_cast<const float*>(x), rows, cols, ld,
                         part);
    return hipGetLastError();
  }
  dim3 grid(static_cast<unsigned>((cols + 255) / 256), static_cast<unsigned>(colsum_blocks(rows))), block(256);
  if (in_dtype == DT_BF16)
    hipLaunchKernelGGL(colsum_partial_kernel<bf16_t>, grid, block, 0, s, static_cast<const bf16_t*>(x), rows, cols,
                       ld, part);
  else
    hipLaunchKernelGGL(colsum_partial_kernel<float>, grid, block, 0, s, static_cast<const float*>(x), rows, cols,
                       ld, part);
  return hipGetLastError();
}

hipError_t sum_parts2(const float* part, int64_t nparts, int cols, int64_t part_stride, int out_dtype, void* out,
                      void* out2, int split, bool accumulate, hipStream_t s) {
  if (cols <= 0 || split < 0 || split > cols) return hipErrorInvalidValue;
  dim3 grid(static_cast<unsigned>((cols + SP_COLS - 1) / SP_COLS)), block(256);
  if (out_dtype == DT_BF16)
    hipLaunchKernelGGL(sum_parts_kernel<bf16_t>, grid, block, 0, s, part, nparts, cols, part_stride,
                       static_cast<bf16_t*>(out), static_cast<bf16_t*>(out2), split, accumulate ? 1 : 0);
  else
    hipLaunchKernelGGL(sum_parts_kernel<float>, grid, block, 0, s, part, nparts, cols, part_stride,
                       static_cast<float*>(out), static_cast<float*>(out2), split, accumulate ? 1 : 0);
  return hipGetLastError();
}

hipError_t sum_parts(const float* part, int64_t nparts, int cols, int64_t part_stride, int out_dtype, void* out,
                     bool accumulate, hipStream_t s) {
  return sum_parts2(part, nparts, cols, part_stride, out_dtype, out, out, cols, accumulate, s);
}

hipError_t embed_fwd(int dtype, const int32_t* tok, const void* wte, const void* wpe, float* x, int64_t n_tok,
                     int T, int V, int d, hipStream_t s) {
  if (n_tok <= 0) return hipSuccess;
  if (T <= 0 || V <= 0 || d <= 0) return hipErrorInvalidValue;
  dim3 grid(static_cast<unsigned>(n_tok)), block(256);
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(embed_fwd_kernel<bf16_t>, grid, block, 0, s, tok, static_cast<const bf16_t*>(wte),
                       static_cast<const bf16_t*>(wpe), x, T, V, d);
  else
    hipLaunchKernelGGL(embed_fwd_kernel<float>, grid, block, 0, s, tok, static_cast<const float*>(wte),
                       static_cast<const float*>(wpe), x, T, V, d);
  return hipGetLastError();
}

hipError_t embed_bwd(int out_dtype, const float* dx, const int32_t* perm, const int32_t* seg, const int32_t* uniq,
                     int n_uniq, void* dwte, void* dwpe, int V, int T, int B, int d, bool accumulate,
                     hipStream_t s) {
  const size_t esz = out_dtype == DT_BF16 ? 2 : 4;
  hipError_t e;
  if (!accumulate) {
    e = fill_zero(dwte, static_cast<int64_t>(V) * d * esz, s);
    if (e != hipSuccess) return e;
  }
  const int ac = accumulate ? 1 : 0;
  if (n_uniq > 0) {
    if (out_dtype == DT_BF16)
      hipLaunchKernelGGL(embed_bwd_wte_kernel<bf16_t>, dim3(n_uniq), dim3(256), 0, s, dx, perm, seg, uniq,
                           static_cast<bf16_t*>(dwte), V, d, ac);
    else
      hipLaunchKernelGGL(embed_bwd_wte_kernel<float>, dim3(n_uniq), dim3(256), 0, s, dx, perm, seg, uniq,
                         static_cast<float*>(dwte), V, d, ac);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (out_dtype == DT_BF16)
    hipLaunchKernelGGL(embed_bwd_wpe_kernel<bf16_t>, dim3(T), dim3(256), 0, s, dx, static_cast<bf16_t*>(dwpe), T, B,
                       d, ac);
  else
    hipLaunchKernelGGL(embed_bwd_wpe_kernel<float>, dim3(T), dim3(256), 0, s, dx, static_cast<float*>(dwpe), T, B, d,
                       ac);
  return hipGetLastError();
}

hipError_t xent_fwd_bwd(int dtype, const float* logits, int64_t ldz, const int32_t* tgt, void* dz, int64_t lddz,
                        float* loss_rows, int64_t rows, int V, float scale, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (V <= 0 || lddz < V || ldz < V) return hipErrorInvalidValue;
  const int esz = dtype == DT_BF16 ? 2 : 4;
  const int nv = static_cast<int>((lddz + 4095) / 4096);  // 16-byte chunks per thread
  if (ldz % 4 == 0 && lddz % 4 == 0 && reinterpret_cast<uintptr_t>(logits) % 16 == 0 &&
      reinterpret_cast<uintptr_t>(dz) % (4 * esz) == 0 && nv <= 16) {
    dim3 g1(static_cast<unsigned>(rows)), b1(1024);
#define ATOM_XR(NV)                                                                                                 \
  do {                                                                                                              \
    if (dtype == DT_BF16)                                                                                           \
      hipLaunchKernelGGL((xent_reg_kernel<bf16_t, NV>), g1, b1, 0, s, logits, ldz, tgt, static_cast<bf16_t*>(dz), \
                         lddz, loss_rows, V, scale);                                                                \
    else                                                                                                            \
      hipLaunchKernelGGL((xent_reg_kernel<float, NV>), g1, b1, 0, s, logits, ldz, tgt, static_cast<float*>(dz),   \
                         lddz, loss_rows, V, scale);                                                                \
  } while (0)
    if (nv <= 1) ATOM_XR(1);
    else if (nv <= 2) ATOM_XR(2);
    else if (nv <= 4) ATOM_XR(4);
    else if (nv <= 8) ATOM_XR(8);
    else if (nv <= 13) ATOM_XR(13);
    else ATOM_XR(16);
#undef ATOM_XR
    return hipGetLastError();
  }
  dim3 grid(static_cast<unsigned>(rows)), block(256);
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(xent_kernel<bf16_t>, grid, block, 0, s, logits, ldz, tgt, static_cast<bf16_t*>(dz), lddz,
                       loss_rows, V, scale);
  else
    hipLaunchKernelGGL(xent_kernel<float>, grid, block, 0, s, logits, ldz, tgt, static_cast<float*>(dz), lddz,
                       loss_rows, V, scale);
  return hipGetLastError();
}

hipError_t sum_fixed(const float* x, int64_t n, float* out, hipStream_t s) {
  hipLaunchKernelGGL(sum_fixed_kernel, dim3(1), dim3(256), 0, s, x, n, out);
  return hipGetLastError();
}

hipError_t convert_f32(int dtype, const float* x, void* y, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(convert_kernel<bf16_t>, dim3(grid_for(n)), dim3(256), 0, s, x, static_cast<bf16_t*>(y), n);
  else
    hipLaunchKernelGGL(convert_kernel<float>, dim3(grid_for(n)), dim3(256), 0, s, x, static_cast<float*>(y), n);
  return hipGetLastError();
}

hipError_t dma_acquire(hipStream_t s) {
  hipLaunchKernelGGL(dma_acquire_kernel, dim3(256), dim3(64), 0, s);
  return hipGetLastError();
}

hipError_t copy_words(const uint32_t* src, uint32_t* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_words_kernel, dim3(grid_for(n)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t copy_bytes(const void* src, void* dst, int64_t bytes, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | static_cast<uintptr_t>(bytes)) & 15)
    return hipErrorInvalidValue;
  const int64_t n16 = bytes / 16;
  const int64_t want = (n16 + 255) / 256;
  const unsigned grid = static_cast<unsigned>(want < 8192 ? (want < 1 ? 1 : want) : 8192);
  hipLaunchKernelGGL(copy16_kernel, dim3(grid), dim3(256), 0, s, static_cast<const uint4*>(src),
                     static_cast<uint4*>(dst), n16);
  return hipGetLastError();
}

hipError_t fill_word(void* p, int64_t bytes, uint32_t word, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(p) | static_cast<uintptr_t>(bytes)) & 15) return hipErrorInvalidValue;
  const int64_t n16 = bytes / 16;
  hipLaunchKernelGGL(fill_word_kernel, dim3(grid_for(n16)), dim3(256), 0, s, static_cast<uint4*>(p), n16, word);
  return hipGetLastError();
}

hipError_t high_water(const void* p, int64_t bytes, uint32_t word, unsigned long long* out, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(p) | static_cast<uintptr_t>(bytes)) & 15) return hipErrorInvalidValue;
  const int64_t n16 = bytes / 16;
  const int64_t want = (n16 + 255) / 256;
  const unsigned grid = static_cast<unsigned>(want < 4096 ? (want < 1 ? 1 : want) : 4096);
  hipLaunchKernelGGL(high_water_kernel, dim3(grid), dim3(256), 0, s, static_cast<const uint4*>(p), n16, word, out);
  return hipGetLastError();
}

hipError_t fill_zero(void* p, int64_t bytes, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  if (reinterpret_cast<uintptr_t>(p) & 15) return hipErrorInvalidValue;
  const int64_t n16 = bytes / 16;
  const int ntail = static_cast<int>(bytes - n16 * 16);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(n16)), dim3(256), 0, s, static_cast<uint4*>(p), n16,
                     static_cast<uint8_t*>(p) + n16 * 16, ntail);
  return hipGetLastError();
}

}  // namespace atom
