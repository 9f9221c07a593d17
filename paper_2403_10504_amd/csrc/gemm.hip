// Dense GEMM on CDNA4 matrix cores with fused epilogues.
//
//   C[m][n] (op)= sum_k A(m,k) * B(k,n),   fp32 accumulation.
//
// Operand layouts (both row-major in memory):
//   A_KC: A(m,k) = A[m*lda + k]   (k contiguous)   else A(m,k) = A[k*lda + m]
//   B_KC: B(k,n) = B[n*ldb + k]   (k contiguous)   else B(k,n) = B[k*ldb + n]
// The three products of a linear layer y = x W^T + b with W stored [out][in]:
//   forward   y  = x  W^T : A = x  (KC),          B = W  (KC)
//   data grad dx = dy W   : A = dy (KC),          B = W  (not KC)
//   weight grad dW = dy^T x: A = dy (not KC),      B = x  (not KC)
//
// Tiling: a BM x BN output tile per workgroup of WM x WN waves (256x256 with
// 16 waves of 64x64 for big problems: four waves per SIMD hide the global
// and LDS latency better than eight waves of 64x128, measured +16 %;
// 128x128 with 4 waves otherwise), 128-byte k tile (64 bf16 or 32 fp32)
// double-buffered in LDS.  Every operand is staged in LDS with k contiguous
// (rows padded to 144 bytes to spread ds_read_b128 over the banks); operands
// that are not k-contiguous in memory are transposed while being written to
// LDS.  Each lane reads 16x16x32 MFMA fragments (see common.h).  Larger
// per-wave tiles raise the MFMA work per byte read from LDS.  Workgroup ids
// are remapped so that neighbouring output tiles, which share A rows or B
// columns, run on the same XCD (each XCD has its own L2).  Problems with few
// output tiles and a long k (weight gradients of narrow layers) split k over
// workgroups; the fp32 partials are summed in split order by a second kernel,
// so the result does not depend on scheduling.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace atom {
namespace {

constexpr int ROW_BYTES = 128, PITCH_BYTES = 144;

// Workgroup tile BM x BN computed by WM x WN waves, each owning a
// (BM/WM) x (BN/WN) block of 16x16 MFMA tiles.
#ifndef ATOM_GEMM_CFG
#define ATOM_GEMM_CFG 256, 256, 4, 4
#endif
template <int BM_, int BN_, int WM_, int WN_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int NT = 64 * WM_ * WN_;
  static constexpr int TM = BM_ / (16 * WM_), TN = BN_ / (16 * WN_);
};
using Big = Cfg<ATOM_GEMM_CFG>;   // large problems
using Small = Cfg<128, 128, 2, 2>; // few output tiles

template <typename T>
struct Tile {
  static constexpr int BK = ROW_BYTES / sizeof(T);    // k per tile
  static constexpr int PITCH = PITCH_BYTES / sizeof(T);
  static constexpr int KV = 16 / sizeof(T);           // elements per 16 bytes
  static constexpr int PAIR = 4 / sizeof(T);          // elements per dword
  static constexpr int NSLICE = BK / 32;
};

// Stages an R-row x BK tile of one operand (rows = m for A, n for B) with NT
// threads.  Registers hold the next tile while the current one is consumed.
template <typename T, bool KC, int R, int NT>
struct Loader {
  using TL = Tile<T>;
  static constexpr int DW = R * ROW_BYTES / 4 / NT;   // dwords per thread
  static constexpr int UPK = R / TL::PAIR;            // !KC: dword units per k row
  static constexpr int UPT = 8 * UPK / NT;            // !KC: units per thread
  static constexpr int NOFF = KC ? DW / 4 : UPT;
  uint32_t r[DW];
  uint32_t off[NOFF];  // byte offsets of this thread's loads inside a full tile

  // Offsets for load_fast (leading dimension ld, elements).
  __device__ void init(int64_t ld, int tid) {
    if constexpr (KC) {
#pragma unroll
      for (int i = 0; i < NOFF; ++i) {
        const int c = tid + NT * i;
        off[i] = static_cast<uint32_t>(((c >> 3) * ld + (c & 7) * TL::KV) * sizeof(T));
      }
    } else {
#pragma unroll
      for (int i = 0; i < NOFF; ++i) {
        const int u = tid + NT * i;
        off[i] = static_cast<uint32_t>(((u / UPK) * TL::KV * ld + (u % UPK) * TL::PAIR) * sizeof(T));
      }
    }
  }

  // Unguarded load of a tile that lies wholly inside the operand (rows
  // r0..r0+R-1 and k0..k0+BK-1): one uniform base pointer and the 32-bit
  // per-thread offsets from init.
  __device__ void load_fast(const T* __restrict__ X, int64_t ld, int r0, int k0) {
    if constexpr (KC) {
      const char* base = reinterpret_cast<const char*>(X + static_cast<int64_t>(r0) * ld + k0);
#pragma unroll
      for (int i = 0; i < NOFF; ++i) {
        const uint4 v = *reinterpret_cast<const uint4*>(base + off[i]);
        r[4 * i + 0] = v.x;
        r[4 * i + 1] = v.y;
        r[4 * i + 2] = v.z;
        r[4 * i + 3] = v.w;
      }
    } else {
      const char* base = reinterpret_cast<const char*>(X + static_cast<int64_t>(k0) * ld + r0);
      const uint32_t step = static_cast<uint32_t>(ld * sizeof(T));
#pragma unroll
      for (int i = 0; i < NOFF; ++i)
#pragma unroll
        for (int j = 0; j < TL::KV; ++j) r[i * TL::KV + j] = *reinterpret_cast<const uint32_t*>(base + off[i] + j * step);
    }
  }

  // KC: rows are contiguous along k, R rows x 8 chunks of 16 bytes.
  // !KC: memory is [k][row]; a unit is KV consecutive k rows x PAIR rows.
  __device__ void load(const T* __restrict__ X, int64_t ld, int Rlim, int K, int r0, int k0, int tid) {
    if constexpr (KC) {
#pragma unroll
      for (int i = 0; i < DW / 4; ++i) {
        const int c = tid + NT * i;
        const int row = c >> 3, kc = c & 7;
        const int gr = r0 + row, gk = k0 + kc * TL::KV;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (gr < Rlim && gk < K) v = *reinterpret_cast<const uint4*>(X + static_cast<int64_t>(gr) * ld + gk);
        r[4 * i + 0] = v.x;
        r[4 * i + 1] = v.y;
        r[4 * i + 2] = v.z;
        r[4 * i + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < UPT; ++i) {
        const int u = tid + NT * i;
        const int kb = u / UPK, rc = u % UPK;
        const int gr = r0 + rc * TL::PAIR;
#pragma unroll
        for (int j = 0; j < TL::KV; ++j) {
          const int gk = k0 + kb * TL::KV + j;
          uint32_t v = 0;
          if (gr < Rlim && gk < K) v = *reinterpret_cast<const uint32_t*>(X + static_cast<int64_t>(gk) * ld + gr);
          r[i * TL::KV + j] = v;
        }
      }
    }
  }

  __device__ void store(T* __restrict__ S, int tid) {
    if constexpr (KC) {
#pragma unroll
      for (int i = 0; i < DW / 4; ++i) {
        const int c = tid + NT * i;
        const int row = c >> 3, kc = c & 7;
        *reinterpret_cast<uint4*>(S + row * TL::PITCH + kc * TL::KV) =
            make_uint4(r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < UPT; ++i) {
        const int u = tid + NT * i;
        const int kb = u / UPK, rc = u % UPK;
        const uint32_t* d = r + i * TL::KV;
        if constexpr (sizeof(T) == 2) {
          // d[j] packs (row 2rc, row 2rc+1) at k = 8kb + j; transpose to two
          // 16-byte rows of 8 consecutive k.
          uint4 lo, hi;
          lo.x = (d[0] & 0xffffu) | (d[1] << 16); hi.x = (d[0] >> 16) | (d[1] & 0xffff0000u);
          lo.y = (d[2] & 0xffffu) | (d[3] << 16); hi.y = (d[2] >> 16) | (d[3] & 0xffff0000u);
          lo.z = (d[4] & 0xffffu) | (d[5] << 16); hi.z = (d[4] >> 16) | (d[5] & 0xffff0000u);
          lo.w = (d[6] & 0xffffu) | (d[7] << 16); hi.w = (d[6] >> 16) | (d[7] & 0xffff0000u);
          *reinterpret_cast<uint4*>(S + (2 * rc) * TL::PITCH + kb * 8) = lo;
          *reinterpret_cast<uint4*>(S + (2 * rc + 1) * TL::PITCH + kb * 8) = hi;
        } else {
          *reinterpret_cast<uint4*>(S + rc * TL::PITCH + kb * 4) = make_uint4(d[0], d[1], d[2], d[3]);
        }
      }
    }
  }
};

template <typename T>
__device__ __forceinline__ void store4(T* p, const float* v, bool vec, int nvalid) {
  if (vec) {
    if constexpr (sizeof(T) == 2) {
      uint2 w;
      w.x = pack_bf16(v[0], v[1]);
      w.y = pack_bf16(v[2], v[3]);
      *reinterpret_cast<uint2*>(p) = w;
    } else {
      *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    }
  } else {
    for (int r = 0; r < nvalid; ++r) p[r] = from_f<T>(v[r]);
  }
}

template <typename T>
__device__ __forceinline__ void load4(const T* p, float* v, bool vec, int nvalid) {
  if (vec) {
    if constexpr (sizeof(T) == 2) {
      uint2 w = *reinterpret_cast<const uint2*>(p);
      v[0] = bf2f(w.x & 0xffff); v[1] = bf2f(w.x >> 16); v[2] = bf2f(w.y & 0xffff); v[3] = bf2f(w.y >> 16);
    } else {
      float4 w = *reinterpret_cast<const float4*>(p);
      v[0] = w.x; v[1] = w.y; v[2] = w.z; v[3] = w.w;
    }
  } else {
    for (int r = 0; r < 4; ++r) v[r] = r < nvalid ? to_f<T>(p[r]) : 0.f;
  }
}

// Epilogue of one 4-wide output fragment: v[r] = C[m][nb + r] before the op.
template <typename T, int EPI>
__device__ __forceinline__ void epilogue4(const GemmArgs& g, int m, int nb, float* v, bool ld_vec) {
  const int nvalid = min(4, g.N - nb);
  const bool vec = ld_vec && nvalid == 4;
  const int64_t off = static_cast<int64_t>(m) * g.ldc + nb;
  if constexpr (EPI == EPI_STORE) {
    store4<T>(static_cast<T*>(g.C) + off, v, vec, nvalid);
  } else if constexpr (EPI == EPI_STORE_F32) {
    store4<float>(static_cast<float*>(g.C) + off, v, vec, nvalid);
  } else if constexpr (EPI == EPI_ACC_F32) {
    float o[4];
    load4<float>(static_cast<const float*>(g.C) + off, o, vec, nvalid);
    for (int r = 0; r < 4; ++r) v[r] += o[r];
    store4<float>(static_cast<float*>(g.C) + off, v, vec, nvalid);
  } else if constexpr (EPI == EPI_BIAS) {
    float b[4];
    load4<T>(static_cast<const T*>(g.bias) + nb, b, nvalid == 4, nvalid);
    for (int r = 0; r < 4; ++r) v[r] += b[r];
    store4<T>(static_cast<T*>(g.C) + off, v, vec, nvalid);
  } else if constexpr (EPI == EPI_BIAS_GELU) {
    float b[4], gv[4];
    load4<T>(static_cast<const T*>(g.bias) + nb, b, nvalid == 4, nvalid);
    for (int r = 0; r < 4; ++r) {
      // g = GELU(u) of the stored (rounded) u, so the backward sees the same u.
      const float u = to_f<T>(from_f<T>(v[r] + b[r]));
      v[r] = u;
      gv[r] = gelu_f(u);
    }
    const int64_t aoff = static_cast<int64_t>(m) * g.ldaux + nb;
    store4<T>(static_cast<T*>(g.aux) + aoff, v, vec && (g.ldaux & 3) == 0, nvalid);
    store4<T>(static_cast<T*>(g.C) + off, gv, vec, nvalid);
  } else if constexpr (EPI == EPI_BIAS_RESID) {
    float b[4], x[4];
    load4<T>(static_cast<const T*>(g.bias) + nb, b, nvalid == 4, nvalid);
    load4<float>(g.resid + off, x, vec, nvalid);
    for (int r = 0; r < 4; ++r) v[r] = x[r] + (v[r] + b[r]);
    store4<float>(static_cast<float*>(g.C) + off, v, vec, nvalid);
  } else if constexpr (EPI == EPI_GELU_BWD) {
    float u[4];
    const int64_t aoff = static_cast<int64_t>(m) * g.ldaux + nb;
    load4<T>(static_cast<const T*>(g.aux) + aoff, u, vec && (g.ldaux & 3) == 0, nvalid);
    for (int r = 0; r < 4; ++r) v[r] *= gelu_grad_f(u[r]);
    store4<T>(static_cast<T*>(g.C) + off, v, vec, nvalid);
  }
}

// Epilogues that read an element operand (C itself, the fp32 residual or the
// saved pre-activation) and epilogues that add the bias.
template <int EPI>
constexpr bool epi_reads_elem() {
  return EPI == EPI_ACC_F32 || EPI == EPI_BIAS_RESID || EPI == EPI_GELU_BWD;
}
template <int EPI>
constexpr bool epi_has_bias() {
  return EPI == EPI_BIAS || EPI == EPI_BIAS_GELU || EPI == EPI_BIAS_RESID;
}

// One output tile per workgroup (blockIdx.x), one k range per split
// (blockIdx.y).  With splits > 1 the raw fp32 sums go to the workspace
// ws[split][M][N] and splitk_reduce applies the epilogue.
template <typename T, bool AKC, bool BKC, int EPI, class CF>
__global__ void __launch_bounds__(CF::NT) gemm_kernel(GemmArgs g) {
  using TL = Tile<T>;
  constexpr int BM = CF::BM, BN = CF::BN, NT = CF::NT, TM = CF::TM, TN = CF::TN;
  __shared__ __attribute__((aligned(16))) T As[2][BM * TL::PITCH];
  __shared__ __attribute__((aligned(16))) T Bs[2][BN * TL::PITCH];

  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wm = w / CF::WN, wn = w % CF::WN;

  // Tile order: XCD-aware remap (consecutive ids go round-robin over the 8
  // XCDs, so give each XCD a contiguous range), then groups of 8 row-tiles
  // sweeping the columns.
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int total = tiles_m * tiles_n;
  int pid = blockIdx.x;
  if ((total & 7) == 0) pid = (pid & 7) * (total >> 3) + (pid >> 3);
  constexpr int GROUP = 8;
  const int per_group = GROUP * tiles_n;
  const int first_m = (pid / per_group) * GROUP;
  const int gsize = min(tiles_m - first_m, GROUP);
  const int pid_m = first_m + (pid % per_group) % gsize;
  const int pid_n = (pid % per_group) / gsize;
  const int m0 = pid_m * BM, n0 = pid_n * BN;

  const T* __restrict__ A = static_cast<const T*>(g.A);
  const T* __restrict__ B = static_cast<const T*>(g.B);

  const int nk_all = (g.K + TL::BK - 1) / TL::BK;
  const int per_split = (nk_all + gridDim.y - 1) / gridDim.y;
  const int kt0 = blockIdx.y * per_split;
  const int kt1 = min(nk_all, kt0 + per_split);

  Loader<T, AKC, BM, NT> la;
  Loader<T, BKC, BN, NT> lb;
  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // operands that are not k-contiguous load tiles wholly inside the operand
  // without bounds checks (measured: no gain for k-contiguous ones)
  const bool kfull = g.K % TL::BK == 0;
  const bool afast = !AKC && kfull && m0 + BM <= g.M, bfast = !BKC && kfull && n0 + BN <= g.N;
  la.init(g.lda, tid);
  lb.init(g.ldb, tid);
  auto load_a = [&](int k0) {
    if (afast) la.load_fast(A, g.lda, m0, k0);
    else la.load(A, g.lda, g.M, g.K, m0, k0, tid);
  };
  auto load_b = [&](int k0) {
    if (bfast) lb.load_fast(B, g.ldb, n0, k0);
    else lb.load(B, g.ldb, g.N, g.K, n0, k0, tid);
  };
  if (kt0 < kt1) {
    load_a(kt0 * TL::BK);
    load_b(kt0 * TL::BK);
    la.store(As[0], tid);
    lb.store(Bs[0], tid);
  }
  __syncthreads();

  for (int kt = kt0; kt < kt1; ++kt) {
    const int cur = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) {
      load_a((kt + 1) * TL::BK);
      load_b((kt + 1) * TL::BK);
    }
    const T* as = As[cur] + (wm * TM * 16 + lr) * TL::PITCH + lg * 8;
    const T* bs = Bs[cur] + (wn * TN * 16 + lr) * TL::PITCH + lg * 8;
#pragma unroll
    for (int s = 0; s < TL::NSLICE; ++s) {
      Frag<T> fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) frag_load(fa[i], as + i * 16 * TL::PITCH + s * 32);
#pragma unroll
      for (int j = 0; j < TN; ++j) frag_load(fb[j], bs + j * 16 * TL::PITCH + s * 32);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) mfma16(acc[i][j], fb[j], fa[i]);
    }
    if (more) {
      la.store(As[cur ^ 1], tid);
      lb.store(Bs[cur ^ 1], tid);
    }
    __syncthreads();
  }

  // acc[i][j][r] = C[m][nb + r]
  if (gridDim.y > 1) {
    float* ws = g.ws + static_cast<int64_t>(blockIdx.y) * g.M * g.N;
    const bool vec_ws = (g.N & 3) == 0;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + (wm * TM + i) * 16 + lr;
      if (m >= g.M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int nb = n0 + (wn * TN + j) * 16 + lg * 4;
        if (nb >= g.N) continue;
        const int nvalid = min(4, g.N - nb);
        float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        store4<float>(ws + static_cast<int64_t>(m) * g.N + nb, v, vec_ws && nvalid == 4, nvalid);
      }
    }
    return;
  }
  const bool ld_vec = (g.ldc & 3) == 0;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + (wm * TM + i) * 16 + lr;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int nb = n0 + (wn * TN + j) * 16 + lg * 4;
      if (nb >= g.N) continue;
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      epilogue4<T, EPI>(g, m, nb, v, ld_vec);
    }
  }
}

// Sum of the split partials in split order, then the epilogue (store in the
// element type, store fp32, or add to fp32).
template <typename T, int EPI>
__global__ void __launch_bounds__(256) splitk_reduce(GemmArgs g, int splits) {
  const int64_t MN = static_cast<int64_t>(g.M) * g.N;
  const int64_t q = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (q >= MN) return;
  const int m = static_cast<int>(q / g.N);
  const int nb = static_cast<int>(q % g.N);
  if ((g.N & 3) == 0) {
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < splits; ++s) {
      const float4 p = *reinterpret_cast<const float4*>(g.ws + s * MN + q);
      v[0] += p.x; v[1] += p.y; v[2] += p.z; v[3] += p.w;
    }
    epilogue4<T, EPI>(g, m, nb, v, (g.ldc & 3) == 0);
  } else {
    for (int e = 0; e < 4 && q + e < MN; ++e) {
      const int mm = static_cast<int>((q + e) / g.N), nn = static_cast<int>((q + e) % g.N);
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      for (int s = 0; s < splits; ++s) v[0] += g.ws[s * MN + q + e];
      GemmArgs g1 = g;
      g1.N = nn + 1;  // one valid column at nn
      epilogue4<T, EPI>(g1, mm, nn, v, false);
    }
  }
}

template <typename T, bool AKC, bool BKC, class CF>
hipError_t launch_cfg(const GemmArgs& g, int epi, int splits, hipStream_t s) {
  const int tiles = ((g.M + CF::BM - 1) / CF::BM) * ((g.N + CF::BN - 1) / CF::BN);
  dim3 grid(tiles, splits), block(CF::NT);
  switch (epi) {
#define ATOM_CASE(E) \
  case E: hipLaunchKernelGGL((gemm_kernel<T, AKC, BKC, E, CF>), grid, block, 0, s, g); break;
    ATOM_CASE(EPI_STORE)
    ATOM_CASE(EPI_STORE_F32)
    ATOM_CASE(EPI_ACC_F32)
    ATOM_CASE(EPI_BIAS)
    ATOM_CASE(EPI_BIAS_GELU)
    ATOM_CASE(EPI_BIAS_RESID)
    ATOM_CASE(EPI_GELU_BWD)
#undef ATOM_CASE
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t MN = static_cast<int64_t>(g.M) * g.N;
  dim3 rgrid(static_cast<unsigned>((MN / 4 + 255) / 256 + 1)), rblock(256);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((splitk_reduce<T, EPI_STORE>), rgrid, rblock, 0, s, g, splits); break;
    case EPI_STORE_F32: hipLaunchKernelGGL((splitk_reduce<T, EPI_STORE_F32>), rgrid, rblock, 0, s, g, splits); break;
    case EPI_ACC_F32: hipLaunchKernelGGL((splitk_reduce<T, EPI_ACC_F32>), rgrid, rblock, 0, s, g, splits); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ------------------------------------------------------------ pipelined
// bf16 GEMM for large problems with a four-stage LDS pipeline fed by direct
// global-to-LDS loads (global_load_lds_dwordx4: no staging registers, no LDS
// store instructions).  256x256 output tile, 16 waves of 64x64, k tile of 32.
// Iteration t waits for its own stage (the loads of the two later stages may
// still be in flight), synchronises the workgroup, starts the loads of tile
// t+3 into the stage iteration t-1 has just finished reading, then computes.
// Each stage is a separate LDS array and the stage rotation is unrolled, so
// the compiler sees which array every load and read touches and inserts no
// waits of its own between them.
//
// LDS layouts (16-byte chunks are XOR-swizzled so that fragment reads are
// free of bank conflicts; a direct load writes 1 KB per wave contiguously, so
// the swizzle is applied to the global address each lane loads):
//   k-contiguous operand  [256 rows][32 k]: row r, chunk c at slot c ^ ((r>>1)&3);
//                         fragments by ds_read_b128.
//   other operand         [32 k][256 rows]: k row k, chunk c (8 rows) at slot
//                         c ^ tr_swz(k); fragments by two ds_read_b64_tr_b16,
//                         each transposing a 4 (k) x 16 (rows) block across 16
//                         lanes.
// Rows beyond the operand are clamped to its last valid row (or 8-row block),
// so they read finite data that only reaches output rows or columns that are
// never stored; k must be a multiple of 32.
#ifndef ATOM_GEMM_PIPE
#define ATOM_GEMM_PIPE 1
#endif
#ifndef P3_ROUNDS
#define P3_ROUNDS 1
#endif
namespace p3 {
constexpr int BM = 256, BN = 256, BK = 32, WM = 4, WN = 4, NT = 64 * WM * WN;
constexpr int TM = BM / (16 * WM), TN = BN / (16 * WN);
constexpr int OPB = BM * BK * 2;  // bytes of one operand tile in one stage


// Workgroup barrier that is also a compiler barrier for memory accesses.
// This wave's LDS reads must have completed (lgkmcnt) before it arrives, as
// the loads issued right after the barrier overwrite the stage they read;
// unlike __syncthreads it does not drain the direct loads still in flight.
__device__ __forceinline__ void barrier_only() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Swizzle of the transposed-read layout: a ds_read_b64_tr_b16 serves 32
// lanes per LDS cycle, i.e. the k rows K0..K0+3 and K0+8..K0+11 of two
// 16-lane groups; 2 (k & 3) + 8 ((k >> 3) & 1) puts their 16 chunks on
// distinct banks (measured: no conflicts, against two conflict cycles per
// read with 2 (k & 3) alone).
__device__ __forceinline__ int tr_swz(int k) { return 2 * (k & 3) + 8 * ((k >> 3) & 1); }

// Per-thread source of its one 16-byte chunk of an operand tile.
template <bool KC>
struct Src {
  const bf16_t* p;  // address for k0 = 0
  int64_t kstep;    // elements to advance per k tile
  __device__ void init(const bf16_t* X, int64_t ld, int r0, int Rlim, int tid) {
    if constexpr (KC) {
      const int r = tid >> 2, slot = tid & 3;
      const int c = slot ^ ((r >> 1) & 3);
      const int rr = min(r0 + r, Rlim - 1);
      p = X + static_cast<int64_t>(rr) * ld + c * 8;
      kstep = BK;
    } else {
      const int k = tid >> 5, slot = tid & 31;
      const int c = slot ^ tr_swz(k);
      const int m = min(r0 + c * 8, Rlim - 8);
      p = X + static_cast<int64_t>(k) * ld + m;
      kstep = static_cast<int64_t>(BK) * ld;
    }
  }
  __device__ __forceinline__ void load(uint8_t* stage, int kt, int w) const {
    lds_dma16(p + kt * kstep, __builtin_amdgcn_readfirstlane(lds_offset(stage) + w * 1024));
  }
};

// Byte offsets inside a stage of this lane's fragment reads of tile rows
// row0..row0+15 (one for k-contiguous operands, two transposed reads
// otherwise); loop-invariant, computed once.
template <bool KC>
struct FragOff {
  uint32_t o[KC ? 1 : 2];
  __device__ void init(int row0, int lane) {
    const int r = lane & 15, g = lane >> 4;
    if constexpr (KC) {
      const int row = row0 + r;
      o[0] = row * 64 + 16 * (g ^ ((row >> 1) & 3));
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = 8 * g + 4 * h + (r >> 2);
        const int m = row0 + 4 * (r & 3);
        o[h] = k * 512 + 16 * ((m >> 3) ^ tr_swz(k)) + 8 * (r & 1);
      }
    }
  }
};

// Fragment (16 rows x 32 k) of one 16-row tile from a stage.
template <bool KC>
__device__ __forceinline__ void frag(Frag<bf16_t>& f, const uint8_t* st, const FragOff<KC>& fo) {
  if constexpr (KC) {
    f.v = *reinterpret_cast<const uint4*>(st + fo.o[0]);
  } else {
    const uint2 lo = ds_read_tr8(st + fo.o[0]), hi = ds_read_tr8(st + fo.o[1]);
    f.v = make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
}

// Wait until at most n of this thread's loads are outstanding (n even, <= 4).
__device__ __forceinline__ void wait_loads(int n) {
  if (n >= 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if (n >= 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

}  // namespace p3

template <bool AKC, bool BKC, int EPI>
__global__ void __launch_bounds__(p3::NT) gemm_p3_kernel(GemmArgs g) {
  using namespace p3;
  __shared__ __attribute__((aligned(1024))) uint8_t sa0[OPB], sa1[OPB], sa2[OPB], sa3[OPB];
  __shared__ __attribute__((aligned(1024))) uint8_t sb0[OPB], sb1[OPB], sb2[OPB], sb3[OPB];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wm = w / WN, wn = w % WN;

  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int total = tiles_m * tiles_n;
  int pid = blockIdx.x;
  if ((total & 7) == 0) pid = (pid & 7) * (total >> 3) + (pid >> 3);
  constexpr int GROUP = 8;
  const int per_group = GROUP * tiles_n;
  const int first_m = (pid / per_group) * GROUP;
  const int gsize = min(tiles_m - first_m, GROUP);
  const int pid_m = first_m + (pid % per_group) % gsize;
  const int pid_n = (pid % per_group) / gsize;
  const int m0 = pid_m * BM, n0 = pid_n * BN;

  Src<AKC> sra;
  Src<BKC> srb;
  sra.init(static_cast<const bf16_t*>(g.A), g.lda, m0, g.M, tid);
  srb.init(static_cast<const bf16_t*>(g.B), g.ldb, n0, g.N, tid);
  const int nk = g.K / BK;

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  FragOff<AKC> foa[TM];
  FragOff<BKC> fob[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) foa[i].init(wm * TM * 16 + i * 16, lane);
#pragma unroll
  for (int j = 0; j < TN; ++j) fob[j].init(wn * TN * 16 + j * 16, lane);

  auto stage_a = [&](int s) -> uint8_t* { return s == 0 ? sa0 : s == 1 ? sa1 : s == 2 ? sa2 : sa3; };
  auto stage_b = [&](int s) -> uint8_t* { return s == 0 ? sb0 : s == 1 ? sb1 : s == 2 ? sb2 : sb3; };

  // prologue: tiles 0, 1, 2
#pragma unroll
  for (int s = 0; s < 3; ++s)
    if (s < nk) {
      sra.load(stage_a(s), s, w);
      srb.load(stage_b(s), s, w);
    }

  auto body = [&](auto S_, int t) {
    constexpr int S = decltype(S_)::value;
    // loads issued for tiles t+1 .. min(t+2, nk-1) may stay in flight
    wait_loads(2 * (min(t + 2, nk - 1) - t));
    barrier_only();
    if (t + 3 < nk) {
      sra.load(stage_a((S + 3) & 3), t + 3, w);
      srb.load(stage_b((S + 3) & 3), t + 3, w);
    }
    const uint8_t* as = stage_a(S);
    const uint8_t* bs = stage_b(S);
    Frag<bf16_t> fa[TM], fb[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) frag<AKC>(fa[i], as, foa[i]);
#pragma unroll
    for (int j = 0; j < TN; ++j) frag<BKC>(fb[j], bs, fob[j]);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) mfma16(acc[i][j], fb[j], fa[i]);
  };
  // four stages per loop iteration, so every stage index is a constant
  for (int t = 0; t < nk; t += 4 * P3_ROUNDS) {
#pragma unroll
    for (int r = 0; r < P3_ROUNDS; ++r) {
      const int tr = t + 4 * r;
      if (tr < nk) body(std::integral_constant<int, 0>{}, tr);
      if (tr + 1 < nk) body(std::integral_constant<int, 1>{}, tr + 1);
      if (tr + 2 < nk) body(std::integral_constant<int, 2>{}, tr + 2);
      if (tr + 3 < nk) body(std::integral_constant<int, 3>{}, tr + 3);
    }
  }

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // every direct load has landed
  // acc[i][j][r] = C[m][nb + r]
  const bool ld_vec = (g.ldc & 3) == 0;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + (wm * TM + i) * 16 + lr;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int nb = n0 + (wn * TN + j) * 16 + lg * 4;
      if (nb >= g.N) continue;
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      epilogue4<bf16_t, EPI>(g, m, nb, v, ld_vec);
    }
  }
}


// Four-wave variant of the pipelined kernel: the same 256x256 tile, k tile
// and LDS layouts, but four waves of 128x128 (one per SIMD, accumulators in
// AGPRs) whose fragment registers are double-buffered, so that the LDS reads
// of tile t+1 are issued between the MFMAs of tile t instead of after a
// barrier that every wave of the CU has to reach first.  A stage is free once
// the barrier that follows the reads of its tile has passed; the loads of
// tile t+4 go into the stage of tile t, so four tiles are in flight.
#ifndef ATOM_GEMM_P4
#define ATOM_GEMM_P4 1
#endif
namespace p4 {
constexpr int BM = 256, BN = 256, BK = 32, WM = 2, WN = 2, NT = 64 * WM * WN;
constexpr int TM = BM / (16 * WM), TN = BN / (16 * WN);
constexpr int OPB = BM * BK * 2;
constexpr int LPT = OPB / (NT * 16);  // direct loads per thread per operand and tile

// Barrier after this wave's LDS reads have completed; the wait is the
// builtin so that the compiler knows those fragment registers are ready.
__device__ __forceinline__ void barrier_after_reads() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), vmcnt and expcnt unconstrained
  asm volatile("s_barrier" ::: "memory");
}

// acc += a b with the accumulator pinned to its AGPRs.  The 256 accumulator
// registers of a wave fill the AGPR file; left to itself the register
// allocator splits them between AGPRs and VGPRs and copies them around every
// MFMA.  Issued in program order (volatile); the kernel supplies the wait
// states between the accumulators' other writes and reads and these MFMAs.
__device__ __forceinline__ void mfma_agpr(f32x4_t& acc, const Frag<bf16_t>& a, const Frag<bf16_t>& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
               : "+a"(acc)
               : "v"(__builtin_bit_cast(bf16x8_t, a.v)), "v"(__builtin_bit_cast(bf16x8_t, b.v)));
}
}  // namespace p4

template <bool AKC, bool BKC, int EPI>
__global__ void __launch_bounds__(p4::NT) __attribute__((amdgpu_waves_per_eu(1, 1))) gemm_p4_kernel(GemmArgs g) {
  using namespace p4;
  using p3::Src;
  using p3::FragOff;
  // stages 0..3 of A, then of B; after the loop, the epilogue's staging
  __shared__ __attribute__((aligned(1024))) uint8_t lds[8 * OPB];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wm = w / WN, wn = w % WN;

  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int total = tiles_m * tiles_n;
  int pid = blockIdx.x;
  if ((total & 7) == 0) pid = (pid & 7) * (total >> 3) + (pid >> 3);
  constexpr int GROUP = 8;
  const int per_group = GROUP * tiles_n;
  const int first_m = (pid / per_group) * GROUP;
  const int gsize = min(tiles_m - first_m, GROUP);
  const int pid_m = first_m + (pid % per_group) % gsize;
  const int pid_n = (pid % per_group) / gsize;
  const int m0 = pid_m * BM, n0 = pid_n * BN;

  // load q of a thread is the 16-byte chunk q * NT + tid of the tile
  Src<AKC> sra[LPT];
  Src<BKC> srb[LPT];
#pragma unroll
  for (int q = 0; q < LPT; ++q) {
    sra[q].init(static_cast<const bf16_t*>(g.A), g.lda, m0, g.M, q * NT + tid);
    srb[q].init(static_cast<const bf16_t*>(g.B), g.ldb, n0, g.N, q * NT + tid);
  }
  // k range of this workgroup: split blockIdx.y of gridDim.y equal ranges
  // (the launcher makes each a multiple of four k tiles)
  const int nk = g.K / BK / static_cast<int>(gridDim.y);
  const int kbase = static_cast<int>(blockIdx.y) * nk;
  // Each XCD starts its k loop at its own eighth of the range (the tile's
  // sum is rotated, the same for every launch of the shape).  Workgroups
  // walk k in step, so without it the whole GPU reads the same column range
  // of every row at once; when both operands are k-contiguous, rows of a long
  // k are 32 KB apart and those addresses share their low bits, which crowds
  // a few memory channels (4096x4096x16384: 500 -> 418 us).  The workgroups
  // of one XCD share operand tiles through its L2, so they keep one offset.
  const int koff = ((total & 7) == 0) ? ((blockIdx.x & 7) * (nk >> 3)) & ~3 : 0;
  auto rot = [&](int kt) {
    const int r = kt + koff;
    return kbase + (r >= nk ? r - nk : r);
  };

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      asm volatile("" : "+a"(acc[i][j]));
    }
  // wait states between the zeroing writes and the first MFMA reading them
  asm volatile("s_nop 7\n\ts_nop 7");

  FragOff<AKC> foa[TM];
  FragOff<BKC> fob[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) foa[i].init(wm * TM * 16 + i * 16, lane);
#pragma unroll
  for (int j = 0; j < TN; ++j) fob[j].init(wn * TN * 16 + j * 16, lane);

  auto stage_a = [&](int s) -> uint8_t* { return lds + s * OPB; };
  auto stage_b = [&](int s) -> uint8_t* { return lds + (4 + s) * OPB; };
  auto load_tile = [&](int s, int kt) {
#pragma unroll
    for (int q = 0; q < LPT; ++q) sra[q].load(stage_a(s), kt, q * (NT / 64) + w);
#pragma unroll
    for (int q = 0; q < LPT; ++q) srb[q].load(stage_b(s), kt, q * (NT / 64) + w);
  };

  Frag<bf16_t> fa0[TM], fb0[TN], fa1[TM], fb1[TN];
  // prologue: tiles 0..3 in flight, fragments of tile 0 in set 0.  Loads
  // past the last tile repeat it (into stages nobody reads again), so every
  // iteration has the same loads outstanding; they land before the exit.
#pragma unroll
  for (int s = 0; s < 4; ++s) load_tile(s, rot(min(s, nk - 1)));
  asm volatile("s_waitcnt vmcnt(24)" ::: "memory");
  barrier_after_reads();
#pragma unroll
  for (int i = 0; i < TM; ++i) p3::frag<AKC>(fa0[i], stage_a(0), foa[i]);
#pragma unroll
  for (int j = 0; j < TN; ++j) p3::frag<BKC>(fb0[j], stage_b(0), fob[j]);

  auto body = [&](auto S_, int t, Frag<bf16_t>(&ca)[TM], Frag<bf16_t>(&cb)[TN], Frag<bf16_t>(&na)[TM],
                  Frag<bf16_t>(&nb)[TN]) {
    constexpr int S = decltype(S_)::value;
    // tile t+1 has landed for every wave, and every wave has read tile t
    asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
    barrier_after_reads();
    const int kt = rot(min(t + 4, nk - 1));
    // per row i: the fragments i of tile t+1 (after the last tile they come
    // from a stale stage and are never used), then the MFMAs of row i of this
    // tile, which hide the reads' latency, with one direct load of tile t+4
    // half way (3-4 % faster than at the row's start; clustering the loads
    // cost 3-5 %)
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      p3::frag<AKC>(na[i], stage_a((S + 1) & 3), foa[i]);
      p3::frag<BKC>(nb[i], stage_b((S + 1) & 3), fob[i]);
#pragma unroll
      for (int j = 0; j < TN / 2; ++j) mfma_agpr(acc[i][j], cb[j], ca[i]);
      if (i < LPT) sra[i].load(stage_a(S), kt, i * (NT / 64) + w);
      else if (i < 2 * LPT) srb[i - LPT].load(stage_b(S), kt, (i - LPT) * (NT / 64) + w);
#pragma unroll
      for (int j = TN / 2; j < TN; ++j) mfma_agpr(acc[i][j], cb[j], ca[i]);
    }
  };
  // nk is a multiple of 4: no tile is conditional inside the loop
  for (int t = 0; t < nk; t += 4) {
    body(std::integral_constant<int, 0>{}, t, fa0, fb0, fa1, fb1);
    body(std::integral_constant<int, 1>{}, t + 1, fa1, fb1, fa0, fb0);
    body(std::integral_constant<int, 2>{}, t + 2, fa0, fb0, fa1, fb1);
    body(std::integral_constant<int, 3>{}, t + 3, fa1, fb1, fa0, fb0);
  }

  // every direct load has landed; wait states between the last MFMAs and
  // the reads of their accumulators
  asm volatile("s_waitcnt vmcnt(0)\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) asm volatile("" : "+a"(acc[i][j]));
  // Epilogue through LDS, 32 rows of the wave's 128x128 block at a time: the
  // accumulators go to a wave-private [32][128] fp32 staging area, and each
  // lane takes back 4 consecutive columns of one row, so a wave's stores (and
  // the epilogue's reads of bias, residual or saved pre-activations) cover
  // two whole 128-column rows instead of 32-byte pieces of 16 rows.
  barrier_after_reads();  // every wave is done with the stages
  constexpr int PITCH = 132;  // floats per staged row; rows 16 bytes of banks apart
  float* stg = reinterpret_cast<float*>(lds) + w * (32 * PITCH);
  const int row0 = m0 + wm * TM * 16, col0 = n0 + wn * TN * 16;
  // N, ldc and ldaux are multiples of 4 (p4_applies): a lane's four columns
  // are all inside the matrix or all past it, and every access is one
  // 4-vector.  They are the same columns in every row the lane stores, so the
  // bias is loaded once and the row pointers advance by a fixed stride.
  const int cc = 4 * (lane & 31), nb = col0 + cc, rsub = lane >> 5;
  const bool col_ok = nb < g.N;
  float bv[4] = {0.f, 0.f, 0.f, 0.f};
  if constexpr (epi_has_bias<EPI>())
    if (col_ok) {
      const uint2 w2 = *reinterpret_cast<const uint2*>(static_cast<const bf16_t*>(g.bias) + nb);
      bv[0] = bf2f(w2.x & 0xffff); bv[1] = bf2f(w2.x >> 16); bv[2] = bf2f(w2.y & 0xffff); bv[3] = bf2f(w2.y >> 16);
    }
  // The element operands (C itself, the fp32 residual or the saved bf16
  // pre-activation) are requested ahead of their use: every CU reaches its
  // epilogue at about the same time, so a load issued just before its use
  // waits out a GPU-wide burst.  bf16 operands go out two blocks of 32 rows
  // ahead (two registers per row), fp32 ones one block ahead.
  // Interior blocks take a branch-free copy of the epilogue: with per-row
  // bounds tests the compiler waits for every load in flight at each test,
  // which defeats the loads issued ahead.
  auto epilogue = [&](auto GUARD_, auto EPI_, const GemmArgs& ga) {
    constexpr bool GUARD = decltype(GUARD_)::value;
    constexpr int E = decltype(EPI_)::value;
    constexpr bool F32_OUT = E == EPI_STORE_F32 || E == EPI_ACC_F32 || E == EPI_BIAS_RESID;
    constexpr bool ELEM = epi_reads_elem<E>();
    constexpr int AHEAD = E == EPI_GELU_BWD ? 2 : 1;
    using Raw = typename std::conditional<E == EPI_GELU_BWD, uint2, float4>::type;
    Raw xr[TM / 2][16];
    auto load_block = [&](int h) {
      const int mq = row0 + h * 32 + rsub;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        if (!GUARD || (mq + 2 * q < ga.M && col_ok)) {
          if constexpr (E == EPI_GELU_BWD)
            xr[h][q] = *reinterpret_cast<const uint2*>(static_cast<const bf16_t*>(ga.aux) +
                                                       static_cast<int64_t>(mq + 2 * q) * ga.ldaux + nb);
          else
            xr[h][q] = *reinterpret_cast<const float4*>((E == EPI_ACC_F32 ? static_cast<const float*>(ga.C) : ga.resid) +
                                                        static_cast<int64_t>(mq + 2 * q) * ga.ldc + nb);
        }
      }
    };
    if constexpr (ELEM) {
#pragma unroll
      for (int h = 0; h <= AHEAD; ++h) load_block(h);
    }
#pragma unroll
    for (int h = 0; h < TM / 2; ++h) {
      if constexpr (ELEM)
        if (h > 0 && h + AHEAD < TM / 2) load_block(h + AHEAD);
      const int mq = row0 + h * 32 + rsub;  // row of q = 0; row q is mq + 2q
      const int64_t cq = static_cast<int64_t>(mq) * ga.ldc + nb, aq = static_cast<int64_t>(mq) * ga.ldaux + nb;
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const f32x4_t& a = acc[2 * h + ii][j];
          *reinterpret_cast<float4*>(stg + (ii * 16 + lr) * PITCH + j * 16 + lg * 4) = make_float4(a[0], a[1], a[2], a[3]);
        }
      float4 sv[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) sv[q] = *reinterpret_cast<const float4*>(stg + (2 * q + rsub) * PITCH + cc);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        if (GUARD && !(mq + 2 * q < ga.M && col_ok)) continue;
        float v[4] = {sv[q].x, sv[q].y, sv[q].z, sv[q].w};
        const int64_t off = cq + 2 * q * ga.ldc;
        float xe[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (E == EPI_GELU_BWD) {
          xe[0] = bf2f(xr[h][q].x & 0xffff); xe[1] = bf2f(xr[h][q].x >> 16);
          xe[2] = bf2f(xr[h][q].y & 0xffff); xe[3] = bf2f(xr[h][q].y >> 16);
        } else if constexpr (ELEM) {
          xe[0] = xr[h][q].x; xe[1] = xr[h][q].y; xe[2] = xr[h][q].z; xe[3] = xr[h][q].w;
        }
        // the arithmetic of epilogue4, in the same order
        if constexpr (E == EPI_ACC_F32) {
          for (int r = 0; r < 4; ++r) v[r] += xe[r];
        } else if constexpr (E == EPI_BIAS) {
          for (int r = 0; r < 4; ++r) v[r] += bv[r];
        } else if constexpr (E == EPI_BIAS_GELU) {
          float gv[4];
          for (int r = 0; r < 4; ++r) {
            const float u = to_f<bf16_t>(from_f<bf16_t>(v[r] + bv[r]));
            v[r] = u;
            gv[r] = gelu_f(u);
          }
          *reinterpret_cast<uint2*>(static_cast<bf16_t*>(ga.aux) + aq + 2 * q * ga.ldaux) =
              make_uint2(pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]));
          for (int r = 0; r < 4; ++r) v[r] = gv[r];
        } else if constexpr (E == EPI_BIAS_RESID) {
          for (int r = 0; r < 4; ++r) v[r] = xe[r] + (v[r] + bv[r]);
        } else if constexpr (E == EPI_GELU_BWD) {
          for (int r = 0; r < 4; ++r) v[r] *= gelu_grad_f(xe[r]);
        }
        if constexpr (F32_OUT)
          *reinterpret_cast<float4*>(static_cast<float*>(ga.C) + off) = make_float4(v[0], v[1], v[2], v[3]);
        else
          *reinterpret_cast<uint2*>(static_cast<bf16_t*>(ga.C) + off) = make_uint2(pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]));
      }
    }
  };
  const bool interior = row0 + TM * 16 <= g.M && col0 + TN * 16 <= g.N;
  if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_F32 || EPI == EPI_ACC_F32) {
    if (gridDim.y > 1) {
      // a split over k: the raw fp32 sums go to ws[split][M][N], and
      // splitk_reduce adds the splits in order and applies the epilogue
      GemmArgs gw = g;
      gw.C = g.ws + static_cast<int64_t>(blockIdx.y) * g.M * g.N;
      gw.ldc = g.N;
      if (interior) epilogue(std::false_type{}, std::integral_constant<int, EPI_STORE_F32>{}, gw);
      else epilogue(std::true_type{}, std::integral_constant<int, EPI_STORE_F32>{}, gw);
      return;
    }
  }
  if (interior) epilogue(std::false_type{}, std::integral_constant<int, EPI>{}, g);
  else epilogue(std::true_type{}, std::integral_constant<int, EPI>{}, g);
}


// The pipelined kernels apply to bf16 problems with k a multiple of 32 and
// (for clamped edge rows) M and N multiples of 8 with 16-byte aligned rows;
// launch_p3 takes those with at least one 256x256 tile per CU.
bool pipe_shape_ok(const GemmArgs& g) {
  return ATOM_GEMM_PIPE && g.K % p3::BK == 0 && g.K > 0 && g.M % 8 == 0 && g.N % 8 == 0 && g.lda % 8 == 0 &&
         g.ldb % 8 == 0 && g.M >= 8 && g.N >= 8;
}

int pipe_tiles(const GemmArgs& g) { return ((g.M + p3::BM - 1) / p3::BM) * ((g.N + p3::BN - 1) / p3::BN); }

bool p3_applies(const GemmArgs& g) { return pipe_shape_ok(g) && pipe_tiles(g) >= 256; }

// The four-wave kernel takes every epilogue when k is a multiple of four k
// tiles and the output rows (and the saved pre-activation's) are 16-byte
// aligned.
bool p4_applies(const GemmArgs& g, int epi) {
  const bool aux = epi == EPI_BIAS_GELU || epi == EPI_GELU_BWD;
  return ATOM_GEMM_P4 && g.K % (4 * p4::BK) == 0 && g.ldc % 4 == 0 && (!aux || g.ldaux % 4 == 0);
}

template <bool AKC, bool BKC>
hipError_t launch_p3(const GemmArgs& g, int epi, hipStream_t s) {
  const int tiles = ((g.M + p3::BM - 1) / p3::BM) * ((g.N + p3::BN - 1) / p3::BN);
  const bool four = p4_applies(g, epi);
  const dim3 grid(tiles);
  switch (epi) {
#define ATOM_CASE4(E)                                                                             \
  case E:                                                                                         \
    if (four) hipLaunchKernelGGL((gemm_p4_kernel<AKC, BKC, E>), grid, dim3(p4::NT), 0, s, g);      \
    else hipLaunchKernelGGL((gemm_p3_kernel<AKC, BKC, E>), grid, dim3(p3::NT), 0, s, g);           \
    break;
#define ATOM_CASE3(E) \
  case E: hipLaunchKernelGGL((gemm_p3_kernel<AKC, BKC, E>), grid, dim3(p3::NT), 0, s, g); break;
    ATOM_CASE4(EPI_STORE)
    ATOM_CASE4(EPI_STORE_F32)
    ATOM_CASE4(EPI_ACC_F32)
    ATOM_CASE4(EPI_BIAS)
    ATOM_CASE4(EPI_BIAS_GELU)
    ATOM_CASE4(EPI_BIAS_RESID)
    ATOM_CASE4(EPI_GELU_BWD)
#undef ATOM_CASE4
#undef ATOM_CASE3
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// The four-wave kernel on fewer 256x256 tiles than CUs (weight gradients of
// the narrower layers): the split count over k, 1 from 192 tiles on, else the
// smallest power of two that brings the workgroups to 192 or more, or the
// largest one the workspace holds if that leaves at least 96; splits need an
// epilogue that can follow their sum and k ranges of whole four-tile steps.
// 0 where the kernel does not apply.
int p4_splits(const GemmArgs& g, int epi, int tiles) {
  if (!pipe_shape_ok(g) || !p4_applies(g, epi)) return 0;
  if (tiles >= 192) return 1;
  if (!(epi == EPI_STORE || epi == EPI_STORE_F32 || epi == EPI_ACC_F32) || !g.ws) return 0;
  int best = 0;
  for (int sp = 2; sp <= 16 && tiles * best < 192; sp *= 2) {
    if (g.K % (4 * p4::BK * sp) != 0 || static_cast<uint64_t>(sp) * g.M * g.N * 4 > g.ws_bytes) break;
    best = sp;
  }
  return tiles * best >= 96 ? best : 0;
}

template <bool AKC, bool BKC>
hipError_t launch_p4_split(const GemmArgs& g, int epi, int tiles, int splits, hipStream_t s) {
  const dim3 grid(tiles, splits);
  switch (epi) {
#define ATOM_CASE(E) \
  case E: hipLaunchKernelGGL((gemm_p4_kernel<AKC, BKC, E>), grid, dim3(p4::NT), 0, s, g); break;
    ATOM_CASE(EPI_STORE)
    ATOM_CASE(EPI_STORE_F32)
    ATOM_CASE(EPI_ACC_F32)
    ATOM_CASE(EPI_BIAS)
    ATOM_CASE(EPI_BIAS_GELU)
    ATOM_CASE(EPI_BIAS_RESID)
    ATOM_CASE(EPI_GELU_BWD)
#undef ATOM_CASE
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t MN = static_cast<int64_t>(g.M) * g.N;
  dim3 rgrid(static_cast<unsigned>((MN / 4 + 255) / 256 + 1)), rblock(256);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((splitk_reduce<bf16_t, EPI_STORE>), rgrid, rblock, 0, s, g, splits); break;
    case EPI_STORE_F32: hipLaunchKernelGGL((splitk_reduce<bf16_t, EPI_STORE_F32>), rgrid, rblock, 0, s, g, splits); break;
    case EPI_ACC_F32: hipLaunchKernelGGL((splitk_reduce<bf16_t, EPI_ACC_F32>), rgrid, rblock, 0, s, g, splits); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Tile configuration and split count for a problem: the large tile when it
// gives at least one workgroup per CU, else the 128x128 tile; a split over k
// when even that leaves the CUs idle and k is long (weight gradients of
// small layers), limited by the workspace.
template <typename T, bool AKC, bool BKC>
hipError_t launch_t(const GemmArgs& g, int epi, hipStream_t s) {
  constexpr int CUS = 256;
  if constexpr (sizeof(T) == 2) {
    if (p3_applies(g)) return launch_p3<AKC, BKC>(g, epi, s);
    const int tiles = pipe_tiles(g), splits = p4_splits(g, epi, tiles);
    if (splits > 0) return launch_p4_split<AKC, BKC>(g, epi, tiles, splits, s);
  }
  const int tiles_big = ((g.M + Big::BM - 1) / Big::BM) * ((g.N + Big::BN - 1) / Big::BN);
  if (tiles_big >= CUS) return launch_cfg<T, AKC, BKC, Big>(g, epi, 1, s);
  const int tiles = ((g.M + Small::BM - 1) / Small::BM) * ((g.N + Small::BN - 1) / Small::BN);
  const int nk = (g.K + Tile<T>::BK - 1) / Tile<T>::BK;
  int splits = 1;
  const bool can_split = epi == EPI_STORE || epi == EPI_STORE_F32 || epi == EPI_ACC_F32;
  if (can_split && g.ws && tiles < 2 * CUS && nk >= 32) {
    splits = std::min((2 * CUS + tiles - 1) / tiles, nk / 16);
    const int64_t per = static_cast<int64_t>(g.M) * g.N * 4;
    splits = static_cast<int>(std::min<int64_t>(splits, static_cast<int64_t>(g.ws_bytes / per)));
    splits = std::max(1, std::min(splits, 16));
  }
  return launch_cfg<T, AKC, BKC, Small>(g, epi, splits, s);
}

}  // namespace

// Shape and alignment rules checked before launch (bounds inside the kernel
// rely on them): K a multiple of 8 (bf16) or 4 (fp32), so a 16-byte k chunk
// is either wholly inside or wholly outside; a k-contiguous operand needs a
// leading dimension that keeps 16-byte chunks aligned; a bf16 operand that is
// not k-contiguous is read as dwords of two rows, so it needs an even row
// count and an even leading dimension; all pointers 16-byte aligned.
hipError_t gemm_check(const GemmArgs& g, int dtype, bool akc, bool bkc) {
  const int kv = dtype == DT_BF16 ? 8 : 4;
  if (g.M < 0 || g.N < 0 || g.K < 0) return hipErrorInvalidValue;
  if (g.K % kv) return hipErrorInvalidValue;
  if (akc ? g.lda % kv : (dtype == DT_BF16 && ((g.lda | g.M) & 1))) return hipErrorInvalidValue;
  if (bkc ? g.ldb % kv : (dtype == DT_BF16 && ((g.ldb | g.N) & 1))) return hipErrorInvalidValue;
  if ((reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.B) | reinterpret_cast<uintptr_t>(g.C)) & 15)
    return hipErrorInvalidValue;
  if (akc ? g.lda < g.K : g.lda < g.M) return hipErrorInvalidValue;
  if (bkc ? g.ldb < g.K : g.ldb < g.N) return hipErrorInvalidValue;
  if (g.ldc < g.N) return hipErrorInvalidValue;
  return hipSuccess;
}

hipError_t gemm(const GemmArgs& g, int dtype, bool akc, bool bkc, int epi, hipStream_t s) {
  hipError_t e = gemm_check(g, dtype, akc, bkc);
  if (e != hipSuccess) return e;
  if (g.M == 0 || g.N == 0) return hipSuccess;
  if (dtype == DT_BF16) {
    if (akc && bkc) return launch_t<bf16_t, true, true>(g, epi, s);
    if (akc && !bkc) return launch_t<bf16_t, true, false>(g, epi, s);
    if (!akc && !bkc) return launch_t<bf16_t, false, false>(g, epi, s);
    return launch_t<bf16_t, false, true>(g, epi, s);
  }
  if (akc && bkc) return launch_t<float, true, true>(g, epi, s);
  if (akc && !bkc) return launch_t<float, true, false>(g, epi, s);
  if (!akc && !bkc) return launch_t<float, false, false>(g, epi, s);
  return launch_t<float, false, true>(g, epi, s);
}

}  // namespace atom
