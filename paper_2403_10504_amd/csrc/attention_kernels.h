// Causal self-attention kernel templates; instantiated by attention.hip
// (bf16: the direct-load kernels attn_fwd_dl, attn_bwd_dkdv_dl,
// attn_bwd_dq_dl) and attention_f32.hip (fp32 validation mode: the
// register-staged kernels below, which stage tiles through registers into
// padded LDS and transpose V, Q, dO or K while storing).
//
// Fused causal self-attention on CDNA4 matrix cores (tiled, online softmax;
// the [T, T] score matrix never leaves registers).
//
// Layout: qkv [B*T][3*d] with q, k, v at column offsets 0, d, 2d and head h at
// h*dh inside each; o [B*T][d]; lse [B][H][T] (natural log of the row sum of
// exp(scale * q.k) over the unmasked keys).  scale = 1/sqrt(dh); key j is
// visible to query i iff j <= i.
//
// Each wave owns G groups of 16 rows; fragments read from LDS are reused by
// all G groups.  Key/query tiles of 64 rows are staged in LDS and, when two
// stages fit, double-buffered: the next tile is loaded into registers while
// the current one is consumed, so global-memory latency overlaps the MFMAs.
//   forward : S^T = K Q^T (lanes hold one query, so the accumulators feed the
//             P V product as B operands directly); online softmax; O += V^T P^T.
//   dK, dV  : a workgroup of W waves owns 16*W keys and loops over the query
//             tiles at or below the diagonal; S = Q K^T, dP = dO V^T,
//             dS = P (dP - D); dV += P^T dO, dK += dS^T Q.
//   dQ      : a workgroup of NW waves owns 16*NW*G queries and loops over key
//             tiles; dQ += dS K.
// Splitting dQ from dK/dV makes every output owned by one workgroup, so the
// backward needs no atomics and is bitwise reproducible.
#pragma once
#include <type_traits>

#include "common.h"
#include "launch.h"

namespace atom {
namespace attn {

constexpr int BT = 64;  // rows per staged tile (keys or queries)
// Lazy rescaling: the running row maximum is only raised when a new score
// exceeds it by more than this (log2 units), so p = 2^(s - m) <= 2^8.  The
// final division by the row sum makes the result independent of the
// reference maximum.
constexpr float RESCALE_LOG2 = 8.f;

// 2^x by the hardware instruction (inputs here are finite or -inf; results
// that would be denormal flush to zero, as p is later rounded anyway).
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
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
  static constexpr int ROWS_BYTES = BT * RP * sizeof(T);
  static constexpr int TRANS_BYTES = DH * TP * sizeof(T);
};

// Register staging of one 64-row tile of a head slice (row stride ld), in
// the natural [row][c] layout (16-byte chunks) or transposed [c][row] (dword
// loads of PAIR columns over KV consecutive rows, transposed in registers).
template <typename T, int DH, int NT, bool TRANS>
struct TileLoader {
  using L = ALay<T, DH>;
  static constexpr int CPR = DH / L::KV;                   // natural: chunks per row
  static constexpr int NCH = BT * CPR / NT;                 // natural: chunks per thread
  static constexpr int PAIR = 4 / sizeof(T);
  static constexpr int UC = DH / PAIR;                      // transposed: dword columns
  static constexpr int UNITS = (BT / L::KV) * UC;
  static constexpr int NU = (UNITS + NT - 1) / NT;          // transposed: units per thread
  static constexpr int NREG = TRANS ? NU * L::KV : NCH * 4;
  uint32_t r[NREG];

  // Rows r0 .. r0+63 of the tile; rows at or beyond nrows read as zero.
  // A tile wholly inside [0, nrows) takes the unchecked path.
  __device__ __forceinline__ void load(const T* __restrict__ base, int64_t ld, int r0, int nrows, int tid) {
    const T* tb = base + static_cast<int64_t>(r0) * ld;
    const bool full = r0 + BT <= nrows;
    if constexpr (!TRANS) {
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int c = tid + NT * i;
        const int rr = c / CPR, k = (c % CPR) * L::KV;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (full || r0 + rr < nrows) v = *reinterpret_cast<const uint4*>(tb + static_cast<int64_t>(rr) * ld + k);
        r[4 * i] = v.x;
        r[4 * i + 1] = v.y;
        r[4 * i + 2] = v.z;
        r[4 * i + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < NU; ++i) {
        const int u = tid + NT * i;
        const int rb = u / UC, cc = (u % UC) * PAIR;
        const T* p = tb + static_cast<int64_t>(rb * L::KV) * ld + cc;
        if (full && (UNITS % NT == 0 || u < UNITS)) {
#pragma unroll
          for (int j = 0; j < L::KV; ++j) r[i * L::KV + j] = *reinterpret_cast<const uint32_t*>(p + j * ld);
        } else {
#pragma unroll
          for (int j = 0; j < L::KV; ++j) {
            const int rr = r0 + rb * L::KV + j;
            r[i * L::KV + j] = (u < UNITS && rr < nrows) ? *reinterpret_cast<const uint32_t*>(p + j * ld) : 0u;
          }
        }
      }
    }
  }

  __device__ __forceinline__ void store(T* S, int tid) {
    if constexpr (!TRANS) {
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int c = tid + NT * i;
        const int rr = c / CPR, k = (c % CPR) * L::KV;
        *reinterpret_cast<uint4*>(S + rr * L::RP + k) = make_uint4(r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < NU; ++i) {
        const int u = tid + NT * i;
        if (u >= UNITS) continue;
        const int rb = u / UC, cc = (u % UC) * PAIR;
        const uint32_t* d = r + i * L::KV;
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
  }
};

// Fragment of a head row (for a register-resident operand): row r, column col.
template <typename T>
__device__ __forceinline__ void frag_global(Frag<T>& f, const T* __restrict__ base, int64_t ld, int r, int nrows,
                                            int col) {
  if (r < nrows) frag_load(f, base + static_cast<int64_t>(r) * ld + col);
  else frag_zero(f);
}

// B-operand fragment for a 32-wide slice from two 16-row tiles of per-lane
// accumulator values x[t][r] (t = 2s, 2s+1): element e < 4 takes x[2s][e],
// e >= 4 takes x[2s+1][e-4].  The matching A operand reads rows
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
__device__ __forceinline__ void store_row4(T* p, const float* v) {
  if constexpr (sizeof(T) == 2) {
    uint2 w;
    w.x = pack_bf16(v[0], v[1]);
    w.y = pack_bf16(v[2], v[3]);
    *reinterpret_cast<uint2*>(p) = w;
  } else {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

// Two stages of `bytes` fit in the LDS budget of one workgroup.
constexpr bool two_stages(int bytes) { return 2 * bytes <= 150 * 1024; }

// ------------------------------------------------------------------ forward
template <typename T, int DH, int G>
// Workgroups per CU the register allocation must allow.  Two forward
// workgroups per CU (two waves per SIMD, within 256 registers) overlap one
// wave's softmax with the other's MFMAs and loads: 1.7x faster at d_head 128.
#ifndef ATOM_ATTN_FWD_OCC
#define ATOM_ATTN_FWD_OCC 2
#endif
#ifndef ATOM_ATTN_DQ_OCC
#define ATOM_ATTN_DQ_OCC 1
#endif
__global__ void __launch_bounds__(256, ATOM_ATTN_FWD_OCC) attn_fwd_kernel(const T* __restrict__ qkv, T* __restrict__ o,
                                                       float* __restrict__ lse, int B, int Tn, int H) {
  using L = ALay<T, DH>;
  constexpr int STAGE = L::ROWS_BYTES + L::TRANS_BYTES;
  constexpr int NBUF = two_stages(STAGE) ? 2 : 1;
  constexpr int BQ = 4 * 16 * G;  // queries per workgroup
  __shared__ __attribute__((aligned(16))) T Ks[NBUF][BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Vt[NBUF][DH * L::TP];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const T* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const T* kb = qb + d;
  const T* vb = qb + 2 * d;
  const int q0 = blockIdx.x * BQ;
  const int qw = q0 + w * 16 * G;  // first query of this wave
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));

  Frag<T> qf[G][L::NS];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int s = 0; s < L::NS; ++s) frag_global(qf[g][s], qb, ld, qw + g * 16 + lr, Tn, 32 * s + 8 * lg);

  f32x4_t acc_o[G][L::NCT];
  float m_i[G], l_i[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_i[g] = -1e30f;
    l_i[g] = 0.f;
#pragma unroll
    for (int c = 0; c < L::NCT; ++c) acc_o[g][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  TileLoader<T, DH, 256, false> lk;
  TileLoader<T, DH, 256, true> lv;
  const int n_kt = min((Tn + BT - 1) / BT, (min(q0 + BQ, Tn) - 1) / BT + 1);
  lk.load(kb, ld, 0, Tn, tid);
  lv.load(vb, ld, 0, Tn, tid);
  lk.store(Ks[0], tid);
  lv.store(Vt[0], tid);
  __syncthreads();

  for (int kt = 0; kt < n_kt; ++kt) {
    const int j0 = kt * BT;
    const int cur = NBUF == 2 ? (kt & 1) : 0;
    const bool more = kt + 1 < n_kt;
    if (NBUF == 2 && more) {
      lk.load(kb, ld, j0 + BT, Tn, tid);
      lv.load(vb, ld, j0 + BT, Tn, tid);
    }
    const T* ks = Ks[cur];
    const T* vt = Vt[cur];
    // the wave's queries that can see part of this key tile
    if (j0 <= qw + 16 * G - 1) {
      float p[G][4][4];
      float mloc[G];
#pragma unroll
      for (int g = 0; g < G; ++g) mloc[g] = -INFINITY;
#pragma unroll
      for (int jt = 0; jt < 4; ++jt) {
        f32x4_t a[G];
#pragma unroll
        for (int g = 0; g < G; ++g) a[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < L::NS; ++s) {
          Frag<T> kf;
          frag_load(kf, ks + (jt * 16 + lr) * L::RP + 32 * s + 8 * lg);
#pragma unroll
          for (int g = 0; g < G; ++g) mfma16(a[g], kf, qf[g][s]);
        }
        const bool edge = j0 + BT > qw || j0 + BT > Tn;  // tile touches the diagonal or the end
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const int qi = qw + g * 16 + lr;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int j = j0 + jt * 16 + 4 * lg + r;
            const float x = (!edge || (j <= qi && j < Tn)) ? a[g][r] * sc : -INFINITY;
            p[g][jt][r] = x;
            mloc[g] = fmaxf(mloc[g], x);
          }
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float mx = fmaxf(mloc[g], __shfl_xor(mloc[g], 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        // raise the reference maximum only when some lane of the wave needs it
        // (a wave-uniform branch, so the rescale of O is skipped together)
        if (__builtin_amdgcn_ballot_w64(mx > m_i[g] + RESCALE_LOG2) != 0) {
          const float m_new = fmaxf(m_i[g], mx);
          const float alpha = ex2(m_i[g] - m_new);
          l_i[g] *= alpha;
          m_i[g] = m_new;
#pragma unroll
          for (int c = 0; c < L::NCT; ++c) acc_o[g][c] *= alpha;
        }
        float lsum = 0.f;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            p[g][jt][r] = ex2(p[g][jt][r] - m_i[g]);
            lsum += p[g][jt][r];
          }
        l_i[g] += lsum;
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        Frag<T> pf[G];
#pragma unroll
        for (int g = 0; g < G; ++g) frag_from_pair(pf[g], p[g], s2);
#pragma unroll
        for (int c = 0; c < L::NCT; ++c) {
          Frag<T> vf;
          frag_pair_rows<T, DH>(vf, vt, c * 16 + lr, s2, lg);
#pragma unroll
          for (int g = 0; g < G; ++g) mfma16(acc_o[g][c], vf, pf[g]);
        }
      }
    }
    if (more) {
      if (NBUF == 1) {
        __syncthreads();
        lk.load(kb, ld, j0 + BT, Tn, tid);
        lv.load(vb, ld, j0 + BT, Tn, tid);
      }
      lk.store(Ks[NBUF == 2 ? (cur ^ 1) : 0], tid);
      lv.store(Vt[NBUF == 2 ? (cur ^ 1) : 0], tid);
    }
    __syncthreads();
  }

#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int qi = qw + g * 16 + lr;
    float l_tot = l_i[g] + __shfl_xor(l_i[g], 16, 64);
    l_tot += __shfl_xor(l_tot, 32, 64);
    if (qi < Tn) {
      const float inv = 1.f / l_tot;
      T* orow = o + (static_cast<int64_t>(b) * Tn + qi) * d + h * DH;
#pragma unroll
      for (int c = 0; c < L::NCT; ++c) {
        float v[4] = {acc_o[g][c][0] * inv, acc_o[g][c][1] * inv, acc_o[g][c][2] * inv, acc_o[g][c][3] * inv};
        store_row4<T>(orow + c * 16 + 4 * lg, v);
      }
      if (lg == 0) lse[(static_cast<int64_t>(b) * H + h) * Tn + qi] = (m_i[g] + log2f(l_tot)) * LN2;
    }
  }
}

// Work item of a workgroup in a [n_x blocks][B*H heads] grid.  Under the
// causal mask the blocks of a head carry unequal work (block x of the
// forward visits x+1 key tiles), so the items are handed out heaviest first
// over all heads: a workgroup that starts late then has little left to do,
// and the kernel does not wait on a heavy block that started behind a run of
// light ones (heaviest-first within each head, one head after another, left
// the 6.7B forward with about 1.1 of its 2 resident waves per SIMD on
// average).  The hardware hands consecutive linear ids to the 8 XCDs in
// turn; when the heads split evenly over them, each XCD takes its own eighth
// of the heads (all their blocks), so one head's K and V stay in one L2.
// heavy_last: block x does work growing with x (forward, dQ); otherwise
// shrinking (dK/dV).
struct BlockId {
  int x, bh;
};
__device__ __forceinline__ BlockId attn_block(bool heavy_last) {
  const int n_x = gridDim.x, n_bh = gridDim.y;
  const int lin = blockIdx.y * n_x + blockIdx.x;
  int rank, bh;  // rank 0 = the heaviest block
  if ((n_bh & 7) == 0) {
    const int per = n_bh >> 3, i = lin >> 3;  // heads per XCD; item index inside the XCD
    rank = i / per;
    bh = (lin & 7) * per + i % per;
  } else {
    rank = lin / n_bh;
    bh = lin % n_bh;
  }
  return BlockId{heavy_last ? n_x - 1 - rank : rank, bh};
}

// ------------------------------------------- forward, bf16, direct loads
// The K and V tiles of a key tile go straight from global memory to LDS
// (global_load_lds_dwordx4, no staging registers, no LDS stores), two stages
// deep: the loads of tile t+1 are issued after the barrier that opens tile t,
// into the stage tile t-1 used.  V stays in its natural [key][dh] layout and
// the A operand of O^T += V^T P^T is read with ds_read_b64_tr_b16.  Each
// fragment read is issued one step ahead of the MFMAs that use it.
//
// Stage layout: K [64][DH] then V [64][DH], rows of DH*2 bytes in 16-byte
// chunks; chunk c of row r sits at slot c ^ kswz(r) (K) or c ^ vswz(r) (V):
//   K: a ds_read_b128 serves 16 lanes per LDS cycle, 16 consecutive rows at
//      one chunk;
//   V: a ds_read_b64_tr_b16 serves 32 lanes, 8 consecutive rows at one
//      aligned chunk pair (vswz is even, so pairs stay pairs).
// Keys past the end read the last row (finite data; their scores are masked
// to -inf, so they weigh zero).
template <int DH, int NT = 256>
struct FwdDL {
  static constexpr int CPR = DH / 8;             // chunks per row
  static constexpr int TILE = BT * DH * 2;       // bytes of a K or V tile
  static constexpr int STAGE = 2 * TILE;
  static constexpr int LPT = TILE / (NT * 16);   // direct loads per thread per tile and operand
  static_assert(DH == 64 || DH == 128, "head size");
  __device__ static int kswz(int r) { return DH == 128 ? (r & 15) : ((r >> 1) & 7); }
  __device__ static int vswz(int r) { return DH == 128 ? 2 * (r & 7) : 2 * ((r >> 1) & 3); }
};

// NW waves of G groups of 16 queries per workgroup.  Waves per SIMD the
// register allocation must allow (the second launch bound): four with eight
// waves of one group (d_h 128: two workgroups per CU, as the LDS allows, in
// 128 registers with a spill of nine; against four waves of two groups at two
// waves per SIMD, 230 registers: 90-92 against 92-96 us at the 6.7B shape,
// 59 against 68-69 at 13B's, whose 40 heads leave the last round of work
// items less full); four with four waves of two groups at d_h 64, where 128
// registers suffice and four workgroups fit the LDS (82 against 88 us at
// GPT-3 Small's shape; five spill).
template <int DH, int G, int NW>
__global__ void __launch_bounds__(64 * NW, (DH == 64 || G == 1) ? 4 : 2)
    attn_fwd_dl_kernel(const bf16_t* __restrict__ qkv, bf16_t* __restrict__ o, float* __restrict__ lse, int B, int Tn,
                       int H) {
  constexpr int NT = 64 * NW;
  using F = FwdDL<DH, NT>;
  constexpr int NS = DH / 32, NCT = DH / 16, BQ = NW * 16 * G, RB = DH * 2;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * F::STAGE];

  // the wave index through readfirstlane, so that everything derived from
  // it (the wave's queries, the diagonal test) is known to be wave-uniform
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const BlockId blk = attn_block(true);
  const int bh = blk.bh, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const bf16_t* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const bf16_t* kb = qb + d;
  const bf16_t* vb = qb + 2 * d;
  const int q0 = blk.x * BQ;
  const int qw = q0 + w * 16 * G;
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));

  Frag<bf16_t> qf[G][NS];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int s = 0; s < NS; ++s) frag_global(qf[g][s], qb, ld, qw + g * 16 + lr, Tn, 32 * s + 8 * lg);

  f32x4_t acc_o[G][NCT];
  float m_i[G], l_i[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_i[g] = -1e30f;
    l_i[g] = 0.f;
#pragma unroll
    for (int c = 0; c < NCT; ++c) acc_o[g][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  // load q of a thread: chunk q*256 + tid of the tile (row, slot).  Its
  // sources for key tile 0 are computed once; a whole tile adds the tile's
  // row offset (a wave-uniform product), only the last, partial tile clamps
  // its rows to the last key.
  const bf16_t* ksrc[F::LPT];
  const bf16_t* vsrc[F::LPT];
#pragma unroll
  for (int q = 0; q < F::LPT; ++q) {
    const int id = q * NT + tid, row = id / F::CPR, slot = id % F::CPR;
    ksrc[q] = kb + static_cast<int64_t>(row) * ld + (slot ^ F::kswz(row)) * 8;
    vsrc[q] = vb + static_cast<int64_t>(row) * ld + (slot ^ F::vswz(row)) * 8;
  }
  auto load_tile = [&](int st, int j0) {
    const uint32_t kl = lds_offset(lds + st * F::STAGE), vl = kl + F::TILE;
    const bool whole = j0 + BT <= Tn;
#pragma unroll
    for (int q = 0; q < F::LPT; ++q) {
      const uint32_t lo = __builtin_amdgcn_readfirstlane((q * NT + w * 64) * 16);
      if (whole) {
        const int64_t off = static_cast<int64_t>(j0) * ld;
        lds_dma16(ksrc[q] + off, kl + lo);
        lds_dma16(vsrc[q] + off, vl + lo);
      } else {
        const int id = q * NT + tid, row = id / F::CPR, slot = id % F::CPR;
        const int64_t gr = static_cast<int64_t>(min(j0 + row, Tn - 1)) * ld;
        lds_dma16(kb + gr + (slot ^ F::kswz(row)) * 8, kl + lo);
        lds_dma16(vb + gr + (slot ^ F::vswz(row)) * 8, vl + lo);
      }
    }
  };
  // fragment addresses inside a stage
  auto kfrag = [&](Frag<bf16_t>& f, const uint8_t* ks, int jt, int s) {
    const int row = jt * 16 + lr;
    f.v = *reinterpret_cast<const uint4*>(ks + row * RB + ((4 * s + lg) ^ F::kswz(row)) * 16);
  };
  auto vfrag = [&](Frag<bf16_t>& f, const uint8_t* vs, int s2, int c) {
    // keys 32 s2 + 4 lg + 0..3 (elements 0..3) and 32 s2 + 16 + 4 lg + 0..3
    // (elements 4..7), the order of the P fragment built from two 16-key tiles
    const int chunk = 2 * c + ((lr & 3) >> 1);
    const int r0 = 32 * s2 + 4 * lg + (lr >> 2), r1 = r0 + 16;
    const uint2 lo = ds_read_tr8(vs + r0 * RB + (chunk ^ F::vswz(r0)) * 16 + 8 * (lr & 1));
    const uint2 hi = ds_read_tr8(vs + r1 * RB + (chunk ^ F::vswz(r1)) * 16 + 8 * (lr & 1));
    f.v = make_uint4(lo.x, lo.y, hi.x, hi.y);
  };

  const int n_kt = min((Tn + BT - 1) / BT, (min(q0 + BQ, Tn) - 1) / BT + 1);
  load_tile(0, 0);
  for (int kt = 0; kt < n_kt; ++kt) {
    const int j0 = kt * BT, cur = kt & 1;
    // tile kt has landed for every wave, and every wave is done with tile kt-1
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    asm volatile("s_barrier" ::: "memory");
    if (kt + 1 < n_kt) load_tile(cur ^ 1, j0 + BT);
    const uint8_t* ks = lds + cur * F::STAGE;
    const uint8_t* vs = ks + F::TILE;
    if (j0 <= qw + 16 * G - 1) {
      float p[G][4][4];
      float mloc[G];
#pragma unroll
      for (int g = 0; g < G; ++g) mloc[g] = -INFINITY;
      // raw scores, masked by selects (not per-element control flow); the
      // scale goes into the max once and into the exponent's FMA.  The mask
      // is a template parameter: the whole scores phase of a tile is one
      // branch-free block, so the maxima of 16 keys overlap the next 16 keys'
      // MFMAs (a test per 16 keys split it into blocks the scheduler does not
      // cross).
      auto score_tile = [&](auto MASK_) {
        constexpr bool MASK = decltype(MASK_)::value;
        Frag<bf16_t> kf[2][NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) kfrag(kf[0][s], ks, 0, s);
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
          if (jt + 1 < 4) {
#pragma unroll
            for (int s = 0; s < NS; ++s) kfrag(kf[(jt + 1) & 1][s], ks, jt + 1, s);
          }
          f32x4_t a[G];
#pragma unroll
          for (int g = 0; g < G; ++g) a[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int g = 0; g < G; ++g) mfma16(a[g], kf[jt & 1][s], qf[g][s]);
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const int qi = qw + g * 16 + lr;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int j = j0 + jt * 16 + 4 * lg + r;
              float x = a[g][r];
              if constexpr (MASK) x = ((j <= qi) & (j < Tn)) ? x : -INFINITY;
              p[g][jt][r] = x;
              mloc[g] = fmaxf(mloc[g], x);
            }
          }
        }
      };
      if (j0 + BT > qw || j0 + BT > Tn) score_tile(std::true_type{});  // tile touches the diagonal or the end
      else score_tile(std::false_type{});
      Frag<bf16_t> vf[2];
      vfrag(vf[0], vs, 0, 0);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float mx = rows4_max(mloc[g]) * sc;
        if (__builtin_amdgcn_ballot_w64(mx > m_i[g] + RESCALE_LOG2) != 0) {
          const float m_new = fmaxf(m_i[g], mx);
          const float alpha = ex2(m_i[g] - m_new);
          l_i[g] *= alpha;
          m_i[g] = m_new;
#pragma unroll
          for (int c = 0; c < NCT; ++c) acc_o[g][c] *= alpha;
        }
        float lsum = 0.f;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            p[g][jt][r] = ex2(__builtin_fmaf(p[g][jt][r], sc, -m_i[g]));
            lsum += p[g][jt][r];
          }
        l_i[g] += lsum;
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        Frag<bf16_t> pf[G];
#pragma unroll
        for (int g = 0; g < G; ++g) frag_from_pair(pf[g], p[g], s2);
#pragma unroll
        for (int c = 0; c < NCT; ++c) {
          const int n = s2 * NCT + c;
          if (n + 1 < 2 * NCT) vfrag(vf[(n + 1) & 1], vs, (n + 1) / NCT, (n + 1) % NCT);
#pragma unroll
          for (int g = 0; g < G; ++g) mfma16(acc_o[g][c], vf[n & 1], pf[g]);
        }
      }
    }
  }

#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int qi = qw + g * 16 + lr;
    const float l_tot = rows4_sum(l_i[g]);
    if (qi < Tn) {
      const float inv = 1.f / l_tot;
      bf16_t* orow = o + (static_cast<int64_t>(b) * Tn + qi) * d + h * DH;
#pragma unroll
      for (int c = 0; c < NCT; ++c) {
        float v[4] = {acc_o[g][c][0] * inv, acc_o[g][c][1] * inv, acc_o[g][c][2] * inv, acc_o[g][c][3] * inv};
        store_row4<bf16_t>(orow + c * 16 + 4 * lg, v);
      }
      if (lg == 0) lse[(static_cast<int64_t>(b) * H + h) * Tn + qi] = (m_i[g] + log2f(l_tot)) * LN2;
    }
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

// bf16: eight consecutive elements per thread (16-byte loads), DH/8 threads
// per (row, head) summed by shuffles in a fixed order.  Head h of row r sits
// at (r*H + h)*DH, so the pairs are contiguous and a workgroup reads one
// contiguous range of O and of dO.
template <int DH>
__global__ void __launch_bounds__(256) attn_delta_bf16_kernel(const bf16_t* __restrict__ o,
                                                              const bf16_t* __restrict__ dout,
                                                              float* __restrict__ delta, int64_t n_pairs, int Tn,
                                                              int H) {
  constexpr int G = DH / 8;
  const int64_t gid = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t idx = gid / G;
  const int sub = static_cast<int>(gid % G);
  float s = 0.f;
  if (idx < n_pairs) {
    const uint4 a = *reinterpret_cast<const uint4*>(o + idx * DH + 8 * sub);
    const uint4 b = *reinterpret_cast<const uint4*>(dout + idx * DH + 8 * sub);
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int k = 0; k < 4; ++k)
      s += bf2f(aw[k] & 0xffff) * bf2f(bw[k] & 0xffff) + bf2f(aw[k] >> 16) * bf2f(bw[k] >> 16);
  }
#pragma unroll
  for (int off = G / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (idx < n_pairs && sub == 0) {
    const int64_t row = idx / H, bb = row / Tn, t = row % Tn;
    const int h = static_cast<int>(idx % H);
    delta[(bb * H + h) * Tn + t] = s;
  }
}

// ------------------------------------------------------ backward: dK, dV
template <typename T, int DH, int W>
__global__ void __launch_bounds__(64 * W) attn_bwd_dkdv_kernel(const T* __restrict__ qkv,
                                                               const T* __restrict__ dout,
                                                               const float* __restrict__ lse,
                                                               const float* __restrict__ delta,
                                                               T* __restrict__ dqkv, int B, int Tn, int H) {
  using L = ALay<T, DH>;
  constexpr int NT = 64 * W;
  constexpr int STAGE = 2 * (L::ROWS_BYTES + L::TRANS_BYTES);
  constexpr int NBUF = two_stages(STAGE) ? 2 : 1;
  constexpr int BKEYS = 16 * W;
  __shared__ __attribute__((aligned(16))) T Qs[NBUF][BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Qt[NBUF][DH * L::TP];
  __shared__ __attribute__((aligned(16))) T Os[NBUF][BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Ot[NBUF][DH * L::TP];
  __shared__ float lse_s[NBUF][BT], del_s[NBUF][BT];

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
  const int k0 = blockIdx.x * BKEYS;
  const int kw = k0 + w * 16;  // this wave's first key
  const int kj = kw + lr;      // this lane's key
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

  TileLoader<T, DH, NT, false> lq, lo;
  TileLoader<T, DH, NT, true> lqt, lot;
  const int qt0 = k0 / BT, n_qt = (Tn + BT - 1) / BT;
  float pre_lse = 0.f, pre_del = 0.f;
  auto load_tile = [&](int i0) {
    lq.load(qb, ld, i0, Tn, tid);
    lqt.load(qb, ld, i0, Tn, tid);
    lo.load(ob, d, i0, Tn, tid);
    lot.load(ob, d, i0, Tn, tid);
    if (tid < BT) {
      const int i = i0 + tid;
      pre_lse = i < Tn ? lse_b[i] * LOG2E : INFINITY;
      pre_del = i < Tn ? del_b[i] : 0.f;
    }
  };
  auto store_tile = [&](int buf) {
    lq.store(Qs[buf], tid);
    lqt.store(Qt[buf], tid);
    lo.store(Os[buf], tid);
    lot.store(Ot[buf], tid);
    if (tid < BT) {
      lse_s[buf][tid] = pre_lse;
      del_s[buf][tid] = pre_del;
    }
  };
  if (qt0 < n_qt) {
    load_tile(qt0 * BT);
    store_tile(0);
  }
  __syncthreads();

  for (int qt = qt0; qt < n_qt; ++qt) {
    const int i0 = qt * BT;
    const int cur = NBUF == 2 ? ((qt - qt0) & 1) : 0;
    const bool more = qt + 1 < n_qt;
    if (NBUF == 2 && more) load_tile(i0 + BT);
    if (i0 + BT - 1 >= kw && kw < Tn) {  // some query of the tile sees some key of this wave
      const T* qs = Qs[cur];
      const T* os = Os[cur];
      const bool edge = i0 < kw + 15;  // diagonal tile: mask
      float p[4][4], ds[4][4];
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        f32x4_t sa = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < L::NS; ++s) {
          Frag<T> qf, of;
          frag_load(qf, qs + (it * 16 + lr) * L::RP + 32 * s + 8 * lg);
          frag_load(of, os + (it * 16 + lr) * L::RP + 32 * s + 8 * lg);
          mfma16(sa, qf, kf[s]);  // S[i][j]: lane holds key kj, queries 4lg + r
          mfma16(dp, of, vf[s]);  // dP[i][j]
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int il = it * 16 + 4 * lg + r;
          const int i = i0 + il;
          const bool vis = !edge || (kj <= i);
          const float pv = (vis && kj < Tn) ? ex2(sa[r] * sc - lse_s[cur][il]) : 0.f;
          p[it][r] = pv;
          ds[it][r] = pv * (dp[r] - del_s[cur][il]);
        }
      }
      const T* ot = Ot[cur];
      const T* qtt = Qt[cur];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        Frag<T> pf, dsf;
        frag_from_pair(pf, p, s2);
        frag_from_pair(dsf, ds, s2);
#pragma unroll
        for (int c = 0; c < L::NCT; ++c) {
          Frag<T> of2, qf2;
          frag_pair_rows<T, DH>(of2, ot, c * 16 + lr, s2, lg);
          frag_pair_rows<T, DH>(qf2, qtt, c * 16 + lr, s2, lg);
          mfma16(acc_dv[c], of2, pf);   // dV^T[c][j]
          mfma16(acc_dk[c], qf2, dsf);  // dK^T[c][j]
        }
      }
    }
    if (more) {
      if (NBUF == 1) {
        __syncthreads();
        load_tile(i0 + BT);
      }
      store_tile(NBUF == 2 ? (cur ^ 1) : 0);
    }
    __syncthreads();
  }

  if (kj < Tn) {
    const float scale = 1.f / sqrtf(static_cast<float>(DH));
    T* row = dqkv + (static_cast<int64_t>(b) * Tn + kj) * ld + h * DH;
#pragma unroll
    for (int c = 0; c < L::NCT; ++c) {
      float vk[4] = {acc_dk[c][0] * scale, acc_dk[c][1] * scale, acc_dk[c][2] * scale, acc_dk[c][3] * scale};
      float vv[4] = {acc_dv[c][0], acc_dv[c][1], acc_dv[c][2], acc_dv[c][3]};
      store_row4<T>(row + d + c * 16 + 4 * lg, vk);
      store_row4<T>(row + 2 * d + c * 16 + 4 * lg, vv);
    }
  }
}

// ----------------------------------------------------------- backward: dQ
template <typename T, int DH, int G, int NW>
__global__ void __launch_bounds__(64 * NW, ATOM_ATTN_DQ_OCC) attn_bwd_dq_kernel(const T* __restrict__ qkv, const T* __restrict__ dout,
                                                          const float* __restrict__ lse,
                                                          const float* __restrict__ delta, T* __restrict__ dqkv,
                                                          int B, int Tn, int H) {
  using L = ALay<T, DH>;
  constexpr int STAGE = 2 * L::ROWS_BYTES + L::TRANS_BYTES;
  constexpr int NBUF = two_stages(STAGE) ? 2 : 1;
  constexpr int BQ = NW * 16 * G;
  constexpr int NT = 64 * NW;
  __shared__ __attribute__((aligned(16))) T Ks[NBUF][BT * L::RP];
  __shared__ __attribute__((aligned(16))) T Kt[NBUF][DH * L::TP];
  __shared__ __attribute__((aligned(16))) T Vs[NBUF][BT * L::RP];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const T* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const T* kb = qb + d;
  const T* vb = qb + 2 * d;
  const T* ob = dout + static_cast<int64_t>(b) * Tn * d + h * DH;
  const int q0 = blockIdx.x * BQ;
  const int qw = q0 + w * 16 * G;
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));

  Frag<T> qf[G][L::NS], of[G][L::NS];
  float lse_i[G], del_i[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int qi = qw + g * 16 + lr;
    lse_i[g] = qi < Tn ? lse[(static_cast<int64_t>(b) * H + h) * Tn + qi] * LOG2E : INFINITY;
    del_i[g] = qi < Tn ? delta[(static_cast<int64_t>(b) * H + h) * Tn + qi] : 0.f;
#pragma unroll
    for (int s = 0; s < L::NS; ++s) {
      frag_global(qf[g][s], qb, ld, qi, Tn, 32 * s + 8 * lg);
      frag_global(of[g][s], ob, d, qi, Tn, 32 * s + 8 * lg);
    }
  }
  f32x4_t acc_dq[G][L::NCT];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int c = 0; c < L::NCT; ++c) acc_dq[g][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  TileLoader<T, DH, NT, false> lk, lv;
  TileLoader<T, DH, NT, true> lkt;
  const int n_kt = min((Tn + BT - 1) / BT, (min(q0 + BQ, Tn) - 1) / BT + 1);
  lk.load(kb, ld, 0, Tn, tid);
  lkt.load(kb, ld, 0, Tn, tid);
  lv.load(vb, ld, 0, Tn, tid);
  lk.store(Ks[0], tid);
  lkt.store(Kt[0], tid);
  lv.store(Vs[0], tid);
  __syncthreads();

  for (int kt = 0; kt < n_kt; ++kt) {
    const int j0 = kt * BT;
    const int cur = NBUF == 2 ? (kt & 1) : 0;
    const bool more = kt + 1 < n_kt;
    if (NBUF == 2 && more) {
      lk.load(kb, ld, j0 + BT, Tn, tid);
      lkt.load(kb, ld, j0 + BT, Tn, tid);
      lv.load(vb, ld, j0 + BT, Tn, tid);
    }
    if (j0 <= qw + 16 * G - 1) {
      const T* ks = Ks[cur];
      const T* vs = Vs[cur];
      const bool edge = j0 + BT > qw || j0 + BT > Tn;
      float ds[G][4][4];
#pragma unroll
      for (int jt = 0; jt < 4; ++jt) {
        f32x4_t sa[G], dp[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
          sa[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
          dp[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int s = 0; s < L::NS; ++s) {
          Frag<T> kf, vf;
          frag_load(kf, ks + (jt * 16 + lr) * L::RP + 32 * s + 8 * lg);
          frag_load(vf, vs + (jt * 16 + lr) * L::RP + 32 * s + 8 * lg);
#pragma unroll
          for (int g = 0; g < G; ++g) {
            mfma16(sa[g], kf, qf[g][s]);  // S^T[j][i]: lane holds one query, keys 4lg + r
            mfma16(dp[g], vf, of[g][s]);  // dP^T[j][i]
          }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const int qi = qw + g * 16 + lr;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int j = j0 + jt * 16 + 4 * lg + r;
            const bool vis = !edge || (j <= qi && j < Tn);
            const float pv = vis ? ex2(sa[g][r] * sc - lse_i[g]) : 0.f;
            ds[g][jt][r] = pv * (dp[g][r] - del_i[g]);
          }
        }
      }
      const T* kt_s = Kt[cur];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        Frag<T> dsf[G];
#pragma unroll
        for (int g = 0; g < G; ++g) frag_from_pair(dsf[g], ds[g], s2);
#pragma unroll
        for (int c = 0; c < L::NCT; ++c) {
          Frag<T> kf2;
          frag_pair_rows<T, DH>(kf2, kt_s, c * 16 + lr, s2, lg);
#pragma unroll
          for (int g = 0; g < G; ++g) mfma16(acc_dq[g][c], kf2, dsf[g]);  // dQ^T[c][i]
        }
      }
    }
    if (more) {
      if (NBUF == 1) {
        __syncthreads();
        lk.load(kb, ld, j0 + BT, Tn, tid);
        lkt.load(kb, ld, j0 + BT, Tn, tid);
        lv.load(vb, ld, j0 + BT, Tn, tid);
      }
      lk.store(Ks[NBUF == 2 ? (cur ^ 1) : 0], tid);
      lkt.store(Kt[NBUF == 2 ? (cur ^ 1) : 0], tid);
      lv.store(Vs[NBUF == 2 ? (cur ^ 1) : 0], tid);
    }
    __syncthreads();
  }

  const float scale = 1.f / sqrtf(static_cast<float>(DH));
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int qi = qw + g * 16 + lr;
    if (qi < Tn) {
      T* row = dqkv + (static_cast<int64_t>(b) * Tn + qi) * ld + h * DH;
#pragma unroll
      for (int c = 0; c < L::NCT; ++c) {
        float v[4] = {acc_dq[g][c][0] * scale, acc_dq[g][c][1] * scale, acc_dq[g][c][2] * scale,
                      acc_dq[g][c][3] * scale};
        store_row4<T>(row + c * 16 + 4 * lg, v);
      }
    }
  }
}

// ----------------------------------------- backward: dK, dV, bf16, direct loads
// Q and dO tiles (natural layout) by direct loads, two stages; both are read
// as row fragments (S = Q K^T, dP = dO V^T) and transposed in pair order
// (dK^T += Q^T dS, dV^T += dO^T P), so both use the two-way swizzle dsw.
// The rows' LSE and D go through registers into small per-stage arrays.
template <int DH>
__device__ __forceinline__ int dsw(int r);

// Launch bounds of both backward kernels: at d_h 64 four waves per SIMD (108
// registers; two eight-wave workgroups per CU: 264 against 291 us for the
// whole backward at GPT-3 Small's shape), at d_h 128 two (244 and 174
// registers, one workgroup per CU; 128 registers would spill).
template <int DH, int W>
__global__ void __launch_bounds__(64 * W, DH == 64 ? 4 : 2) attn_bwd_dkdv_dl_kernel(const bf16_t* __restrict__ qkv,
                                                                  const bf16_t* __restrict__ dout,
                                                                  const float* __restrict__ lse,
                                                                  const float* __restrict__ delta,
                                                                  bf16_t* __restrict__ dqkv, int B, int Tn, int H) {
  using F = FwdDL<DH>;
  constexpr int NS = DH / 32, NCT = DH / 16, NT = 64 * W, RB = DH * 2, BKEYS = 16 * W;
  constexpr int LPT = F::TILE / (NT * 16);
  static_assert(LPT >= 1 && F::TILE % (NT * 16) == 0, "tile split");
  constexpr int STAGE = 2 * F::TILE + 2 * BT * 4;  // Q, dO, LSE (log2 units), D of one 64-query tile
  // Two query tiles per pipeline stage, so one barrier per 128 queries: the
  // wave's work between barriers doubles (373 against 377 us for the whole
  // backward at the 6.7B shape, 262 against 273 at d_h 64); the loop over
  // the two stays rolled (unrolled, 40 bytes spill at d_h 128)
  constexpr int SUB = 2;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * SUB * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const BlockId blk = attn_block(false);  // key block x sees the queries from x on
  const int bh = blk.bh, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const bf16_t* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const bf16_t* kb = qb + d;
  const bf16_t* vb = qb + 2 * d;
  const bf16_t* ob = dout + static_cast<int64_t>(b) * Tn * d + h * DH;  // dO, row stride d
  const float* lse_b = lse + (static_cast<int64_t>(b) * H + h) * Tn;
  const float* del_b = delta + (static_cast<int64_t>(b) * H + h) * Tn;
  const int k0 = blk.x * BKEYS;
  const int kw = k0 + w * 16;  // this wave's first key
  const int kj = kw + lr;      // this lane's key
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));

  Frag<bf16_t> kf[NS], vf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    frag_global(kf[s], kb, ld, kj, Tn, 32 * s + 8 * lg);
    frag_global(vf[s], vb, ld, kj, Tn, 32 * s + 8 * lg);
  }
  f32x4_t acc_dk[NCT], acc_dv[NCT];
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    acc_dk[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc_dv[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  auto load_tile = [&](int st, int i0) {
    const uint32_t ql = lds_offset(lds + st * STAGE), ol = ql + F::TILE;
#pragma unroll
    for (int q = 0; q < LPT; ++q) {
      const int id = q * NT + tid, row = id / F::CPR, slot = id % F::CPR;
      const int r = min(i0 + row, Tn - 1);
      const uint32_t lo = __builtin_amdgcn_readfirstlane((q * NT + w * 64) * 16);
      lds_dma16(qb + static_cast<int64_t>(r) * ld + (slot ^ dsw<DH>(row)) * 8, ql + lo);
      lds_dma16(ob + static_cast<int64_t>(r) * d + (slot ^ dsw<DH>(row)) * 8, ol + lo);
    }
  };
  // LSE and D of a tile's rows: read into registers, stored to LDS after the
  // tile's compute (rows past the end get LSE = +inf, so their P is 0)
  float pre_lse = 0.f, pre_del = 0.f;
  // (thread tid < SUB*BT reads row tid % BT of sub-tile tid / BT)
  auto read_rows = [&](int i0) {
    if (tid < SUB * BT) {
      const int i = i0 + tid;
      pre_lse = i < Tn ? lse_b[i] * LOG2E : INFINITY;
      pre_del = i < Tn ? del_b[i] : 0.f;
    }
  };
  auto store_rows = [&](int st) {
    if (tid < SUB * BT) {
      float* rows = reinterpret_cast<float*>(lds + (st * SUB + tid / BT) * STAGE + 2 * F::TILE);
      rows[tid % BT] = pre_lse;
      rows[BT + tid % BT] = pre_del;
    }
  };
  auto rowfrag = [&](Frag<bf16_t>& f, const uint8_t* st, int it, int s) {
    const int row = it * 16 + lr, chunk = 4 * s + lg;
    f.v = *reinterpret_cast<const uint4*>(st + row * RB + (chunk ^ dsw<DH>(row)) * 16);
  };
  auto trfrag = [&](Frag<bf16_t>& f, const uint8_t* st, int s2, int c) {
    const int chunk = 2 * c + ((lr & 3) >> 1);
    const int r0 = 32 * s2 + 4 * lg + (lr >> 2), r1 = r0 + 16;
    const uint2 lo = ds_read_tr8(st + r0 * RB + (chunk ^ dsw<DH>(r0)) * 16 + 8 * (lr & 1));
    const uint2 hi = ds_read_tr8(st + r1 * RB + (chunk ^ dsw<DH>(r1)) * 16 + 8 * (lr & 1));
    f.v = make_uint4(lo.x, lo.y, hi.x, hi.y);
  };

  const int qt0 = k0 / BT, n_qt = (Tn + BT - 1) / BT;
  const bool tail_keys = kw + 16 > Tn;  // some of this wave's keys are past the end
  // the SUB tiles from query tile qt into stage st (tiles past the end are skipped)
  auto load_stage = [&](int st, int qt) {
#pragma unroll
    for (int u = 0; u < SUB; ++u)
      if (qt + u < n_qt) load_tile(st * SUB + u, (qt + u) * BT);
  };
  if (qt0 < n_qt) {
    load_stage(0, qt0);
    read_rows(qt0 * BT);
    store_rows(0);
  }
  for (int qs0 = qt0; qs0 < n_qt; qs0 += SUB) {
    const int cur = ((qs0 - qt0) / SUB) & 1;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    asm volatile("s_barrier" ::: "memory");
    const bool more = qs0 + SUB < n_qt;
    if (more) {
      load_stage(cur ^ 1, qs0 + SUB);
      read_rows((qs0 + SUB) * BT);
    }
#pragma unroll 1
    for (int u = 0; u < SUB; ++u) {
      const int qt = qs0 + u, i0 = qt * BT, stg = cur * SUB + u;
      if (qt >= n_qt) break;
      if (i0 + BT - 1 >= kw && kw < Tn) {  // some query of the tile sees some key of this wave
        const uint8_t* qs = lds + stg * STAGE;
        const uint8_t* os = qs + F::TILE;
        const float* lse_s = reinterpret_cast<const float*>(qs + 2 * F::TILE);
        const float* del_s = lse_s + BT;
        float p[4][4], ds[4][4];
        const bool mask = i0 < kw + 15 || tail_keys;  // diagonal tile or keys past the end
        if constexpr (DH == 128) {
          // One branch-free block per tile (the mask a template parameter), so
          // the exponentials of 16 queries overlap the next 16 queries' MFMAs;
          // LDS reads stay in their 16-query step (sched_barrier lets only VALU
          // and MFMA cross), else the scheduler hoists every step's fragments
          // and spills (380 against 393 us for the backward at the 6.7B shape).
          auto score_tile = [&](auto MASK_) {
            constexpr bool MASK = decltype(MASK_)::value;
#pragma unroll
            for (int it = 0; it < 4; ++it) {
              Frag<bf16_t> qf[NS], of[NS];
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                rowfrag(qf[s], qs, it, s);
                rowfrag(of[s], os, it, s);
              }
              f32x4_t sa = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                mfma16(sa, qf[s], kf[s]);  // S[i][j]: lane holds key kj, queries 4lg + r
                mfma16(dp, of[s], vf[s]);  // dP[i][j]
              }
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int il = it * 16 + 4 * lg + r;
                float pv = ex2(__builtin_fmaf(sa[r], sc, -lse_s[il]));
                if constexpr (MASK) pv = ((kj <= i0 + il) & (kj < Tn)) ? pv : 0.f;
                p[it][r] = pv;
                ds[it][r] = pv * (dp[r] - del_s[il]);
              }
              __builtin_amdgcn_sched_barrier(0x000A);
            }
          };
          if (mask) score_tile(std::true_type{});
          else score_tile(std::false_type{});
        } else {
          // d_h 64: fragments one step ahead and the mask a runtime test (the
          // branch-free form spills within the 128 registers of four waves per SIMD)
          Frag<bf16_t> qf[2][NS], of[2][NS];
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            rowfrag(qf[0][s], qs, 0, s);
            rowfrag(of[0][s], os, 0, s);
          }
#pragma unroll
          for (int it = 0; it < 4; ++it) {
            if (it + 1 < 4) {
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                rowfrag(qf[(it + 1) & 1][s], qs, it + 1, s);
                rowfrag(of[(it + 1) & 1][s], os, it + 1, s);
              }
            }
            f32x4_t sa = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < NS; ++s) {
              mfma16(sa, qf[it & 1][s], kf[s]);
              mfma16(dp, of[it & 1][s], vf[s]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int il = it * 16 + 4 * lg + r;
              float pv = ex2(__builtin_fmaf(sa[r], sc, -lse_s[il]));
              if (mask) pv = ((kj <= i0 + il) & (kj < Tn)) ? pv : 0.f;
              p[it][r] = pv;
              ds[it][r] = pv * (dp[r] - del_s[il]);
            }
          }
        }
        Frag<bf16_t> ot2[2], qt2[2];
        trfrag(ot2[0], os, 0, 0);
        trfrag(qt2[0], qs, 0, 0);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          Frag<bf16_t> pf, dsf;
          frag_from_pair(pf, p, s2);
          frag_from_pair(dsf, ds, s2);
#pragma unroll
          for (int c = 0; c < NCT; ++c) {
            const int n = s2 * NCT + c;
            if (n + 1 < 2 * NCT) {
              trfrag(ot2[(n + 1) & 1], os, (n + 1) / NCT, (n + 1) % NCT);
              trfrag(qt2[(n + 1) & 1], qs, (n + 1) / NCT, (n + 1) % NCT);
            }
            mfma16(acc_dv[c], ot2[n & 1], pf);   // dV^T[c][j]
            mfma16(acc_dk[c], qt2[n & 1], dsf);  // dK^T[c][j]
          }
        }
      }
    }
    if (more) store_rows(cur ^ 1);
  }

  if (kj < Tn) {
    const float scale = 1.f / sqrtf(static_cast<float>(DH));
    bf16_t* row = dqkv + (static_cast<int64_t>(b) * Tn + kj) * ld + h * DH;
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      float vk[4] = {acc_dk[c][0] * scale, acc_dk[c][1] * scale, acc_dk[c][2] * scale, acc_dk[c][3] * scale};
      float vv[4] = {acc_dv[c][0], acc_dv[c][1], acc_dv[c][2], acc_dv[c][3]};
      store_row4<bf16_t>(row + d + c * 16 + 4 * lg, vk);
      store_row4<bf16_t>(row + 2 * d + c * 16 + 4 * lg, vv);
    }
  }
}

// -------------------------------------------- backward: dQ, bf16, direct loads
// K and V tiles by direct loads, two stages (as in the forward).  K is read
// both ways, as row fragments for S^T = K Q^T and transposed (pair order)
// for dQ^T += K^T dS^T, so its slots use one swizzle that serves both access
// patterns: dsw(r) = 2 (r & 7) for 16-chunk rows, 2 ((r >> 1) & 3) for
// 8-chunk rows, the transposed reads' swizzle of the forward's V.  Measured
// with the bank-conflict counter on both read forms at both widths: these
// leave ds_read_b128 of 16 rows at one chunk conflict-free (4 LDS cycles per
// instruction) as well as the transposed reads (2 cycles); flipping the low
// bit for rows 8-15 too, so that 16 consecutive rows take 16 distinct
// chunks, makes ds_read_b128 take 8 cycles (dK/dV 171 -> 162 us at the 6.7B
// shape without it).
template <int DH>
__device__ __forceinline__ int dsw(int r) {
  return DH == 128 ? 2 * (r & 7) : 2 * ((r >> 1) & 3);
}

template <int DH, int NW>
__global__ void __launch_bounds__(64 * NW, DH == 64 ? 4 : 2) attn_bwd_dq_dl_kernel(const bf16_t* __restrict__ qkv,
                                                                const bf16_t* __restrict__ dout,
                                                                const float* __restrict__ lse,
                                                                const float* __restrict__ delta,
                                                                bf16_t* __restrict__ dqkv, int B, int Tn, int H) {
  using F = FwdDL<DH>;
  constexpr int NS = DH / 32, NCT = DH / 16, BQ = NW * 16, NT = 64 * NW, RB = DH * 2;
  constexpr int LPT = F::TILE / (NT * 16);  // direct loads per thread per tile and operand
  static_assert(LPT >= 1 && F::TILE % (NT * 16) == 0, "tile split");
  // Two key tiles per pipeline stage, one barrier per 128 keys (at d_h 64
  // 254-260 against 272 us for the whole backward at GPT-3 Small's shape;
  // unchanged at d_h 128, where one workgroup per CU leaves the LDS for it)
  constexpr int SUB = 2;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * SUB * F::STAGE];

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const BlockId blk = attn_block(true);
  const int bh = blk.bh, b = bh / H, h = bh % H;
  const int d = H * DH;
  const int64_t ld = 3 * static_cast<int64_t>(d);
  const bf16_t* qb = qkv + static_cast<int64_t>(b) * Tn * ld + h * DH;
  const bf16_t* kb = qb + d;
  const bf16_t* vb = qb + 2 * d;
  const bf16_t* ob = dout + static_cast<int64_t>(b) * Tn * d + h * DH;
  const int q0 = blk.x * BQ;
  const int qw = q0 + w * 16;
  const int qi = qw + lr;
  const float sc = LOG2E / sqrtf(static_cast<float>(DH));

  Frag<bf16_t> qf[NS], of[NS];
  const float lse_i = qi < Tn ? lse[(static_cast<int64_t>(b) * H + h) * Tn + qi] * LOG2E : INFINITY;
  const float del_i = qi < Tn ? delta[(static_cast<int64_t>(b) * H + h) * Tn + qi] : 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    frag_global(qf[s], qb, ld, qi, Tn, 32 * s + 8 * lg);
    frag_global(of[s], ob, d, qi, Tn, 32 * s + 8 * lg);
  }
  f32x4_t acc_dq[NCT];
#pragma unroll
  for (int c = 0; c < NCT; ++c) acc_dq[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  auto load_tile = [&](int st, int j0) {
    const uint32_t kl = lds_offset(lds + st * F::STAGE), vl = kl + F::TILE;
#pragma unroll
    for (int q = 0; q < LPT; ++q) {
      const int id = q * NT + tid, row = id / F::CPR, slot = id % F::CPR;
      const int64_t gr = static_cast<int64_t>(min(j0 + row, Tn - 1)) * ld;
      const uint32_t lo = __builtin_amdgcn_readfirstlane((q * NT + w * 64) * 16);
      lds_dma16(kb + gr + (slot ^ dsw<DH>(row)) * 8, kl + lo);
      lds_dma16(vb + gr + (slot ^ F::kswz(row)) * 8, vl + lo);
    }
  };
  auto rowfrag = [&](Frag<bf16_t>& f, const uint8_t* st, int jt, int s, bool dual) {
    const int row = jt * 16 + lr, chunk = 4 * s + lg;
    f.v = *reinterpret_cast<const uint4*>(st + row * RB + (chunk ^ (dual ? dsw<DH>(row) : F::kswz(row))) * 16);
  };
  auto trfrag = [&](Frag<bf16_t>& f, const uint8_t* st, int s2, int c) {
    const int chunk = 2 * c + ((lr & 3) >> 1);
    const int r0 = 32 * s2 + 4 * lg + (lr >> 2), r1 = r0 + 16;
    const uint2 lo = ds_read_tr8(st + r0 * RB + (chunk ^ dsw<DH>(r0)) * 16 + 8 * (lr & 1));
    const uint2 hi = ds_read_tr8(st + r1 * RB + (chunk ^ dsw<DH>(r1)) * 16 + 8 * (lr & 1));
    f.v = make_uint4(lo.x, lo.y, hi.x, hi.y);
  };

  const int n_kt = min((Tn + BT - 1) / BT, (min(q0 + BQ, Tn) - 1) / BT + 1);
  // the SUB key tiles from tile kt into stage st (tiles past the last are skipped)
  auto load_stage = [&](int st, int kt) {
#pragma unroll
    for (int u = 0; u < SUB; ++u)
      if (kt + u < n_kt) load_tile(st * SUB + u, (kt + u) * BT);
  };
  load_stage(0, 0);
  for (int ks0 = 0; ks0 < n_kt; ks0 += SUB) {
    const int cur = (ks0 / SUB) & 1;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    asm volatile("s_barrier" ::: "memory");
    if (ks0 + SUB < n_kt) load_stage(cur ^ 1, ks0 + SUB);
#pragma unroll 1
    for (int u = 0; u < SUB; ++u) {
      const int kt = ks0 + u, j0 = kt * BT, stg = cur * SUB + u;
      if (kt >= n_kt) break;
      if (j0 <= qw + 15) {
        const uint8_t* ks = lds + stg * F::STAGE;
        const uint8_t* vs = ks + F::TILE;
        float ds[4][4];
        // one branch-free block per tile (the mask a template parameter)
        auto score_tile = [&](auto MASK_) {
          constexpr bool MASK = decltype(MASK_)::value;
          Frag<bf16_t> kf[2][NS], vf[2][NS];
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            rowfrag(kf[0][s], ks, 0, s, true);
            rowfrag(vf[0][s], vs, 0, s, false);
          }
#pragma unroll
          for (int jt = 0; jt < 4; ++jt) {
            if (jt + 1 < 4) {
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                rowfrag(kf[(jt + 1) & 1][s], ks, jt + 1, s, true);
                rowfrag(vf[(jt + 1) & 1][s], vs, jt + 1, s, false);
              }
            }
            f32x4_t sa = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < NS; ++s) {
              mfma16(sa, kf[jt & 1][s], qf[s]);  // S^T[j][i]: lane holds one query, keys 4lg + r
              mfma16(dp, vf[jt & 1][s], of[s]);  // dP^T[j][i]
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int j = j0 + jt * 16 + 4 * lg + r;
              float pv = ex2(__builtin_fmaf(sa[r], sc, -lse_i));
              if constexpr (MASK) pv = ((j <= qi) & (j < Tn)) ? pv : 0.f;
              ds[jt][r] = pv * (dp[r] - del_i);
            }
          }
        };
        if (j0 + BT > qw || j0 + BT > Tn) score_tile(std::true_type{});
        else score_tile(std::false_type{});
        Frag<bf16_t> kt2[2];
        trfrag(kt2[0], ks, 0, 0);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          Frag<bf16_t> dsf;
          frag_from_pair(dsf, ds, s2);
#pragma unroll
          for (int c = 0; c < NCT; ++c) {
            const int n = s2 * NCT + c;
            if (n + 1 < 2 * NCT) trfrag(kt2[(n + 1) & 1], ks, (n + 1) / NCT, (n + 1) % NCT);
            mfma16(acc_dq[c], kt2[n & 1], dsf);  // dQ^T[c][i]
          }
        }
      }
    }
  }

  if (qi < Tn) {
    const float scale = 1.f / sqrtf(static_cast<float>(DH));
    bf16_t* row = dqkv + (static_cast<int64_t>(b) * Tn + qi) * ld + h * DH;
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      float v[4] = {acc_dq[c][0] * scale, acc_dq[c][1] * scale, acc_dq[c][2] * scale, acc_dq[c][3] * scale};
      store_row4<bf16_t>(row + c * 16 + 4 * lg, v);
    }
  }
}

// Query groups per wave in the forward (G), waves per dK/dV workgroup (W),
// and query groups (GQ) and waves (WQ) of the dQ kernel; bf16 takes the
// direct-load kernels, fp32 the register-staged ones.  dQ: eight waves of 16
// queries (two waves per SIMD within the register file) beat four waves of 32
// queries (one wave per SIMD): 1.14x.  The bf16 forward at d_h 128 takes
// ATOM_FWD_G128 groups per wave in workgroups of ATOM_FWD_NW128 waves (one
// group, eight waves: see attn_fwd_dl_kernel), at d_h 64 two groups in four.
#ifndef ATOM_FWD_G128
#define ATOM_FWD_G128 1
#endif
#ifndef ATOM_FWD_NW128
#define ATOM_FWD_NW128 8
#endif
template <typename T, int DH>
struct ACfg {
  static constexpr int G = sizeof(T) == 2 ? 2 : 1;
  static constexpr int W = sizeof(T) == 2 ? 8 : 4;
  static constexpr int GQ = 1;
  static constexpr int WQ = sizeof(T) == 2 ? 8 : 4;
};

template <typename T, int DH>
hipError_t fwd_t(const void* qkv, void* o, float* lse, int B, int Tn, int H, hipStream_t s) {
  constexpr int G = ACfg<T, DH>::G;
  if constexpr (sizeof(T) == 2) {
    constexpr int FG = DH == 128 ? ATOM_FWD_G128 : 2, FNW = DH == 128 ? ATOM_FWD_NW128 : 4;
    dim3 grid((Tn + 16 * FG * FNW - 1) / (16 * FG * FNW), B * H), block(64 * FNW);
    hipLaunchKernelGGL((attn_fwd_dl_kernel<DH, FG, FNW>), grid, block, 0, s, static_cast<const bf16_t*>(qkv),
                       static_cast<bf16_t*>(o), lse, B, Tn, H);
  } else {
    dim3 grid((Tn + 64 * G - 1) / (64 * G), B * H), block(256);
    hipLaunchKernelGGL((attn_fwd_kernel<T, DH, G>), grid, block, 0, s, static_cast<const T*>(qkv), static_cast<T*>(o),
                       lse, B, Tn, H);
  }
  return hipGetLastError();
}

template <typename T, int DH>
hipError_t bwd_t(const void* qkv, const void* o, const void* dout, const float* lse, float* delta, void* dqkv, int B,
                 int Tn, int H, hipStream_t s) {
  constexpr int W = ACfg<T, DH>::W;
  const int64_t n_rows = static_cast<int64_t>(B) * Tn;
  if constexpr (sizeof(T) == 2)
    hipLaunchKernelGGL(attn_delta_bf16_kernel<DH>, dim3(static_cast<unsigned>((n_rows * H * (DH / 8) + 255) / 256)),
                       dim3(256), 0, s, static_cast<const bf16_t*>(o), static_cast<const bf16_t*>(dout), delta,
                       n_rows * H, Tn, H);
  else
    hipLaunchKernelGGL(attn_delta_kernel<T>, dim3(static_cast<unsigned>((n_rows * H + 3) / 4)), dim3(256), 0, s,
                       static_cast<const T*>(o), static_cast<const T*>(dout), delta, n_rows, Tn, H, DH);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if constexpr (sizeof(T) == 2)
    hipLaunchKernelGGL((attn_bwd_dkdv_dl_kernel<DH, W>), dim3((Tn + 16 * W - 1) / (16 * W), B * H), dim3(64 * W), 0,
                       s, static_cast<const bf16_t*>(qkv), static_cast<const bf16_t*>(dout), lse, delta,
                       static_cast<bf16_t*>(dqkv), B, Tn, H);
  else
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, DH, W>), dim3((Tn + 16 * W - 1) / (16 * W), B * H), dim3(64 * W), 0,
                       s, static_cast<const T*>(qkv), static_cast<const T*>(dout), lse, delta, static_cast<T*>(dqkv),
                       B, Tn, H);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  constexpr int GQ = ACfg<T, DH>::GQ, WQ = ACfg<T, DH>::WQ;
  if constexpr (sizeof(T) == 2)
    hipLaunchKernelGGL((attn_bwd_dq_dl_kernel<DH, WQ>), dim3((Tn + 16 * WQ - 1) / (16 * WQ), B * H), dim3(64 * WQ), 0,
                       s, static_cast<const bf16_t*>(qkv), static_cast<const bf16_t*>(dout), lse, delta,
                       static_cast<bf16_t*>(dqkv), B, Tn, H);
  else
    hipLaunchKernelGGL((attn_bwd_dq_kernel<T, DH, GQ, WQ>), dim3((Tn + 16 * WQ * GQ - 1) / (16 * WQ * GQ), B * H),
                       dim3(64 * WQ), 0, s, static_cast<const T*>(qkv), static_cast<const T*>(dout), lse, delta,
                       static_cast<T*>(dqkv), B, Tn, H);
  return hipGetLastError();
}

}  // namespace attn
}  // namespace atom
