// Internal launchers of the libatom kernels (host side).  Every launcher only
// enqueues work on the given stream and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace atom {

enum { DT_F32 = 0, DT_BF16 = 1 };

enum Epilogue {
  EPI_STORE = 0,       // C = acc                          (element type)
  EPI_STORE_F32 = 1,   // C = acc                          (fp32)
  EPI_ACC_F32 = 2,     // C += acc                         (fp32)
  EPI_BIAS = 3,        // C = acc + bias[n]                (element type)
  EPI_BIAS_GELU = 4,   // aux = acc + bias[n]; C = GELU(aux)
  EPI_BIAS_RESID = 5,  // C = resid + (acc + bias[n])      (fp32)
  EPI_GELU_BWD = 6,    // C = acc * GELU'(aux)             (element type)
};

struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  const void* bias;
  const float* resid;
  void* aux;
  int64_t lda, ldb, ldc, ldaux;
  int M, N, K;
  float* ws;          // optional fp32 workspace for a split over k (may be null)
  uint64_t ws_bytes;  // its size; a split needs splits * M * N * 4 bytes
};

hipError_t gemm_check(const GemmArgs& g, int dtype, bool a_kcontig, bool b_kcontig);
hipError_t gemm(const GemmArgs& g, int dtype, bool a_kcontig, bool b_kcontig, int epi, hipStream_t s);

// LayerNorm over rows of length d (d % 64 == 0, d <= 8192).
//   y = (x - mean) * rstd * gamma + beta, x fp32, y element type.
hipError_t layernorm_fwd(int dtype, const float* x, const void* gamma, const void* beta, void* y, float* mean,
                         float* rstd, int64_t rows, int d, hipStream_t s);
// dres (+)= LN backward of dy; also writes dres_lp (element-type copy of the
// updated dres, may be null) and per-block partial column sums of dy*xhat and
// dy into part[nblk][2][d] (nblk from layernorm_bwd_blocks).
int64_t layernorm_bwd_blocks(int64_t rows, int d);
hipError_t layernorm_bwd(int dtype, const void* dy, const float* x, const float* mean, const float* rstd,
                         const void* gamma, float* dres, void* dres_lp, bool accumulate, float* part, int64_t rows,
                         int d, hipStream_t s);

// Deterministic column sums of a [rows][cols] matrix in two passes.
int64_t colsum_blocks(int64_t rows);
hipError_t colsum_partial(int in_dtype, const void* x, int64_t rows, int cols, int64_t ld, float* part,
                          hipStream_t s);
// out[j] (op)= sum over nparts of part[p][j] (+ stride between slabs); out
// type: DT_F32 with accumulate flag, or the element type (overwrite).
hipError_t sum_parts(const float* part, int64_t nparts, int cols, int64_t part_stride, int out_dtype, void* out,
                     bool accumulate, hipStream_t s);
// The same with two targets of one dtype and mode in one launch: columns
// c < split go to out[c], the rest to out2[c - split].
hipError_t sum_parts2(const float* part, int64_t nparts, int cols, int64_t part_stride, int out_dtype, void* out,
                      void* out2, int split, bool accumulate, hipStream_t s);

// Embedding: x[n] = wte[tok[n]] + wpe[n % T] (x fp32); ids outside [0, V)
// give NaN rows.
hipError_t embed_fwd(int dtype, const int32_t* tok, const void* wte, const void* wpe, float* x, int64_t n_tok,
                     int T, int V, int d, hipStream_t s);
// dwte rows of the listed unique tokens = sum of dx rows in `perm` order;
// all other rows zero (unless accumulate); dwpe[t] (op)= sum_b dx[b*T + t].
hipError_t embed_bwd(int out_dtype, const float* dx, const int32_t* perm, const int32_t* seg,
                     const int32_t* uniq, int n_uniq, void* dwte, void* dwpe, int V, int T, int B, int d,
                     bool accumulate, hipStream_t s);

// Cross-entropy rows: logits fp32 [rows][ldz] (V valid columns); writes
// dz = (softmax - onehot) * scale in the element type ([rows][lddz], padding
// columns up to lddz zeroed) and loss_rows[r] = logsumexp - z[y].
hipError_t xent_fwd_bwd(int dtype, const float* logits, int64_t ldz, const int32_t* tgt, void* dz, int64_t lddz,
                        float* loss_rows, int64_t rows, int V, float scale, hipStream_t s);

// Sum of n fp32 values in a fixed order, result in out[0] (fp32).
hipError_t sum_fixed(const float* x, int64_t n, float* out, hipStream_t s);

// fp32 -> element type conversion (n elements).
hipError_t convert_f32(int dtype, const float* x, void* y, int64_t n, hipStream_t s);
hipError_t fill_zero(void* p, int64_t bytes, hipStream_t s);
// Working-memory probe: fill `bytes` (a multiple of 16, 16-byte aligned) with
// a 32-bit word; high_water raises *out (a device counter) to 1 + the index of
// the last 16-byte unit that no longer holds it.
hipError_t fill_word(void* p, int64_t bytes, uint32_t word, hipStream_t s);
hipError_t high_water(const void* p, int64_t bytes, uint32_t word, unsigned long long* out, hipStream_t s);
// Streaming device copy of `bytes` (multiple of 16, 16-byte aligned).
hipError_t copy_bytes(const void* src, void* dst, int64_t bytes, hipStream_t s);
// Copy n 32-bit words on stream s by a kernel; src may be mapped pinned host
// memory (small uploads that must not occupy a DMA engine).
hipError_t copy_words(const uint32_t* src, uint32_t* dst, int64_t n, hipStream_t s);
// Makes device memory written by a DMA engine (after the host saw the copy
// complete) visible to the kernels enqueued after it on stream s.
hipError_t dma_acquire(hipStream_t s);

// Causal attention on a fused qkv [B*T][3*d] (element type), heads of dh in
// {64, 128}.  o [B*T][d], lse [B][H][T] fp32 (natural log).
hipError_t attn_fwd(int dtype, const void* qkv, void* o, float* lse, int B, int T, int H, int dh,
                    hipStream_t s);
// Backward: delta [B][H][T] fp32 scratch; dqkv [B*T][3*d].
hipError_t attn_bwd(int dtype, const void* qkv, const void* o, const void* dout, const float* lse, float* delta,
                    void* dqkv, int B, int T, int H, int dh, hipStream_t s);

}  // namespace atom
