/*
 * atom_kernels.h - kernel-level entry points of libatom.
 *
 * The swapped step (atom.h) composes these kernels; they are exported on
 * their own so each can be checked against a reference in isolation.  All
 * pointers are device pointers except where noted; `stream` is a hipStream_t
 * (NULL = the default stream).  Every call only enqueues work and returns
 * ATOM_OK, ATOM_EINVAL (shape, alignment or dtype not supported) or ATOM_EHIP
 * (launch failed).  dtype is ATOM_F32 or ATOM_BF16 (bf16 tensors are raw
 * 16-bit patterns); accumulation is fp32 in every kernel.
 */
#ifndef ATOM_KERNELS_H
#define ATOM_KERNELS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Epilogues of atom_k_gemm. */
enum {
  ATOM_EPI_STORE = 0,       /* C = acc                        (dtype)  */
  ATOM_EPI_STORE_F32 = 1,   /* C = acc                        (fp32)   */
  ATOM_EPI_ACC_F32 = 2,     /* C += acc                       (fp32)   */
  ATOM_EPI_BIAS = 3,        /* C = acc + bias[n]              (dtype)  */
  ATOM_EPI_BIAS_GELU = 4,   /* aux = acc + bias[n]; C = GELU(aux)     */
  ATOM_EPI_BIAS_RESID = 5,  /* C = resid + acc + bias[n]      (fp32)   */
  ATOM_EPI_GELU_BWD = 6     /* C = acc * GELU'(aux)           (dtype)  */
};

/* Matrix product of a linear layer y = x W^T + b and its two gradients
 * (the decoder-block GEMMs of the GPT-3 model, Section III-B).
 *   C[m][n] = sum_k A(m,k) B(k,n), with
 *   A(m,k) = a_kcontig ? A[m*lda + k] : A[k*lda + m],
 *   B(k,n) = b_kcontig ? B[n*ldb + k] : B[k*ldb + n].
 * C, resid, aux are row-major with leading dimensions ldc (resid shares ldc)
 * and ldaux.  Requirements: K % 8 == 0 (bf16) or K % 4 == 0 (fp32); the
 * leading dimension of a k-contiguous operand a multiple of 8 (bf16) or 4
 * (fp32); for bf16 an operand that is not k-contiguous needs an even row
 * count and an even leading dimension; A, B, C 16-byte aligned.
 * ws (fp32, ws_bytes, 16-byte aligned, may be NULL) lets a problem with few
 * output tiles and a long k split k over workgroups for the store epilogues
 * (STORE, STORE_F32, ACC_F32); the partials are summed in a fixed order. */
int atom_k_gemm(int dtype, int a_kcontig, int b_kcontig, int epi, int M, int N, int K, const void* A, int64_t lda,
                const void* B, int64_t ldb, void* C, int64_t ldc, const void* bias, const float* resid, void* aux,
                int64_t ldaux, float* ws, uint64_t ws_bytes, void* stream);

/* LayerNorm forward over rows of d (d % 64 == 0, d <= 8192), eps 1e-5,
 * biased variance: y = (x - mean) * rstd * gamma + beta.  x fp32 [rows][d];
 * y dtype; mean, rstd fp32 [rows]. */
int atom_k_layernorm_fwd(int dtype, const float* x, const void* gamma, const void* beta, void* y, float* mean,
                         float* rstd, int64_t rows, int d, void* stream);

/* Scratch floats atom_k_layernorm_bwd needs in `part`. */
int64_t atom_k_layernorm_bwd_part_floats(int64_t rows, int d);

/* LayerNorm backward: dx = rstd * (g' - mean(g') - xhat * mean(g' xhat)),
 * g' = dy * gamma; dres (fp32) = dx or dres + dx (accumulate); dres_lp
 * (dtype, may be NULL) receives the updated dres rounded; dgamma, dbeta
 * (fp32 [d]) = column sums of dy * xhat and dy (fixed order). */
int atom_k_layernorm_bwd(int dtype, const void* dy, const float* x, const float* mean, const float* rstd,
                         const void* gamma, float* dres, void* dres_lp, int accumulate, float* dgamma, float* dbeta,
                         float* part, int64_t rows, int d, void* stream);

/* Causal self-attention on qkv [B*T][3*d] (q, k, v at column offsets 0, d,
 * 2d; head h at h*dh), dh in {64, 128}, scale 1/sqrt(dh): o [B*T][d] and
 * lse [B][H][T] (natural-log row log-sum-exp of the scaled scores). */
int atom_k_attn_fwd(int dtype, const void* qkv, void* o, float* lse, int B, int T, int H, int dh, void* stream);

/* Its backward: dqkv [B*T][3*d] from dout [B*T][d]; delta is fp32 scratch
 * of [B][H][T]. */
int atom_k_attn_bwd(int dtype, const void* qkv, const void* o, const void* dout, const float* lse, float* delta,
                    void* dqkv, int B, int T, int H, int dh, void* stream);

/* atom_k_attn_bwd for callers that cannot allocate (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): the same kernels,
 * with the D scratch in a library-owned device array of
 * ATOM_ATTN_NOALLOC_MAX_ROWS floats (4 MiB per GPU, held until the process
 * ends) instead of a `delta` argument.  Allocates nothing.  B * H * T above
 * the limit: ATOM_EINVAL.  Every call on one GPU uses the same array, so
 * calls that overlap on one GPU (different streams, or threads) race; calls
 * in order on one stream do not.  Nothing in the array must start at zero. */
#define ATOM_ATTN_NOALLOC_MAX_ROWS (1 << 20)
int atom_k_attn_bwd_noalloc(int dtype, const void* qkv, const void* o, const void* dout, const float* lse,
                            void* dqkv, int B, int T, int H, int dh, void* stream);

/* Scratch floats atom_k_colsum needs in `part`. */
int64_t atom_k_colsum_part_floats(int64_t rows, int cols);

/* out[j] = sum over rows of x[r][j] (x dtype [rows][cols], out fp32),
 * fixed order. */
int atom_k_colsum(int dtype, const void* x, int64_t rows, int cols, float* out, float* part, void* stream);

/* Softmax cross-entropy rows: logits fp32 [rows][ldz] with V valid columns,
 * target ids tgt[rows]; dz = (softmax - onehot) * scale (dtype, row pitch
 * lddz, columns V..lddz-1 zeroed); loss_rows = logsumexp - z[y] (NaN for a
 * target outside [0, V), which is never read). */
int atom_k_xent(int dtype, const float* logits, int64_t ldz, const int32_t* tgt, void* dz, int64_t lddz,
                float* loss_rows, int64_t rows, int V, float scale, void* stream);

/* Token and position embedding (node 0 of the layer chain):
 * x[n][c] = wte[tok[n]][c] + wpe[n % T][c]; x fp32 [n_tok][d].  A token id
 * outside [0, V) yields a NaN row (no out-of-range read). */
int atom_k_embed_fwd(int dtype, const int32_t* tok, const void* wte, const void* wpe, float* x, int64_t n_tok,
                     int T, int V, int d, void* stream);

/* Plain device copy of `bytes` (a multiple of 16; both pointers 16-byte
 * aligned, not overlapping): reads and writes each byte once.  Measurement
 * only: its known traffic calibrates the HBM byte counters. */
int atom_k_copy(const void* src, void* dst, int64_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ATOM_KERNELS_H */
