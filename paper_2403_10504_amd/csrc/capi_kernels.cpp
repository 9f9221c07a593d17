// extern "C" wrappers of the kernel launchers (include/atom_kernels.h).
#include <hip/hip_runtime.h>

#include "../../include/atom.h"
#include "../../include/atom_kernels.h"
#include "launch.h"

using namespace atom;

namespace {
inline int st(hipError_t e) {
  if (e == hipSuccess) return ATOM_OK;
  if (e == hipErrorInvalidValue) return ATOM_EINVAL;
  return ATOM_EHIP;
}
inline hipStream_t S(void* s) { return static_cast<hipStream_t>(s); }
inline bool dt_ok(int dt) { return dt == ATOM_F32 || dt == ATOM_BF16; }
}  // namespace

extern "C" {

int atom_k_gemm(int dtype, int a_kcontig, int b_kcontig, int epi, int M, int N, int K, const void* A, int64_t lda,
                const void* B, int64_t ldb, void* C, int64_t ldc, const void* bias, const float* resid, void* aux,
                int64_t ldaux, float* ws, uint64_t ws_bytes, void* stream) {
  if (!dt_ok(dtype) || !A || !B || !C || epi < ATOM_EPI_STORE || epi > ATOM_EPI_GELU_BWD) return ATOM_EINVAL;
  if ((epi == ATOM_EPI_BIAS || epi == ATOM_EPI_BIAS_GELU || epi == ATOM_EPI_BIAS_RESID) && !bias) return ATOM_EINVAL;
  if ((epi == ATOM_EPI_BIAS_GELU || epi == ATOM_EPI_GELU_BWD) && (!aux || ldaux < N)) return ATOM_EINVAL;
  if (epi == ATOM_EPI_BIAS_RESID && !resid) return ATOM_EINVAL;
  GemmArgs g{};
  g.A = A;
  g.B = B;
  g.C = C;
  g.bias = bias;
  g.resid = resid;
  g.aux = aux;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.ldaux = ldaux;
  g.M = M;
  g.N = N;
  g.K = K;
  g.ws = ws;
  g.ws_bytes = ws ? ws_bytes : 0;
  return st(gemm(g, dtype, a_kcontig != 0, b_kcontig != 0, epi, S(stream)));
}

int atom_k_layernorm_fwd(int dtype, const float* x, const void* gamma, const void* beta, void* y, float* mean,
                         float* rstd, int64_t rows, int d, void* stream) {
  if (!dt_ok(dtype) || !x || !gamma || !beta || !y || !mean || !rstd) return ATOM_EINVAL;
  return st(layernorm_fwd(dtype, x, gamma, beta, y, mean, rstd, rows, d, S(stream)));
}

int64_t atom_k_layernorm_bwd_part_floats(int64_t rows, int d) { return layernorm_bwd_blocks(rows, d) * 2 * d; }

int atom_k_layernorm_bwd(int dtype, const void* dy, const float* x, const float* mean, const float* rstd,
                         const void* gamma, float* dres, void* dres_lp, int accumulate, float* dgamma, float* dbeta,
                         float* part, int64_t rows, int d, void* stream) {
  if (!dt_ok(dtype) || !dy || !x || !mean || !rstd || !gamma || !dres || !dgamma || !dbeta || !part) return ATOM_EINVAL;
  int s = st(layernorm_bwd(dtype, dy, x, mean, rstd, gamma, dres, dres_lp, accumulate != 0, part, rows, d, S(stream)));
  if (s != ATOM_OK) return s;
  const int64_t np = layernorm_bwd_blocks(rows, d);
  s = st(sum_parts(part, np, d, 2 * static_cast<int64_t>(d), DT_F32, dgamma, false, S(stream)));
  if (s != ATOM_OK) return s;
  return st(sum_parts(part + d, np, d, 2 * static_cast<int64_t>(d), DT_F32, dbeta, false, S(stream)));
}

int atom_k_attn_fwd(int dtype, const void* qkv, void* o, float* lse, int B, int T, int H, int dh, void* stream) {
  if (!dt_ok(dtype) || !qkv || !o || !lse) return ATOM_EINVAL;
  return st(attn_fwd(dtype, qkv, o, lse, B, T, H, dh, S(stream)));
}

int atom_k_attn_bwd(int dtype, const void* qkv, const void* o, const void* dout, const float* lse, float* delta,
                    void* dqkv, int B, int T, int H, int dh, void* stream) {
  if (!dt_ok(dtype) || !qkv || !o || !dout || !lse || !delta || !dqkv) return ATOM_EINVAL;
  return st(attn_bwd(dtype, qkv, o, dout, lse, delta, dqkv, B, T, H, dh, S(stream)));
}

int64_t atom_k_colsum_part_floats(int64_t rows, int cols) { return colsum_blocks(rows) * cols; }

int atom_k_colsum(int dtype, const void* x, int64_t rows, int cols, float* out, float* part, void* stream) {
  if (!dt_ok(dtype) || !x || !out || !part) return ATOM_EINVAL;
  int s = st(colsum_partial(dtype, x, rows, cols, cols, part, S(stream)));
  if (s != ATOM_OK) return s;
  return st(sum_parts(part, colsum_blocks(rows), cols, cols, DT_F32, out, false, S(stream)));
}

int atom_k_xent(int dtype, const float* logits, int64_t ldz, const int32_t* tgt, void* dz, int64_t lddz,
                float* loss_rows, int64_t rows, int V, float scale, void* stream) {
  if (!dt_ok(dtype) || !logits || !tgt || !dz || !loss_rows) return ATOM_EINVAL;
  return st(xent_fwd_bwd(dtype, logits, ldz, tgt, dz, lddz, loss_rows, rows, V, scale, S(stream)));
}

int atom_k_embed_fwd(int dtype, const int32_t* tok, const void* wte, const void* wpe, float* x, int64_t n_tok, int T,
                     int V, int d, void* stream) {
  if (!dt_ok(dtype) || !tok || !wte || !wpe || !x || T <= 0 || V <= 0 || d <= 0) return ATOM_EINVAL;
  return st(embed_fwd(dtype, tok, wte, wpe, x, n_tok, T, V, d, S(stream)));
}

int atom_k_copy(const void* src, void* dst, int64_t bytes, void* stream) {
  if (!src || !dst || bytes < 0 || bytes % 16) return ATOM_EINVAL;
  return st(copy_bytes(src, dst, bytes, S(stream)));
}

}  // extern "C"
