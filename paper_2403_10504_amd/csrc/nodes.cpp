// A node's forward and backward composed from the kernels: the decoder
// block (LayerNorm, QKV, attention, output projection, MLP, residuals), the
// LM head with the cross-entropy, and the embedding; weight and gradient
// addresses in the group slots; the GEMM probe.
#include "context.h"

namespace atom {
namespace rt {

float* ckpt_ptr(atom_ctx* c, int idx, int micro) {
  return reinterpret_cast<float*>(A(c, c->lay.ckpt) + static_cast<uint64_t>(ck_entry(c, idx, micro)) *
                                                          c->lay.ckpt_bytes_each);
}

// Device pointer of a weight tensor of `node` in its group's slot.
const void* wptr(atom_ctx* c, int node, int t) {
  const int g = c->node_group[node];
  const uint64_t in_group = c->node_off[node] - c->group_off[g];
  return A(c, c->lay.wslots + static_cast<uint64_t>(slot_of(c, c->par, g)) * c->plan.slot_bytes + in_group +
                  c->tens[node][t].offset);
}

GradTarget gptr(atom_ctx* c, int node, int t, int micro) {
  const int g = c->node_group[node];
  const uint64_t in_group = c->node_off[node] - c->group_off[g] + c->tens[node][t].offset;
  if (use_accslot(c)) return {A(c, c->lay.accslot + 2 * in_group), DT_F32, micro > 0};
  const int gs = c->gslot_of[GI(c, c->par, g)];
  return {A(c, c->lay.gslots + static_cast<uint64_t>(gs) * c->plan.slot_bytes + in_group),
          c->dt == DT_BF16 ? DT_BF16 : DT_F32, micro > 0};
}

int wgrad_epi(const GradTarget& t) {
  if (t.dtype == DT_F32) return t.accumulate ? EPI_ACC_F32 : EPI_STORE_F32;
  return EPI_STORE;
}

// Waits (on the compute stream) for the weights of the node's group and for
// the gradient slot the group will write.
int prepare_group(atom_ctx* c, int node, bool grads) {
  const int g = c->node_group[node];
  const int gi = GI(c, c->par, g);
  if (!c->resident[gi]) return fail(c, ATOM_ESTATE, "group " + std::to_string(g) + " is not swapped in");
  if (c->need_wait[gi]) {
    {
      std::unique_lock<std::mutex> l(c->xm);
      c->xcv.wait(l, [c, gi] { return c->load_done[gi] >= c->load_req[gi]; });
    }
    KCHK(c, dma_acquire(c->cs));
    c->need_wait[gi] = 0;
  }
  if (grads && !c->gclaimed[gi]) {
    // every copy out of the gradient slot issued so far must have finished
    const int gs = c->next_gslot;
    c->next_gslot = (gs + 1) % c->R;
    std::unique_lock<std::mutex> l(c->xm);
    c->xcv.wait(l, [c, gs] { return c->gs_freed[gs] >= c->gs_issued[gs]; });
    c->gslot_of[gi] = gs;
    c->gclaimed[gi] = 1;
  }
  return ATOM_OK;
}

int finish_group_use(atom_ctx* c, int node) {
  const int gi = GI(c, c->par, c->node_group[node]);
  HIPCHK(c, hipEventRecord(c->ev_lastuse[gi], c->cs));
  c->lastuse_recorded[gi] = 1;
  return ATOM_OK;
}

GemmArgs gargs(const void* A_, int64_t lda, const void* B_, int64_t ldb, void* C_, int64_t ldc, int M, int N,
               int K) {
  GemmArgs g{};
  g.A = A_;
  g.B = B_;
  g.C = C_;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.ldaux = ldc;
  g.M = M;
  g.N = N;
  g.K = K;
  return g;
}


// Drain recorded probe events (after the compute stream has finished them).
int probe_collect(atom_ctx* c) {
  for (int i = 0; i < c->probe_pending; ++i) {
    float ms = 0.f;
    HIPCHK(c, hipEventElapsedTime(&ms, c->probe_ev[2 * i], c->probe_ev[2 * i + 1]));
    c->probe_seconds += ms * 1e-3;
    c->probe_flops += c->probe_flop[i];
    c->probe_bytes += c->probe_byte[i];
    c->probe_launches += 1;
  }
  c->probe_pending = 0;
  return ATOM_OK;
}

// Every GEMM of the step goes through here so the probe can time it.
// alg_m (if >= 0) is the algorithmic row count the probe counts instead of
// g.M: the LM head's weight gradient runs over the padded vocabulary Vp but
// computes V useful rows.
hipError_t run_gemm(atom_ctx* c, const GemmArgs& g, bool akc, bool bkc, int epi, int alg_m = -1) {
  const bool probe = c->probe_epi == epi && c->probe_akc == static_cast<int>(akc) &&
                     c->probe_bkc == static_cast<int>(bkc) && c->probe_pending < PROBE_MAX;
  if (probe) {
    hipError_t e = hipEventRecord(c->probe_ev[2 * c->probe_pending], c->cs);
    if (e != hipSuccess) return e;
  }
  GemmArgs gw = g;
  gw.ws = reinterpret_cast<float*>(A(c, c->lay.splitk));
  gw.ws_bytes = c->lay.splitk_bytes;
  hipError_t e = gemm(gw, c->dt, akc, bkc, epi, c->cs);
  if (e != hipSuccess || !probe) return e;
  e = hipEventRecord(c->probe_ev[2 * c->probe_pending + 1], c->cs);
  if (e != hipSuccess) return e;
  const double M = alg_m >= 0 ? alg_m : g.M;
  c->probe_flop[c->probe_pending] = 2.0 * M * g.N * static_cast<double>(g.K);
  // algorithmic bytes: both operands read once, the output written once
  // (fp32 or the element type), plus what the epilogue reads
  const double ein = c->e;
  const double eout = (epi == EPI_STORE_F32 || epi == EPI_ACC_F32 || epi == EPI_BIAS_RESID) ? 4.0 : ein;
  double extra = 0.0;
  if (epi == EPI_ACC_F32 || epi == EPI_BIAS_RESID) extra += 4.0 * M * g.N;
  if (epi == EPI_BIAS_GELU || epi == EPI_GELU_BWD) extra += ein * M * g.N;
  c->probe_byte[c->probe_pending] = ein * (M * g.K + static_cast<double>(g.K) * g.N) + eout * M * g.N + extra;
  c->probe_pending += 1;
  return hipSuccess;
}

// Tensor indices inside a block node.
enum { T_LN1G, T_LN1B, T_WQKV, T_BQKV, T_WO, T_BO, T_LN2G, T_LN2B, T_WFC, T_BFC, T_WPR, T_BPR };
enum { T_WTE, T_WPE };
enum { T_LNFG, T_LNFB, T_WHEAD };

// Forward of block `node` on micro-batch `micro`; recompute == true stops
// before the last projection (the backward does not need the block output).
int block_forward(atom_ctx* c, int node, int micro, bool recompute) {
  const int dt = c->dt, d = c->d, f = c->f;
  const int64_t N = c->N;
  hipStream_t s = c->cs;
  const float* x = ckpt_ptr(c, node - 1, micro);
  const auto& L = c->lay;
  void* a = WS(c, L.a);
  void* qkv = WS(c, L.qkv);
  void* o = WS(c, L.o);
  float* x1 = reinterpret_cast<float*>(WS(c, L.x1));
  void* cc = WS(c, L.c);
  void* u = WS(c, L.u);
  void* g = WS(c, L.g);
  float* mu1 = reinterpret_cast<float*>(WS(c, L.mu1));
  float* rs1 = reinterpret_cast<float*>(WS(c, L.rs1));
  float* mu2 = reinterpret_cast<float*>(WS(c, L.mu2));
  float* rs2 = reinterpret_cast<float*>(WS(c, L.rs2));
  float* lse = reinterpret_cast<float*>(WS(c, L.lse));

  KCHK(c, layernorm_fwd(dt, x, wptr(c, node, T_LN1G), wptr(c, node, T_LN1B), a, mu1, rs1, N, d, s));
  GemmArgs q = gargs(a, d, wptr(c, node, T_WQKV), d, qkv, 3 * d, static_cast<int>(N), 3 * d, d);
  q.bias = wptr(c, node, T_BQKV);
  KCHK(c, run_gemm(c, q, true, true, EPI_BIAS));
  KCHK(c, attn_fwd(dt, qkv, o, lse, c->B, c->T, c->H, c->dh, s));
  GemmArgs po = gargs(o, d, wptr(c, node, T_WO), d, x1, d, static_cast<int>(N), d, d);
  po.bias = wptr(c, node, T_BO);
  po.resid = x;
  KCHK(c, run_gemm(c, po, true, true, EPI_BIAS_RESID));
  KCHK(c, layernorm_fwd(dt, x1, wptr(c, node, T_LN2G), wptr(c, node, T_LN2B), cc, mu2, rs2, N, d, s));
  GemmArgs fc = gargs(cc, d, wptr(c, node, T_WFC), d, g, f, static_cast<int>(N), f, d);
  fc.bias = wptr(c, node, T_BFC);
  fc.aux = u;
  fc.ldaux = f;
  KCHK(c, run_gemm(c, fc, true, true, EPI_BIAS_GELU));
  if (!recompute) {
    GemmArgs pr = gargs(g, f, wptr(c, node, T_WPR), f, ckpt_ptr(c, node, micro), d, static_cast<int>(N), d, f);
    pr.bias = wptr(c, node, T_BPR);
    pr.resid = x1;
    KCHK(c, run_gemm(c, pr, true, true, EPI_BIAS_RESID));
  }
  return ATOM_OK;
}

// Bias gradient: column sums of x [N][cols] (dtype in_dt) into target.
int bias_grad(atom_ctx* c, int in_dt, const void* x, int cols, float* part, const GradTarget& t) {
  KCHK(c, colsum_partial(in_dt, x, c->N, cols, cols, part, c->cs));
  KCHK(c, sum_parts(part, colsum_blocks(c->N), cols, cols, t.dtype, t.p, t.accumulate, c->cs));
  return ATOM_OK;
}

// LayerNorm backward into dres (accumulate) plus gamma/beta gradients.
int ln_grad(atom_ctx* c, const void* dy, const float* x, const float* mu, const float* rs, const void* gamma,
            float* dres, void* dres_lp, bool acc, float* part, const GradTarget& tg, const GradTarget& tb) {
  const int d = c->d;
  KCHK(c, layernorm_bwd(c->dt, dy, x, mu, rs, gamma, dres, dres_lp, acc, part, c->N, d, c->cs));
  const int64_t np = layernorm_bwd_blocks(c->N, d);
  // the partials are [np][2d], gamma's columns then beta's
  if (tg.dtype == tb.dtype && tg.accumulate == tb.accumulate) {
    KCHK(c, sum_parts2(part, np, 2 * d, 2 * static_cast<int64_t>(d), tg.dtype, tg.p, tb.p, d, tg.accumulate, c->cs));
  } else {
    KCHK(c, sum_parts(part, np, d, 2 * static_cast<int64_t>(d), tg.dtype, tg.p, tg.accumulate, c->cs));
    KCHK(c, sum_parts(part + d, np, d, 2 * static_cast<int64_t>(d), tb.dtype, tb.p, tb.accumulate, c->cs));
  }
  return ATOM_OK;
}

int block_backward(atom_ctx* c, int node, int micro) {
  int st = block_forward(c, node, micro, true);
  if (st != ATOM_OK) return st;
  const int dt = c->dt, d = c->d, f = c->f;
  const int Nn = static_cast<int>(c->N);
  hipStream_t s = c->cs;
  const auto& L = c->lay;
  const float* x = ckpt_ptr(c, node - 1, micro);
  float* dres = reinterpret_cast<float*>(A(c, L.dres)) + static_cast<int64_t>(micro) * c->N * d;
  void* dlp = dt == DT_BF16 ? static_cast<void*>(A(c, L.dres_lp) + static_cast<uint64_t>(micro) * c->N * d * 2)
                            : static_cast<void*>(dres);
  void* dres_lp_out = dt == DT_BF16 ? dlp : nullptr;
  void* a = WS(c, L.a);
  void* qkv = WS(c, L.qkv);
  void* o = WS(c, L.o);
  float* x1 = reinterpret_cast<float*>(WS(c, L.x1));
  void* cc = WS(c, L.c);
  void* u = WS(c, L.u);
  void* g = WS(c, L.g);
  float* mu1 = reinterpret_cast<float*>(WS(c, L.mu1));
  float* rs1 = reinterpret_cast<float*>(WS(c, L.rs1));
  float* mu2 = reinterpret_cast<float*>(WS(c, L.mu2));
  float* rs2 = reinterpret_cast<float*>(WS(c, L.rs2));
  float* lse = reinterpret_cast<float*>(WS(c, L.lse));
  float* delta = reinterpret_cast<float*>(WS(c, L.delta));
  void* du = WS(c, L.du);
  void* dbuf = WS(c, L.dbuf);
  void* dout = WS(c, L.dout);
  void* dqkv = WS(c, L.dqkv);
  float* part = reinterpret_cast<float*>(WS(c, L.part));

  // MLP output projection: x2 = x1 + g W_pr^T + b_pr
  GradTarget t = gptr(c, node, T_BPR, micro);
  if ((st = bias_grad(c, DT_F32, dres, d, part, t)) != ATOM_OK) return st;
  t = gptr(c, node, T_WPR, micro);
  KCHK(c, run_gemm(c, gargs(dlp, d, g, f, t.p, f, d, f, Nn), false, false, wgrad_epi(t)));
  GemmArgs gd = gargs(dlp, d, wptr(c, node, T_WPR), f, du, f, Nn, f, d);
  gd.aux = u;
  gd.ldaux = f;
  KCHK(c, run_gemm(c, gd, true, false, EPI_GELU_BWD));
  // MLP input projection: u = c W_fc^T + b_fc
  t = gptr(c, node, T_BFC, micro);
  if ((st = bias_grad(c, dt, du, f, part, t)) != ATOM_OK) return st;
  t = gptr(c, node, T_WFC, micro);
  KCHK(c, run_gemm(c, gargs(du, f, cc, d, t.p, d, f, d, Nn), false, false, wgrad_epi(t)));
  KCHK(c, run_gemm(c, gargs(du, f, wptr(c, node, T_WFC), d, dbuf, d, Nn, d, f), true, false, EPI_STORE));
  // LN2
  st = ln_grad(c, dbuf, x1, mu2, rs2, wptr(c, node, T_LN2G), dres, dres_lp_out, true, part,
               gptr(c, node, T_LN2G, micro), gptr(c, node, T_LN2B, micro));
  if (st != ATOM_OK) return st;
  // attention output projection: x1 = x + o W_o^T + b_o
  t = gptr(c, node, T_BO, micro);
  if ((st = bias_grad(c, DT_F32, dres, d, part, t)) != ATOM_OK) return st;
  t = gptr(c, node, T_WO, micro);
  KCHK(c, run_gemm(c, gargs(dlp, d, o, d, t.p, d, d, d, Nn), false, false, wgrad_epi(t)));
  KCHK(c, run_gemm(c, gargs(dlp, d, wptr(c, node, T_WO), d, dout, d, Nn, d, d), true, false, EPI_STORE));
  // attention
  KCHK(c, attn_bwd(dt, qkv, o, dout, lse, delta, dqkv, c->B, c->T, c->H, c->dh, s));
  // QKV projection: qkv = a W_qkv^T + b_qkv
  t = gptr(c, node, T_BQKV, micro);
  if ((st = bias_grad(c, dt, dqkv, 3 * d, part, t)) != ATOM_OK) return st;
  t = gptr(c, node, T_WQKV, micro);
  KCHK(c, run_gemm(c, gargs(dqkv, 3 * d, a, d, t.p, d, 3 * d, d, Nn), false, false, wgrad_epi(t)));
  KCHK(c, run_gemm(c, gargs(dqkv, 3 * d, wptr(c, node, T_WQKV), d, dbuf, d, Nn, d, 3 * d), true, false, EPI_STORE));
  // LN1
  return ln_grad(c, dbuf, x, mu1, rs1, wptr(c, node, T_LN1G), dres, dres_lp_out, true, part,
                 gptr(c, node, T_LN1G, micro), gptr(c, node, T_LN1B, micro));
}

// Head: final LN, logits in token chunks, cross-entropy, and the head's
// backward, which initialises dres for the micro-batch.
int head_forward_backward(atom_ctx* c, int node, int micro) {
  const int dt = c->dt, d = c->d;
  const int64_t N = c->N, Vp = c->Vp;
  hipStream_t s = c->cs;
  const auto& L = c->lay;
  const float* x = ckpt_ptr(c, c->L, micro);
  void* yhat = WS(c, L.yhat);
  float* fmu = reinterpret_cast<float*>(WS(c, L.fmu));
  float* frs = reinterpret_cast<float*>(WS(c, L.frs));
  float* logits = reinterpret_cast<float*>(WS(c, L.logits));
  uint8_t* dz = WS(c, L.dz);
  void* dyhat = WS(c, L.dyhat);
  float* part = reinterpret_cast<float*>(WS(c, L.hpart));
  float* dres = reinterpret_cast<float*>(A(c, L.dres)) + static_cast<int64_t>(micro) * N * d;
  void* dres_lp_out = dt == DT_BF16 ? static_cast<void*>(A(c, L.dres_lp) + static_cast<uint64_t>(micro) * N * d * 2)
                                    : nullptr;
  const int32_t* tgt = reinterpret_cast<const int32_t*>(A(c, L.tok_tgt + c->par * L.tok_stride)) +
                       static_cast<int64_t>(micro) * N;
  float* loss_rows = reinterpret_cast<float*>(A(c, L.loss_rows)) + static_cast<int64_t>(micro) * N;
  const float scale = 1.0f / static_cast<float>(static_cast<double>(c->C) * static_cast<double>(N));

  KCHK(c, layernorm_fwd(dt, x, wptr(c, node, T_LNFG), wptr(c, node, T_LNFB), yhat, fmu, frs, N, d, s));
  const void* W = wptr(c, node, T_WHEAD);
  for (int64_t r0 = 0; r0 < N; r0 += HEAD_CHUNK) {
    const int rows = static_cast<int>(std::min<int64_t>(HEAD_CHUNK, N - r0));
    KCHK(c, run_gemm(c, gargs(static_cast<uint8_t*>(yhat) + r0 * d * c->e, d, W, d, logits, Vp, rows,
                              static_cast<int>(Vp), d),
                     true, true, EPI_STORE_F32));
    KCHK(c, xent_fwd_bwd(dt, logits, Vp, tgt + r0, dz + r0 * Vp * c->e, Vp, loss_rows + r0, rows, c->V, scale, s));
  }
  KCHK(c, run_gemm(c, gargs(dz, Vp, W, d, dyhat, d, static_cast<int>(N), d, static_cast<int>(Vp)), true, false,
                   EPI_STORE));
  GradTarget t = gptr(c, node, T_WHEAD, micro);
  KCHK(c, run_gemm(c, gargs(dz, Vp, yhat, d, t.p, d, static_cast<int>(Vp), d, static_cast<int>(N)), false, false,
                   wgrad_epi(t), c->V));
  return ln_grad(c, dyhat, x, fmu, frs, wptr(c, node, T_LNFG), dres, dres_lp_out, false, part,
                 gptr(c, node, T_LNFG, micro), gptr(c, node, T_LNFB, micro));
}

int embed_forward(atom_ctx* c, int micro) {
  const int32_t* tok = reinterpret_cast<const int32_t*>(A(c, c->lay.tok_in + c->par * c->lay.tok_stride)) +
                       static_cast<int64_t>(micro) * c->N;
  // with row-sparse embedding transfers the ids address the step's packed rows
  KCHK(c, embed_fwd(c->dt, tok, wptr(c, 0, T_WTE), wptr(c, 0, T_WPE), ckpt_ptr(c, 0, micro), c->N, c->T,
                    emb_vocab(c, c->par), c->d, c->cs));
  return ATOM_OK;
}

int embed_backward(atom_ctx* c, int micro) {
  const auto& L = c->lay;
  const int64_t N = c->N;
  const uint64_t ts = c->par * L.tok_stride;
  const float* dres = reinterpret_cast<const float*>(A(c, L.dres)) + static_cast<int64_t>(micro) * N * c->d;
  const int32_t* perm = reinterpret_cast<const int32_t*>(A(c, L.emb_perm + ts)) + static_cast<int64_t>(micro) * N;
  const int32_t* seg = reinterpret_cast<const int32_t*>(A(c, L.emb_seg + ts)) + static_cast<int64_t>(micro) * (N + 1);
  const int32_t* uniq = reinterpret_cast<const int32_t*>(A(c, L.emb_uniq + ts)) + static_cast<int64_t>(micro) * N;
  GradTarget te = gptr(c, 0, T_WTE, micro), tp = gptr(c, 0, T_WPE, micro);
  KCHK(c, embed_bwd(te.dtype, dres, perm, seg, uniq, c->n_uniq[c->par][micro], te.p, tp.p, emb_vocab(c, c->par), c->T,
                    c->B, c->d, te.accumulate, c->cs));
  return ATOM_OK;
}

}  // namespace rt
}  // namespace atom
