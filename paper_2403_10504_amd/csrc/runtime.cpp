// Runtime of the swapped GPT step: the context, the pinned host model, the
// swap engine (weights in on one system DMA engine, gradients out on another,
// each fed by its own worker thread that waits on compute-stream events), the
// composition of each
// node's forward and backward from the kernels, host-side gradient
// accumulation, and the schedule of whole steps.
//
// Schedule (Section IV: one stream runs the current sub-model, another
// prefetches the next; completed sub-models are swapped out; the last forward
// sub-model is not swapped out before the backward).  With K weight slots:
//   forward : load groups 0..K-1; after group j's forward is enqueued, load
//             group j+K into the slot group j frees;
//   backward: the last K groups are still resident; after group j's backward
//             its gradients are copied out and group j-K is reloaded into the
//             slot group j just freed.
// A pipelined call runs several steps of one global batch back to back (the
// host model does not change inside it, as the optimizer runs only when the
// global batch is complete, Section III-E): once the backward has freed the
// slot of one of the last K groups, the next step's swap-in of a first group
// starts in it, so the next step's weights stream in while this step's
// backward computes and its gradients stream out.  Consecutive steps use
// opposite slot orders (group j in slot j mod K, then K-1-(j mod K)), which
// makes the slots free in exactly the order the next step needs them.  Each
// step still loads every weight and drains every gradient.
//
// Gradients of a group go to one of the plan's gradient slots (claimed
// round-robin in backward order), are copied to pinned host memory (one buffer
// shared by the steps in flight: a group's copy waits until the group's
// previous gradients have been accumulated) on the
// system DMA engine, and a host thread adds them to the fp32 accumulators.
//
// Transfers.  Both directions run on the GPU's system DMA (SDMA) engines
// through ROCr, each on its own fixed engine and its own worker thread, so
// they never queue behind each other or behind HIP's own copies, and take no
// compute unit (HIP moves device-to-host data with a copy kernel, which the
// training kernels starve).  A weight copy waits (on the host) for the last
// compute that used its slot; a gradient copy waits for the group's backward.
// The calling thread only enqueues compute: before a group's first kernel it
// waits on the host for the group's weight copy to have finished (then
// enqueues a cache acquire so kernels see the DMA-written weights), and
// before a group reuses a gradient slot, for the copy out of that slot (so
// gradient copies may lag the backward by as many groups as there are
// gradient slots).  Every kernel reduces in a fixed
// order, so a step gives bitwise the same result for any plan and any
// pipelining.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>
#include <unistd.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <deque>
#include <functional>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "launch.h"
#include "layout.h"
#include "transfer.h"

namespace atom {

// ------------------------------------------------------------ host pool
// Fixed pool of threads for the host gradient accumulation.
class HostPool {
 public:
  explicit HostPool(int n) : n_(std::max(1, n)) {
    for (int i = 1; i < n_; ++i) th_.emplace_back([this, i] { loop(i); });
  }
  ~HostPool() {
    {
      std::lock_guard<std::mutex> l(m_);
      stop_ = true;
      ++gen_;
    }
    cv_.notify_all();
    for (auto& t : th_) t.join();
  }
  int size() const { return n_; }
  // Runs fn(i) for i in [0, n) on all threads; returns when all are done.
  // Not reentrant (one job at a time): during steps only the accumulation
  // thread calls it; the context's other users (zeroing, optimizer) first
  // drain every copy and the accumulation queue (sync_all), so no two
  // callers overlap.
  void run(const std::function<void(int)>& fn) {
    {
      std::lock_guard<std::mutex> l(m_);
      fn_ = &fn;
      pending_ = n_ - 1;
      ++gen_;
    }
    cv_.notify_all();
    fn(0);
    std::unique_lock<std::mutex> l(m_);
    done_cv_.wait(l, [this] { return pending_ == 0; });
    fn_ = nullptr;
  }

 private:
  void loop(int i) {
    uint64_t seen = 0;
    for (;;) {
      const std::function<void(int)>* f;
      {
        std::unique_lock<std::mutex> l(m_);
        cv_.wait(l, [&] { return gen_ != seen; });
        seen = gen_;
        if (stop_) return;
        f = fn_;
      }
      (*f)(i);
      {
        std::lock_guard<std::mutex> l(m_);
        if (--pending_ == 0) done_cv_.notify_one();
      }
    }
  }
  int n_;
  std::vector<std::thread> th_;
  std::mutex m_;
  std::condition_variable cv_, done_cv_;
  const std::function<void(int)>* fn_ = nullptr;
  int pending_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

}  // namespace atom

using namespace atom;

struct Range {
  uint64_t off, n;  // element offset and count within the host model
};

// Group g of a step with parity p is the "instance" gi = p * G + g: the two
// steps a pipelined call keeps in flight have separate residency and events.
struct atom_ctx {
  atom_config cfg{};
  atom_plan plan{};
  ArenaLayout lay{};
  uint8_t* arena = nullptr;
  hipStream_t cs = nullptr;
  int L = 0, G = 0, K = 0, C = 0, H = 0, dh = 0, dt = 0, e = 0, d = 0, f = 0, V = 0, B = 0, T = 0;
  int64_t N = 0, Vp = 0;
  int par = 0;       // parity of the step the compute stream is being given work for

  // host model (pinned), per-node ranges
  uint8_t* h_w = nullptr;             // weights, working dtype
  uint8_t* h_g = nullptr;             // gradients of the last step, working dtype
  float* h_acc = nullptr;             // fp32 accumulators (element-indexed like h_w)
  uint64_t model_bytes = 0;
  std::vector<uint64_t> node_off, node_bytes;
  std::vector<std::vector<TensorDesc>> tens;
  std::vector<int> node_group;
  std::vector<uint64_t> group_off, group_bytes;
  std::vector<std::vector<Range>> group_ranges;  // tensors of each group (for accumulation)

  // residency and events, indexed by group instance
  std::vector<int> slot_owner;  // instance whose weights occupy the slot (-1: none)
  std::vector<char> resident, need_wait, gclaimed, lastuse_recorded;
  std::vector<hipEvent_t> ev_lastuse, ev_gready;

  // transfers (see the file comment); counters are guarded by xm
  Worker* h2d_worker = nullptr;
  Worker* d2h_worker = nullptr;
  DmaEngine dma;     // device-to-host
  DmaEngine dma_in;  // host-to-device
  std::mutex xm;
  std::condition_variable xcv;
  std::vector<uint64_t> load_req, load_done;  // per instance: weight copies requested / finished
  std::vector<int> d2h_pending;               // per instance: gradient copies not yet finished
  int R = 2;                                // gradient slots
  std::vector<uint64_t> gs_issued, gs_freed;  // per gradient slot: copies out issued / finished
  std::vector<int> gslot_of;                // per instance: gradient slot of its current claim
  int next_gslot = 0;                       // round-robin claim order

  // Host checkpoints (ATOM_CKPT_HOST).  Block input idx (0..L) of micro-batch
  // m lives in ring entry (idx % CKPT_RING) * C + m.  Inputs the ring
  // overwrites in the forward are copied to pinned host memory on the D2H
  // engine after the kernel that wrote them, and restored on the H2D engine
  // once the last kernel that read the entry's later occupant has run.
  bool ck_host = false;
  // weights retained across the steps of one atom_steps call (every group
  // in a slot of its own); retain_active while such a call runs
  bool retain = false, retain_active = false;
  uint8_t* h_ck = nullptr;                        // pinned [(L+1)][C][N][d] fp32
  std::vector<int> ck_holder;                     // per ring entry: index it holds (-1: none)
  std::vector<char> ck_wait;                      // per ring entry: a restore the compute stream has not waited for
  std::vector<uint64_t> ck_out_req, ck_out_done;  // per (idx, m): copies to the host issued / finished
  std::vector<uint64_t> ck_in_req, ck_in_done;    // per (idx, m): restores issued / finished
  std::vector<hipEvent_t> ev_ckw, ev_cku;         // per ring entry: after its writer / its last reader
  std::vector<char> cku_recorded;

  // per-step validation state, by parity
  bool tokens_ok[2] = {false, false};
  std::vector<char> fwd_done[2], bwd_done[2];  // [node][micro]
  std::vector<int> n_uniq[2];                  // per micro
  int32_t* h_tok[2] = {nullptr, nullptr};      // pinned token staging
  hipEvent_t ev_tok[2] = {nullptr, nullptr};
  bool tok_recorded[2] = {false, false};

  // host accumulation
  HostPool* pool = nullptr;
  std::thread acc_thread;
  std::mutex acc_m;
  std::condition_variable acc_cv, acc_done_cv;
  std::deque<int> acc_q;  // group instances
  std::vector<int> acc_pending;
  int acc_busy = 0;
  bool acc_stop = false;
  int acc_error = 0;
  std::string acc_errmsg;
  double acc_seconds = 0;

  // GEMM probe (measurement): events around launches of one instantiation
  int probe_akc = -1, probe_bkc = -1, probe_epi = -1;
  std::vector<hipEvent_t> probe_ev;  // 2 per launch
  std::vector<double> probe_flop, probe_byte;  // per pending launch
  int probe_pending = 0;
  int64_t probe_launches = 0;
  double probe_seconds = 0, probe_flops = 0, probe_bytes = 0;

  // host optimizer (atom_optimizer_init / atom_optimizer_step): fp32 master
  // weights and the two AdamW moments, element-indexed like h_w (pageable)
  float* h_master = nullptr;
  float* h_m = nullptr;
  float* h_v = nullptr;

  // node profile (atom_profile_nodes): events around each node's forward
  // and backward, per micro-batch
  bool profiling = false;
  std::vector<hipEvent_t> prof_ev;  // [node][micro][fwd, bwd][begin, end]

  atom_stats stats{};
  std::string err;
};

namespace {

// Failure text of the last atom_ctx_create on this thread (no context exists
// to hold it).
thread_local std::string g_create_error;

int fail(atom_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg;
  return code;
}

#define HIPCHK(ctx, expr)                                                                 \
  do {                                                                                    \
    hipError_t _e = (expr);                                                               \
    if (_e != hipSuccess)                                                                 \
      return fail(ctx, ATOM_EHIP, std::string(#expr) + ": " + hipGetErrorString(_e));     \
  } while (0)

#define KCHK(ctx, expr)                                                                       \
  do {                                                                                        \
    hipError_t _e = (expr);                                                                   \
    if (_e != hipSuccess)                                                                     \
      return fail(ctx, ATOM_EHIP, std::string("kernel launch ") + #expr + ": " + hipGetErrorString(_e)); \
  } while (0)

inline uint8_t* A(atom_ctx* c, uint64_t off) { return c->arena + off; }
inline uint8_t* WS(atom_ctx* c, uint64_t off) { return c->arena + c->lay.ws + off; }
inline int GI(atom_ctx* c, int par, int g) { return par * c->G + g; }

// Weight slot of group g in a step of parity par (see the file comment).
inline int slot_of(atom_ctx* c, int par, int g) {
  const int r = g % c->K;
  return par == 0 || c->retain_active ? r : c->K - 1 - r;
}

// Device entry of block input idx (the output of node idx) of a micro-batch.
inline int ck_entry(atom_ctx* c, int idx, int micro) { return (c->ck_host ? idx % CKPT_RING : idx) * c->C + micro; }
inline bool ck_evicted(atom_ctx* c, int idx) { return c->ck_host && idx + CKPT_RING <= c->L; }
inline size_t ck_key(atom_ctx* c, int idx, int micro) { return static_cast<size_t>(idx) * c->C + micro; }

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

// Gradient target of a tensor: fp32 accumulation slot (bf16 with C > 1) or
// the group's gradient slot in the working dtype.
struct GradTarget {
  void* p;
  int dtype;  // DT_F32 or DT_BF16
  bool accumulate;
};

bool use_accslot(atom_ctx* c) { return c->dt == DT_BF16 && c->C > 1; }

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

constexpr int PROBE_MAX = 4096;

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
  KCHK(c, sum_parts(part, np, d, 2 * static_cast<int64_t>(d), tg.dtype, tg.p, tg.accumulate, c->cs));
  KCHK(c, sum_parts(part + d, np, d, 2 * static_cast<int64_t>(d), tb.dtype, tb.p, tb.accumulate, c->cs));
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
  KCHK(c, embed_fwd(c->dt, tok, wptr(c, 0, T_WTE), wptr(c, 0, T_WPE), ckpt_ptr(c, 0, micro), c->N, c->T, c->V, c->d,
                    c->cs));
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
  KCHK(c, embed_bwd(te.dtype, dres, perm, seg, uniq, c->n_uniq[c->par][micro], te.p, tp.p, c->V, c->T, c->B, c->d,
                    te.accumulate, c->cs));
  return ATOM_OK;
}

// ------------------------------------------------------ host accumulation
template <typename T>
void accum_range(float* acc, const T* g, uint64_t n);
template <>
void accum_range<float>(float* acc, const float* g, uint64_t n) {
  for (uint64_t i = 0; i < n; ++i) acc[i] += g[i];
}
template <>
void accum_range<uint16_t>(float* acc, const uint16_t* g, uint64_t n) {
  for (uint64_t i = 0; i < n; ++i) {
    uint32_t u = static_cast<uint32_t>(g[i]) << 16;
    float v;
    memcpy(&v, &u, 4);
    acc[i] += v;
  }
}

void accumulate_group(atom_ctx* c, int gi) {
  const int par = gi / c->G, g = gi % c->G;
  const uint8_t* hg = c->h_g;
  const auto& rs = c->group_ranges[g];
  uint64_t total = 0;
  for (auto& r : rs) total += r.n;
  const int nt = c->pool->size();
  c->pool->run([&](int ti) {
    // split the concatenated ranges into nt equal pieces
    const uint64_t lo = total * ti / nt, hi = total * (ti + 1) / nt;
    uint64_t pos = 0;
    for (auto& r : rs) {
      const uint64_t a = std::max(lo, pos), b = std::min(hi, pos + r.n);
      if (a < b) {
        const uint64_t off = r.off + (a - pos);
        if (c->dt == DT_BF16)
          accum_range<uint16_t>(c->h_acc + off, reinterpret_cast<const uint16_t*>(hg) + off, b - a);
        else
          accum_range<float>(c->h_acc + off, reinterpret_cast<const float*>(hg) + off, b - a);
      }
      pos += r.n;
    }
  });
}

void acc_loop(atom_ctx* c) {
  for (;;) {
    int gi;
    {
      std::unique_lock<std::mutex> l(c->acc_m);
      c->acc_cv.wait(l, [c] { return c->acc_stop || !c->acc_q.empty(); });
      if (c->acc_q.empty()) return;
      gi = c->acc_q.front();
      c->acc_q.pop_front();
    }
    // queued only once its gradient copy has finished
    auto t0 = std::chrono::steady_clock::now();
    accumulate_group(c, gi);
    c->acc_seconds += std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    {
      std::lock_guard<std::mutex> l(c->acc_m);
      --c->acc_pending[gi];
      --c->acc_busy;
    }
    c->acc_done_cv.notify_all();
  }
}

int wait_accum(atom_ctx* c) {
  std::unique_lock<std::mutex> l(c->acc_m);
  c->acc_done_cv.wait(l, [c] { return c->acc_busy == 0; });
  if (c->acc_error) {
    const int e = c->acc_error;
    c->acc_error = 0;
    return fail(c, e, c->acc_errmsg);
  }
  return ATOM_OK;
}

// The host buffer of instance gi is rewritten by its next gradient copy only
// after the previous one has been added to the accumulators.
void wait_accum_group(atom_ctx* c, int g) {
  std::unique_lock<std::mutex> l(c->acc_m);
  c->acc_done_cv.wait(l, [c, g] { return c->acc_pending[g] == 0 && c->acc_pending[c->G + g] == 0; });
}

bool group_bwd_complete(atom_ctx* c, int par, int g) {
  for (int n = c->plan.first[g]; n <= c->plan.last[g]; ++n)
    for (int m = 0; m < c->C; ++m) {
      const size_t k = static_cast<size_t>(n) * c->C + m;
      if (n == c->L + 1 ? !c->fwd_done[par][k] : !c->bwd_done[par][k]) return false;
    }
  return true;
}

// Clears the per-step state of parity par (called when a step's tokens are set).
void reset_step_state(atom_ctx* c, int par) {
  std::fill(c->fwd_done[par].begin(), c->fwd_done[par].end(), 0);
  std::fill(c->bwd_done[par].begin(), c->bwd_done[par].end(), 0);
  for (int g = 0; g < c->G; ++g) c->gclaimed[GI(c, par, g)] = 0;
}

// Every group of both parities is considered not resident: the next step
// loads all weights again (the host model may have changed).
void drop_residency(atom_ctx* c) {
  std::fill(c->resident.begin(), c->resident.end(), 0);
  std::fill(c->need_wait.begin(), c->need_wait.end(), 0);
}

// Retained weights: group g's slot, loaded in an earlier step of the same
// call, serves the step of parity par without a copy.  Every group runs in
// every step, so the compute stream has already waited for that load (and
// acquired the DMA-written data); kernels on it run in order, so the step of
// parity par reads the slot only after the previous step is done with it.
int hand_over(atom_ctx* c, int par, int g) {
  const int gi = GI(c, par, g), pi = GI(c, par ^ 1, g);
  if (!c->resident[pi] || c->need_wait[pi])
    return fail(c, ATOM_ESTATE, "group " + std::to_string(g) + " was not used before its hand-over");
  c->resident[pi] = 0;
  c->resident[gi] = 1;
  c->need_wait[gi] = 0;
  c->lastuse_recorded[gi] = 0;
  c->slot_owner[slot_of(c, par, g)] = gi;
  return ATOM_OK;
}

// Token preprocessing on the host and an asynchronous upload on the compute
// stream into token slot par.  Ids are validated before anything is copied.
int upload_tokens(atom_ctx* c, int par, const int32_t* tokens) {
  const int64_t N = c->N, T = c->T, C = c->C;
  for (int64_t i = 0; i < C * c->B * (T + 1); ++i)
    if (tokens[i] < 0 || tokens[i] >= c->V) return fail(c, ATOM_EINVAL, "token id out of range");
  if (c->tok_recorded[par]) HIPCHK(c, hipEventSynchronize(c->ev_tok[par]));  // staging slot free
  // staging layout: [inp C*N][tgt C*N][perm C*N][seg C*(N+1)][uniq C*N]
  int32_t* inp = c->h_tok[par];
  int32_t* tgt = inp + C * N;
  int32_t* perm = tgt + C * N;
  int32_t* seg = perm + C * N;
  int32_t* uniq = seg + C * (N + 1);
  std::vector<int32_t> count(c->V), start(c->V);
  for (int64_t m = 0; m < C; ++m) {
    for (int64_t b = 0; b < c->B; ++b)
      for (int64_t t = 0; t < T; ++t) {
        inp[m * N + b * T + t] = tokens[(m * c->B + b) * (T + 1) + t];
        tgt[m * N + b * T + t] = tokens[(m * c->B + b) * (T + 1) + t + 1];
      }
    // stable counting sort of token positions by token id
    std::fill(count.begin(), count.end(), 0);
    for (int64_t n = 0; n < N; ++n) ++count[inp[m * N + n]];
    int nu = 0, pos = 0;
    for (int v = 0; v < c->V; ++v) {
      start[v] = pos;
      if (count[v]) {
        uniq[m * N + nu] = v;
        seg[m * (N + 1) + nu] = pos;
        ++nu;
      }
      pos += count[v];
    }
    seg[m * (N + 1) + nu] = pos;
    for (int64_t n = 0; n < N; ++n) perm[m * N + start[inp[m * N + n]]++] = static_cast<int32_t>(n);
    c->n_uniq[par][m] = nu;
  }
  const auto& L = c->lay;
  const uint64_t ts = par * L.tok_stride;
  // Uploaded by a kernel on the compute stream, reading the pinned staging
  // buffer: a DMA copy queued on the compute stream would hold its DMA engine
  // until the compute stream reached it, delaying transfers queued behind it.
  auto up = [&](uint64_t off, const int32_t* src, int64_t n) {
    return copy_words(reinterpret_cast<const uint32_t*>(src), reinterpret_cast<uint32_t*>(A(c, off + ts)), n, c->cs);
  };
  KCHK(c, up(L.tok_in, inp, C * N));
  KCHK(c, up(L.tok_tgt, tgt, C * N));
  KCHK(c, up(L.emb_perm, perm, C * N));
  KCHK(c, up(L.emb_seg, seg, C * (N + 1)));
  KCHK(c, up(L.emb_uniq, uniq, C * N));
  HIPCHK(c, hipEventRecord(c->ev_tok[par], c->cs));
  c->tok_recorded[par] = true;
  c->tokens_ok[par] = true;
  reset_step_state(c, par);
  return ATOM_OK;
}

int swap_in_impl(atom_ctx* c, int par, int g) {
  const int gi = GI(c, par, g);
  if (c->resident[gi]) return fail(c, ATOM_ESTATE, "group " + std::to_string(g) + " is already resident");
  const int s = slot_of(c, par, g);
  const int prev = c->slot_owner[s];
  // the copy waits for the last compute that used the slot's previous occupant
  hipEvent_t wait_ev = nullptr;
  if (prev >= 0 && prev != gi) {
    if (c->resident[prev]) {
      // the previous occupant must have been used since it was loaded
      if (!c->lastuse_recorded[prev] && c->need_wait[prev])
        return fail(c, ATOM_ESTATE, "slot holds group " + std::to_string(prev % c->G) + " that was never used");
      c->resident[prev] = 0;
    }
    if (c->lastuse_recorded[prev]) wait_ev = c->ev_lastuse[prev];
  } else if (prev == gi && c->lastuse_recorded[gi]) {
    wait_ev = c->ev_lastuse[gi];
  }
  uint8_t* dst = A(c, c->lay.wslots + static_cast<uint64_t>(s) * c->plan.slot_bytes);
  const uint8_t* src = c->h_w + c->group_off[g];
  const uint64_t bytes = c->group_bytes[g];
  uint64_t gen;
  {
    std::lock_guard<std::mutex> l(c->xm);
    gen = ++c->load_req[gi];
  }
  c->h2d_worker->submit([c, gi, wait_ev, dst, src, bytes, gen]() -> std::string {
    std::string err;
    hipError_t e = hipSuccess;
    if (wait_ev)
      while ((e = hipEventQuery(wait_ev)) == hipErrorNotReady) usleep(POLL_US);
    if (e != hipSuccess) err = std::string("waiting for the slot: ") + hipGetErrorString(e);
    if (err.empty()) err = c->dma_in.copy(dst, src, bytes);
    {
      // published even on failure, so no waiter hangs; the error surfaces at the next sync
      std::lock_guard<std::mutex> l(c->xm);
      c->load_done[gi] = gen;
    }
    c->xcv.notify_all();
    return err;
  });
  c->slot_owner[s] = gi;
  c->resident[gi] = 1;
  c->need_wait[gi] = 1;
  c->lastuse_recorded[gi] = 0;
  c->stats.h2d_bytes += bytes;
  c->stats.swap_ins += 1;
  return ATOM_OK;
}

// ------------------------------------------------------ host checkpoints
// Wait (on the host) until ring entry e's occupant needs nothing more from
// the DMA engines: its copy to the host and any restore into it finished.
void ckpt_settle(atom_ctx* c, int e, int micro) {
  const int prev = c->ck_holder[e];
  if (prev < 0 || !ck_evicted(c, prev)) return;
  const size_t kp = ck_key(c, prev, micro);
  std::unique_lock<std::mutex> l(c->xm);
  c->xcv.wait(l, [c, kp] { return c->ck_out_done[kp] >= c->ck_out_req[kp] && c->ck_in_done[kp] >= c->ck_in_req[kp]; });
}

// Records that the compute stream has enqueued its last use (so far) of ring
// entry e; a restore into e waits for it.
int ckpt_used(atom_ctx* c, int e) {
  HIPCHK(c, hipEventRecord(c->ev_cku[e], c->cs));
  c->cku_recorded[e] = 1;
  return ATOM_OK;
}

// Copies block input idx of a micro-batch to the host once the kernel that
// wrote it has run (D2H engine).
int ckpt_out(atom_ctx* c, int idx, int micro) {
  const int e = ck_entry(c, idx, micro);
  const size_t k = ck_key(c, idx, micro);
  HIPCHK(c, hipEventRecord(c->ev_ckw[e], c->cs));
  const uint64_t bytes = c->lay.ckpt_bytes_each;
  uint8_t* dst = c->h_ck + k * bytes;
  const float* src = ckpt_ptr(c, idx, micro);
  hipEvent_t ev = c->ev_ckw[e];
  uint64_t gen;
  {
    std::lock_guard<std::mutex> l(c->xm);
    gen = ++c->ck_out_req[k];
  }
  // ev is recorded again only by the next writer of the entry, which first
  // waits for this copy (ckpt_settle)
  c->d2h_worker->submit([c, k, ev, dst, src, bytes, gen]() -> std::string {
    std::string err;
    hipError_t r;
    while ((r = hipEventQuery(ev)) == hipErrorNotReady) usleep(POLL_US);
    if (r != hipSuccess) err = std::string("waiting for a checkpoint: ") + hipGetErrorString(r);
    if (err.empty()) err = c->dma.copy(dst, src, bytes);
    {
      std::lock_guard<std::mutex> l(c->xm);
      c->ck_out_done[k] = gen;
    }
    c->xcv.notify_all();
    return err;
  });
  c->stats.d2h_bytes += bytes;
  return ATOM_OK;
}

// Restores block input idx of a micro-batch into its ring entry (H2D
// engine) after the last use of the entry's current occupant and after the
// copy of idx to the host.  No-op when the entry already holds idx.
int ckpt_restore(atom_ctx* c, int idx, int micro) {
  const int e = ck_entry(c, idx, micro);
  if (c->ck_holder[e] == idx) return ATOM_OK;
  if (!ck_evicted(c, idx))
    return fail(c, ATOM_ESTATE, "block input " + std::to_string(idx) + " is not on the device");
  const size_t k = ck_key(c, idx, micro);
  hipEvent_t wait_ev = c->cku_recorded[e] ? c->ev_cku[e] : nullptr;
  const uint64_t bytes = c->lay.ckpt_bytes_each;
  const uint8_t* src = c->h_ck + k * bytes;
  float* dst = ckpt_ptr(c, idx, micro);
  uint64_t gen, out_gen;
  {
    std::lock_guard<std::mutex> l(c->xm);
    if (c->ck_out_req[k] == 0) return fail(c, ATOM_ESTATE, "block input " + std::to_string(idx) + " never computed");
    gen = ++c->ck_in_req[k];
    out_gen = c->ck_out_req[k];
  }
  c->h2d_worker->submit([c, k, wait_ev, dst, src, bytes, gen, out_gen]() -> std::string {
    {
      std::unique_lock<std::mutex> l(c->xm);
      c->xcv.wait(l, [c, k, out_gen] { return c->ck_out_done[k] >= out_gen; });
    }
    std::string err;
    hipError_t r = hipSuccess;
    if (wait_ev)
      while ((r = hipEventQuery(wait_ev)) == hipErrorNotReady) usleep(POLL_US);
    if (r != hipSuccess) err = std::string("waiting for a checkpoint entry: ") + hipGetErrorString(r);
    if (err.empty()) err = c->dma_in.copy(dst, src, bytes);
    {
      std::lock_guard<std::mutex> l(c->xm);
      c->ck_in_done[k] = gen;
    }
    c->xcv.notify_all();
    return err;
  });
  c->ck_holder[e] = idx;
  c->ck_wait[e] = 1;
  c->cku_recorded[e] = 0;
  c->stats.h2d_bytes += bytes;
  return ATOM_OK;
}

// Makes block input idx readable by the next kernel on the compute stream
// (restoring it if needed and waiting for the restore).
int ckpt_ready(atom_ctx* c, int idx, int micro) {
  const int e = ck_entry(c, idx, micro);
  int st = ckpt_restore(c, idx, micro);
  if (st != ATOM_OK) return st;
  if (c->ck_wait[e]) {
    const size_t k = ck_key(c, idx, micro);
    {
      std::unique_lock<std::mutex> l(c->xm);
      c->xcv.wait(l, [c, k] { return c->ck_in_done[k] >= c->ck_in_req[k]; });
    }
    KCHK(c, dma_acquire(c->cs));
    c->ck_wait[e] = 0;
  }
  return ATOM_OK;
}

// Working-memory probe (atom_profile_nodes): the union workspace is filled
// with this word before each node runs, and a counter per node and direction
// records how far into the workspace the node's kernels wrote.  No data in
// the workspace outlives the node that wrote it, so the fill changes nothing.
constexpr uint32_t HWM_WORD = 0xFFC0FFEEu;  // a NaN in fp32, two NaNs in bf16

unsigned long long* hwm_counter(atom_ctx* c, int node, int dir) {
  return reinterpret_cast<unsigned long long*>(A(c, c->lay.hwm)) + 2 * node + dir;
}

int fwd_impl(atom_ctx* c, int node, int micro) {
  const int par = c->par;
  if (!c->tokens_ok[par]) return fail(c, ATOM_ESTATE, "tokens not set");
  if (node > 0 && !c->fwd_done[par][static_cast<size_t>(node - 1) * c->C + micro])
    return fail(c, ATOM_ESTATE, "input of node " + std::to_string(node) + " not computed");
  int st = prepare_group(c, node, node == c->L + 1);
  if (st != ATOM_OK) return st;
  if (c->ck_host) {
    if (node > 0 && (st = ckpt_ready(c, node - 1, micro)) != ATOM_OK) return st;
    if (node <= c->L) {
      // the node's output goes into a ring entry whose occupant must be settled
      const int e = ck_entry(c, node, micro);
      ckpt_settle(c, e, micro);
      c->ck_holder[e] = node;
      c->ck_wait[e] = 0;
    }
  }
  const size_t pe = (static_cast<size_t>(node) * c->C + micro) * 4;
  if (c->profiling) {
    KCHK(c, fill_word(WS(c, 0), static_cast<int64_t>(c->lay.ws_bytes), HWM_WORD, c->cs));
    HIPCHK(c, hipEventRecord(c->prof_ev[pe], c->cs));
  }
  if (node == 0) st = embed_forward(c, micro);
  else if (node <= c->L) st = block_forward(c, node, micro, false);
  else st = head_forward_backward(c, node, micro);
  if (st != ATOM_OK) return st;
  if (c->profiling) {
    HIPCHK(c, hipEventRecord(c->prof_ev[pe + 1], c->cs));
    KCHK(c, high_water(WS(c, 0), static_cast<int64_t>(c->lay.ws_bytes), HWM_WORD, hwm_counter(c, node, 0), c->cs));
  }
  if (c->ck_host) {
    if (node > 0 && (st = ckpt_used(c, ck_entry(c, node - 1, micro))) != ATOM_OK) return st;
    if (node <= c->L && (st = ckpt_used(c, ck_entry(c, node, micro))) != ATOM_OK) return st;
    if (ck_evicted(c, node) && (st = ckpt_out(c, node, micro)) != ATOM_OK) return st;
  }
  c->fwd_done[par][static_cast<size_t>(node) * c->C + micro] = 1;
  return finish_group_use(c, node);
}

int bwd_impl(atom_ctx* c, int node, int micro) {
  const int par = c->par;
  const size_t k = static_cast<size_t>(node) * c->C + micro;
  const size_t up = static_cast<size_t>(node + 1) * c->C + micro;
  const bool up_done = node + 1 == c->L + 1 ? c->fwd_done[par][up] : c->bwd_done[par][up];
  if (!up_done) return fail(c, ATOM_ESTATE, "gradient of node " + std::to_string(node) + " output not computed");
  if (c->bwd_done[par][k]) return fail(c, ATOM_ESTATE, "backward already done");
  int st = prepare_group(c, node, true);
  if (st != ATOM_OK) return st;
  if (c->ck_host && node > 0 && (st = ckpt_ready(c, node - 1, micro)) != ATOM_OK) return st;
  const size_t pe = (static_cast<size_t>(node) * c->C + micro) * 4 + 2;
  if (c->profiling) {
    KCHK(c, fill_word(WS(c, 0), static_cast<int64_t>(c->lay.ws_bytes), HWM_WORD, c->cs));
    HIPCHK(c, hipEventRecord(c->prof_ev[pe], c->cs));
  }
  st = node == 0 ? embed_backward(c, micro) : block_backward(c, node, micro);
  if (st != ATOM_OK) return st;
  if (c->profiling) {
    HIPCHK(c, hipEventRecord(c->prof_ev[pe + 1], c->cs));
    KCHK(c, high_water(WS(c, 0), static_cast<int64_t>(c->lay.ws_bytes), HWM_WORD, hwm_counter(c, node, 1), c->cs));
  }
  if (c->ck_host && node > 0 && (st = ckpt_used(c, ck_entry(c, node - 1, micro))) != ATOM_OK) return st;
  c->bwd_done[par][k] = 1;
  return finish_group_use(c, node);
}

int swap_out_impl(atom_ctx* c, int par, int g) {
  const int gi = GI(c, par, g);
  if (!group_bwd_complete(c, par, g))
    return fail(c, ATOM_ESTATE, "group " + std::to_string(g) + " backward incomplete");
  const int gs = c->gslot_of[gi];
  uint8_t* gsl = A(c, c->lay.gslots + static_cast<uint64_t>(gs) * c->plan.slot_bytes);
  if (use_accslot(c)) {
    // fp32 accumulation slot -> working dtype in the gradient slot, per tensor
    for (int n = c->plan.first[g]; n <= c->plan.last[g]; ++n)
      for (auto& t : c->tens[n]) {
        const uint64_t in_group = c->node_off[n] - c->group_off[g] + t.offset;
        KCHK(c, convert_f32(c->dt, reinterpret_cast<const float*>(A(c, c->lay.accslot + 2 * in_group)),
                            gsl + in_group, static_cast<int64_t>(t.bytes / c->e), c->cs));
      }
  }
  {
    // the instance's previous copy (two steps back) has finished with its event
    std::unique_lock<std::mutex> l(c->xm);
    c->xcv.wait(l, [c, gi] { return c->d2h_pending[gi] == 0; });
    c->d2h_pending[gi] += 1;
    c->gs_issued[gs] += 1;
  }
  HIPCHK(c, hipEventRecord(c->ev_gready[gi], c->cs));
  uint8_t* dst = c->h_g + c->group_off[g];
  const uint64_t bytes = c->group_bytes[g];
  c->d2h_worker->submit([c, gi, gs, dst, gsl, bytes]() -> std::string {
    // the group's range of the host buffer has been added to the accumulators
    // (copies run in submission order, so an earlier step's copy of the group
    // has already queued its accumulation)
    wait_accum_group(c, gi % c->G);
    std::string err;
    hipError_t e;
    while ((e = hipEventQuery(c->ev_gready[gi])) == hipErrorNotReady) usleep(POLL_US);
    if (e != hipSuccess) err = std::string("waiting for gradients: ") + hipGetErrorString(e);
    if (err.empty()) err = c->dma.copy(dst, gsl, bytes);
    if (err.empty()) {
      std::lock_guard<std::mutex> l(c->acc_m);
      c->acc_q.push_back(gi);
      ++c->acc_pending[gi];
      ++c->acc_busy;
    }
    c->acc_cv.notify_one();
    {
      std::lock_guard<std::mutex> l(c->xm);
      c->gs_freed[gs] += 1;
      c->d2h_pending[gi] -= 1;
    }
    c->xcv.notify_all();
    return err;
  });
  c->stats.d2h_bytes += bytes;
  c->stats.swap_outs += 1;
  return ATOM_OK;
}

// Sum of the step's per-token losses into loss slot `slot` (compute stream).
int reduce_loss(atom_ctx* c, int slot) {
  float* lr = reinterpret_cast<float*>(A(c, c->lay.loss_rows));
  float* lo = reinterpret_cast<float*>(A(c, c->lay.loss_out)) + slot;
  KCHK(c, sum_fixed(lr, static_cast<int64_t>(c->C) * c->N, lo, c->cs));
  return ATOM_OK;
}

int sync_all(atom_ctx* c) {
  // the workers only wait for work already enqueued, so they drain
  const std::string e_in = c->h2d_worker->drain();
  const std::string e_out = c->d2h_worker->drain();
  HIPCHK(c, hipStreamSynchronize(c->cs));
  if (!e_in.empty()) return fail(c, ATOM_EHIP, e_in);
  if (!e_out.empty()) return fail(c, ATOM_EHIP, e_out);
  int st = probe_collect(c);
  if (st != ATOM_OK) return st;
  return wait_accum(c);
}

// n steps with pipelined swapping (see the file comment); losses[s] is the
// mean loss of step s.
int run_steps(atom_ctx* c, const int32_t* tokens, int n, float* losses) {
  const int G = c->G, K = c->K, C = c->C;
  const atom_plan& p = c->plan;
  const int64_t tok_per_step = static_cast<int64_t>(C) * c->B * (c->T + 1);
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  drop_residency(c);
  std::fill(c->slot_owner.begin(), c->slot_owner.end(), -1);
  // with retention and a slot per group, each group is loaded once per call
  const bool keep = c->retain && G <= K;
  c->retain_active = keep;
#define STEP(expr)                  \
  do {                              \
    if ((st = (expr)) != ATOM_OK) { \
      sync_all(c);                  \
      if (keep) {                   \
        c->retain_active = false;   \
        drop_residency(c);          \
      }                             \
      return st;                    \
    }                               \
  } while (0)
  STEP(upload_tokens(c, 0, tokens));
  for (int j = 0; j < std::min(G, K); ++j) STEP(swap_in_impl(c, 0, j));
  for (int s = 0; s < n; ++s) {
    const int par = s & 1, nxt = par ^ 1;
    const bool more = s + 1 < n;
    c->par = par;
    if (keep && s > 0)
      for (int g = 0; g < G; ++g) STEP(hand_over(c, par, g));
    // forward (the head also runs its backward and starts the residual gradient)
    for (int j = 0; j < G; ++j) {
      for (int node = p.first[j]; node <= p.last[j]; ++node)
        for (int m = 0; m < C; ++m) {
          STEP(fwd_impl(c, node, m));
          // host checkpoints: the head was the last reader of input L's entry
          if (c->ck_host && node == c->L + 1 && c->L - CKPT_RING >= 0) STEP(ckpt_restore(c, c->L - CKPT_RING, m));
        }
      if (j + K < G) STEP(swap_in_impl(c, par, j + K));
    }
    STEP(reduce_loss(c, s));
    if (more) STEP(upload_tokens(c, nxt, tokens + (s + 1) * tok_per_step));
    // backward, with reloads; slots the last K groups free take the next step's first groups
    for (int j = G - 1; j >= 0; --j) {
      for (int node = std::min(p.last[j], c->L); node >= p.first[j]; --node)
        for (int m = 0; m < C; ++m) {
          STEP(bwd_impl(c, node, m));
          // host checkpoints: this block was the last reader of input node-1's entry
          if (c->ck_host && node - 1 - CKPT_RING >= 0) STEP(ckpt_restore(c, node - 1 - CKPT_RING, m));
        }
      STEP(swap_out_impl(c, par, j));
      if (j - K >= 0) STEP(swap_in_impl(c, par, j - K));
      else if (more && !keep) STEP(swap_in_impl(c, nxt, K - 1 - j));
    }
  }
#undef STEP
  c->par = 0;
  if (keep) {
    // the next call loads everything again (the host model may change
    // between calls), in the usual slot order
    c->retain_active = false;
    drop_residency(c);
  }
  st = sync_all(c);
  if (st != ATOM_OK) return st;
  if (losses) {
    HIPCHK(c, hipMemcpy(losses, A(c, c->lay.loss_out), n * sizeof(float), hipMemcpyDeviceToHost));
    const float inv = 1.0f / static_cast<float>(static_cast<double>(C) * static_cast<double>(c->N));
    for (int s = 0; s < n; ++s) losses[s] *= inv;
  }
  return ATOM_OK;
}

}  // namespace

// ---------------------------------------------------------------- C ABI
extern "C" {

int atom_ctx_create(const atom_config* cfg, const atom_plan* plan, void* dev_arena, uint64_t arena_bytes,
                    void* compute_stream, atom_ctx** out) {
  if (!out) return ATOM_EINVAL;
  *out = nullptr;
  g_create_error = "invalid argument";
  if (!cfg || !plan || !dev_arena || !compute_stream) return ATOM_EINVAL;
  if (!check_config(*cfg).empty()) return ATOM_EINVAL;
  const int n = cfg->n_layer + 2;
  if (plan->n_nodes != n || plan->n_groups < 1 || plan->n_groups > n || plan->n_slots < 1 ||
      plan->n_slots > plan->n_groups || plan->accum != cfg->accum)
    return ATOM_EINVAL;
  if (plan->first[0] != 0 || plan->last[plan->n_groups - 1] != n - 1) return ATOM_EINVAL;
  for (int g = 0; g < plan->n_groups; ++g) {
    if (plan->first[g] > plan->last[g]) return ATOM_EINVAL;
    if (g > 0 && plan->first[g] != plan->last[g - 1] + 1) return ATOM_EINVAL;
  }
  if (plan->n_slots < std::min(plan->n_groups, 2)) return ATOM_EINVAL;
  if (plan->n_gslots < 2 || plan->n_gslots > ATOM_MAX_GSLOTS) return ATOM_EINVAL;
  if (reinterpret_cast<uintptr_t>(dev_arena) & (ALIGN - 1)) return ATOM_EINVAL;

  atom_ctx* c = new atom_ctx();
  c->cfg = *cfg;
  c->plan = *plan;
  c->L = cfg->n_layer;
  c->G = plan->n_groups;
  c->K = plan->n_slots;
  c->C = cfg->accum;
  c->H = cfg->n_head;
  c->d = cfg->d_model;
  c->dh = c->d / c->H;
  c->f = cfg->d_mlp;
  c->V = cfg->vocab;
  c->Vp = vocab_padded(cfg->vocab);
  c->B = cfg->batch;
  c->T = cfg->seq_len;
  c->N = static_cast<int64_t>(c->B) * c->T;
  c->dt = cfg->dtype == ATOM_BF16 ? DT_BF16 : DT_F32;
  c->e = elem_bytes(*cfg);
  c->ck_host = cfg->ckpt == ATOM_CKPT_HOST;

  // host ranges per node and group
  c->tens.resize(n);
  c->node_off.resize(n);
  c->node_bytes.resize(n);
  c->node_group.resize(n);
  uint64_t off = 0;
  for (int i = 0; i < n; ++i) {
    c->node_off[i] = off;
    c->node_bytes[i] = node_tensors(*cfg, i, &c->tens[i]);
    off += c->node_bytes[i];
  }
  c->model_bytes = off;
  uint64_t smax = 0;
  c->group_off.resize(c->G);
  c->group_bytes.resize(c->G);
  c->group_ranges.resize(c->G);
  for (int g = 0; g < c->G; ++g) {
    c->group_off[g] = c->node_off[plan->first[g]];
    uint64_t b = 0;
    for (int i = plan->first[g]; i <= plan->last[g]; ++i) {
      c->node_group[i] = g;
      b += c->node_bytes[i];
      for (auto& t : c->tens[i])
        c->group_ranges[g].push_back({(c->node_off[i] + t.offset) / c->e, t.bytes / c->e});
    }
    c->group_bytes[g] = b;
    smax = std::max(smax, b);
  }
  if (smax > plan->slot_bytes) {
    delete c;
    return ATOM_EINVAL;
  }
  c->lay = arena_layout(*cfg, plan->slot_bytes, plan->n_slots, plan->n_gslots);
  c->R = plan->n_gslots;
  c->gs_issued.assign(c->R, 0);
  c->gs_freed.assign(c->R, 0);
  if (arena_bytes < c->lay.arena_bytes) {
    delete c;
    return ATOM_EBUDGET;
  }
  c->arena = static_cast<uint8_t*>(dev_arena);
  c->cs = static_cast<hipStream_t>(compute_stream);

  // pinned host model, two gradient buffers, token staging
  const int64_t tok_words = static_cast<int64_t>(c->C) * (5 * c->N + 1);
  struct PinnedBuf {
    uint8_t** p;
    uint64_t bytes;
    const char* what;
  };
  const PinnedBuf bufs[] = {{&c->h_w, c->model_bytes, "host weights"},
                            {&c->h_g, c->model_bytes, "host gradients"},
                            {reinterpret_cast<uint8_t**>(&c->h_tok[0]), static_cast<uint64_t>(tok_words) * 4,
                             "token staging (even steps)"},
                            {reinterpret_cast<uint8_t**>(&c->h_tok[1]), static_cast<uint64_t>(tok_words) * 4,
                             "token staging (odd steps)"}};
  for (const auto& b : bufs) {
    const hipError_t e = hipHostMalloc(reinterpret_cast<void**>(b.p), b.bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
      *b.p = nullptr;
      g_create_error = std::string("hipHostMalloc of ") + std::to_string(b.bytes) + " bytes for " + b.what +
                       " failed: " + hipGetErrorString(e);
      atom_ctx_destroy(c);
      return ATOM_ENOMEM_HOST;
    }
  }
  if (c->ck_host) {
    const uint64_t ck_bytes = static_cast<uint64_t>(std::max(1, ckpt_evicted(*cfg))) * c->C * c->lay.ckpt_bytes_each;
    const hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&c->h_ck), ck_bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
      c->h_ck = nullptr;
      g_create_error = "hipHostMalloc of " + std::to_string(ck_bytes) + " bytes for host checkpoints failed: " +
                       hipGetErrorString(e);
      atom_ctx_destroy(c);
      return ATOM_ENOMEM_HOST;
    }
  }
  const uint64_t n_elem = c->model_bytes / c->e;
  if (posix_memalign(reinterpret_cast<void**>(&c->h_acc), 4096, n_elem * 4) != 0) {
    c->h_acc = nullptr;
    g_create_error = "allocation of " + std::to_string(n_elem * 4) + " bytes for the fp32 accumulators failed";
    atom_ctx_destroy(c);
    return ATOM_ENOMEM_HOST;
  }
  // accumulation threads: the cores minus two for the calling thread and the
  // transfer workers (at most 16; the sum is bound by host memory bandwidth)
  unsigned hw = std::thread::hardware_concurrency();
  int nthreads = static_cast<int>(std::min(16u, std::max(1u, hw > 3 ? hw - 2 : 1u)));
  c->pool = new HostPool(nthreads);
  {
    // zero host buffers in parallel
    const uint64_t nb = c->model_bytes;
    c->pool->run([&](int ti) {
      const int nt = c->pool->size();
      const uint64_t lo = nb * ti / nt, hi = nb * (ti + 1) / nt;
      memset(c->h_w + lo, 0, hi - lo);
      memset(c->h_g + lo, 0, hi - lo);
      const uint64_t elo = n_elem * ti / nt, ehi = n_elem * (ti + 1) / nt;
      memset(c->h_acc + elo, 0, (ehi - elo) * 4);
    });
  }
  const int GI2 = 2 * c->G;
  c->slot_owner.assign(c->K, -1);
  c->resident.assign(GI2, 0);
  c->need_wait.assign(GI2, 0);
  c->gclaimed.assign(GI2, 0);
  c->lastuse_recorded.assign(GI2, 0);
  c->acc_pending.assign(GI2, 0);
  c->load_req.assign(GI2, 0);
  c->load_done.assign(GI2, 0);
  c->d2h_pending.assign(GI2, 0);
  c->gslot_of.assign(GI2, 0);
  {
    const size_t ring = static_cast<size_t>(CKPT_RING) * c->C, keys = static_cast<size_t>(c->L + 1) * c->C;
    c->ck_holder.assign(ring, -1);
    c->ck_wait.assign(ring, 0);
    c->cku_recorded.assign(ring, 0);
    c->ck_out_req.assign(keys, 0);
    c->ck_out_done.assign(keys, 0);
    c->ck_in_req.assign(keys, 0);
    c->ck_in_done.assign(keys, 0);
  }
  for (int par = 0; par < 2; ++par) {
    c->fwd_done[par].assign(static_cast<size_t>(n) * c->C, 0);
    c->bwd_done[par].assign(static_cast<size_t>(n) * c->C, 0);
    c->n_uniq[par].assign(c->C, 0);
  }
  auto mk = [&](std::vector<hipEvent_t>& v, unsigned flags, size_t count) {
    v.assign(count, nullptr);
    for (auto& e : v)
      if (hipEventCreateWithFlags(&e, flags) != hipSuccess) return false;
    return true;
  };
  const size_t n_ring = c->ck_host ? static_cast<size_t>(CKPT_RING) * c->C : 0;
  if (!mk(c->ev_lastuse, hipEventDisableTiming, GI2) || !mk(c->ev_gready, hipEventDisableTiming, GI2) ||
      !mk(c->ev_ckw, hipEventDisableTiming, n_ring) || !mk(c->ev_cku, hipEventDisableTiming, n_ring) ||
      hipEventCreateWithFlags(&c->ev_tok[0], hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_tok[1], hipEventDisableTiming) != hipSuccess) {
    g_create_error = "event creation failed";
    atom_ctx_destroy(c);
    return ATOM_EHIP;
  }
  c->probe_ev.assign(2 * PROBE_MAX, nullptr);
  c->probe_flop.assign(PROBE_MAX, 0.0);
  c->probe_byte.assign(PROBE_MAX, 0.0);
  for (auto& e : c->probe_ev)
    if (hipEventCreate(&e) != hipSuccess) {
      atom_ctx_destroy(c);
      return ATOM_EHIP;
    }
  {
    int dev = 0;
    std::string e = hipGetDevice(&dev) == hipSuccess ? c->dma.init(dev, true) : "hipGetDevice failed";
    if (e.empty()) e = c->dma_in.init(dev, false);
    if (e.empty()) e = c->dma.check_known(c->arena, "the device arena");
    if (e.empty()) e = c->dma.check_known(c->h_w, "the pinned host model");
    if (!e.empty()) {
      g_create_error = "DMA engines: " + e;
      atom_ctx_destroy(c);
      return ATOM_EHIP;
    }
  }
  c->acc_thread = std::thread(acc_loop, c);
  c->h2d_worker = new Worker();
  c->d2h_worker = new Worker();
  *out = c;
  return ATOM_OK;
}

void atom_ctx_destroy(atom_ctx* c) {
  if (!c) return;
  // workers first (gradient copies hand work to the accumulation thread)
  if (c->h2d_worker) (void)c->h2d_worker->drain();
  if (c->d2h_worker) (void)c->d2h_worker->drain();
  delete c->h2d_worker;
  delete c->d2h_worker;
  if (c->cs) (void)hipStreamSynchronize(c->cs);
  if (c->acc_thread.joinable()) {
    {
      std::lock_guard<std::mutex> l(c->acc_m);
      c->acc_stop = true;
    }
    c->acc_cv.notify_all();
    c->acc_thread.join();
  }
  for (auto* v : {&c->ev_lastuse, &c->ev_gready, &c->probe_ev, &c->ev_ckw, &c->ev_cku, &c->prof_ev})
    for (auto e : *v)
      if (e) (void)hipEventDestroy(e);
  for (auto e : c->ev_tok)
    if (e) (void)hipEventDestroy(e);
  delete c->pool;
  if (c->h_w) (void)hipHostFree(c->h_w);
  if (c->h_g) (void)hipHostFree(c->h_g);
  for (auto p : c->h_tok)
    if (p) (void)hipHostFree(p);
  if (c->h_ck) (void)hipHostFree(c->h_ck);
  free(c->h_acc);
  free(c->h_master);
  free(c->h_m);
  free(c->h_v);
  delete c;
}

int atom_host_tensor(atom_ctx* c, int32_t node, int32_t which, void** ptr, uint64_t* bytes) {
  if (!c || !ptr || node < 0 || node > c->L + 1 || which < 0 || which > 2) return fail(c, ATOM_EINVAL, "bad argument");
  const uint64_t off = c->node_off[node];
  if (which == 0) *ptr = c->h_w + off;
  else if (which == 1) *ptr = c->h_acc + off / c->e;
  else *ptr = c->h_g + off;
  if (bytes) *bytes = which == 1 ? c->node_bytes[node] / c->e * 4 : c->node_bytes[node];
  return ATOM_OK;
}

int atom_zero_grads(atom_ctx* c) {
  if (!c) return ATOM_EINVAL;
  // gradient copies still in flight (e.g. from a manual atom_swap_out) end
  // in an accumulation: wait for all of them, not only the queued ones
  int s = sync_all(c);
  if (s != ATOM_OK) return s;
  memset(c->h_acc, 0, c->model_bytes / c->e * 4);
  return ATOM_OK;
}

int atom_set_tokens(atom_ctx* c, const int32_t* tokens) {
  if (!c || !tokens) return fail(c, ATOM_EINVAL, "null tokens");
  c->par = 0;
  int st = upload_tokens(c, 0, tokens);
  if (st != ATOM_OK) return st;
  HIPCHK(c, hipStreamSynchronize(c->cs));
  drop_residency(c);
  return ATOM_OK;
}

int atom_swap_in(atom_ctx* c, int32_t g) {
  if (!c || g < 0 || g >= c->G) return fail(c, ATOM_EINVAL, "bad group");
  return swap_in_impl(c, c->par, g);
}

int atom_block_fwd(atom_ctx* c, int32_t node, int32_t micro) {
  if (!c || node < 0 || node > c->L + 1 || micro < 0 || micro >= c->C) return fail(c, ATOM_EINVAL, "bad node/micro");
  return fwd_impl(c, node, micro);
}

int atom_block_bwd(atom_ctx* c, int32_t node, int32_t micro) {
  if (!c || node < 0 || node > c->L || micro < 0 || micro >= c->C) return fail(c, ATOM_EINVAL, "bad node/micro");
  return bwd_impl(c, node, micro);
}

int atom_swap_out(atom_ctx* c, int32_t g) {
  if (!c || g < 0 || g >= c->G) return fail(c, ATOM_EINVAL, "bad group");
  return swap_out_impl(c, c->par, g);
}

int atom_sync(atom_ctx* c, float* loss_out) {
  if (!c) return ATOM_EINVAL;
  if (loss_out) {
    int st = reduce_loss(c, 0);
    if (st != ATOM_OK) return st;
    float v = 0.f;
    HIPCHK(c, hipMemcpyAsync(&v, A(c, c->lay.loss_out), 4, hipMemcpyDeviceToHost, c->cs));
    HIPCHK(c, hipStreamSynchronize(c->cs));
    *loss_out = v / static_cast<float>(static_cast<double>(c->C) * static_cast<double>(c->N));
  }
  return sync_all(c);
}

int atom_steps(atom_ctx* c, const int32_t* tokens, int32_t n, float* losses) {
  if (!c || !tokens || n < 1 || n > MAX_STEPS_PER_CALL) return fail(c, ATOM_EINVAL, "bad step count");
  const int64_t total = static_cast<int64_t>(n) * c->C * c->B * (c->T + 1);
  for (int64_t i = 0; i < total; ++i)
    if (tokens[i] < 0 || tokens[i] >= c->V) return fail(c, ATOM_EINVAL, "token id out of range");
  auto t0 = std::chrono::steady_clock::now();
  c->stats = atom_stats{};
  c->acc_seconds = 0;
  const int st = run_steps(c, tokens, n, losses);
  c->stats.step_s = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count() / n;
  c->stats.host_accum_s = c->acc_seconds / n;
  return st;
}

int atom_set_retention(atom_ctx* c, int32_t on) {
  if (!c) return ATOM_EINVAL;
  c->retain = on != 0;
  return ATOM_OK;
}

int atom_step(atom_ctx* c, const int32_t* tokens, float* loss_out) {
  float loss = 0.f;
  const int st = atom_steps(c, tokens, 1, &loss);
  if (st == ATOM_OK && loss_out) *loss_out = loss;
  return st;
}

int atom_probe_gemm(atom_ctx* c, int32_t akc, int32_t bkc, int32_t epi) {
  if (!c) return ATOM_EINVAL;
  HIPCHK(c, hipStreamSynchronize(c->cs));
  int st = probe_collect(c);
  if (st != ATOM_OK) return st;
  c->probe_akc = akc ? 1 : 0;
  c->probe_bkc = bkc ? 1 : 0;
  c->probe_epi = epi;
  c->probe_launches = 0;
  c->probe_seconds = 0;
  c->probe_flops = 0;
  c->probe_bytes = 0;
  return ATOM_OK;
}

int atom_probe_read(atom_ctx* c, int64_t* launches, double* seconds, double* flops, double* bytes) {
  if (!c) return ATOM_EINVAL;
  HIPCHK(c, hipStreamSynchronize(c->cs));
  int st = probe_collect(c);
  if (st != ATOM_OK) return st;
  if (launches) *launches = c->probe_launches;
  if (seconds) *seconds = c->probe_seconds;
  if (flops) *flops = c->probe_flops;
  if (bytes) *bytes = c->probe_bytes;
  return ATOM_OK;
}

int atom_link_bench(atom_ctx* c, uint64_t bytes, int32_t iters, double* h2d, double* d2h, double* bidir) {
  if (!c || iters < 1) return ATOM_EINVAL;
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  const uint64_t region = static_cast<uint64_t>(c->K) * c->plan.slot_bytes;
  // two device halves so both directions can run at once on distinct memory
  const uint64_t n = std::min<uint64_t>(std::min<uint64_t>(bytes, region / 2), c->model_bytes) / 256 * 256;
  if (n == 0) return fail(c, ATOM_EINVAL, "no room for the link benchmark");
  uint8_t* dev0 = A(c, c->lay.wslots);
  uint8_t* dev1 = dev0 + n;
  std::string err;
  // the engines a step uses, each direction on its own thread
  std::string err_in;
  auto timed = [&](bool up, bool down) -> double {
    auto t0 = std::chrono::steady_clock::now();
    std::thread t_in([&] {
      for (int i = 0; i < iters && up && err_in.empty(); ++i) err_in = c->dma_in.copy(dev0, c->h_w, n);
    });
    for (int i = 0; i < iters && down && err.empty(); ++i) err = c->dma.copy(c->h_g, dev1, n);
    t_in.join();
    return std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  };
  timed(true, true);  // warm-up
  const double tu = timed(true, false), td = timed(false, true), tb = timed(true, true);
  // slots no longer hold any group's weights
  std::fill(c->slot_owner.begin(), c->slot_owner.end(), -1);
  drop_residency(c);
  if (err.empty()) err = err_in;
  if (!err.empty()) return fail(c, ATOM_EHIP, err);
  const double gb = static_cast<double>(n) * iters / 1e9;
  if (h2d) *h2d = gb / tu;
  if (d2h) *d2h = gb / td;
  if (bidir) *bidir = 2.0 * gb / tb;
  return ATOM_OK;
}

int atom_optimizer_init(atom_ctx* c) {
  if (!c) return ATOM_EINVAL;
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  const uint64_t n = c->model_bytes / c->e;
  float** bufs[] = {&c->h_master, &c->h_m, &c->h_v};
  for (float** b : bufs)
    if (!*b && posix_memalign(reinterpret_cast<void**>(b), 4096, n * 4) != 0) {
      *b = nullptr;
      return fail(c, ATOM_ENOMEM_HOST, "allocation of the optimizer state failed");
    }
  c->pool->run([&](int ti) {
    const int nt = c->pool->size();
    const uint64_t lo = n * ti / nt, hi = n * (ti + 1) / nt;
    for (uint64_t i = lo; i < hi; ++i) {
      if (c->dt == DT_BF16) {
        const uint32_t u = static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(c->h_w)[i]) << 16;
        memcpy(&c->h_master[i], &u, 4);
      } else {
        c->h_master[i] = reinterpret_cast<const float*>(c->h_w)[i];
      }
    }
    memset(c->h_m + lo, 0, (hi - lo) * 4);
    memset(c->h_v + lo, 0, (hi - lo) * 4);
  });
  return ATOM_OK;
}

namespace {
// fp32 -> bf16 bits, round to nearest even (finite inputs).
inline uint16_t host_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
}  // namespace

int atom_optimizer_step(atom_ctx* c, const atom_adamw* hp, float grad_scale, int32_t step) {
  if (!c || !hp || step < 1) return fail(c, ATOM_EINVAL, "bad optimizer arguments");
  if (!c->h_master) return fail(c, ATOM_ESTATE, "atom_optimizer_init was not called");
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  // per-tensor element ranges with their decay flag
  struct Seg {
    uint64_t off, n;
    bool decay;
  };
  std::vector<Seg> segs;
  uint64_t total = 0;
  for (int node = 0; node <= c->L + 1; ++node)
    for (const auto& t : c->tens[node]) {
      const bool decay = t.name == "w_qkv" || t.name == "w_o" || t.name == "w_fc" || t.name == "w_pr" ||
                         t.name == "w_head";
      segs.push_back({(c->node_off[node] + t.offset) / c->e, t.bytes / c->e, decay});
      total += t.bytes / c->e;
    }
  const float lr = hp->lr, b1 = hp->beta1, b2 = hp->beta2, eps = hp->eps, wd = hp->weight_decay;
  // 1 - beta and the bias corrections in double: in fp32 they would lose
  // most of their digits to cancellation (1 - 0.999^2 keeps about three)
  const double b1d = b1, b2d = b2;
  const float c1 = static_cast<float>(1.0 - b1d), c2 = static_cast<float>(1.0 - b2d);
  const float bc1 = static_cast<float>(1.0 - std::pow(b1d, step));
  const float bc2 = static_cast<float>(1.0 - std::pow(b2d, step));
  const bool bf = c->dt == DT_BF16;
  c->pool->run([&](int ti) {
    const int nt = c->pool->size();
    const uint64_t lo = total * ti / nt, hi = total * (ti + 1) / nt;
    uint64_t pos = 0;
    for (const Seg& sg : segs) {
      const uint64_t a = std::max(lo, pos), b = std::min(hi, pos + sg.n);
      if (a < b) {
        const float keep = sg.decay ? 1.f - lr * wd : 1.f;
        for (uint64_t k = sg.off + (a - pos), e = sg.off + (b - pos); k < e; ++k) {
          const float g = c->h_acc[k] * grad_scale;
          const float m = b1 * c->h_m[k] + c1 * g;
          const float v = b2 * c->h_v[k] + c2 * g * g;
          c->h_m[k] = m;
          c->h_v[k] = v;
          const float p = c->h_master[k] * keep - lr * (m / bc1) / (std::sqrt(v / bc2) + eps);
          c->h_master[k] = p;
          if (bf) reinterpret_cast<uint16_t*>(c->h_w)[k] = host_bf16(p);
          else reinterpret_cast<float*>(c->h_w)[k] = p;
          c->h_acc[k] = 0.f;
        }
      }
      pos += sg.n;
    }
  });
  return ATOM_OK;
}

int atom_profile_nodes(atom_ctx* c, const int32_t* tokens, atom_node_cost* out, int32_t n) {
  if (!c || !tokens || !out || n != c->L + 2) return fail(c, ATOM_EINVAL, "bad argument");
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  // copy times of each node alone on the step's DMA engines (best of three)
  uint8_t* dev = A(c, c->lay.wslots);
  for (int i = 0; i < n; ++i) {
    double best_in = 1e30, best_out = 1e30;
    for (int rep = 0; rep < 3; ++rep) {
      auto t0 = std::chrono::steady_clock::now();
      std::string e = c->dma_in.copy(dev, c->h_w + c->node_off[i], c->node_bytes[i]);
      auto t1 = std::chrono::steady_clock::now();
      if (e.empty()) e = c->dma.copy(c->h_g + c->node_off[i], dev, c->node_bytes[i]);
      auto t2 = std::chrono::steady_clock::now();
      if (!e.empty()) return fail(c, ATOM_EHIP, e);
      best_in = std::min(best_in, std::chrono::duration<double>(t1 - t0).count());
      best_out = std::min(best_out, std::chrono::duration<double>(t2 - t1).count());
    }
    out[i].weight_bytes = c->node_bytes[i];
    out[i].t_load = best_in;
    out[i].t_store = best_out;
  }
  std::fill(c->slot_owner.begin(), c->slot_owner.end(), -1);
  drop_residency(c);
  // kernel times of each node in one step of the context's plan
  const size_t ne = static_cast<size_t>(n) * c->C * 4;
  if (c->prof_ev.size() != ne) {
    for (auto e : c->prof_ev)
      if (e) (void)hipEventDestroy(e);
    c->prof_ev.assign(ne, nullptr);
    for (auto& e : c->prof_ev) HIPCHK(c, hipEventCreate(&e));
  }
  // one step to warm up (the first launch of a kernel loads its code), then
  // the timed one
  st = run_steps(c, tokens, 1, nullptr);
  if (st != ATOM_OK) return st;
  KCHK(c, fill_zero(A(c, c->lay.hwm), static_cast<int64_t>(n) * 2 * 8, c->cs));
  c->profiling = true;
  c->stats = atom_stats{};
  st = run_steps(c, tokens, 1, nullptr);
  c->profiling = false;
  if (st != ATOM_OK) return st;
  std::vector<unsigned long long> hwm(static_cast<size_t>(n) * 2);
  HIPCHK(c, hipMemcpy(hwm.data(), A(c, c->lay.hwm), hwm.size() * 8, hipMemcpyDeviceToHost));
  const uint64_t cut = static_cast<uint64_t>(c->N) * c->d * 4;
  for (int i = 0; i < n; ++i) {
    double f = 0, b = 0;
    for (int m = 0; m < c->C; ++m) {
      const size_t pe = (static_cast<size_t>(i) * c->C + m) * 4;
      float ms = 0.f;
      HIPCHK(c, hipEventElapsedTime(&ms, c->prof_ev[pe], c->prof_ev[pe + 1]));
      f += ms * 1e-3;
      if (i <= c->L) {
        HIPCHK(c, hipEventElapsedTime(&ms, c->prof_ev[pe + 2], c->prof_ev[pe + 3]));
        b += ms * 1e-3;
      }
    }
    out[i].t_fwd = f / c->C;
    out[i].t_bwd = b / c->C;
    out[i].mem_bytes = 16 * std::max(hwm[2 * i], hwm[2 * i + 1]);
    out[i].cut_bytes = i <= c->L ? cut : 4;
  }
  return ATOM_OK;
}

int atom_ctx_config(const atom_ctx* c, atom_config* cfg, atom_plan* plan) {
  if (!c) return ATOM_EINVAL;
  if (cfg) *cfg = c->cfg;
  if (plan) *plan = c->plan;
  return ATOM_OK;
}

int atom_get_stats(atom_ctx* c, atom_stats* out) {
  if (!c || !out) return ATOM_EINVAL;
  *out = c->stats;
  return ATOM_OK;
}

const char* atom_last_error(const atom_ctx* c) {
  if (!c) return g_create_error.c_str();
  return c->err.c_str();
}

}  // extern "C"
