// Internal state of a swapped-step context (struct atom_ctx) and what the
// runtime's units share: nodes.cpp composes a node's forward and backward
// from the kernels, schedule.cpp moves weights, gradients and checkpoints
// and runs whole steps, host_accum.cpp adds gradients into the host
// accumulators and runs the host optimizer, runtime.cpp is the C ABI.
#pragma once

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
  // Runs fn(i) for i in [0, active) (active <= size(); the other threads
  // skip the job); returns when all are done.  Not reentrant (one job at a
  // time): during steps only the accumulation thread calls it; the context's
  // other users (zeroing, optimizer) first drain every copy and the
  // accumulation queue (sync_all), so no two callers overlap.
  void run(const std::function<void(int)>& fn, int active) {
    {
      std::lock_guard<std::mutex> l(m_);
      fn_ = &fn;
      active_ = std::max(1, std::min(active, n_));
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
      bool run_it;
      {
        std::unique_lock<std::mutex> l(m_);
        cv_.wait(l, [&] { return gen_ != seen; });
        seen = gen_;
        if (stop_) return;
        f = fn_;
        run_it = i < active_;
      }
      if (run_it) (*f)(i);
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
  int active_ = 1;
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

  // Row-sparse embedding transfers (atom_set_embedding_rows): a step's
  // token ids are remapped to the positions of the distinct ids it uses
  // (ascending); group 0's swap-in copies only those rows of wte, packed at
  // the start of the slot's wte region, and its swap-out only their
  // gradients, packed the same way in the gradient slot and in h_g; the host
  // accumulation adds each packed row to its own row.
  bool emb_rows_on = false;
  bool emb_packed[2] = {false, false};  // the parity's tokens address packed rows
  std::vector<int32_t> emb_rows[2];     // the parity's distinct token ids, ascending
  std::vector<int32_t> acc_rows0;       // rows of group 0's queued accumulation (empty: dense)
  std::vector<int32_t> g_rows0;         // rows of the packed node-0 gradient in h_g (empty: dense)
  uint8_t* h_emb_stage = nullptr;       // pinned staging of the packed rows of a swap-in

  // per-step validation state, by parity
  bool tokens_ok[2] = {false, false};
  std::vector<char> fwd_done[2], bwd_done[2];  // [node][micro]
  std::vector<int> n_uniq[2];                  // per micro
  int32_t* h_tok[2] = {nullptr, nullptr};      // pinned token staging
  hipEvent_t ev_tok[2] = {nullptr, nullptr};
  bool tok_recorded[2] = {false, false};

  // host accumulation (acc_threads of the pool's threads while steps run,
  // all of them for work that runs alone)
  HostPool* pool = nullptr;
  int acc_threads = 1;
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
  // weights and the two AdamW moments, element-indexed like h_w
  float* h_master = nullptr;
  float* h_m = nullptr;
  float* h_v = nullptr;
  bool opt_pinned = false;  // the three buffers are pinned (else pageable)
  // update armed for the next step call (atom_optimizer_arm): its last step's
  // swap-outs carry ACC_UPDATE, and the accumulation thread updates each such
  // group right after adding its gradients (upd_capture: set while that
  // step's backward is being enqueued)
  bool upd_armed = false, upd_capture = false;
  atom_adamw upd_hp{};
  float upd_scale = 1.f;
  int32_t upd_step = 0;
  int upd_groups = 0;        // groups the current call has updated
  double upd_seconds = 0;    // host time of those updates

  // node profile (atom_profile_nodes): events around each node's forward
  // and backward, per micro-batch
  bool profiling = false;
  std::vector<hipEvent_t> prof_ev;  // [node][micro][fwd, bwd][begin, end]

  atom_stats stats{};
  std::string err;
};

namespace atom {
namespace rt {

constexpr int PROBE_MAX = 4096;  // GEMM launches a probe records per call

inline int fail(atom_ctx* c, int code, const std::string& msg) {
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

// wte is node 0's first tensor: its byte offset in node 0 (= in group 0),
// its bytes, and the bytes of one row.
inline uint64_t wte_off(atom_ctx* c) { return c->tens[0][0].offset; }
inline uint64_t wte_bytes(atom_ctx* c) { return c->tens[0][0].bytes; }
inline uint64_t wte_row_bytes(atom_ctx* c) { return static_cast<uint64_t>(c->d) * c->e; }
// Rows of wte the kernels of a step of parity par address.
inline int emb_vocab(atom_ctx* c, int par) {
  return c->emb_packed[par] ? static_cast<int>(c->emb_rows[par].size()) : c->V;
}

// Gradient target of a tensor: fp32 accumulation slot (bf16 with C > 1) or
// the group's gradient slot in the working dtype.
struct GradTarget {
  void* p;
  int dtype;  // DT_F32 or DT_BF16
  bool accumulate;
};

inline bool use_accslot(atom_ctx* c) { return c->dt == DT_BF16 && c->C > 1; }

// ----------------------------------------------------- shared functions
// nodes.cpp: a node's forward and backward composed from the kernels
float* ckpt_ptr(atom_ctx* c, int idx, int micro);
const void* wptr(atom_ctx* c, int node, int t);
GradTarget gptr(atom_ctx* c, int node, int t, int micro);
int prepare_group(atom_ctx* c, int node, bool grads);
int finish_group_use(atom_ctx* c, int node);
int probe_collect(atom_ctx* c);
int block_forward(atom_ctx* c, int node, int micro, bool recompute);
int block_backward(atom_ctx* c, int node, int micro);
int head_forward_backward(atom_ctx* c, int node, int micro);
int embed_forward(atom_ctx* c, int micro);
int embed_backward(atom_ctx* c, int micro);

// host_accum.cpp: host gradient accumulation (and the optimizer's update)
constexpr int ACC_UPDATE = 1 << 24;  // flag on a queued instance: update the group after adding
void acc_loop(atom_ctx* c);
void adamw_nodes(atom_ctx* c, int first, int last, const atom_adamw& hp, float grad_scale, int32_t step, int nt);
int wait_accum(atom_ctx* c);
void wait_accum_group(atom_ctx* c, int g);

// schedule.cpp: residency, transfers, checkpoints and whole steps
bool group_bwd_complete(atom_ctx* c, int par, int g);
void reset_step_state(atom_ctx* c, int par);
void drop_residency(atom_ctx* c);
int upload_tokens(atom_ctx* c, int par, const int32_t* tokens);
int swap_in_impl(atom_ctx* c, int par, int g);
int fwd_impl(atom_ctx* c, int node, int micro);
int bwd_impl(atom_ctx* c, int node, int micro);
int swap_out_impl(atom_ctx* c, int par, int g);
int reduce_loss(atom_ctx* c, int slot);
int sync_all(atom_ctx* c);
int run_steps(atom_ctx* c, const int32_t* tokens, int n, float* losses);

}  // namespace rt
}  // namespace atom
