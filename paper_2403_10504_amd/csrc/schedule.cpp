// Schedule of the swapped GPT step: weight-slot residency, the swap engine
// (weights in on one system DMA engine, gradients out on another, each fed
// by its own worker thread that waits on compute-stream events), host
// checkpoints, and whole steps, one at a time or pipelined.
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
#include <system_error>

#include "context.h"

namespace atom {
namespace rt {

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
  for (int64_t m = 0; m < C; ++m)
    for (int64_t b = 0; b < c->B; ++b)
      for (int64_t t = 0; t < T; ++t) {
        inp[m * N + b * T + t] = tokens[(m * c->B + b) * (T + 1) + t];
        tgt[m * N + b * T + t] = tokens[(m * c->B + b) * (T + 1) + t + 1];
      }
  std::vector<int32_t> count(c->V), start(c->V);
  // row-sparse embedding: the step's distinct ids in ascending order, and
  // the inputs remapped to their positions (targets keep the ids)
  c->emb_packed[par] = c->emb_rows_on;
  c->emb_rows[par].clear();
  if (c->emb_rows_on) {
    for (int64_t i = 0; i < C * N; ++i) count[inp[i]] = 1;
    for (int v = 0; v < c->V; ++v)
      if (count[v]) {
        start[v] = static_cast<int32_t>(c->emb_rows[par].size());
        c->emb_rows[par].push_back(v);
      }
    for (int64_t i = 0; i < C * N; ++i) inp[i] = start[inp[i]];
  }
  const int Vr = emb_vocab(c, par);
  for (int64_t m = 0; m < C; ++m) {
    // stable counting sort of token positions by (remapped) token id
    std::fill(count.begin(), count.end(), 0);
    for (int64_t n = 0; n < N; ++n) ++count[inp[m * N + n]];
    int nu = 0, pos = 0;
    for (int v = 0; v < Vr; ++v) {
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
  // row-sparse embedding: group 0 (node 0 first) takes only the step's rows of wte
  std::vector<int32_t> rows;
  if (g == 0 && c->emb_packed[par]) rows = c->emb_rows[par];
  const uint64_t moved = rows.empty() ? bytes : bytes - wte_bytes(c) + rows.size() * wte_row_bytes(c);
  uint64_t gen;
  {
    std::lock_guard<std::mutex> l(c->xm);
    gen = ++c->load_req[gi];
  }
  c->h2d_worker->submit([c, gi, wait_ev, dst, src, bytes, gen, rows]() -> std::string {
    std::string err;
    hipError_t e = hipSuccess;
    if (wait_ev)
      while ((e = hipEventQuery(wait_ev)) == hipErrorNotReady) usleep(POLL_US);
    if (e != hipSuccess) err = std::string("waiting for the slot: ") + hipGetErrorString(e);
    if (err.empty() && rows.empty()) err = c->dma_in.copy(dst, src, bytes);
    if (err.empty() && !rows.empty()) {
      // the rows packed in pinned staging, copied to the start of the wte
      // region; then whatever the group holds around wte
      const uint64_t wo = wte_off(c), rb = wte_row_bytes(c), we = wo + wte_bytes(c);
      // four threads for the copy of the rows (the swap-in waits for it; one
      // thread packs about 15 GB/s)
      const size_t nr = rows.size();
      const int np = nr * rb >= (8u << 20) ? 4 : 1;
      auto pack = [&](int t) {
        for (size_t i = nr * t / np, e = nr * (t + 1) / np; i < e; ++i)
          memcpy(c->h_emb_stage + i * rb, src + wo + static_cast<uint64_t>(rows[i]) * rb, rb);
      };
      std::vector<std::thread> helpers;
      int t_done = np;  // helpers 1..t_done-1 started; the rest is packed here
      for (int t = 1; t < np; ++t) {
        try {
          helpers.emplace_back(pack, t);
        } catch (const std::system_error&) {
          t_done = t;
          break;
        }
      }
      pack(0);
      for (int t = t_done; t < np; ++t) pack(t);
      for (auto& h : helpers) h.join();
      err = c->dma_in.copy(dst + wo, c->h_emb_stage, rows.size() * rb);
      if (err.empty() && wo > 0) err = c->dma_in.copy(dst, src, wo);
      if (err.empty()) err = c->dma_in.copy(dst + we, src + we, bytes - we);
    }
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
  c->stats.h2d_bytes += moved;
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
  // row-sparse embedding: group 0's wte gradient is the step's rows, packed
  std::vector<int32_t> rows;
  if (g == 0 && c->emb_packed[par]) rows = c->emb_rows[par];
  if (use_accslot(c)) {
    // fp32 accumulation slot -> working dtype in the gradient slot, per tensor
    for (int n = c->plan.first[g]; n <= c->plan.last[g]; ++n)
      for (size_t ti = 0; ti < c->tens[n].size(); ++ti) {
        const auto& t = c->tens[n][ti];
        const uint64_t in_group = c->node_off[n] - c->group_off[g] + t.offset;
        const uint64_t tb = n == 0 && ti == 0 && !rows.empty() ? rows.size() * wte_row_bytes(c) : t.bytes;
        KCHK(c, convert_f32(c->dt, reinterpret_cast<const float*>(A(c, c->lay.accslot + 2 * in_group)),
                            gsl + in_group, static_cast<int64_t>(tb / c->e), c->cs));
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
  const uint64_t moved = rows.empty() ? bytes : bytes - wte_bytes(c) + rows.size() * wte_row_bytes(c);
  const int job = gi | (c->upd_capture ? ACC_UPDATE : 0);  // the armed update follows this accumulation
  c->d2h_worker->submit([c, gi, gs, dst, gsl, bytes, job, rows]() -> std::string {
    // the group's range of the host buffer has been added to the accumulators
    // (copies run in submission order, so an earlier step's copy of the group
    // has already queued its accumulation)
    wait_accum_group(c, gi % c->G);
    std::string err;
    hipError_t e;
    while ((e = hipEventQuery(c->ev_gready[gi])) == hipErrorNotReady) usleep(POLL_US);
    if (e != hipSuccess) err = std::string("waiting for gradients: ") + hipGetErrorString(e);
    if (err.empty() && rows.empty()) err = c->dma.copy(dst, gsl, bytes);
    if (err.empty() && !rows.empty()) {
      // the packed rows to the start of h_g's wte region, then the rest of the group
      const uint64_t wo = wte_off(c), we = wo + wte_bytes(c);
      err = c->dma.copy(dst + wo, gsl + wo, rows.size() * wte_row_bytes(c));
      if (err.empty() && wo > 0) err = c->dma.copy(dst, gsl, wo);
      if (err.empty()) err = c->dma.copy(dst + we, gsl + we, bytes - we);
    }
    if (err.empty() && gi % c->G == 0) {
      // no accumulation of group 0 is queued (waited for above): its rows,
      // and the layout of node 0's gradient in h_g, are this copy's
      c->acc_rows0 = rows;
      c->g_rows0 = rows;
    }
    if (err.empty()) {
      std::lock_guard<std::mutex> l(c->acc_m);
      c->acc_q.push_back(job);
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
  c->stats.d2h_bytes += moved;
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
      c->upd_capture = false;       \
      sync_all(c);                  \
      c->upd_armed = false;         \
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
    // backward, with reloads; slots the last K groups free take the next step's first groups.
    // An armed optimizer update rides on the last step's swap-outs: each group's
    // gradients are then complete for the global batch once they are added.
    c->upd_capture = c->upd_armed && !more;
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
  c->upd_capture = false;
  c->par = 0;
  if (keep) {
    // the next call loads everything again (the host model may change
    // between calls), in the usual slot order
    c->retain_active = false;
    drop_residency(c);
  }
  st = sync_all(c);
  if (c->upd_armed) {
    // every group has been updated (or an accumulation failed): the host model
    // changed, so no weights on the device are current
    c->upd_armed = false;
    drop_residency(c);
  }
  if (st != ATOM_OK) return st;
  if (losses) {
    HIPCHK(c, hipMemcpy(losses, A(c, c->lay.loss_out), n * sizeof(float), hipMemcpyDeviceToHost));
    const float inv = 1.0f / static_cast<float>(static_cast<double>(C) * static_cast<double>(c->N));
    for (int s = 0; s < n; ++s) losses[s] *= inv;
  }
  return ATOM_OK;
}

}  // namespace rt
}  // namespace atom
