// C ABI of the swapped step: context creation (pinned host model, arena
// layout, DMA engines and worker threads), the per-group calls, whole steps,
// measurement hooks (GEMM probe, link benchmark, node profile) and stats.
#include <sched.h>

#include "context.h"

using namespace atom::rt;

namespace {

// Failure text of the last atom_ctx_create on this thread (no context exists
// to hold it).
thread_local std::string g_create_error;

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
  // host threads: the CPUs this process may run on, less two for the
  // calling thread and the transfer workers, at most 16.  Work that runs
  // alone (zeroing, the optimizer step) uses all of them.  The accumulation
  // that runs beside the step's copies uses six fewer: the sum is bound by
  // host memory bandwidth, so more threads add no speed and take bandwidth
  // from the DMA engines' copies (6.7B pipelined step with 14 threads on 16
  // CPUs: 302 ms, also at nice 10; with 8-10 threads 286-288 ms, the same
  // accumulation time; with 4, too few to keep up, 324 ms).
  cpu_set_t cpus;
  const int n_cpu = sched_getaffinity(0, sizeof(cpus), &cpus) == 0 ? CPU_COUNT(&cpus)
                                                                   : static_cast<int>(std::thread::hardware_concurrency());
  c->pool = new HostPool(std::max(1, std::min(16, n_cpu - 2)));
  c->acc_threads = std::max(1, std::min(16, n_cpu - 6));
  {
    // zero host buffers in parallel
    const uint64_t nb = c->model_bytes;
    const int nt = c->pool->size();
    c->pool->run([&](int ti) {
      const uint64_t lo = nb * ti / nt, hi = nb * (ti + 1) / nt;
      memset(c->h_w + lo, 0, hi - lo);
      memset(c->h_g + lo, 0, hi - lo);
      const uint64_t elo = n_elem * ti / nt, ehi = n_elem * (ti + 1) / nt;
      memset(c->h_acc + elo, 0, (ehi - elo) * 4);
    }, nt);
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
  if (c->h_emb_stage) (void)hipHostFree(c->h_emb_stage);
  free(c->h_acc);
  for (float* p : {c->h_master, c->h_m, c->h_v}) {
    if (p && c->opt_pinned) (void)hipHostFree(p);
    else free(p);
  }
  delete c;
}

int atom_host_tensor(atom_ctx* c, int32_t node, int32_t which, void** ptr, uint64_t* bytes) {
  if (!c || !ptr || node < 0 || node > c->L + 1 || which < 0 || which > 5) return fail(c, ATOM_EINVAL, "bad argument");
  if (which >= 3 && !c->h_master) return fail(c, ATOM_ESTATE, "atom_optimizer_init was not called");
  if (which == 2 && node == 0 && !c->g_rows0.empty()) {
    // the last node-0 gradient arrived as packed rows of wte: spread them to
    // their rows (the others are zero), once every copy has landed
    int st = sync_all(c);
    if (st != ATOM_OK) return st;
    uint8_t* w = c->h_g + c->node_off[0] + wte_off(c);
    const uint64_t rb = wte_row_bytes(c), nr = c->g_rows0.size();
    std::vector<uint8_t> packed(w, w + nr * rb);
    memset(w, 0, wte_bytes(c));
    for (uint64_t i = 0; i < nr; ++i) memcpy(w + static_cast<uint64_t>(c->g_rows0[i]) * rb, packed.data() + i * rb, rb);
    c->g_rows0.clear();
  }
  const uint64_t off = c->node_off[node], eoff = off / c->e;
  switch (which) {
    case 0: *ptr = c->h_w + off; break;
    case 1: *ptr = c->h_acc + eoff; break;
    case 2: *ptr = c->h_g + off; break;
    case 3: *ptr = c->h_master + eoff; break;
    case 4: *ptr = c->h_m + eoff; break;
    default: *ptr = c->h_v + eoff; break;
  }
  const bool f32 = which == 1 || which >= 3;
  if (bytes) *bytes = f32 ? c->node_bytes[node] / c->e * 4 : c->node_bytes[node];
  return ATOM_OK;
}

int atom_zero_grads(atom_ctx* c) {
  if (!c) return ATOM_EINVAL;
  // gradient copies still in flight (e.g. from a manual atom_swap_out) end
  // in an accumulation: wait for all of them, not only the queued ones
  int s = sync_all(c);
  if (s != ATOM_OK) return s;
  // on every pool thread (nothing else runs on the pool after sync_all)
  const uint64_t n = c->model_bytes / c->e;
  const int nt = c->pool->size();
  c->pool->run([&](int ti) {
    const uint64_t lo = n * ti / nt, hi = n * (ti + 1) / nt;
    memset(c->h_acc + lo, 0, (hi - lo) * 4);
  }, nt);
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
  c->upd_seconds = 0;
  c->upd_groups = 0;
  const int st = run_steps(c, tokens, n, losses);
  c->stats.step_s = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count() / n;
  c->stats.host_accum_s = c->acc_seconds / n;
  c->stats.host_update_s = c->upd_seconds;
  c->stats.updated_groups = c->upd_groups;
  return st;
}

int atom_set_retention(atom_ctx* c, int32_t on) {
  if (!c) return ATOM_EINVAL;
  if (on && c->emb_rows_on)
    return fail(c, ATOM_ESTATE, "retention across steps needs whole embedding loads (atom_set_embedding_rows off)");
  c->retain = on != 0;
  return ATOM_OK;
}

int atom_set_embedding_rows(atom_ctx* c, int32_t on) {
  if (!c) return ATOM_EINVAL;
  if (on && c->retain)
    return fail(c, ATOM_ESTATE, "row-sparse embedding transfers need retention across steps off");
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  if (on && !c->h_emb_stage) {
    // a step uses at most min(V, C*B*T) distinct ids
    const uint64_t rows = std::min<uint64_t>(c->V, static_cast<uint64_t>(c->C) * c->N);
    const hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&c->h_emb_stage), rows * wte_row_bytes(c),
                                       hipHostMallocDefault);
    if (e != hipSuccess) {
      c->h_emb_stage = nullptr;
      return fail(c, ATOM_ENOMEM_HOST, std::string("hipHostMalloc of the embedding-row staging failed: ") +
                                           hipGetErrorString(e));
    }
  }
  c->emb_rows_on = on != 0;
  // the next step sets its tokens (remapped or not) and loads every group
  drop_residency(c);
  c->tokens_ok[0] = c->tokens_ok[1] = false;
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
  out->opt_state_pinned = c->h_master && c->opt_pinned ? 1 : 0;
  return ATOM_OK;
}

const char* atom_last_error(const atom_ctx* c) {
  if (!c) return g_create_error.c_str();
  return c->err.c_str();
}

}  // extern "C"
