// Static analysis of the swapped step: node layout, node costs, arena
// layout and the partition search (Section III-D, Algorithm 1).
//
// Readings of the algorithm (the paper's listing is garbled in places):
//  * Search space: with step size 1 the search visits every way to cut the
//    topologically sorted chain into contiguous sub-models; that set is
//    enumerated directly (all 2^(n-1) compositions) for n <= 16 nodes.  For
//    longer chains the search uses the structure of GPT-3 (identical decoder
//    blocks, noted in Section III-D as the knowledge that shrinks the search):
//    the embedding alone or with the first block, the head alone or with the
//    last block, and the remaining blocks in runs of s.
//  * Memory (hard): the executing group and the one being preloaded must be
//    co-resident.  Groups live in equal weight slots of the largest group's
//    size S next to two or more gradient slots (plus a 2S fp32 accumulation
//    slot for bf16 with C > 1) and the reserved memory.  A node's working
//    memory m_i is recomputed from its input checkpoint in the backward, so
//    one workspace serves every node in turn: the reserve holds max m_i, not
//    a sum over a sub-model.
//  * Overlap: C * t^f(g_j) >= t^u(g_{j+1}) in the forward and the mirrored
//    condition for groups reloaded in the backward.
//  * Selection: among partitions meeting memory and overlap, the smallest
//    total cut size (the paper's rule), then the smallest predicted step
//    time, then the lexicographically smallest list of group end nodes.  When
//    no partition meets overlap (on MI355X at C = 1 the host link cannot keep
//    up with per-block compute), strict mode returns nothing, like the
//    paper's search; otherwise the fastest memory-feasible partition is taken
//    (then fewest bytes loaded, smallest cut, end list).
//  * Predicted times: an event model of the runtime's issue order on three
//    servers (compute stream, host-to-device engine, device-to-host engine),
//    the two copy engines sharing the host link (each at `duplex` of its
//    rate alone while both run).
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <string>
#include <vector>

#include "layout.h"

namespace atom {

std::string check_config(const atom_config& c) {
  if (c.n_layer < 1 || c.d_model <= 0 || c.n_head <= 0 || c.d_mlp <= 0 || c.vocab <= 0 || c.seq_len <= 0 ||
      c.batch <= 0 || c.accum <= 0)
    return "all config sizes must be positive";
  if (c.n_layer + 2 > ATOM_MAX_NODES) return "too many layers";
  if (c.dtype != ATOM_F32 && c.dtype != ATOM_BF16) return "dtype must be ATOM_F32 or ATOM_BF16";
  if (c.ckpt != ATOM_CKPT_DEVICE && c.ckpt != ATOM_CKPT_HOST) return "unknown checkpoint policy";
  if (c.d_model % c.n_head) return "d_model must be divisible by n_head";
  const int dh = c.d_model / c.n_head;
  if (dh != 64 && dh != 128) return "head dimension d_model/n_head must be 64 or 128";
  if (c.d_model % 64 || c.d_model > 8192) return "d_model must be a multiple of 64 and at most 8192";
  if (c.d_mlp % 8) return "d_mlp must be a multiple of 8";
  if (static_cast<int64_t>(c.batch) * c.seq_len > (1LL << 30)) return "batch * seq_len too large";
  return "";
}

uint64_t node_tensors(const atom_config& c, int node, std::vector<TensorDesc>* out) {
  const int64_t d = c.d_model, f = c.d_mlp, V = c.vocab, T = c.seq_len, e = elem_bytes(c);
  std::vector<std::pair<std::string, std::pair<int64_t, int64_t>>> t;
  if (node == 0) {
    t = {{"wte", {V, d}}, {"wpe", {T, d}}};
  } else if (node >= 1 && node <= c.n_layer) {
    t = {{"ln1_g", {d, 1}}, {"ln1_b", {d, 1}}, {"w_qkv", {3 * d, d}}, {"b_qkv", {3 * d, 1}},
         {"w_o", {d, d}},   {"b_o", {d, 1}},   {"ln2_g", {d, 1}},     {"ln2_b", {d, 1}},
         {"w_fc", {f, d}},  {"b_fc", {f, 1}},  {"w_pr", {d, f}},      {"b_pr", {d, 1}}};
  } else if (node == c.n_layer + 1) {
    t = {{"lnf_g", {d, 1}}, {"lnf_b", {d, 1}}, {"w_head", {vocab_padded(V), d}}};
  } else {
    return 0;
  }
  uint64_t off = 0;
  if (out) out->clear();
  for (auto& x : t) {
    const uint64_t bytes = static_cast<uint64_t>(x.second.first * x.second.second * e);
    if (out) out->push_back({x.first, x.second.first, x.second.second, off, bytes});
    off = align_up(off + bytes);
  }
  return off;
}

ArenaLayout arena_layout(const atom_config& c, uint64_t slot_bytes, int n_slots, int n_gslots) {
  ArenaLayout a{};
  const uint64_t N = static_cast<uint64_t>(c.batch) * c.seq_len, d = c.d_model, f = c.d_mlp, C = c.accum;
  const uint64_t L = c.n_layer, H = c.n_head, e = elem_bytes(c);
  const uint64_t Vp = vocab_padded(c.vocab);
  const uint64_t BHT = static_cast<uint64_t>(c.batch) * H * c.seq_len;
  uint64_t off = 0;
  auto take = [&](uint64_t bytes) {
    const uint64_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  // token arrays, twice: consecutive steps of a pipelined call alternate
  const uint64_t tok0 = off;
  a.tok_in = take(C * N * 4);
  a.tok_tgt = take(C * N * 4);
  a.emb_perm = take(C * N * 4);
  a.emb_seg = take(C * (N + 1) * 4);
  a.emb_uniq = take(C * N * 4);
  a.tok_stride = off - tok0;
  take(a.tok_stride);
  a.ckpt_bytes_each = N * d * 4;
  a.ckpt = take((c.ckpt == ATOM_CKPT_DEVICE ? L + 1 : CKPT_RING) * C * a.ckpt_bytes_each);
  a.dres = take(C * N * d * 4);
  a.dres_lp = c.dtype == ATOM_BF16 ? take(C * N * d * 2) : a.dres;
  a.loss_rows = take(C * N * 4);
  a.loss_out = take(MAX_STEPS_PER_CALL * 4);
  a.hwm = take(static_cast<uint64_t>(ATOM_MAX_NODES) * 2 * 8);
  a.splitk_bytes = SPLITK_BYTES;
  a.splitk = take(a.splitk_bytes);
  // partial-sum scratch: column sums over ceil(N/16) row blocks, or LayerNorm
  // partials (at most one per 8-row block, two rows of d each)
  a.part_floats = std::max((N + 15) / 16 * std::max(3 * d, f), (N + 7) / 8 * 2 * d);
  // block workspace
  uint64_t w = 0;
  auto wtake = [&](uint64_t bytes) {
    const uint64_t o = w;
    w = align_up(w + bytes);
    return o;
  };
  a.a = wtake(N * d * e);
  a.qkv = wtake(N * 3 * d * e);
  a.o = wtake(N * d * e);
  a.x1 = wtake(N * d * 4);
  a.c = wtake(N * d * e);
  a.u = wtake(N * f * e);
  a.g = wtake(N * f * e);
  a.mu1 = wtake(N * 4);
  a.rs1 = wtake(N * 4);
  a.mu2 = wtake(N * 4);
  a.rs2 = wtake(N * 4);
  a.lse = wtake(BHT * 4);
  a.delta = wtake(BHT * 4);
  a.du = wtake(N * f * e);
  a.dbuf = wtake(N * d * e);
  a.dout = wtake(N * d * e);
  a.dqkv = wtake(N * 3 * d * e);
  a.part = wtake(a.part_floats * 4);
  a.block_ws = w;
  // head workspace
  w = 0;
  a.yhat = wtake(N * d * e);
  a.fmu = wtake(N * 4);
  a.frs = wtake(N * 4);
  a.logits = wtake(std::min<uint64_t>(N, HEAD_CHUNK) * Vp * 4);
  a.dz = wtake(N * Vp * e);
  a.dyhat = wtake(N * d * e);
  a.hpart = wtake(a.part_floats * 4);
  a.head_ws = w;
  a.ws_bytes = std::max(a.block_ws, a.head_ws);
  a.ws = take(a.ws_bytes);
  a.reserve_bytes = off;
  a.wslots = take(static_cast<uint64_t>(n_slots) * slot_bytes);
  a.gslots = take(static_cast<uint64_t>(n_gslots) * slot_bytes);
  a.accslot = (c.dtype == ATOM_BF16 && c.accum > 1) ? take(2 * slot_bytes) : 0;
  a.arena_bytes = off;
  return a;
}

namespace {

using Groups = std::vector<std::pair<int, int>>;

// ---------------------------------------------------------------- schedule
// Jobs of a call of n steps in the runtime's issue order, and an event run
// of them.  Servers: 0 = compute stream, 1 = host-to-device engine, 2 =
// device-to-host engine; each runs its jobs in issue order, a job starting
// once the server is free and every job it depends on has ended.
enum { SX = 0, SI = 1, SO = 2 };
enum { K_LOAD, K_FWD, K_CKOUT, K_RESTORE, K_BWD, K_GCOPY };

struct Job {
  int server, step, kind;
  double dur;
  int dep[4];
  int ndep;
};

struct Model {
  const atom_node_cost* c;
  int n, L, C, K, R;
  bool ck_host;
  double t_ck_out, t_ck_in;  // one node's block input (all micro-batches) each way
};

struct JobList {
  std::vector<Job> jobs;
  int add(int server, double dur, std::initializer_list<int> deps, int step, int kind) {
    Job j{server, step, kind, dur, {-1, -1, -1, -1}, 0};
    for (int d : deps)
      if (d >= 0) j.dep[j.ndep++] = d;
    jobs.push_back(j);
    return static_cast<int>(jobs.size()) - 1;
  }
};

double sum_load(const Model& m, int a, int b) {
  double t = 0.0;
  for (int i = a; i <= b; ++i) t += m.c[i].t_load;
  return t;
}

double sum_store(const Model& m, int a, int b) {
  double t = 0.0;
  for (int i = a; i <= b; ++i) t += m.c[i].t_store;
  return t;
}

// retain: every group has a slot of its own and keeps its weights from one
// step of the call to the next, so only step 0 loads (the later steps' loads
// are zero-length jobs at the same place in the issue order).
void build_jobs(const Model& m, const Groups& g, int n_steps, bool retain, JobList* out) {
  const int G = static_cast<int>(g.size()), K = m.K, R = m.R, L = m.L, head = L + 1;
  auto evicted = [&](int i) { return m.ck_host && i >= 0 && i + CKPT_RING <= L; };
  JobList& J = *out;
  J.jobs.clear();
  // load[s][j], reload[j] (current step), per node fwd / ckout / restore
  std::vector<std::vector<int>> load(n_steps + 1, std::vector<int>(G, -1));
  std::vector<int> reload(G, -1), fwd(m.n, -1), ckout(m.n, -1), restore(m.n, -1), last_c(G, -1), claim_of(G, -1);
  std::vector<int> claims;  // gradient copy releasing each claim's slot (-1 until issued)
  auto claim = [&]() {
    const int k = static_cast<int>(claims.size());
    claims.push_back(-1);
    return k >= R ? claims[k - R] : -1;
  };
  for (int j = 0; j < std::min(G, K); ++j) load[0][j] = J.add(SI, sum_load(m, g[j].first, g[j].second), {}, 0, K_LOAD);
  for (int s = 0; s < n_steps; ++s) {
    std::fill(fwd.begin(), fwd.end(), -1);
    std::fill(ckout.begin(), ckout.end(), -1);
    std::fill(restore.begin(), restore.end(), -1);
    std::fill(claim_of.begin(), claim_of.end(), -1);
    std::fill(reload.begin(), reload.end(), -1);
    for (int j = 0; j < G; ++j) {
      for (int node = g[j].first; node <= g[j].second; ++node) {
        const int d_load = node == g[j].first ? load[s][j] : -1;
        int d_claim = -1;
        if (node == head) {
          claim_of[j] = static_cast<int>(claims.size());
          d_claim = claim();
        }
        const int d_ck = evicted(node - CKPT_RING) ? ckout[node - CKPT_RING] : -1;
        fwd[node] = J.add(SX, m.C * m.c[node].t_fwd, {d_load, d_claim, d_ck}, s, K_FWD);
        if (evicted(node)) ckout[node] = J.add(SO, m.t_ck_out, {fwd[node]}, s, K_CKOUT);
        if (m.ck_host && node == head && L - CKPT_RING >= 0)
          restore[L - CKPT_RING] = J.add(SI, m.t_ck_in, {fwd[node], ckout[L - CKPT_RING]}, s, K_RESTORE);
      }
      last_c[j] = fwd[g[j].second];
      if (j + K < G)
        load[s][j + K] = J.add(SI, sum_load(m, g[j + K].first, g[j + K].second), {fwd[g[j].second]}, s, K_LOAD);
    }
    for (int j = G - 1; j >= 0; --j) {
      bool first = true;
      for (int node = std::min(g[j].second, L); node >= g[j].first; --node) {
        int d_w = -1, d_claim = -1, d_ck = -1;
        if (first) {
          if (j < G - K) d_w = reload[j];
          if (claim_of[j] < 0) {
            claim_of[j] = static_cast<int>(claims.size());
            d_claim = claim();
          }
          first = false;
        }
        if (node >= 1 && evicted(node - 1)) d_ck = restore[node - 1];
        last_c[j] = J.add(SX, m.C * m.c[node].t_bwd, {d_w, d_claim, d_ck}, s, K_BWD);
        if (m.ck_host && node - 1 - CKPT_RING >= 0) {
          const int i = node - 1 - CKPT_RING;
          restore[i] = J.add(SI, m.t_ck_in, {last_c[j], ckout[i]}, s, K_RESTORE);
        }
      }
      const int gc = J.add(SO, sum_store(m, g[j].first, g[j].second), {last_c[j]}, s, K_GCOPY);
      claims[claim_of[j]] = gc;
      if (j - K >= 0)
        reload[j - K] = J.add(SI, sum_load(m, g[j - K].first, g[j - K].second), {last_c[j]}, s, K_LOAD);
      else if (s + 1 < n_steps)
        load[s + 1][K - 1 - j] =
            J.add(SI, retain ? 0.0 : sum_load(m, g[K - 1 - j].first, g[K - 1 - j].second), {last_c[j]}, s, K_LOAD);
    }
  }
}

// End time of every job; false on a deadlock (cannot happen: every job
// depends only on jobs issued before it).
bool run_jobs(const JobList& J, double duplex, std::vector<double>* end_out) {
  const int nj = static_cast<int>(J.jobs.size());
  std::vector<double>& end = *end_out;
  end.assign(nj, 0.0);
  std::vector<char> done(nj, 0);
  std::vector<int> queue[3];
  for (int i = 0; i < nj; ++i) queue[J.jobs[i].server].push_back(i);
  size_t nxt[3] = {0, 0, 0};
  int run[3] = {-1, -1, -1};
  double rem[3] = {0.0, 0.0, 0.0};
  double t = 0.0;
  for (;;) {
    bool progress = true;
    while (progress) {
      progress = false;
      for (int sv = 0; sv < 3; ++sv) {
        if (run[sv] >= 0 || nxt[sv] >= queue[sv].size()) continue;
        const int k = queue[sv][nxt[sv]];
        const Job& jb = J.jobs[k];
        bool ready = true;
        for (int d = 0; d < jb.ndep; ++d)
          if (!done[jb.dep[d]]) ready = false;
        if (!ready) continue;
        ++nxt[sv];
        progress = true;
        if (jb.dur <= 0.0) {
          end[k] = t;
          done[k] = 1;
        } else {
          run[sv] = k;
          rem[sv] = jb.dur;
        }
      }
    }
    if (run[0] < 0 && run[1] < 0 && run[2] < 0) break;
    const bool both = run[SI] >= 0 && run[SO] >= 0;
    double rate[3], tau[3];
    double dt = 0.0;
    bool have = false;
    for (int sv = 0; sv < 3; ++sv) {
      rate[sv] = (both && sv != SX) ? duplex : 1.0;
      if (run[sv] < 0) continue;
      tau[sv] = rem[sv] / rate[sv];
      if (!have || tau[sv] < dt) dt = tau[sv];
      have = true;
    }
    const double t_new = t + dt;
    for (int sv = 0; sv < 3; ++sv) {
      if (run[sv] < 0) continue;
      if (tau[sv] == dt) {
        end[run[sv]] = t_new;
        done[run[sv]] = 1;
        run[sv] = -1;
        rem[sv] = 0.0;
      } else {
        rem[sv] = rem[sv] - rate[sv] * dt;
      }
    }
    t = t_new;
  }
  for (int i = 0; i < nj; ++i)
    if (!done[i]) return false;
  return true;
}

// Step end times (last compute job or last gradient copy of each step) and
// the forward end of step 0.
bool simulate(const Model& m, const Groups& g, int n_steps, bool retain, double duplex, std::vector<double>* ends,
              double* t_fwd) {
  JobList J;
  build_jobs(m, g, n_steps, retain, &J);
  std::vector<double> end;
  if (!run_jobs(J, duplex, &end)) return false;
  ends->assign(n_steps, 0.0);
  double tf = 0.0;
  for (size_t i = 0; i < J.jobs.size(); ++i) {
    const Job& jb = J.jobs[i];
    if (jb.server == SX || jb.kind == K_GCOPY) (*ends)[jb.step] = std::max((*ends)[jb.step], end[i]);
    if (jb.step == 0 && jb.kind == K_FWD) tf = std::max(tf, end[i]);
  }
  if (t_fwd) *t_fwd = tf;
  return true;
}

constexpr int PIPE_STEPS = 4;

// ---------------------------------------------------------------- search
struct Eval {
  bool ok = false, overlap = false;
  int K = 0, R = 0;
  uint64_t S = 0, arena = 0, h2d = 0, d2h = 0, cut = 0;
  double t_fwd = 0, t_first = 0, t_step = 0;
};

struct Search {
  const atom_node_cost* c;
  int n, L, C, dtype;
  uint64_t budget, base, work;
  bool ck_host;
  double t_ck_out, t_ck_in, duplex;
};

// Memory, overlap, bytes and cut of a partition (no simulation).  The
// weight and gradient slot counts follow from the budget, or are given
// (k_fixed, r_fixed >= 1: a plan built for a given partition).
Eval check(const Search& p, const Groups& g, int k_fixed = 0, int r_fixed = 0) {
  Eval ev;
  const int G = static_cast<int>(g.size());
  std::vector<uint64_t> W(G, 0);
  std::vector<double> F(G, 0.0), B(G, 0.0), U(G, 0.0);
  uint64_t S = 0;
  for (int j = 0; j < G; ++j) {
    double tf = 0.0, tb = 0.0, tu = 0.0;
    for (int i = g[j].first; i <= g[j].second; ++i) {
      W[j] += p.c[i].weight_bytes;
      tf += p.c[i].t_fwd;
      tb += p.c[i].t_bwd;
      tu += p.c[i].t_load;
    }
    F[j] = p.C * tf;
    B[j] = p.C * tb;
    U[j] = tu;
    S = std::max(S, W[j]);
  }
  const uint64_t acc = (p.C > 1 && p.dtype == ATOM_BF16) ? 2 * S : 0;
  const uint64_t fixed = p.base + p.work + 2 * S + acc;
  if (S == 0 || p.budget < fixed) return ev;
  const uint64_t kmax = (p.budget - fixed) / S;
  const int K = k_fixed > 0 ? k_fixed : static_cast<int>(std::min<uint64_t>(static_cast<uint64_t>(G), kmax));
  if (K < std::min(G, 2) || K > G || static_cast<uint64_t>(K) > kmax) return ev;
  const uint64_t left = p.budget - fixed - static_cast<uint64_t>(K) * S;
  ev.ok = true;
  ev.K = K;
  ev.R = r_fixed > 0 ? r_fixed : static_cast<int>(std::min<uint64_t>(ATOM_MAX_GSLOTS, 2 + left / S));
  if (static_cast<uint64_t>(ev.R - 2) > left / S) ev.ok = false;
  ev.S = S;
  ev.arena = fixed + static_cast<uint64_t>(K) * S + static_cast<uint64_t>(ev.R - 2) * S;
  bool ov = true;
  for (int j = 0; j + 1 < G; ++j)
    if (F[j] < U[j + 1]) ov = false;
  for (int j = 0; j + 1 < G; ++j)
    if (j < G - K && B[j + 1] < U[j]) ov = false;
  ev.overlap = ov;
  uint64_t tot = 0, rel = 0;
  for (int j = 0; j < G; ++j) {
    tot += W[j];
    if (j < G - K) rel += W[j];
  }
  ev.h2d = tot + rel;
  ev.d2h = tot;
  for (int j = 0; j + 1 < G; ++j) ev.cut += p.c[g[j].second].cut_bytes;
  return ev;
}

bool predict(const Search& p, const Groups& g, Eval* ev) {
  const Model m{p.c, p.n, p.L, p.C, ev->K, ev->R, p.ck_host, p.t_ck_out, p.t_ck_in};
  std::vector<double> ends;
  if (!simulate(m, g, 1, false, p.duplex, &ends, &ev->t_fwd)) return false;
  ev->t_first = ends[0];
  if (!simulate(m, g, PIPE_STEPS, false, p.duplex, &ends, nullptr)) return false;
  ev->t_step = (ends[PIPE_STEPS - 1] - ends[PIPE_STEPS - 3]) / 2.0;
  return true;
}

bool lex_less(const Groups& a, const Groups& b) {
  for (size_t i = 0; i < std::min(a.size(), b.size()); ++i)
    if (a[i].second != b[i].second) return a[i].second < b[i].second;
  return a.size() < b.size();
}

bool paper_better(const Eval& a, const Groups& ga, const Eval& b, const Groups& gb) {
  if (a.cut != b.cut) return a.cut < b.cut;
  if (a.t_step != b.t_step) return a.t_step < b.t_step;
  return lex_less(ga, gb);
}

bool time_better(const Eval& a, const Groups& ga, const Eval& b, const Groups& gb) {
  if (a.t_step != b.t_step) return a.t_step < b.t_step;
  if (a.h2d != b.h2d) return a.h2d < b.h2d;
  if (a.cut != b.cut) return a.cut < b.cut;
  return lex_less(ga, gb);
}

// Candidate partitions: every composition for short chains, the structured
// family otherwise.
std::vector<Groups> candidates(int n, bool* exhaustive) {
  std::vector<Groups> out;
  Groups g;
  *exhaustive = n <= 16;
  if (*exhaustive) {
    const uint64_t total = 1ULL << (n - 1);
    for (uint64_t mask = 0; mask < total; ++mask) {
      g.clear();
      int start = 0;
      for (int i = 0; i < n - 1; ++i)
        if (mask >> i & 1ULL) {
          g.push_back({start, i});
          start = i + 1;
        }
      g.push_back({start, n - 1});
      out.push_back(g);
    }
    return out;
  }
  const int L = n - 2;
  std::vector<Groups> seen;
  for (int e = 0; e <= 1; ++e)
    for (int hh = 0; hh <= 1; ++hh) {
      const int lo = 1 + e, hi = L - hh, m = hi - lo + 1;
      if (m < 0) continue;
      for (int s = 1; s <= std::max(m, 1); ++s) {
        g.clear();
        g.push_back({0, e});
        if (m > 0) {
          const int r = m % s;
          int start = lo;
          if (r) {
            g.push_back({start, start + r - 1});
            start += r;
          }
          while (start <= hi) {
            g.push_back({start, start + s - 1});
            start += s;
          }
        }
        g.push_back({L + 1 - hh, L + 1});
        if (std::find(out.begin(), out.end(), g) == out.end()) out.push_back(g);
      }
    }
  return out;
}

// Seconds per byte of the host link each way, from the nodes' copy times.
void link_rates(const atom_node_cost* c, int n, double* in_s_per_b, double* out_s_per_b) {
  double tl = 0.0, ts = 0.0;
  uint64_t w = 0;
  for (int i = 0; i < n; ++i) {
    tl += c[i].t_load;
    ts += c[i].t_store;
    w += c[i].weight_bytes;
  }
  *in_s_per_b = w ? tl / static_cast<double>(w) : 0.0;
  *out_s_per_b = w ? ts / static_cast<double>(w) : 0.0;
}

Search make_search(const atom_config& cfg, uint64_t budget, uint64_t base, const atom_node_cost* c, int n,
                   double duplex) {
  Search p{};
  p.c = c;
  p.n = n;
  p.L = n - 2;
  p.C = cfg.accum;
  p.dtype = cfg.dtype;
  p.budget = budget;
  p.base = base;
  p.work = 0;
  for (int i = 0; i < n; ++i) p.work = std::max(p.work, c[i].mem_bytes);
  p.ck_host = cfg.ckpt == ATOM_CKPT_HOST;
  const double ckb = static_cast<double>(ckpt_xfer_bytes(cfg) / std::max(1, ckpt_evicted(cfg)));
  double rin = 0.0, rout = 0.0;
  link_rates(c, n, &rin, &rout);
  p.t_ck_in = p.ck_host ? ckb * rin : 0.0;
  p.t_ck_out = p.ck_host ? ckb * rout : 0.0;
  p.duplex = duplex > 0.0 ? duplex : ATOM_DEFAULT_DUPLEX;
  return p;
}

void fill_plan(const atom_config& cfg, const Search& p, const Groups& g, const Eval& ev, atom_plan* out) {
  memset(out, 0, sizeof(*out));
  out->n_nodes = p.n;
  out->n_groups = static_cast<int32_t>(g.size());
  out->n_slots = ev.K;
  out->n_gslots = ev.R;
  out->overlap_ok = ev.overlap ? 1 : 0;
  out->accum = cfg.accum;
  for (size_t i = 0; i < g.size(); ++i) {
    out->first[i] = g[i].first;
    out->last[i] = g[i].second;
  }
  out->budget_bytes = p.budget;
  out->reserve_bytes = p.base + p.work;
  out->work_bytes = p.work;
  out->slot_bytes = ev.S;
  out->arena_bytes = ev.arena;
  out->h2d_bytes = ev.h2d + ckpt_xfer_bytes(cfg);
  out->d2h_bytes = ev.d2h + ckpt_xfer_bytes(cfg);
  out->cut_bytes = ev.cut;
  out->pred_fwd_s = ev.t_fwd;
  out->pred_first_step_s = ev.t_first;
  out->pred_step_s = ev.t_step;
  out->duplex = p.duplex;
}

}  // namespace
}  // namespace atom

using namespace atom;

extern "C" {

const char* atom_version(void) { return "atom-mi355x 0.2 (gfx950)"; }

const char* atom_status_string(int s) {
  switch (s) {
    case ATOM_OK: return "ok";
    case ATOM_EINVAL: return "invalid argument";
    case ATOM_ENOPLAN: return "no partition fits the device budget";
    case ATOM_EBUDGET: return "arena smaller than the plan requires";
    case ATOM_EHIP: return "HIP runtime error";
    case ATOM_ESTATE: return "call-order violation";
    case ATOM_ENOMEM_HOST: return "pinned host allocation failed";
    default: return "unknown status";
  }
}

int atom_node_layout(const atom_config* cfg, int32_t node, atom_tensor_desc* out, int32_t max, int32_t* n_out,
                     uint64_t* node_bytes) {
  if (!cfg || !check_config(*cfg).empty() || node < 0 || node > cfg->n_layer + 1) return ATOM_EINVAL;
  std::vector<TensorDesc> t;
  const uint64_t nb = node_tensors(*cfg, node, &t);
  if (n_out) *n_out = static_cast<int32_t>(t.size());
  if (node_bytes) *node_bytes = nb;
  if (out) {
    for (int i = 0; i < static_cast<int>(t.size()) && i < max; ++i) {
      memset(&out[i], 0, sizeof(out[i]));
      strncpy(out[i].name, t[i].name.c_str(), sizeof(out[i].name) - 1);
      out[i].rows = static_cast<int32_t>(t[i].rows);
      out[i].cols = static_cast<int32_t>(t[i].cols);
      out[i].offset = t[i].offset;
      out[i].bytes = t[i].bytes;
    }
  }
  return ATOM_OK;
}

int atom_node_costs(const atom_config* cfg, atom_node_cost* out, int32_t n) {
  if (!cfg || !out || !check_config(*cfg).empty() || n != cfg->n_layer + 2) return ATOM_EINVAL;
  const double N = static_cast<double>(cfg->batch) * cfg->seq_len, d = cfg->d_model, f = cfg->d_mlp;
  const double T = cfg->seq_len, Vp = static_cast<double>(vocab_padded(cfg->vocab));
  // Assumed rates for the analytic model: half of the dense MFMA peak
  // (bf16 2.5 PFLOP/s, fp32 157.3 TFLOP/s), 50 GB/s host link each way and
  // 4 TB/s effective HBM for the embedding.
  const double rate = (cfg->dtype == ATOM_BF16 ? 2.5e15 : 157.3e12) * 0.5;
  const double link = 50e9, hbm = 4e12;
  const ArenaLayout lay = arena_layout(*cfg, 0, 0, 0);
  const uint64_t cut = static_cast<uint64_t>(cfg->batch) * cfg->seq_len * cfg->d_model * 4;
  for (int i = 0; i < n; ++i) {
    const uint64_t wb = node_tensors(*cfg, i, nullptr);
    out[i].weight_bytes = wb;
    out[i].t_load = static_cast<double>(wb) / link;
    out[i].t_store = static_cast<double>(wb) / link;
    if (i == 0) {
      out[i].mem_bytes = 0;
      out[i].cut_bytes = cut;
      out[i].t_fwd = N * d * 12.0 / hbm;
      out[i].t_bwd = N * d * 12.0 / hbm;
    } else if (i <= cfg->n_layer) {
      out[i].mem_bytes = lay.block_ws;
      out[i].cut_bytes = cut;
      const double fwd = 2.0 * N * (4.0 * d * d + 2.0 * d * f) + 2.0 * N * T * d;  // causal half of 4NTd
      out[i].t_fwd = fwd / rate;
      out[i].t_bwd = 3.0 * fwd / rate;  // recompute + data and weight gradients
    } else {
      out[i].mem_bytes = lay.head_ws;
      out[i].cut_bytes = 4;  // the loss; never a cut (the head is the last node)
      out[i].t_fwd = 6.0 * N * d * Vp / rate;  // logits, data and weight gradients of the head
      out[i].t_bwd = 0.0;
    }
  }
  return ATOM_OK;
}

int atom_reserve_bytes(const atom_config* cfg, uint64_t* out) {
  if (!cfg || !out || !check_config(*cfg).empty()) return ATOM_EINVAL;
  *out = arena_layout(*cfg, 0, 0, 0).reserve_bytes;
  return ATOM_OK;
}

int atom_plan_search(const atom_config* cfg, uint64_t budget, uint64_t base, const atom_node_cost* costs, int32_t n,
                     const atom_plan_opts* opts, atom_plan* out) {
  if (!cfg || !costs || !out || n < 3 || n > ATOM_MAX_NODES || n != cfg->n_layer + 2 || cfg->accum < 1)
    return ATOM_EINVAL;
  if (opts && (opts->duplex < 0.0 || opts->duplex > 1.0)) return ATOM_EINVAL;
  const Search p = make_search(*cfg, budget, base, costs, n, opts ? opts->duplex : 0.0);
  bool exhaustive = false;
  const std::vector<Groups> cand = candidates(n, &exhaustive);
  // pass 1: memory, overlap and cut of every candidate
  std::vector<Eval> ev(cand.size());
  bool any_ok = false, any_ov = false;
  uint64_t min_cut = UINT64_MAX;
  for (size_t i = 0; i < cand.size(); ++i) {
    ev[i] = check(p, cand[i]);
    if (!ev[i].ok) continue;
    any_ok = true;
    if (ev[i].overlap) {
      any_ov = true;
      min_cut = std::min(min_cut, ev[i].cut);
    }
  }
  if (!any_ok || (!any_ov && opts && opts->strict)) return ATOM_ENOPLAN;
  // pass 2: predicted times where they decide (the minimum-cut partitions
  // meeting overlap, or every memory-feasible one for the fallback)
  int best = -1;
  for (size_t i = 0; i < cand.size(); ++i) {
    if (!ev[i].ok) continue;
    if (any_ov && (!ev[i].overlap || ev[i].cut != min_cut)) continue;
    if (!predict(p, cand[i], &ev[i])) return ATOM_EINVAL;
    if (best < 0 || (any_ov ? paper_better(ev[i], cand[i], ev[best], cand[best])
                            : time_better(ev[i], cand[i], ev[best], cand[best])))
      best = static_cast<int>(i);
  }
  fill_plan(*cfg, p, cand[best], ev[best], out);
  out->rule = any_ov ? ATOM_RULE_PAPER : ATOM_RULE_TIME;
  out->exhaustive = exhaustive ? 1 : 0;
  out->n_evaluated = static_cast<int64_t>(cand.size());
  uint64_t W = 0, Smin = 0;
  for (int i = 0; i < n; ++i) {
    W += costs[i].weight_bytes;
    Smin = std::max<uint64_t>(Smin, costs[i].weight_bytes);
  }
  // Lower bound on host-to-device bytes for any schedule in this memory
  // model: every weight once, plus what cannot stay resident into the
  // backward (the budget minus the reserve, two gradient slots and the
  // weights of the group being executed).
  const uint64_t reserve = p.base + p.work;
  const uint64_t keep = budget > reserve + 3 * Smin ? budget - reserve - 3 * Smin : 0;
  out->forced_h2d_bytes = W + (W > keep ? W - keep : 0) + ckpt_xfer_bytes(*cfg);
  return ATOM_OK;
}

int atom_plan_partition(const atom_config* cfg, uint64_t budget, const atom_node_cost* costs, int32_t n_costs,
                        const atom_plan_opts* opts, atom_plan* out) {
  if (!cfg || !out || !check_config(*cfg).empty()) return ATOM_EINVAL;
  const int n = cfg->n_layer + 2;
  std::vector<atom_node_cost> analytic(n), c(n);
  atom_node_costs(cfg, analytic.data(), n);
  if (costs) {
    if (n_costs != n) return ATOM_EINVAL;
    for (int i = 0; i < n; ++i) {
      c[i] = costs[i];
      // the arena carves each node's workspace at its analytic size
      c[i].mem_bytes = std::max(costs[i].mem_bytes, analytic[i].mem_bytes);
    }
  } else {
    c = analytic;
  }
  const ArenaLayout a0 = arena_layout(*cfg, 0, 0, 0);
  const uint64_t base = a0.reserve_bytes - a0.ws_bytes;
  int s = atom_plan_search(cfg, budget, base, c.data(), n, opts, out);
  if (s != ATOM_OK) return s;
  // Slot sizes are multiples of the 256-byte alignment and the reserve
  // already includes its padding, so the carved arena is exactly the size the
  // search assumed.
  const ArenaLayout a = arena_layout(*cfg, out->slot_bytes, out->n_slots, out->n_gslots);
  // (a node's m_i above the carved workspace cannot come from a measurement
  // of the kernels, which write only inside their regions)
  if (a.reserve_bytes != out->reserve_bytes) return ATOM_EINVAL;
  if (a.arena_bytes != out->arena_bytes || a.arena_bytes > budget) return ATOM_ENOPLAN;
  return ATOM_OK;
}

int atom_plan_fixed(const atom_config* cfg, int32_t n_groups, const int32_t* last, int32_t n_slots,
                    int32_t n_gslots, atom_plan* out) {
  if (!cfg || !last || !out || !check_config(*cfg).empty()) return ATOM_EINVAL;
  if (n_gslots < 2 || n_gslots > ATOM_MAX_GSLOTS) return ATOM_EINVAL;
  const int n = cfg->n_layer + 2;
  if (n_groups < 1 || n_groups > n || n_slots < std::min<int32_t>(n_groups, 2) || n_slots > n_groups) return ATOM_EINVAL;
  Groups g;
  int start = 0;
  for (int i = 0; i < n_groups; ++i) {
    if (last[i] < start || last[i] >= n) return ATOM_EINVAL;
    g.push_back({start, last[i]});
    start = last[i] + 1;
  }
  if (start != n) return ATOM_EINVAL;
  std::vector<atom_node_cost> c(n);
  atom_node_costs(cfg, c.data(), n);
  uint64_t S = 0;
  for (auto& x : g) {
    uint64_t w = 0;
    for (int i = x.first; i <= x.second; ++i) w += c[i].weight_bytes;
    S = std::max(S, w);
  }
  const ArenaLayout lay = arena_layout(*cfg, S, n_slots, n_gslots);
  const uint64_t base = lay.reserve_bytes - lay.ws_bytes;
  Search p = make_search(*cfg, lay.arena_bytes, base, c.data(), n, 0.0);
  Eval ev = check(p, g, n_slots, n_gslots);
  if (!ev.ok || ev.K != n_slots || ev.R != n_gslots || ev.arena != lay.arena_bytes) return ATOM_EINVAL;
  if (!predict(p, g, &ev)) return ATOM_EINVAL;
  fill_plan(*cfg, p, g, ev, out);
  out->rule = ATOM_RULE_FIXED;
  out->forced_h2d_bytes = out->h2d_bytes;
  out->n_evaluated = 1;
  return ATOM_OK;
}

int atom_plan_predict(const atom_config* cfg, const atom_plan* plan, const atom_node_cost* costs, int32_t n_costs,
                      double duplex, int32_t n_steps, int32_t retain, double* ends, double* fwd_s) {
  if (!cfg || !plan || !ends || !check_config(*cfg).empty() || n_steps < 1 || n_steps > MAX_STEPS_PER_CALL)
    return ATOM_EINVAL;
  const int n = cfg->n_layer + 2;
  if (plan->n_nodes != n || plan->n_groups < 1 || plan->n_groups > n || plan->n_slots < 1 ||
      plan->n_slots > plan->n_groups || plan->n_gslots < 2 || plan->n_gslots > ATOM_MAX_GSLOTS ||
      duplex < 0.0 || duplex > 1.0)
    return ATOM_EINVAL;
  Groups g;
  for (int i = 0; i < plan->n_groups; ++i) {
    if (plan->first[i] > plan->last[i] || (i > 0 && plan->first[i] != plan->last[i - 1] + 1)) return ATOM_EINVAL;
    g.push_back({plan->first[i], plan->last[i]});
  }
  if (g.front().first != 0 || g.back().second != n - 1) return ATOM_EINVAL;
  std::vector<atom_node_cost> c(n);
  if (costs) {
    if (n_costs != n) return ATOM_EINVAL;
    for (int i = 0; i < n; ++i) c[i] = costs[i];
  } else {
    atom_node_costs(cfg, c.data(), n);
  }
  const Search p = make_search(*cfg, 0, 0, c.data(), n, duplex);
  const Model m{c.data(), n, n - 2, cfg->accum, plan->n_slots, plan->n_gslots, p.ck_host, p.t_ck_out, p.t_ck_in};
  std::vector<double> e;
  // as atom_set_retention: no effect unless every group has a slot of its own
  const bool ret = retain != 0 && plan->n_slots == plan->n_groups;
  if (!simulate(m, g, n_steps, ret, p.duplex, &e, fwd_s)) return ATOM_EINVAL;
  for (int s = 0; s < n_steps; ++s) ends[s] = e[s];
  return ATOM_OK;
}

}  // extern "C"
