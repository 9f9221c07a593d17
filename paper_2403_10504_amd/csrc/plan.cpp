// Static analysis of the swapped step: node layout, node costs, arena
// layout and the partition search (Section III-D, Algorithm 1).
//
// Readings of the algorithm (the paper's listing is garbled in places):
//  * Search space: with step size 1 the search visits every way to cut the
//    topologically sorted chain into contiguous sub-models; that set is
//    enumerated directly (all 2^(n-1) compositions) for n <= 20 nodes.  For
//    longer chains the search uses the structure of GPT-3 (identical decoder
//    blocks, noted in Section III-D as the knowledge that shrinks the search):
//    the embedding alone or with the first block, the head alone or with the
//    last block, and the remaining blocks in runs of s.
//  * Memory (hard): the executing group and the one being preloaded must be
//    co-resident.  Groups live in equal weight slots of the largest group's
//    size S next to two gradient slots (plus a 2S fp32 accumulation slot for
//    bf16 with C > 1) and the reserved activation memory.
//  * Overlap (soft): C * t^f(g_j) >= t^u(g_{j+1}) in the forward and the
//    mirrored condition for groups reloaded in the backward; reported as
//    overlap_ok, not required, because on MI355X the host link cannot keep
//    up with per-block compute at C = 1.
//  * Objective: smallest predicted step time of the three-stream schedule,
//    then fewest bytes loaded (the model runs loads and stores at full rate
//    each, so reloads that overlap the gradient stores look free although
//    both directions share the host link), then fewest groups (the paper's
//    minimum total cut size: every cut is one [B, T, d] activation), then the
//    lexicographically smallest list of group end nodes.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>
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
  const uint64_t block_ws = w;
  // head workspace
  w = 0;
  a.yhat = wtake(N * d * e);
  a.fmu = wtake(N * 4);
  a.frs = wtake(N * 4);
  a.logits = wtake(std::min<uint64_t>(N, HEAD_CHUNK) * Vp * 4);
  a.dz = wtake(N * Vp * e);
  a.dyhat = wtake(N * d * e);
  a.hpart = wtake(a.part_floats * 4);
  const uint64_t head_ws = w;
  a.ws_bytes = std::max(block_ws, head_ws);
  a.ws = take(a.ws_bytes);
  a.reserve_bytes = off;
  a.wslots = take(static_cast<uint64_t>(n_slots) * slot_bytes);
  a.gslots = take(static_cast<uint64_t>(n_gslots) * slot_bytes);
  a.accslot = (c.dtype == ATOM_BF16 && c.accum > 1) ? take(2 * slot_bytes) : 0;
  a.arena_bytes = off;
  return a;
}

namespace {

struct Sums {
  std::vector<double> F, B, U, S;
  std::vector<uint64_t> W;
};

Sums group_sums(const std::vector<std::pair<int, int>>& g, const atom_node_cost* c, int accum) {
  Sums s;
  for (auto& x : g) {
    double tf = 0.0, tb = 0.0, tu = 0.0, ts = 0.0;
    uint64_t w = 0;
    for (int i = x.first; i <= x.second; ++i) {
      tf += c[i].t_fwd;
      tb += c[i].t_bwd;
      tu += c[i].t_load;
      ts += c[i].t_store;
      w += c[i].weight_bytes;
    }
    s.F.push_back(static_cast<double>(accum) * tf);
    s.B.push_back(static_cast<double>(accum) * tb);
    s.U.push_back(tu);
    s.S.push_back(ts);
    s.W.push_back(w);
  }
  return s;
}

struct Eval {
  bool ok = false;
  int K = 0;
  uint64_t S = 0, arena = 0, h2d = 0, d2h = 0;
  double t_fwd = 0, t_step = 0;
  bool overlap = false;
};

Eval evaluate(const std::vector<std::pair<int, int>>& g, const atom_node_cost* c, uint64_t budget,
              uint64_t reserve, int accum, int dtype) {
  Eval ev;
  const Sums s = group_sums(g, c, accum);
  const int G = static_cast<int>(g.size());
  uint64_t S = 0;
  for (uint64_t w : s.W) S = std::max(S, w);
  const uint64_t grad = 2 * S + ((accum > 1 && dtype == ATOM_BF16) ? 2 * S : 0);
  if (S == 0 || budget < reserve + grad) return ev;
  const uint64_t kmax = (budget - reserve - grad) / S;
  const int K = static_cast<int>(std::min<uint64_t>(static_cast<uint64_t>(G), kmax));
  if (K < std::min(G, 2)) return ev;
  ev.ok = true;
  ev.K = K;
  ev.S = S;
  ev.arena = reserve + static_cast<uint64_t>(K) * S + grad;

  // three-stream schedule
  double h = 0.0, cc = 0.0, dd = 0.0;
  std::vector<double> fend(G, 0.0), bend(G, 0.0), dend(G, 0.0);
  for (int j = 0; j < G; ++j) {
    const double fr = j >= K ? fend[j - K] : 0.0;
    const double le = std::max(h, fr) + s.U[j];
    h = le;
    fend[j] = std::max(cc, le) + s.F[j];
    cc = fend[j];
  }
  ev.t_fwd = cc;
  for (int j = G - 1; j >= 0; --j) {
    double ready = 0.0;
    if (j < G - K) {
      const double le = std::max(h, bend[j + K]) + s.U[j];
      h = le;
      ready = le;
    }
    const double gfree = (j + 2 <= G - 1) ? dend[j + 2] : 0.0;
    bend[j] = std::max(std::max(cc, ready), gfree) + s.B[j];
    cc = bend[j];
    dend[j] = std::max(dd, bend[j]) + s.S[j];
    dd = dend[j];
  }
  ev.t_step = std::max(cc, dd);

  bool ov = true;
  for (int j = 0; j + 1 < G; ++j)
    if (s.F[j] < s.U[j + 1]) ov = false;
  for (int j = 0; j + 1 < G; ++j)
    if (j < G - K && s.B[j + 1] < s.U[j]) ov = false;
  ev.overlap = ov;

  uint64_t tot = 0, rel = 0;
  for (int j = 0; j < G; ++j) {
    tot += s.W[j];
    if (j < G - K) rel += s.W[j];
  }
  ev.h2d = tot + rel;
  ev.d2h = tot;
  return ev;
}

bool better(const Eval& a, const std::vector<std::pair<int, int>>& ga, const Eval& b,
            const std::vector<std::pair<int, int>>& gb) {
  if (a.t_step != b.t_step) return a.t_step < b.t_step;
  if (a.h2d != b.h2d) return a.h2d < b.h2d;
  if (ga.size() != gb.size()) return ga.size() < gb.size();
  for (size_t i = 0; i < ga.size(); ++i)
    if (ga[i].second != gb[i].second) return ga[i].second < gb[i].second;
  return false;
}

}  // namespace
}  // namespace atom

using namespace atom;

extern "C" {

const char* atom_version(void) { return "atom-mi355x 0.1 (gfx950)"; }

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
  for (int i = 0; i < n; ++i) {
    const uint64_t wb = node_tensors(*cfg, i, nullptr);
    out[i].weight_bytes = wb;
    out[i].t_load = static_cast<double>(wb) / link;
    out[i].t_store = static_cast<double>(wb) / link;
    if (i == 0) {
      out[i].t_fwd = N * d * 12.0 / hbm;
      out[i].t_bwd = N * d * 12.0 / hbm;
    } else if (i <= cfg->n_layer) {
      const double fwd = 2.0 * N * (4.0 * d * d + 2.0 * d * f) + 2.0 * N * T * d;  // causal half of 4NTd
      out[i].t_fwd = fwd / rate;
      out[i].t_bwd = 3.0 * fwd / rate;  // recompute + data and weight gradients
    } else {
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

int atom_plan_search(const atom_config* cfg, uint64_t budget, uint64_t reserve, const atom_node_cost* costs,
                     int32_t n, atom_plan* out) {
  if (!cfg || !costs || !out || n < 1 || n > ATOM_MAX_NODES || cfg->accum < 1) return ATOM_EINVAL;
  const int accum = cfg->accum, dtype = cfg->dtype;
  std::vector<std::pair<int, int>> best_g, g;
  Eval best;
  int64_t evaluated = 0;
  auto consider = [&](const std::vector<std::pair<int, int>>& cand) {
    ++evaluated;
    Eval ev = evaluate(cand, costs, budget, reserve, accum, dtype);
    if (!ev.ok) return;
    if (!best.ok || better(ev, cand, best, best_g)) {
      best = ev;
      best_g = cand;
    }
  };
  const bool exhaustive = n <= 20;
  if (exhaustive) {
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
      consider(g);
    }
  } else {
    const int L = n - 2;
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
          consider(g);
        }
      }
  }
  if (!best.ok) return ATOM_ENOPLAN;
  memset(out, 0, sizeof(*out));
  out->n_nodes = n;
  out->n_groups = static_cast<int32_t>(best_g.size());
  out->n_slots = best.K;
  out->n_gslots = 2;
  out->overlap_ok = best.overlap ? 1 : 0;
  out->exhaustive = exhaustive ? 1 : 0;
  out->accum = accum;
  for (size_t i = 0; i < best_g.size(); ++i) {
    out->first[i] = best_g[i].first;
    out->last[i] = best_g[i].second;
  }
  out->budget_bytes = budget;
  out->reserve_bytes = reserve;
  out->slot_bytes = best.S;
  out->arena_bytes = best.arena;
  out->h2d_bytes = best.h2d + ckpt_xfer_bytes(*cfg);
  out->d2h_bytes = best.d2h + ckpt_xfer_bytes(*cfg);
  uint64_t W = 0, Smin = 0;
  for (int i = 0; i < n; ++i) {
    W += costs[i].weight_bytes;
    Smin = std::max<uint64_t>(Smin, costs[i].weight_bytes);
  }
  // Lower bound on host-to-device bytes for any schedule in this memory
  // model: every weight once, plus what cannot stay resident into the
  // backward (the budget minus the reserve, two gradient slots and the
  // weights of the group being executed).
  const uint64_t keep = budget > reserve + 3 * Smin ? budget - reserve - 3 * Smin : 0;
  out->forced_h2d_bytes = W + (W > keep ? W - keep : 0) + ckpt_xfer_bytes(*cfg);
  out->pred_fwd_s = best.t_fwd;
  out->pred_step_s = best.t_step;
  out->n_evaluated = evaluated;
  return ATOM_OK;
}

int atom_plan_fixed(const atom_config* cfg, int32_t n_groups, const int32_t* last, int32_t n_slots,
                    int32_t n_gslots, atom_plan* out) {
  if (!cfg || !last || !out || !check_config(*cfg).empty()) return ATOM_EINVAL;
  if (n_gslots < 2 || n_gslots > ATOM_MAX_GSLOTS) return ATOM_EINVAL;
  const int n = cfg->n_layer + 2;
  if (n_groups < 1 || n_groups > n || n_slots < std::min<int32_t>(n_groups, 2) || n_slots > n_groups) return ATOM_EINVAL;
  std::vector<std::pair<int, int>> g;
  int start = 0;
  for (int i = 0; i < n_groups; ++i) {
    if (last[i] < start || last[i] >= n) return ATOM_EINVAL;
    g.push_back({start, last[i]});
    start = last[i] + 1;
  }
  if (start != n) return ATOM_EINVAL;
  std::vector<atom_node_cost> c(n);
  atom_node_costs(cfg, c.data(), n);
  uint64_t reserve = 0;
  atom_reserve_bytes(cfg, &reserve);
  uint64_t S = 0;
  for (auto& x : g) {
    uint64_t w = 0;
    for (int i = x.first; i <= x.second; ++i) w += c[i].weight_bytes;
    S = std::max(S, w);
  }
  const uint64_t grad = 2 * S + ((cfg->accum > 1 && cfg->dtype == ATOM_BF16) ? 2 * S : 0);
  const uint64_t budget = reserve + static_cast<uint64_t>(n_slots) * S + grad;
  Eval ev = evaluate(g, c.data(), budget, reserve, cfg->accum, cfg->dtype);
  if (!ev.ok || ev.K != n_slots) return ATOM_EINVAL;
  memset(out, 0, sizeof(*out));
  out->n_nodes = n;
  out->n_groups = n_groups;
  out->n_slots = n_slots;
  out->n_gslots = n_gslots;
  out->overlap_ok = ev.overlap ? 1 : 0;
  out->accum = cfg->accum;
  for (int i = 0; i < n_groups; ++i) {
    out->first[i] = g[i].first;
    out->last[i] = g[i].second;
  }
  out->reserve_bytes = reserve;
  out->slot_bytes = S;
  out->arena_bytes = arena_layout(*cfg, S, n_slots, n_gslots).arena_bytes;
  out->budget_bytes = out->arena_bytes;
  out->h2d_bytes = ev.h2d + ckpt_xfer_bytes(*cfg);
  out->d2h_bytes = ev.d2h + ckpt_xfer_bytes(*cfg);
  out->forced_h2d_bytes = out->h2d_bytes;
  out->pred_fwd_s = ev.t_fwd;
  out->pred_step_s = ev.t_step;
  out->n_evaluated = 1;
  return ATOM_OK;
}

int atom_plan_partition(const atom_config* cfg, uint64_t budget, const atom_node_cost* costs, int32_t n_costs,
                        atom_plan* out) {
  if (!cfg || !out || !check_config(*cfg).empty()) return ATOM_EINVAL;
  const int n = cfg->n_layer + 2;
  std::vector<atom_node_cost> c(n);
  if (costs) {
    if (n_costs != n) return ATOM_EINVAL;
    for (int i = 0; i < n; ++i) c[i] = costs[i];
  } else {
    int s = atom_node_costs(cfg, c.data(), n);
    if (s != ATOM_OK) return s;
  }
  uint64_t reserve = 0;
  atom_reserve_bytes(cfg, &reserve);
  int s = atom_plan_search(cfg, budget, reserve, c.data(), n, out);
  if (s != ATOM_OK) return s;
  // Slot sizes are multiples of the 256-byte alignment and the reserve
  // already includes its padding, so the carved arena is exactly the size the
  // search assumed.
  const ArenaLayout a = arena_layout(*cfg, out->slot_bytes, out->n_slots, 2);
  if (a.arena_bytes != out->arena_bytes || a.arena_bytes > budget) return ATOM_ENOPLAN;
  // leftover budget -> extra gradient slots
  const uint64_t extra = (budget - a.arena_bytes) / out->slot_bytes;
  out->n_gslots = static_cast<int32_t>(std::min<uint64_t>(ATOM_MAX_GSLOTS, 2 + extra));
  out->arena_bytes = arena_layout(*cfg, out->slot_bytes, out->n_slots, out->n_gslots).arena_bytes;
  if (out->arena_bytes > budget) return ATOM_ENOPLAN;
  return ATOM_OK;
}

}  // extern "C"
