// Host gradient accumulation: after a group's gradients reach pinned host
// memory, the accumulation thread adds them into the fp32 accumulators on the
// host thread pool (the gradient of the global batch, Section III-E).
#include "context.h"

namespace atom {
namespace rt {

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
  const int g = gi % c->G;
  const uint8_t* hg = c->h_g;
  const auto& rows = c->acc_rows0;  // group 0 with row-sparse embedding: wte's packed rows
  const uint64_t wte_el = (c->node_off[0] + wte_off(c)) / c->e;
  std::vector<Range> rs;
  for (const Range& r : c->group_ranges[g])
    if (!(g == 0 && !rows.empty() && r.off == wte_el)) rs.push_back(r);
  uint64_t total = 0;
  for (auto& r : rs) total += r.n;
  const int nt = c->acc_threads;
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
  }, nt);
  if (g == 0 && !rows.empty()) {
    // packed row i of h_g's wte region goes to row rows[i]; every other row
    // of the gradient is zero, which adds nothing
    const uint64_t d = c->d, nr = rows.size();
    c->pool->run([&](int ti) {
      for (uint64_t i = nr * ti / nt, e = nr * (ti + 1) / nt; i < e; ++i) {
        float* acc = c->h_acc + wte_el + static_cast<uint64_t>(rows[i]) * d;
        if (c->dt == DT_BF16)
          accum_range<uint16_t>(acc, reinterpret_cast<const uint16_t*>(hg) + wte_el + i * d, d);
        else
          accum_range<float>(acc, reinterpret_cast<const float*>(hg) + wte_el + i * d, d);
      }
    }, nt);
  }
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
inline uint16_t host_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// AdamW over the parameters of nodes first..last (Section V-B; the formula
// atom_optimizer_step documents), on the host thread pool: reads the
// accumulators, updates the fp32 master and the moments, writes the
// working-dtype weights and zeroes the accumulators.  Each element's
// arithmetic is the same whatever the range and the thread split, so an update
// group by group equals one over the whole model bit for bit.
void adamw_nodes(atom_ctx* c, int first, int last, const atom_adamw& hp, float grad_scale, int32_t step, int nt) {
  // per-tensor element ranges with their decay flag
  struct Seg {
    uint64_t off, n;
    bool decay;
  };
  std::vector<Seg> segs;
  uint64_t total = 0;
  for (int node = first; node <= last; ++node)
    for (const auto& t : c->tens[node]) {
      const bool decay = t.name == "w_qkv" || t.name == "w_o" || t.name == "w_fc" || t.name == "w_pr" ||
                         t.name == "w_head";
      segs.push_back({(c->node_off[node] + t.offset) / c->e, t.bytes / c->e, decay});
      total += t.bytes / c->e;
    }
  const float lr = hp.lr, b1 = hp.beta1, b2 = hp.beta2, eps = hp.eps, wd = hp.weight_decay;
  // 1 - beta and the bias corrections in double: in fp32 they would lose
  // most of their digits to cancellation (1 - 0.999^2 keeps about three)
  const double b1d = b1, b2d = b2;
  const float c1 = static_cast<float>(1.0 - b1d), c2 = static_cast<float>(1.0 - b2d);
  const float bc1 = static_cast<float>(1.0 - std::pow(b1d, step));
  const float bc2 = static_cast<float>(1.0 - std::pow(b2d, step));
  const bool bf = c->dt == DT_BF16;
  c->pool->run([&](int ti) {
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
  }, nt);
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
    const bool update = (gi & ACC_UPDATE) != 0;
    gi &= ~ACC_UPDATE;
    // queued only once its gradient copy has finished
    auto t0 = std::chrono::steady_clock::now();
    accumulate_group(c, gi);
    auto t1 = std::chrono::steady_clock::now();
    c->acc_seconds += std::chrono::duration<double>(t1 - t0).count();
    if (update) {
      // the last gradients of the global batch for this group are in: apply
      // the armed optimizer step to its parameters now, while the GPU runs
      // the backward of the groups before it
      const int g = gi % c->G;
      adamw_nodes(c, c->plan.first[g], c->plan.last[g], c->upd_hp, c->upd_scale, c->upd_step,
                  c->acc_threads);
      c->upd_seconds += std::chrono::duration<double>(std::chrono::steady_clock::now() - t1).count();
      ++c->upd_groups;
    }
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

}  // namespace rt
}  // namespace atom

using namespace atom::rt;

extern "C" {

int atom_optimizer_init(atom_ctx* c) {
  if (!c) return ATOM_EINVAL;
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  const uint64_t n = c->model_bytes / c->e;
  // Pinned when the system grants it; the GPU never reads this state, so when
  // pinning is refused (the swap buffers already hold most of what the system
  // lets the GPU map) the state goes to pageable memory, which the host
  // arithmetic reads at the same speed.  The three buffers share one kind.
  if (!c->h_master) {
    float** bufs[] = {&c->h_master, &c->h_m, &c->h_v};
    c->opt_pinned = true;
    for (float** b : bufs) {
      if (hipHostMalloc(reinterpret_cast<void**>(b), n * 4, hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        *b = nullptr;
        c->opt_pinned = false;
        break;
      }
    }
    if (!c->opt_pinned) {
      for (float** b : bufs)
        if (*b) (void)hipHostFree(*b);
      for (float** b : bufs) {
        *b = nullptr;
        if (posix_memalign(reinterpret_cast<void**>(b), 4096, n * 4) != 0) {
          *b = nullptr;
          for (float** f : bufs) {
            free(*f);
            *f = nullptr;
          }
          return fail(c, ATOM_ENOMEM_HOST, "allocation of the optimizer state (" + std::to_string(3 * n * 4) +
                                               " bytes) failed");
        }
      }
    }
  }
  const int nt = c->pool->size();
  c->pool->run([&](int ti) {
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
  }, nt);
  return ATOM_OK;
}

int atom_optimizer_step(atom_ctx* c, const atom_adamw* hp, float grad_scale, int32_t step) {
  if (!c || !hp || step < 1) return fail(c, ATOM_EINVAL, "bad optimizer arguments");
  if (!c->h_master) return fail(c, ATOM_ESTATE, "atom_optimizer_init was not called");
  int st = sync_all(c);
  if (st != ATOM_OK) return st;
  adamw_nodes(c, 0, c->L + 1, *hp, grad_scale, step, c->pool->size());
  drop_residency(c);
  return ATOM_OK;
}

int atom_optimizer_arm(atom_ctx* c, const atom_adamw* hp, float grad_scale, int32_t step) {
  if (!c || !hp || step < 1) return fail(c, ATOM_EINVAL, "bad optimizer arguments");
  if (!c->h_master) return fail(c, ATOM_ESTATE, "atom_optimizer_init was not called");
  c->upd_hp = *hp;
  c->upd_scale = grad_scale;
  c->upd_step = step;
  c->upd_armed = true;
  return ATOM_OK;
}

}  // extern "C"
