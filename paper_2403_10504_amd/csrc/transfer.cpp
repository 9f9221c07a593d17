// Host-link transfer machinery: FIFO worker threads and device-to-host copies
// on the system DMA engine (ROCr).
#include "transfer.h"

#include <hip/hip_runtime.h>

#include <unistd.h>

#include <cstdio>
#include <cstdlib>

namespace atom {

// ------------------------------------------------------------------ Worker
Worker::Worker() : th_([this] { loop(); }) {}

Worker::~Worker() {
  {
    std::lock_guard<std::mutex> l(m_);
    stop_ = true;
  }
  cv_.notify_all();
  th_.join();
}

void Worker::submit(Job job) {
  {
    std::lock_guard<std::mutex> l(m_);
    q_.push_back(std::move(job));
  }
  cv_.notify_one();
}

std::string Worker::drain() {
  std::unique_lock<std::mutex> l(m_);
  idle_cv_.wait(l, [this] { return q_.empty() && !busy_; });
  std::string e;
  e.swap(err_);
  return e;
}

bool Worker::failed() {
  std::lock_guard<std::mutex> l(m_);
  return !err_.empty();
}

void Worker::loop() {
  for (;;) {
    Job job;
    {
      std::unique_lock<std::mutex> l(m_);
      cv_.wait(l, [this] { return stop_ || !q_.empty(); });
      if (q_.empty()) return;  // stop requested and nothing left
      job = std::move(q_.front());
      q_.pop_front();
      busy_ = true;
    }
    std::string e = job();
    {
      std::lock_guard<std::mutex> l(m_);
      if (!e.empty() && err_.empty()) err_ = e;
      busy_ = false;
    }
    idle_cv_.notify_all();
  }
}

// --------------------------------------------------------------- DmaEngine
namespace {

struct AgentSearch {
  uint32_t bdf;  // (bus << 8) | (device << 3) | function
  uint32_t domain;
  int n_match = 0;
  hsa_agent_t gpu{}, cpu{};
  bool have_cpu = false;
};

hsa_status_t visit_agent(hsa_agent_t a, void* data) {
  auto* s = static_cast<AgentSearch*>(data);
  hsa_device_type_t type;
  if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &type) != HSA_STATUS_SUCCESS) return HSA_STATUS_SUCCESS;
  if (type == HSA_DEVICE_TYPE_CPU) {
    if (!s->have_cpu) {
      s->cpu = a;
      s->have_cpu = true;
    }
  } else if (type == HSA_DEVICE_TYPE_GPU) {
    uint32_t bdf = 0, domain = 0;
    if (hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_BDFID), &bdf) != HSA_STATUS_SUCCESS)
      return HSA_STATUS_SUCCESS;
    if (hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_DOMAIN), &domain) != HSA_STATUS_SUCCESS)
      domain = 0;
    // function bits are ignored: a GPU is function 0 of its device
    if ((bdf >> 3) == (s->bdf >> 3) && domain == s->domain) {
      s->gpu = a;
      s->n_match += 1;
    }
  }
  return HSA_STATUS_SUCCESS;
}

std::string hsa_err(const char* what, hsa_status_t st) {
  const char* msg = nullptr;
  hsa_status_string(st, &msg);
  return std::string(what) + ": " + (msg ? msg : "unknown ROCr error");
}

}  // namespace

DmaEngine::~DmaEngine() {
  if (ready_) hsa_signal_destroy(sig_);
  if (inited_) hsa_shut_down();
}

std::string DmaEngine::init(int hip_device, bool to_host) {
  to_host_ = to_host;
  int bus = 0, dev = 0, domain = 0;
  if (hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, hip_device) != hipSuccess ||
      hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, hip_device) != hipSuccess ||
      hipDeviceGetAttribute(&domain, hipDeviceAttributePciDomainID, hip_device) != hipSuccess)
    return "cannot read the PCI location of the HIP device";
  // The HIP runtime has initialised ROCr already; this takes a reference.
  hsa_status_t st = hsa_init();
  if (st != HSA_STATUS_SUCCESS) return hsa_err("hsa_init", st);
  inited_ = true;
  AgentSearch s;
  s.bdf = (static_cast<uint32_t>(bus) << 8) | (static_cast<uint32_t>(dev) << 3);
  s.domain = static_cast<uint32_t>(domain);
  st = hsa_iterate_agents(visit_agent, &s);
  if (st != HSA_STATUS_SUCCESS) return hsa_err("hsa_iterate_agents", st);
  if (s.n_match != 1 || !s.have_cpu) {
    char b[128];
    snprintf(b, sizeof b, "no unique ROCr agent for PCI %04x:%02x:%02x (%d matches)", domain, bus, dev, s.n_match);
    return b;
  }
  gpu_ = s.gpu;
  cpu_ = s.cpu;
  st = hsa_signal_create(0, 0, nullptr, &sig_);
  if (st != HSA_STATUS_SUCCESS) return hsa_err("hsa_signal_create", st);
  // A fixed engine keeps every gradient copy off the engine the weight copies
  // use; with the runtime's per-copy choice a copy now and then queued behind
  // other transfers for over 100 ms.
  uint32_t pref = 0;
  const hsa_status_t ps = to_host ? hsa_amd_memory_get_preferred_copy_engine(cpu_, gpu_, &pref)
                                  : hsa_amd_memory_get_preferred_copy_engine(gpu_, cpu_, &pref);
  if (ps == HSA_STATUS_SUCCESS && pref != 0) engine_ = pref & (~pref + 1);
  ready_ = true;
  return "";
}

std::string DmaEngine::check_known(const void* p, const char* what) {
  hsa_amd_pointer_info_t info{};
  info.size = sizeof(info);
  const hsa_status_t st = hsa_amd_pointer_info(const_cast<void*>(p), &info, nullptr, nullptr, nullptr);
  if (st != HSA_STATUS_SUCCESS) return hsa_err("hsa_amd_pointer_info", st);
  if (info.type == HSA_EXT_POINTER_TYPE_UNKNOWN)
    return std::string(what) + " is unknown to the ROCr runtime this library is bound to (a second ROCr copy "
           "in the process?)";
  return "";
}

std::string DmaEngine::copy(void* dst, const void* src, uint64_t bytes) {
  if (!ready_) return "DMA engine is not initialised";
  if (bytes == 0) return "";
  hsa_signal_store_screlease(sig_, 1);
  const hsa_agent_t da = to_host_ ? cpu_ : gpu_, sa = to_host_ ? gpu_ : cpu_;
  hsa_status_t st =
      engine_ ? hsa_amd_memory_async_copy_on_engine(dst, da, src, sa, bytes, 0, nullptr, sig_,
                                                    static_cast<hsa_amd_sdma_engine_id_t>(engine_), true)
              : hsa_amd_memory_async_copy(dst, da, src, sa, bytes, 0, nullptr, sig_);
  if (st != HSA_STATUS_SUCCESS) return hsa_err("hsa_amd_memory_async_copy", st);
  // The engine decrements the signal to 0 when done, below 0 on error.  Poll
  // with short sleeps: an interrupt-driven wait occasionally woke up over
  // 100 ms late, which stalls the backward waiting for the gradient slot.
  hsa_signal_value_t v;
  while ((v = hsa_signal_load_scacquire(sig_)) >= 1) usleep(POLL_US);
  if (v < 0) return "DMA copy failed";
  return "";
}

}  // namespace atom
