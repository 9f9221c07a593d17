// Host-link transfer machinery of the swap engine.
//
// Worker: a FIFO thread that runs submitted jobs in order, so that calls into
// the HIP runtime which may block the calling thread (a copy whose stream
// dependency is still pending) never stall the thread that feeds the compute
// stream.
//
// DmaEngine: copies between device memory and pinned host memory on one of
// the GPU's system DMA (SDMA) engines through the ROCr API.  Used for
// device-to-host gradient copies:  The HIP runtime moves device-to-pinned-host data with a copy
// kernel; under the training kernels, which occupy every compute unit, such a
// kernel is starved of compute units and a 0.4 GB gradient copy can take
// several times its link time.  The DMA engine needs no compute unit.  A copy
// here is synchronous for its calling (worker) thread; ordering against the
// compute stream is established by the caller on the host (wait for the
// producer's event before the copy; publish completion afterwards).
#pragma once

#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>
#include <stdint.h>

#include <condition_variable>
#include <deque>
#include <functional>
#include <mutex>
#include <string>
#include <thread>

namespace atom {

class Worker {
 public:
  // A job returns an empty string on success, else an error description.
  using Job = std::function<std::string()>;
  Worker();
  ~Worker();
  void submit(Job job);
  // Waits until every submitted job has run.  Returns the first error since
  // the last drain (empty if none) and clears it.
  std::string drain();
  // True once a job has failed (until drained); later jobs still run.
  bool failed();

 private:
  void loop();
  std::thread th_;
  std::mutex m_;
  std::condition_variable cv_, idle_cv_;
  std::deque<Job> q_;
  bool busy_ = false, stop_ = false;
  std::string err_;
};

// Sleep between polls of a copy or event that is still in flight.
constexpr int POLL_US = 50;

class DmaEngine {
 public:
  ~DmaEngine();
  // Finds the ROCr agent of HIP device `hip_device` (by PCI location) and the
  // host agent, picks the engine (the lowest the runtime recommends for the
  // direction) and creates the completion signal.  Empty string on success.
  std::string init(int hip_device, bool to_host);
  // Copies `bytes` (device -> pinned host if to_host, else the reverse) on
  // the engine and waits for the copy to finish.  Empty string on success.
  std::string copy(void* dst, const void* src, uint64_t bytes);
  // Checks that `p` (device memory or pinned host memory the HIP runtime
  // allocated) is known to the ROCr instance this library calls.  A process
  // can hold two ROCr copies (a profiler may preload its own); the copies
  // must run on the one the HIP runtime uses.  Empty string on success.
  std::string check_known(const void* p, const char* what);
  bool ready() const { return ready_; }

 private:
  hsa_agent_t gpu_{}, cpu_{};
  hsa_signal_t sig_{};
  uint32_t engine_ = 0;  // one SDMA engine id bit, 0: the runtime's choice
  bool to_host_ = true;
  bool ready_ = false, inited_ = false;
};

}  // namespace atom
