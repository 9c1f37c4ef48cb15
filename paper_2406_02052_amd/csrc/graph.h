// Cache of instantiated HIP graphs, one per distinct call signature (kind of
// call plus the device pointers it was given).  A cached call replays its
// graph on a private stream that is fenced with events to the caller's
// stream, so launch cost on the host is one graph launch per call.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <functional>
#include <list>
#include <map>
#include <vector>

namespace petra {

// First failure among the HIP runtime calls of an enqueue sequence (event
// records, cross-stream waits, device copies).  Enqueue code notes every
// status here instead of dropping it; the C ABI call that enqueued the work
// reports the failure as PETRA_ERR_HIP and clears it.
struct HipStatus {
  hipError_t err = hipSuccess;
  const char* what = nullptr;
  void note(hipError_t e, const char* call) {
    if (e != hipSuccess && err == hipSuccess) {
      err = e;
      what = call;
    }
  }
  void clear() {
    err = hipSuccess;
    what = nullptr;
  }
};
#define PETRA_HIP(status, call) (status).note((call), #call)

class GraphCache {
 public:
  using Key = std::vector<uintptr_t>;
  ~GraphCache();
  // Run `enqueue` (which launches work on the stream it is given, possibly
  // forking to other streams through events) as a graph keyed by `key`.
  // `lane` (0 or 1) selects one of two private replay streams, so that two
  // independent calls of one owner can replay concurrently.
  hipError_t run(const Key& key, hipStream_t caller, const std::function<void(hipStream_t)>& enqueue,
                 int lane = 0);
  void clear();
  size_t size() const { return execs_.size(); }
  static constexpr size_t kMaxGraphs = 64;

 private:
  hipError_t ensure();
  hipStream_t cap_[2] = {nullptr, nullptr};
  hipEvent_t in_[2] = {nullptr, nullptr}, out_[2] = {nullptr, nullptr};
  std::map<Key, hipGraphExec_t> execs_;
  std::list<Key> order_;
};

}  // namespace petra
