#include "graph.h"

namespace petra {

GraphCache::~GraphCache() {
  clear();
  for (int i = 0; i < 2; ++i) {
    if (in_[i]) (void)hipEventDestroy(in_[i]);
    if (out_[i]) (void)hipEventDestroy(out_[i]);
    if (cap_[i]) (void)hipStreamDestroy(cap_[i]);
  }
}

void GraphCache::clear() {
  for (auto& kv : execs_) (void)hipGraphExecDestroy(kv.second);
  execs_.clear();
  order_.clear();
}

hipError_t GraphCache::ensure() {
  if (cap_[1]) return hipSuccess;
  hipError_t e;
  for (int i = 0; i < 2; ++i) {
    if (!cap_[i] && (e = hipStreamCreateWithFlags(&cap_[i], hipStreamNonBlocking)) != hipSuccess) return e;
    if (!in_[i] && (e = hipEventCreateWithFlags(&in_[i], hipEventDisableTiming)) != hipSuccess) return e;
    if (!out_[i] && (e = hipEventCreateWithFlags(&out_[i], hipEventDisableTiming)) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t GraphCache::run(const Key& key, hipStream_t caller,
                           const std::function<void(hipStream_t)>& enqueue, int lane) {
  hipError_t e = ensure();
  if (e != hipSuccess) return e;
  lane = lane ? 1 : 0;
  hipStream_t cap = cap_[lane];
  auto it = execs_.find(key);
  if (it == execs_.end()) {
    if (execs_.size() >= kMaxGraphs) {  // evict the oldest signature
      auto old = execs_.find(order_.front());
      if (old != execs_.end()) {
        (void)hipGraphExecDestroy(old->second);
        execs_.erase(old);
      }
      order_.pop_front();
    }
    if ((e = hipStreamBeginCapture(cap, hipStreamCaptureModeThreadLocal)) != hipSuccess) return e;
    enqueue(cap);
    hipGraph_t g = nullptr;
    const hipError_t launch_err = hipGetLastError();
    e = hipStreamEndCapture(cap, &g);
    if (launch_err != hipSuccess) e = launch_err;
    if (e != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return e;
    }
    hipGraphExec_t x = nullptr;
    e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) return e;
    it = execs_.emplace(key, x).first;
    order_.push_back(key);
  }
  if ((e = hipEventRecord(in_[lane], caller)) != hipSuccess) return e;
  if ((e = hipStreamWaitEvent(cap, in_[lane], 0)) != hipSuccess) return e;
  if ((e = hipGraphLaunch(it->second, cap)) != hipSuccess) return e;
  if ((e = hipEventRecord(out_[lane], cap)) != hipSuccess) return e;
  return hipStreamWaitEvent(caller, out_[lane], 0);
}

}  // namespace petra
