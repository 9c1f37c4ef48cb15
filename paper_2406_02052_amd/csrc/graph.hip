#include "graph.h"

namespace petra {

GraphCache::~GraphCache() {
  clear();
  if (in_) (void)hipEventDestroy(in_);
  if (out_) (void)hipEventDestroy(out_);
  if (cap_) (void)hipStreamDestroy(cap_);
}

void GraphCache::clear() {
  for (auto& kv : execs_) (void)hipGraphExecDestroy(kv.second);
  execs_.clear();
  order_.clear();
}

hipError_t GraphCache::ensure() {
  if (cap_) return hipSuccess;
  hipError_t e;
  if ((e = hipStreamCreateWithFlags(&cap_, hipStreamNonBlocking)) != hipSuccess) return e;
  if ((e = hipEventCreateWithFlags(&in_, hipEventDisableTiming)) != hipSuccess) return e;
  return hipEventCreateWithFlags(&out_, hipEventDisableTiming);
}

hipError_t GraphCache::run(const Key& key, hipStream_t caller,
                           const std::function<void(hipStream_t)>& enqueue) {
  hipError_t e = ensure();
  if (e != hipSuccess) return e;
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
    if ((e = hipStreamBeginCapture(cap_, hipStreamCaptureModeThreadLocal)) != hipSuccess) return e;
    enqueue(cap_);
    hipGraph_t g = nullptr;
    const hipError_t launch_err = hipGetLastError();
    e = hipStreamEndCapture(cap_, &g);
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
  if ((e = hipEventRecord(in_, caller)) != hipSuccess) return e;
  if ((e = hipStreamWaitEvent(cap_, in_, 0)) != hipSuccess) return e;
  if ((e = hipGraphLaunch(it->second, cap_)) != hipSuccess) return e;
  if ((e = hipEventRecord(out_, cap_)) != hipSuccess) return e;
  return hipStreamWaitEvent(caller, out_, 0);
}

}  // namespace petra
