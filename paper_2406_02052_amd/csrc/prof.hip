#include "prof.h"

namespace petra {

thread_local LaunchEvents g_launch_events;

const char* kernel_class_name(int k) {
  static const char* names[K_NUM_CLASSES] = {
      "conv_fprop", "conv_dgrad", "conv_wgrad", "wgrad_reduce", "bn_finalize",
      "bn_bwd_finalize", "combine_fwd", "combine_bwd", "sgd_update",
      "refresh_weights"};
  return (k >= 0 && k < K_NUM_CLASSES) ? names[k] : "?";
}

Profiler::~Profiler() {
  for (auto& r : recs_) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  for (auto e : pool_) (void)hipEventDestroy(e);
}

hipEvent_t Profiler::take() {
  if (!pool_.empty()) {
    hipEvent_t e = pool_.back();
    pool_.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void Profiler::begin(hipStream_t st) {
  (void)st;
  if (!enabled) return;
  pending_ = take();
  pending_stop_ = take();
  if (pending_ == nullptr || pending_stop_ == nullptr) {
    pending_ = pending_stop_ = nullptr;
    return;
  }
  g_launch_events.start = pending_;
  g_launch_events.stop = pending_stop_;
}

void Profiler::end(int kind, hipStream_t st, double fl, double by) {
  (void)st;
  g_launch_events = LaunchEvents{};
  if (!enabled || pending_ == nullptr) return;
  recs_.push_back(ProfRecord{kind, pending_, pending_stop_, fl, by});
  pending_ = pending_stop_ = nullptr;
}

hipError_t Profiler::collect() {
  for (auto& r : recs_) {
    hipError_t e = hipEventSynchronize(r.stop);
    if (e != hipSuccess) return e;
    float t = 0.f;
    e = hipEventElapsedTime(&t, r.start, r.stop);
    if (e != hipSuccess) return e;
    launches[r.kind] += 1;
    ms[r.kind] += t;
    flops[r.kind] += r.flops;
    bytes[r.kind] += r.bytes;
    pool_.push_back(r.start);
    pool_.push_back(r.stop);
  }
  recs_.clear();
  return hipSuccess;
}

void Profiler::reset() {
  for (int k = 0; k < K_NUM_CLASSES; ++k) {
    launches[k] = 0;
    ms[k] = flops[k] = bytes[k] = 0.0;
  }
}

}  // namespace petra
