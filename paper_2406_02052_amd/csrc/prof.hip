#include "prof.h"

#include <cxxabi.h>
#include <dlfcn.h>

#include <cstdlib>

namespace petra {

std::string kernel_symbol_name(const void* kernel) {
  Dl_info info{};
  if (kernel == nullptr || dladdr(kernel, &info) == 0 || info.dli_sname == nullptr ||
      info.dli_saddr != kernel)
    return "?";
  int status = 0;
  char* d = abi::__cxa_demangle(info.dli_sname, nullptr, nullptr, &status);
  std::string n = d != nullptr ? d : info.dli_sname;
  std::free(d);
  // "void petra::k<...>(args)" -> "petra::k<...>": the argument list is the
  // last parenthesised group at template depth 0
  if (n.compare(0, 5, "void ") == 0) n = n.substr(5);
  int depth = 0;
  size_t cut = std::string::npos;
  for (size_t i = 0; i < n.size(); ++i) {
    if (n[i] == '<') ++depth;
    if (n[i] == '>') --depth;
    if (n[i] == '(' && depth == 0) cut = i;
  }
  return cut == std::string::npos ? n : n.substr(0, cut);
}

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
  const void* kernel = g_launch_events.fn;
  g_launch_events = LaunchEvents{};
  if (!enabled || pending_ == nullptr) return;
  recs_.push_back(ProfRecord{kind, pending_, pending_stop_, fl, by, kernel});
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
    KernelStat* ks = nullptr;
    for (KernelStat& k : kernels)
      if (k.kernel == r.kernel && k.kind == r.kind) ks = &k;
    if (ks == nullptr) {
      kernels.push_back(KernelStat{r.kernel, r.kind, kernel_symbol_name(r.kernel)});
      ks = &kernels.back();
    }
    ks->launches += 1;
    ks->ms += t;
    ks->flops += r.flops;
    ks->bytes += r.bytes;
    pool_.push_back(r.start);
    pool_.push_back(r.stop);
  }
  recs_.clear();
  return hipSuccess;
}

void Profiler::reset() {
  kernels.clear();
  for (int k = 0; k < K_NUM_CLASSES; ++k) {
    launches[k] = 0;
    ms[k] = flops[k] = bytes[k] = 0.0;
  }
}

}  // namespace petra
