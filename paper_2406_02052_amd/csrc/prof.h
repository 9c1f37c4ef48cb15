// Optional per-launch timing with HIP events on the launching stream, used by
// the benchmark to measure each kernel class's average duration live.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <string>
#include <vector>

namespace petra {

enum KernelClass {
  K_CONV_FPROP = 0, K_CONV_DGRAD, K_CONV_WGRAD, K_WGRAD_REDUCE, K_BN_FINALIZE, K_BN_BWD_FINALIZE,
  K_COMBINE_FWD, K_COMBINE_BWD, K_SGD, K_REFRESH, K_NUM_CLASSES
};

const char* kernel_class_name(int k);

// Start/stop events that the next kernel launch attaches to its dispatch
// (set by Profiler::begin, cleared by Profiler::end; null when not profiling),
// and the host handle of the kernel that launch used.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  const void* fn = nullptr;
};
extern thread_local LaunchEvents g_launch_events;

// Every kernel launch of the library goes through this macro: with profiling
// on, the runtime timestamps the dispatch itself (kernel start to end), so the
// per-launch durations are kernel durations, not event-packet intervals.
#define PETRA_LAUNCH(kernel, grid, block, shmem, stream, ...)                                  \
  do {                                                                                         \
    ::petra::g_launch_events.fn = reinterpret_cast<const void*>(kernel);                   \
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ::petra::g_launch_events.start,  \
                          ::petra::g_launch_events.stop, 0, __VA_ARGS__);                      \
  } while (0)

struct ProfRecord {
  int kind;
  hipEvent_t start, stop;
  double flops, bytes;
  const void* kernel;
};

// Totals of one kernel (template instance) within one class.
struct KernelStat {
  const void* kernel = nullptr;
  int kind = 0;
  std::string name;   // demangled symbol, e.g. "petra::sgd_kernel"
  long launches = 0;
  double ms = 0.0, flops = 0.0, bytes = 0.0;
};

// Demangled name of a kernel from its host handle ("?" if not found).
std::string kernel_symbol_name(const void* kernel);

class Profiler {
 public:
  ~Profiler();
  bool enabled = false;
  // Bracket exactly one kernel launch of class `kind` (no-op when disabled): the
  // launch in between carries the start/stop events on its dispatch.
  void begin(hipStream_t st);
  void end(int kind, hipStream_t st, double flops, double bytes);
  // Aggregate finished records (synchronises on their events) into totals.
  hipError_t collect();
  void reset();
  long launches[K_NUM_CLASSES] = {};
  double ms[K_NUM_CLASSES] = {};
  double flops[K_NUM_CLASSES] = {};
  double bytes[K_NUM_CLASSES] = {};
  std::vector<KernelStat> kernels;   // per kernel instance, in order of first launch

 private:
  std::vector<hipEvent_t> pool_;
  std::vector<ProfRecord> recs_;
  hipEvent_t pending_ = nullptr, pending_stop_ = nullptr;
  hipEvent_t take();
};

}  // namespace petra
