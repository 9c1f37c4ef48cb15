// extern "C" entry points of petra.h: argument validation, error reporting
// and dispatch to the stage program.  Nothing here allocates device memory.
#include <cstdint>
#include <cstdio>
#include <functional>
#include <mutex>
#include <new>
#include <string>

#include "net.h"
#include "stage.h"

struct petra_stage {
  petra::Stage* impl;
};

struct petra_net {
  petra::Net* impl;
};

namespace {

thread_local std::string g_last_error;

petra_status fail(petra_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

petra_status ok() { return PETRA_OK; }

petra_status check_hip(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(PETRA_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
  return PETRA_OK;
}

bool pow2_multiple_of_8(int c) {
  if (c < 8 || c > 512 || c % 8 != 0) return false;
  const int g = c / 8;
  return (g & (g - 1)) == 0;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// [a, a+n) and [b, b+n) overlap without being identical.
bool partial_overlap(const void* a, const void* b, size_t n) {
  const char* x = static_cast<const char*>(a);
  const char* y = static_cast<const char*>(b);
  if (x == y) return false;
  return x < y + n && y < x + n;
}

bool any_overlap(const void* a, const void* b, size_t n) {
  const char* x = static_cast<const char*>(a);
  const char* y = static_cast<const char*>(b);
  return x < y + n && y < x + n;
}

petra_status check_ready(const petra_stage* st) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  if (!st->impl->bound()) return fail(PETRA_ERR_STATE, "stage buffers not bound");
  if (!st->impl->has_workspace())
    return fail(PETRA_ERR_WORKSPACE,
                "no workspace bound (such a handle serves petra_stage_forward_noalloc only)");
  return PETRA_OK;
}

petra_status check_act(const void* p, const char* name) {
  if (p == nullptr) return fail(PETRA_ERR_INVALID_ARG, std::string("null pointer: ") + name);
  if (!aligned16(p)) return fail(PETRA_ERR_ALIGN, std::string("misaligned pointer: ") + name);
  return PETRA_OK;
}

petra_status check_fwd(const petra::Stage& s, const void* x1, const void* x2, const void* y1,
                       const void* y2) {
  petra_status r;
  if ((r = check_act(x1, "x1")) || (r = check_act(x2, "x2")) || (r = check_act(y1, "y1")) ||
      (r = check_act(y2, "y2")))
    return r;
  const size_t n = static_cast<size_t>(s.M) * s.desc.c_half * s.esz;
  if (any_overlap(x1, x2, n) || any_overlap(y1, y2, n) || any_overlap(x1, y2, n) ||
      any_overlap(x2, y1, n) || partial_overlap(x1, y1, n) || partial_overlap(x2, y2, n))
    return fail(PETRA_ERR_ALIAS, "forward buffers overlap (only x1==y1, x2==y2 allowed)");
  return PETRA_OK;
}

petra_status check_bwd(const petra::Stage& s, const void* y1, const void* y2, const void* dy1,
                       const void* dy2, const void* x1, const void* x2, const void* dx1,
                       const void* dx2) {
  petra_status r;
  if ((r = check_act(y1, "y1")) || (r = check_act(y2, "y2")) || (r = check_act(dy1, "dy1")) ||
      (r = check_act(dy2, "dy2")) || (r = check_act(x1, "x1")) || (r = check_act(x2, "x2")) ||
      (r = check_act(dx1, "dx1")) || (r = check_act(dx2, "dx2")))
    return r;
  const size_t n = static_cast<size_t>(s.M) * s.desc.c_half * s.esz;
  const void* in[4] = {y1, y2, dy1, dy2};
  const void* out[4] = {x1, x2, dx1, dx2};
  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) {
      if (i < j && (any_overlap(in[i], in[j], n) || any_overlap(out[i], out[j], n)))
        return fail(PETRA_ERR_ALIAS, "backward inputs or outputs overlap each other");
      if (i == j ? partial_overlap(in[i], out[j], n) : any_overlap(in[i], out[j], n))
        return fail(PETRA_ERR_ALIAS,
                    "backward buffers overlap (only x1==y1, x2==y2, dx1==dy1, dx2==dy2 allowed)");
    }
  return PETRA_OK;
}

enum CallKind : uintptr_t { CALL_FWD = 1, CALL_BWD, CALL_UPD, CALL_SYNC };

// Enqueue `work` on `stream`, through the stage's graph cache unless graphs are
// off or per-launch profiling is active.
petra_status hip_status(petra::HipStatus& h, const char* where) {
  if (h.err == hipSuccess) return PETRA_OK;
  const std::string msg = std::string(where) + ": " + h.what + ": " + hipGetErrorString(h.err);
  h.clear();
  return fail(PETRA_ERR_HIP, msg);
}

petra_status launch_status(petra::Stage& s, const char* where) {
  if (s.launch_error) {
    s.launch_error = false;
    s.hip_status.clear();
    return fail(PETRA_ERR_STATE, std::string(where) + ": internal error: unsupported kernel variant");
  }
  const petra_status r = hip_status(s.hip_status, where);
  if (r) return r;
  return check_hip(where);
}

// Status of the net's own runtime calls and of every stage program it enqueued.
petra_status net_status(petra::Net& n, const char* where) {
  petra_status r = hip_status(n.hip_status, where);
  for (petra::NetStage& ns : n.st) {
    const petra_status q = ns.has_blocks ? launch_status(*ns.blocks, where) : PETRA_OK;
    if (r == PETRA_OK) r = q;
  }
  if (r) return r;
  return check_hip(where);
}

petra_status launch(petra::Stage& s, const petra::GraphCache::Key& key, hipStream_t stream,
                    const char* where, const std::function<void(hipStream_t)>& work) {
  if (s.use_graphs && !s.prof.enabled) {
    const hipError_t e = s.graphs.run(key, stream, work);
    if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
    return launch_status(s, where);
  }
  work(stream);
  return launch_status(s, where);
}

uintptr_t P(const void* p) { return reinterpret_cast<uintptr_t>(p); }

}  // namespace

// Scratch of petra_stage_forward_noalloc: one array per device, held from the
// library's code object load until the process ends.  Host code never uses
// its name as an address: the device address comes from hipGetSymbolAddress,
// once per device, and is kept in g_scratch below.
static __device__ __align__(256) unsigned char scratch[PETRA_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`.
hipError_t static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

const char* petra_status_str(petra_status s) {
  switch (s) {
    case PETRA_OK: return "PETRA_OK";
    case PETRA_ERR_INVALID_ARG: return "PETRA_ERR_INVALID_ARG";
    case PETRA_ERR_SHAPE: return "PETRA_ERR_SHAPE";
    case PETRA_ERR_DTYPE: return "PETRA_ERR_DTYPE";
    case PETRA_ERR_ALIGN: return "PETRA_ERR_ALIGN";
    case PETRA_ERR_WORKSPACE: return "PETRA_ERR_WORKSPACE";
    case PETRA_ERR_STATE: return "PETRA_ERR_STATE";
    case PETRA_ERR_HIP: return "PETRA_ERR_HIP";
    case PETRA_ERR_ALIAS: return "PETRA_ERR_ALIAS";
  }
  return "PETRA_ERR_UNKNOWN";
}

const char* petra_last_error(void) { return g_last_error.c_str(); }

petra_status petra_stage_create(const petra_stage_desc* d, petra_stage** out) {
  g_last_error.clear();
  if (d == nullptr || out == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  if (d->dtype != PETRA_FP32 && d->dtype != PETRA_BF16)
    return fail(PETRA_ERR_DTYPE, "dtype must be PETRA_FP32 or PETRA_BF16");
  if (d->kind != PETRA_BLOCK_BASIC && d->kind != PETRA_BLOCK_BOTTLENECK)
    return fail(PETRA_ERR_INVALID_ARG, "unknown block kind");
  if (d->n < 1 || d->h < 1 || d->w < 1 || d->num_blocks < 1)
    return fail(PETRA_ERR_SHAPE, "n, h, w and num_blocks must be positive");
  if (!pow2_multiple_of_8(d->c_half))
    return fail(PETRA_ERR_SHAPE, "c_half must be 8 times a power of two, at most 512");
  if (d->kind == PETRA_BLOCK_BOTTLENECK && !pow2_multiple_of_8(d->c_mid))
    return fail(PETRA_ERR_SHAPE, "c_mid must be 8 times a power of two, at most 512");
  const long m = static_cast<long>(d->n) * d->h * d->w;
  const long cm = d->kind == PETRA_BLOCK_BOTTLENECK && d->c_mid > d->c_half ? d->c_mid : d->c_half;
  // every kernel addresses a tensor with 32-bit byte offsets below its
  // out-of-range sentinel (2^31): each half-tensor must stay below 2 GiB
  const long esz = d->dtype == PETRA_BF16 ? 2 : 4;
  if (m * cm * esz >= (1L << 31) || m >= (1L << 30))
    return fail(PETRA_ERR_SHAPE, "activation too large (N*H*W*C*element size must stay below 2^31 bytes)");
  if (!(d->bn_eps > 0.f) || d->bn_momentum < 0.f || d->bn_momentum > 1.f)
    return fail(PETRA_ERR_INVALID_ARG, "bn_eps must be > 0 and bn_momentum in [0, 1]");
  const int convs = d->num_blocks * 2 * (d->kind == PETRA_BLOCK_BASIC ? 2 : 3);
  if (convs > petra::MAX_WEIGHT_SEGS)
    return fail(PETRA_ERR_SHAPE, "too many blocks for one stage handle");
  petra_stage* h = new (std::nothrow) petra_stage;
  if (h == nullptr) return fail(PETRA_ERR_INVALID_ARG, "host allocation failed");
  h->impl = new (std::nothrow) petra::Stage(*d);
  if (h->impl == nullptr) {
    delete h;
    return fail(PETRA_ERR_INVALID_ARG, "host allocation failed");
  }
  *out = h;
  return ok();
}

petra_status petra_stage_destroy(petra_stage* st) {
  if (st == nullptr) return PETRA_OK;
  delete st->impl;
  delete st;
  return PETRA_OK;
}

petra_status petra_stage_query(const petra_stage* st, int64_t* n_params, int32_t* n_tensors,
                               int64_t* n_bn_channels, size_t* workspace_bytes) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  const petra::Stage& s = *st->impl;
  if (n_params) *n_params = s.n_params;
  if (n_tensors) *n_tensors = static_cast<int32_t>(s.infos.size());
  if (n_bn_channels) *n_bn_channels = s.n_bnch;
  if (workspace_bytes) *workspace_bytes = s.ws_need;
  return ok();
}

petra_status petra_stage_param_info(const petra_stage* st, int32_t index, petra_param_info* out) {
  if (st == nullptr || st->impl == nullptr || out == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "null argument");
  const petra::Stage& s = *st->impl;
  if (index < 0 || index >= static_cast<int32_t>(s.infos.size()))
    return fail(PETRA_ERR_INVALID_ARG, "tensor index out of range");
  *out = s.infos[index];
  return ok();
}

petra_status petra_stage_bind(petra_stage* st, float* params, float* grad_accum, float* momentum,
                              float* run_mean, float* run_var, void* workspace,
                              size_t workspace_bytes) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  if (!params || !grad_accum || !momentum || !run_mean || !run_var)
    return fail(PETRA_ERR_INVALID_ARG, "null buffer");
  const bool no_ws = workspace == nullptr && workspace_bytes == 0;
  if (!no_ws && (workspace == nullptr || workspace_bytes < st->impl->ws_need))
    return fail(PETRA_ERR_WORKSPACE, "workspace missing or smaller than petra_stage_query()");
  const void* ptrs[6] = {params, grad_accum, momentum, run_mean, run_var, workspace};
  for (const void* p : ptrs)
    if (!aligned16(p)) return fail(PETRA_ERR_ALIGN, "buffers must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(PETRA_ERR_ALIGN, "workspace must be 256-byte aligned");
  st->impl->bind(params, grad_accum, momentum, run_mean, run_var, workspace);
  return ok();
}

petra_status petra_stage_set_optimizer(petra_stage* st, const petra_sgd* opt) {
  if (st == nullptr || st->impl == nullptr || opt == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "null argument");
  if (!(opt->lr >= 0.f) || !(opt->momentum >= 0.f) || opt->momentum >= 1.f ||
      !(opt->weight_decay >= 0.f) || opt->accum_k < 1)
    return fail(PETRA_ERR_INVALID_ARG, "need lr >= 0, 0 <= momentum < 1, weight_decay >= 0, accum_k >= 1");
  st->impl->opt = *opt;
  st->impl->graphs.clear();  // cached graphs carry the old settings in their arguments
  return ok();
}

petra_status petra_stage_set_graphs(petra_stage* st, int32_t enable) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  st->impl->use_graphs = enable != 0;
  st->impl->graphs.clear();
  return ok();
}

petra_status petra_stage_set_streams(petra_stage* st, int32_t n) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  if (n < 1 || n > 3) return fail(PETRA_ERR_INVALID_ARG, "streams must be 1, 2 or 3");
  st->impl->bwd_streams = n;
  st->impl->graphs.clear();
  return ok();
}

petra_status petra_stage_sync_weights(petra_stage* st, void* stream) {
  petra_status r = check_ready(st);
  if (r) return r;
  if ((r = check_hip("before petra_stage_sync_weights"))) return r;
  petra::Stage& s = *st->impl;
  return launch(s, {CALL_SYNC}, static_cast<hipStream_t>(stream), "petra_stage_sync_weights",
                [&](hipStream_t q) { s.sync_weights(q); });
}

petra_status petra_stage_forward(petra_stage* st, const void* x1, const void* x2, void* y1,
                                 void* y2, void* stream) {
  petra_status r = check_ready(st);
  if (r) return r;
  if ((r = check_fwd(*st->impl, x1, x2, y1, y2))) return r;
  if ((r = check_hip("before petra_stage_forward"))) return r;
  petra::Stage& s = *st->impl;
  return launch(s, {CALL_FWD, P(x1), P(x2), P(y1), P(y2)}, static_cast<hipStream_t>(stream),
                "petra_stage_forward", [&](hipStream_t q) { s.forward(x1, x2, y1, y2, q); });
}

petra_status petra_stage_forward_noalloc(petra_stage* st, const void* x1, const void* x2,
                                         void* y1, void* y2, void* stream) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  petra::Stage& s = *st->impl;
  if (!s.bound()) return fail(PETRA_ERR_STATE, "stage buffers not bound");
  petra_status r;
  if ((r = check_fwd(s, x1, x2, y1, y2))) return r;
  if (s.fwd_need > static_cast<size_t>(PETRA_STATIC_SCRATCH_BYTES))
    return fail(PETRA_ERR_WORKSPACE,
                "petra_stage_forward_noalloc: the stage's forward needs " +
                    std::to_string(s.fwd_need) + " bytes of scratch; the static scratch holds " +
                    std::to_string(static_cast<size_t>(PETRA_STATIC_SCRATCH_BYTES)));
  if ((r = check_hip("before petra_stage_forward_noalloc"))) return r;
  void* base = nullptr;
  const hipError_t e = static_scratch(&base);
  if (e != hipSuccess)
    return fail(PETRA_ERR_HIP, std::string("petra_stage_forward_noalloc: scratch address: ") +
                                   hipGetErrorString(e));
  s.forward_on(static_cast<char*>(base), x1, x2, y1, y2, static_cast<hipStream_t>(stream));
  return launch_status(s, "petra_stage_forward_noalloc");
}

petra_status petra_stage_reconstruct_backward(petra_stage* st, const void* y1, const void* y2,
                                              const void* dy1, const void* dy2, void* x1,
                                              void* x2, void* dx1, void* dx2, void* stream) {
  petra_status r = check_ready(st);
  if (r) return r;
  if ((r = check_bwd(*st->impl, y1, y2, dy1, dy2, x1, x2, dx1, dx2))) return r;
  if ((r = check_hip("before petra_stage_reconstruct_backward"))) return r;
  petra::Stage& s = *st->impl;
  const hipError_t se = s.ensure_streams();
  if (se != hipSuccess) return fail(PETRA_ERR_HIP, std::string("stream setup: ") + hipGetErrorString(se));
  r = launch(s, {CALL_BWD, P(y1), P(y2), P(dy1), P(dy2), P(x1), P(x2), P(dx1), P(dx2)},
             static_cast<hipStream_t>(stream), "petra_stage_reconstruct_backward",
             [&](hipStream_t q) { s.backward(y1, y2, dy1, dy2, x1, x2, dx1, dx2, q); });
  if (r == PETRA_OK) s.count_backward();
  return r;
}

petra_status petra_stage_update(petra_stage* st, void* stream, int32_t* updated) {
  petra_status r = check_ready(st);
  if (r) return r;
  if ((r = check_hip("before petra_stage_update"))) return r;
  petra::Stage& s = *st->impl;
  const bool due = s.update_due();
  if (updated) *updated = due ? 1 : 0;
  if (!due) return ok();
  r = launch(s, {CALL_UPD}, static_cast<hipStream_t>(stream), "petra_stage_update",
             [&](hipStream_t q) { s.update_kernels(q); });
  if (r == PETRA_OK) s.mark_updated();
  return r;
}

petra_status petra_stage_step(petra_stage* st, const void* x1, const void* x2, void* y1, void* y2,
                              const void* yb1, const void* yb2, const void* dyb1,
                              const void* dyb2, void* xb1, void* xb2, void* dxb1, void* dxb2,
                              void* stream, int32_t* updated) {
  petra_status r = check_ready(st);
  if (r) return r;
  petra::Stage& s = *st->impl;
  if ((r = check_fwd(s, x1, x2, y1, y2))) return r;
  if ((r = check_bwd(s, yb1, yb2, dyb1, dyb2, xb1, xb2, dxb1, dxb2))) return r;
  const size_t n = static_cast<size_t>(s.M) * s.desc.c_half * s.esz;
  const void* f[4] = {x1, x2, y1, y2};
  const void* b[8] = {yb1, yb2, dyb1, dyb2, xb1, xb2, dxb1, dxb2};
  for (const void* p : f)
    for (const void* q : b)
      if (any_overlap(p, q, n))
        return fail(PETRA_ERR_ALIAS, "forward and backward buffers of a step overlap");
  if ((r = check_hip("before petra_stage_step"))) return r;
  const hipError_t e = s.ensure_streams();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("stream setup: ") + hipGetErrorString(e));
  // The update follows this step's backward (Eq. 5); whether it fires is decided
  // on the host from the backward count before the work is enqueued.
  s.count_backward();
  const bool due = s.update_due();
  hipStream_t main = static_cast<hipStream_t>(stream);
  // fork: the forward runs on its own stream after prior work on `main`, the
  // backward on `main` itself; join: the update (and later work on `main`)
  // follow both passes.  With graphs on, each pass replays the graph of its
  // standalone call (two replay lanes), so the step shares them.
  PETRA_HIP(s.hip_status, hipEventRecord(s.ev_fork, main));
  PETRA_HIP(s.hip_status, hipStreamWaitEvent(s.s_fwd, s.ev_fork, 0));
  if (s.use_graphs && !s.prof.enabled) {
    hipError_t ge = s.graphs.run({CALL_FWD, P(x1), P(x2), P(y1), P(y2)}, s.s_fwd,
                                 [&](hipStream_t c) { s.forward(x1, x2, y1, y2, c); }, 1);
    if (ge == hipSuccess)
      ge = s.graphs.run({CALL_BWD, P(yb1), P(yb2), P(dyb1), P(dyb2), P(xb1), P(xb2), P(dxb1), P(dxb2)},
                        main, [&](hipStream_t c) {
                          s.backward(yb1, yb2, dyb1, dyb2, xb1, xb2, dxb1, dxb2, c);
                        }, 0);
    PETRA_HIP(s.hip_status, hipEventRecord(s.ev_fwd, s.s_fwd));
    PETRA_HIP(s.hip_status, hipStreamWaitEvent(main, s.ev_fwd, 0));
    if (ge == hipSuccess && due)
      ge = s.graphs.run({CALL_UPD}, main, [&](hipStream_t c) { s.update_kernels(c); }, 0);
    r = ge != hipSuccess
            ? fail(PETRA_ERR_HIP, std::string("petra_stage_step: ") + hipGetErrorString(ge))
            : launch_status(s, "petra_stage_step");
  } else {
    if (s.defer_wgrad && s.bwd_streams == 1 && !s.prof.enabled) {
      // the forward stream is idle once the forward is done: the backward puts
      // most of its deferred weight gradients there (after the forward's
      // launches; the join below covers them)
      s.forward(x1, x2, y1, y2, s.s_fwd);
      s.backward(yb1, yb2, dyb1, dyb2, xb1, xb2, dxb1, dxb2, main, s.s_fwd);
    } else {
      // the backward is the longer chain: enqueue it first so its first kernels
      // do not wait behind the host time of the forward's launches
      s.backward(yb1, yb2, dyb1, dyb2, xb1, xb2, dxb1, dxb2, main);
      s.forward(x1, x2, y1, y2, s.s_fwd);
    }
    PETRA_HIP(s.hip_status, hipEventRecord(s.ev_fwd, s.s_fwd));
    PETRA_HIP(s.hip_status, hipStreamWaitEvent(main, s.ev_fwd, 0));
    if (due) s.update_kernels(main);
    r = launch_status(s, "petra_stage_step");
  }
  if (r == PETRA_OK && due) s.mark_updated();
  if (updated) *updated = (r == PETRA_OK && due) ? 1 : 0;
  return r;
}

// ---------------------------------------------------------------------------
// multi-stage schedule
// ---------------------------------------------------------------------------

petra_status petra_net_create(const petra_net_desc* d, petra_net** out) {
  g_last_error.clear();
  if (d == nullptr || out == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  if (d->dtype != PETRA_FP32 && d->dtype != PETRA_BF16)
    return fail(PETRA_ERR_DTYPE, "dtype must be PETRA_FP32 or PETRA_BF16");
  if (d->num_stages < 1 || d->num_stages > PETRA_MAX_STAGES)
    return fail(PETRA_ERR_SHAPE, "num_stages must be in [1, PETRA_MAX_STAGES]");
  if (d->n < 1 || d->h < 1 || d->w < 1 || d->blocks_per_stage < 1)
    return fail(PETRA_ERR_SHAPE, "n, h, w and blocks_per_stage must be positive");
  if (d->c_img < 1 || d->c_img > 8) return fail(PETRA_ERR_SHAPE, "c_img must be in [1, 8]");
  if (d->classes < 1 || d->classes > 64) return fail(PETRA_ERR_SHAPE, "classes must be in [1, 64]");
  const int div = 1 << (d->num_stages - 1);
  if (d->h % div != 0 || d->w % div != 0)
    return fail(PETRA_ERR_SHAPE, "h and w must be divisible by 2^(num_stages-1)");
  for (int j = 0; j < d->num_stages; ++j) {
    if (d->widths[j] % 2 != 0 || !pow2_multiple_of_8(d->widths[j] / 2))
      return fail(PETRA_ERR_SHAPE, "widths[j]/2 must be 8 times a power of two, at most 512");
    const long m = static_cast<long>(d->n) * (d->h >> j) * (d->w >> j);
    const long esz = d->dtype == PETRA_BF16 ? 2 : 4;
    if (m * d->widths[j] * esz >= (1L << 31))
      return fail(PETRA_ERR_SHAPE, "activation too large (N*H*W*C*element size must stay below 2^31 bytes)");
  }
  if (!(d->bn_eps > 0.f) || d->bn_momentum < 0.f || d->bn_momentum > 1.f)
    return fail(PETRA_ERR_INVALID_ARG, "bn_eps must be > 0 and bn_momentum in [0, 1]");
  if (d->blocks_per_stage * 4 > petra::MAX_WEIGHT_SEGS)
    return fail(PETRA_ERR_SHAPE, "too many blocks per stage");
  if ((d->input_buffer != 0 && d->input_buffer != 1) ||
      (d->param_buffer != 0 && d->param_buffer != 1) ||
      (d->split_stages != 0 && d->split_stages != 1))
    return fail(PETRA_ERR_INVALID_ARG, "input_buffer, param_buffer and split_stages must be 0 or 1");
  petra_net* h = new (std::nothrow) petra_net;
  if (h == nullptr) return fail(PETRA_ERR_INVALID_ARG, "host allocation failed");
  h->impl = new (std::nothrow) petra::Net(*d);
  if (h->impl == nullptr) {
    delete h;
    return fail(PETRA_ERR_INVALID_ARG, "host allocation failed");
  }
  *out = h;
  return ok();
}

petra_status petra_net_num_stages(const petra_net* net, int32_t* stages) {
  if (net == nullptr || net->impl == nullptr || stages == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "null argument");
  *stages = net->impl->J;
  return ok();
}

petra_status petra_net_destroy(petra_net* net) {
  if (net == nullptr) return PETRA_OK;
  delete net->impl;
  delete net;
  return PETRA_OK;
}

petra_status petra_net_query(const petra_net* net, int64_t* n_params, int32_t* n_tensors,
                             int64_t* n_bn_channels, size_t* workspace_bytes) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  const petra::Net& s = *net->impl;
  if (n_params) *n_params = s.n_params;
  if (n_tensors) *n_tensors = static_cast<int32_t>(s.infos.size());
  if (n_bn_channels) *n_bn_channels = s.n_bnch;
  if (workspace_bytes) *workspace_bytes = s.ws_need;
  return ok();
}

petra_status petra_net_param_info(const petra_net* net, int32_t index, petra_param_info* out) {
  if (net == nullptr || net->impl == nullptr || out == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "null argument");
  const petra::Net& s = *net->impl;
  if (index < 0 || index >= static_cast<int32_t>(s.infos.size()))
    return fail(PETRA_ERR_INVALID_ARG, "tensor index out of range");
  *out = s.infos[index];
  return ok();
}

petra_status petra_net_bind(petra_net* net, float* params, float* grad_accum, float* momentum,
                            float* run_mean, float* run_var, void* workspace,
                            size_t workspace_bytes) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  if (!params || !grad_accum || !momentum || !run_mean || !run_var)
    return fail(PETRA_ERR_INVALID_ARG, "null buffer");
  if (workspace == nullptr || workspace_bytes < net->impl->ws_need)
    return fail(PETRA_ERR_WORKSPACE, "workspace missing or smaller than petra_net_query()");
  const void* ptrs[5] = {params, grad_accum, momentum, run_mean, run_var};
  for (const void* p : ptrs)
    if (!aligned16(p)) return fail(PETRA_ERR_ALIGN, "buffers must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(PETRA_ERR_ALIGN, "workspace must be 256-byte aligned");
  net->impl->bind(params, grad_accum, momentum, run_mean, run_var, workspace);
  return ok();
}

petra_status petra_net_set_optimizer(petra_net* net, const petra_sgd* opt) {
  if (net == nullptr || net->impl == nullptr || opt == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "null argument");
  if (!(opt->lr >= 0.f) || !(opt->momentum >= 0.f) || opt->momentum >= 1.f ||
      !(opt->weight_decay >= 0.f) || opt->accum_k < 1)
    return fail(PETRA_ERR_INVALID_ARG, "need lr >= 0, 0 <= momentum < 1, weight_decay >= 0, accum_k >= 1");
  net->impl->opt = *opt;
  for (petra::NetStage& s : net->impl->st) {
    if (!s.has_blocks) continue;
    s.blocks->opt = *opt;
    s.blocks->graphs.clear();
  }
  return ok();
}

petra_status petra_net_sync_weights(petra_net* net, void* stream) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  if (!net->impl->bound()) return fail(PETRA_ERR_STATE, "net buffers not bound");
  petra_status r;
  if ((r = check_hip("before petra_net_sync_weights"))) return r;
  net->impl->sync_weights(static_cast<hipStream_t>(stream));
  return net_status(*net->impl, "petra_net_sync_weights");
}

petra_status petra_net_tick(petra_net* net, const void* images, const int32_t* labels,
                            float* loss, void* stream, int32_t* loss_written) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  petra::Net& s = *net->impl;
  if (!s.bound()) return fail(PETRA_ERR_STATE, "net buffers not bound");
  if ((images == nullptr) != (labels == nullptr))
    return fail(PETRA_ERR_INVALID_ARG, "images and labels must both be given or both be NULL");
  if (images != nullptr && !s.feeding)
    return fail(PETRA_ERR_STATE, "feeding cannot resume after a tick without input");
  if (images != nullptr && (!aligned16(images) || !aligned16(labels)))
    return fail(PETRA_ERR_ALIGN, "images and labels must be 16-byte aligned");
  if (images != nullptr && s.fed != s.t)
    return fail(PETRA_ERR_STATE, "micro-batch m must enter at tick m");
  petra_status r;
  if ((r = check_hip("before petra_net_tick"))) return r;
  const hipError_t e = s.ensure_streams();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("stream setup: ") + hipGetErrorString(e));
  if (images == nullptr) s.feeding = false;
  const bool wrote = s.tick(images, labels, loss, static_cast<hipStream_t>(stream));
  if (loss_written) *loss_written = wrote ? 1 : 0;
  return net_status(s, "petra_net_tick");
}

namespace {

int64_t net_in_flight(const petra::Net& s) {
  // micro-batch m finishes its last backward (stage 0) at tick m + 2J - 2
  int64_t done = s.t - (2 * static_cast<int64_t>(s.J) - 2);
  if (done < 0) done = 0;
  if (done > s.fed) done = s.fed;
  return s.fed - done;
}

}  // namespace

petra_status petra_net_drain(petra_net* net, float* losses, void* stream, int32_t* n_losses,
                             int32_t* ticks_run) {
  if (n_losses) *n_losses = 0;
  if (ticks_run) *ticks_run = 0;
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  petra::Net& s = *net->impl;
  if (!s.bound()) return fail(PETRA_ERR_STATE, "net buffers not bound");
  if (losses != nullptr && !aligned16(losses)) return fail(PETRA_ERR_ALIGN, "losses must be 16-byte aligned");
  petra_status r;
  if ((r = check_hip("before petra_net_drain"))) return r;
  const hipError_t e = s.ensure_streams();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("stream setup: ") + hipGetErrorString(e));
  s.feeding = false;
  int32_t nl = 0, nt = 0;
  // micro-batch m leaves stage 0 at tick m + 2J - 2, so at most 2J - 2 ticks remain;
  // at most J - 1 of the micro-batches in flight still have to reach the head
  while (net_in_flight(s) > 0) {
    float* slot = losses != nullptr && nl < s.J ? losses + nl : nullptr;
    if (s.tick(nullptr, nullptr, slot, static_cast<hipStream_t>(stream)) && slot != nullptr) ++nl;
    ++nt;
    if ((r = net_status(s, "petra_net_drain"))) break;
  }
  if (n_losses) *n_losses = nl;
  if (ticks_run) *ticks_run = nt;
  return r;
}

petra_status petra_net_state(const petra_net* net, int64_t* ticks, int64_t* fed,
                             int64_t* in_flight) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  const petra::Net& s = *net->impl;
  if (ticks) *ticks = s.t;
  if (fed) *fed = s.fed;
  if (in_flight) *in_flight = net_in_flight(s);
  return ok();
}

petra_status petra_net_set_backward(petra_net* net, int32_t mode) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  if (mode < 0 || mode > 3) return fail(PETRA_ERR_INVALID_ARG, "mode must be a petra_bwd_mode");
  const petra_net_desc& d = net->impl->desc;
  if (((mode & PETRA_BWD_INPUT_BUFFER) && !d.input_buffer) ||
      ((mode & PETRA_BWD_PARAM_BUFFER) && !d.param_buffer))
    return fail(PETRA_ERR_STATE, "the variant needs a buffer the net does not keep");
  net->impl->bwd_mode = mode;
  return ok();
}

petra_status petra_net_stage_params(const petra_net* net, int32_t stage, int64_t* offset,
                                    int64_t* numel) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  const petra::Net& n = *net->impl;
  if (stage < 0 || stage >= n.J) return fail(PETRA_ERR_INVALID_ARG, "stage out of range");
  if (offset) *offset = n.st[stage].off_front_w;
  if (numel) *numel = n.st[stage].n_span;
  return ok();
}

petra_status petra_net_memory(const petra_net* net, int32_t stage, petra_net_mem* out) {
  if (net == nullptr || net->impl == nullptr || out == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "null argument");
  const petra::Net& n = *net->impl;
  if (stage < 0 || stage >= n.J) return fail(PETRA_ERR_INVALID_ARG, "stage out of range");
  const int64_t* m = n.st[stage].mem;
  out->params = m[petra::MEM_PARAMS];
  out->weight_copies = m[petra::MEM_WEIGHT_COPIES];
  out->activation_buffer = m[petra::MEM_ACTIVATION_BUFFER];
  out->input_buffer = m[petra::MEM_INPUT_BUFFER];
  out->param_buffer = m[petra::MEM_PARAM_BUFFER];
  out->scratch = m[petra::MEM_SCRATCH];
  out->total = 0;
  for (int c = 0; c < petra::MEM_COUNT; ++c) out->total += m[c];
  return ok();
}

petra_status petra_net_probe_tick(petra_net* net, int32_t mode, float* grad_out, void* stream) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  petra::Net& s = *net->impl;
  if (!s.bound()) return fail(PETRA_ERR_STATE, "net buffers not bound");
  if (mode < 0 || mode > 3) return fail(PETRA_ERR_INVALID_ARG, "mode must be a petra_bwd_mode");
  if (((mode & PETRA_BWD_INPUT_BUFFER) && !s.desc.input_buffer) ||
      ((mode & PETRA_BWD_PARAM_BUFFER) && !s.desc.param_buffer))
    return fail(PETRA_ERR_STATE, "the variant needs a buffer the net does not keep");
  if (grad_out == nullptr) return fail(PETRA_ERR_INVALID_ARG, "grad_out is required");
  if (!aligned16(grad_out)) return fail(PETRA_ERR_ALIGN, "grad_out must be 16-byte aligned");
  petra_status r;
  if ((r = check_hip("before petra_net_probe_tick"))) return r;
  const hipError_t e = s.ensure_streams();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("stream setup: ") + hipGetErrorString(e));
  s.probe_tick(mode, grad_out, static_cast<hipStream_t>(stream));
  return net_status(s, "petra_net_probe_tick");
}

petra_status petra_net_probe_backprop(petra_net* net, const void* images, const int32_t* labels,
                                      float* grad_out, void* stream) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  petra::Net& s = *net->impl;
  if (!s.bound()) return fail(PETRA_ERR_STATE, "net buffers not bound");
  if (images == nullptr || labels == nullptr || grad_out == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "images, labels and grad_out are required");
  if (!aligned16(images) || !aligned16(labels) || !aligned16(grad_out))
    return fail(PETRA_ERR_ALIGN, "images, labels and grad_out must be 16-byte aligned");
  petra_status r;
  if ((r = check_hip("before petra_net_probe_backprop"))) return r;
  const hipError_t e = s.ensure_streams();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("stream setup: ") + hipGetErrorString(e));
  s.probe_backprop(images, labels, grad_out, static_cast<hipStream_t>(stream));
  return net_status(s, "petra_net_probe_backprop");
}

petra_status petra_net_backprop_step(petra_net* net, const void* images, const int32_t* labels,
                                     float* loss, void* stream) {
  if (net == nullptr || net->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null net handle");
  petra::Net& s = *net->impl;
  if (!s.bound()) return fail(PETRA_ERR_STATE, "net buffers not bound");
  if (images == nullptr || labels == nullptr)
    return fail(PETRA_ERR_INVALID_ARG, "images and labels are required");
  if (!aligned16(images) || !aligned16(labels) || (loss != nullptr && !aligned16(loss)))
    return fail(PETRA_ERR_ALIGN, "images, labels and loss must be 16-byte aligned");
  if (net_in_flight(s) != 0)
    return fail(PETRA_ERR_STATE, "micro-batches of the tick schedule are still in flight");
  petra_status r;
  if ((r = check_hip("before petra_net_backprop_step"))) return r;
  const hipError_t e = s.ensure_streams();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("stream setup: ") + hipGetErrorString(e));
  s.backprop_step(images, labels, loss, static_cast<hipStream_t>(stream));
  return net_status(s, "petra_net_backprop_step");
}

petra_status petra_stage_profile(petra_stage* st, int32_t enable) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  petra::Profiler& p = st->impl->prof;
  const hipError_t e = p.collect();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("profile: ") + hipGetErrorString(e));
  p.reset();
  p.enabled = enable != 0;
  return ok();
}

petra_status petra_stage_profile_read(petra_stage* st, int32_t kernel_class, const char** name,
                                      int64_t* launches, double* total_ms, double* flops,
                                      double* bytes) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  if (kernel_class < 0 || kernel_class >= petra::K_NUM_CLASSES)
    return fail(PETRA_ERR_INVALID_ARG, "kernel class out of range");
  petra::Profiler& p = st->impl->prof;
  const hipError_t e = p.collect();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("profile: ") + hipGetErrorString(e));
  if (name) *name = petra::kernel_class_name(kernel_class);
  if (launches) *launches = p.launches[kernel_class];
  if (total_ms) *total_ms = p.ms[kernel_class];
  if (flops) *flops = p.flops[kernel_class];
  if (bytes) *bytes = p.bytes[kernel_class];
  return ok();
}

petra_status petra_stage_profile_kernel(petra_stage* st, int32_t index, const char** name,
                                        int32_t* kernel_class, int64_t* launches,
                                        double* total_ms, double* flops, double* bytes) {
  if (st == nullptr || st->impl == nullptr) return fail(PETRA_ERR_INVALID_ARG, "null stage handle");
  petra::Profiler& p = st->impl->prof;
  const hipError_t e = p.collect();
  if (e != hipSuccess) return fail(PETRA_ERR_HIP, std::string("profile: ") + hipGetErrorString(e));
  if (index < 0 || index >= static_cast<int32_t>(p.kernels.size()))
    return fail(PETRA_ERR_INVALID_ARG, "kernel index out of range");
  const petra::KernelStat& k = p.kernels[index];
  if (name) *name = k.name.c_str();
  if (kernel_class) *kernel_class = k.kind;
  if (launches) *launches = k.launches;
  if (total_ms) *total_ms = k.ms;
  if (flops) *flops = k.flops;
  if (bytes) *bytes = k.bytes;
  return ok();
}

}  // extern "C"
