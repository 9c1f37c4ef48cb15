// Host-side program of one reversible stage: layer tables, workspace plan and
// the kernel sequences of the forward, the reconstruct+VJP backward and the
// update (internal to the library; the C ABI wraps it).
#pragma once

#include <string>
#include <vector>

#include "../../include/petra.h"
#include "kernels.h"
#include "graph.h"
#include "prof.h"

namespace petra {

struct ConvLayer {
  int cin, cout, r, s, pad;
  int64_t w_off;   // offset of the KRSC weight in the flat buffers and the forward copy
  int64_t dg_off;  // offset in the transposed/flipped copy
  int bn;          // BN layer that follows
};

struct BnLayer {
  int c;
  int64_t g_off, b_off;  // gamma / beta offsets in the flat buffers
  int64_t run_off;       // offset into the running-statistics arrays
};

struct ResidualFn {
  int nconv;
  int conv[3];
};

struct Block {
  ResidualFn f, g;
};

// Device scratch of one residual function's pass, carved from the workspace.
// The forward uses one set; the backward alternates two sets between
// consecutive residual functions, so the recompute of the next function can run
// while the gradient chain of the current one still reads its own set.
struct Scratch {
  void* h[3] = {nullptr, nullptr, nullptr};  // pre-BN conv outputs of the function
  void* d1[2] = {nullptr, nullptr};          // masked gradients dz of inner layers (backward)
  float* part = nullptr;                     // BN statistic partials of the recompute [tiles][3][c]
  float* gpart = nullptr;                    // BN-backward partials of the last BN [tiles][2][c]
  float* bpart = nullptr;                    // BN-backward partials of an inner BN [tiles][2][c]
  float* bnp = nullptr;                      // per layer: scale, shift, mean, rstd, ca, cb, cc
  int gtiles = 0;                            // tile count of gpart (host side, set at enqueue)
  float* vec(int layer, int which, int cmax) const { return bnp + (layer * 8 + which) * cmax; }
};

enum { V_SCALE = 0, V_SHIFT, V_MEAN, V_RSTD, V_CA, V_CB, V_CC };

class Stage {
 public:
  explicit Stage(const petra_stage_desc& d);
  ~Stage();

  petra_stage_desc desc;
  int dt;
  size_t esz;
  long M;
  int cmax;
  std::vector<ConvLayer> convs;
  std::vector<BnLayer> bns;
  std::vector<Block> blocks;
  std::vector<petra_param_info> infos;
  int64_t n_params = 0, n_conv = 0, n_bnch = 0, max_wnumel = 0;
  WeightSegTable segs{};

  // Workspace plan (byte offsets).
  size_t ws_need = 0;
  size_t fwd_need = 0;   // leading workspace bytes the forward uses (copies + scratch set)
  size_t off_wfwd = 0, off_wdg = 0;
  struct ScratchPlan {
    size_t h[3], d1[2], part, gpart, bpart, bnp;
  };
  static constexpr size_t NO_BUF = ~static_cast<size_t>(0);   // a buffer the set does not hold
  // Residual functions whose last conv is the bf16 1x1 32 -> 128: every
  // coupling (forward add and reconstruction) recomputes that conv's output
  // from the layer's input; in the forward the conv writes its BN statistics
  // only (the forward set holds no buffer for it).
  bool couple_fwd = false;
  // ... and the coupling also runs the next function's first conv (1x1 128 -> 32)
  bool couple_next = false;
  ScratchPlan plan_f{};
  std::vector<ScratchPlan> plan_b;   // 2 sets, or one per residual function (defer_wgrad)
  // Weight gradients wait until the end of a single-stream backward and run as
  // one launch per kernel configuration (the first function's only when the
  // call is not in place); their inputs then stay alive: one scratch set per
  // function, and the reconstructed inputs and input gradients of blocks 1.. in
  // their own buffers (4 half-width tensors per block).
  bool defer_wgrad = false;
  size_t off_inter = 0;
  size_t off_wpart = 0;
  int64_t wpart_floats = 0;

  // Bound buffers.
  float* theta = nullptr;
  float* grad = nullptr;
  float* mom = nullptr;
  float* rmean = nullptr;
  float* rvar = nullptr;
  char* ws = nullptr;
  void* wfwd = nullptr;
  void* wdg = nullptr;
  const float* v_th = nullptr;   // active parameter view (see set_view)
  const void* v_wf = nullptr;
  const void* v_wd = nullptr;
  Scratch sf;
  std::vector<Scratch> sb;
  float* wpart = nullptr;  // weight-gradient split partials, one region per conv layer
  std::vector<int64_t> wpart_off;       // float offset of each conv layer's region
  std::vector<TrSeg> pending_reduce;    // reduces deferred to the end of the backward
  std::vector<WgradArgs> pending_wgrad; // weight gradients deferred to the end of the backward
  bool defer_cur = false;               // the function being enqueued defers its weight gradients
  // launch the deferred weight gradients and reduces collected so far on q
  void flush_deferred(hipStream_t q);

  petra_sgd opt{0.1f, 0.9f, 0.0f, 1, 1};
  int64_t bwd_count = 0, last_update = 0;

  Profiler prof;
  bool launch_error = false;  // a conv variant was requested that no kernel implements
  HipStatus hip_status;       // first failed runtime call of the current enqueue

  hipStream_t s_fwd = nullptr, s_bwd = nullptr;
  // Backward streams: the recompute of residual functions runs ahead on s_rec,
  // the weight gradients on s_wg, the input-gradient chain on the caller's stream.
  hipStream_t s_rec = nullptr, s_wg = nullptr;
  hipEvent_t ev_fork = nullptr, ev_fwd = nullptr, ev_bwd = nullptr;
  hipEvent_t ev_start = nullptr, ev_d = nullptr, ev_rec_end = nullptr, ev_side = nullptr;
  hipEvent_t ev_rec[2] = {nullptr, nullptr};     // recompute of set p done (h, BN statistics)
  hipEvent_t ev_gdone[2] = {nullptr, nullptr};   // input-gradient chain done with set p
  hipEvent_t ev_wgdone[2] = {nullptr, nullptr};  // weight gradients done with set p

  bool bound() const { return theta != nullptr; }
  bool has_workspace() const { return ws != nullptr; }
  void bind(float* th, float* gr, float* mo, float* rm, float* rv, void* w);
  void sync_weights(hipStream_t st);
  // Kernel sequences (enqueue only; no host-side bookkeeping).
  void forward(const void* x1, const void* x2, void* y1, void* y2, hipStream_t st);
  // The forward with its compute copies and scratch set laid out at `base` as in
  // the first fwd_need bytes of the workspace (the copies refreshed first).
  void forward_on(char* base, const void* x1, const void* x2, void* y1, void* y2,
                  hipStream_t st);
  // The forward on a given scratch set (the backward's sb[0] for a recompute that
  // runs on the backward's stream while another forward may be in flight).
  void forward_with(const void* x1, const void* x2, void* y1, void* y2, Scratch& s,
                    hipStream_t st);
  // Reconstruction only (x = inverse of the blocks at y), on scratch sb[0].
  void reconstruct(const void* y1, const void* y2, void* x1, void* x2, hipStream_t st);
  // Parameters the forward, backward and reconstruction read: the bound master
  // (BN) parameters and compute copies unless a view of another version of the
  // same layout is set (a stashed copy); the update always writes the bound ones.
  void set_view(const float* th, const void* wf, const void* wd) { v_th = th; v_wf = wf; v_wd = wd; }
  void reset_view() { v_th = theta; v_wf = wfwd; v_wd = wdg; }
  // side (optional, single-stream deferred mode only): a stream that is idle
  // during the second half of the backward; the weight gradients collected by
  // the middle and by the last function run there (one event each), and the
  // caller joins it before the update.
  void backward(const void* y1, const void* y2, const void* dy1, const void* dy2, void* x1,
                void* x2, void* dx1, void* dx2, hipStream_t st, hipStream_t side = nullptr);
  void update_kernels(hipStream_t st);
  // Host-side accumulation bookkeeping: count one backward; does the update fire now?
  void count_backward() { ++bwd_count; }
  bool update_due() const;
  void mark_updated() { last_update = bwd_count; }
  hipError_t ensure_streams();

  GraphCache graphs;
  bool use_graphs = false;
  // 1: one stream; 2: + weight gradients; 3: + recompute ahead.  Set in the
  // constructor: one stream for basic blocks (each cross-stream event costs more
  // host time than the overlap gains there), three for bottleneck blocks (their
  // HBM-bound 1x1 convs overlap well).
  int bwd_streams = 1;

 private:
  // One residual function of the backward, in the order the backward visits them.
  struct BwdFn {
    const ResidualFn* fn;
    const void* u;     // function input (recomputed from)
    const void* v;     // output-side stream: the reconstruction is v - Phi(u)
    const void* d;     // gradient of the coupling output
    const void* rg;    // residual gradient added to the input gradient
    void* xrec;        // reconstructed stream
    void* dout;        // input gradient: rg + dPhi/du^T d
  };
  Scratch carve(const ScratchPlan& p, char* base, bool bwd) const;
  // stats_only_last: the last conv writes its BN partials only (the forward's
  // coupling recomputes its output; see couple_fwd)
  // first_done: the first conv already ran (its output in s.h[0], its BN
  // partials in s.part, written by the previous function's coupling); only its
  // finalize is enqueued.
  void fn_recompute(const ResidualFn& fn, const void* u, Scratch& s, bool running,
                    hipStream_t st, bool stats_only_last = false, bool first_done = false);
  // Forward of one residual function (y = r + fn(u)).  With next set and
  // couple_next, the coupling also runs next's first conv on y; returns
  // whether it did (then next's forward passes first_done).
  bool fn_forward(const ResidualFn& fn, const void* u, const void* r, void* y, Scratch& s,
                  hipStream_t st, bool first_done = false, const ResidualFn* next = nullptr);
  void fn_grad(const BwdFn& f, Scratch& s, const BwdFn* next, Scratch* sn, hipStream_t st,
               hipStream_t wst, hipStream_t rs, bool wait_prev_wg, int parity, int part,
               const void** dsrc_io);
  // Coupling output of a residual function whose convs s holds (recomputed):
  // out = r + BN_L(h_L), or r - BN_L(h_L) with sub (the reconstruction); with
  // couple_fwd h_L is recomputed from h_{L-1}, else read from s.h[L].
  // With next / ns (and couple_next), the same launch also runs next's first
  // conv on out, into ns->h[0] and ns->part (then next's recompute passes
  // first_done); returns whether it did.
  bool coupling(const ResidualFn& fn, Scratch& s, const void* r, void* out, bool sub,
                hipStream_t st, const ResidualFn* next = nullptr, Scratch* ns = nullptr);
  bool conv(const ConvArgs& a, int ep, hipStream_t st);
  ConvArgs conv_args(const ConvLayer& cv) const;
  void wgrad_splits(const ConvLayer& cv, int* splits, int* rows_per_split) const;
};

}  // namespace petra
