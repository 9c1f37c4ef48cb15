// One-GPU PETRA schedule over a network split into J stages (host side).
//
// Stage j = a non-reversible front layer (stage 0: 3x3 conv on the images,
// BN, ReLU; stage j > 0: 1x1 stride-2 conv on the previous stage's output, BN)
// followed by reversible blocks (a Stage); the last stage ends with the
// softmax cross-entropy head.  At tick t stage j runs the forward of micro-batch
// t - j and the backward of micro-batch t - (2J - 2 - j), both with its current
// parameters, then its update; all stages of a tick run concurrently on their
// own streams and the tick ends with a join on the caller's stream.
#pragma once

#include <memory>
#include <string>
#include <vector>

#include "../../include/petra.h"
#include "stage.h"

namespace petra {

struct NetStage {
  int j = 0;
  bool first = false, last = false;
  int H = 0, W = 0, C = 0;          // block resolution and full width
  int Hin = 0, Win = 0, Cin = 0;    // front input (Cin padded to 8 for the images)
  int cin_real = 0;                 // front input channels in the master weight
  int R = 1, stride = 1, pad = 0;   // front conv geometry
  long M = 0, Min = 0;              // rows of the block activations / front input
  std::unique_ptr<Stage> blocks;
  // flat parameter layout (elements)
  int64_t off_front_w = 0, n_front_w = 0, off_fc_w = 0, n_fc_w = 0;
  int64_t off_blocks = 0, off_front_g = 0, off_front_b = 0, off_fc_b = 0;
  int64_t off_decay = 0, n_decay = 0, off_plain = 0, n_plain = 0;
  int64_t run_front = 0, run_blocks = 0;
  // workspace plan (byte offsets) and bound pointers
  int ring_depth = 0;
  size_t o_blocks_ws = 0, o_ring = 0, o_wfwd = 0, o_wdg = 0;
  size_t o_fh = 0, o_fx1 = 0, o_fx2 = 0, o_fpart = 0, o_fbnp = 0;          // forward front
  size_t o_bh = 0, o_bpart = 0, o_bbnp = 0, o_dh = 0, o_wpart = 0, o_dtmp = 0;  // backward front
  size_t o_xr1 = 0, o_xr2 = 0, o_dx1 = 0, o_dx2 = 0;                      // block backward outputs
  size_t o_msg[2][2] = {{0, 0}, {0, 0}};   // gradient message to stage j-1 [parity][half]
  size_t o_y1 = 0, o_y2 = 0, o_g1 = 0, o_g2 = 0;                          // last stage
  size_t o_pooled = 0, o_dlogits = 0, o_lossn = 0, o_labels = 0;
  size_t ring_slot_bytes = 0;
  int wsplits = 0, wrows = 0;
  hipStream_t sf = nullptr, sb = nullptr;
  hipEvent_t ev_f = nullptr, ev_b = nullptr;
};

class Net {
 public:
  explicit Net(const petra_net_desc& d);
  ~Net();

  petra_net_desc desc;
  int dt;
  size_t esz;
  int J;
  std::vector<NetStage> st;
  std::vector<petra_param_info> infos;
  int64_t n_params = 0, n_bnch = 0;
  size_t ws_need = 0;
  WeightSegTable front_segs{};
  int64_t front_max_numel = 0;
  size_t o_front_wfwd = 0, o_front_wdg = 0;

  float* theta = nullptr;
  float* grad = nullptr;
  float* mom = nullptr;
  float* rmean = nullptr;
  float* rvar = nullptr;
  char* ws = nullptr;
  petra_sgd opt{0.1f, 0.9f, 0.0f, 1, 1};

  int64_t t = 0;       // ticks run
  int64_t fed = 0;     // micro-batches fed
  bool feeding = true;
  hipEvent_t ev_tick = nullptr;

  bool bound() const { return theta != nullptr; }
  void bind(float* th, float* gr, float* mo, float* rm, float* rv, void* w);
  hipError_t ensure_streams();
  void sync_weights(hipStream_t s);
  // One tick; returns whether a loss was written.
  bool tick(const void* images, const int32_t* labels, float* loss, hipStream_t caller);
  // One micro-batch through plain reversible backpropagation on stream q: the
  // forward of every stage in order, the head, then every stage's backward from
  // the last to the first (each followed by its update when due).  Front
  // layers keep their forward output instead of recomputing it.  Uses ring
  // slot 0 and message parity 0: no micro-batch of the tick schedule may be in
  // flight.
  void backprop_step(const void* images, const int32_t* labels, float* loss, hipStream_t q);

 private:
  template <typename P> P* at(size_t off) const { return reinterpret_cast<P*>(ws + off); }
  void* ring_slot(const NetStage& s, int64_t m, int half) const;
  void front_forward(NetStage& s, const void* in1, const void* in2, hipStream_t q,
                     bool keep = false);
  void front_backward(NetStage& s, const void* in1, const void* in2, const void* d1,
                      const void* d2, int parity, hipStream_t q, bool recompute = true);
  void head(NetStage& s, const void* y1, const void* y2, const int32_t* labels, float* loss,
            hipStream_t q);
  void stage_update(NetStage& s, hipStream_t q);
};

}  // namespace petra
