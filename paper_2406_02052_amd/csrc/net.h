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

// Device bytes of a stage by purpose (memory accounting of Tables 3 and 6).
enum { MEM_PARAMS = 0, MEM_WEIGHT_COPIES, MEM_ACTIVATION_BUFFER, MEM_INPUT_BUFFER,
       MEM_PARAM_BUFFER, MEM_SCRATCH, MEM_COUNT };

struct NetStage {
  int j = 0;
  int level = 0;                    // network level (width index) the stage belongs to
  bool first = false, last = false;
  bool has_front = true;            // opens with the stem / a downsampling layer
  bool has_blocks = true;           // holds reversible blocks
  int fseg = -1;                    // its front weight in front_segs
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
  int64_t n_span = 0;               // the stage's parameters: [off_front_w, off_front_w + n_span)
  // workspace plan (byte offsets) and bound pointers
  int ring_depth = 0;
  size_t o_blocks_ws = 0, o_ring = 0, o_wfwd = 0, o_wdg = 0;
  size_t o_fh = 0, o_fx1 = 0, o_fx2 = 0, o_fpart = 0, o_fbnp = 0;          // forward front
  size_t o_bh = 0, o_bpart = 0, o_bbnp = 0, o_dh = 0, o_wpart = 0, o_dtmp = 0;  // backward front
  size_t o_xr1 = 0, o_xr2 = 0, o_dx1 = 0, o_dx2 = 0;                      // block backward outputs
  size_t o_msg[2][2] = {{0, 0}, {0, 0}};   // gradient message to stage j-1 [parity][half]
  size_t o_y1 = 0, o_y2 = 0, o_g1 = 0, o_g2 = 0;                          // last stage
  // stage without front: forward input by micro-batch parity, the input it
  // reconstructs for stage j - 1 by tick parity, and the backprop pass's input
  size_t o_fin[2][2] = {{0, 0}, {0, 0}};
  size_t o_xmsg[2][2] = {{0, 0}, {0, 0}};
  size_t o_bpin = 0;
  size_t o_pooled = 0, o_dlogits = 0, o_lossn = 0, o_labels = 0;
  size_t ring_slot_bytes = 0;
  // buffer variants (Table 4): per micro-batch in flight, the blocks' input
  // (input buffer) and the parameters of the forward (parameter buffer: fp32
  // span, then the blocks' and the front's compute copies); rx/ry hold the
  // reconstructed input and the recomputed output of the variant backward
  int buf_depth = 0;
  size_t o_ib = 0, ib_slot_bytes = 0;
  size_t o_ps = 0, ps_slot_bytes = 0, ps_bwf = 0, ps_bwd = 0, ps_fwf = 0, ps_fwd = 0;
  size_t o_rx1 = 0, o_rx2 = 0, o_ry1 = 0, o_ry2 = 0;
  int wsplits = 0, wrows = 0;
  hipStream_t sf = nullptr, sb = nullptr;
  hipEvent_t ev_f = nullptr, ev_b = nullptr;
  int64_t mem[MEM_COUNT] = {0, 0, 0, 0, 0, 0};
  int64_t bwd_count = 0;            // backward passes (stages without blocks)
};

// Parameters a front layer's backward reads: the live ones or a stashed copy.
struct FrontView {
  const void* wf;      // forward compute copy [C][R][R][Cin]
  const void* wd;      // transposed compute copy
  const float* gamma;
  const float* beta;
};

class Net {
 public:
  explicit Net(const petra_net_desc& d);
  ~Net();

  petra_net_desc desc;
  int dt;
  size_t esz;
  int J;            // stages (levels, or levels x (1 + blocks) with split_stages)
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

  // Backward variant of the ticks: bit 0 stored block inputs, bit 1 stashed
  // parameters (each needs its buffer kept, desc.input_buffer/param_buffer).
  int bwd_mode = 0;
  size_t o_probe_run = 0;   // running-statistics sink of the probes [2][n_bnch]

  int64_t t = 0;       // ticks run
  int64_t fed = 0;     // micro-batches fed
  bool feeding = true;
  HipStatus hip_status;  // first failed runtime call of the current enqueue
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
  // Gradient probes (App. B), no state change: the unscaled parameter
  // gradients that the backward passes of the next tick would produce in
  // variant `mode`, or the end-to-end gradient of one micro-batch at the
  // current parameters; both into gout [n_params] (zeroed first).
  void probe_tick(int mode, float* gout, hipStream_t q);
  void probe_backprop(const void* images, const int32_t* labels, float* gout, hipStream_t q);

 private:
  template <typename P> P* at(size_t off) const { return reinterpret_cast<P*>(ws + off); }
  // Slot m of the stage's input ring; m < 0: the extra slot of the backprop pass.
  void* ring_slot(const NetStage& s, int64_t m, int half) const;
  void* ib_slot(const NetStage& s, int64_t m, int half) const;
  char* ps_slot(const NetStage& s, int64_t m) const;
  FrontView front_view(const NetStage& s) const;
  FrontView stash_front_view(const NetStage& s, int64_t m) const;
  void stash_params(NetStage& s, int64_t m, hipStream_t q);
  // The stage's forward input for micro-batch m (m < 0: the backprop pass),
  // where its output goes, and the output / output gradient its backward gets.
  void* fwd_in(const NetStage& s, int64_t m, int half) const;
  void* fwd_dest(const NetStage& s, int64_t m, int half) const;
  const void* bwd_y(const NetStage& s, int64_t m, int parity, int half) const;
  const void* bwd_g(const NetStage& s, int parity, int half) const;
  // Forward of one stage (front, blocks); buffers: keep the variant buffers.
  void stage_forward(NetStage& s, int64_t m, hipStream_t q, bool keep, bool buffers);
  void front_forward(NetStage& s, const void* in1, const void* in2, hipStream_t q,
                     bool keep = false, void* out1 = nullptr, void* out2 = nullptr);
  void front_backward(NetStage& s, const void* in1, const void* in2, const void* d1,
                      const void* d2, int parity, hipStream_t q, bool recompute = true,
                      const FrontView* fv = nullptr);
  // Blocks + front backward of micro-batch mb given the block output (by) and
  // its gradient (bg), in variant `mode`; the message goes to parity `parity`.
  void backward_stage(NetStage& s, int64_t mb, int mode, int parity, hipStream_t q,
                      const void* by1, const void* by2, const void* bg1, const void* bg2,
                      hipStream_t side = nullptr, bool recompute = true);
  void backprop_pass(const void* images, const int32_t* labels, float* loss, bool update,
                     hipStream_t q);
  // count one backward of the stage; does its update fire now?
  bool count_and_due(NetStage& s);
  struct Redirect;
  void head(NetStage& s, const void* y1, const void* y2, const int32_t* labels, float* loss,
            hipStream_t q);
  void stage_update(NetStage& s, hipStream_t q);
};

}  // namespace petra
