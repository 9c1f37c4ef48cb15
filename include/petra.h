/*
 * petra.h -- C ABI of the MI355X (gfx950) PETRA reversible-stage library.
 *
 * PETRA trains a network split into stages; each stage keeps one copy of its
 * parameters and, per time step, runs the forward of one micro-batch and the
 * backward of another with the same current parameters, then updates them in
 * place (paper: Sec. 3.3, Eq. 5 and Alg. 1).  For a reversible stage the
 * backward first rebuilds the stage input from its output (Sec. 3.2, Eq. 4),
 * so no activation is kept between the two passes.
 *
 * Conventions shared by every call below
 *  - All tensors are device pointers into memory the caller owns.  The library
 *    owns only the host-side handle and the HIP streams/events it creates for
 *    itself; no call allocates or frees device memory.
 *  - Activations are NHWC.  A stage activation with C channels is passed as two
 *    contiguous half-tensors x1 (channels [0, C/2)) and x2 (channels [C/2, C)),
 *    each [N][H][W][C/2], of the stage's storage type (fp32 or bf16).
 *  - Parameters live in flat fp32 buffers whose layout the library defines and
 *    reports through petra_stage_param_info(): conv weights are KRSC
 *    ([C_out][R][S][C_in]).  Gradient accumulator and momentum buffers use the
 *    same layout.  BN running statistics are two fp32 arrays (mean, variance)
 *    of petra_stage_query()'s n_bn_channels entries.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Compute calls only
 *    enqueue work and return; buffers must stay alive until the stream has
 *    drained them.
 *  - Argument, shape, alignment and state errors are detected on the host
 *    before anything is enqueued and return a non-zero status; nothing is
 *    launched in that case.  An asynchronous HIP error is reported as
 *    PETRA_ERR_HIP by the call that observes it.  petra_last_error() gives
 *    a readable message for the calling thread.  The library never aborts.
 *  - Device pointers must be 16-byte aligned.  A handle must not be used by
 *    two host threads at once.
 */
#ifndef PETRA_H
#define PETRA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PETRA_OK = 0,
  PETRA_ERR_INVALID_ARG = 1, /* null pointer, bad enum, bad hyper-parameter   */
  PETRA_ERR_SHAPE = 2,       /* unsupported or inconsistent sizes             */
  PETRA_ERR_DTYPE = 3,       /* unsupported storage type                      */
  PETRA_ERR_ALIGN = 4,       /* a device pointer is not 16-byte aligned       */
  PETRA_ERR_WORKSPACE = 5,   /* workspace missing or too small                */
  PETRA_ERR_STATE = 6,       /* call out of order (e.g. compute before bind)  */
  PETRA_ERR_HIP = 7,         /* a HIP runtime call failed                     */
  PETRA_ERR_ALIAS = 8        /* two buffers overlap where that is not allowed */
} petra_status;

typedef enum { PETRA_FP32 = 0, PETRA_BF16 = 1 } petra_dtype; /* storage; accumulation is fp32 */

typedef enum {
  PETRA_BLOCK_BASIC = 0,      /* conv3x3-BN-ReLU-conv3x3-BN                        */
  PETRA_BLOCK_BOTTLENECK = 1  /* conv1x1-BN-ReLU-conv3x3-BN-ReLU-conv1x1-BN         */
} petra_block_kind;

typedef enum {
  PETRA_ROLE_CONV_WEIGHT = 0,
  PETRA_ROLE_BN_GAMMA = 1,
  PETRA_ROLE_BN_BETA = 2,
  PETRA_ROLE_FC_WEIGHT = 3,
  PETRA_ROLE_FC_BIAS = 4
} petra_param_role;

/* One reversible stage: num_blocks reversible blocks y1 = x1 + F(x2),
 * y2 = x2 + G(y1) (Sec. 3.2, Fig. 2) at a fixed activation shape.
 * Each block has two residual functions F and G of the given kind, acting on
 * one stream of c_half channels (c_mid = inner width of a bottleneck).
 * BN runs in training mode with batch statistics over N*H*W (eps bn_eps);
 * running statistics use momentum bn_momentum and move only during the
 * backward recompute (Sec. 4.1, "Model adaptations").
 * Limits: c_half and c_mid are 8 times a power of two, at most 512;
 * N*H*W*max(c_half, c_mid)*element size < 2^31 bytes (every tensor is
 * addressed with 32-bit byte offsets); PETRA_ERR_SHAPE otherwise. */
typedef struct {
  int32_t n, h, w;
  int32_t c_half;
  int32_t c_mid;
  int32_t num_blocks;
  int32_t kind;   /* petra_block_kind */
  int32_t dtype;  /* petra_dtype      */
  float bn_eps;
  float bn_momentum;
} petra_stage_desc;

/* SGD with momentum (Nesterov when nesterov != 0) and gradient accumulation
 * over accum_k backward steps with averaging (Sec. 4.1; Alg. 1).  Weight decay
 * applies to conv/FC weights only, never to BN parameters or biases. */
typedef struct {
  float lr;
  float momentum;
  float weight_decay;
  int32_t nesterov;
  int32_t accum_k;
} petra_sgd;

/* Placement of one parameter tensor in the flat fp32 buffers.  Tensors are
 * indexed in canonical order: block b, function F then G, conv l, and for
 * each conv its weight, BN gamma, BN beta. */
typedef struct {
  int64_t offset;        /* element offset into the flat buffers           */
  int64_t numel;
  int32_t role;          /* petra_param_role                                */
  int32_t ndim;
  int32_t shape[4];      /* KRSC for conv weights, [C] for BN parameters    */
  int32_t weight_decay;  /* 1 if weight decay applies                       */
  int32_t bn_index;      /* BN layer index for gamma/beta (and the conv it follows), else -1 */
} petra_param_info;

typedef struct petra_stage petra_stage;

/* Status name, e.g. "PETRA_ERR_SHAPE". */
const char* petra_status_str(petra_status s);
/* Message of the calling thread's last failed call ("" if none). */
const char* petra_last_error(void);

/* Build a handle from a description (host only, no device work). */
petra_status petra_stage_create(const petra_stage_desc* desc, petra_stage** out);
petra_status petra_stage_destroy(petra_stage* st);

/* Sizes the caller must allocate: n_params fp32 elements for each of the
 * parameter, gradient-accumulator and momentum buffers; n_tensors parameter
 * tensors; n_bn_channels fp32 elements for each running-statistics array;
 * workspace_bytes of device scratch (compute copies of the weights, one
 * block's intermediates for the forward and for the backward, partial sums). */
petra_status petra_stage_query(const petra_stage* st, int64_t* n_params, int32_t* n_tensors,
                               int64_t* n_bn_channels, size_t* workspace_bytes);
petra_status petra_stage_param_info(const petra_stage* st, int32_t index, petra_param_info* out);

/* Attach caller-owned device buffers.  params: fp32 master weights theta;
 * grad_accum: the accumulator Delta; momentum: optimizer state; run_mean /
 * run_var: BN running statistics; workspace: scratch of at least
 * workspace_bytes.  The caller initialises params, zeroes grad_accum and
 * momentum, and sets run_mean = 0, run_var = 1; then calls
 * petra_stage_sync_weights().  workspace = NULL with workspace_bytes = 0 binds
 * a handle for petra_stage_forward_noalloc only. */
petra_status petra_stage_bind(petra_stage* st, float* params, float* grad_accum, float* momentum,
                              float* run_mean, float* run_var, void* workspace,
                              size_t workspace_bytes);

/* Optimizer settings used by petra_stage_update() and the (1/k) gradient
 * scale of petra_stage_reconstruct_backward(). */
petra_status petra_stage_set_optimizer(petra_stage* st, const petra_sgd* opt);

/* Graph replay (default off): each distinct call (kind of call and the device
 * pointers passed) is captured once into a HIP graph and replayed on a private
 * stream ordered with events after prior work on the caller's stream and
 * before later work on it; set_optimizer() drops the cached graphs.
 * enable = 0 launches every kernel directly (on the caller's stream and the
 * stage's side streams). */
petra_status petra_stage_set_graphs(petra_stage* st, int32_t enable);

/* Streams used by one backward call: 1 = every kernel on one stream; 2 = the
 * weight gradients on a second stream; 3 = in addition the recompute of the
 * next residual function on a third stream, overlapped with the input-gradient
 * chain of the current one.  Default: 1 for every block kind (with one stream
 * the weight gradients wait for the end of the backward and run grouped, which
 * fills the chip better than per-layer launches beside the chain).  Results
 * are identical in every mode.
 * PETRA_ERR_INVALID_ARG outside [1, 3]. */
petra_status petra_stage_set_streams(petra_stage* st, int32_t n);

/* Refresh the storage-type compute copies of the conv weights from the fp32
 * master (needed once after the caller writes params directly). */
petra_status petra_stage_sync_weights(petra_stage* st, void* stream);

/* Forward of the stage with the current parameters (Eq. 5, first line):
 * blocks 1..B in order.  Reads x1, x2; writes y1, y2.  In place is allowed
 * (x1 == y1 and/or x2 == y2); no other overlap.  BN uses batch statistics and
 * leaves the running statistics untouched. */
petra_status petra_stage_forward(petra_stage* st, const void* x1, const void* x2, void* y1,
                                 void* y2, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the forward
 * of petra_stage_forward, with the same arguments, aliasing rules and result
 * bits, that needs no workspace.  Its scratch -- the compute copies of the
 * conv weights, refreshed from params on every call, and one residual
 * function's pre-BN tensors and BN partial sums -- lives in a static device
 * array of PETRA_STATIC_SCRATCH_BYTES that the library holds on each device it
 * runs on until the process ends.  The call allocates nothing and always
 * launches directly (no graph cache, no timing events).  The handle may be
 * bound with workspace = NULL and workspace_bytes = 0 (every other compute
 * call then returns PETRA_ERR_WORKSPACE).  PETRA_ERR_WORKSPACE when the stage's
 * forward needs more scratch than the array holds (about 2 bytes per conv
 * weight plus N*H*W*(sum of one residual function's conv output widths)*element
 * size).  Runs on the current device.  Every call on a device shares that
 * device's array: calls that overlap in time on one device (other streams or
 * threads) race and must be ordered by the caller. */
#define PETRA_STATIC_SCRATCH_BYTES (64u << 20)
petra_status petra_stage_forward_noalloc(petra_stage* st, const void* x1, const void* x2,
                                         void* y1, void* y2, void* stream);

/* Backward of the stage with the current parameters (Eq. 5, lines 2-4;
 * Alg. 1): blocks B..1, each rebuilding its input from its output
 * (x2 = y2 - G(y1), x1 = y1 - F(x2), Eq. 4) while recomputing the graph of G
 * and F, then taking the vector-Jacobian products through them.
 * Inputs: the stage output y1, y2 and its gradient dy1, dy2.
 * Outputs: the reconstructed input x1, x2 and the input gradient dx1, dx2.
 * Adds (1/accum_k) of the parameter gradient to grad_accum and updates the BN
 * running statistics.  In place is allowed for x1 == y1, x2 == y2,
 * dx1 == dy1, dx2 == dy2; no other overlap. */
petra_status petra_stage_reconstruct_backward(petra_stage* st, const void* y1, const void* y2,
                                              const void* dy1, const void* dy2, void* x1,
                                              void* x2, void* dx1, void* dx2, void* stream);

/* Parameter update (Eq. 5, last line; Alg. 1): when the number of backward
 * calls so far is a multiple of accum_k (and no update has run since the last
 * backward), applies the optimizer to params from grad_accum, zeroes
 * grad_accum and refreshes the compute copies.  *updated (nullable) receives
 * 1 if the update ran. */
petra_status petra_stage_update(petra_stage* st, void* stream, int32_t* updated);

/* One PETRA stage step (Eq. 5): the forward of one micro-batch (x -> y) and
 * the backward of another (yb, dyb -> xb, dxb) run concurrently on two
 * library-owned streams, both reading the current parameters; the update
 * follows both.  All work is ordered after prior work on `stream`, and later
 * work on `stream` is ordered after it.  Aliasing rules of the two calls
 * apply; the forward and backward buffers must not overlap each other. */
petra_status petra_stage_step(petra_stage* st, const void* x1, const void* x2, void* y1, void* y2,
                              const void* yb1, const void* yb2, const void* dyb1,
                              const void* dyb2, void* xb1, void* xb2, void* dxb1, void* dxb2,
                              void* stream, int32_t* updated);

/* ------------------------------------------------------------------------
 * Multi-stage schedule on one GPU (Alg. 1, Eq. 5; delays of App. B).
 *
 * The network is split into num_stages stages.  Stage 0 opens with a 3x3 conv
 * (pad 1) + BN + ReLU on the images; stage j > 0 opens with a non-reversible
 * 1x1 stride-2 conv + BN on the previous stage's output (both streams taken as
 * one tensor, x1 first); each stage then runs blocks_per_stage reversible basic
 * blocks at width widths[j] (two streams of widths[j]/2 channels); the last
 * stage ends with global average pooling, a linear layer with bias and softmax
 * cross-entropy averaged over the micro-batch (Sec. 4.1, "Model adaptations").
 *
 * petra_net_tick() runs one time step of every stage: stage j (0-based) runs
 * the forward of micro-batch t - j and the backward of micro-batch
 * t - (2 num_stages - 2 - j), both with its current parameters, and then its
 * update, so the delay between a stage's forward and backward of the same
 * micro-batch is 2(num_stages - 1 - j).  Front layers keep their input in a
 * ring of micro-batches and recompute it on the backward (Sec. 3.2,
 * "Non-reversible stages"); the reversible blocks rebuild their input from
 * their output.  All stages of a tick run concurrently on library streams; the
 * tick is ordered after prior work on `stream` and later work on `stream`
 * follows it.
 *
 * Limits: h and w divisible by 2^(num_stages-1); widths[j]/2 is 8 times a
 * power of two, at most 512; c_img <= 8; classes <= 64; num_stages <= 8;
 * every stage's activation below 2^31 bytes (as for a stage).
 * ------------------------------------------------------------------------ */
#define PETRA_MAX_STAGES 8

typedef struct {
  int32_t n, h, w, c_img;              /* micro-batch of images [n][h][w][c_img] */
  int32_t num_stages;
  int32_t widths[PETRA_MAX_STAGES];    /* full width of each stage (both streams) */
  int32_t blocks_per_stage;
  int32_t classes;
  int32_t dtype;                       /* petra_dtype */
  float bn_eps;
  float bn_momentum;
  /* Buffers kept per micro-batch in flight, for the backward variants of
   * Table 4 (petra_net_set_backward) and the gradient probes: the blocks'
   * input (input buffer) and the parameters of the forward (parameter
   * buffer, a weight stash).  0 = PETRA's setting (neither). */
  int32_t input_buffer;
  int32_t param_buffer;
  /* 0: one stage per level (front layer + its blocks).  1: the paper's
   * per-layer split (Table 6, App. B): every front layer (stem, downsampling)
   * and every reversible block is a stage of its own, the last block also
   * owning the head, so num_stages x (1 + blocks_per_stage) stages; a
   * reversible stage below another one rebuilds its input from the
   * reconstruction that stage sends back.  num_stages then counts levels. */
  int32_t split_stages;
} petra_net_desc;

typedef struct petra_net petra_net;

petra_status petra_net_create(const petra_net_desc* desc, petra_net** out);
petra_status petra_net_destroy(petra_net* net);
/* Number of stages of the schedule (num_stages, or the per-layer split's count). */
petra_status petra_net_num_stages(const petra_net* net, int32_t* stages);
/* Sizes as for a stage.  Parameter tensors in canonical order: per stage j,
 * the front conv weight (KRSC, [w_j][3][3][c_img] or [w_j][1][1][w_{j-1}]), its
 * BN gamma and beta, the reversible blocks' tensors in the stage order, and
 * for the last stage the linear weight [classes][w_last] and bias [classes]. */
petra_status petra_net_query(const petra_net* net, int64_t* n_params, int32_t* n_tensors,
                             int64_t* n_bn_channels, size_t* workspace_bytes);
petra_status petra_net_param_info(const petra_net* net, int32_t index, petra_param_info* out);
/* Caller-owned buffers as for petra_stage_bind (workspace 256-byte aligned). */
petra_status petra_net_bind(petra_net* net, float* params, float* grad_accum, float* momentum,
                            float* run_mean, float* run_var, void* workspace,
                            size_t workspace_bytes);
petra_status petra_net_set_optimizer(petra_net* net, const petra_sgd* opt);
petra_status petra_net_sync_weights(petra_net* net, void* stream);
/* One tick.  images: the next micro-batch [n][h][w][c_img] in the storage type
 * and labels: its [n] int32 class ids (device pointers), or both NULL once the
 * input has ended (then only the micro-batches in flight advance; feeding
 * cannot resume).  loss (nullable, device fp32): receives the mean loss of the
 * micro-batch that reached the head in this tick; *loss_written (nullable)
 * tells whether one did. */
petra_status petra_net_tick(petra_net* net, const void* images, const int32_t* labels,
                            float* loss, void* stream, int32_t* loss_written);
/* Drain the pipeline (Alg. 1 once the input has ended): runs ticks without
 * input until no micro-batch is in flight, so every micro-batch fed so far
 * has had its backward in every stage and its updates applied.  Feeding cannot
 * resume afterwards.  losses (nullable, device fp32, at least petra_net_num_stages()
 * entries, 16-byte aligned): entry i receives the mean loss of the i-th
 * micro-batch that reaches the head during the drain; *n_losses (nullable)
 * their count; *ticks_run (nullable) the ticks this call ran (0 if nothing
 * was in flight).  Ordered after prior work on `stream`; later work on
 * `stream` follows every tick. */
petra_status petra_net_drain(petra_net* net, float* losses, void* stream, int32_t* n_losses,
                             int32_t* ticks_run);
/* Ticks run so far, micro-batches fed, and micro-batches still in flight. */
petra_status petra_net_state(const petra_net* net, int64_t* ticks, int64_t* fed,
                             int64_t* in_flight);
/* Backward variants of the ticks (Table 4; App. B): which of the kept buffers
 * the backward of a non-last stage uses.  RECONSTRUCT is PETRA: the blocks'
 * input is rebuilt from their output with the current parameters and the VJP
 * taken there.  INPUT_BUFFER takes the VJP at the stored block input with the
 * current parameters; PARAM_BUFFER at the input reconstructed with the current
 * parameters, with the parameters the forward used (blocks and front layer);
 * DELAYED uses both buffers, the standard delayed gradient.  The last stage
 * has no delay, so every variant is the PETRA backward there. */
typedef enum {
  PETRA_BWD_RECONSTRUCT = 0,
  PETRA_BWD_INPUT_BUFFER = 1,
  PETRA_BWD_PARAM_BUFFER = 2,
  PETRA_BWD_DELAYED = 3
} petra_bwd_mode;
/* Sets the variant of the following ticks (default: the buffers kept).
 * PETRA_ERR_STATE if it needs a buffer the description did not ask for. */
petra_status petra_net_set_backward(petra_net* net, int32_t mode);
/* Stage `stage`'s parameters are elements [*offset, *offset + *numel) of the
 * flat buffers (front layer, blocks, and the head for the last stage). */
petra_status petra_net_stage_params(const petra_net* net, int32_t stage, int64_t* offset,
                                    int64_t* numel);
/* Device memory of stage `stage` by purpose, in bytes (Tables 3 and 6).  The
 * first field counts the caller-owned fp32 buffers (parameters, accumulator,
 * momentum, running statistics); the rest are the stage's parts of the
 * workspace, which sum with the other stages' to petra_net_query()'s
 * workspace_bytes. */
typedef struct {
  int64_t params;             /* fp32 parameters, accumulator, momentum, running stats */
  int64_t weight_copies;      /* compute copies of the conv weights (forward, transposed) */
  int64_t activation_buffer;  /* the front layer's input, one per micro-batch in flight */
  int64_t input_buffer;       /* the blocks' input per micro-batch in flight (if kept) */
  int64_t param_buffer;       /* stashed parameters per micro-batch in flight (if kept) */
  int64_t scratch;            /* one micro-batch's working set, messages, the rest */
  int64_t total;
} petra_net_mem;
petra_status petra_net_memory(const petra_net* net, int32_t stage, petra_net_mem* out);
/* Gradient probes for the gradient-quality diagnostics (App. B); neither
 * changes parameters, accumulators, running statistics, counters or the
 * micro-batches in flight.  grad_out: device fp32 [n_params], 16-byte aligned,
 * zeroed and then filled with unscaled gradients (no 1/accum_k); ordered on
 * `stream` after prior work.
 * petra_net_probe_tick: the gradients the backward passes of the next tick
 * would compute in variant `mode` (stages without a backward then stay zero).
 * petra_net_probe_backprop: the end-to-end gradient of one micro-batch
 * (images, labels as for petra_net_tick) at the current parameters. */
petra_status petra_net_probe_tick(petra_net* net, int32_t mode, float* grad_out, void* stream);
petra_status petra_net_probe_backprop(petra_net* net, const void* images, const int32_t* labels,
                                      float* grad_out, void* stream);
/* Reversible backpropagation baseline (Sec. 4.2 and Table 5, the comparison
 * of iteration times): one micro-batch through the same network and kernels
 * with exact gradients and no overlap.  The forward of every stage in order
 * (front layers keep their output, reversible blocks keep nothing), the loss
 * head, then the backward of every stage from the last to the first, the
 * blocks rebuilding their inputs from their outputs; each stage applies its
 * update (petra_net_set_optimizer; accum_k counts these steps) right after its
 * backward, which the stages below do not read.  All work is ordered on
 * `stream`.  images [n][h][w][c_img] (storage type) and labels [n] int32 are
 * device pointers (16-byte aligned); loss (nullable, device fp32) receives the
 * micro-batch's mean loss.  Does not advance the tick counters.
 * PETRA_ERR_STATE while micro-batches of petra_net_tick are in flight (the
 * step would update parameters they have yet to use in their backward). */
petra_status petra_net_backprop_step(petra_net* net, const void* images, const int32_t* labels,
                                     float* loss, void* stream);

/* Measurement support (not part of the method).  petra_stage_profile(st, 1)
 * clears the counters and starts bracketing every kernel launch of the stage
 * with HIP events on the stream the kernel is launched on; 0 stops it.
 * petra_stage_profile_read() waits for the recorded events and returns, for
 * kernel class `kernel_class` (0 .. until it returns PETRA_ERR_INVALID_ARG),
 * its name, launch count, summed device time in ms and the summed algorithmic
 * flops and bytes of those launches (compulsory traffic of each launch: every
 * operand read once, every result written once). */
petra_status petra_stage_profile(petra_stage* st, int32_t enable);
petra_status petra_stage_profile_read(petra_stage* st, int32_t kernel_class, const char** name,
                                      int64_t* launches, double* total_ms, double* flops,
                                      double* bytes);
/* The same totals per kernel (template instance) and class, index 0 .. until
 * it returns PETRA_ERR_INVALID_ARG, in order of first launch since the
 * profile was enabled: *name receives the kernel's demangled symbol as the
 * profiler tools print it (valid until the next petra_stage_profile call),
 * *kernel_class its class index for petra_stage_profile_read. */
petra_status petra_stage_profile_kernel(petra_stage* st, int32_t index, const char** name,
                                        int32_t* kernel_class, int64_t* launches,
                                        double* total_ms, double* flops, double* bytes);

#ifdef __cplusplus
}
#endif

#endif /* PETRA_H */
