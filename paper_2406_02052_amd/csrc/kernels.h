// Kernel argument blocks and host-side launchers (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace petra {

enum { DT_FP32 = 0, DT_BF16 = 1 };
// Epilogues: BN statistics of the output; ReLU mask of the layer below plus its
// BN-backward partials; residual add; residual add plus the BN-backward
// partials of the stored result against a BN layer given by ep_h/ep_mean/ep_rstd.
enum { EP_STATS = 0, EP_MASK = 1, EP_RESID = 2, EP_RESID_STATS = 3 };
// Prologues applied to the gathered input: none; BN-apply + ReLU
// (pro_scale/pro_shift); BN backward (pro_h, pro_ca/cb/cc/mean).
enum { PRO_NONE = 0, PRO_RELU = 1, PRO_BWD = 2 };

// Implicit-GEMM convolution (forward, or input gradient with transposed weights).
struct ConvArgs {
  const void* src;         // input [N][H][W][c_split] (or first half of a concat)
  const void* src2;        // optional second input [N][H][W][c_in - c_split], channels >= c_split
  int c_split;             // channels held by src (== c_in without src2)
  const float* pro_scale;  // optional prologue: input -> max(scale*x + shift, 0) per input channel
  const float* pro_shift;
  // optional prologue (with pro_h set): input d -> ca*d + cb*(h - mean) + cc per input
  // channel, h read from pro_h at the same position (BN input gradient formed on the fly)
  const void* pro_h;
  const float* pro_ca;
  const float* pro_cb;
  const float* pro_cc;
  const float* pro_mean;
  const void* wt;          // [c_out][k_tot], k = (r, s, c)
  void* out;               // [m][c_out]
  const void* resid;       // EP_RESID: out = resid + conv (may alias out); null: out = conv
  const void* ep_h;        // EP_MASK / EP_RESID_STATS: pre-BN tensor of that BN layer, [m][c_out]
  const float* ep_scale;   // EP_MASK: BN scale/shift of the layer below
  const float* ep_shift;
  const float* ep_mean;    // EP_MASK / EP_RESID_STATS: BN mean/rstd of that layer
  const float* ep_rstd;
  float* partials;         // EP_STATS: [tiles][3][c_out] (rows, sum, centred sum of squares);
                           // EP_MASK / EP_RESID_STATS: [tiles][2][c_out] (sum g, sum g*xhat)
  int n, h, w, c_in, p, q, c_out, r, s, stride, pad, k_tot, m;
};

// Weight gradient partials over split row chunks.
struct WgradArgs {
  const void* dh;          // output-side gradient [m][c_out]
  const void* src;         // conv input (as in ConvArgs)
  const void* src2;
  int c_split;
  const float* pro_scale;
  const float* pro_shift;
  // optional (with dh_h set): the output-side operand is ca*dh + cb*(h - mean) + cc per
  // output channel, h read from dh_h [m][c_out]
  const void* dh_h;
  const float* dh_ca;
  const float* dh_cb;
  const float* dh_cc;
  const float* dh_mean;
  float* partials;         // [splits][c_out][k_tot]
  int n, h, w, c_in, p, q, c_out, r, s, stride, pad, k_tot, m;
  int rows_per_split, splits;
};

constexpr int CONV_BM = 128;  // rows per conv output tile (= partial-sum tile)

// Launches the conv; false (nothing launched) for an unsupported epilogue /
// prologue pair (EP_STATS takes PRO_NONE or PRO_RELU, the others PRO_NONE or
// PRO_BWD).
bool conv_gemm(int dtype, const ConvArgs& a, int ep, hipStream_t st);
// Number of partial-sum rows (output row tiles) conv_gemm writes for these
// arguments and epilogue.
int conv_row_tiles(int dtype, const ConvArgs& a, int ep);
// With a.out == nullptr, conv_gemm's streaming 1x1 forward (EP_STATS) writes
// the BN partials only.  conv1x1_couple then forms the coupling output
// a.out = a.resid +/- (scale h + shift) with h = that conv of
// relu(pro_scale * a.src + pro_shift), recomputed bit for bit as the
// statistics pass rounded it (a.out may alias a.resid); false, with nothing
// launched, where it does not apply (conv1x1_couple_ok: bf16 1x1 32 -> 128).
// With next, the coupling output (sum or reconstruction) is also fed to the next
// residual function's first conv, the 1x1 128 -> 32 (weights next->wt): its
// pre-BN output goes to next->out and its BN partials to next->partials,
// exactly as conv_gemm (EP_STATS, no prologue) would write them from the
// stored coupling output (the same partial rows: conv_row_tiles of that conv).
struct NextConv {
  const void* wt;   // [32][128] weights (c_out x c_in) of the next function's first conv
  void* out;        // [m][32] its pre-BN output
  float* partials;  // [tiles][3][32] its BN partials (tiles = conv_row_tiles of that conv)
};
bool conv1x1_couple_ok(int dtype, const ConvArgs& a);
// Whether the coupling of `a` can also run `next` (that first conv, EP_STATS).
bool conv1x1_couple_next_ok(int dtype, const ConvArgs& a, const ConvArgs& next);
bool conv1x1_couple(int dtype, const ConvArgs& a, const float* scale, const float* shift,
                    bool sub, hipStream_t st, const NextConv* next = nullptr);
void conv_wgrad(int dtype, const WgradArgs& a, hipStream_t st);
// Transposed-read weight-gradient kernel: configuration (0 = not applicable)
// and its split count (partial rows) for these arguments; conv_wgrad uses it
// whenever it applies, with a.splits set to that count.
int wgrad_tr_plan(int dtype, const WgradArgs& a, int* splits);
// Several layers' transposed-read weight gradients in one launch (each entry
// as for conv_wgrad, partials to its own a.partials); false, with nothing
// launched, unless that kernel applies to every entry with one configuration.
constexpr int MAX_WG_GROUP = 16;
struct WgGroupTable {
  int n;
  long block_begin[MAX_WG_GROUP];
  WgradArgs a[MAX_WG_GROUP];
};
bool conv_wgrad_tr_group(int dtype, const WgradArgs* args, int n, hipStream_t st);
// Halo-tile weight-gradient kernel selection (0 = not applicable) and the
// number of pixel tiles it splits over.
int wgrad_halo_shape(int dtype, const WgradArgs& a);
int wgrad_halo_tiles(int dtype, const WgradArgs& a);
void wgrad_reduce(const float* part, int splits, long numel, float inv_k, float* grad,
                  hipStream_t st);
// Split reduce of the transposed-read kernel's fragment-ordered partials
// (a.partials, a.splits) into grad[o][k] += inv_k * sum; false when that
// kernel does not apply to these arguments (use wgrad_reduce then).
bool wgrad_tr_reduce(int dtype, const WgradArgs& a, float inv_k, float* grad, hipStream_t st);
// Deferred form: one layer's reduce as a table entry (partials at base +
// part_off, gradient at grad_base + w_off), false when the transposed-read
// kernel does not apply; wgrad_tr_reduce_group then reduces many layers in one
// launch (per element the same fixed order as wgrad_tr_reduce).
struct TrMap {
  int wo, of, wc, cf, wt, tpw, bo, bc, nz, c_in, k_tot;
};
struct TrSeg {
  long part_off, w_off, numel, block_begin;
  int splits;
  TrMap mp;
};
constexpr int MAX_TR_SEGS = 32;
struct TrSegTable {
  int n;
  TrSeg seg[MAX_TR_SEGS];
};
bool wgrad_tr_segment(int dtype, const WgradArgs& a, long part_off, long w_off, TrSeg* seg);
void wgrad_tr_reduce_group(const float* base, const TrSeg* segs, int nseg, float inv_k,
                           float* grad_base, hipStream_t st);

// BN statistics: partials [tiles][3][c] of (rows, sum h, sum (h - tile mean)^2)
// combined across tiles with Chan's pairwise formula in fp64 (m rows in all).
// Writes scale = gamma*rstd, shift = beta - mean*scale, mean, rstd; when
// run_mean != nullptr also moves the running statistics (unbiased variance).
void bn_stats_finalize(const float* partials, int tiles, int c, long m, const float* gamma,
                       const float* beta, float eps, float* scale, float* shift, float* mean,
                       float* rstd, float* run_mean, float* run_var, float momentum,
                       hipStream_t st);

// BN backward: partials [tiles][2][c] of (sum d, sum d*xhat).  Adds
// inv_k*dgamma, inv_k*dbeta to the gradient accumulator and writes the
// coefficients of dh = ca*d + cb*(h - mean) + cc.
void bn_bwd_finalize(const float* partials, int tiles, int c, long m, const float* gamma,
                     const float* mean, const float* rstd, float inv_k, float* dgamma,
                     float* dbeta, float* ca, float* cb, float* cc, hipStream_t st);

// Row-chunk count used by the reducing elementwise kernel for m rows.
int ew_tiles(long m, int c);

// y = r + scale*h + shift  (forward coupling add)
void combine_fwd(int dtype, const void* r, const void* h, const float* scale, const float* shift,
                 void* y, long m, int c, hipStream_t st);
// x = v - (scale*h + shift)  (reconstruction only).
void combine_rec(int dtype, const void* v, const void* h, const float* scale, const float* shift,
                 void* x, long m, int c, hipStream_t st);
// x = v - (scale*h + shift)  (reconstruction), with partials of (sum d, sum d*xhat).
void combine_bwd(int dtype, const void* v, const void* h, const void* d, const float* scale,
                 const float* shift, const float* mean, const float* rstd, void* x,
                 float* partials, long m, int c, hipStream_t st);

// Conv weight tensors inside the flat parameter buffer, for the refresh of
// the storage-type compute copies.
struct WeightSeg {
  int64_t off;     // element offset of the master [c_out][r][s][c_in] in the flat buffer
  int64_t fwd_off; // element offset of the forward copy [c_out][r][s][c_in_pad] (pads zeroed)
  int64_t dg_off;  // element offset of the transposed/flipped copy [c_in][r][s][c_out]
  int c_out, r, s, c_in, c_in_pad;
};

constexpr int MAX_WEIGHT_SEGS = 96;
struct WeightSegTable {
  int nseg;
  WeightSeg seg[MAX_WEIGHT_SEGS];
};

// SGD step over the flat buffers (elements [0, n_decay) get weight decay),
// zeroing the accumulator.
void sgd_update(float* theta, float* accum, float* mom, int64_t n, int64_t n_decay, float lr,
                float momentum, float wd, int nesterov, hipStream_t st);
// Write the forward and transposed compute copies of the conv weights listed
// in the table; max_numel bounds the padded size of the largest segment.
void refresh_weights(int dtype, const float* theta, const WeightSegTable& segs, int64_t max_numel,
                     void* fwd_copy, void* dg_copy, hipStream_t st);

// ---- multi-stage network helpers ------------------------------------------
// dst[m][0..8) = src[m][0..c_img) zero-padded to 8 channels (c_img <= 8).
void pad_channels8(int dtype, const void* src, int c_img, void* dst, long m, hipStream_t st);
void copy_i32(const int32_t* src, int32_t* dst, int n, hipStream_t st);
// out1/out2 [m][c/2] = (relu)(scale*h + shift) of h [m][c], split into halves.
void bn_apply_split(int dtype, const void* h, const float* scale, const float* shift, int relu,
                    void* out1, void* out2, long m, int c, hipStream_t st);
// BN backward over an input gradient given as halves d1/d2 [m][c/2] of h [m][c]
// (optionally through the ReLU that followed the BN): partial sums of
// (dz, dz*xhat) per tile, then dh = ca*dz + cb*(h - mean) + cc.
int split_tiles(long m, int c);
void split_bwd_partials(int dtype, const void* d1, const void* d2, const void* h,
                        const float* scale, const float* shift, const float* mean,
                        const float* rstd, int relu, float* partials, long m, int c,
                        hipStream_t st);
void split_bwd_apply(int dtype, const void* d1, const void* d2, const void* h,
                     const float* scale, const float* shift, const float* ca, const float* cb,
                     const float* cc, const float* mean, int relu, void* dh, long m, int c,
                     hipStream_t st);
// dst1/dst2 [n][h][w][c/2]: rows of src [n*(h/2)*(w/2)][c] at even pixels, zero elsewhere.
void scatter_stride2_split(int dtype, const void* src, void* dst1, void* dst2, int n, int h,
                           int w, int c, hipStream_t st);
// Head: global average pool of [x1|x2] ([n][hw][c/2] each), linear layer
// (fp32 weight [k][c], bias [k]), softmax cross-entropy against labels.
// Writes pooled [n][c], dlogits [n][k] (already divided by n), per-image loss
// [n] and the input gradient halves g1/g2.
void head_forward_backward(int dtype, const void* x1, const void* x2, int n, int hw, int c,
                           const float* wfc, const float* bfc, int k, const int32_t* labels,
                           float* pooled, float* dlogits, float* loss_n, void* g1, void* g2,
                           hipStream_t st);
// grad_w += inv_k * dlogits^T pooled; grad_b += inv_k * sum dlogits; loss = mean(loss_n).
void head_param_grads(const float* pooled, const float* dlogits, const float* loss_n, int n,
                      int c, int k, float inv_k, float* grad_w, float* grad_b, float* loss,
                      hipStream_t st);
// Split-K reduce for weights stored with padded input channels:
// grad[o][tap][c] += inv_k * sum_split part[split][o][tap][c_pad] for c < c_real.
void wgrad_reduce_pad(const float* part, int splits, int c_out, int taps, int c_pad, int c_real,
                      float inv_k, float* grad, hipStream_t st);

}  // namespace petra
