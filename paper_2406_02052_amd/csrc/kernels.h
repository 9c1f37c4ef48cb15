// Kernel argument blocks and host-side launchers (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace petra {

enum { DT_FP32 = 0, DT_BF16 = 1 };
enum { EP_STATS = 0, EP_MASK = 1, EP_RESID = 2 };

// Implicit-GEMM convolution (forward, or input gradient with transposed weights).
struct ConvArgs {
  const void* src;         // input [N][H][W][c_split] (or first half of a concat)
  const void* src2;        // optional second input [N][H][W][c_in - c_split], channels >= c_split
  int c_split;             // channels held by src (== c_in without src2)
  const float* pro_scale;  // optional prologue: input -> max(scale*x + shift, 0) per input channel
  const float* pro_shift;
  const void* wt;          // [c_out][k_tot], k = (r, s, c)
  void* out;               // [m][c_out]
  const void* resid;       // EP_RESID: out = resid + conv (may alias out)
  const void* ep_h;        // EP_MASK: pre-BN tensor of the layer below, [m][c_out]
  const float* ep_scale;   // EP_MASK: BN scale/shift/mean/rstd of that layer
  const float* ep_shift;
  const float* ep_mean;
  const float* ep_rstd;
  float* partials;         // EP_STATS / EP_MASK: [tiles_m][2][c_out]
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
  float* partials;         // [splits][c_out][k_tot]
  int n, h, w, c_in, p, q, c_out, r, s, stride, pad, k_tot, m;
  int rows_per_split, splits;
};

constexpr int CONV_BM = 128;  // rows per conv output tile (= partial-sum tile)

void conv_gemm(int dtype, const ConvArgs& a, int ep, hipStream_t st);
// Number of partial-sum rows (output row tiles) conv_gemm writes for these arguments.
int conv_row_tiles(int dtype, const ConvArgs& a);
void conv_wgrad(int dtype, const WgradArgs& a, hipStream_t st);
// Halo-tile weight-gradient kernel selection (0 = not applicable) and the
// number of pixel tiles it splits over.
int wgrad_halo_shape(int dtype, const WgradArgs& a);
int wgrad_halo_tiles(int dtype, const WgradArgs& a);
void wgrad_reduce(const float* part, int splits, long numel, float inv_k, float* grad,
                  hipStream_t st);

// BN statistics: partials [tiles][2][c] of (sum h, sum h^2) over m rows.
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
// x = v - (scale*h + shift)  (reconstruction), with partials of (sum d, sum d*xhat).
void combine_bwd(int dtype, const void* v, const void* h, const void* d, const float* scale,
                 const float* shift, const float* mean, const float* rstd, void* x,
                 float* partials, long m, int c, hipStream_t st);
// out = ca*d + cb*(h - mean) + cc  (BN input gradient); may run in place on d.
void bn_bwd_apply(int dtype, const void* d, const void* h, const float* ca, const float* cb,
                  const float* cc, const float* mean, void* out, long m, int c, hipStream_t st);

// Conv weight tensors inside the flat parameter buffer, for the refresh of
// the storage-type compute copies.
struct WeightSeg {
  int64_t off;     // element offset of [c_out][r][s][c_in] in the flat buffer (== in fwd copy)
  int64_t dg_off;  // element offset of the transposed/flipped copy [c_in][r][s][c_out]
  int c_out, r, s, c_in;
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
// in the table (segments sorted by offset, covering [0, n_conv)).
void refresh_weights(int dtype, const float* theta, const WeightSegTable& segs, int64_t n_conv,
                     void* fwd_copy, void* dg_copy, hipStream_t st);

}  // namespace petra
