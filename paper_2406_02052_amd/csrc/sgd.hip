// In-place parameter update and compute-copy refresh (gfx950).
//
// One pass over the flat fp32 buffers applies SGD with momentum (Nesterov or
// heavy ball, no dampening, weight decay on the leading conv-weight range
// only) and zeroes the gradient accumulator; a second pass rounds the conv
// weights into the storage-type copies read by the forward/backward kernels:
// the KRSC copy and the transposed, R/S-flipped copy used for input gradients.
#include "common.h"
#include "kernels.h"
#include "prof.h"

namespace petra {

namespace sgdk {

__global__ __launch_bounds__(256) void sgd_kernel(float* __restrict__ theta, float* __restrict__ accum,
                                                  float* __restrict__ mom, int64_t n, int64_t n_decay,
                                                  float lr, float mu, float wd, int nesterov) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const float p = theta[i];
    const float g = accum[i] + (i < n_decay ? wd * p : 0.f);
    const float b = fmaf(mu, mom[i], g);
    mom[i] = b;
    theta[i] = p - lr * (nesterov ? fmaf(mu, b, g) : b);
    accum[i] = 0.f;
  }
}

// blockIdx.y = segment; threads stride over its padded forward layout.
template <typename T>
__global__ __launch_bounds__(256) void refresh_kernel(const float* __restrict__ theta, WeightSegTable segs,
                                                      T* __restrict__ fwd, T* __restrict__ dg) {
  const WeightSeg& sg = segs.seg[blockIdx.y];
  const int64_t n = static_cast<int64_t>(sg.c_out) * sg.r * sg.s * sg.c_in_pad;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const int ci = static_cast<int>(i % sg.c_in_pad);
    const int64_t t1 = i / sg.c_in_pad;
    const int s = static_cast<int>(t1 % sg.s);
    const int64_t t2 = t1 / sg.s;
    const int r = static_cast<int>(t2 % sg.r);
    const int o = static_cast<int>(t2 / sg.r);
    float v = 0.f;
    if (ci < sg.c_in) {
      v = theta[sg.off + ((static_cast<int64_t>(o) * sg.r + r) * sg.s + s) * sg.c_in + ci];
      const int64_t j = sg.dg_off +
                        ((static_cast<int64_t>(ci) * sg.r + (sg.r - 1 - r)) * sg.s + (sg.s - 1 - s)) * sg.c_out + o;
      store1(dg + j, v);
    }
    store1(fwd + sg.fwd_off + i, v);
  }
}

unsigned grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  return static_cast<unsigned>(b);
}

}  // namespace sgdk
using namespace sgdk;

void sgd_update(float* theta, float* accum, float* mom, int64_t n, int64_t n_decay, float lr,
                float momentum, float wd, int nesterov, hipStream_t st) {
  PETRA_LAUNCH(sgd_kernel, dim3(grid_for(n)), dim3(256), 0, st, theta, accum, mom, n, n_decay,
                     lr, momentum, wd, nesterov);
}

void refresh_weights(int dtype, const float* theta, const WeightSegTable& segs, int64_t max_numel,
                     void* fwd_copy, void* dg_copy, hipStream_t st) {
  if (segs.nseg <= 0) return;
  dim3 grid(grid_for(max_numel), segs.nseg);
  if (dtype == DT_BF16)
    PETRA_LAUNCH(refresh_kernel<bf16_t>, grid, dim3(256), 0, st, theta, segs,
                       static_cast<bf16_t*>(fwd_copy), static_cast<bf16_t*>(dg_copy));
  else
    PETRA_LAUNCH(refresh_kernel<float>, grid, dim3(256), 0, st, theta, segs,
                       static_cast<float*>(fwd_copy), static_cast<float*>(dg_copy));
}

}  // namespace petra
