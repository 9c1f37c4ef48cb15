// In-place parameter update and compute-copy refresh (gfx950).
//
// One pass over the flat fp32 buffers applies SGD with momentum (Nesterov or
// heavy ball, no dampening, weight decay on the leading conv-weight range
// only) and zeroes the gradient accumulator; a second pass rounds the conv
// weights into the storage-type copies read by the forward/backward kernels:
// the KRSC copy and the transposed, R/S-flipped copy used for input gradients.
#include "common.h"
#include "kernels.h"

namespace petra {

namespace {

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

template <typename T>
__global__ __launch_bounds__(256) void refresh_kernel(const float* __restrict__ theta, WeightSegTable segs,
                                                      int64_t n_conv, T* __restrict__ fwd,
                                                      T* __restrict__ dg) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n_conv;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    int lo = 0, hi = segs.nseg - 1;
    while (lo < hi) {  // last segment with off <= i
      const int mid = (lo + hi + 1) >> 1;
      if (segs.seg[mid].off <= i) lo = mid; else hi = mid - 1;
    }
    const WeightSeg& sg = segs.seg[lo];
    const int64_t local = i - sg.off;
    const int ci = static_cast<int>(local % sg.c_in);
    const int64_t t1 = local / sg.c_in;
    const int s = static_cast<int>(t1 % sg.s);
    const int64_t t2 = t1 / sg.s;
    const int r = static_cast<int>(t2 % sg.r);
    const int o = static_cast<int>(t2 / sg.r);
    const float v = theta[i];
    store1(fwd + i, v);
    const int64_t j = sg.dg_off +
                      ((static_cast<int64_t>(ci) * sg.r + (sg.r - 1 - r)) * sg.s + (sg.s - 1 - s)) * sg.c_out + o;
    store1(dg + j, v);
  }
}

unsigned grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  return static_cast<unsigned>(b);
}

}  // namespace

void sgd_update(float* theta, float* accum, float* mom, int64_t n, int64_t n_decay, float lr,
                float momentum, float wd, int nesterov, hipStream_t st) {
  hipLaunchKernelGGL(sgd_kernel, dim3(grid_for(n)), dim3(256), 0, st, theta, accum, mom, n, n_decay,
                     lr, momentum, wd, nesterov);
}

void refresh_weights(int dtype, const float* theta, const WeightSegTable& segs, int64_t n_conv,
                     void* fwd_copy, void* dg_copy, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(refresh_kernel<bf16_t>, dim3(grid_for(n_conv)), dim3(256), 0, st, theta, segs,
                       n_conv, static_cast<bf16_t*>(fwd_copy), static_cast<bf16_t*>(dg_copy));
  else
    hipLaunchKernelGGL(refresh_kernel<float>, dim3(grid_for(n_conv)), dim3(256), 0, st, theta, segs,
                       n_conv, static_cast<float*>(fwd_copy), static_cast<float*>(dg_copy));
}

}  // namespace petra
