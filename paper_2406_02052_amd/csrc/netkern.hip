// Kernels of the multi-stage network: image ingest, the non-reversible front
// layers' BN passes on split activations, the stride-2 input-gradient scatter,
// the softmax cross-entropy head and the padded-channel split-K reduce.
#include "common.h"
#include "kernels.h"
#include "prof.h"

namespace petra {

namespace netk {

unsigned grid_of(long n, long per_block = 256) {
  long b = (n + per_block - 1) / per_block;
  if (b > 65536) b = 65536;
  if (b < 1) b = 1;
  return static_cast<unsigned>(b);
}

template <typename T>
__global__ __launch_bounds__(256) void pad8_kernel(const T* src, int c_img, T* dst, long m) {
  for (long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; i < m * 8;
       i += static_cast<long>(gridDim.x) * 256) {
    const long row = i >> 3;
    const int c = static_cast<int>(i & 7);
    dst[i] = c < c_img ? src[row * c_img + c] : T{};
  }
}

__global__ void copy_i32_kernel(const int32_t* src, int32_t* dst, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

template <typename T>
__global__ __launch_bounds__(256) void bn_apply_split_kernel(const T* h, const float* scale,
                                                             const float* shift, int relu, T* o1,
                                                             T* o2, long m, int c) {
  const int c8 = c / 8, half = c / 2;
  for (long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; i < m * c8;
       i += static_cast<long>(gridDim.x) * 256) {
    const long row = i / c8;
    const int ch = static_cast<int>(i - row * c8) * 8;
    float v[8];
    Vec8<T>::load(h + row * c + ch, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = fmaf(scale[ch + j], v[j], shift[ch + j]);
      if (relu) v[j] = fmaxf(v[j], 0.f);
    }
    T* dst = ch < half ? o1 + row * half + ch : o2 + row * half + (ch - half);
    Vec8<T>::store(dst, v);
  }
}

// Gradient of the BN output (optionally masked by the ReLU after it), read
// from the two half tensors.
template <typename T>
__device__ __forceinline__ void load_dz(const T* d1, const T* d2, const T* h, const float* scale,
                                        const float* shift, int relu, long row, int ch, int c,
                                        float* dz, float* hv) {
  const int half = c / 2;
  const T* src = ch < half ? d1 + row * half + ch : d2 + row * half + (ch - half);
  Vec8<T>::load(src, dz);
  Vec8<T>::load(h + row * c + ch, hv);
  if (relu) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (!(fmaf(scale[ch + j], hv[j], shift[ch + j]) > 0.f)) dz[j] = 0.f;
  }
}

int split_rows_per_tile(long m, int c) {
  const int rows_per_pass = 256 / (c / 8);
  long want = (m + 1023) / 1024;
  long rpt = ((want + rows_per_pass - 1) / rows_per_pass) * rows_per_pass;
  if (rpt < rows_per_pass) rpt = rows_per_pass;
  return static_cast<int>(rpt);
}

template <typename T>
__global__ __launch_bounds__(256) void split_bwd_partials_kernel(
    const T* d1, const T* d2, const T* h, const float* scale, const float* shift,
    const float* mean, const float* rstd, int relu, float* partials, long m, int c,
    int rows_per_tile) {
  const int c8 = c / 8;
  const int rows_per_pass = 256 / c8;
  const int tid = threadIdx.x;
  const int cg = tid % c8, rr = tid / c8;
  const int ch = cg * 8;
  const long row0 = static_cast<long>(blockIdx.x) * rows_per_tile;
  const long row1 = min(m, row0 + rows_per_tile);
  float s1[8], s2[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) s1[j] = s2[j] = 0.f;
  if (rr < rows_per_pass) {
    for (long row = row0 + rr; row < row1; row += rows_per_pass) {
      float dz[8], hv[8];
      load_dz(d1, d2, h, scale, shift, relu, row, ch, c, dz, hv);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        s1[j] += dz[j];
        s2[j] += dz[j] * ((hv[j] - mean[ch + j]) * rstd[ch + j]);
      }
    }
  }
  __shared__ float buf[2][256][9];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    buf[0][tid][j] = s1[j];
    buf[1][tid][j] = s2[j];
  }
  __syncthreads();
  for (int i = tid; i < 2 * c; i += 256) {
    const int which = i / c, chh = i - which * c;
    const int g = chh / 8, j = chh - g * 8;
    float t = 0.f;
    for (int q = 0; q < rows_per_pass; ++q) t += buf[which][q * c8 + g][j];
    partials[(static_cast<long>(blockIdx.x) * 2 + which) * c + chh] = t;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void split_bwd_apply_kernel(
    const T* d1, const T* d2, const T* h, const float* scale, const float* shift, const float* ca,
    const float* cb, const float* cc, const float* mean, int relu, T* dh, long m, int c) {
  const int c8 = c / 8;
  for (long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; i < m * c8;
       i += static_cast<long>(gridDim.x) * 256) {
    const long row = i / c8;
    const int ch = static_cast<int>(i - row * c8) * 8;
    float dz[8], hv[8], o[8];
    load_dz(d1, d2, h, scale, shift, relu, row, ch, c, dz, hv);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      o[j] = fmaf(ca[ch + j], dz[j], fmaf(cb[ch + j], hv[j] - mean[ch + j], cc[ch + j]));
    Vec8<T>::store(dh + row * c + ch, o);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void scatter2_kernel(const T* src, T* dst1, T* dst2, int n,
                                                       int h, int w, int c) {
  const int c8 = c / 8, half = c / 2;
  const int h2 = h / 2, w2 = w / 2;
  const long total = static_cast<long>(n) * h * w * c8;
  for (long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; i < total;
       i += static_cast<long>(gridDim.x) * 256) {
    const long pix = i / c8;
    const int ch = static_cast<int>(i - pix * c8) * 8;
    const int x = static_cast<int>(pix % w);
    const int y = static_cast<int>((pix / w) % h);
    const long img = pix / (static_cast<long>(h) * w);
    float v[8];
    if ((x & 1) == 0 && (y & 1) == 0 && (y >> 1) < h2 && (x >> 1) < w2) {
      const long srow = (img * h2 + (y >> 1)) * w2 + (x >> 1);
      Vec8<T>::load(src + srow * c + ch, v);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.f;
    }
    T* dst = ch < half ? dst1 + pix * half + ch : dst2 + pix * half + (ch - half);
    Vec8<T>::store(dst, v);
  }
}

// One block per image.  c <= 1024, k <= 64.
template <typename T>
__global__ __launch_bounds__(256) void head_kernel(const T* x1, const T* x2, int hw, int c,
                                                   const float* wfc, const float* bfc, int k,
                                                   const int32_t* labels, int n, float* pooled,
                                                   float* dlogits, float* loss_n, T* g1, T* g2) {
  __shared__ float sp[1024];
  __shared__ float sl[64];
  __shared__ float sdp[1024];
  const int img = blockIdx.x;
  const int tid = threadIdx.x;
  const int half = c / 2;
  for (int ch = tid; ch < c; ch += 256) {
    const T* src = ch < half ? x1 + static_cast<long>(img) * hw * half + ch
                             : x2 + static_cast<long>(img) * hw * half + (ch - half);
    float acc = 0.f;
    for (int p = 0; p < hw; ++p) acc += load1(src + static_cast<long>(p) * half);
    const float v = acc / static_cast<float>(hw);
    sp[ch] = v;
    pooled[static_cast<long>(img) * c + ch] = v;
  }
  __syncthreads();
  const int lane = tid & 63, wave = tid >> 6;
  for (int j = wave; j < k; j += 4) {
    float acc = 0.f;
    for (int ch = lane; ch < c; ch += 64) acc += sp[ch] * wfc[static_cast<long>(j) * c + ch];
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (lane == 0) sl[j] = acc + bfc[j];
  }
  __syncthreads();
  if (tid == 0) {
    float mx = sl[0];
    for (int j = 1; j < k; ++j) mx = fmaxf(mx, sl[j]);
    double se = 0.0;
    for (int j = 0; j < k; ++j) se += exp(static_cast<double>(sl[j] - mx));
    const double lse = log(se);
    const int raw = labels[img];
    const bool valid = raw >= 0 && raw < k;   // an out-of-range label yields a NaN loss
    const int lab = valid ? raw : 0;
    loss_n[img] = valid ? static_cast<float>(lse - (sl[lab] - mx)) : __int_as_float(0x7fc00000);
    for (int j = 0; j < k; ++j) {
      double p = exp(static_cast<double>(sl[j] - mx) - lse);
      if (j == lab) p -= 1.0;
      sl[j] = static_cast<float>(p / n);
      dlogits[static_cast<long>(img) * k + j] = sl[j];
    }
  }
  __syncthreads();
  for (int ch = tid; ch < c; ch += 256) {
    float acc = 0.f;
    for (int j = 0; j < k; ++j) acc += sl[j] * wfc[static_cast<long>(j) * c + ch];
    sdp[ch] = acc / static_cast<float>(hw);
  }
  __syncthreads();
  for (long i = tid; i < static_cast<long>(hw) * c; i += 256) {
    const int p = static_cast<int>(i / c);
    const int ch = static_cast<int>(i - static_cast<long>(p) * c);
    T* dst = ch < half ? g1 + (static_cast<long>(img) * hw + p) * half + ch
                       : g2 + (static_cast<long>(img) * hw + p) * half + (ch - half);
    store1(dst, sdp[ch]);
  }
}

__global__ __launch_bounds__(256) void head_grads_kernel(const float* pooled, const float* dlogits,
                                                         const float* loss_n, int n, int c, int k,
                                                         float inv_k, float* gw, float* gb,
                                                         float* loss) {
  const long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  if (i < static_cast<long>(k) * c) {
    const int j = static_cast<int>(i / c), ch = static_cast<int>(i - static_cast<long>(j) * c);
    float acc = 0.f;
    for (int r = 0; r < n; ++r) acc += dlogits[static_cast<long>(r) * k + j] * pooled[static_cast<long>(r) * c + ch];
    gw[i] += inv_k * acc;
  }
  if (blockIdx.x == 0 && threadIdx.x < k) {
    float acc = 0.f;
    for (int r = 0; r < n; ++r) acc += dlogits[static_cast<long>(r) * k + threadIdx.x];
    gb[threadIdx.x] += inv_k * acc;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && loss != nullptr) {
    double acc = 0.0;
    for (int r = 0; r < n; ++r) acc += loss_n[r];
    *loss = static_cast<float>(acc / n);
  }
}

__global__ __launch_bounds__(256) void wgrad_reduce_pad_kernel(const float* part, int splits,
                                                               int c_out, int taps, int c_pad,
                                                               int c_real, float inv_k,
                                                               float* grad) {
  const long numel = static_cast<long>(c_out) * taps * c_real;
  const long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= numel) return;
  const int cr = static_cast<int>(i % c_real);
  const long ot = i / c_real;  // o * taps + tap
  const long src = ot * c_pad + cr;
  const long stride = static_cast<long>(c_out) * taps * c_pad;
  float s = 0.f;
  for (int t = 0; t < splits; ++t) s += part[t * stride + src];
  grad[i] += inv_k * s;
}

}  // namespace netk
using namespace netk;

void pad_channels8(int dtype, const void* src, int c_img, void* dst, long m, hipStream_t st) {
  if (dtype == DT_BF16)
    PETRA_LAUNCH(pad8_kernel<bf16_t>, dim3(grid_of(m * 8)), dim3(256), 0, st,
                       static_cast<const bf16_t*>(src), c_img, static_cast<bf16_t*>(dst), m);
  else
    PETRA_LAUNCH(pad8_kernel<float>, dim3(grid_of(m * 8)), dim3(256), 0, st,
                       static_cast<const float*>(src), c_img, static_cast<float*>(dst), m);
}

void copy_i32(const int32_t* src, int32_t* dst, int n, hipStream_t st) {
  PETRA_LAUNCH(copy_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, st, src, dst, n);
}

void bn_apply_split(int dtype, const void* h, const float* scale, const float* shift, int relu,
                    void* out1, void* out2, long m, int c, hipStream_t st) {
  const unsigned g = grid_of(m * (c / 8));
  if (dtype == DT_BF16)
    PETRA_LAUNCH(bn_apply_split_kernel<bf16_t>, dim3(g), dim3(256), 0, st,
                       static_cast<const bf16_t*>(h), scale, shift, relu,
                       static_cast<bf16_t*>(out1), static_cast<bf16_t*>(out2), m, c);
  else
    PETRA_LAUNCH(bn_apply_split_kernel<float>, dim3(g), dim3(256), 0, st,
                       static_cast<const float*>(h), scale, shift, relu,
                       static_cast<float*>(out1), static_cast<float*>(out2), m, c);
}

int split_tiles(long m, int c) {
  const int rpt = split_rows_per_tile(m, c);
  return static_cast<int>((m + rpt - 1) / rpt);
}

void split_bwd_partials(int dtype, const void* d1, const void* d2, const void* h,
                        const float* scale, const float* shift, const float* mean,
                        const float* rstd, int relu, float* partials, long m, int c,
                        hipStream_t st) {
  const int rpt = split_rows_per_tile(m, c);
  const int tiles = static_cast<int>((m + rpt - 1) / rpt);
  if (dtype == DT_BF16)
    PETRA_LAUNCH(split_bwd_partials_kernel<bf16_t>, dim3(tiles), dim3(256), 0, st,
                       static_cast<const bf16_t*>(d1), static_cast<const bf16_t*>(d2),
                       static_cast<const bf16_t*>(h), scale, shift, mean, rstd, relu, partials, m,
                       c, rpt);
  else
    PETRA_LAUNCH(split_bwd_partials_kernel<float>, dim3(tiles), dim3(256), 0, st,
                       static_cast<const float*>(d1), static_cast<const float*>(d2),
                       static_cast<const float*>(h), scale, shift, mean, rstd, relu, partials, m,
                       c, rpt);
}

void split_bwd_apply(int dtype, const void* d1, const void* d2, const void* h,
                     const float* scale, const float* shift, const float* ca, const float* cb,
                     const float* cc, const float* mean, int relu, void* dh, long m, int c,
                     hipStream_t st) {
  const unsigned g = grid_of(m * (c / 8));
  if (dtype == DT_BF16)
    PETRA_LAUNCH(split_bwd_apply_kernel<bf16_t>, dim3(g), dim3(256), 0, st,
                       static_cast<const bf16_t*>(d1), static_cast<const bf16_t*>(d2),
                       static_cast<const bf16_t*>(h), scale, shift, ca, cb, cc, mean, relu,
                       static_cast<bf16_t*>(dh), m, c);
  else
    PETRA_LAUNCH(split_bwd_apply_kernel<float>, dim3(g), dim3(256), 0, st,
                       static_cast<const float*>(d1), static_cast<const float*>(d2),
                       static_cast<const float*>(h), scale, shift, ca, cb, cc, mean, relu,
                       static_cast<float*>(dh), m, c);
}

void scatter_stride2_split(int dtype, const void* src, void* dst1, void* dst2, int n, int h,
                           int w, int c, hipStream_t st) {
  const unsigned g = grid_of(static_cast<long>(n) * h * w * (c / 8));
  if (dtype == DT_BF16)
    PETRA_LAUNCH(scatter2_kernel<bf16_t>, dim3(g), dim3(256), 0, st,
                       static_cast<const bf16_t*>(src), static_cast<bf16_t*>(dst1),
                       static_cast<bf16_t*>(dst2), n, h, w, c);
  else
    PETRA_LAUNCH(scatter2_kernel<float>, dim3(g), dim3(256), 0, st,
                       static_cast<const float*>(src), static_cast<float*>(dst1),
                       static_cast<float*>(dst2), n, h, w, c);
}

void head_forward_backward(int dtype, const void* x1, const void* x2, int n, int hw, int c,
                           const float* wfc, const float* bfc, int k, const int32_t* labels,
                           float* pooled, float* dlogits, float* loss_n, void* g1, void* g2,
                           hipStream_t st) {
  if (dtype == DT_BF16)
    PETRA_LAUNCH(head_kernel<bf16_t>, dim3(n), dim3(256), 0, st,
                       static_cast<const bf16_t*>(x1), static_cast<const bf16_t*>(x2), hw, c, wfc,
                       bfc, k, labels, n, pooled, dlogits, loss_n, static_cast<bf16_t*>(g1),
                       static_cast<bf16_t*>(g2));
  else
    PETRA_LAUNCH(head_kernel<float>, dim3(n), dim3(256), 0, st,
                       static_cast<const float*>(x1), static_cast<const float*>(x2), hw, c, wfc,
                       bfc, k, labels, n, pooled, dlogits, loss_n, static_cast<float*>(g1),
                       static_cast<float*>(g2));
}

void head_param_grads(const float* pooled, const float* dlogits, const float* loss_n, int n,
                      int c, int k, float inv_k, float* grad_w, float* grad_b, float* loss,
                      hipStream_t st) {
  const long total = static_cast<long>(k) * c;
  PETRA_LAUNCH(head_grads_kernel, dim3(grid_of(total)), dim3(256), 0, st, pooled, dlogits,
                     loss_n, n, c, k, inv_k, grad_w, grad_b, loss);
}

void wgrad_reduce_pad(const float* part, int splits, int c_out, int taps, int c_pad, int c_real,
                      float inv_k, float* grad, hipStream_t st) {
  const long numel = static_cast<long>(c_out) * taps * c_real;
  PETRA_LAUNCH(wgrad_reduce_pad_kernel, dim3(grid_of(numel)), dim3(256), 0, st, part, splits,
                     c_out, taps, c_pad, c_real, inv_k, grad);
}

}  // namespace petra
