// Batch-normalisation statistics, BN backward coefficients and the fused
// elementwise passes of the reversible coupling (gfx950).
//
// Statistics arrive as per-tile partial sums written by the producing kernel
// (the conv epilogue or combine_bwd); the finalize kernels combine them in a
// fixed order in fp64, so results are run-to-run deterministic.
#include "common.h"
#include "kernels.h"
#include "prof.h"

namespace petra {

namespace bnk {

// Finalize kernels: one 256-thread block per channel.  Thread t takes tiles
// t, t + 256, ... (loads of up to FIN_U tiles in flight), then the block's
// sums are combined in a fixed tree: xor-shuffle levels inside each wave,
// then the four wave results in order.  Deterministic run to run.  The
// summation order does not depend on FIN_U; FIN_U = 2 keeps the statistics
// finalize at 44 VGPRs, so that one of its waves fits on a SIMD beside two
// waves of the whole-image conv (up to 232 VGPRs each).  With FIN_U = 4 (64
// VGPRs) it waited for a CU that conv did not hold (ImageNet32-shaped stage
// step 3.131 -> 3.117 ms).
constexpr int FIN_THREADS = 256;
constexpr int FIN_U = 2;
static_assert(FIN_THREADS == 256, "the wave results are combined as four");

// Sum of (a, b) over partials[tile][2][c] for channel ch.
__device__ void reduce_partials(const float* partials, int tiles, int c, int ch, double& s1,
                                double& s2) {
  __shared__ double red[2][FIN_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double a = 0.0, b = 0.0;
  for (int base = tid; base < tiles; base += FIN_THREADS * FIN_U) {
    float va[FIN_U], vb[FIN_U];
#pragma unroll
    for (int u = 0; u < FIN_U; ++u) {
      const int t = base + u * FIN_THREADS;
      const bool ok = t < tiles;
      va[u] = ok ? partials[(static_cast<long>(t) * 2) * c + ch] : 0.f;
      vb[u] = ok ? partials[(static_cast<long>(t) * 2 + 1) * c + ch] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < FIN_U; ++u) {
      a += va[u];
      b += vb[u];
    }
  }
  for (int off = 1; off < 64; off <<= 1) {
    a += __shfl_xor(a, off, 64);
    b += __shfl_xor(b, off, 64);
  }
  if (lane == 0) {
    red[0][wave] = a;
    red[1][wave] = b;
  }
  __syncthreads();
  s1 = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
  s2 = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
}

// partials[tile][3][c] = (rows n_t, sum S_t, centred sum of squares Q_t) ->
// fp64 totals for ch.  Every tile is re-centred on one shift K, the first
// tile's mean: sum_x (x - K)^2 = sum_t [Q_t + n_t (m_t - K)^2] and
// sum_x (x - K) = sum_t n_t (m_t - K), with m_t = S_t / n_t.  Those are plain
// sums (one fixed-order block reduction of three fp64 values), and
// mean = K + B/N, M2 = A - B^2/N.  K lies within a tile's spread of the mean,
// so the subtraction loses a few bits of fp64 at most.
__device__ void reduce_stats(const float* partials, int tiles, int c, int ch, double& n,
                             double& mean, double& m2) {
  __shared__ double red[3][FIN_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float n0 = tiles > 0 ? partials[ch] : 0.f;
  const float s0 = tiles > 0 ? partials[c + ch] : 0.f;
  double na = 0.0, aa = 0.0, ba = 0.0;
  double k = 0.0;
  bool have_k = false;
  for (int base = tid; base < tiles; base += FIN_THREADS * FIN_U) {
    float vn[FIN_U], vs[FIN_U], vq[FIN_U];
#pragma unroll
    for (int u = 0; u < FIN_U; ++u) {
      const int t = base + u * FIN_THREADS;
      const bool ok = t < tiles;
      const long row = static_cast<long>(t) * 3;
      vn[u] = ok ? partials[row * c + ch] : 0.f;
      vs[u] = ok ? partials[(row + 1) * c + ch] : 0.f;
      vq[u] = ok ? partials[(row + 2) * c + ch] : 0.f;
    }
    if (!have_k) {
      k = n0 > 0.f ? static_cast<double>(s0) / n0 : 0.0;
      have_k = true;
    }
#pragma unroll
    for (int u = 0; u < FIN_U; ++u) {
      if (vn[u] > 0.f) {
        const double nt = vn[u];
        const double d = static_cast<double>(vs[u]) / nt - k;
        na += nt;
        ba += nt * d;
        aa += static_cast<double>(vq[u]) + nt * d * d;
      }
    }
  }
  if (!have_k) k = n0 > 0.f ? static_cast<double>(s0) / n0 : 0.0;
  // xor butterfly: every lane ends with the same (commutative) sums
  for (int off = 1; off < 64; off <<= 1) {
    na += __shfl_xor(na, off, 64);
    aa += __shfl_xor(aa, off, 64);
    ba += __shfl_xor(ba, off, 64);
  }
  if (lane == 0) {
    red[0][wave] = na;
    red[1][wave] = aa;
    red[2][wave] = ba;
  }
  __syncthreads();
  n = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
  const double A = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
  const double B = (red[2][0] + red[2][1]) + (red[2][2] + red[2][3]);
  if (n > 0.0) {
    mean = k + B / n;
    m2 = fmax(A - B * B / n, 0.0);
  } else {
    mean = 0.0;
    m2 = 0.0;
  }
}

__global__ __launch_bounds__(FIN_THREADS) void bn_stats_finalize_kernel(
    const float* partials, int tiles, int c, long m, const float* gamma, const float* beta,
    float eps, float* scale, float* shift, float* mean_out, float* rstd_out, float* run_mean,
    float* run_var, float momentum) {
  const int ch = blockIdx.x;
  double n, mean, m2;
  reduce_stats(partials, tiles, c, ch, n, mean, m2);
  if (threadIdx.x != 0) return;
  (void)m;
  const double var = n > 0.0 ? m2 / n : 0.0;   // biased batch variance
  const double rstd = 1.0 / sqrt(var + static_cast<double>(eps));
  const double sc = static_cast<double>(gamma[ch]) * rstd;
  scale[ch] = static_cast<float>(sc);
  shift[ch] = static_cast<float>(static_cast<double>(beta[ch]) - mean * sc);
  mean_out[ch] = static_cast<float>(mean);
  rstd_out[ch] = static_cast<float>(rstd);
  if (run_mean != nullptr) {
    const double mom = momentum;
    const double unbiased = n > 1.0 ? var * n / (n - 1.0) : var;
    run_mean[ch] = static_cast<float>((1.0 - mom) * run_mean[ch] + mom * mean);
    run_var[ch] = static_cast<float>((1.0 - mom) * run_var[ch] + mom * unbiased);
  }
}

__global__ __launch_bounds__(FIN_THREADS) void bn_bwd_finalize_kernel(
    const float* partials, int tiles, int c, long m, const float* gamma, const float* mean,
    const float* rstd, float inv_k, float* dgamma, float* dbeta, float* ca, float* cb, float* cc) {
  const int ch = blockIdx.x;
  double sd, sdx;
  reduce_partials(partials, tiles, c, ch, sd, sdx);
  if (threadIdx.x != 0) return;
  (void)mean;
  dbeta[ch] += inv_k * static_cast<float>(sd);
  dgamma[ch] += inv_k * static_cast<float>(sdx);
  const double g = gamma[ch], r = rstd[ch], md = static_cast<double>(m);
  // dh = g*r*(d - sd/m - xhat*sdx/m), xhat = (h - mean)*r
  ca[ch] = static_cast<float>(g * r);
  cb[ch] = static_cast<float>(-g * r * r * sdx / md);
  cc[ch] = static_cast<float>(-g * r * sd / md);
}

template <typename T>
__global__ __launch_bounds__(256) void combine_fwd_kernel(const T* r, const T* h,
                                                          const float* scale, const float* shift,
                                                          T* y, long total8, int c8) {
  for (long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; i < total8;
       i += static_cast<long>(gridDim.x) * 256) {
    const int ch = static_cast<int>(i % c8) * 8;
    float rv[8], hv[8], o[8];
    Vec8<T>::load(r + i * 8, rv);
    Vec8<T>::load(h + i * 8, hv);
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = rv[j] + fmaf(scale[ch + j], hv[j], shift[ch + j]);
    Vec8<T>::store(y + i * 8, o);
  }
}

// x = v - (scale*h + shift): the reconstruction of a coupling input.
template <typename T>
__global__ __launch_bounds__(256) void combine_rec_kernel(const T* v, const T* h,
                                                          const float* scale, const float* shift,
                                                          T* x, long total8, int c8) {
  for (long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x; i < total8;
       i += static_cast<long>(gridDim.x) * 256) {
    const int ch = static_cast<int>(i % c8) * 8;
    float vv[8], hv[8], o[8];
    Vec8<T>::load(v + i * 8, vv);
    Vec8<T>::load(h + i * 8, hv);
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = vv[j] - fmaf(scale[ch + j], hv[j], shift[ch + j]);
    Vec8<T>::store(x + i * 8, o);
  }
}

// Each block owns rows [tile*rows_per_tile, ...) and writes one partial row.
template <typename T>
__global__ __launch_bounds__(256) void combine_bwd_kernel(const T* v, const T* h, const T* d,
                                                          const float* scale, const float* shift,
                                                          const float* mean, const float* rstd,
                                                          T* x, float* partials, long m, int c,
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
    float sc[8], sh[8], mu[8], rs[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      sc[j] = scale[ch + j];
      sh[j] = shift[ch + j];
      mu[j] = mean[ch + j];
      rs[j] = rstd[ch + j];
    }
    for (long row = row0 + rr; row < row1; row += rows_per_pass) {
      const long off = row * c + ch;
      float vv[8], hv[8], dv[8], o[8];
      Vec8<T>::load(v + off, vv);
      Vec8<T>::load(h + off, hv);
      Vec8<T>::load(d + off, dv);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        o[j] = vv[j] - fmaf(sc[j], hv[j], sh[j]);
        s1[j] += dv[j];
        s2[j] += dv[j] * ((hv[j] - mu[j]) * rs[j]);
      }
      Vec8<T>::store(x + off, o);
    }
  }
  // Fixed-order reduction over the rows_per_pass thread rows of each channel.
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

int ew_rows_per_tile(long m, int c) {
  const int rows_per_pass = 256 / (c / 8);
  long want = (m + 1023) / 1024;
  long rpt = ((want + rows_per_pass - 1) / rows_per_pass) * rows_per_pass;
  if (rpt < rows_per_pass) rpt = rows_per_pass;
  return static_cast<int>(rpt);
}

unsigned ew_grid(long total8) {
  long b = (total8 + 255) / 256;
  if (b > 65536) b = 65536;
  if (b < 1) b = 1;
  return static_cast<unsigned>(b);
}

}  // namespace bnk
using namespace bnk;

int ew_tiles(long m, int c) {
  const int rpt = ew_rows_per_tile(m, c);
  return static_cast<int>((m + rpt - 1) / rpt);
}

void bn_stats_finalize(const float* partials, int tiles, int c, long m, const float* gamma,
                       const float* beta, float eps, float* scale, float* shift, float* mean,
                       float* rstd, float* run_mean, float* run_var, float momentum,
                       hipStream_t st) {
  PETRA_LAUNCH(bn_stats_finalize_kernel, dim3(c), dim3(FIN_THREADS), 0, st, partials, tiles, c, m, gamma,
                     beta, eps, scale, shift, mean, rstd, run_mean, run_var, momentum);
}

void bn_bwd_finalize(const float* partials, int tiles, int c, long m, const float* gamma,
                     const float* mean, const float* rstd, float inv_k, float* dgamma,
                     float* dbeta, float* ca, float* cb, float* cc, hipStream_t st) {
  PETRA_LAUNCH(bn_bwd_finalize_kernel, dim3(c), dim3(FIN_THREADS), 0, st, partials, tiles, c, m, gamma,
                     mean, rstd, inv_k, dgamma, dbeta, ca, cb, cc);
}

void combine_fwd(int dtype, const void* r, const void* h, const float* scale, const float* shift,
                 void* y, long m, int c, hipStream_t st) {
  const long total8 = m * c / 8;
  if (dtype == DT_BF16)
    PETRA_LAUNCH(combine_fwd_kernel<bf16_t>, dim3(ew_grid(total8)), dim3(256), 0, st,
                       static_cast<const bf16_t*>(r), static_cast<const bf16_t*>(h), scale, shift,
                       static_cast<bf16_t*>(y), total8, c / 8);
  else
    PETRA_LAUNCH(combine_fwd_kernel<float>, dim3(ew_grid(total8)), dim3(256), 0, st,
                       static_cast<const float*>(r), static_cast<const float*>(h), scale, shift,
                       static_cast<float*>(y), total8, c / 8);
}

void combine_rec(int dtype, const void* v, const void* h, const float* scale, const float* shift,
                 void* x, long m, int c, hipStream_t st) {
  const long total8 = m * c / 8;
  if (dtype == DT_BF16)
    PETRA_LAUNCH(combine_rec_kernel<bf16_t>, dim3(ew_grid(total8)), dim3(256), 0, st,
                       static_cast<const bf16_t*>(v), static_cast<const bf16_t*>(h), scale, shift,
                       static_cast<bf16_t*>(x), total8, c / 8);
  else
    PETRA_LAUNCH(combine_rec_kernel<float>, dim3(ew_grid(total8)), dim3(256), 0, st,
                       static_cast<const float*>(v), static_cast<const float*>(h), scale, shift,
                       static_cast<float*>(x), total8, c / 8);
}

void combine_bwd(int dtype, const void* v, const void* h, const void* d, const float* scale,
                 const float* shift, const float* mean, const float* rstd, void* x,
                 float* partials, long m, int c, hipStream_t st) {
  const int rpt = ew_rows_per_tile(m, c);
  const int tiles = static_cast<int>((m + rpt - 1) / rpt);
  if (dtype == DT_BF16)
    PETRA_LAUNCH(combine_bwd_kernel<bf16_t>, dim3(tiles), dim3(256), 0, st,
                       static_cast<const bf16_t*>(v), static_cast<const bf16_t*>(h),
                       static_cast<const bf16_t*>(d), scale, shift, mean, rstd,
                       static_cast<bf16_t*>(x), partials, m, c, rpt);
  else
    PETRA_LAUNCH(combine_bwd_kernel<float>, dim3(tiles), dim3(256), 0, st,
                       static_cast<const float*>(v), static_cast<const float*>(h),
                       static_cast<const float*>(d), scale, shift, mean, rstd,
                       static_cast<float*>(x), partials, m, c, rpt);
}

}  // namespace petra
