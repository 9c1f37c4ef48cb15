// Implicit-GEMM convolution kernels for gfx950 (MFMA, wave64).
//
// Forward and input-gradient convolutions share one kernel: the input
// gradient of a stride-1 convolution is a forward convolution of the output
// gradient with the weights transposed to [C_in][R][S][C_out] and flipped in
// R and S (that copy is written by the weight-refresh kernel).
//
// GEMM view (NHWC activations, [C_out][K] weights with K = R*S*C_in):
//   rows    m = (n, p, q)           M = N*P*Q
//   columns o                        C_out
//   reduce  k = (r, s, c)            K = R*S*C_in
// A[m][k] is gathered on the fly from the input (zero outside the image,
// optional BN-apply + ReLU prologue of the layer below); B[k][o] is the
// weight row o.  A and B fragments go straight from global memory (L1/L2
// cached) into MFMA operand registers: an 8-wide run of k always lies in one
// filter tap because C_in is a multiple of 8.
//
// The weight gradient uses a second kernel whose reduction runs over m; both
// of its operands are staged through LDS transposed to k-contiguous rows, and
// the reduction is split over row chunks whose fp32 partial sums are reduced
// in a fixed order by wgrad_reduce (deterministic, no float atomics).
#include "common.h"
#include "kernels.h"

namespace petra {

namespace {

struct RowPos {
  int n, p, q;
  bool valid;
};

template <typename T>
__device__ __forceinline__ const T* src_pixel(const ConvArgs& a, int n, int ih, int iw, int c) {
  const long pix = (static_cast<long>(n) * a.h + ih) * a.w + iw;
  if (a.src2 != nullptr && c >= a.c_split)
    return static_cast<const T*>(a.src2) + pix * (a.c_in - a.c_split) + (c - a.c_split);
  return static_cast<const T*>(a.src) + pix * a.c_split + c;
}

// Gather 8 consecutive input channels of one im2col element group.
template <typename T, bool PRO>
__device__ __forceinline__ void gather_a(const ConvArgs& a, const RowPos& rp, bool kvalid, int fr,
                                         int fs, int c, Raw8<T>& f) {
  const int ih = rp.p * a.stride + fr - a.pad;
  const int iw = rp.q * a.stride + fs - a.pad;
  if (!(rp.valid && kvalid && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w)) {
    f.zero();
    return;
  }
  const T* ptr = src_pixel<T>(a, rp.n, ih, iw, c);
  f.load(ptr);
  if constexpr (PRO) {
    float v[8];
    f.to_f32(v);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = fmaxf(fmaf(a.pro_scale[c + j], v[j], a.pro_shift[c + j]), 0.f);
    f.from_f32(v);
  }
}

}  // namespace

// One workgroup = 4 waves computing a BM x BN output tile; the waves form a
// WAVES_M x (4 / WAVES_M) grid, each owning FM x FN 16x16 MFMA tiles.
template <typename T, int BM, int BN, int WAVES_M, int EP, bool PRO>
__global__ __launch_bounds__(256) void conv_gemm_kernel(ConvArgs a) {
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 16, FN = TN / 16;
  static_assert(FM >= 1 && FN >= 1 && TM % 16 == 0 && TN % 16 == 0, "tile");

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int lr = lane & 15, lg = lane >> 4;
  const int row_base = blockIdx.x * BM + wm * TM;
  const int col_base = blockIdx.y * BN + wn * TN;
  const int pq = a.p * a.q;

  RowPos rows[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int m = row_base + fm * 16 + lr;
    rows[fm].valid = m < a.m;
    const int mm = rows[fm].valid ? m : 0;
    rows[fm].n = mm / pq;
    const int rem = mm - rows[fm].n * pq;
    rows[fm].p = rem / a.q;
    rows[fm].q = rem - rows[fm].p * a.q;
  }
  const T* wt = static_cast<const T*>(a.wt);

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < a.k_tot; k0 += 32) {
    const int k = k0 + lg * 8;
    const bool kvalid = k < a.k_tot;
    const int kk = kvalid ? k : 0;
    const int tap = kk / a.c_in;
    const int c = kk - tap * a.c_in;
    const int fr = tap / a.s;
    const int fs = tap - fr * a.s;
    Frag<T> af[FM], bfr[FN];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      Raw8<T> r;
      gather_a<T, PRO>(a, rows[fm], kvalid, fr, fs, c, r);
      af[fm].set(r);
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int col = col_base + fn * 16 + lr;
      Raw8<T> r;
      if (kvalid && col < a.c_out)
        r.load(wt + static_cast<long>(col) * a.k_tot + k);
      else
        r.zero();
      bfr[fn].set(r);
    }
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma(af[fm], bfr[fn], acc[fm][fn]);
  }

  // Epilogue.  Lane (lr, lg) of tile (fm, fn) holds rows 4*lg + j, column lr.
  T* out = static_cast<T*>(a.out);
  float s1[FN], s2[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) s1[fn] = s2[fn] = 0.f;
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int col = col_base + fn * 16 + lr;
    const bool cvalid = col < a.c_out;
    float e_scale = 0.f, e_shift = 0.f, e_mean = 0.f, e_rstd = 0.f;
    if constexpr (EP == EP_MASK) {
      if (cvalid) {
        e_scale = a.ep_scale[col];
        e_shift = a.ep_shift[col];
        e_mean = a.ep_mean[col];
        e_rstd = a.ep_rstd[col];
      }
    }
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = row_base + fm * 16 + lg * 4 + j;
        if (!(cvalid && row < a.m)) continue;
        const long idx = static_cast<long>(row) * a.c_out + col;
        const float v = acc[fm][fn][j];
        if constexpr (EP == EP_STATS) {
          // statistics of the stored tensor, so BN normalises exactly what it reads back
          const float vs = quant(v, out);
          store1(out + idx, vs);
          s1[fn] += vs;
          s2[fn] += vs * vs;
        } else if constexpr (EP == EP_MASK) {
          const float hl = load1(static_cast<const T*>(a.ep_h) + idx);
          const float o = fmaf(e_scale, hl, e_shift);
          const float dz = quant(o > 0.f ? v : 0.f, out);
          store1(out + idx, dz);
          s1[fn] += dz;
          s2[fn] += dz * ((hl - e_mean) * e_rstd);
        } else {
          const float rv = load1(static_cast<const T*>(a.resid) + idx);
          store1(out + idx, rv + v);
        }
      }
    }
  }
  if constexpr (EP == EP_STATS || EP == EP_MASK) {
    __shared__ float red[WAVES_M][2][BN];
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const float t1 = sum_lane_groups(s1[fn]);
      const float t2 = sum_lane_groups(s2[fn]);
      if (lg == 0) {
        red[wm][0][wn * TN + fn * 16 + lr] = t1;
        red[wm][1][wn * TN + fn * 16 + lr] = t2;
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 2 * BN; i += 256) {
      const int which = i / BN, cl = i - which * BN;
      const int col = blockIdx.y * BN + cl;
      if (col >= a.c_out) continue;
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < WAVES_M; ++w) t += red[w][which][cl];
      a.partials[(static_cast<long>(blockIdx.x) * 2 + which) * a.c_out + col] = t;
    }
  }
}

// Weight gradient partials over one chunk of rows:
//   part[split][o][k] = sum_{m in chunk} dh[m][o] * A[m][k]
// BO x BK output tile, 4 waves in a 2 x 2 grid; rows advance 32 at a time.
template <typename T, int BO, int BK, bool PRO>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a) {
  constexpr int PITCH = 40;  // elements per LDS row: 32 rows of m + pad (16B-aligned rows)
  constexpr int FO = BO / 32, FK = BK / 32;
  __shared__ __attribute__((aligned(16))) T sA[BO * PITCH];
  __shared__ __attribute__((aligned(16))) T sB[BK * PITCH];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wo = wave & 1, wk = wave >> 1;
  const int lr = lane & 15, lg = lane >> 4;
  const int k0 = blockIdx.x * BK, o0 = blockIdx.y * BO;
  const int m_begin = blockIdx.z * a.rows_per_split;
  const int m_end = min(a.m, m_begin + a.rows_per_split);
  const int pq = a.p * a.q;
  const T* dh = static_cast<const T*>(a.dh);

  // Per-thread load roles (fixed over the loop).
  const int a_row = tid / (BO / 8), a_og = tid % (BO / 8);
  const bool a_active = tid < 32 * (BO / 8);
  const int b_row = tid / (BK / 8), b_kg = tid % (BK / 8);
  const bool b_active = tid < 32 * (BK / 8);
  const int kb = k0 + b_kg * 8;
  const bool kb_valid = kb < a.k_tot;
  const int kbb = kb_valid ? kb : 0;
  const int tap = kbb / a.c_in;
  const int cb = kbb - tap * a.c_in;
  const int fr = tap / a.s, fs = tap - fr * a.s;

  f32x4_t acc[FO][FK];
#pragma unroll
  for (int i = 0; i < FO; ++i)
#pragma unroll
    for (int j = 0; j < FK; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  ConvArgs ca;  // reuse the gather helper
  ca.src = a.src; ca.src2 = a.src2; ca.c_split = a.c_split;
  ca.pro_scale = a.pro_scale; ca.pro_shift = a.pro_shift;
  ca.h = a.h; ca.w = a.w; ca.c_in = a.c_in; ca.stride = a.stride; ca.pad = a.pad;

  for (int mb = m_begin; mb < m_end; mb += 32) {
    if (a_active) {
      const int m = mb + a_row;
      const int o = o0 + a_og * 8;
      Raw8<T> r;
      if (m < m_end && o < a.c_out)
        r.load(dh + static_cast<long>(m) * a.c_out + o);
      else
        r.zero();
#pragma unroll
      for (int j = 0; j < 8; ++j) r.put(j, &sA[(a_og * 8 + j) * PITCH + a_row]);
    }
    if (b_active) {
      const int m = mb + b_row;
      RowPos rp;
      rp.valid = m < m_end;
      const int mm = rp.valid ? m : 0;
      rp.n = mm / pq;
      const int rem = mm - rp.n * pq;
      rp.p = rem / a.q;
      rp.q = rem - rp.p * a.q;
      Raw8<T> r;
      gather_a<T, PRO>(ca, rp, kb_valid, fr, fs, cb, r);
#pragma unroll
      for (int j = 0; j < 8; ++j) r.put(j, &sB[(b_kg * 8 + j) * PITCH + b_row]);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < FO; ++i) {
      Frag<T> fa;
      fa.load(&sA[(wo * (BO / 2) + i * 16 + lr) * PITCH + lg * 8]);
#pragma unroll
      for (int j = 0; j < FK; ++j) {
        Frag<T> fb;
        fb.load(&sB[(wk * (BK / 2) + j * 16 + lr) * PITCH + lg * 8]);
        acc[i][j] = mfma(fa, fb, acc[i][j]);
      }
    }
    __syncthreads();
  }

  float* part = a.partials + static_cast<long>(blockIdx.z) * a.c_out * a.k_tot;
#pragma unroll
  for (int i = 0; i < FO; ++i)
#pragma unroll
    for (int j = 0; j < FK; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int o = o0 + wo * (BO / 2) + i * 16 + lg * 4 + e;
        const int k = k0 + wk * (BK / 2) + j * 16 + lr;
        if (o < a.c_out && k < a.k_tot) part[static_cast<long>(o) * a.k_tot + k] = acc[i][j][e];
      }
}

// grad[o*K + k] += inv_k * sum_split part[split][o][k]   (fixed split order)
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ part, int splits,
                                                           long numel, float inv_k,
                                                           float* __restrict__ grad) {
  const long i = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= numel) return;
  float s = 0.f;
  for (int t = 0; t < splits; ++t) s += part[static_cast<long>(t) * numel + i];
  grad[i] += inv_k * s;
}

// ---------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------

namespace {

template <typename T, int BN, int WM, int EP, bool PRO>
void launch_gemm(const ConvArgs& a, hipStream_t st) {
  constexpr int BM = 128;
  dim3 grid((a.m + BM - 1) / BM, (a.c_out + BN - 1) / BN);
  hipLaunchKernelGGL((conv_gemm_kernel<T, BM, BN, WM, EP, PRO>), grid, dim3(256), 0, st, a);
}

template <typename T, int EP, bool PRO>
void launch_gemm_tiles(const ConvArgs& a, hipStream_t st) {
  if (a.c_out <= 16)
    launch_gemm<T, 16, 4, EP, PRO>(a, st);
  else if (a.c_out <= 32)
    launch_gemm<T, 32, 4, EP, PRO>(a, st);
  else if (a.c_out <= 64)
    launch_gemm<T, 64, 2, EP, PRO>(a, st);
  else
    launch_gemm<T, 128, 2, EP, PRO>(a, st);
}

template <typename T>
void conv_gemm_t(const ConvArgs& a, int ep, hipStream_t st) {
  const bool pro = a.pro_scale != nullptr;
  if (ep == EP_STATS) {
    if (pro) launch_gemm_tiles<T, EP_STATS, true>(a, st);
    else launch_gemm_tiles<T, EP_STATS, false>(a, st);
  } else if (ep == EP_MASK) {
    launch_gemm_tiles<T, EP_MASK, false>(a, st);
  } else {
    launch_gemm_tiles<T, EP_RESID, false>(a, st);
  }
}

template <typename T, int BO, int BK>
void launch_wgrad_bk(const WgradArgs& a, hipStream_t st) {
  dim3 grid((a.k_tot + BK - 1) / BK, (a.c_out + BO - 1) / BO, a.splits);
  if (a.pro_scale != nullptr)
    hipLaunchKernelGGL((wgrad_kernel<T, BO, BK, true>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((wgrad_kernel<T, BO, BK, false>), grid, dim3(256), 0, st, a);
}

template <typename T>
void wgrad_t(const WgradArgs& a, hipStream_t st) {
  if (a.c_out <= 32)
    launch_wgrad_bk<T, 32, 64>(a, st);
  else
    launch_wgrad_bk<T, 64, 64>(a, st);
}

}  // namespace

void conv_gemm(int dtype, const ConvArgs& a, int ep, hipStream_t st) {
  if (dtype == DT_BF16)
    conv_gemm_t<bf16_t>(a, ep, st);
  else
    conv_gemm_t<float>(a, ep, st);
}

void conv_wgrad(int dtype, const WgradArgs& a, hipStream_t st) {
  if (dtype == DT_BF16)
    wgrad_t<bf16_t>(a, st);
  else
    wgrad_t<float>(a, st);
}

void wgrad_reduce(const float* part, int splits, long numel, float inv_k, float* grad,
                  hipStream_t st) {
  const long blocks = (numel + 255) / 256;
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                     part, splits, numel, inv_k, grad);
}

}  // namespace petra
