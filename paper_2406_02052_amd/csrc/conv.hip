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
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "prof.h"

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

// Prologue on 8 consecutive input channels c..c+7 of a loaded chunk r (hr: the
// same chunk of pro_h for PRO_BWD).  Tables t0..t3: scale, shift for PRO_RELU;
// ca, cb, cc, mean for PRO_BWD (LDS or global).  The result is rounded to T, as
// the materialised tensor would be.
template <typename T, int PRO>
__device__ __forceinline__ void pro8(Raw8<T>& r, const Raw8<T>& hr, const float* t0,
                                     const float* t1, const float* t2, const float* t3, int c) {
  if constexpr (PRO == PRO_NONE) return;
  float v[8];
  r.to_f32(v);
  if constexpr (PRO == PRO_RELU) {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = fmaxf(fmaf(t0[c + j], v[j], t1[c + j]), 0.f);
  } else {
    float h[8];
    hr.to_f32(h);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = fmaf(t0[c + j], v[j], fmaf(t1[c + j], h[j] - t3[c + j], t2[c + j]));
  }
  r.from_f32(v);
}

// Gather 8 consecutive input channels of one im2col element group.
template <typename T, int PRO>
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
  if constexpr (PRO == PRO_RELU) {
    pro8<T, PRO>(f, f, a.pro_scale, a.pro_shift, nullptr, nullptr, c);
  } else if constexpr (PRO == PRO_BWD) {
    Raw8<T> hr;
    hr.load(static_cast<const T*>(a.pro_h) + (ptr - static_cast<const T*>(a.src)));
    pro8<T, PRO>(f, hr, a.pro_ca, a.pro_cb, a.pro_cc, a.pro_mean, c);
  }
}

// Output-side operand of the weight gradient: with dh_h set, 8 channels o..o+7
// of the BN input gradient are formed from the loaded chunk (coefficients in
// registers: ca, cb, cc, mean), rounded to T as the materialised tensor would be.
template <typename T>
__device__ __forceinline__ void dh_bwd8(Raw8<T>& r, const T* hptr, const float (&k)[4][8]) {
  Raw8<T> hr;
  hr.load(hptr);
  float v[8], h[8];
  r.to_f32(v);
  hr.to_f32(h);
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = fmaf(k[0][j], v[j], fmaf(k[1][j], h[j] - k[3][j], k[2][j]));
  r.from_f32(v);
}

__device__ __forceinline__ void dh_coeffs(const WgradArgs& a, int o, float (&k)[4][8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const bool ok = a.dh_h != nullptr && o + j < a.c_out;
    k[0][j] = ok ? a.dh_ca[o + j] : 0.f;
    k[1][j] = ok ? a.dh_cb[o + j] : 0.f;
    k[2][j] = ok ? a.dh_cc[o + j] : 0.f;
    k[3][j] = ok ? a.dh_mean[o + j] : 0.f;
  }
}

// BN statistics of one output tile, mean-centred: per column the number of
// valid rows, their sum and the sum of squared deviations from the tile mean
// (of the values as stored in T), written to partials[tile][3][c_out].  Works
// on the MFMA accumulator layout: lane (lr, lg) of tile (fm, fn) holds column
// wn*TN + fn*16 + lr, rows fm*16 + lg*4 + j; valid(fm, j) says whether that row
// is a real output row.
template <typename T, int FM, int FN, int WAVES_M, int TN, int BN, typename Valid>
__device__ void tile_stats(const f32x4_t (&acc)[FM][FN], Valid valid, int wm, int wn, int lane,
                           int n0, int c_out, float* partials, int tile) {
  __shared__ float red[WAVES_M][3][BN];
  const int lr = lane & 15, lg = lane >> 4;
  const T* tag = nullptr;
  // Branch-free: invalid rows contribute zero (their weight vm is 0).
  float vm[FM][4], q[FM][FN][4];
  float cnt = 0.f;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      vm[fm][j] = valid(fm, j) ? 1.f : 0.f;
      cnt += vm[fm][j];
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) q[fm][fn][j] = vm[fm][j] * quant(acc[fm][fn][j], tag);
    }
  float sum[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    float t = 0.f;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int j = 0; j < 4; ++j) t += q[fm][fn][j];
    sum[fn] = t;
  }
  cnt = sum_lane_groups(cnt);
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    sum[fn] = sum_lane_groups(sum[fn]);
    if (lg == 0) {
      red[wm][0][wn * TN + fn * 16 + lr] = sum[fn];
      red[wm][1][wn * TN + fn * 16 + lr] = cnt;
    }
  }
  __syncthreads();
  float m2[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int cl = wn * TN + fn * 16 + lr;
    float S = 0.f, N = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES_M; ++w) {
      S += red[w][0][cl];
      N += red[w][1][cl];
    }
    const float mean = N > 0.f ? S / N : 0.f;
    float t = 0.f;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float d = q[fm][fn][j] - mean;
        t += vm[fm][j] * (d * d);
      }
    m2[fn] = sum_lane_groups(t);
    if (lg == 0) red[wm][2][wn * TN + fn * 16 + lr] = m2[fn];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < BN; i += blockDim.x) {
    const int col = n0 + i;
    if (col >= c_out) continue;
    float S = 0.f, N = 0.f, Q = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES_M; ++w) {
      S += red[w][0][i];
      N += red[w][1][i];
      Q += red[w][2][i];
    }
    partials[(static_cast<long>(tile) * 3 + 0) * c_out + col] = N;
    partials[(static_cast<long>(tile) * 3 + 1) * c_out + col] = S;
    partials[(static_cast<long>(tile) * 3 + 2) * c_out + col] = Q;
  }
}

}  // namespace

// Epilogue slice in LDS: column-major, 16 rows + 4 pad per column, so every
// lane writes its four accumulator rows with one aligned 16-byte store
// (conflict-free across the 16 lanes of a store pass).
constexpr int EP_RP = 20;

// One workgroup = 4 waves computing a BM x BN output tile; the waves form a
// WAVES_M x (4 / WAVES_M) grid, each owning FM x FN 16x16 MFMA tiles.
template <typename T, int BM, int BN, int WAVES_M, int EP, int PRO>
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
      }
    }
    if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
      if (cvalid) {
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
          store1(out + idx, v);
        } else if constexpr (EP == EP_MASK) {
          const float hl = load1(static_cast<const T*>(a.ep_h) + idx);
          const float o = fmaf(e_scale, hl, e_shift);
          const float dz = quant(o > 0.f ? v : 0.f, out);
          store1(out + idx, dz);
          s1[fn] += dz;
          s2[fn] += dz * ((hl - e_mean) * e_rstd);
        } else {
          const float rv = a.resid != nullptr ? load1(static_cast<const T*>(a.resid) + idx) : 0.f;
          store1(out + idx, rv + v);
          if constexpr (EP == EP_RESID_STATS) {
            const float g = quant(rv + v, out);
            const float hl = load1(static_cast<const T*>(a.ep_h) + idx);
            s1[fn] += g;
            s2[fn] += g * ((hl - e_mean) * e_rstd);
          }
        }
      }
    }
  }
  if constexpr (EP == EP_STATS) {
    // statistics of the stored tensor, so BN normalises exactly what it reads back
    tile_stats<T, FM, FN, WAVES_M, TN, BN>(
        acc, [&](int fm, int j) { return row_base + fm * 16 + lg * 4 + j < a.m; }, wm, wn, lane,
        blockIdx.y * BN, a.c_out, a.partials, blockIdx.x);
  }
  if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
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

// Staged variant for bf16 with C_in a multiple of 32 (every stage conv of the
// bf16 workloads).  Per 32-wide reduction step (one filter tap, 32 input
// channels) all 256 threads gather the A tile (im2col rows, prologue applied)
// and the B tile into registers one step ahead, park them in a double-buffered
// LDS stage, and the 4 waves feed MFMA from LDS.  The epilogue goes through LDS
// one 16-row slice per wave at a time so that every lane stores 16 contiguous
// bytes of one output row.
template <int BM, int BN, int WAVES_M, int EP, int PRO>
__global__ __launch_bounds__(256) void conv_staged_kernel(ConvArgs a) {
  using T = bf16_t;
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 16, FN = TN / 16;
  constexpr int PITCH = 40;                  // bf16 per LDS row: 32 k + 8 pad (80 B)
  constexpr int A_CHUNKS = BM * 4 / 256;     // 16-byte A chunks per thread and step
  constexpr int B_CHUNKS = (BN * 4 + 255) / 256;  // 16-byte B chunks per thread and step
  static_assert(BM * 4 % 256 == 0, "tile");
  constexpr int STAGE_ELEMS = (BM + BN) * PITCH;
  constexpr int EPI_FLOATS = 4 * TN * EP_RP;
  constexpr int LDS_BYTES = (2 * STAGE_ELEMS * 2 > EPI_FLOATS * 4) ? 2 * STAGE_ELEMS * 2 : EPI_FLOATS * 4;
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  __shared__ float pro_tab[PRO == PRO_BWD ? 4 : 2][512];
  __shared__ float red[WAVES_M][2][BN];

  T* stage_base = reinterpret_cast<T*>(lds);
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int lr = lane & 15, lg = lane >> 4;
  const int m0 = blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int pq = a.p * a.q;
  const int csteps = a.c_in / 32;
  const int steps = a.r * a.s * csteps;

  if constexpr (PRO == PRO_RELU) {
    for (int i = tid; i < a.c_in; i += 256) {
      pro_tab[0][i] = a.pro_scale[i];
      pro_tab[1][i] = a.pro_shift[i];
    }
  } else if constexpr (PRO == PRO_BWD) {
    for (int i = tid; i < a.c_in; i += 256) {
      pro_tab[0][i] = a.pro_ca[i];
      pro_tab[1][i] = a.pro_cb[i];
      pro_tab[2][i] = a.pro_cc[i];
      pro_tab[3][i] = a.pro_mean[i];
    }
  }

  // Fixed per-thread load roles.
  int a_row[A_CHUNKS], a_sub[A_CHUNKS], a_ih0[A_CHUNKS], a_iw0[A_CHUNKS];
  long a_pix0[A_CHUNKS];
  bool a_ok[A_CHUNKS];
#pragma unroll
  for (int i = 0; i < A_CHUNKS; ++i) {
    const int q = tid + 256 * i;
    a_row[i] = q >> 2;
    a_sub[i] = q & 3;
    const int m = m0 + a_row[i];
    a_ok[i] = m < a.m;
    const int mm = a_ok[i] ? m : 0;
    const int n = mm / pq;
    const int rem = mm - n * pq;
    const int pp = rem / a.q;
    const int qq = rem - pp * a.q;
    a_ih0[i] = pp * a.stride - a.pad;
    a_iw0[i] = qq * a.stride - a.pad;
    a_pix0[i] = static_cast<long>(n) * a.h * a.w;
  }
  int b_col[B_CHUNKS], b_sub[B_CHUNKS];
  bool b_in[B_CHUNKS], b_ok[B_CHUNKS];
#pragma unroll
  for (int i = 0; i < B_CHUNKS; ++i) {
    const int q = tid + 256 * i;
    b_col[i] = q >> 2;
    b_sub[i] = q & 3;
    b_in[i] = q < BN * 4;
    b_ok[i] = b_in[i] && (n0 + b_col[i]) < a.c_out;
  }
  // Buffer resources: rows outside the image and columns past c_out load zeros
  // without branches, so the next step's loads stay in flight.
  const long in_bytes = static_cast<long>(a.n) * a.h * a.w * a.c_in * 2;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_proh = make_rsrc(PRO == PRO_BWD ? a.pro_h : a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_wt = make_rsrc(a.wt, static_cast<long>(a.c_out) * a.k_tot * 2);
  if constexpr (PRO != PRO_NONE) __syncthreads();

  Raw8<T> ra[A_CHUNKS], rb[B_CHUNKS];
  Raw8<T> rah[PRO == PRO_BWD ? A_CHUNKS : 1];
  uint32_t avalid = 0;
  int step_c0 = 0;
  auto load_step = [&](int step) {
    const int tap = step / csteps;
    const int c0 = (step - tap * csteps) * 32;
    const int fr = tap / a.s, fs = tap - fr * a.s;
    step_c0 = c0;
    avalid = 0;
#pragma unroll
    for (int i = 0; i < A_CHUNKS; ++i) {
      const int ih = a_ih0[i] + fr, iw = a_iw0[i] + fs;
      const int c = c0 + a_sub[i] * 8;
      const bool ok = a_ok[i] && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
      const uint32_t off =
          ok ? static_cast<uint32_t>(((a_pix0[i] + static_cast<long>(ih) * a.w + iw) * a.c_in + c) * 2) : BUF_OOB;
      ra[i].set(buf_load16(r_src, off));
      if constexpr (PRO == PRO_BWD) rah[i].set(buf_load16(r_proh, off));
      avalid |= ok ? 1u << i : 0u;
    }
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i) {
      const uint32_t off =
          b_ok[i] ? static_cast<uint32_t>(((n0 + b_col[i]) * a.k_tot + tap * a.c_in + c0 + b_sub[i] * 8) * 2)
                  : BUF_OOB;
      rb[i].set(buf_load16(r_wt, off));
    }
  };
  // prologue of the loaded A chunks (padding stays zero)
  auto pro_step = [&]() {
    if constexpr (PRO != PRO_NONE) {
#pragma unroll
      for (int i = 0; i < A_CHUNKS; ++i) {
        pro8<T, PRO>(ra[i], rah[PRO == PRO_BWD ? i : 0], pro_tab[0], pro_tab[1],
                     pro_tab[PRO == PRO_BWD ? 2 : 0], pro_tab[PRO == PRO_BWD ? 3 : 0],
                     step_c0 + a_sub[i] * 8);
        if (!((avalid >> i) & 1u)) ra[i].zero();
      }
    }
  };
  auto park = [&](int buf) {
    T* sA = stage_base + buf * STAGE_ELEMS;
    T* sB = sA + BM * PITCH;
#pragma unroll
    for (int i = 0; i < A_CHUNKS; ++i)
      *reinterpret_cast<uint4*>(sA + a_row[i] * PITCH + a_sub[i] * 8) =
          make_uint4(ra[i].w[0], ra[i].w[1], ra[i].w[2], ra[i].w[3]);
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i)
      if (b_in[i])
        *reinterpret_cast<uint4*>(sB + b_col[i] * PITCH + b_sub[i] * 8) =
            make_uint4(rb[i].w[0], rb[i].w[1], rb[i].w[2], rb[i].w[3]);
  };

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  load_step(0);
  pro_step();
  park(0);
  __syncthreads();
  for (int step = 0; step < steps; ++step) {
    const int buf = step & 1;
    if (step + 1 < steps) load_step(step + 1);
    const T* sA = stage_base + buf * STAGE_ELEMS;
    const T* sB = sA + BM * PITCH;
    Frag<T> af[FM], bfr[FN];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) af[fm].load(sA + (wm * TM + fm * 16 + lr) * PITCH + lg * 8);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) bfr[fn].load(sB + (wn * TN + fn * 16 + lr) * PITCH + lg * 8);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma(af[fm], bfr[fn], acc[fm][fn]);
    if (step + 1 < steps) {
      pro_step();
      park(buf ^ 1);
    }
    __syncthreads();
  }

  if constexpr (EP == EP_STATS) {
    tile_stats<T, FM, FN, WAVES_M, TN, BN>(
        acc, [&](int fm, int j) { return m0 + wm * TM + fm * 16 + lg * 4 + j < a.m; }, wm, wn,
        lane, n0, a.c_out, a.partials, blockIdx.x);
  }
  // Epilogue: per 16-row slice, stage fp32 results of each wave in LDS
  // (column-major, one 16-byte store per fragment), then each lane handles 8
  // consecutive columns of one row.
  float* ep = reinterpret_cast<float*>(lds) + wave * TN * EP_RP;
  constexpr int CG = TN / 8;                  // column groups per slice row
  constexpr int TASKS = 16 * CG;              // (row, group) tasks per slice
  const int my_cg = lane % CG;
  const int col = n0 + wn * TN + my_cg * 8;
  const bool cvalid = col < a.c_out;
  float s1[8], s2[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) s1[j] = s2[j] = 0.f;
  float es[8], esh[8], emu[8], ers[8];
  if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      es[j] = cvalid && EP == EP_MASK ? a.ep_scale[col + j] : 0.f;
      esh[j] = cvalid && EP == EP_MASK ? a.ep_shift[col + j] : 0.f;
      emu[j] = cvalid ? a.ep_mean[col + j] : 0.f;
      ers[j] = cvalid ? a.ep_rstd[col + j] : 0.f;
    }
  }
  T* out = static_cast<T*>(a.out);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
      *reinterpret_cast<f32x4_t*>(ep + (fn * 16 + lr) * EP_RP + lg * 4) = acc[fm][fn];
    __syncthreads();
    for (int t = lane; t < TASKS; t += 64) {
      const int rr = t / CG;
      const int row = m0 + wm * TM + fm * 16 + rr;
      if (!(cvalid && row < a.m)) continue;
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = ep[(my_cg * 8 + j) * EP_RP + rr];
      const long idx = static_cast<long>(row) * a.c_out + col;
      Raw8<T> o;
      if constexpr (EP == EP_STATS) {
        o.from_f32(v);
      } else if constexpr (EP == EP_MASK) {
        Raw8<T> hr;
        hr.load(static_cast<const T*>(a.ep_h) + idx);
        float hl[8];
        hr.to_f32(hl);
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = fmaf(es[j], hl[j], esh[j]) > 0.f ? v[j] : 0.f;
        o.from_f32(v);
        o.to_f32(v);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          s1[j] += v[j];
          s2[j] += v[j] * ((hl[j] - emu[j]) * ers[j]);
        }
      } else {
        if (a.resid != nullptr) {  // without a residual the epilogue is a plain store
          Raw8<T> rr8;
          rr8.load(static_cast<const T*>(a.resid) + idx);
          float rv[8];
          rr8.to_f32(rv);
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] += rv[j];
        }
        o.from_f32(v);
        if constexpr (EP == EP_RESID_STATS) {  // BN-backward partials of the stored values
          Raw8<T> hr;
          hr.load(static_cast<const T*>(a.ep_h) + idx);
          float hl[8];
          hr.to_f32(hl);
          o.to_f32(v);
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            s1[j] += v[j];
            s2[j] += v[j] * ((hl[j] - emu[j]) * ers[j]);
          }
        }
      }
      *reinterpret_cast<uint4*>(out + idx) = make_uint4(o.w[0], o.w[1], o.w[2], o.w[3]);
    }
    __syncthreads();
  }
  if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
    // lanes with the same column group: lane % CG equal -> xor over the higher lane bits
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      for (int off = CG; off < 64; off <<= 1) {
        s1[j] += __shfl_xor(s1[j], off, 64);
        s2[j] += __shfl_xor(s2[j], off, 64);
      }
    }
    if (lane < CG) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        red[wm][0][wn * TN + lane * 8 + j] = s1[j];
        red[wm][1][wn * TN + lane * 8 + j] = s2[j];
      }
    }
    __syncthreads();
    for (int i = tid; i < 2 * BN; i += 256) {
      const int which = i / BN, cl = i - which * BN;
      const int c = n0 + cl;
      if (c >= a.c_out) continue;
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < WAVES_M; ++w) t += red[w][which][cl];
      a.partials[(static_cast<long>(blockIdx.x) * 2 + which) * a.c_out + c] = t;
    }
  }
}

// Epilogue operands of one lane of epilogue_cp (the pre-BN tensor of the BN
// below, the residual), loaded at the same offsets; a kernel that knows its
// tile from the start issues them with its first operand loads, so their
// latency hides behind the MFMAs instead of stalling the epilogue.
template <int FM, int FN>
struct EpiOps {
  u32x2_t h[FM][FN], r[FM][FN];
};

template <int TW, int FM, int FN, int TM, int TN, int EP>
__device__ __forceinline__ void epilogue_load(EpiOps<FM, FN>& o, const ConvArgs& a, int img,
                                              int p0, int q0, int n0, int wm, int wn, int lane) {
  constexpr bool GRAD = EP == EP_MASK || EP == EP_RESID_STATS;
  constexpr bool RES = EP == EP_RESID || EP == EP_RESID_STATS;
  if constexpr (GRAD || RES) {
    const int lr = lane & 15, lg = lane >> 4;
    const long out_bytes = static_cast<long>(a.m) * a.c_out * 2;
    const __amdgpu_buffer_rsrc_t r_eph = make_rsrc(a.ep_h != nullptr ? a.ep_h : a.out, out_bytes);
    const __amdgpu_buffer_rsrc_t r_res = make_rsrc(a.resid != nullptr ? a.resid : a.out,
                                                   a.resid != nullptr ? out_bytes : 0);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int i = wm * TM + fm * 16 + lr;
      const int ph = i / TW, pw = i - ph * TW;
      const bool vm = p0 + ph < a.h && q0 + pw < a.w;
      const long pix = (static_cast<long>(img) * a.h + p0 + ph) * a.w + q0 + pw;
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int c0 = n0 + wn * TN + fn * 16 + lg * 4;
        const uint32_t boff =
            vm && c0 < a.c_out ? static_cast<uint32_t>((pix * a.c_out + c0) * 2) : BUF_OOB;
        if constexpr (GRAD) o.h[fm][fn] = buf_load8(r_eph, boff);
        if constexpr (RES) o.r[fm][fn] = buf_load8(r_res, boff);
      }
    }
  }
}

// Epilogue for accumulators issued as D[cout][pixel] (the MFMA's A operand is
// the weight fragment): lane (lr, lg) of fragment (fm, fn) holds output channels
// n0 + wn*TN + fn*16 + lg*4 + e of tile pixel wm*TM + fm*16 + lr, pixel i of the
// TH x TW tile at (p0 + i / TW, q0 + i % TW) of image img.  Each lane stores its
// 4 channels directly (8 bytes, buffer store: pixels past the image are
// dropped); BN statistics are shifted sums per lane, summed over the 16 pixel
// lanes with DPP and over the WAVES_M waves in LDS, written as partial row
// blockIdx.x.  Epilogues as in conv_gemm_kernel.
template <int TW, int FM, int FN, int WAVES_M, int TM, int TN, int BN, int EP>
__device__ __forceinline__ void epilogue_cp(const f32x4_t (&acc)[FM][FN], const ConvArgs& a,
                                            int img, int p0, int q0, int n0, int wm, int wn,
                                            int lane, int tid, int nthreads,
                                            float (*red)[3][BN],
                                            const EpiOps<FM, FN>* pre = nullptr) {
  const int lr = lane & 15, lg = lane >> 4;
  const long out_bytes = static_cast<long>(a.m) * a.c_out * 2;
  const __amdgpu_buffer_rsrc_t r_out = make_rsrc(a.out, out_bytes);
  const __amdgpu_buffer_rsrc_t r_eph = make_rsrc(a.ep_h != nullptr ? a.ep_h : a.out, out_bytes);
  const __amdgpu_buffer_rsrc_t r_res = make_rsrc(a.resid != nullptr ? a.resid : a.out,
                                                 a.resid != nullptr ? out_bytes : 0);
  constexpr bool STATS = EP == EP_STATS;
  constexpr bool GRAD = EP == EP_MASK || EP == EP_RESID_STATS;
  float es[FN][4], esh[FN][4], emu[FN][4], ers[FN][4];
  bool cok[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int c0 = n0 + wn * TN + fn * 16 + lg * 4;
    cok[fn] = c0 < a.c_out;   // c_out is a multiple of 8 and of 4
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      es[fn][e] = esh[fn][e] = emu[fn][e] = ers[fn][e] = 0.f;
      if constexpr (GRAD) {
        if (cok[fn]) {
          es[fn][e] = EP == EP_MASK ? a.ep_scale[c0 + e] : 0.f;
          esh[fn][e] = EP == EP_MASK ? a.ep_shift[c0 + e] : 0.f;
          emu[fn][e] = a.ep_mean[c0 + e];
          ers[fn][e] = a.ep_rstd[c0 + e];
        }
      }
    }
  }
  float sa[FN][4], sb[FN][4], kk[FN][4];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn)
#pragma unroll
    for (int e = 0; e < 4; ++e) sa[fn][e] = sb[fn][e] = kk[fn][e] = 0.f;
  float nv = 0.f;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int i = wm * TM + fm * 16 + lr;
    const int ph = i / TW, pw = i - ph * TW;
    const bool vm = p0 + ph < a.h && q0 + pw < a.w;
    nv += vm ? 1.f : 0.f;
    const long pix = (static_cast<long>(img) * a.h + p0 + ph) * a.w + q0 + pw;
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const bool ok = vm && cok[fn];
      const uint32_t boff =
          ok ? static_cast<uint32_t>((pix * a.c_out + n0 + wn * TN + fn * 16 + lg * 4) * 2) : BUF_OOB;
      float v[4] = {acc[fm][fn][0], acc[fm][fn][1], acc[fm][fn][2], acc[fm][fn][3]};
      float hl[4] = {0.f, 0.f, 0.f, 0.f};
      if constexpr (GRAD) {
        const u32x2_t hw = pre != nullptr ? pre->h[fm][fn] : buf_load8(r_eph, boff);
        hl[0] = __uint_as_float(hw.x << 16); hl[1] = __uint_as_float(hw.x & 0xffff0000u);
        hl[2] = __uint_as_float(hw.y << 16); hl[3] = __uint_as_float(hw.y & 0xffff0000u);
      }
      if constexpr (EP == EP_RESID || EP == EP_RESID_STATS) {
        // a null residual reads zeros
        const u32x2_t rw = pre != nullptr ? pre->r[fm][fn] : buf_load8(r_res, boff);
        v[0] += __uint_as_float(rw.x << 16); v[1] += __uint_as_float(rw.x & 0xffff0000u);
        v[2] += __uint_as_float(rw.y << 16); v[3] += __uint_as_float(rw.y & 0xffff0000u);
      }
      if constexpr (EP == EP_MASK) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = fmaf(es[fn][e], hl[e], esh[fn][e]) > 0.f ? v[e] : 0.f;
      }
      const uint32_t w0 = pack_bf16x2(v[0], v[1]), w1 = pack_bf16x2(v[2], v[3]);
      buf_store8(u32x2_t{w0, w1}, r_out, boff);
      // statistics of the stored values
      v[0] = __uint_as_float(w0 << 16); v[1] = __uint_as_float(w0 & 0xffff0000u);
      v[2] = __uint_as_float(w1 << 16); v[3] = __uint_as_float(w1 & 0xffff0000u);
      if constexpr (STATS) {
        if (fm == 0) {
          // shift per channel: the stored value of this wave's first pixel
#pragma unroll
          for (int e = 0; e < 4; ++e) kk[fn][e] = __shfl(v[e], lane & 48, 64);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float d = vm ? v[e] - kk[fn][e] : 0.f;
          sa[fn][e] += d;
          sb[fn][e] = fmaf(d, d, sb[fn][e]);
        }
      } else if constexpr (GRAD) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float g = vm ? v[e] : 0.f;
          sa[fn][e] += g;
          sb[fn][e] += g * ((hl[e] - emu[fn][e]) * ers[fn][e]);
        }
      }
    }
  }
  if constexpr (STATS || GRAD) {
    const float n16 = sum16(nv);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = sum16(sa[fn][e]), y = sum16(sb[fn][e]);
        if (lr == 0) {
          const int c = wn * TN + fn * 16 + lg * 4 + e;
          if constexpr (STATS) {
            const float md = n16 > 0.f ? x / n16 : 0.f;
            red[wm][0][c] = n16;
            red[wm][1][c] = kk[fn][e] + md;                            // mean
            red[wm][2][c] = n16 > 0.f ? fmaxf(y - x * md, 0.f) : 0.f;  // centred M2
          } else {
            red[wm][1][c] = x;
            red[wm][2][c] = y;
          }
        }
      }
    __syncthreads();
    for (int c = tid; c < BN; c += nthreads) {
      const int col = n0 + c;
      if (col >= a.c_out) continue;
      float* pr = a.partials;
      const long row = static_cast<long>(blockIdx.x);
      if constexpr (STATS) {
        float n = 0.f, mean = 0.f, m2 = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES_M; ++w) {
          const float nb = red[w][0][c];
          if (nb > 0.f) {
            const float nn = n + nb, rb = nb / nn, d = red[w][1][c] - mean;
            mean += d * rb;
            m2 += red[w][2][c] + d * d * n * rb;
            n = nn;
          }
        }
        pr[(row * 3 + 0) * a.c_out + col] = n;
        pr[(row * 3 + 1) * a.c_out + col] = n * mean;
        pr[(row * 3 + 2) * a.c_out + col] = m2;
      } else {
        float t1 = 0.f, t2 = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES_M; ++w) {
          t1 += red[w][1][c];
          t2 += red[w][2][c];
        }
        pr[(row * 2 + 0) * a.c_out + col] = t1;
        pr[(row * 2 + 1) * a.c_out + col] = t2;
      }
    }
  }
}

// Halo-tile variant for 3x3 / stride 1 / pad 1 bf16 convolutions with C_in a
// multiple of 32.  A workgroup owns a TH x TW patch of output pixels of one
// image; per 32-channel chunk it loads the (TH+2) x (TW+2) input patch once into
// LDS (BN-apply + ReLU prologue applied there, once per element, zero padding
// kept zero) and runs the 9 taps from LDS by shifting the pixel index, while the
// 32-channel weight slab of each (chunk, tap) step streams through a double
// buffer.  The next chunk's patch and the next slab are fetched into registers
// one step ahead.  HB = number of patch buffers (1 when there is one chunk).
// FB (C_in == 32, a single chunk): all nine slabs are staged with the patch up
// front, so the nine taps run from LDS behind a single barrier.
template <int TH, int TW, int BN, int WAVES_M, int HB, int EP, int PRO, bool FB>
__global__ __launch_bounds__(256) void conv_halo_kernel(ConvArgs a) {
  using T = bf16_t;
  constexpr int BM = TH * TW;
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 16, FN = TN / 16;
  static_assert(TM % 16 == 0 && TN % 16 == 0, "tile");
  constexpr int HTH = TH + 2, HTW = TW + 2, HPIX = HTH * HTW;
  constexpr int HP = 40;                              // bf16 per patch pixel (32 + pad)
  static_assert(!FB || HB == 1, "a single chunk has one patch buffer");
  constexpr int NSLAB = FB ? 9 : 2;
  constexpr int H_CHUNKS = (HPIX * 4 + 255) / 256;    // 16-byte patch chunks per thread
  constexpr int B_CHUNKS = ((FB ? 9 : 1) * BN * 4 + 255) / 256;
  // weight slab rows of 64 bytes (32 bf16), the four 16-byte chunks permuted
  // by bits 1-2 of the row: conflict-free fragment reads
  constexpr int PATCH = HPIX * HP;
  constexpr int SLAB = BN * 32;
  constexpr int MAIN_BYTES = (HB * PATCH + NSLAB * SLAB) * 2;
  constexpr int LDS_BYTES = MAIN_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  __shared__ float pro_tab[PRO == PRO_BWD ? 4 : 2][512];
  __shared__ float red3[WAVES_M][3][BN];

  T* patch_base = reinterpret_cast<T*>(lds);
  T* slab_base = patch_base + HB * PATCH;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int lr = lane & 15, lg = lane >> 4;
  const int w_off = lr * 32 + ((lg ^ ((lr >> 1) & 3)) * 8);   // weight fragment rows
  const int tiles_x = (a.w + TW - 1) / TW, tiles_y = (a.h + TH - 1) / TH;
  const int tx = blockIdx.x % tiles_x;
  const int ty = (blockIdx.x / tiles_x) % tiles_y;
  const int img = blockIdx.x / (tiles_x * tiles_y);
  const int p0 = ty * TH, q0 = tx * TW;
  const int n0 = blockIdx.y * BN;
  const int chunks = a.c_in / 32;
  const int steps = chunks * 9;
  const long img_base = static_cast<long>(img) * a.h * a.w;

  // Operands come through buffer resources: padding and columns past c_out
  // load as zeros without branches, so the next chunk's loads stay in flight
  // while the current one is multiplied.
  const __amdgpu_buffer_rsrc_t r_src =
      make_rsrc(a.src, static_cast<long>(a.n) * a.h * a.w * a.c_in * 2);
  const __amdgpu_buffer_rsrc_t r_proh =
      make_rsrc(PRO == PRO_BWD ? a.pro_h : a.src, static_cast<long>(a.n) * a.h * a.w * a.c_in * 2);
  const __amdgpu_buffer_rsrc_t r_wt = make_rsrc(a.wt, static_cast<long>(a.c_out) * a.k_tot * 2);
  Raw8<T> rh[H_CHUNKS], rb[B_CHUNKS];
  Raw8<T> rhh[PRO == PRO_BWD ? H_CHUNKS : 1];   // pro_h at the patch positions
  uint32_t hvalid = 0;   // bit i: patch chunk i lies inside the image
  auto load_patch = [&](int chunk) {
    const int c0 = chunk * 32;
    hvalid = 0;
#pragma unroll
    for (int i = 0; i < H_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int hp = q >> 2, sub = q & 3;
      const int hy = hp / HTW, hx = hp - hy * HTW;
      const int ih = p0 - 1 + hy, iw = q0 - 1 + hx;
      const bool ok = hp < HPIX && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
      const uint32_t off =
          ok ? static_cast<uint32_t>(((img_base + static_cast<long>(ih) * a.w + iw) * a.c_in + c0 + sub * 8) * 2)
             : BUF_OOB;
      rh[i].set(buf_load16(r_src, off));
      if constexpr (PRO == PRO_BWD) rhh[i].set(buf_load16(r_proh, off));
      hvalid |= ok ? 1u << i : 0u;
    }
  };
  // Prologue on the loaded patch; padding stays zero.
  auto pro_patch = [&](int chunk) {
    if constexpr (PRO != PRO_NONE) {
#pragma unroll
      for (int i = 0; i < H_CHUNKS; ++i) {
        const int c = chunk * 32 + ((tid + 256 * i) & 3) * 8;
        pro8<T, PRO>(rh[i], rhh[PRO == PRO_BWD ? i : 0], pro_tab[0], pro_tab[1],
                     pro_tab[PRO == PRO_BWD ? 2 : 0], pro_tab[PRO == PRO_BWD ? 3 : 0], c);
        if (!((hvalid >> i) & 1u)) rh[i].zero();
      }
    }
  };
  auto park_patch = [&](int buf) {
    T* dst = patch_base + buf * PATCH;
#pragma unroll
    for (int i = 0; i < H_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int hp = q >> 2, sub = q & 3;
      if (hp < HPIX)
        *reinterpret_cast<uint4*>(dst + hp * HP + sub * 8) = make_uint4(rh[i].w[0], rh[i].w[1], rh[i].w[2], rh[i].w[3]);
    }
  };
  // One (chunk, tap) slab, or with FB all nine taps of chunk 0 (slab t = tap t).
  auto load_slab = [&](int step) {
    const int chunk = step / 9, tap0 = step - chunk * 9;
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int tap = FB ? q / (BN * 4) : tap0;
      const int rem = FB ? q - (q / (BN * 4)) * (BN * 4) : q;
      const int col = rem >> 2, sub = rem & 3;
      const bool ok = q < (FB ? 9 : 1) * BN * 4 && n0 + col < a.c_out;
      const uint32_t off =
          ok ? static_cast<uint32_t>(((n0 + col) * a.k_tot + tap * a.c_in + chunk * 32 + sub * 8) * 2) : BUF_OOB;
      rb[i].set(buf_load16(r_wt, off));
    }
  };
  auto park_slab = [&](int buf) {
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      if (q >= (FB ? 9 : 1) * BN * 4) continue;
      const int tap = FB ? q / (BN * 4) : 0;
      const int rem = q - tap * (BN * 4);
      T* dst = slab_base + (FB ? tap : buf) * SLAB;
      const int row = rem >> 2, sub = rem & 3;
      *reinterpret_cast<uint4*>(dst + row * 32 + ((sub ^ ((row >> 1) & 3)) * 8)) =
          make_uint4(rb[i].w[0], rb[i].w[1], rb[i].w[2], rb[i].w[3]);
    }
  };

  // Patch-pixel offset of each MFMA row this lane feeds (tap (0,0)).
  int rowpix[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int i = wm * TM + fm * 16 + lr;
    const int ph = i / TW, pw = i - ph * TW;
    rowpix[fm] = ph * HTW + pw;
  }

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Operand loads go out first, then this tile's epilogue operands; the
  // prologue table is fetched while they fly.
  load_patch(0);
  load_slab(0);
  EpiOps<FM, FN> epi;
  epilogue_load<TW, FM, FN, TM, TN, EP>(epi, a, img, p0, q0, n0, wm, wn, lane);
  if constexpr (PRO == PRO_RELU) {
    for (int i = tid; i < a.c_in; i += 256) {
      pro_tab[0][i] = a.pro_scale[i];
      pro_tab[1][i] = a.pro_shift[i];
    }
    __syncthreads();
  } else if constexpr (PRO == PRO_BWD) {
    for (int i = tid; i < a.c_in; i += 256) {
      pro_tab[0][i] = a.pro_ca[i];
      pro_tab[1][i] = a.pro_cb[i];
      pro_tab[2][i] = a.pro_cc[i];
      pro_tab[3][i] = a.pro_mean[i];
    }
    __syncthreads();
  }
  pro_patch(0);
  park_patch(0);
  park_slab(0);
  __syncthreads();
  if constexpr (FB) {
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int fr = tap / 3, fs = tap - fr * 3;
      const int toff = fr * HTW + fs;
      const T* sb = slab_base + tap * SLAB;
      Frag<T> af[FM], bfr[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) af[fm].load(patch_base + (rowpix[fm] + toff) * HP + lg * 8);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) bfr[fn].load(sb + (wn * TN + fn * 16) * 32 + w_off);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma(bfr[fn], af[fm], acc[fm][fn]);
    }
  }
  // Chunks x nine unrolled taps.  Every prefetch is unconditional (past the
  // end it re-reads the last chunk / slab into the buffer not being read), so
  // the number of loads in flight is fixed and the waits stay tight: the next
  // chunk's patch is in flight for all nine taps, each next slab for one tap.
  for (int chunk = 0; chunk < (FB ? 0 : chunks); ++chunk) {
    if constexpr (HB > 1) load_patch(min(chunk + 1, chunks - 1));
    const T* pt = patch_base + (HB > 1 ? (chunk & 1) : 0) * PATCH;
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int step = chunk * 9 + tap;
      load_slab(min(step + 1, steps - 1));
      const T* sb = slab_base + (step & 1) * SLAB;
      const int toff = (tap / 3) * HTW + (tap % 3);
      Frag<T> af[FM], bfr[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) af[fm].load(pt + (rowpix[fm] + toff) * HP + lg * 8);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) bfr[fn].load(sb + (wn * TN + fn * 16) * 32 + w_off);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma(bfr[fn], af[fm], acc[fm][fn]);
      park_slab((step + 1) & 1);
      if constexpr (HB > 1) {
        if (tap == 8) {
          pro_patch(min(chunk + 1, chunks - 1));
          park_patch((chunk + 1) & 1);
        }
      }
      __syncthreads();
    }
  }

  // acc holds D[cout][pixel] (weights are the MFMA's A operand)
  epilogue_cp<TW, FM, FN, WAVES_M, TM, TN, BN, EP>(acc, a, img, p0, q0, n0, wm, wn, lane, tid, 256,
                                                   red3, &epi);
}

template <int TH, int TW, int BN, int WAVES_M, int CH, int EP, int PRO>
__global__ __launch_bounds__(256, 2) void conv_fp_kernel(ConvArgs a) {
  using T = bf16_t;
  constexpr int BM = TH * TW;
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 16, FN = TN / 16;
  static_assert(TM % 16 == 0 && TN % 16 == 0, "tile");
  constexpr int HTH = TH + 2, HTW = TW + 2, HPIX = HTH * HTW;
  constexpr int HP = 40;                              // bf16 per patch pixel and chunk (32 + pad)
  constexpr int PLANE = HPIX * HP;                    // one chunk of the patch
  constexpr int P_CHUNKS = (HPIX * 4 + 255) / 256;    // 16-byte loads per thread and chunk
  constexpr int STEPS = CH * 9;
  constexpr int D = 3;                                // weight prefetch depth (steps)
  constexpr int MAIN_BYTES = CH * PLANE * 2;
  constexpr int LDS_BYTES = MAIN_BYTES;
  constexpr bool BWD = PRO == PRO_BWD;
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  __shared__ float pro_tab[BWD ? 4 : 2][PRO == PRO_NONE ? 1 : CH * 32];
  __shared__ float red3[WAVES_M][3][BN];

  T* patch = reinterpret_cast<T*>(lds);
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int lr = lane & 15, lg = lane >> 4;
  const int tiles_x = (a.w + TW - 1) / TW, tiles_y = (a.h + TH - 1) / TH;
  const int tx = blockIdx.x % tiles_x;
  const int ty = (blockIdx.x / tiles_x) % tiles_y;
  const int img = blockIdx.x / (tiles_x * tiles_y);
  const int p0 = ty * TH, q0 = tx * TW;
  const int n0 = blockIdx.y * BN;
  const long img_base = static_cast<long>(img) * a.h * a.w;
  const long in_bytes = static_cast<long>(a.n) * a.h * a.w * a.c_in * 2;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_proh = make_rsrc(BWD ? a.pro_h : a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_wt = make_rsrc(a.wt, static_cast<long>(a.c_out) * a.k_tot * 2);

  // Weight fragments of step s: lane (lr, lg) of fragment fn holds output
  // channel n0 + wn*TN + fn*16 + lr, k = tap*C_in + chunk*32 + lg*8 .. +7.
  uint32_t wrow[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int col = n0 + wn * TN + fn * 16 + lr;
    wrow[fn] = col < a.c_out ? static_cast<uint32_t>(col * a.k_tot + lg * 8) * 2u : BUF_OOB;
  }
  Frag<T> wb[D][FN];
  auto load_w = [&](int s, int slot) {
    const int chunk = s / 9, tap = s - chunk * 9;
    const uint32_t koff = static_cast<uint32_t>(tap * a.c_in + chunk * 32) * 2u;
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const uint32_t off = wrow[fn] == BUF_OOB ? BUF_OOB : wrow[fn] + koff;
      wb[slot][fn].v = __builtin_bit_cast(bf16x8_t, buf_load16(r_wt, off));
    }
  };
#pragma unroll
  for (int d = 0; d < D; ++d) load_w(d, d);

  if constexpr (PRO == PRO_RELU) {
    for (int i = tid; i < a.c_in; i += 256) {
      pro_tab[0][i] = a.pro_scale[i];
      pro_tab[1][i] = a.pro_shift[i];
    }
  } else if constexpr (BWD) {
    for (int i = tid; i < a.c_in; i += 256) {
      pro_tab[0][i] = a.pro_ca[i];
      pro_tab[1][i] = a.pro_cb[i];
      pro_tab[2][i] = a.pro_cc[i];
      pro_tab[3][i] = a.pro_mean[i];
    }
  }

  // Patch fill, one chunk at a time with the next chunk's loads in flight.
  int p_off[P_CHUNKS];
  uint32_t pvalid = 0;
#pragma unroll
  for (int i = 0; i < P_CHUNKS; ++i) {
    const int q = tid + 256 * i;
    const int hp = q >> 2, sub = q & 3;
    const int hy = hp / HTW, hx = hp - hy * HTW;
    const int ih = p0 - 1 + hy, iw = q0 - 1 + hx;
    const bool ok = hp < HPIX && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
    p_off[i] = ok ? static_cast<int>(((img_base + static_cast<long>(ih) * a.w + iw) * a.c_in + sub * 8) * 2) : -1;
    pvalid |= ok ? 1u << i : 0u;
  }
  Raw8<T> ph[2][P_CHUNKS], phh[2][BWD ? P_CHUNKS : 1];
  auto load_chunk = [&](int c, int slot) {
#pragma unroll
    for (int i = 0; i < P_CHUNKS; ++i) {
      const uint32_t off = p_off[i] >= 0 ? static_cast<uint32_t>(p_off[i] + c * 64) : BUF_OOB;
      ph[slot][i].set(buf_load16(r_src, off));
      if constexpr (BWD) phh[slot][i].set(buf_load16(r_proh, off));
    }
  };
  auto park_chunk = [&](int c, int slot) {
    T* dst = patch + c * PLANE;
#pragma unroll
    for (int i = 0; i < P_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int hp = q >> 2, sub = q & 3;
      if (hp >= HPIX) continue;
      Raw8<T> r = ph[slot][i];
      if constexpr (PRO != PRO_NONE) {
        pro8<T, PRO>(r, phh[slot][BWD ? i : 0], pro_tab[0], pro_tab[1], pro_tab[BWD ? 2 : 0],
                     pro_tab[BWD ? 3 : 0], c * 32 + sub * 8);
        if (!((pvalid >> i) & 1u)) r.zero();
      }
      *reinterpret_cast<uint4*>(dst + hp * HP + sub * 8) = make_uint4(r.w[0], r.w[1], r.w[2], r.w[3]);
    }
  };
  load_chunk(0, 0);
  if constexpr (PRO != PRO_NONE) __syncthreads();   // prologue table
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    if (c + 1 < CH) load_chunk(c + 1, (c + 1) & 1);
    park_chunk(c, c & 1);
  }
  __syncthreads();

  int rowpix[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int i = wm * TM + fm * 16 + lr;
    const int ph_ = i / TW, pw = i - ph_ * TW;
    rowpix[fm] = ph_ * HTW + pw;
  }
  f32x4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Patch fragments of step s (double-buffered one step ahead).
  Frag<T> af[2][FM];
  auto load_a = [&](int s, int buf) {
    const int chunk = s / 9, tap = s - chunk * 9;
    const T* pt = patch + chunk * PLANE + ((tap / 3) * HTW + (tap % 3)) * HP + lg * 8;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) af[buf][fm].load(pt + rowpix[fm] * HP);
  };
  load_a(0, 0);
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int slot = s % D;
    Frag<T> cur[FN];
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) cur[fn] = wb[slot][fn];
    // refill this slot D steps ahead (past the end: reload the last step) and
    // fetch the next step's patch fragments; the scheduling barriers keep the
    // compiler from sinking these loads down to their uses
    load_w(s + D < STEPS ? s + D : STEPS - 1, slot);
    if (s + 1 < STEPS) load_a(s + 1, (s + 1) & 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma(cur[fn], af[s & 1][fm], acc[fm][fn]);
    __builtin_amdgcn_sched_barrier(0);
  }

  // acc holds D[cout][pixel] (weights are the MFMA's A operand)
  epilogue_cp<TW, FM, FN, WAVES_M, TM, TN, BN, EP>(acc, a, img, p0, q0, n0, wm, wn, lane, tid, 256,
                                                   red3);
}

// Whole-image 3x3 / stride 1 / pad 1 conv for the MFMA-bound shapes: one
// 512-thread workgroup per TH x TW image (TW = 16: a 16-pixel MFMA fragment is
// one image row), C_in = 32 * CH, C_out = 128.
//  * The reduction runs chunk-major (k step s = c * 9 + tap over the 32-channel
//    input chunks c), so the MFMAs start as soon as chunk 0 of the (TH+2) x
//    (TW+2) input patch is in LDS; the later chunks are loaded meanwhile
//    (prologue applied while parking) and parked one slab before their first
//    use.
//  * Weights go through double-buffered LDS slabs of one tap row (3 k steps of
//    32 channels, 64 bytes of every weight row each), loaded two slabs ahead,
//    one barrier per slab.
//  * LDS rows are 64 bytes (32 bf16) with the four 16-byte chunks of a row
//    permuted by bits 1-2 of the row index: the 16 consecutive rows a fragment
//    read touches then fall in distinct banks (ds_read_b128 measured at full
//    LDS bandwidth, against half of it for 80- or 144-byte padded rows).
//  * The MFMA is issued as D[cout][pixel] = W x patch^T: each lane ends with 4
//    consecutive output channels of one pixel, stored directly (8 bytes), and
//    the BN statistics are shifted sums in registers reduced once at the end.
// The tile is the whole image (the launcher checks h = TH, w = TW), so every
// output pixel is valid.  Partial row of the statistics = blockIdx.x (the image).
template <int TH, int TW, int CH, int EP, int PRO, int NWM, int NWN>
__global__ __launch_bounds__(64 * NWM * NWN, 1) void conv_img_kernel(ConvArgs a) {
  using T = bf16_t;
  constexpr int NT = 64 * NWM * NWN;
  constexpr int WAVES_M = NWM, WAVES_N = NWN;
  constexpr int BN = 128, BM = TH * TW;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 16, FN = TN / 16;
  static_assert(TW == 16 && TM % 16 == 0 && TN % 16 == 0, "fragments are image rows");
  static_assert(NT == BN * 4, "one 16-byte weight load per thread and k step");
  constexpr int HTH = TH + 2, HTW = TW + 2, HPIX = HTH * HTW;
  constexpr int PLANE = HPIX * 32;                   // bf16 per input chunk (64 bytes per pixel)
  constexpr int P_CHUNKS = (HPIX * 4 + NT - 1) / NT; // 16-byte patch loads per thread and chunk
  constexpr int WPLANE = BN * 32;                    // bf16 per k step of a weight slab
  constexpr int SLAB = 3 * WPLANE;                   // one tap row: 3 k steps
  constexpr int SLABS = CH * 3;                      // slab j: chunk j / 3, tap row j % 3
  constexpr bool BWD = PRO == PRO_BWD;
  constexpr bool STATS = EP == EP_STATS;
  constexpr int NCS = 1;                             // input chunks in flight in registers
  __shared__ __attribute__((aligned(16))) T lds[CH * PLANE + 2 * SLAB];
  __shared__ float pro_tab[BWD ? 4 : 2][PRO == PRO_NONE ? 1 : CH * 32];
  __shared__ float red[WAVES_M][3][BN];

  T* patch = lds;
  T* slabs = lds + CH * PLANE;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int lr = lane & 15, lg = lane >> 4;
  const int img = blockIdx.x;
  const long img_base = static_cast<long>(img) * a.h * a.w;
  const long in_bytes = static_cast<long>(a.n) * a.h * a.w * a.c_in * 2;
  const long out_bytes = static_cast<long>(a.m) * BN * 2;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_proh = make_rsrc(BWD ? a.pro_h : a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_wt = make_rsrc(a.wt, static_cast<long>(BN) * a.k_tot * 2);
  const __amdgpu_buffer_rsrc_t r_out = make_rsrc(a.out, out_bytes);
  const __amdgpu_buffer_rsrc_t r_eph = make_rsrc(a.ep_h != nullptr ? a.ep_h : a.out, out_bytes);
  const __amdgpu_buffer_rsrc_t r_res = make_rsrc(a.resid != nullptr ? a.resid : a.out,
                                                 a.resid != nullptr ? out_bytes : 0);

  // Weight slab j (chunk c = j / 3, tap row dy = j % 3), k step u = dx: input
  // channels c*32 .. c*32+31 of tap 3 dy + dx.  Thread t loads 16 bytes of row
  // t / 4 per k step, so 4 neighbouring threads read one 64-byte run.
  const int s_row = tid >> 2, s_sub = tid & 3;
  const uint32_t s_gl = static_cast<uint32_t>((s_row * a.k_tot + s_sub * 8) * 2);
  const int s_lds = s_row * 32 + ((s_sub ^ ((s_row >> 1) & 3)) * 8);
  u32x4_t rs[2][3];
  auto load_slab = [&](u32x4_t* r, int j) {
    const int c = j / 3, dy = j - c * 3;
#pragma unroll
    for (int u = 0; u < 3; ++u)
      r[u] = buf_load16(r_wt, s_gl + static_cast<uint32_t>(((3 * dy + u) * a.c_in + c * 32) * 2));
  };
  auto park_slab = [&](const u32x4_t* r, int buf) {
#pragma unroll
    for (int u = 0; u < 3; ++u)
      *reinterpret_cast<u32x4_t*>(slabs + buf * SLAB + u * WPLANE + s_lds) = r[u];
  };
  load_slab(rs[0], 0);
  if (SLABS > 1) load_slab(rs[1], 1);

  if constexpr (PRO == PRO_RELU) {
    for (int i = tid; i < a.c_in; i += NT) {
      pro_tab[0][i] = a.pro_scale[i];
      pro_tab[1][i] = a.pro_shift[i];
    }
  } else if constexpr (BWD) {
    for (int i = tid; i < a.c_in; i += NT) {
      pro_tab[0][i] = a.pro_ca[i];
      pro_tab[1][i] = a.pro_cb[i];
      pro_tab[2][i] = a.pro_cc[i];
      pro_tab[3][i] = a.pro_mean[i];
    }
  }

  // Input patch: thread t takes 16-byte pieces q = t + NT i (patch pixel q / 4,
  // channels (q % 4) * 8 .. + 7 of a chunk).
  int p_off[P_CHUNKS];
  uint32_t pvalid = 0;
#pragma unroll
  for (int i = 0; i < P_CHUNKS; ++i) {
    const int q = tid + NT * i;
    const int hp = q >> 2, sub = q & 3;
    const int hy = hp / HTW, hx = hp - hy * HTW;
    const int ih = hy - 1, iw = hx - 1;
    const bool ok = hp < HPIX && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
    p_off[i] = ok ? static_cast<int>(((img_base + static_cast<long>(ih) * a.w + iw) * a.c_in + sub * 8) * 2) : -1;
    pvalid |= ok ? 1u << i : 0u;
  }
  Raw8<T> ph[NCS][P_CHUNKS], phh[NCS][BWD ? P_CHUNKS : 1];
  auto load_chunk = [&](int c) {
    const int slot = c % NCS;
#pragma unroll
    for (int i = 0; i < P_CHUNKS; ++i) {
      const uint32_t off = p_off[i] >= 0 ? static_cast<uint32_t>(p_off[i] + c * 64) : BUF_OOB;
      ph[slot][i].set(buf_load16(r_src, off));
      if constexpr (BWD) phh[slot][i].set(buf_load16(r_proh, off));
    }
  };
  auto park_chunk = [&](int c) {
    const int slot = c % NCS;
    T* dst = patch + c * PLANE;
#pragma unroll
    for (int i = 0; i < P_CHUNKS; ++i) {
      const int q = tid + NT * i;
      const int hp = q >> 2, sub = q & 3;
      if (hp >= HPIX) continue;
      Raw8<T> r = ph[slot][i];
      if constexpr (PRO != PRO_NONE) {
        pro8<T, PRO>(r, phh[slot][BWD ? i : 0], pro_tab[0], pro_tab[1], pro_tab[BWD ? 2 : 0],
                     pro_tab[BWD ? 3 : 0], c * 32 + sub * 8);
        if (!((pvalid >> i) & 1u)) r.zero();
      }
      *reinterpret_cast<uint4*>(dst + hp * 32 + ((sub ^ ((hp >> 1) & 3)) * 8)) =
          make_uint4(r.w[0], r.w[1], r.w[2], r.w[3]);
    }
  };
#pragma unroll
  for (int c = 0; c < NCS && c < CH; ++c) load_chunk(c);
  if constexpr (PRO != PRO_NONE) __syncthreads();   // prologue table
  park_chunk(0);
  if (NCS < CH) load_chunk(NCS);
  park_slab(rs[0], 0);
  __syncthreads();

  // Fragment addresses.  Weights: row wn*TN + fn*16 + lr of a k-step plane,
  // whose chunk permutation is (lr >> 1) & 3.  Patch: fragment fm of tap
  // (dy, dx) reads pixel (rb + fm + dy) * HTW + dx + lr of a chunk plane (rb =
  // wm * FM, the wave's first image row); bits 1-2 of that index are
  // (rb + fm + dy + ((dx + lr) >> 1)) & 3, so the lane's offsets for the 3
  // values of dx and the 4 values of (fm + dy) & 3 are computed once here.
  const int rb = wm * FM;
  const int w_off = (wn * TN + lr) * 32 + ((lg ^ ((lr >> 1) & 3)) * 8);
  int p_tab[3][4];
#pragma unroll
  for (int dx = 0; dx < 3; ++dx)
#pragma unroll
    for (int k = 0; k < 4; ++k)
      p_tab[dx][k] = (rb * HTW + dx + lr) * 32 + ((lg ^ ((k + rb + ((dx + lr) >> 1)) & 3)) * 8);

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Slab j: slab j + 2 into the register set that held slab j, MFMAs on slab j
  // from LDS buffer j % 2, slab j + 1 (loaded an iteration earlier) parked into
  // the other buffer, and before the last slab of a chunk the next chunk parked.
#pragma unroll
  for (int j = 0; j < SLABS; ++j) {
    const int c = j / 3, dy = j - c * 3, buf = j & 1;
    if (j + 2 < SLABS) load_slab(rs[j & 1], j + 2);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int dx = 0; dx < 3; ++dx) {
      Frag<T> wf[FN], pf[FM];
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) wf[fn].load(slabs + buf * SLAB + dx * WPLANE + fn * 16 * 32 + w_off);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        pf[fm].load(patch + c * PLANE + (fm + dy) * HTW * 32 + p_tab[dx][(fm + dy) & 3]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma(wf[fn], pf[fm], acc[fm][fn]);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (dy == 2 && c + 1 < CH) {
      park_chunk(c + 1);
      if (c + 1 + NCS < CH) load_chunk(c + 1 + NCS);
    }
    if (j + 1 < SLABS) park_slab(rs[(j + 1) & 1], buf ^ 1);
    __syncthreads();
  }

  // Epilogue: lane (lr, lg) holds channels wn*TN + fn*16 + lg*4 + e of pixel
  // wm*TM + fm*16 + lr.
  float es[FN][4], esh[FN][4], emu[FN][4], ers[FN][4];
  if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = wn * TN + fn * 16 + lg * 4 + e;
        es[fn][e] = EP == EP_MASK ? a.ep_scale[c] : 0.f;
        esh[fn][e] = EP == EP_MASK ? a.ep_shift[c] : 0.f;
        emu[fn][e] = a.ep_mean[c];
        ers[fn][e] = a.ep_rstd[c];
      }
  }
  float sa[FN][4], sb2[FN][4], kk[FN][4];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn)
#pragma unroll
    for (int e = 0; e < 4; ++e) sa[fn][e] = sb2[fn][e] = kk[fn][e] = 0.f;
  float nv = 0.f;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    // image row rb + fm, column lr: every pixel of the tile is in the image
    constexpr bool vm = true;
    nv += 1.f;
    const uint32_t pixoff =
        static_cast<uint32_t>(((img_base + static_cast<long>(rb + fm) * TW + lr) * BN) * 2);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const uint32_t boff = vm ? pixoff + (wn * TN + fn * 16 + lg * 4) * 2 : BUF_OOB;
      float v[4] = {acc[fm][fn][0], acc[fm][fn][1], acc[fm][fn][2], acc[fm][fn][3]};
      float hl[4] = {0.f, 0.f, 0.f, 0.f};
      if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
        const u32x2_t hw = buf_load8(r_eph, boff);
        hl[0] = __uint_as_float(hw.x << 16); hl[1] = __uint_as_float(hw.x & 0xffff0000u);
        hl[2] = __uint_as_float(hw.y << 16); hl[3] = __uint_as_float(hw.y & 0xffff0000u);
      }
      if constexpr (EP == EP_RESID || EP == EP_RESID_STATS) {
        const u32x2_t rw = buf_load8(r_res, boff);   // a null residual reads zeros
        v[0] += __uint_as_float(rw.x << 16); v[1] += __uint_as_float(rw.x & 0xffff0000u);
        v[2] += __uint_as_float(rw.y << 16); v[3] += __uint_as_float(rw.y & 0xffff0000u);
      }
      if constexpr (EP == EP_MASK) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = fmaf(es[fn][e], hl[e], esh[fn][e]) > 0.f ? v[e] : 0.f;
      }
      const uint32_t w0 = pack_bf16x2(v[0], v[1]), w1 = pack_bf16x2(v[2], v[3]);
      buf_store8(u32x2_t{w0, w1}, r_out, boff);
      // statistics of the stored values
      v[0] = __uint_as_float(w0 << 16); v[1] = __uint_as_float(w0 & 0xffff0000u);
      v[2] = __uint_as_float(w1 << 16); v[3] = __uint_as_float(w1 & 0xffff0000u);
      if constexpr (STATS) {
        if (fm == 0) {
          // shift per channel: the value at this wave's first pixel
#pragma unroll
          for (int e = 0; e < 4; ++e) kk[fn][e] = __shfl(v[e], lane & 48, 64);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float d = vm ? v[e] - kk[fn][e] : 0.f;
          sa[fn][e] += d;
          sb2[fn][e] = fmaf(d, d, sb2[fn][e]);
        }
      } else if constexpr (EP != EP_RESID) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float g = vm ? v[e] : 0.f;
          sa[fn][e] += g;
          sb2[fn][e] += g * ((hl[e] - emu[fn][e]) * ers[fn][e]);
        }
      }
    }
  }
  if constexpr (EP != EP_RESID) {
    const float n16 = sum16(nv);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = sum16(sa[fn][e]), y = sum16(sb2[fn][e]);
        if (lr == 0) {
          const int c = wn * TN + fn * 16 + lg * 4 + e;
          if constexpr (STATS) {
            const float md = n16 > 0.f ? x / n16 : 0.f;
            red[wm][0][c] = n16;
            red[wm][1][c] = kk[fn][e] + md;                          // mean
            red[wm][2][c] = n16 > 0.f ? fmaxf(y - x * md, 0.f) : 0.f;  // centred M2
          } else {
            red[wm][1][c] = x;
            red[wm][2][c] = y;
          }
        }
      }
    __syncthreads();
    if (tid < BN) {
      const int c = tid;
      float* pr = a.partials;
      const long row = static_cast<long>(blockIdx.x);
      if constexpr (STATS) {
        float n = 0.f, mean = 0.f, m2 = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES_M; ++w) {
          const float nb = red[w][0][c];
          if (nb > 0.f) {
            const float nn = n + nb, rb = nb / nn, d = red[w][1][c] - mean;
            mean += d * rb;
            m2 += red[w][2][c] + d * d * n * rb;
            n = nn;
          }
        }
        pr[(row * 3 + 0) * BN + c] = n;
        pr[(row * 3 + 1) * BN + c] = n * mean;
        pr[(row * 3 + 2) * BN + c] = m2;
      } else {
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES_M; ++w) {
          s1 += red[w][1][c];
          s2 += red[w][2][c];
        }
        pr[(row * 2 + 0) * BN + c] = s1;
        pr[(row * 2 + 1) * BN + c] = s2;
      }
    }
  }
}

// [16 pixels][N] bf16 tile of one unit of the 1x1 kernels, in a wave-private
// LDS slice.  The MFMA leaves each lane 4 channels (8 bytes) of one pixel; the
// global side moves whole rows instead, every lane 16 contiguous bytes, so one
// load or store instruction covers 1 KB of consecutive rows.  LDS operations of
// a wave complete in order, so no barrier is needed between writes and reads,
// nor before the next unit overwrites the slice.
template <int N>
struct UnitTile {
  static constexpr int ROW = N / 2 + 2;        // 32-bit words per pixel row (+ pad)
  static constexpr int CHUNKS = 16 * N / 8;    // 16-byte chunks per unit
  static_assert(CHUNKS % 64 == 0, "whole chunks per lane");
  static constexpr int PER_LANE = CHUNKS / 64;
  uint32_t w[16 * ROW];
  __device__ __forceinline__ void put(int lr, int lg, int nb, uint32_t w0, uint32_t w1) {
    uint32_t* p = w + lr * ROW + (nb * 16 + lg * 4) / 2;
    *reinterpret_cast<u32x2_t*>(p) = u32x2_t{w0, w1};
  }
  __device__ __forceinline__ u32x2_t get(int lr, int lg, int nb) const {
    return *reinterpret_cast<const u32x2_t*>(w + lr * ROW + (nb * 16 + lg * 4) / 2);
  }
  // row-major loads of the unit's rows of a [m][N] tensor (zeros past m)
  static __device__ __forceinline__ void load_rows(__amdgpu_buffer_rsrc_t r, int u, long m,
                                                   int lane, u32x4_t* q) {
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) {
      const int c = lane + 64 * i;
      const int px = c / (N / 8), ch = c - px * (N / 8);
      const long pix = static_cast<long>(u) * 16 + px;
      q[i] = buf_load16(r, pix < m ? static_cast<uint32_t>((pix * N + ch * 8) * 2) : BUF_OOB);
    }
  }
  __device__ __forceinline__ void park_rows(const u32x4_t* q, int lane) {
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) {
      const int c = lane + 64 * i;
      const int px = c / (N / 8), ch = c - px * (N / 8);
      uint32_t* p = w + px * ROW + ch * 4;
      *reinterpret_cast<u32x2_t*>(p) = u32x2_t{q[i][0], q[i][1]};
      *reinterpret_cast<u32x2_t*>(p + 2) = u32x2_t{q[i][2], q[i][3]};
    }
  }
  // stores the unit's valid rows (pixels u*16 .. u*16 + 15 below m) through r_out
  __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t r_out, int u, long m, int lane) {
#pragma unroll
    for (int i = 0; i < CHUNKS / 64; ++i) {
      const int q = lane + 64 * i;
      const int px = q / (N / 8), ch = q - px * (N / 8);
      const uint32_t* p = w + px * ROW + ch * 4;
      const u32x4_t v = u32x4_t{p[0], p[1], p[2], p[3]};
      const long pix = static_cast<long>(u) * 16 + px;
      const uint32_t off = pix < m ? static_cast<uint32_t>((pix * N + ch * 8) * 2) : BUF_OOB;
      buf_store16(v, r_out, off);
    }
  }
};

// 1x1 / stride 1 bf16 convolution with the BN-statistics epilogue, for the
// HBM-bound bottleneck widths (C_in x C_out = 128 x 32 and 32 x 128).  There is
// no LDS staging: a wave loads the 16 x K activation block of a 16-pixel unit
// straight into MFMA operand registers (each lane 16 contiguous bytes of one
// pixel), keeps every weight fragment in registers for the whole launch, and
// issues D[cout][pixel] so that each lane stores 4 consecutive output channels
// of one pixel (8 bytes).  Waves stream over units g, g + W, g + 2W, ... with
// the next unit's loads in flight during the current unit's MFMAs and stores;
// no barrier until the end.  BN moments are shifted sums in registers (shift:
// the stored value of the wave's first pixel, per channel), combined over the
// four waves once per workgroup: partial row = blockIdx.x.  ST = false: the
// statistics only (nothing stored; the coupling kernel below recomputes the
// output where it is consumed).
template <int K, int N, int PRO, bool ST = true>
__global__ __launch_bounds__(256) void conv1x1_kernel(ConvArgs a, int units) {
  using T = bf16_t;
  constexpr int KB = K / 32, NB = N / 16;
  static_assert(K % 32 == 0 && N % 16 == 0 && PRO != PRO_BWD, "1x1 shape");
  constexpr int PK = PRO == PRO_RELU ? KB : 1;
  __shared__ float red[4][3][N];
  __shared__ __attribute__((aligned(16))) UnitTile<N> otile[4];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const long m = a.m;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, m * K * 2);
  const __amdgpu_buffer_rsrc_t r_out = make_rsrc(a.out, m * N * 2);
  const __amdgpu_buffer_rsrc_t r_wt = make_rsrc(a.wt, static_cast<long>(N) * K * 2);

  auto load_unit = [&](int u, u32x4_t* x) {
    const long pix = static_cast<long>(u) * 16 + lr;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const uint32_t off =
          pix < m ? static_cast<uint32_t>((pix * K + kb * 32 + lg * 8) * 2) : BUF_OOB;
      x[kb] = buf_load16(r_src, off);
    }
  };
  const int W = gridDim.x * 4;
  int u = blockIdx.x * 4 + wave;
  u32x4_t xr[KB], xn[KB];
  if (u < units) load_unit(u, xr);

  // weight fragments: lane (lr, lg) holds W[nb*16 + lr][kb*32 + lg*8 .. +7]
  Frag<T> wf[NB][KB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      Raw8<T> r;
      r.set(buf_load16(r_wt, static_cast<uint32_t>(((nb * 16 + lr) * K + kb * 32 + lg * 8) * 2)));
      wf[nb][kb].set(r);
    }
  // BN-apply + ReLU constants of this lane's input channels
  float ps[PK][8], pt[PK][8];
  if constexpr (PRO == PRO_RELU) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        ps[kb][j] = a.pro_scale[kb * 32 + lg * 8 + j];
        pt[kb][j] = a.pro_shift[kb * 32 + lg * 8 + j];
      }
  }

  float sa[NB][4], sb[NB][4], kk[NB][4];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) sa[nb][e] = sb[nb][e] = kk[nb][e] = 0.f;
  float nv = 0.f;
  bool first = true;
  // one unit; FULL: all 16 pixels inside the tensor (every unit but a ragged last one)
  auto unit = [&](auto full_t) {
    constexpr bool FULL = decltype(full_t)::value;
    Frag<T> xf[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      Raw8<T> r;
      r.set(xr[kb]);
      if constexpr (PRO == PRO_RELU) {
        float v[8];
        r.to_f32(v);
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = fmaxf(fmaf(ps[kb][j], v[j], pt[kb][j]), 0.f);
        r.from_f32(v);   // rounded to bf16, as the materialised activation
      }
      xf[kb].set(r);
    }
    const long pix = static_cast<long>(u) * 16 + lr;
    const bool vm = FULL || pix < m;
    nv += vm ? 1.f : 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) acc = mfma(wf[nb][kb], xf[kb], acc);
      const uint32_t w0 = pack_bf16x2(acc[0], acc[1]), w1 = pack_bf16x2(acc[2], acc[3]);
      if constexpr (ST) otile[wave].put(lr, lg, nb, w0, w1);
      // statistics of the stored values
      float v[4];
      v[0] = __uint_as_float(w0 << 16); v[1] = __uint_as_float(w0 & 0xffff0000u);
      v[2] = __uint_as_float(w1 << 16); v[3] = __uint_as_float(w1 & 0xffff0000u);
      if (first) {
        // the unit's first pixel is inside the image (u < units)
#pragma unroll
        for (int e = 0; e < 4; ++e) kk[nb][e] = __shfl(v[e], lane & 48, 64);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float d = vm ? v[e] - kk[nb][e] : 0.f;
        sa[nb][e] += d;
        sb[nb][e] = fmaf(d, d, sb[nb][e]);
      }
    }
    if constexpr (ST) otile[wave].store(r_out, u, m, lane);
  };
  for (; u < units; u += W) {
    const int un = u + W;
    if (un < units) load_unit(un, xn);
    if ((static_cast<long>(u) + 1) * 16 <= m)
      unit(std::true_type{});
    else
      unit(std::false_type{});
    first = false;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) xr[kb] = xn[kb];
  }
  // per wave: (n, mean, centred M2) of every channel; then Chan over the waves
  const float n16 = sum16(nv);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = sum16(sa[nb][e]), y = sum16(sb[nb][e]);
      if (lr == 0) {
        const int c = nb * 16 + lg * 4 + e;
        const float md = n16 > 0.f ? x / n16 : 0.f;
        red[wave][0][c] = n16;
        red[wave][1][c] = kk[nb][e] + md;
        red[wave][2][c] = n16 > 0.f ? fmaxf(y - x * md, 0.f) : 0.f;
      }
    }
  __syncthreads();
  for (int c = tid; c < N; c += 256) {
    float n = 0.f, mean = 0.f, m2 = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float nb = red[w][0][c];
      if (nb > 0.f) {
        const float nn = n + nb, rb = nb / nn, d = red[w][1][c] - mean;
        mean += d * rb;
        m2 += red[w][2][c] + d * d * n * rb;
        n = nn;
      }
    }
    const long row = blockIdx.x;
    a.partials[(row * 3 + 0) * N + c] = n;
    a.partials[(row * 3 + 1) * N + c] = n * mean;
    a.partials[(row * 3 + 2) * N + c] = m2;
  }
}

// Coupling of a residual function whose last layer is a streaming 1x1 conv
// (the forward add of Eq. 4, or the reconstruction's subtraction): out =
// r + (scale h + shift), or r - (scale h + shift) with SUB, where h is that
// conv's output as the statistics pass rounds it to bf16 (same operands, same
// MFMA order, same rounding: the same bits) -- recomputed from the layer's
// input (C_in = K channels, read once) instead of being stored at C_out = N
// channels and read back.  The BN of h enters through ep_scale / ep_shift, the
// layer's own BN-apply + ReLU prologue through pro_scale / pro_shift as in
// conv1x1_kernel.  Each wave streams 16-pixel units with the input and
// residual rows of the next unit in flight; the residual goes through the
// wave's LDS tile into the MFMA layout and the result back out as whole rows.
// out may alias resid: a unit's rows are read before they are written, by the
// one wave that owns the unit.
// NX: the coupling output is also the input of the next residual function,
// whose first layer is the 1x1 N -> K conv: the unit's output rows, still in
// the LDS tile, feed that conv's MFMAs directly, and its output (stored at
// nx.out) and BN partials (nx.partials, row = blockIdx.x) are exactly what
// conv1x1_kernel<N, K, PRO_NONE> would produce from the stored output: the
// same grid, units per wave, operands, MFMA order, rounding and statistics.

template <int K, int N, bool SUB, bool NX>
__global__ __launch_bounds__(256) void conv1x1_couple_kernel(ConvArgs a, int units, NextConv nx) {
  using T = bf16_t;
  constexpr int KB = K / 32, NB = N / 16;
  constexpr int KB2 = N / 32, NB2 = K / 16;   // the next conv: N -> K
  using Tile = UnitTile<N>;
  using Tile2 = UnitTile<K>;
  constexpr int CH = Tile::PER_LANE;
  __shared__ __attribute__((aligned(16))) Tile otile[4];   // residual in, result out
  __shared__ __attribute__((aligned(16))) Tile2 ntile[NX ? 4 : 1];
  __shared__ float red[NX ? 4 : 1][3][K];
  __shared__ float cst[2][NX ? N : 1];   // BN of h (scale, shift) when registers are short
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const long m = a.m;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, m * K * 2);
  const __amdgpu_buffer_rsrc_t r_out = make_rsrc(a.out, m * N * 2);
  const __amdgpu_buffer_rsrc_t r_res = make_rsrc(a.resid, m * N * 2);
  const __amdgpu_buffer_rsrc_t r_wt = make_rsrc(a.wt, static_cast<long>(N) * K * 2);
  const __amdgpu_buffer_rsrc_t r_nout = make_rsrc(NX ? nx.out : a.out, NX ? m * K * 2 : 0);
  const __amdgpu_buffer_rsrc_t r_nwt =
      make_rsrc(NX ? nx.wt : a.wt, NX ? static_cast<long>(K) * N * 2 : 0);
  if constexpr (NX) {
    for (int c = tid; c < N; c += 256) {
      cst[0][c] = a.ep_scale[c];
      cst[1][c] = a.ep_shift[c];
    }
  }
  struct Unit {
    u32x4_t x[KB];
    u32x4_t rs[CH];
  };
  auto load_unit = [&](int u, Unit& d) {
    const long pix = static_cast<long>(u) * 16 + lr;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const uint32_t off =
          pix < m ? static_cast<uint32_t>((pix * K + kb * 32 + lg * 8) * 2) : BUF_OOB;
      d.x[kb] = buf_load16(r_src, off);
    }
    Tile::load_rows(r_res, u, m, lane, d.rs);
  };
  const int W = gridDim.x * 4;
  int u = blockIdx.x * 4 + wave;
  Unit cur, nxt;
  if (u < units) load_unit(u, cur);

  Frag<T> wf[NB][KB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      Raw8<T> r;
      r.set(buf_load16(r_wt, static_cast<uint32_t>(((nb * 16 + lr) * K + kb * 32 + lg * 8) * 2)));
      wf[nb][kb].set(r);
    }
  // the next conv's weight fragments (as conv1x1_kernel<N, K> holds them)
  Frag<T> wf2[NX ? NB2 : 1][NX ? KB2 : 1];
  if constexpr (NX) {
#pragma unroll
    for (int nb = 0; nb < NB2; ++nb)
#pragma unroll
      for (int kb = 0; kb < KB2; ++kb) {
        Raw8<T> r;
        r.set(buf_load16(r_nwt,
                         static_cast<uint32_t>(((nb * 16 + lr) * N + kb * 32 + lg * 8) * 2)));
        wf2[nb][kb].set(r);
      }
  }
  float ps[KB][8], pt[KB][8];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      ps[kb][j] = a.pro_scale[kb * 32 + lg * 8 + j];
      pt[kb][j] = a.pro_shift[kb * 32 + lg * 8 + j];
    }
  float cs[NX ? 1 : NB][4], csh[NX ? 1 : NB][4];
  if constexpr (!NX) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cs[nb][e] = a.ep_scale[nb * 16 + lg * 4 + e];
        csh[nb][e] = a.ep_shift[nb * 16 + lg * 4 + e];
      }
  }
  // the next conv's BN moments: shifted sums per lane, as in conv1x1_kernel
  float sa[NX ? NB2 : 1][4], sb[NX ? NB2 : 1][4], kk[NX ? NB2 : 1][4];
#pragma unroll
  for (int nb = 0; nb < (NX ? NB2 : 1); ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) sa[nb][e] = sb[nb][e] = kk[nb][e] = 0.f;
  float nv = 0.f;
  bool first = true;
  if constexpr (NX) __syncthreads();   // cst
  auto unit = [&](auto full_t) {
    constexpr bool FULL = decltype(full_t)::value;
    Frag<T> xf[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      Raw8<T> r;
      r.set(cur.x[kb]);
      float v[8];
      r.to_f32(v);
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = fmaxf(fmaf(ps[kb][j], v[j], pt[kb][j]), 0.f);
      r.from_f32(v);   // rounded to bf16, as the materialised activation
      xf[kb].set(r);
    }
    otile[wave].park_rows(cur.rs, lane);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) acc = mfma(wf[nb][kb], xf[kb], acc);
      // h as the statistics pass rounds it
      const uint32_t h0 = pack_bf16x2(acc[0], acc[1]), h1 = pack_bf16x2(acc[2], acc[3]);
      float h[4];
      h[0] = __uint_as_float(h0 << 16); h[1] = __uint_as_float(h0 & 0xffff0000u);
      h[2] = __uint_as_float(h1 << 16); h[3] = __uint_as_float(h1 & 0xffff0000u);
      const u32x2_t rw = otile[wave].get(lr, lg, nb);
      float r[4];
      r[0] = __uint_as_float(rw.x << 16); r[1] = __uint_as_float(rw.x & 0xffff0000u);
      r[2] = __uint_as_float(rw.y << 16); r[3] = __uint_as_float(rw.y & 0xffff0000u);
      float o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = nb * 16 + lg * 4 + e;
        const float f = NX ? fmaf(cst[0][c], h[e], cst[1][c])
                           : fmaf(cs[NX ? 0 : nb][e], h[e], csh[NX ? 0 : nb][e]);
        o[e] = SUB ? r[e] - f : r[e] + f;
      }
      otile[wave].put(lr, lg, nb, pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
    }
    otile[wave].store(r_out, u, m, lane);
    if constexpr (NX) {
      // the next conv on the unit's output rows: lane (lr, lg) takes channels
      // kb * 32 + lg * 8 .. + 7 of pixel lr, as a row load of the stored tensor would
      Frag<T> yf[KB2];
#pragma unroll
      for (int kb = 0; kb < KB2; ++kb) {
        const uint32_t* p = otile[wave].w + lr * Tile::ROW + (kb * 32 + lg * 8) / 2;
        const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(p);
        const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(p + 2);
        Raw8<T> rr;
        rr.set(u32x4_t{lo.x, lo.y, hi.x, hi.y});
        yf[kb].set(rr);
      }
      const long pix = static_cast<long>(u) * 16 + lr;
      const bool vm = FULL || pix < m;
      nv += vm ? 1.f : 0.f;
#pragma unroll
      for (int nb = 0; nb < NB2; ++nb) {
        f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB2; ++kb) acc = mfma(wf2[nb][kb], yf[kb], acc);
        const uint32_t w0 = pack_bf16x2(acc[0], acc[1]), w1 = pack_bf16x2(acc[2], acc[3]);
        ntile[wave].put(lr, lg, nb, w0, w1);
        float v[4];
        v[0] = __uint_as_float(w0 << 16); v[1] = __uint_as_float(w0 & 0xffff0000u);
        v[2] = __uint_as_float(w1 << 16); v[3] = __uint_as_float(w1 & 0xffff0000u);
        if (first) {
#pragma unroll
          for (int e = 0; e < 4; ++e) kk[nb][e] = __shfl(v[e], lane & 48, 64);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float d = vm ? v[e] - kk[nb][e] : 0.f;
          sa[nb][e] += d;
          sb[nb][e] = fmaf(d, d, sb[nb][e]);
        }
      }
      ntile[wave].store(r_nout, u, m, lane);
    }
  };
  for (; u < units; u += W) {
    const int un = u + W;
    if (un < units) load_unit(un, nxt);
    if ((static_cast<long>(u) + 1) * 16 <= m)
      unit(std::true_type{});
    else
      unit(std::false_type{});
    first = false;
    cur = nxt;
  }
  if constexpr (NX) {
    // per wave: (n, mean, centred M2) of every channel; then Chan over the
    // waves (the reduction of conv1x1_kernel)
    const float n16 = sum16(nv);
#pragma unroll
    for (int nb = 0; nb < NB2; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = sum16(sa[nb][e]), y = sum16(sb[nb][e]);
        if (lr == 0) {
          const int c = nb * 16 + lg * 4 + e;
          const float md = n16 > 0.f ? x / n16 : 0.f;
          red[wave][0][c] = n16;
          red[wave][1][c] = kk[nb][e] + md;
          red[wave][2][c] = n16 > 0.f ? fmaxf(y - x * md, 0.f) : 0.f;
        }
      }
    __syncthreads();
    for (int c = tid; c < K; c += 256) {
      float n = 0.f, mean = 0.f, m2 = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float nb = red[w][0][c];
        if (nb > 0.f) {
          const float nn = n + nb, rb = nb / nn, d = red[w][1][c] - mean;
          mean += d * rb;
          m2 += red[w][2][c] + d * d * n * rb;
          n = nn;
        }
      }
      const long row = blockIdx.x;
      nx.partials[(row * 3 + 0) * K + c] = n;
      nx.partials[(row * 3 + 1) * K + c] = n * mean;
      nx.partials[(row * 3 + 2) * K + c] = m2;
    }
  }
}

// Input-gradient form of the streaming 1x1 kernel: out = conv(dh) with the
// layer's transposed weights (here K and N are the layer's C_out and C_in).
// Prologue: PRO_BWD forms the BN input gradient ca d + cb (h - mean) + cc of
// the layer's BN as the output gradient d is loaded (h read at the same
// position), rounded to bf16 as the materialised gradient.  Epilogues as in the
// other conv kernels: EP_MASK (ReLU mask of the BN below plus its backward
// partials), EP_RESID (residual add), EP_RESID_STATS (residual add plus the
// BN-backward partials of the stored result against ep_h).  Every operand of
// the next unit, the epilogue's included, is in flight during the current one.
template <int K, int N, int EP, int PRO>
__global__ __launch_bounds__(256) void conv1x1_bwd_kernel(ConvArgs a, int units) {
  using T = bf16_t;
  constexpr int KB = K / 32, NB = N / 16;
  constexpr bool GRAD = EP == EP_MASK || EP == EP_RESID_STATS;
  constexpr bool RES = EP == EP_RESID || EP == EP_RESID_STATS;
  constexpr bool BWD = PRO == PRO_BWD;
  static_assert(K % 32 == 0 && N % 16 == 0 && EP != EP_STATS && PRO != PRO_RELU, "1x1 shape");
  constexpr int PK = BWD ? KB : 1;
  constexpr int EN = GRAD ? NB : 1;
  __shared__ float red[4][2][N];
  __shared__ __attribute__((aligned(16))) UnitTile<N> otile[4];   // residual in, result out
  __shared__ __attribute__((aligned(16))) UnitTile<N> etile[GRAD ? 4 : 1];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const long m = a.m;
  const long in_bytes = m * K * 2, out_bytes = m * N * 2;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_h = make_rsrc(BWD ? a.pro_h : a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_out = make_rsrc(a.out, out_bytes);
  const __amdgpu_buffer_rsrc_t r_eph = make_rsrc(a.ep_h != nullptr ? a.ep_h : a.out, out_bytes);
  // a null residual reads zeros
  const __amdgpu_buffer_rsrc_t r_res =
      make_rsrc(a.resid != nullptr ? a.resid : a.out, a.resid != nullptr ? out_bytes : 0);
  const __amdgpu_buffer_rsrc_t r_wt = make_rsrc(a.wt, static_cast<long>(N) * K * 2);

  using Tile = UnitTile<N>;
  constexpr int CH = Tile::PER_LANE;
  struct Unit {
    u32x4_t x[KB], h[PK];
    u32x4_t eh[GRAD ? CH : 1], rs[RES ? CH : 1];   // epilogue operands, row-major
  };
  auto load_unit = [&](int u, Unit& d) {
    const long pix = static_cast<long>(u) * 16 + lr;
    const bool in = pix < m;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const uint32_t off = in ? static_cast<uint32_t>((pix * K + kb * 32 + lg * 8) * 2) : BUF_OOB;
      d.x[kb] = buf_load16(r_src, off);
      if constexpr (BWD) d.h[kb] = buf_load16(r_h, off);
    }
    if constexpr (GRAD) Tile::load_rows(r_eph, u, m, lane, d.eh);
    if constexpr (RES) Tile::load_rows(r_res, u, m, lane, d.rs);
  };
  const int W = gridDim.x * 4;
  int u = blockIdx.x * 4 + wave;
  Unit cur, nxt;
  if (u < units) load_unit(u, cur);

  Frag<T> wf[NB][KB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      Raw8<T> r;
      r.set(buf_load16(r_wt, static_cast<uint32_t>(((nb * 16 + lr) * K + kb * 32 + lg * 8) * 2)));
      wf[nb][kb].set(r);
    }
  // BN-backward constants of this lane's input channels, and the epilogue's
  // per-output-channel constants
  float pca[PK][8], pcb[PK][8], pcc[PK][8], pmu[PK][8];
  if constexpr (BWD) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int c = kb * 32 + lg * 8 + j;
        pca[kb][j] = a.pro_ca[c];
        pcb[kb][j] = a.pro_cb[c];
        pcc[kb][j] = a.pro_cc[c];
        pmu[kb][j] = a.pro_mean[c];
      }
  }
  float es[EN][4], esh[EN][4], emu[EN][4], ers[EN][4];
  if constexpr (GRAD) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = nb * 16 + lg * 4 + e;
        es[nb][e] = EP == EP_MASK ? a.ep_scale[c] : 0.f;
        esh[nb][e] = EP == EP_MASK ? a.ep_shift[c] : 0.f;
        emu[nb][e] = a.ep_mean[c];
        ers[nb][e] = a.ep_rstd[c];
      }
  }

  float sa[NB][4], sb[NB][4];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) sa[nb][e] = sb[nb][e] = 0.f;
  for (; u < units; u += W) {
    const int un = u + W;
    if (un < units) load_unit(un, nxt);
    Frag<T> xf[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      Raw8<T> r;
      r.set(cur.x[kb]);
      if constexpr (BWD) {
        Raw8<T> hr;
        hr.set(cur.h[kb]);
        float v[8], h[8];
        r.to_f32(v);
        hr.to_f32(h);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[j] = fmaf(pca[kb][j], v[j], fmaf(pcb[kb][j], h[j] - pmu[kb][j], pcc[kb][j]));
        r.from_f32(v);   // rounded to bf16, as the materialised gradient
      }
      xf[kb].set(r);
    }
    const long pix = static_cast<long>(u) * 16 + lr;
    const bool vm = pix < m;
    // epilogue operands to the MFMA layout: each lane reads back 4 channels of its pixel
    if constexpr (RES) otile[wave].park_rows(cur.rs, lane);
    if constexpr (GRAD) etile[wave].park_rows(cur.eh, lane);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) acc = mfma(wf[nb][kb], xf[kb], acc);
      float v[4] = {acc[0], acc[1], acc[2], acc[3]};
      if constexpr (RES) {
        const u32x2_t rw = otile[wave].get(lr, lg, nb);
        v[0] += __uint_as_float(rw.x << 16); v[1] += __uint_as_float(rw.x & 0xffff0000u);
        v[2] += __uint_as_float(rw.y << 16); v[3] += __uint_as_float(rw.y & 0xffff0000u);
      }
      float hl[4] = {0.f, 0.f, 0.f, 0.f};
      if constexpr (GRAD) {
        const u32x2_t hw = etile[wave].get(lr, lg, nb);
        hl[0] = __uint_as_float(hw.x << 16); hl[1] = __uint_as_float(hw.x & 0xffff0000u);
        hl[2] = __uint_as_float(hw.y << 16); hl[3] = __uint_as_float(hw.y & 0xffff0000u);
      }
      if constexpr (EP == EP_MASK) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = fmaf(es[nb][e], hl[e], esh[nb][e]) > 0.f ? v[e] : 0.f;
      }
      const uint32_t w0 = pack_bf16x2(v[0], v[1]), w1 = pack_bf16x2(v[2], v[3]);
      otile[wave].put(lr, lg, nb, w0, w1);
      if constexpr (GRAD) {
        // partials of the stored values
        v[0] = __uint_as_float(w0 << 16); v[1] = __uint_as_float(w0 & 0xffff0000u);
        v[2] = __uint_as_float(w1 << 16); v[3] = __uint_as_float(w1 & 0xffff0000u);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float g = vm ? v[e] : 0.f;
          sa[nb][e] += g;
          sb[nb][e] += g * ((hl[e] - emu[nb][e]) * ers[nb][e]);
        }
      }
    }
    otile[wave].store(r_out, u, m, lane);
    cur = nxt;
  }
  if constexpr (GRAD) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = sum16(sa[nb][e]), y = sum16(sb[nb][e]);
        if (lr == 0) {
          const int c = nb * 16 + lg * 4 + e;
          red[wave][0][c] = x;
          red[wave][1][c] = y;
        }
      }
    __syncthreads();
    for (int c = tid; c < N; c += 256) {
      float t1 = 0.f, t2 = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        t1 += red[w][0][c];
        t2 += red[w][1][c];
      }
      const long row = blockIdx.x;
      a.partials[(row * 2 + 0) * N + c] = t1;
      a.partials[(row * 2 + 1) * N + c] = t2;
    }
  }
}

// Persistent 3x3 / stride 1 / pad 1 conv for 32 -> 32 bf16 channels (the
// HBM-bound shapes: C/2 = 32 at 32x32 and 56x56).  A workgroup takes tiles
// g, g + G, g + 2G, ... of TH x TW output pixels; while the MFMAs of one tile
// run, the input patch of the next one is already in flight into registers, so
// loads, multiplies and stores of successive tiles overlap.  The 9 x 2 weight
// fragments stay in registers for the whole launch.  The MFMA is issued as
// D[cout][pixel] = W x patch^T, so each lane ends up with 4 consecutive output
// channels of one pixel and stores them directly (8 bytes).  Statistics are
// combined across the workgroup's tiles in registers (Chan's formula for the
// BN moments, plain fixed-order sums for the gradient partials) and written
// once per workgroup: partial row = blockIdx.x.
template <int TH, int TW, int EP, int PRO>
__global__ __launch_bounds__(256, 2) void conv32_kernel(ConvArgs a, int ntiles) {
  using T = bf16_t;
  constexpr int NR = TH * TW;                          // output pixels per tile
  constexpr int FM = (NR + 63) / 64;                   // 16-pixel fragments per wave
  constexpr int HTH = TH + 2, HTW = TW + 2, HPIX = HTH * HTW;
  constexpr int HP = 40;                               // bf16 per patch pixel (32 + 8 pad)
  constexpr int PATCH = HPIX * HP;
  constexpr int H_CHUNKS = (HPIX * 4 + 255) / 256;
  constexpr bool BWD = PRO == PRO_BWD;
  __shared__ __attribute__((aligned(16))) T lds[2 * PATCH];
  __shared__ float pro_tab[4][32];
  __shared__ float red[4][3][32];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int G = gridDim.x;
  // XCD-aware numbering: workgroups that share an L2 take neighbouring tiles
  const int g = (G % 8 == 0) ? (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8 : blockIdx.x;
  const int tiles_x = (a.w + TW - 1) / TW, tiles_y = (a.h + TH - 1) / TH;
  // Activations go through buffer resources: out-of-range offsets read zero
  // (halo padding) or drop the store (rows past the image), with no branches.
  const long in_bytes = static_cast<long>(a.n) * a.h * a.w * 64;
  const long out_bytes = static_cast<long>(a.m) * 64;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_proh = make_rsrc(BWD ? a.pro_h : a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_out = make_rsrc(a.out, out_bytes);
  const __amdgpu_buffer_rsrc_t r_eph = make_rsrc(a.ep_h != nullptr ? a.ep_h : a.out, out_bytes);
  const __amdgpu_buffer_rsrc_t r_res = make_rsrc(a.resid != nullptr ? a.resid : a.out,
                                                 a.resid != nullptr ? out_bytes : 0);

  if (tid < 32) {
    if constexpr (PRO == PRO_RELU) {
      pro_tab[0][tid] = a.pro_scale[tid];
      pro_tab[1][tid] = a.pro_shift[tid];
    } else if constexpr (BWD) {
      pro_tab[0][tid] = a.pro_ca[tid];
      pro_tab[1][tid] = a.pro_cb[tid];
      pro_tab[2][tid] = a.pro_cc[tid];
      pro_tab[3][tid] = a.pro_mean[tid];
    }
  }

  auto origin = [&](int t, int& img, int& p0, int& q0) {
    const int tx = t % tiles_x;
    const int ty = (t / tiles_x) % tiles_y;
    img = t / (tiles_x * tiles_y);
    p0 = ty * TH;
    q0 = tx * TW;
  };
  u32x4_t rh[H_CHUNKS];
  u32x4_t rhh[BWD ? H_CHUNKS : 1];
  uint32_t hvalid = 0;
  // Per-thread patch chunks are fixed: patch row/column and the element offset
  // relative to the tile origin.
  int ch_y[H_CHUNKS], ch_x[H_CHUNKS], ch_rel[H_CHUNKS];
#pragma unroll
  for (int i = 0; i < H_CHUNKS; ++i) {
    const int q = tid + 256 * i;
    const int hp = q >> 2, sub = q & 3;
    const int hy = hp / HTW, hx = hp - hy * HTW;
    ch_y[i] = hp < HPIX ? hy - 1 : -(1 << 20);   // rows past the patch never load
    ch_x[i] = hx - 1;
    ch_rel[i] = ((hy - 1) * a.w + (hx - 1)) * 32 + sub * 8;
  }
  auto load_patch = [&](int t) {
    int img, p0, q0;
    origin(t, img, p0, q0);
    const int tbase = ((img * a.h + p0) * a.w + q0) * 32;
    hvalid = 0;
#pragma unroll
    for (int i = 0; i < H_CHUNKS; ++i) {
      const int ih = p0 + ch_y[i], iw = q0 + ch_x[i];
      const bool ok = static_cast<unsigned>(ih) < static_cast<unsigned>(a.h) &&
                      static_cast<unsigned>(iw) < static_cast<unsigned>(a.w);
      const uint32_t off = ok ? static_cast<uint32_t>(tbase + ch_rel[i]) * 2u : BUF_OOB;
      rh[i] = buf_load16(r_src, off);
      if constexpr (BWD) rhh[i] = buf_load16(r_proh, off);
      hvalid |= ok ? 1u << i : 0u;
    }
  };
  auto park_patch = [&](int buf) {
    T* dst = lds + buf * PATCH;
#pragma unroll
    for (int i = 0; i < H_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int hp = q >> 2, sub = q & 3;
      if (hp >= HPIX) continue;
      u32x4_t v = rh[i];
      if constexpr (PRO != PRO_NONE) {
        Raw8<T> r, hr;
        r.w[0] = v.x; r.w[1] = v.y; r.w[2] = v.z; r.w[3] = v.w;
        if constexpr (BWD) {
          hr.w[0] = rhh[i].x; hr.w[1] = rhh[i].y; hr.w[2] = rhh[i].z; hr.w[3] = rhh[i].w;
        }
        pro8<T, PRO>(r, hr, pro_tab[0], pro_tab[1], pro_tab[BWD ? 2 : 0], pro_tab[BWD ? 3 : 0],
                     sub * 8);
        const bool ok = (hvalid >> i) & 1u;   // padding stays zero
        v = u32x4_t{ok ? r.w[0] : 0u, ok ? r.w[1] : 0u, ok ? r.w[2] : 0u, ok ? r.w[3] : 0u};
      }
      *reinterpret_cast<u32x4_t*>(dst + hp * HP + sub * 8) = v;
    }
  };

  // Weight fragments: lane (lr, lg) holds output channel fn*16 + lr, inputs lg*8..+7 of tap.
  Frag<T> wf[9][2];
  {
    const T* wt = static_cast<const T*>(a.wt);
#pragma unroll
    for (int tap = 0; tap < 9; ++tap)
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) wf[tap][fn].load(wt + (fn * 16 + lr) * a.k_tot + tap * 32 + lg * 8);
  }
  // Loads are unconditional (a workgroup past the last tile, and the prefetch
  // after its last tile, re-read tile ntiles - 1) so that the number of loads in
  // flight is the same on every path and the waits stay tight.
  int t = g;
  load_patch(min(t, ntiles - 1));
  if constexpr (PRO != PRO_NONE) __syncthreads();   // prologue table
  // Patch offset of each fragment's pixel lr (tap (0,0)); rows past NR are padding.
  int rowpix[FM], rowi[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int i = (wave * FM + fm) * 16 + lr;
    rowi[fm] = i;
    const int ii = i < NR ? i : 0;
    const int ph = ii / TW, pw = ii - ph * TW;
    rowpix[fm] = ph * HTW + pw;
  }
  // This lane's 8 output channels: fn*16 + lg*4 + e.
  float es[2][4], esh[2][4], emu[2][4], ers[2][4];
  if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
#pragma unroll
    for (int fn = 0; fn < 2; ++fn)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = fn * 16 + lg * 4 + e;
        es[fn][e] = EP == EP_MASK ? a.ep_scale[c] : 0.f;
        esh[fn][e] = EP == EP_MASK ? a.ep_shift[c] : 0.f;
        emu[fn][e] = a.ep_mean[c];
        ers[fn][e] = a.ep_rstd[c];
      }
  }
  // Running per-lane statistics.  EP_STATS: count and sums of (v - K), (v - K)^2
  // with K a per-channel shift taken from the first tile (keeps the moments
  // free of cancellation); gradient epilogues: sums of g and g*xhat.
  float st_n = 0.f, st_a[2][4], st_b[2][4], st_k[2][4];
  bool have_k = false;
#pragma unroll
  for (int fn = 0; fn < 2; ++fn)
#pragma unroll
    for (int e = 0; e < 4; ++e) st_a[fn][e] = st_b[fn][e] = st_k[fn][e] = 0.f;

  int buf = 0;
  for (; t < ntiles; t += G) {
    park_patch(buf);
    __syncthreads();
    int img, p0, q0;
    origin(t, img, p0, q0);
    load_patch(min(t + G, ntiles - 1));
    f32x4_t acc[FM][2];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) acc[fm][0] = acc[fm][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const T* pt = lds + buf * PATCH;
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int toff = (tap / 3) * HTW + (tap % 3);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        Frag<T> pb;
        pb.load(pt + (rowpix[fm] + toff) * HP + lg * 8);
        acc[fm][0] = mfma(wf[tap][0], pb, acc[fm][0]);
        acc[fm][1] = mfma(wf[tap][1], pb, acc[fm][1]);
      }
    }
    // Epilogue: lane holds channels fn*16 + lg*4 + e of pixel rowi[fm].
    bool vm[FM];
    uint32_t pix[FM];
    float nv = 0.f;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int i = rowi[fm];
      const int ii = i < NR ? i : 0;
      const int ph = ii / TW, pw = ii - ph * TW;
      vm[fm] = i < NR && p0 + ph < a.h && q0 + pw < a.w;
      pix[fm] = vm[fm] ? static_cast<uint32_t>(((img * a.h + p0 + ph) * a.w + q0 + pw) * 64) : BUF_OOB;
      nv += vm[fm] ? 1.f : 0.f;
    }
    float q[FM][2][4];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        float v[4] = {acc[fm][fn][0], acc[fm][fn][1], acc[fm][fn][2], acc[fm][fn][3]};
        // byte offset of channels fn*16 + lg*4 .. +3 (past the end for padding rows)
        const uint32_t boff = vm[fm] ? pix[fm] + (fn * 16 + lg * 4) * 2 : BUF_OOB;
        float hl[4] = {0.f, 0.f, 0.f, 0.f}, rv[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (EP == EP_MASK || EP == EP_RESID_STATS || EP == EP_RESID) {
          if constexpr (EP != EP_RESID) {
            const u32x2_t hw = buf_load8(r_eph, boff);
            hl[0] = __uint_as_float(hw.x << 16); hl[1] = __uint_as_float(hw.x & 0xffff0000u);
            hl[2] = __uint_as_float(hw.y << 16); hl[3] = __uint_as_float(hw.y & 0xffff0000u);
          }
          if constexpr (EP != EP_MASK) {
            // a null residual has a zero-sized resource: reads give zero
            const u32x2_t rw = buf_load8(r_res, boff);
            rv[0] = __uint_as_float(rw.x << 16); rv[1] = __uint_as_float(rw.x & 0xffff0000u);
            rv[2] = __uint_as_float(rw.y << 16); rv[3] = __uint_as_float(rw.y & 0xffff0000u);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if constexpr (EP == EP_MASK)
              v[e] = fmaf(es[fn][e], hl[e], esh[fn][e]) > 0.f ? v[e] : 0.f;
            else
              v[e] += rv[e];
          }
        }
        // one conversion per pair; statistics use the stored values
        const uint32_t w0 = pack_bf16x2(v[0], v[1]), w1 = pack_bf16x2(v[2], v[3]);
        buf_store8(u32x2_t{w0, w1}, r_out, boff);
        v[0] = __uint_as_float(w0 << 16); v[1] = __uint_as_float(w0 & 0xffff0000u);
        v[2] = __uint_as_float(w1 << 16); v[3] = __uint_as_float(w1 & 0xffff0000u);
        if constexpr (EP == EP_MASK || EP == EP_RESID_STATS) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float g = vm[fm] ? v[e] : 0.f;
            st_a[fn][e] += g;
            st_b[fn][e] += g * ((hl[e] - emu[fn][e]) * ers[fn][e]);
          }
        } else if constexpr (EP == EP_STATS) {
#pragma unroll
          for (int e = 0; e < 4; ++e) q[fm][fn][e] = vm[fm] ? v[e] : 0.f;
        }
      }
    }
    if constexpr (EP == EP_STATS) {
      if (!have_k) {
        // shift: the stored value of the wave's first pixel of this tile, per channel
#pragma unroll
        for (int fn = 0; fn < 2; ++fn)
#pragma unroll
          for (int e = 0; e < 4; ++e) st_k[fn][e] = __shfl(q[0][fn][e], lane & 48, 64);
        have_k = true;
      }
      st_n += nv;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < 2; ++fn)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float d = vm[fm] ? q[fm][fn][e] - st_k[fn][e] : 0.f;
            st_a[fn][e] += d;
            st_b[fn][e] = fmaf(d, d, st_b[fn][e]);
          }
    }
    buf ^= 1;
  }

  // Workgroup partials: lane sums over the 16 pixels lanes, then the four waves in order.
  if constexpr (EP != EP_RESID) {
    const float n16 = sum16(st_n);
#pragma unroll
    for (int fn = 0; fn < 2; ++fn)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = sum16(st_a[fn][e]), y = sum16(st_b[fn][e]);
        if constexpr (EP == EP_STATS) {
          // (count, mean, centred M2) of this wave from the shifted sums
          const float mean_d = n16 > 0.f ? x / n16 : 0.f;
          st_a[fn][e] = st_k[fn][e] + mean_d;
          st_b[fn][e] = n16 > 0.f ? fmaxf(y - x * mean_d, 0.f) : 0.f;
        } else {
          st_a[fn][e] = x;
          st_b[fn][e] = y;
        }
      }
    if (lr == 0) {
#pragma unroll
      for (int fn = 0; fn < 2; ++fn)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int c = fn * 16 + lg * 4 + e;
          red[wave][0][c] = n16;
          red[wave][1][c] = st_a[fn][e];
          red[wave][2][c] = st_b[fn][e];
        }
    }
    __syncthreads();
    if (tid < 32) {
      const int c = tid;
      float* pr = a.partials;
      const long row = static_cast<long>(blockIdx.x);
      if constexpr (EP == EP_STATS) {
        float n = 0.f, mean = 0.f, m2 = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float nb = red[w][0][c];
          if (nb > 0.f) {
            const float nn = n + nb, rb = nb / nn, d = red[w][1][c] - mean;
            mean += d * rb;
            m2 += red[w][2][c] + d * d * n * rb;
            n = nn;
          }
        }
        pr[(row * 3 + 0) * 32 + c] = n;
        pr[(row * 3 + 1) * 32 + c] = n * mean;
        pr[(row * 3 + 2) * 32 + c] = m2;
      } else {
        const float s1 = (red[0][1][c] + red[1][1][c]) + (red[2][1][c] + red[3][1][c]);
        const float s2 = (red[0][2][c] + red[1][2][c]) + (red[2][2][c] + red[3][2][c]);
        pr[(row * 2 + 0) * 32 + c] = s1;
        pr[(row * 2 + 1) * 32 + c] = s2;
      }
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

  ConvArgs ca{};  // reuse the gather helper
  ca.src = a.src; ca.src2 = a.src2; ca.c_split = a.c_split;
  ca.pro_scale = a.pro_scale; ca.pro_shift = a.pro_shift;
  ca.h = a.h; ca.w = a.w; ca.c_in = a.c_in; ca.stride = a.stride; ca.pad = a.pad;
  const bool dhb = a.dh_h != nullptr;
  float dk[4][8];
  dh_coeffs(a, o0 + a_og * 8, dk);

  for (int mb = m_begin; mb < m_end; mb += 32) {
    if (a_active) {
      const int m = mb + a_row;
      const int o = o0 + a_og * 8;
      Raw8<T> r;
      if (m < m_end && o < a.c_out) {
        r.load(dh + static_cast<long>(m) * a.c_out + o);
        if (dhb) dh_bwd8(r, static_cast<const T*>(a.dh_h) + static_cast<long>(m) * a.c_out + o, dk);
      } else {
        r.zero();
      }
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
      gather_a<T, PRO ? PRO_RELU : PRO_NONE>(ca, rp, kb_valid, fr, fs, cb, r);
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

// bf16 weight gradient, 64 rows per step: register prefetch one step ahead,
// double-buffered LDS, and each thread transposes a pair of rows into 32-bit
// LDS words (two consecutive m of one channel), so both operands become
// m-contiguous rows that feed MFMA directly.
template <int BO, int BK, bool PRO, bool CAT>
__global__ __launch_bounds__(256) void wgrad_staged_kernel(WgradArgs a) {
  using T = bf16_t;
  constexpr int RS = 64;                    // rows (m) per step
  constexpr int PITCH = RS + 8;             // bf16 per LDS row (144 B)
  constexpr int FO = BO / 32, FK = BK / 32;
  constexpr int A_TASKS = 32 * (BO / 8);    // (row pair, 8-channel group) tasks of dh
  constexpr int B_TASKS = 32 * (BK / 8);    // (row pair, 8-column group) tasks of the input
  static_assert(A_TASKS <= 256 && B_TASKS <= 256, "tile");
  constexpr int BUF = (BO + BK) * PITCH;
  __shared__ __attribute__((aligned(16))) T lds[2 * BUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wo = wave & 1, wk = wave >> 1;
  const int lr = lane & 15, lg = lane >> 4;
  const int k0 = blockIdx.x * BK, o0 = blockIdx.y * BO;
  const int m_begin = blockIdx.z * a.rows_per_split;
  const int m_end = min(a.m, m_begin + a.rows_per_split);
  const int steps = (m_end - m_begin + RS - 1) / RS;
  const int pq = a.p * a.q;
  const T* dh = static_cast<const T*>(a.dh);

  const bool a_on = tid < A_TASKS;
  const int a_pair = tid / (BO / 8), a_og = tid % (BO / 8);
  const int a_o = o0 + a_og * 8;
  const bool a_ook = a_on && a_o < a.c_out;
  const bool b_on = tid < B_TASKS;
  const int b_pair = tid / (BK / 8), b_kg = tid % (BK / 8);
  const int kb = k0 + b_kg * 8;
  const bool kb_ok = b_on && kb < a.k_tot;
  const int kbb = kb_ok ? kb : 0;
  const int tap = kbb / a.c_in;
  const int cb = kbb - tap * a.c_in;
  const int fr = tap / a.s, fs = tap - fr * a.s;

  ConvArgs ca{};
  ca.src = a.src; ca.src2 = a.src2; ca.c_split = a.c_split;
  ca.pro_scale = a.pro_scale; ca.pro_shift = a.pro_shift;
  ca.h = a.h; ca.w = a.w; ca.c_in = a.c_in; ca.stride = a.stride; ca.pad = a.pad;
  const bool dhb = a.dh_h != nullptr;
  float dk[4][8];
  dh_coeffs(a, a_o, dk);

  Raw8<T> ra[2], rb[2], rah[2];
  uint32_t aval = 0, bval = 0;
  // Without a concatenated second input, operands come through buffer
  // resources: rows past the split, padding and channels past the end load
  // zeros without branches, so the next step's loads stay in flight.  The
  // BN-backward (dh) and BN-apply + ReLU prologues run when the step is parked.
  const long in_bytes = static_cast<long>(a.n) * a.h * a.w * a.c_split * 2;
  const long out_bytes = static_cast<long>(a.m) * a.c_out * 2;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_dh = make_rsrc(a.dh, out_bytes);
  const __amdgpu_buffer_rsrc_t r_dhh = make_rsrc(dhb ? a.dh_h : a.dh, out_bytes);
  auto load_step = [&](int step) {
    const int mb = m_begin + step * RS;
    aval = bval = 0;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int m = mb + 2 * a_pair + e;
      const int mm = mb + 2 * b_pair + e;
      if constexpr (!CAT) {
        const bool oka = a_ook && m < m_end;
        const uint32_t offa = oka ? static_cast<uint32_t>((static_cast<long>(m) * a.c_out + a_o) * 2) : BUF_OOB;
        ra[e].set(buf_load16(r_dh, offa));
        rah[e].set(buf_load16(r_dhh, offa));
        aval |= oka ? 1u << e : 0u;
        const bool vb = b_on && mm < m_end;
        const int m2 = vb ? mm : 0;
        const int n = m2 / pq;
        const int rem = m2 - n * pq;
        const int pp = rem / a.q, qq = rem - pp * a.q;
        const int ih = pp * a.stride + fr - a.pad, iw = qq * a.stride + fs - a.pad;
        const bool okb = vb && kb_ok && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
        const uint32_t offb =
            okb ? static_cast<uint32_t>((((static_cast<long>(n) * a.h + ih) * a.w + iw) * a.c_split + cb) * 2) : BUF_OOB;
        rb[e].set(buf_load16(r_src, offb));
        bval |= okb ? 1u << e : 0u;
      } else {
        if (a_ook && m < m_end) {
          ra[e].load(dh + static_cast<long>(m) * a.c_out + a_o);
          if (dhb) dh_bwd8(ra[e], static_cast<const T*>(a.dh_h) + static_cast<long>(m) * a.c_out + a_o, dk);
        } else {
          ra[e].zero();
        }
        RowPos rp;
        rp.valid = b_on && mm < m_end;
        const int m2 = rp.valid ? mm : 0;
        rp.n = m2 / pq;
        const int rem = m2 - rp.n * pq;
        rp.p = rem / a.q;
        rp.q = rem - rp.p * a.q;
        gather_a<T, PRO ? PRO_RELU : PRO_NONE>(ca, rp, kb_ok, fr, fs, cb, rb[e]);
      }
    }
  };
  float bsc[8], bsh[8];   // BN-apply of this thread's 8 input channels (fixed)
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    bsc[j] = PRO && !CAT && kb_ok ? a.pro_scale[cb + j] : 0.f;
    bsh[j] = PRO && !CAT && kb_ok ? a.pro_shift[cb + j] : 0.f;
  }
  auto pro_step = [&]() {
    if constexpr (!CAT) {
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        if (dhb) {
          float v[8], h[8];
          ra[e].to_f32(v);
          rah[e].to_f32(h);
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = fmaf(dk[0][j], v[j], fmaf(dk[1][j], h[j] - dk[3][j], dk[2][j]));
          ra[e].from_f32(v);
          if (!((aval >> e) & 1u)) ra[e].zero();
        }
        if constexpr (PRO) {
          float v[8];
          rb[e].to_f32(v);
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = fmaxf(fmaf(bsc[j], v[j], bsh[j]), 0.f);
          rb[e].from_f32(v);
          if (!((bval >> e) & 1u)) rb[e].zero();
        }
      }
    }
  };
  auto pair_word = [](const Raw8<T>& lo, const Raw8<T>& hi, int j) -> uint32_t {
    const uint32_t a0 = lo.w[j >> 1], b0 = hi.w[j >> 1];
    return (j & 1) ? ((a0 >> 16) | (b0 & 0xffff0000u)) : ((a0 & 0xffffu) | (b0 << 16));
  };
  auto park = [&](int buf) {
    T* sA = lds + buf * BUF;
    T* sB = sA + BO * PITCH;
    if (a_on) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        *reinterpret_cast<uint32_t*>(sA + (a_og * 8 + j) * PITCH + 2 * a_pair) = pair_word(ra[0], ra[1], j);
    }
    if (b_on) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        *reinterpret_cast<uint32_t*>(sB + (b_kg * 8 + j) * PITCH + 2 * b_pair) = pair_word(rb[0], rb[1], j);
    }
  };

  f32x4_t acc[FO][FK];
#pragma unroll
  for (int i = 0; i < FO; ++i)
#pragma unroll
    for (int j = 0; j < FK; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (steps > 0) {
    load_step(0);
    pro_step();
    park(0);
  }
  __syncthreads();
  for (int step = 0; step < steps; ++step) {
    const int buf = step & 1;
    if (step + 1 < steps) load_step(step + 1);
    const T* sA = lds + buf * BUF;
    const T* sB = sA + BO * PITCH;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      Frag<T> fa[FO], fb[FK];
#pragma unroll
      for (int i = 0; i < FO; ++i) fa[i].load(sA + (wo * (BO / 2) + i * 16 + lr) * PITCH + kk * 32 + lg * 8);
#pragma unroll
      for (int j = 0; j < FK; ++j) fb[j].load(sB + (wk * (BK / 2) + j * 16 + lr) * PITCH + kk * 32 + lg * 8);
#pragma unroll
      for (int i = 0; i < FO; ++i)
#pragma unroll
        for (int j = 0; j < FK; ++j) acc[i][j] = mfma(fa[i], fb[j], acc[i][j]);
    }
    if (step + 1 < steps) {
      pro_step();
      park(buf ^ 1);
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

// Halo-tile weight gradient for 3x3 / stride 1 / pad 1 bf16 convolutions with
// C_in a multiple of 32:
//   part[split][o][(tap, c)] = sum over the split's pixels of dh[pix][o] * x[pix + tap][c]
// A workgroup owns one output-channel tile (BO), one 32-channel input chunk
// and a strided set of TH x TW pixel tiles.  Per pixel tile it stores dh
// transposed ([o][pixel]) and the (TH+2)-row input patch transposed three
// times, pre-shifted by 0, 1 and 2 columns ([c][row][col + s]), so that the
// MFMA operands of every tap are 16-byte aligned LDS rows.  The BN-apply +
// ReLU prologue runs once per patch element.  The next tile is fetched into
// registers while the current one is multiplied; the 9 taps accumulate in
// registers across all tiles of the split.
template <int TH, int TW, int BO, bool PRO>
__global__ __launch_bounds__(256) void wgrad_halo_kernel(WgradArgs a) {
  using T = bf16_t;
  constexpr int NPIX = TH * TW;
  static_assert(NPIX % 32 == 0 && TW % 8 == 0 && 256 % (BO / 8) == 0, "tile");
  constexpr int HTH = TH + 2, HTW = TW + 2, HPIX = HTH * HTW;
  constexpr int HROW = HTH * TW + 8;        // bf16 per channel row of one shifted copy
  constexpr int DROW = NPIX + 8;            // bf16 per output-channel row of dh^T
  constexpr int OT = BO / 16;               // output-channel MFMA tiles
  constexpr int WPO = 4 / OT;               // waves per output-channel tile
  constexpr int NP = 18 / WPO;              // (tap, 16-channel half) pairs per wave
  static_assert(OT * WPO == 4 && NP * WPO == 18, "waves");
  constexpr int H_CHUNKS = (HPIX * 4 + 255) / 256;
  constexpr int D_CHUNKS = (NPIX * (BO / 8) + 255) / 256;
  __shared__ __attribute__((aligned(16))) T sh[3 * 32 * HROW];
  __shared__ __attribute__((aligned(16))) T sd[BO * DROW];
  __shared__ float pro_tab[2][32];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int ot = wave % OT, part = wave / OT;
  const int o0 = blockIdx.y * BO;
  const int chunk = blockIdx.z;
  const int c0 = chunk * 32;
  const int tiles_x = (a.w + TW - 1) / TW, tiles_y = (a.h + TH - 1) / TH;
  const int ntiles = tiles_x * tiles_y * a.n;

  if constexpr (PRO) {
    if (tid < 32) {
      pro_tab[0][tid] = a.pro_scale[c0 + tid];
      pro_tab[1][tid] = a.pro_shift[c0 + tid];
    }
    __syncthreads();
  }

  const bool dhb = a.dh_h != nullptr;
  float dk[4][8];
  dh_coeffs(a, o0 + (tid % (BO / 8)) * 8, dk);   // this thread's output-channel group is fixed
  // Buffer resources: padding and rows past the image load zeros without
  // branches, so the next tile's loads stay in flight during the MFMAs.
  const long in_bytes = static_cast<long>(a.n) * a.h * a.w * a.c_in * 2;
  const long out_bytes = static_cast<long>(a.m) * a.c_out * 2;
  const __amdgpu_buffer_rsrc_t r_src = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_dh = make_rsrc(a.dh, out_bytes);
  const __amdgpu_buffer_rsrc_t r_dhh = make_rsrc(dhb ? a.dh_h : a.dh, out_bytes);
  Raw8<T> rh[H_CHUNKS], rd[D_CHUNKS], rdh[D_CHUNKS];
  uint32_t hval = 0, dval = 0;
  auto tile_origin = [&](int t, int& img, int& p0, int& q0) {
    const int tx = t % tiles_x;
    const int ty = (t / tiles_x) % tiles_y;
    img = t / (tiles_x * tiles_y);
    p0 = ty * TH;
    q0 = tx * TW;
  };
  auto load_tile = [&](int t) {
    int img, p0, q0;
    tile_origin(t, img, p0, q0);
    const long base = static_cast<long>(img) * a.h * a.w;
    hval = dval = 0;
#pragma unroll
    for (int i = 0; i < H_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int hp = q >> 2, sub = q & 3;
      const int hy = hp / HTW, hx = hp - hy * HTW;
      const int ih = p0 - 1 + hy, iw = q0 - 1 + hx;
      const bool ok = hp < HPIX && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
      const uint32_t off =
          ok ? static_cast<uint32_t>(((base + static_cast<long>(ih) * a.w + iw) * a.c_in + c0 + sub * 8) * 2)
             : BUF_OOB;
      rh[i].set(buf_load16(r_src, off));
      hval |= ok ? 1u << i : 0u;
    }
#pragma unroll
    for (int i = 0; i < D_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int pix = q / (BO / 8), og = q % (BO / 8);
      const int ph = pix / TW, pw = pix - ph * TW;
      const int pp = p0 + ph, qq = q0 + pw;
      const bool ok = pix < NPIX && pp < a.h && qq < a.w && o0 + og * 8 < a.c_out;
      const uint32_t off =
          ok ? static_cast<uint32_t>(((base + static_cast<long>(pp) * a.w + qq) * a.c_out + o0 + og * 8) * 2)
             : BUF_OOB;
      rd[i].set(buf_load16(r_dh, off));
      rdh[i].set(buf_load16(r_dhh, off));
      dval |= ok ? 1u << i : 0u;
    }
  };
  // Prologues on the landed registers (padding stays zero), then the
  // transposed LDS layout.
  auto park_tile = [&]() {
#pragma unroll
    for (int i = 0; i < H_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int hp = q >> 2, sub = q & 3;
      if (hp >= HPIX) continue;
      if constexpr (PRO) {
        float v[8];
        rh[i].to_f32(v);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[j] = fmaxf(fmaf(pro_tab[0][sub * 8 + j], v[j], pro_tab[1][sub * 8 + j]), 0.f);
        rh[i].from_f32(v);
        if (!((hval >> i) & 1u)) rh[i].zero();
      }
      const int hy = hp / HTW, hx = hp - hy * HTW;
#pragma unroll
      for (int sft = 0; sft < 3; ++sft) {
        const int col = hx - sft;
        if (col < 0 || col >= TW) continue;
        T* dst = sh + sft * 32 * HROW + hy * TW + col;
#pragma unroll
        for (int j = 0; j < 8; ++j) rh[i].put(j, dst + (sub * 8 + j) * HROW);
      }
    }
#pragma unroll
    for (int i = 0; i < D_CHUNKS; ++i) {
      const int q = tid + 256 * i;
      const int pix = q / (BO / 8), og = q % (BO / 8);
      if (pix >= NPIX) continue;
      if (dhb) {
        Raw8<T> r = rd[i];
        float v[8], h[8];
        r.to_f32(v);
        rdh[i].to_f32(h);
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = fmaf(dk[0][j], v[j], fmaf(dk[1][j], h[j] - dk[3][j], dk[2][j]));
        r.from_f32(v);
        if (!((dval >> i) & 1u)) r.zero();
        rd[i] = r;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) rd[i].put(j, sd + (og * 8 + j) * DROW + pix);
    }
  };

  f32x4_t acc[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Loads are unconditional (the prefetch after the last tile re-reads tile
  // ntiles - 1) so the number of loads in flight is the same on every path.
  int t = blockIdx.x;
  load_tile(min(t, ntiles - 1));
  for (; t < ntiles; t += gridDim.x) {
    __syncthreads();            // previous tile's operands fully consumed
    park_tile();
    __syncthreads();
    load_tile(min(t + static_cast<int>(gridDim.x), ntiles - 1));
#pragma unroll
    for (int g = 0; g < NPIX / 32; ++g) {
      const int pix = g * 32 + lg * 8;
      const int ph = pix / TW, pw = pix - ph * TW;
      Frag<T> fa;
      fa.load(sd + (ot * 16 + lr) * DROW + pix);
#pragma unroll
      for (int pi = 0; pi < NP; ++pi) {
        const int pr = part + pi * WPO;          // 0..17
        const int tap = pr >> 1, half = pr & 1;
        const int fr = tap / 3, fs = tap - fr * 3;
        Frag<T> fb;
        fb.load(sh + fs * 32 * HROW + (half * 16 + lr) * HROW + (ph + fr) * TW + pw);
        acc[pi] = mfma(fa, fb, acc[pi]);
      }
    }
  }

  float* outp = a.partials + static_cast<long>(blockIdx.x) * a.c_out * a.k_tot;
#pragma unroll
  for (int pi = 0; pi < NP; ++pi) {
    const int pr = part + pi * WPO;
    const int tap = pr >> 1, half = pr & 1;
    const int k = tap * a.c_in + c0 + half * 16 + lr;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int o = o0 + ot * 16 + lg * 4 + e;
      if (o < a.c_out) outp[static_cast<long>(o) * a.k_tot + k] = acc[pi][e];
    }
  }
}

// Weight gradient on transposing LDS reads (gfx950 ds_read_b64_tr_b16):
//   part[split][o][tap*C_in + c] = sum over the split's pixels of dh[px][o] * x[px + tap][c]
// Both MFMA operands need pixels along the reduction, but the tensors are
// channel-contiguous.  The tiles stay in LDS exactly as loaded ([pixel][channel]);
// each operand fragment is two transposing reads: in a group of 16 lanes, lane
// 4r + q supplies the address of 4 channels (q-th quarter of a 16-channel run)
// of pixel r, and lane j receives channel j of the 4 pixels.  A workgroup owns
// BO output x BC input channels and all R*R taps, and sums a strided set of
// TH x TW pixel tiles; the next tile is in flight while the current one is
// multiplied (double-buffered LDS, one barrier per tile).  Waves split the
// output: WO x WC channel blocks of OF x CF fragments, and WT groups of taps.
template <int R, int TH, int TW, int WO, int OF, int WC, int CF, int WT, int WP, bool DH>
__device__ __forceinline__ void wgrad_tr_body(const WgradArgs& a, int bx, int by, int bz,
                                              int splits, int nbz) {
  const bool PRO = a.pro_scale != nullptr;   // BN-apply + ReLU prologue of the conv input
  using T = bf16_t;
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  constexpr int NW = WO * WC * WT;                    // waves of one pixel group
  constexpr int NT = 64 * NW * WP;
  constexpr int TAPS = R * R, TPW = TAPS / WT;
  static_assert(TPW * WT == TAPS, "taps per wave");
  constexpr int BO = WO * OF * 16, BC = WC * CF * 16;
  constexpr int NPIX = TH * TW;
  static_assert(NPIX % (32 * WP) == 0, "pixel tile");
  constexpr int KSTEPS = NPIX / 32 / WP;             // k-steps per pixel group and tile
  constexpr int PAD = R / 2;
  constexpr int HTH = TH + 2 * PAD, HTW = TW + 2 * PAD, HPIX = HTH * HTW;
  constexpr int PO = BO + 16, PC = BC + 16;          // LDS row pitches (bf16)
  constexpr int DG = BO / 8, XG = BC / 8;            // 16-byte groups per row
  static_assert(NT % DG == 0 && NT % XG == 0, "fixed channel group per thread");
  constexpr int D_PT = (NPIX * DG + NT - 1) / NT;
  constexpr int X_PT = (HPIX * XG + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) T sd[2][NPIX * PO];
  __shared__ __attribute__((aligned(16))) T sx[2][HPIX * PC];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wo = wave % WO, wc = (wave / WO) % WC, wt = (wave / (WO * WC)) % WT;
  const int wp = wave / NW;   // pixel group: k-steps wp, wp + WP, ... of each tile
  const int li = lane & 15, kg = lane >> 4;
  const int o0 = by * BO, c0 = bz * BC;
  // 1x1: no halo; tiles are runs of NPIX consecutive pixels of the flat [m] index
  constexpr bool FLAT = R == 1;
  const int tiles_x = (a.w + TW - 1) / TW, tiles_y = (a.h + TH - 1) / TH;
  const int ntiles = FLAT ? (a.m + NPIX - 1) / NPIX : tiles_x * tiles_y * a.n;

  const long in_bytes = static_cast<long>(a.n) * a.h * a.w * a.c_in * 2;
  const long out_bytes = static_cast<long>(a.m) * a.c_out * 2;
  const __amdgpu_buffer_rsrc_t r_x = make_rsrc(a.src, in_bytes);
  const __amdgpu_buffer_rsrc_t r_d = make_rsrc(a.dh, out_bytes);
  const __amdgpu_buffer_rsrc_t r_h = make_rsrc(DH ? a.dh_h : a.dh, out_bytes);

  // Fixed channel groups of this thread and their prologue coefficients.
  const int og = tid % DG, cg = tid % XG;
  float dk[4][8], xs[8], xsh[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int o = o0 + og * 8 + j, c = c0 + cg * 8 + j;
    dk[0][j] = DH ? a.dh_ca[o] : 0.f;
    dk[1][j] = DH ? a.dh_cb[o] : 0.f;
    dk[2][j] = DH ? a.dh_cc[o] : 0.f;
    dk[3][j] = DH ? a.dh_mean[o] : 0.f;
    xs[j] = PRO ? a.pro_scale[c] : 0.f;
    xsh[j] = PRO ? a.pro_shift[c] : 0.f;
  }

  Raw8<T> rd[D_PT], rdh[DH ? D_PT : 1], rx[X_PT];
  uint32_t dval = 0, xval = 0;
  auto load_tile = [&](int t) {
    const int tx = t % tiles_x, ty = (t / tiles_x) % tiles_y, img = t / (tiles_x * tiles_y);
    const int p0 = ty * TH, q0 = tx * TW;
    dval = xval = 0;
#pragma unroll
    for (int i = 0; i < D_PT; ++i) {
      const int px = (tid + NT * i) / DG;
      const int pp = p0 + px / TW, qq = q0 + px % TW;
      const long m = FLAT ? static_cast<long>(t) * NPIX + px : (static_cast<long>(img) * a.h + pp) * a.w + qq;
      const bool ok = px < NPIX && (FLAT ? m < a.m : pp < a.h && qq < a.w);
      const uint32_t off = ok ? static_cast<uint32_t>((m * a.c_out + o0 + og * 8) * 2) : BUF_OOB;
      rd[i].set(buf_load16(r_d, off));
      if constexpr (DH) rdh[i].set(buf_load16(r_h, off));
      dval |= ok ? 1u << i : 0u;
    }
#pragma unroll
    for (int i = 0; i < X_PT; ++i) {
      const int hp = (tid + NT * i) / XG;
      const int ih = p0 - PAD + hp / HTW, iw = q0 - PAD + hp % HTW;
      const long m = FLAT ? static_cast<long>(t) * NPIX + hp : (static_cast<long>(img) * a.h + ih) * a.w + iw;
      const bool ok = hp < HPIX && (FLAT ? m < a.m : ih >= 0 && ih < a.h && iw >= 0 && iw < a.w);
      const uint32_t off = ok ? static_cast<uint32_t>((m * a.c_in + c0 + cg * 8) * 2) : BUF_OOB;
      rx[i].set(buf_load16(r_x, off));
      xval |= ok ? 1u << i : 0u;
    }
  };
  auto park_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < D_PT; ++i) {
      const int px = (tid + NT * i) / DG;
      if (px >= NPIX) continue;
      Raw8<T> r = rd[i];
      if constexpr (DH) {
        float v[8], h[8];
        r.to_f32(v);
        rdh[i].to_f32(h);
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = fmaf(dk[0][j], v[j], fmaf(dk[1][j], h[j] - dk[3][j], dk[2][j]));
        r.from_f32(v);
        if (!((dval >> i) & 1u)) r.zero();
      }
      *reinterpret_cast<uint4*>(&sd[buf][px * PO + og * 8]) = make_uint4(r.w[0], r.w[1], r.w[2], r.w[3]);
    }
#pragma unroll
    for (int i = 0; i < X_PT; ++i) {
      const int hp = (tid + NT * i) / XG;
      if (hp >= HPIX) continue;
      Raw8<T> r = rx[i];
      if (PRO) {
        float v[8];
        r.to_f32(v);
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = fmaxf(fmaf(xs[j], v[j], xsh[j]), 0.f);
        r.from_f32(v);
        if (!((xval >> i) & 1u)) r.zero();   // padding stays zero
      }
      *reinterpret_cast<uint4*>(&sx[buf][hp * PC + cg * 8]) = make_uint4(r.w[0], r.w[1], r.w[2], r.w[3]);
    }
  };
  // two transposing reads give one bf16 MFMA operand: 8 pixels x one channel
  auto tr_frag = [](const T* p0, const T* p1) {
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4i16*)(p0));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4i16*)(p1));
    Frag<T> f;
    f.v = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    return f;
  };

  // Per-lane LDS offsets of the transposing reads (independent of the tile):
  // rows kg*8 + (li>>2) (+4) of k-step ks, quarter (li&3) of the 16-channel run.
  int da[KSTEPS], xa[KSTEPS], xb[KSTEPS];
#pragma unroll
  for (int ks = 0; ks < KSTEPS; ++ks) {
    const int pa = (ks * WP + wp) * 32 + kg * 8 + (li >> 2), pb = pa + 4;
    const int qo = (li & 3) * 4;
    da[ks] = pa * PO + wo * OF * 16 + qo;
    xa[ks] = ((pa / TW) * HTW + pa % TW) * PC + wc * CF * 16 + qo;
    xb[ks] = ((pb / TW) * HTW + pb % TW) * PC + wc * CF * 16 + qo;
  }
  // LDS offsets of this wave's taps (patch row/column shift), in elements
  int u_off[TPW];
#pragma unroll
  for (int u = 0; u < TPW; ++u) {
    const int tap = wt * TPW + u;
    u_off[u] = ((tap / R) * HTW + tap % R) * PC;
  }

  f32x4_t acc[OF][CF][TPW];
#pragma unroll
  for (int of = 0; of < OF; ++of)
#pragma unroll
    for (int cf = 0; cf < CF; ++cf)
#pragma unroll
      for (int u = 0; u < TPW; ++u) acc[of][cf][u] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Loads are unconditional (re-reading the last tile past the end) so the
  // number of loads in flight does not depend on the path.
  int t = bx;
  load_tile(min(t, ntiles - 1));
  int buf = 0;
  for (; t < ntiles; t += splits) {
    park_tile(buf);
    __syncthreads();
    load_tile(min(t + splits, ntiles - 1));
    const T* sdb = sd[buf];
    const T* sxb = sx[buf];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      Frag<T> fa[OF];
#pragma unroll
      for (int of = 0; of < OF; ++of)
        fa[of] = tr_frag(sdb + da[ks] + of * 16, sdb + da[ks] + 4 * PO + of * 16);
#pragma unroll
      for (int u = 0; u < TPW; ++u) {
        const int toff = u_off[u];
#pragma unroll
        for (int cf = 0; cf < CF; ++cf) {
          const Frag<T> fb = tr_frag(sxb + xa[ks] + toff + cf * 16, sxb + xb[ks] + toff + cf * 16);
#pragma unroll
          for (int of = 0; of < OF; ++of) acc[of][cf][u] = mfma(fa[of], fb, acc[of][cf][u]);
        }
      }
    }
    buf ^= 1;
  }

  // Pixel groups 1.. add their sums into group 0 through LDS, one group per
  // round (fixed order).
  constexpr int NFRAG = OF * CF * TPW;
  if constexpr (WP > 1) {
    f32x4_t* xch = reinterpret_cast<f32x4_t*>(&sx[0][0]);   // tiles are no longer read
    static_assert(NW * NFRAG * 64 * 16 <= static_cast<int>(sizeof(sx)), "exchange space");
#pragma unroll
    for (int g = 1; g < WP; ++g) {
      __syncthreads();
      if (wp == g) {
#pragma unroll
        for (int of = 0; of < OF; ++of)
#pragma unroll
          for (int cf = 0; cf < CF; ++cf)
#pragma unroll
            for (int u = 0; u < TPW; ++u)
              xch[((wave % NW) * NFRAG + (of * CF + cf) * TPW + u) * 64 + lane] = acc[of][cf][u];
      }
      __syncthreads();
      if (wp == 0) {
#pragma unroll
        for (int of = 0; of < OF; ++of)
#pragma unroll
          for (int cf = 0; cf < CF; ++cf)
#pragma unroll
            for (int u = 0; u < TPW; ++u)
              acc[of][cf][u] += xch[(wave * NFRAG + (of * CF + cf) * TPW + u) * 64 + lane];
      }
    }
    if (wp > 0) return;
  }
  // Partials in fragment order: every (wave, fragment) owns 256 consecutive
  // floats, lane l at 4 l .. 4 l + 3, so each wave writes whole cache lines;
  // wgrad_tr_reduce maps them back to [o][k].
  const long wg_base = (static_cast<long>(by) * nbz + bz) * NW + wave;
  float* outp = a.partials + static_cast<long>(bx) * a.c_out * a.k_tot;
#pragma unroll
  for (int of = 0; of < OF; ++of)
#pragma unroll
    for (int cf = 0; cf < CF; ++cf)
#pragma unroll
      for (int u = 0; u < TPW; ++u) {
        const long blk = ((wg_base * OF + of) * CF + cf) * TPW + u;
        *reinterpret_cast<f32x4_t*>(outp + blk * 256 + lane * 4) = acc[of][cf][u];
      }
}

template <int R, int TH, int TW, int WO, int OF, int WC, int CF, int WT, int WP, bool DH>
__global__ __launch_bounds__(64 * WO * WC * WT * WP) void wgrad_tr_kernel(WgradArgs a) {
  wgrad_tr_body<R, TH, TW, WO, OF, WC, CF, WT, WP, DH>(a, blockIdx.x, blockIdx.y, blockIdx.z,
                                                       gridDim.x, gridDim.z);
}

// Several layers' weight gradients (same configuration) in one launch: block b
// belongs to the last entry whose first block is <= b; within an entry blocks
// run over (split, output block, input block) as the single-layer grid does.
template <int R, int TH, int TW, int WO, int OF, int WC, int CF, int WT, int WP, bool DH>
__global__ __launch_bounds__(64 * WO * WC * WT * WP) void wgrad_tr_group_kernel(WgGroupTable tab) {
  constexpr int BO = WO * OF * 16, BC = WC * CF * 16;
  const long b = blockIdx.x;
  int i = 0;
  for (int e = 1; e < tab.n; ++e)
    if (tab.block_begin[e] <= b) i = e;
  const WgradArgs& a = tab.a[i];
  const long local = b - tab.block_begin[i];
  const int nby = a.c_out / BO, nbz = a.c_in / BC;
  const int bx = static_cast<int>(local % a.splits);
  const long r = local / a.splits;
  wgrad_tr_body<R, TH, TW, WO, OF, WC, CF, WT, WP, DH>(a, bx, static_cast<int>(r % nby),
                                                       static_cast<int>(r / nby), a.splits, nbz);
}

// Fixed-order sum over the splits of the fragment-ordered partials of
// wgrad_tr_kernel, scaled by inv_k and added to grad[o][k].  One thread per
// lane-quad (4 consecutive partial floats = 4 output channels of one k).
// Reduce of fragment-ordered partials: 16 quads per block; the 16 thread rows
// take splits r, r + 16, ... and the row sums are combined in a fixed order.
// blk is the block's index within its layer's partials.
__device__ __forceinline__ void tr_reduce_block(const float* __restrict__ part, int splits,
                                                long numel, const TrMap& mp, float inv_k,
                                                float* __restrict__ grad, long blk_index) {
  __shared__ f32x4_t red[16][17];
  const int tq = threadIdx.x & 15, tr = threadIdx.x >> 4;
  const long q = blk_index * 16 + tq;   // quad index
  const bool live = q * 4 < numel;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  if (live) {
    int sp = tr;
    for (; sp + 48 < splits; sp += 64) {
      f32x4_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const f32x4_t*>(part + (sp + 16 * u) * numel + q * 4);
#pragma unroll
      for (int u = 0; u < 4; ++u) acc += v[u];
    }
    for (; sp < splits; sp += 16) acc += *reinterpret_cast<const f32x4_t*>(part + sp * numel + q * 4);
  }
  red[tr][tq] = acc;
  __syncthreads();
  if (tr != 0 || !live) return;
#pragma unroll
  for (int r = 1; r < 16; ++r) acc += red[r][tq];
  // decode (block, lane) -> (o, k)
  const int lane = static_cast<int>(q & 63);
  long blk = q >> 6;
  const int u = static_cast<int>(blk % mp.tpw); blk /= mp.tpw;
  const int cf = static_cast<int>(blk % mp.cf); blk /= mp.cf;
  const int of = static_cast<int>(blk % mp.of); blk /= mp.of;
  const int nw = mp.wo * mp.wc * mp.wt;
  const int wave = static_cast<int>(blk % nw); blk /= nw;
  const int bz = static_cast<int>(blk % mp.nz), by = static_cast<int>(blk / mp.nz);
  const int wo = wave % mp.wo, wc = (wave / mp.wo) % mp.wc, wt = wave / (mp.wo * mp.wc);
  const int li = lane & 15, kg = lane >> 4;
  const int tap = wt * mp.tpw + u;
  const int k = tap * mp.c_in + bz * mp.bc + (wc * mp.cf + cf) * 16 + li;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int o = by * mp.bo + (wo * mp.of + of) * 16 + kg * 4 + e;
    grad[static_cast<long>(o) * mp.k_tot + k] += inv_k * acc[e];
  }
}

__global__ __launch_bounds__(256) void wgrad_tr_reduce_kernel(const float* __restrict__ part,
                                                              int splits, long numel, TrMap mp,
                                                              float inv_k, float* __restrict__ grad) {
  tr_reduce_block(part, splits, numel, mp, inv_k, grad, blockIdx.x);
}

// Several layers' reduces in one launch: block b belongs to the last segment
// whose first block is <= b (segments start on whole blocks).
__global__ __launch_bounds__(256) void wgrad_tr_reduce_group_kernel(TrSegTable tab,
                                                                    const float* __restrict__ base,
                                                                    float inv_k,
                                                                    float* __restrict__ grad_base) {
  const long b = blockIdx.x;
  int sidx = 0;
  for (int i = 1; i < tab.n; ++i)
    if (tab.seg[i].block_begin <= b) sidx = i;
  const TrSeg& sg = tab.seg[sidx];
  tr_reduce_block(base + sg.part_off, sg.splits, sg.numel, sg.mp, inv_k, grad_base + sg.w_off,
                  b - sg.block_begin);
}

// grad[o*K + k] += inv_k * sum_split part[split][o][k]   (fixed order)
// A block owns 32 consecutive elements; its 8 thread rows take interleaved
// split ranges, and the 8 row sums are combined in a fixed order.
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ part, int splits,
                                                           long numel, float inv_k,
                                                           float* __restrict__ grad) {
  __shared__ float red[8][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const long i = static_cast<long>(blockIdx.x) * 32 + tx;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  if (i < numel) {
    int t = ty;
    for (; t + 24 < splits; t += 32) {
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] += part[static_cast<long>(t + 8 * u) * numel + i];
    }
    for (; t < splits; t += 8) acc[0] += part[static_cast<long>(t) * numel + i];
  }
  red[ty][tx] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  if (ty == 0 && i < numel) {
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) s += red[r][tx];
    grad[i] += inv_k * s;
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------

namespace {

// Supported (epilogue, prologue) pairs: statistics with no prologue or BN-apply
// + ReLU (forward convs); every gradient epilogue with no prologue or the BN
// backward prologue (input-gradient convs).  f receives both as constants.
template <int E, int P> struct EpPro {
  static constexpr int ep = E, pro = P;
};

template <typename F>
bool dispatch_ep_pro(int ep, int pro, F&& f) {
  if (ep == EP_STATS) {
    if (pro == PRO_NONE) { f(EpPro<EP_STATS, PRO_NONE>{}); return true; }
    if (pro == PRO_RELU) { f(EpPro<EP_STATS, PRO_RELU>{}); return true; }
    return false;
  }
  if (pro == PRO_RELU) return false;
  const bool bwd = pro == PRO_BWD;
  if (ep == EP_MASK) {
    if (bwd) f(EpPro<EP_MASK, PRO_BWD>{}); else f(EpPro<EP_MASK, PRO_NONE>{});
    return true;
  }
  if (ep == EP_RESID) {
    if (bwd) f(EpPro<EP_RESID, PRO_BWD>{}); else f(EpPro<EP_RESID, PRO_NONE>{});
    return true;
  }
  if (ep == EP_RESID_STATS) {
    if (bwd) f(EpPro<EP_RESID_STATS, PRO_BWD>{}); else f(EpPro<EP_RESID_STATS, PRO_NONE>{});
    return true;
  }
  return false;
}

int pro_mode(const ConvArgs& a) {
  return a.pro_h != nullptr ? PRO_BWD : (a.pro_scale != nullptr ? PRO_RELU : PRO_NONE);
}

template <typename T, int BN, int WM>
bool launch_gemm(const ConvArgs& a, int ep, hipStream_t st) {
  constexpr int BM = 128;
  dim3 grid((a.m + BM - 1) / BM, (a.c_out + BN - 1) / BN);
  return dispatch_ep_pro(ep, pro_mode(a), [&](auto k) {
    PETRA_LAUNCH((conv_gemm_kernel<T, BM, BN, WM, decltype(k)::ep, decltype(k)::pro>), grid,
                       dim3(256), 0, st, a);
  });
}

template <typename T>
bool conv_gemm_t(const ConvArgs& a, int ep, hipStream_t st) {
  if (a.c_out <= 16) return launch_gemm<T, 16, 4>(a, ep, st);
  if (a.c_out <= 32) return launch_gemm<T, 32, 4>(a, ep, st);
  if (a.c_out <= 64) return launch_gemm<T, 64, 2>(a, ep, st);
  return launch_gemm<T, 128, 2>(a, ep, st);
}

template <int BM, int BN, int WM>
bool launch_staged(const ConvArgs& a, int ep, hipStream_t st) {
  dim3 grid((a.m + BM - 1) / BM, (a.c_out + BN - 1) / BN);
  return dispatch_ep_pro(ep, pro_mode(a), [&](auto k) {
    PETRA_LAUNCH((conv_staged_kernel<BM, BN, WM, decltype(k)::ep, decltype(k)::pro>), grid,
                       dim3(256), 0, st, a);
  });
}

bool launch_staged_tiles(const ConvArgs& a, int ep, hipStream_t st) {
  if (a.c_out <= 32) return launch_staged<256, 32, 4>(a, ep, st);
  if (a.c_out <= 64) return launch_staged<128, 64, 2>(a, ep, st);
  return launch_staged<128, 128, 2>(a, ep, st);
}

// Halo-tile geometry for a 3x3 stride-1 bf16 conv, or tw = 0 when it does not apply.
struct HaloShape { int th, tw, bn, wm, hb; };

HaloShape halo_shape(int dtype, const ConvArgs& a) {
  HaloShape z{0, 0, 0, 0, 0};
  if (!(dtype == DT_BF16 && a.src2 == nullptr && a.r == 3 && a.s == 3 && a.stride == 1 &&
        a.pad == 1 && a.c_in % 32 == 0 && a.c_in <= 512 && a.c_out % 8 == 0 && a.p == a.h &&
        a.q == a.w))
    return z;
  // byte offsets of the buffer loads/stores are 32-bit
  if (static_cast<long>(a.m) * std::max(a.c_in, a.c_out) * 2 >= static_cast<long>(BUF_OOB)) return z;
  const int hb = a.c_in > 32 ? 2 : 1;
  if (a.w == 32 && a.c_out <= 32) return HaloShape{8, 32, 32, 4, hb};
  if (a.w == 16 && a.c_out <= 64) return HaloShape{8, 16, 64, 2, hb};
  if (a.w == 16) return HaloShape{8, 16, 128, 2, hb};
  if (a.w == 56 && a.c_out <= 32 && a.c_in == 32) return HaloShape{4, 56, 32, 2, 1};
  return z;
}

template <int TH, int TW, int BN, int WM, int HB, bool FB>
bool launch_halo(const ConvArgs& a, int ep, hipStream_t st) {
  const int tiles = ((a.w + TW - 1) / TW) * ((a.h + TH - 1) / TH) * a.n;
  dim3 grid(tiles, (a.c_out + BN - 1) / BN);
  return dispatch_ep_pro(ep, pro_mode(a), [&](auto k) {
    PETRA_LAUNCH((conv_halo_kernel<TH, TW, BN, WM, HB, decltype(k)::ep, decltype(k)::pro, FB>),
                       grid, dim3(256), 0, st, a);
  });
}

// IMG_WM x IMG_WN waves per image, each 64 pixels x 64 channels (measured:
// 2 x 2 waves of 128 x 64, with a third fewer LDS reads per MFMA but one wave
// per SIMD, ran 17 % slower).
constexpr int IMG_WM = 4, IMG_WN = 2;
template <int TH, int TW, int CH>
bool launch_img(const ConvArgs& a, int ep, hipStream_t st) {
  // the tile is the whole image, and every weight row is c_in * 9 long
  if (a.h != TH || a.w != TW || a.c_in != 32 * CH || a.c_out != 128 || a.k_tot != 9 * a.c_in)
    return false;
  return dispatch_ep_pro(ep, pro_mode(a), [&](auto k) {
    PETRA_LAUNCH((conv_img_kernel<TH, TW, CH, decltype(k)::ep, decltype(k)::pro, IMG_WM, IMG_WN>),
                 dim3(a.n), dim3(64 * IMG_WM * IMG_WN), 0, st, a);
  });
}

// Whole-image kernel: 16 x 16 images, C_in 128, C_out 128.
bool use_img(int dtype, const ConvArgs& a) {
  return dtype == DT_BF16 && a.src2 == nullptr && a.r == 3 && a.s == 3 && a.stride == 1 &&
         a.pad == 1 && a.h == 16 && a.w == 16 && a.p == 16 && a.q == 16 && a.c_in == 128 &&
         a.c_out == 128 && a.k_tot == 1152 &&
         static_cast<long>(a.n) * a.h * a.w * 256 < static_cast<long>(BUF_OOB);
}

template <int TH, int TW, int BN, int WM, int CH>
bool launch_fp(const ConvArgs& a, int ep, hipStream_t st) {
  const int tiles = ((a.w + TW - 1) / TW) * ((a.h + TH - 1) / TH) * a.n;
  dim3 grid(tiles, (a.c_out + BN - 1) / BN);
  return dispatch_ep_pro(ep, pro_mode(a), [&](auto k) {
    PETRA_LAUNCH((conv_fp_kernel<TH, TW, BN, WM, CH, decltype(k)::ep, decltype(k)::pro>),
                       grid, dim3(256), 0, st, a);
  });
}

// Persistent 32 -> 32 kernel: tile geometry and grid (th == 0: not used).  It
// wins where the image is wide enough for several tiles per workgroup (56 wide);
// at 32 x 32 the one-shot halo kernel is faster.
struct C32Shape { int th, tw, tiles, grid; };

C32Shape conv32_shape(int dtype, const ConvArgs& a) {
  C32Shape z{0, 0, 0, 0};
  if (!(dtype == DT_BF16 && a.src2 == nullptr && a.r == 3 && a.s == 3 && a.stride == 1 &&
        a.pad == 1 && a.c_in == 32 && a.c_out == 32 && a.p == a.h && a.q == a.w &&
        a.k_tot == 288 && a.w == 56))
    return z;
  // byte offsets of the buffer loads/stores are 32-bit
  if (static_cast<long>(a.n) * a.h * a.w * 64 >= static_cast<long>(BUF_OOB)) return z;
  // the input-gradient form (BN-backward prologue) holds two patches of the
  // next tile in registers: two-row tiles keep it within 256 VGPRs (four-row
  // tiles spill; measured at 64x56x56x32, 33.7 us -> 22.8 us per launch)
  C32Shape c{pro_mode(a) == PRO_BWD ? 2 : 4, 56, 0, 0};
  c.tiles = ((a.w + c.tw - 1) / c.tw) * ((a.h + c.th - 1) / c.th) * a.n;
  const int per = (c.tiles + 511) / 512;
  c.grid = ((c.tiles + per - 1) / per + 7) / 8 * 8;
  return c;
}

bool launch_conv32(const C32Shape& c, const ConvArgs& a, int ep, hipStream_t st) {
  return dispatch_ep_pro(ep, pro_mode(a), [&](auto k) {
    constexpr int TH = decltype(k)::pro == PRO_BWD ? 2 : 4;
    PETRA_LAUNCH((conv32_kernel<TH, 56, decltype(k)::ep, decltype(k)::pro>), dim3(c.grid),
                       dim3(256), 0, st, a, c.tiles);
  });
}

// Streaming 1x1 kernels (conv1x1_kernel, conv1x1_bwd_kernel): stride-1 1x1
// bf16 convs of the bottleneck widths.  Grid: one workgroup per CU
// (C1_GRID = the MI355X CU count) or fewer; the grid is also the number of
// partial rows.  Measured per bottleneck stage step (64x56x56, 12544 units):
// 256 workgroups 1.933 ms, 512: 1.949, 392: 1.962, 784: 1.985, 3136: 2.40;
// with fewer workgroups than CU slots the kernels of the step's other streams
// run beside it.
constexpr int C1_GRID = 256;

bool use_1x1(int dtype, const ConvArgs& a, int ep) {
  // every epilogue; the prologue follows from the arguments (EP_STATS takes
  // none or BN-apply + ReLU, the gradient epilogues none or the BN backward)
  if (!(dtype == DT_BF16 && a.src2 == nullptr && a.r == 1 && a.s == 1 && a.stride == 1 &&
        a.pad == 0 && a.p == a.h && a.q == a.w && a.k_tot == a.c_in))
    return false;
  if (ep == EP_STATS ? a.pro_h != nullptr : a.pro_scale != nullptr && a.pro_h == nullptr)
    return false;
  if (!((a.c_in == 128 && a.c_out == 32) || (a.c_in == 32 && a.c_out == 128))) return false;
  // byte offsets of the buffer loads/stores are 32-bit
  return static_cast<long>(a.m) * 128 * 2 < static_cast<long>(BUF_OOB);
}

int conv1x1_units(const ConvArgs& a) { return (a.m + 15) / 16; }

int conv1x1_grid(const ConvArgs& a) {
  return std::max(1, std::min(C1_GRID, (conv1x1_units(a) + 3) / 4));
}

template <int K, int N>
void launch_1x1_kn(const ConvArgs& a, hipStream_t st) {
  const dim3 grid(conv1x1_grid(a));
  const bool relu = pro_mode(a) == PRO_RELU;
  if (a.out == nullptr) {   // statistics only
    if (relu)
      PETRA_LAUNCH((conv1x1_kernel<K, N, PRO_RELU, false>), grid, dim3(256), 0, st, a,
                   conv1x1_units(a));
    else
      PETRA_LAUNCH((conv1x1_kernel<K, N, PRO_NONE, false>), grid, dim3(256), 0, st, a,
                   conv1x1_units(a));
  } else if (relu) {
    PETRA_LAUNCH((conv1x1_kernel<K, N, PRO_RELU>), grid, dim3(256), 0, st, a, conv1x1_units(a));
  } else {
    PETRA_LAUNCH((conv1x1_kernel<K, N, PRO_NONE>), grid, dim3(256), 0, st, a, conv1x1_units(a));
  }
}


template <int K, int N>
bool launch_1x1_bwd_kn(const ConvArgs& a, int ep, hipStream_t st) {
  const dim3 grid(conv1x1_grid(a));
  return dispatch_ep_pro(ep, pro_mode(a), [&](auto k) {
    if constexpr (decltype(k)::ep != EP_STATS)
      PETRA_LAUNCH((conv1x1_bwd_kernel<K, N, decltype(k)::ep, decltype(k)::pro>), grid,
                   dim3(256), 0, st, a, conv1x1_units(a));
  });
}

bool launch_1x1(const ConvArgs& a, int ep, hipStream_t st) {
  if (ep != EP_STATS)
    return a.c_in == 128 ? launch_1x1_bwd_kn<128, 32>(a, ep, st)
                         : launch_1x1_bwd_kn<32, 128>(a, ep, st);
  if (a.c_in == 128)
    launch_1x1_kn<128, 32>(a, st);
  else
    launch_1x1_kn<32, 128>(a, st);
  return true;
}

// Returns -1 when no halo kernel applies, else whether the launch was made.
int launch_halo_any(int dtype, const ConvArgs& a, int ep, hipStream_t st) {
  if (use_img(dtype, a)) return launch_img<16, 16, 4>(a, ep, st) ? 1 : 0;
  const C32Shape c32 = conv32_shape(dtype, a);
  if (c32.th != 0) return launch_conv32(c32, a, ep, st) ? 1 : 0;
  const HaloShape h = halo_shape(dtype, a);
  if (h.tw == 0) return -1;
  bool ok;
  // a single 32-channel chunk (HB == 1) stages all nine weight slabs at once
  if (h.tw == 32)
    ok = h.hb == 1 ? launch_halo<8, 32, 32, 4, 1, true>(a, ep, st)
                   : launch_halo<8, 32, 32, 4, 2, false>(a, ep, st);
  else if (h.tw == 16 && h.bn == 64)
    ok = h.hb == 1 ? launch_halo<8, 16, 64, 2, 1, true>(a, ep, st)
         : a.c_in == 64 ? launch_fp<8, 16, 64, 2, 2>(a, ep, st)
         : a.c_in == 128 ? launch_fp<8, 16, 64, 2, 4>(a, ep, st)
                         : launch_halo<8, 16, 64, 2, 2, false>(a, ep, st);
  else if (h.tw == 16)
    ok = h.hb == 1 ? launch_halo<8, 16, 128, 2, 1, false>(a, ep, st)
         : a.c_in == 64 ? launch_fp<8, 16, 128, 2, 2>(a, ep, st)
         : a.c_in == 128 ? launch_fp<8, 16, 128, 2, 4>(a, ep, st)
                         : launch_halo<8, 16, 128, 2, 2, false>(a, ep, st);
  else
    ok = launch_halo<4, 56, 32, 2, 1, true>(a, ep, st);
  return ok ? 1 : 0;
}

bool use_staged(int dtype, const ConvArgs& a) {
  return dtype == DT_BF16 && a.src2 == nullptr && a.c_in % 32 == 0 && a.c_out % 8 == 0 &&
         a.c_in <= 512 && a.c_out >= 16 &&
         // byte offsets of the buffer loads/stores are 32-bit
         static_cast<long>(a.n) * a.h * a.w * a.c_in * 2 < static_cast<long>(BUF_OOB) &&
         static_cast<long>(a.m) * a.c_out * 2 < static_cast<long>(BUF_OOB);
}

template <typename T, int BO, int BK>
void launch_wgrad_bk(const WgradArgs& a, hipStream_t st) {
  dim3 grid((a.k_tot + BK - 1) / BK, (a.c_out + BO - 1) / BO, a.splits);
  if (a.pro_scale != nullptr)
    PETRA_LAUNCH((wgrad_kernel<T, BO, BK, true>), grid, dim3(256), 0, st, a);
  else
    PETRA_LAUNCH((wgrad_kernel<T, BO, BK, false>), grid, dim3(256), 0, st, a);
}

}  // namespace

// Transposed-read weight gradient: configuration for these arguments (0: not
// applicable) and the split count it uses.
int wgrad_tr_plan(int dtype, const WgradArgs& a, int* splits) {
  if (!(dtype == DT_BF16 && a.src2 == nullptr && a.stride == 1 && a.r == a.s &&
        (a.r == 3 || a.r == 1) && a.pad == a.r / 2 && a.p == a.h && a.q == a.w &&
        a.dh_h != nullptr))
    return 0;
  if (static_cast<long>(a.n) * a.h * a.w * a.c_in * 2 >= static_cast<long>(BUF_OOB) ||
      static_cast<long>(a.m) * a.c_out * 2 >= static_cast<long>(BUF_OOB))
    return 0;
  int cfg = 0, th = 0, tw = 0, bo = 0, bc = 0;
  if (a.r == 3 && a.c_in == 32 && a.c_out == 32 && (a.w == 32 || a.w == 56)) {
    cfg = a.w == 32 ? 1 : 2; th = 4; tw = a.w; bo = 32; bc = 32;
  } else if (a.r == 3 && a.c_in % 64 == 0 && a.c_out % 64 == 0 && a.w == 16) {
    cfg = 3; th = 8; tw = 16; bo = 64; bc = 64;
  } else if (a.r == 3 && a.c_in % 64 == 0 && a.c_out % 64 == 0 && a.w == 8) {
    cfg = 4; th = 8; tw = 8; bo = 64; bc = 64;
  } else if (a.r == 1 && a.c_in == 128 && a.c_out == 32) {
    cfg = 5; th = 1; tw = 128; bo = 32; bc = 128;
  } else if (a.r == 1 && a.c_in == 32 && a.c_out == 128) {
    cfg = 6; th = 1; tw = 128; bo = 128; bc = 32;
  } else {
    return 0;
  }
  const int ntiles = a.r == 1 ? (a.m + th * tw - 1) / (th * tw)
                              : ((a.w + tw - 1) / tw) * ((a.h + th - 1) / th) * a.n;
  const int per = (a.c_out / bo) * (a.c_in / bc);
  // about half a workgroup per CU and layer: the backward launches the weight
  // gradients of all but one layer together, so fewer, longer splits win.  The
  // bottleneck plans (2, 5, 6), whose grouped launches run beside the backward
  // chain on the forward stream, take three quarters (measured at 64x56x56:
  // 32 / 64 / 128 / 192 / 256 splits per layer, step 1.737 / 1.620 / 1.562 /
  // 1.554 / 1.560 ms); the 16x16 plan (3) a little less (ImageNet32-shaped
  // stage with 16 / 24 / 32 splits per layer: 3.065 / 3.056 / 3.078 ms; 48
  // splits on another box 3.20 against 3.09 ms with 32).  CIFAR-shaped: 64 /
  // 96 / 128 splits 0.414 / 0.412 / 0.412 ms, 192 on another box 0.420 ms.
  // The 8x8 plan (4) in the 4-stage schedule: budget 32 / 48 / 64 / 128 / 192,
  // tick 3.047 / 3.045 / 3.044 / 3.065 / 3.081 ms.
  const int budget = (cfg == 2 || cfg == 5 || cfg == 6) ? 192 : cfg == 3 ? 96 : cfg == 4 ? 64 : 128;
  if (splits) *splits = std::max(1, std::min(ntiles, budget / per));
  return cfg;
}

namespace {
template <int R, int TH, int TW, int WO, int OF, int WC, int CF, int WT, int WP>
TrMap tr_map(const WgradArgs& a) {
  constexpr int BO = WO * OF * 16, BC = WC * CF * 16;
  (void)WP;
  return TrMap{WO, OF, WC, CF, WT, R * R / WT, BO, BC, a.c_in / BC, a.c_in, a.k_tot};
}

template <int R, int TH, int TW, int WO, int OF, int WC, int CF, int WT, int WP>
void launch_wgrad_tr(const WgradArgs& a, hipStream_t st) {
  constexpr int BO = WO * OF * 16, BC = WC * CF * 16;
  dim3 grid(a.splits, a.c_out / BO, a.c_in / BC);
  dim3 block(64 * WO * WC * WT * WP);
  PETRA_LAUNCH((wgrad_tr_kernel<R, TH, TW, WO, OF, WC, CF, WT, WP, true>), grid, block, 0, st, a);
}

template <int R, int TH, int TW, int WO, int OF, int WC, int CF, int WT, int WP>
void launch_wgrad_tr_group(const WgradArgs* args, int n, hipStream_t st) {
  constexpr int BO = WO * OF * 16, BC = WC * CF * 16;
  for (int i0 = 0; i0 < n; i0 += MAX_WG_GROUP) {
    WgGroupTable tab{};
    tab.n = std::min(MAX_WG_GROUP, n - i0);
    long blocks = 0;
    for (int i = 0; i < tab.n; ++i) {
      tab.a[i] = args[i0 + i];
      tab.block_begin[i] = blocks;
      blocks += static_cast<long>(tab.a[i].splits) * (tab.a[i].c_out / BO) * (tab.a[i].c_in / BC);
    }
    PETRA_LAUNCH((wgrad_tr_group_kernel<R, TH, TW, WO, OF, WC, CF, WT, WP, true>),
                 dim3(static_cast<unsigned>(blocks)), dim3(64 * WO * WC * WT * WP), 0, st, tab);
  }
}
}  // namespace

namespace {

// Template arguments of the transposed-read weight gradient per plan (R, TH,
// TW, WO, OF, WC, CF, WT, WP).  Plan 3 (3x3, 16x16 images, 64 x 64 channel
// blocks) splits the 9 taps over three waves (WT = 3: 12 waves, three per
// SIMD, a 64 x 16 x 3 accumulator tile per wave) rather than one wave per SIMD
// holding all 9 taps: the operand parking of the next tile then overlaps other
// waves' MFMAs.  Measured at 256x16x16, 128 -> 128: 68.0 -> 56.7 us per layer,
// ImageNet32-shaped stage step 3.067 -> 2.919 ms, although 11 VGPRs spill.
bool tr_map_of(int dtype, const WgradArgs& a, TrMap* out) {
  int sp = 0;
  TrMap& mp = *out;
  switch (wgrad_tr_plan(dtype, a, &sp)) {
    case 1: mp = tr_map<3, 4, 32, 1, 2, 1, 2, 3, 4>(a); return true;
    case 2: mp = tr_map<3, 4, 56, 1, 2, 1, 2, 3, 1>(a); return true;
    case 3: mp = tr_map<3, 8, 16, 1, 4, 4, 1, 3, 1>(a); return true;
    case 4: mp = tr_map<3, 8, 8, 1, 4, 4, 1, 1, 1>(a); return true;
    case 5: mp = tr_map<1, 1, 128, 1, 2, 4, 2, 1, 1>(a); return true;
    case 6: mp = tr_map<1, 1, 128, 4, 2, 1, 2, 1, 1>(a); return true;
    default: return false;
  }
}

}  // namespace

bool wgrad_tr_segment(int dtype, const WgradArgs& a, long part_off, long w_off, TrSeg* seg) {
  TrSeg sg{};
  if (!tr_map_of(dtype, a, &sg.mp)) return false;
  sg.part_off = part_off;
  sg.w_off = w_off;
  sg.numel = static_cast<long>(a.c_out) * a.k_tot;
  sg.splits = a.splits;
  *seg = sg;
  return true;
}

void wgrad_tr_reduce_group(const float* base, const TrSeg* segs, int nseg, float inv_k,
                           float* grad_base, hipStream_t st) {
  for (int i0 = 0; i0 < nseg; i0 += MAX_TR_SEGS) {
    TrSegTable tab{};
    tab.n = std::min(MAX_TR_SEGS, nseg - i0);
    long blocks = 0;
    for (int i = 0; i < tab.n; ++i) {
      tab.seg[i] = segs[i0 + i];
      tab.seg[i].block_begin = blocks;
      blocks += (tab.seg[i].numel / 4 + 15) / 16;
    }
    PETRA_LAUNCH(wgrad_tr_reduce_group_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                 st, tab, base, inv_k, grad_base);
  }
}

bool wgrad_tr_reduce(int dtype, const WgradArgs& a, float inv_k, float* grad, hipStream_t st) {
  int sp = 0;
  TrMap mp{};
  switch (wgrad_tr_plan(dtype, a, &sp)) {
    case 1: mp = tr_map<3, 4, 32, 1, 2, 1, 2, 3, 4>(a); break;
    case 2: mp = tr_map<3, 4, 56, 1, 2, 1, 2, 3, 1>(a); break;
    case 3: mp = tr_map<3, 8, 16, 1, 4, 4, 1, 3, 1>(a); break;
    case 4: mp = tr_map<3, 8, 8, 1, 4, 4, 1, 1, 1>(a); break;
    case 5: mp = tr_map<1, 1, 128, 1, 2, 4, 2, 1, 1>(a); break;
    case 6: mp = tr_map<1, 1, 128, 4, 2, 1, 2, 1, 1>(a); break;
    default: return false;
  }
  const long numel = static_cast<long>(a.c_out) * a.k_tot;
  const long quads = numel / 4;
  PETRA_LAUNCH(wgrad_tr_reduce_kernel, dim3(static_cast<unsigned>((quads + 15) / 16)), dim3(256), 0,
               st, a.partials, a.splits, numel, mp, inv_k, grad);
  return true;
}

bool conv_wgrad_tr_group(int dtype, const WgradArgs* args, int n, hipStream_t st) {
  if (n <= 0) return true;
  int sp = 0;
  const int plan = wgrad_tr_plan(dtype, args[0], &sp);
  for (int i = 1; i < n; ++i)
    if (wgrad_tr_plan(dtype, args[i], &sp) != plan) return false;
  switch (plan) {
    case 1: launch_wgrad_tr_group<3, 4, 32, 1, 2, 1, 2, 3, 4>(args, n, st); return true;
    case 2: launch_wgrad_tr_group<3, 4, 56, 1, 2, 1, 2, 3, 1>(args, n, st); return true;
    case 3: launch_wgrad_tr_group<3, 8, 16, 1, 4, 4, 1, 3, 1>(args, n, st); return true;
    case 4: launch_wgrad_tr_group<3, 8, 8, 1, 4, 4, 1, 1, 1>(args, n, st); return true;
    case 5: launch_wgrad_tr_group<1, 1, 128, 1, 2, 4, 2, 1, 1>(args, n, st); return true;
    case 6: launch_wgrad_tr_group<1, 1, 128, 4, 2, 1, 2, 1, 1>(args, n, st); return true;
    default: return false;
  }
}

bool conv_wgrad_tr(int dtype, const WgradArgs& a, hipStream_t st) {
  int sp = 0;
  switch (wgrad_tr_plan(dtype, a, &sp)) {
    case 1: launch_wgrad_tr<3, 4, 32, 1, 2, 1, 2, 3, 4>(a, st); return true;
    case 2: launch_wgrad_tr<3, 4, 56, 1, 2, 1, 2, 3, 1>(a, st); return true;
    case 3: launch_wgrad_tr<3, 8, 16, 1, 4, 4, 1, 3, 1>(a, st); return true;
    case 4: launch_wgrad_tr<3, 8, 8, 1, 4, 4, 1, 1, 1>(a, st); return true;
    case 5: launch_wgrad_tr<1, 1, 128, 1, 2, 4, 2, 1, 1>(a, st); return true;
    case 6: launch_wgrad_tr<1, 1, 128, 4, 2, 1, 2, 1, 1>(a, st); return true;
    default: return false;
  }
}

// 0: no halo kernel; 1: 4x32 tiles, 32 output channels per group; 2: 8x16 tiles, 64.
int wgrad_halo_shape(int dtype, const WgradArgs& a) {
  if (!(dtype == DT_BF16 && a.src2 == nullptr && a.r == 3 && a.s == 3 && a.stride == 1 &&
        a.pad == 1 && a.c_in % 32 == 0 && a.c_out % 8 == 0 && a.p == a.h && a.q == a.w))
    return 0;
  if (a.w == 32 && a.c_out <= 32) return 1;
  if (a.w == 16 && a.c_out % 64 == 0) return 2;
  return 0;
}

int wgrad_halo_tiles(int dtype, const WgradArgs& a) {
  const int shape = wgrad_halo_shape(dtype, a);
  if (shape == 1) return ((a.w + 31) / 32) * ((a.h + 3) / 4) * a.n;
  if (shape == 2) return ((a.w + 15) / 16) * ((a.h + 7) / 8) * a.n;
  return 0;
}

namespace {

template <int BO, int BK>
void launch_wgrad_staged(const WgradArgs& a, hipStream_t st) {
  dim3 grid((a.k_tot + BK - 1) / BK, (a.c_out + BO - 1) / BO, a.splits);
  const bool pro = a.pro_scale != nullptr, cat = a.src2 != nullptr;
  if (cat) {
    if (pro)
      PETRA_LAUNCH((wgrad_staged_kernel<BO, BK, true, true>), grid, dim3(256), 0, st, a);
    else
      PETRA_LAUNCH((wgrad_staged_kernel<BO, BK, false, true>), grid, dim3(256), 0, st, a);
  } else {
    if (pro)
      PETRA_LAUNCH((wgrad_staged_kernel<BO, BK, true, false>), grid, dim3(256), 0, st, a);
    else
      PETRA_LAUNCH((wgrad_staged_kernel<BO, BK, false, false>), grid, dim3(256), 0, st, a);
  }
}

template <int TH, int TW, int BO>
void launch_wgrad_halo(const WgradArgs& a, hipStream_t st) {
  dim3 grid(a.splits, (a.c_out + BO - 1) / BO, a.c_in / 32);
  if (a.pro_scale != nullptr)
    PETRA_LAUNCH((wgrad_halo_kernel<TH, TW, BO, true>), grid, dim3(256), 0, st, a);
  else
    PETRA_LAUNCH((wgrad_halo_kernel<TH, TW, BO, false>), grid, dim3(256), 0, st, a);
}

template <typename T>
void wgrad_t(const WgradArgs& a, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    const int shape = wgrad_halo_shape(DT_BF16, a);
    if (shape == 1) { launch_wgrad_halo<4, 32, 32>(a, st); return; }
    if (shape == 2) { launch_wgrad_halo<8, 16, 64>(a, st); return; }
    if (a.c_out <= 32)
      launch_wgrad_staged<32, 64>(a, st);
    else
      launch_wgrad_staged<64, 64>(a, st);
    return;
  }
  if (a.c_out <= 32)
    launch_wgrad_bk<T, 32, 64>(a, st);
  else
    launch_wgrad_bk<T, 64, 64>(a, st);
}

}  // namespace

bool conv1x1_couple_ok(int dtype, const ConvArgs& a) {
  return use_1x1(dtype, a, EP_STATS) && a.c_in == 32 && a.c_out == 128;
}

bool conv1x1_couple_next_ok(int dtype, const ConvArgs& a, const ConvArgs& next) {
  return conv1x1_couple_ok(dtype, a) && use_1x1(dtype, next, EP_STATS) && next.c_in == 128 &&
         next.c_out == 32 && next.m == a.m && next.pro_scale == nullptr &&
         conv_row_tiles(dtype, next, EP_STATS) == conv1x1_grid(a);
}

bool conv1x1_couple(int dtype, const ConvArgs& a, const float* scale, const float* shift,
                    bool sub, hipStream_t st, const NextConv* next) {
  if (!conv1x1_couple_ok(dtype, a) || pro_mode(a) != PRO_RELU || a.resid == nullptr ||
      a.out == nullptr || scale == nullptr || shift == nullptr)
    return false;
  if (next != nullptr &&
      (next->wt == nullptr || next->out == nullptr || next->partials == nullptr))
    return false;
  ConvArgs b = a;
  b.ep_scale = scale;
  b.ep_shift = shift;
  const dim3 grid(conv1x1_grid(b));
  const NextConv nx = next != nullptr ? *next : NextConv{};
  if (next != nullptr && sub)
    PETRA_LAUNCH((conv1x1_couple_kernel<32, 128, true, true>), grid, dim3(256), 0, st, b,
                 conv1x1_units(b), nx);
  else if (next != nullptr)
    PETRA_LAUNCH((conv1x1_couple_kernel<32, 128, false, true>), grid, dim3(256), 0, st, b,
                 conv1x1_units(b), nx);
  else if (sub)
    PETRA_LAUNCH((conv1x1_couple_kernel<32, 128, true, false>), grid, dim3(256), 0, st, b,
                 conv1x1_units(b), nx);
  else
    PETRA_LAUNCH((conv1x1_couple_kernel<32, 128, false, false>), grid, dim3(256), 0, st, b,
                 conv1x1_units(b), nx);
  return true;
}

int conv_row_tiles(int dtype, const ConvArgs& a, int ep) {
  if (use_1x1(dtype, a, ep)) return conv1x1_grid(a);
  if (use_img(dtype, a)) return a.n;
  const C32Shape c32 = conv32_shape(dtype, a);
  if (c32.th != 0) return c32.grid;
  const HaloShape hs = halo_shape(dtype, a);
  if (hs.tw != 0) return ((a.w + hs.tw - 1) / hs.tw) * ((a.h + hs.th - 1) / hs.th) * a.n;
  int bm = CONV_BM;
  if (use_staged(dtype, a)) bm = a.c_out <= 32 ? 256 : 128;
  return (a.m + bm - 1) / bm;
}

bool conv_gemm(int dtype, const ConvArgs& a, int ep, hipStream_t st) {
  if (use_1x1(dtype, a, ep)) return launch_1x1(a, ep, st);
  const int h = launch_halo_any(dtype, a, ep, st);
  if (h >= 0) return h == 1;
  if (use_staged(dtype, a)) return launch_staged_tiles(a, ep, st);
  if (dtype == DT_BF16) return conv_gemm_t<bf16_t>(a, ep, st);
  return conv_gemm_t<float>(a, ep, st);
}

void conv_wgrad(int dtype, const WgradArgs& a, hipStream_t st) {
  if (conv_wgrad_tr(dtype, a, st)) return;
  if (dtype == DT_BF16)
    wgrad_t<bf16_t>(a, st);
  else
    wgrad_t<float>(a, st);
}

void wgrad_reduce(const float* part, int splits, long numel, float inv_k, float* grad,
                  hipStream_t st) {
  const long blocks = (numel + 31) / 32;
  PETRA_LAUNCH(wgrad_reduce_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st,
                     part, splits, numel, inv_k, grad);
}

}  // namespace petra
