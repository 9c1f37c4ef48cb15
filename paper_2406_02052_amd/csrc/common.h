// Shared device helpers for the gfx950 kernels: storage types, 8-element
// vector loads/stores, MFMA fragment types and wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace petra {

// Storage types.  bf16 is kept as its raw 16-bit pattern.
struct bf16_t { uint16_t bits; };

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 (lo in bits 0-15), round to nearest even.  gfx950
// converts a pair in one instruction (v_cvt_pk_bf16_f32); it agrees bit for bit
// with integer round-to-nearest-even on every non-NaN input and keeps NaN NaN.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// fp32 -> bf16, round to nearest even.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// Eight consecutive elements of a tensor, widened to fp32.
template <typename T> struct Vec8;

template <> struct Vec8<bf16_t> {
  static __device__ __forceinline__ void load(const bf16_t* p, float* o) {
    uint4 v = *reinterpret_cast<const uint4*>(p);
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = __uint_as_float(w[i] << 16);
      o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ void store(bf16_t* p, const float* o) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(o[2 * i], o[2 * i + 1]);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

template <> struct Vec8<float> {
  static __device__ __forceinline__ void load(const float* p, float* o) {
    float4 a = reinterpret_cast<const float4*>(p)[0];
    float4 b = reinterpret_cast<const float4*>(p)[1];
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
  static __device__ __forceinline__ void store(float* p, const float* o) {
    reinterpret_cast<float4*>(p)[0] = make_float4(o[0], o[1], o[2], o[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(o[4], o[5], o[6], o[7]);
  }
};

// Value a float takes once stored as T (bf16: round to nearest even).
__device__ __forceinline__ float quant(float v, const float*) { return v; }
__device__ __forceinline__ float quant(float v, const bf16_t*) { return bf16_to_f32(f32_to_bf16(v)); }

__device__ __forceinline__ float load1(const float* p) { return *p; }
__device__ __forceinline__ float load1(const bf16_t* p) { return bf16_to_f32(p->bits); }
__device__ __forceinline__ void store1(float* p, float v) { *p = v; }
__device__ __forceinline__ void store1(bf16_t* p, float v) { p->bits = f32_to_bf16(v); }

// Eight consecutive raw elements (bit-exact; no rounding on the way through).
template <typename T> struct Raw8;

template <> struct Raw8<bf16_t> {
  uint32_t w[4];
  __device__ __forceinline__ void zero() { w[0] = w[1] = w[2] = w[3] = 0u; }
  __device__ __forceinline__ void load(const bf16_t* p) {
    uint4 v = *reinterpret_cast<const uint4*>(p);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
  template <typename V>
  __device__ __forceinline__ void set(const V& v) {
    w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
  }
  __device__ __forceinline__ void to_f32(float* o) const {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = __uint_as_float(w[i] << 16);
      o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ __forceinline__ void from_f32(const float* o) {
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(o[2 * i], o[2 * i + 1]);
  }
  // Store element j into a 16-bit LDS/global slot.
  __device__ __forceinline__ void put(int j, bf16_t* dst) const {
    dst->bits = static_cast<uint16_t>(w[j >> 1] >> ((j & 1) * 16));
  }
};

template <> struct Raw8<float> {
  float v[8];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 0.f;
  }
  __device__ __forceinline__ void load(const float* p) { Vec8<float>::load(p, v); }
  __device__ __forceinline__ void to_f32(float* o) const {
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = v[i];
  }
  __device__ __forceinline__ void from_f32(const float* o) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = o[i];
  }
  __device__ __forceinline__ void put(int j, float* dst) const { *dst = v[j]; }
};

// MFMA operand fragment: each lane of a 16x16 tile contributes 8 values of
// the reduction dimension.  For bf16 that is one v_mfma_f32_16x16x32_bf16; for
// fp32 it is eight v_mfma_f32_16x16x4_f32 (element j of every lane group forms
// the j-th instruction's operand, which covers the same 32-wide k range).
template <typename T> struct Frag;

template <> struct Frag<bf16_t> {
  bf16x8_t v;
  __device__ __forceinline__ void set(const Raw8<bf16_t>& r) {
    v = __builtin_bit_cast(bf16x8_t, make_uint4(r.w[0], r.w[1], r.w[2], r.w[3]));
  }
  __device__ __forceinline__ void load(const bf16_t* p) {
    v = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p));
  }
};

template <> struct Frag<float> {
  float v[8];
  __device__ __forceinline__ void set(const Raw8<float>& r) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = r.v[i];
  }
  __device__ __forceinline__ void load(const float* p) { Vec8<float>::load(p, v); }
};

__device__ __forceinline__ f32x4_t mfma(const Frag<bf16_t>& a, const Frag<bf16_t>& b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4_t mfma(const Frag<float>& a, const Frag<float>& b, f32x4_t c) {
#pragma unroll
  for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], c, 0, 0, 0);
  return c;
}

// Sum over the 16 lanes of a DPP row (lanes 16 r .. 16 r + 15), returned in
// every lane of the row: pairs and quads by quad permutes, then the row's
// half-mirror and mirror.  Four VALU ops with DPP modifiers, no LDS traffic.
__device__ __forceinline__ float sum16(float v) {
  int x = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false));  // [1,0,3,2]
  x = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false));  // [2,3,0,1]
  x = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false)); // half mirror
  x = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false)); // mirror
  return v;
}

// Sum over the 4 lane groups (lanes l, l^16, l^32, l^48) of a wave64.
__device__ __forceinline__ float sum_lane_groups(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}

// Buffer resources (raw, stride 0) over [p, p + bytes): a load at a byte offset
// past the end returns zeros and a store there is dropped, which gives
// branch-free zero padding and masked stores.  Offsets are 32-bit.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
constexpr uint32_t BUF_OOB = 0x80000000u;   // an offset past every buffer used here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, static_cast<int>(bytes),
                                           0x00020000);
}
__device__ __forceinline__ u32x4_t buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, 0);
}
__device__ __forceinline__ u32x2_t buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(off), 0, 0);
}
__device__ __forceinline__ void buf_store8(u32x2_t v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, static_cast<int>(off), 0, 0);
}
__device__ __forceinline__ void buf_store16(u32x4_t v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, static_cast<int>(off), 0, 0);
}

}  // namespace petra
