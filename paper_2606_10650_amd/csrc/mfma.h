// MFMA fragments for gfx950 (CDNA4), 32x32 output tiles, K = 16 per step.
//
// A fragment (32 x 16): lane l holds row l % 32 and the 8 k-values of lane half
// l / 32 (element e <-> k index 8 * (l / 32) + e).  B fragment (16 x 32): lane l
// holds column l % 32 and the same 8 k-values.  The product pairs element e of
// a lane half of A with element e of the same lane half of B, so any fixed
// assignment of (lane half, element) to k that A and B share gives the same sum.
// Output (32 x 32, 16 floats per lane): lane l holds column l % 32 and rows
// 8 * (r / 4) + 4 * (l / 32) + r % 4 for r = 0..15.
#pragma once
#include "dla_common.h"

namespace dla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <typename Tin>
struct Frag;

// bfloat16 inputs: one v_mfma_f32_32x32x16_bf16 per K = 16 step.
template <>
struct Frag<bf16_t> {
  using T = bf16x8;
  __device__ static __forceinline__ T load(const bf16_t* p) {  // 8 consecutive values
    return *reinterpret_cast<const T*>(p);
  }
  __device__ static __forceinline__ T from_floats(const float* x) {
    T r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = (__bf16)x[e];
    return r;
  }
  __device__ static __forceinline__ T zero() {
    T r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = (__bf16)0.f;
    return r;
  }
  __device__ static __forceinline__ void mma(f32x16& acc, const T& a, const T& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
  }
};

// float32 inputs: eight v_mfma_f32_32x32x2_f32 per K = 16 step (element e of
// each lane half is one K = 2 product).
template <>
struct Frag<float> {
  using T = f32x8;
  __device__ static __forceinline__ T load(const float* p) {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    T r;
    r[0] = a.x; r[1] = a.y; r[2] = a.z; r[3] = a.w;
    r[4] = b.x; r[5] = b.y; r[6] = b.z; r[7] = b.w;
    return r;
  }
  __device__ static __forceinline__ T from_floats(const float* x) {
    T r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = x[e];
    return r;
  }
  __device__ static __forceinline__ T zero() {
    T r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = 0.f;
    return r;
  }
  __device__ static __forceinline__ void mma(f32x16& acc, const T& a, const T& b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc, 0, 0, 0);
  }
};

__device__ __forceinline__ f32x16 zero16() {
  f32x16 r;
#pragma unroll
  for (int i = 0; i < 16; ++i) r[i] = 0.f;
  return r;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // 16 bytes, first-class
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// element e of a 16-byte piece of elements of type Tin
template <typename Tin>
__device__ __forceinline__ Tin piece_elem(const u32x4& v, int e);
template <>
__device__ __forceinline__ bf16_t piece_elem<bf16_t>(const u32x4& v, int e) {
  bf16_t r;
  r.x = static_cast<uint16_t>(v[e >> 1] >> (16 * (e & 1)));
  return r;
}
template <>
__device__ __forceinline__ float piece_elem<float>(const u32x4& v, int e) {
  return __uint_as_float(v[e]);
}

// 8 operand values from two runs of 4 consecutive elements (each run aligned
// to 4 elements)
template <typename Tin>
__device__ __forceinline__ typename Frag<Tin>::T load_4x2(const Tin* p0, const Tin* p1);
template <>
__device__ __forceinline__ bf16x8 load_4x2<bf16_t>(const bf16_t* p0, const bf16_t* p1) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 lo = *reinterpret_cast<const bf16x4*>(p0);
  const bf16x4 hi = *reinterpret_cast<const bf16x4*>(p1);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}
template <>
__device__ __forceinline__ f32x8 load_4x2<float>(const float* p0, const float* p1) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  const f32x4 lo = *reinterpret_cast<const f32x4*>(p0);
  const f32x4 hi = *reinterpret_cast<const f32x4*>(p1);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// 4 consecutive elements as floats (8-byte aligned for bfloat16, 16 for float32)
__device__ __forceinline__ void load4f(const bf16_t* p, float (&x)[4]) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  x[0] = __uint_as_float(u.x << 16);
  x[1] = __uint_as_float(u.x & 0xFFFF0000u);
  x[2] = __uint_as_float(u.y << 16);
  x[3] = __uint_as_float(u.y & 0xFFFF0000u);
}
__device__ __forceinline__ void load4f(const float* p, float (&x)[4]) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  x[0] = v.x;
  x[1] = v.y;
  x[2] = v.z;
  x[3] = v.w;
}

// row (within the 32-row tile) of output element r held by lane l
__device__ __forceinline__ int out_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

}  // namespace dla
