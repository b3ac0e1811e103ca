// Internal definitions shared by the libdla HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dla.h"

namespace dla {

constexpr uint32_t kMagic = 0x31414C44u;  // 'DLA1'
constexpr uint32_t kVersion = 2u;
constexpr size_t kHeaderBytes = 256;

struct CacheHeader {
  uint32_t magic;
  uint32_t version;
  int32_t B, H, C, dk, dv;
  uint32_t flags;
  int32_t state_dtype;
};

// Whether a cache header describes the descriptor a call was given.  Every
// kernel of a prefill or decode step checks it before touching anything else,
// so a call whose descriptor differs from the cache's (a larger capacity, more
// heads, another state type) cannot index past the buffer.
__host__ __device__ inline bool header_matches(const CacheHeader& hd, const dla_cache_desc& d) {
  return hd.magic == kMagic && hd.version == kVersion && hd.B == d.B && hd.H == d.H &&
         hd.C == d.C && hd.dk == d.d_k && hd.dv == d.d_v && hd.state_dtype == d.state_dtype;
}

__device__ __forceinline__ bool cache_matches(const char* cache, const dla_cache_desc& d) {
  return header_matches(*reinterpret_cast<const CacheHeader*>(cache), d);
}

// The first kernel of a call records a refused call in the header's flags.
__device__ __forceinline__ void flag_mismatch(char* cache) {
  if (blockIdx.x == 0 && threadIdx.x == 0)
    atomicOr(&reinterpret_cast<CacheHeader*>(cache)->flags, DLA_FLAG_CACHE_MISMATCH);
}

__host__ __device__ inline size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workgroups per head of a decode step at most; each leaves a partial output
// of d_v floats in the head's metadata (see decode.hip).
constexpr int kMaxSplit = 16;

// Scratch of a split decode step in each head's metadata: the decisions
// (64 bytes reserved), then the partial outputs float [kMaxSplit][d_v].
__host__ __device__ inline size_t meta_record_offset(int C) {
  return round_up(32 + 24 * (size_t)C, 64);
}

__host__ __device__ inline size_t meta_stride(int C, int dv) {
  return round_up(meta_record_offset(C) + 64 + (size_t)kMaxSplit * dv * sizeof(float), 256);
}

__device__ __forceinline__ char* decode_record(char* meta, int C) {
  return meta + meta_record_offset(C);
}
__device__ __forceinline__ float* decode_partials(char* meta, int C) {
  return reinterpret_cast<float*>(meta + meta_record_offset(C) + 64);
}

// Per-head metadata (chronological arrays).  See dla.h for the byte layout.
struct Meta {
  int32_t* m;
  double* G;
  int64_t* tokens;
  double* F;
  double* ibar;
  int32_t* n;
  int32_t* perm;
};

__host__ __device__ inline Meta meta_at(char* base, int C) {
  Meta r;
  r.m = reinterpret_cast<int32_t*>(base);
  r.G = reinterpret_cast<double*>(base + 8);
  r.tokens = reinterpret_cast<int64_t*>(base + 16);
  r.F = reinterpret_cast<double*>(base + 32);
  r.ibar = r.F + C;
  r.n = reinterpret_cast<int32_t*>(r.ibar + C);
  r.perm = r.n + C;
  return r;
}

// Bytes of one stored state element (float32 or bfloat16 storage).
__host__ __device__ inline size_t state_elem_bytes(const dla_cache_desc& d) {
  return d.state_dtype == DLA_BF16 ? 2 : 4;
}

inline dla_cache_layout layout_of(const dla_cache_desc& d) {
  dla_cache_layout L;
  const size_t nh = (size_t)d.B * d.H;
  const size_t D = (size_t)d.d_k * d.d_v;
  L.meta_offset = kHeaderBytes;
  L.meta_stride = meta_stride(d.C, d.d_v);
  L.states_offset = round_up(L.meta_offset + nh * L.meta_stride, 256);
  const size_t end = L.states_offset + nh * (size_t)d.C * D * state_elem_bytes(d);
  if (d.state_dtype == DLA_BF16) {
    L.open_offset = round_up(end, 256);
    L.total_bytes = L.open_offset + nh * D * sizeof(float);
  } else {
    L.open_offset = 0;
    L.total_bytes = end;
  }
  return L;
}

// ---------------------------------------------------------------------------
// element types: float32, or bfloat16 kept as raw 16-bit patterns
// ---------------------------------------------------------------------------
struct bf16_t {
  uint16_t x;
};

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v.x) << 16);
}

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  // round to nearest even (inputs here are finite)
  uint32_t u = __float_as_uint(v);
  u += 0x7FFFu + ((u >> 16) & 1u);
  bf16_t r;
  r.x = static_cast<uint16_t>(u >> 16);
  return r;
}

// ---------------------------------------------------------------------------
// wavefront (64 lanes) and block reductions
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------------------
// DPP lane moves (GFX9 controls): row_shr:n = 0x110 + n, wave_shr:1 = 0x138,
// row_bcast:15 = 0x142 (to rows 1 and 3), row_bcast:31 = 0x143 (to rows 2
// and 3).  A lane with no source lane, or outside the row mask, gets `old`.
// Scans built from them compose the earlier lanes into each lane with the
// classic row_shr 1/2/4/8 + row_bcast 15/31 ladder; lane 63 ends with the whole
// wavefront.
// ---------------------------------------------------------------------------
template <int CTRL, int RMASK>
__device__ __forceinline__ float dpp_f(float old, float x) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(x), CTRL, RMASK, 0xF, false));
}
template <int CTRL, int RMASK>
__device__ __forceinline__ int dpp_i(int old, int x) {
  return __builtin_amdgcn_update_dpp(old, x, CTRL, RMASK, 0xF, false);
}
template <int CTRL, int RMASK>
__device__ __forceinline__ double dpp_d(double old, double x) {
  const long long o = __double_as_longlong(old), v = __double_as_longlong(x);
  const int lo = dpp_i<CTRL, RMASK>((int)o, (int)v);
  const int hi = dpp_i<CTRL, RMASK>((int)(o >> 32), (int)(v >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}
__device__ __forceinline__ double readlane_d(double x, int l) {
  const long long v = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)v, l);
  const int hi = __builtin_amdgcn_readlane((int)(v >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Inclusive scan of affine maps x -> A x + B over the lanes: lane i ends with
// map_i o ... o map_0.
template <int CTRL, int RMASK>
__device__ __forceinline__ void affine_step(float& A, float& B) {
  const float Ao = dpp_f<CTRL, RMASK>(1.f, A);
  const float Bo = dpp_f<CTRL, RMASK>(0.f, B);
  B = A * Bo + B;
  A = A * Ao;
}
__device__ __forceinline__ void wave_scan_affine(float& A, float& B) {
  affine_step<0x111, 0xF>(A, B);
  affine_step<0x112, 0xF>(A, B);
  affine_step<0x114, 0xF>(A, B);
  affine_step<0x118, 0xF>(A, B);
  affine_step<0x142, 0xA>(A, B);
  affine_step<0x143, 0xC>(A, B);
}

// Sum of a float over the wavefront through DPP row shifts and broadcasts
// (every lane gets it).
__device__ __forceinline__ float wave_total_dpp(float x) {
  x += dpp_f<0x111, 0xF>(0.f, x);
  x += dpp_f<0x112, 0xF>(0.f, x);
  x += dpp_f<0x114, 0xF>(0.f, x);
  x += dpp_f<0x118, 0xF>(0.f, x);
  x += dpp_f<0x142, 0xA>(0.f, x);
  x += dpp_f<0x143, 0xC>(0.f, x);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

// Sum of a double over the wavefront (every lane gets it).
template <int CTRL, int RMASK>
__device__ __forceinline__ void sum_step_d(double& x) {
  x += dpp_d<CTRL, RMASK>(0.0, x);
}
__device__ __forceinline__ double wave_sum_d(double x) {
  sum_step_d<0x111, 0xF>(x);
  sum_step_d<0x112, 0xF>(x);
  sum_step_d<0x114, 0xF>(x);
  sum_step_d<0x118, 0xF>(x);
  sum_step_d<0x142, 0xA>(x);
  sum_step_d<0x143, 0xC>(x);
  return readlane_d(x, 63);
}

// Lowest value over the wavefront, ties to the lowest index (every lane gets
// both).
template <int CTRL, int RMASK>
__device__ __forceinline__ void argmin_step(double& best, int& bi) {
  const double ob = dpp_d<CTRL, RMASK>(INFINITY, best);
  const int oi = dpp_i<CTRL, RMASK>(0x7fffffff, bi);
  if (ob < best || (ob == best && oi < bi)) {
    best = ob;
    bi = oi;
  }
}
__device__ __forceinline__ void wave_argmin_d(double& best, int& bi) {
  argmin_step<0x111, 0xF>(best, bi);
  argmin_step<0x112, 0xF>(best, bi);
  argmin_step<0x114, 0xF>(best, bi);
  argmin_step<0x118, 0xF>(best, bi);
  argmin_step<0x142, 0xA>(best, bi);
  argmin_step<0x143, 0xC>(best, bi);
  best = readlane_d(best, 63);
  bi = __builtin_amdgcn_readlane(bi, 63);
}

// Sum of two values over a 256-thread block; every thread gets the result.
// red must hold 8 floats.
__device__ __forceinline__ void block_sum2_256(float& a, float& b, float* red) {
  a = wave_sum(a);
  b = wave_sum(b);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    red[w] = a;
    red[4 + w] = b;
  }
  __syncthreads();
  a = (red[0] + red[1]) + (red[2] + red[3]);
  b = (red[4] + red[5]) + (red[6] + red[7]);
}

// The State Information Score from the three scalars of a rank-one token
// state s = k v^T against a state S:  a = |k|^2 |v|^2, b = |S|^2, c = k^T S v.
// With RMSNorm N(X) = X / sqrt(|X|^2/D + eps_rms):
//   |N(s) - N(S)|^2 = a/rs^2 + b/rS^2 - 2c/(rs rS),   |N(S)| = sqrt(b)/rS.
__device__ __forceinline__ double info_score(double a, double b, double c, double D, double eps,
                                             double eps_rms) {
  const double rs2 = a / D + eps_rms;
  const double rS2 = b / D + eps_rms;
  const double num = a / rs2 + b / rS2 - 2.0 * c / sqrt(rs2 * rS2);
  // rounding can take num a little below 0; a NaN (non-finite inputs) passes
  // through, as the score of the definition would be NaN
  return sqrt(num < 0.0 ? 0.0 : num) / (sqrt(b / rS2) + eps);
}

// The same score in float32 (the prefill scans).
__device__ __forceinline__ float score_f(float a, float b, float c, float D, float eps,
                                         float eps_rms) {
  const float rs2 = a / D + eps_rms;
  const float rS2 = b / D + eps_rms;
  const float num = a / rs2 + b / rS2 - 2.f * c * rsqrtf(rs2 * rS2);
  // rounding can take num a little below 0; a NaN (non-finite inputs) passes
  // through, as the score of the definition would be NaN
  return sqrtf(num < 0.f ? 0.f : num) / (sqrtf(b / rS2) + eps);
}

}  // namespace dla
