// Prefill entry (internal): arguments, workspace layout and launchers.
#pragma once
#include "dla_common.h"

namespace dla {

struct PrefillArgs {
  dla_cache_desc desc;
  char* cache;
  size_t meta_offset, meta_stride, states_offset;
  const void* q;
  const void* k;
  const void* v;
  const float* g;
  const void* lam;
  void* out;
  int8_t* b_out;
  int32_t* merge_out;
  float* score_out;
  const int8_t* b_ovr;
  const int32_t* m_ovr;
  int T;
  float tau, eps, eps_rms;
  int skip_readout;
  dla_dtype in_dtype, out_dtype;
  char* workspace;
};

// Workspace regions (per head, 256-byte aligned):
//   Gtok   double [nh][T]   cumulative log-decay after each token (global frame)
//   death  int32  [nh][T]   -1: token t is not the first token of a state;
//                           T: it starts a state that is never merged away;
//                           t' in (t, T): its state was merged into its left
//                           neighbour at token t' (Alg. 2)
//   init   per head: int32 m0, int32 pad, double G0, double F0[C], int32 perm0[C],
//          int32 death0[C] (the cache's metadata before the call, and the death
//          token of the states present before the call)
//   shadow [nh][C][d_v/32][d_k/16][2][32][8] elements of the input dtype: a copy
//          of each state (by physical slot) in the per-lane order of the MFMA
//          A operand, for the readout stage
struct PrefillWS {
  double* Gtok;
  int32_t* death;
  char* init;
  size_t init_stride;
  char* shadow;
};

__host__ __device__ inline size_t ws_init_stride(int C) { return round_up(16 + 16 * (size_t)C, 256); }

__host__ __device__ inline size_t dtype_bytes(dla_dtype t) { return t == DLA_F32 ? 4 : 2; }

__host__ __device__ inline PrefillWS ws_layout(char* base, int nh, int T, int C) {
  PrefillWS w;
  size_t off = 0;
  w.Gtok = reinterpret_cast<double*>(base + off);
  off = round_up(off + (size_t)nh * T * sizeof(double), 256);
  w.death = reinterpret_cast<int32_t*>(base + off);
  off = round_up(off + (size_t)nh * T * sizeof(int32_t), 256);
  w.init = base + off;
  w.init_stride = ws_init_stride(C);
  off = round_up(off + (size_t)nh * w.init_stride, 256);
  w.shadow = base + off;
  return w;
}

inline size_t prefill_workspace_bytes(const dla_cache_desc& d, int T, dla_dtype in) {
  const size_t nh = (size_t)d.B * d.H;
  size_t off = round_up(nh * T * sizeof(double), 256);
  off = round_up(off + nh * T * sizeof(int32_t), 256);
  off = round_up(off + nh * ws_init_stride(d.C), 256);
  off += nh * (size_t)d.C * d.d_k * d.d_v * dtype_bytes(in);
  return off;
}

struct InitView {
  int32_t* m0;
  double* G0;
  double* F0;
  int32_t* perm0;
  int32_t* death0;
};

__host__ __device__ inline InitView init_at(const PrefillWS& w, int h, int C) {
  char* p = w.init + (size_t)h * w.init_stride;
  InitView v;
  v.m0 = reinterpret_cast<int32_t*>(p);
  v.G0 = reinterpret_cast<double*>(p + 8);
  v.F0 = reinterpret_cast<double*>(p + 16);
  v.perm0 = reinterpret_cast<int32_t*>(p + 16 + 8 * (size_t)C);
  v.death0 = v.perm0 + C;
  return v;
}

hipError_t launch_prefill_prep(const PrefillArgs& a, hipStream_t s);
hipError_t launch_prefill_scan(const PrefillArgs& a, hipStream_t s);
hipError_t launch_prefill_readout(const PrefillArgs& a, hipStream_t s);
// whether the readout stage's working set fits in LDS for this shape
bool prefill_readout_supported(const dla_cache_desc& d, dla_dtype in_dtype);

// Stages in order; ev (nullable) receives an event before the first stage and
// after each stage.
inline hipError_t launch_prefill(const PrefillArgs& a, hipStream_t s, void* const* ev) {
  hipError_t (*stages[DLA_PREFILL_STAGES])(const PrefillArgs&, hipStream_t) = {
      launch_prefill_prep, launch_prefill_scan, launch_prefill_readout};
  if (ev && hipEventRecord((hipEvent_t)ev[0], s) != hipSuccess) return hipErrorInvalidValue;
  for (int i = 0; i < DLA_PREFILL_STAGES; ++i) {
    hipError_t e = stages[i](a, s);
    if (e != hipSuccess) return e;
    if (ev && hipEventRecord((hipEvent_t)ev[i + 1], s) != hipSuccess) return hipErrorInvalidValue;
  }
  return hipSuccess;
}

}  // namespace dla
