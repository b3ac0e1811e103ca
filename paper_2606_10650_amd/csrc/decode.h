// Decode step entry (internal).
#pragma once
#include "dla_common.h"

namespace dla {

struct DecodeArgs {
  dla_cache_desc desc;
  char* cache;
  size_t meta_offset, meta_stride, states_offset, open_offset;
  int nsplit;  // workgroups per head (1 .. kMaxSplit)
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
  // Gated DeltaNet form (Sec. 2.2, eq. delta_rule_rnn): beta [B*H] step sizes
  // of the delta rule on the newest state, or null for the gated form
  const float* beta;
  // tokens between consecutive heads in every per-token array (q, k, v, g,
  // beta, lambda, out, exports, overrides): 1 for a decode step, T for a step
  // of a sequence of T tokens laid out [B][H][T]
  long long hs;
  float tau, eps, eps_rms;
  int skip_readout;
};

hipError_t launch_decode(const DecodeArgs& a, int nheads, int dk, int dv, dla_dtype in,
                         dla_dtype out, hipStream_t s);
// workgroups per head for nheads heads of capacity C
int decode_splits(int nheads, int C);

}  // namespace dla
