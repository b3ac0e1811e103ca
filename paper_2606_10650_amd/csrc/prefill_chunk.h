// Definitions shared by the update (stage 3) and readout (stage 4) kernels of
// the prefill: chunk geometry, LDS strides, pool addressing and a block-wide
// prefix count.
#pragma once
#include "mfma.h"
#include "prefill.h"

namespace dla {

template <int DK, typename Tin>
struct ChunkP {
  static constexpr int E = (int)sizeof(Tin);
  static constexpr int NT = readout_nt(E);   // 32-token tiles per wave (readout)
  static constexpr int RL = chunk_len(E);    // tokens per chunk
  static constexpr int KS = DK / 16;         // K = 16 steps over d_k
  static constexpr int EPP = 16 / E;         // elements per 16 bytes
  static constexpr int SLICE = DK * NC;      // elements per (state, column group)
  static constexpr int SLICE16 = SLICE * E / 16;  // 16-byte pieces per slice
  // LDS row strides (elements), padded by 16 bytes so that lanes reading
  // consecutive rows hit distinct banks
  static constexpr int VTS = RL + EPP;        // transposed values [NC][VTS]
  static constexpr int KRS = DK + EPP;        // key block, row-major [32][KRS]
  static constexpr int KBUF = 32 * KRS;
  static constexpr int KROW16 = DK * E / 16;  // 16-byte pieces per key row
};

// Slice of pool object `obj` of head h for column group cg.  Element (k, c) of
// the slice (k < d_k, c < 32) sits at ((k / 16) * 2 + (k % 16) / 8) * 256 + c * 8
// + k % 8: lane l of an MFMA A operand for K step ks reads the 8 elements at
// ((ks * 2 + l / 32) * 32 + l % 32) * 8.
template <typename Tin>
__device__ __forceinline__ Tin* pool_slice(char* pool, int h, int P_cap, int obj, int cg, int ncg,
                                           int slice) {
  return reinterpret_cast<Tin*>(pool) + (((size_t)h * P_cap + obj) * ncg + cg) * slice;
}

// Exclusive prefix count over n <= 1024 flags in a block of NTHR threads:
// out[i] = number of set flags before i.  Returns the total.  red: NWAVE ints.
template <typename F>
__device__ int block_excl_count(int n, F flag, int32_t* out, int32_t* red) {
  constexpr int PER = 1024 / NTHR;
  const int tid = threadIdx.x;
  int f[PER];
  int local = 0;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int i = PER * tid + u;
    f[u] = (i < n) ? (flag(i) ? 1 : 0) : 0;
    local += f[u];
  }
  int incl = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if ((tid & 63) >= o) incl += y;
  }
  __syncthreads();
  if ((tid & 63) == 63) red[tid >> 6] = incl;
  __syncthreads();
  int base = 0;
  for (int w = 0; w < (tid >> 6); ++w) base += red[w];
  int run = base + incl - local;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int i = PER * tid + u;
    if (i < n) out[i] = run;
    run += f[u];
  }
  int total = 0;
#pragma unroll
  for (int w = 0; w < NWAVE; ++w) total += red[w];
  __syncthreads();
  return total;
}

}  // namespace dla
