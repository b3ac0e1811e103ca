// Decode step of the DLA layer: one token per head against a resident cache.
//
// The step is bound by HBM bandwidth: every live state (d_k x d_v) is streamed
// once for the readout o = sum_j lambda_j q^T S_j (eq. capacity_bounded_output),
// and at most three states are written (the merged pair of Alg. 2, the state
// that closes when a new one opens, and the new or accumulated newest state).
// States decay lazily: a slot stores S~ with the true state exp(G - F_j) S~, so
// untouched states are never rewritten.
//
// Storage: float32 slots, or bfloat16 slots for the closed states with the
// newest state of each head in a float32 open region.  The decisions read only
// the newest state, the counts and the aggregated scores, so they do not depend
// on the storage type.
//
// Work split: one workgroup of 256 threads per head when there are enough heads
// to fill the chip.  With few heads, NS workgroups per head: each takes the
// step's decisions (identical arithmetic on identical data, so every workgroup
// of a head reaches the same ones) and streams one contiguous range of the
// pre-merge states, the merged pair never split between two ranges, leaving
// its partial output (and, for the first, the decisions) in a small area of
// the head's metadata; a second kernel, one workgroup per head, then sums the
// partials in split order, writes the output and the newest state, and updates
// the metadata.  The kernel boundary orders the two: no workgroup waits for
// another, and no device-scope fence is needed (one per workgroup, with the L2
// write-back it implies, made the split step 2.4 times slower).
//
// Gated DeltaNet form (with step sizes beta): the newest state follows the
// delta rule while it accumulates, S <- (I - beta k k^T) S + beta k v^T, and a
// new state is beta k v^T; closed states only decay.  The erase needs S^T k,
// reduced from the newest state's registers at the end of the step.
//
// Thread mapping inside a state: element group tid + 256 r (4 consecutive
// elements) of the row-major d_k x d_v array, i.e. thread tid owns the 4
// columns 4*(tid % (d_v/4)) .. +3 of the rows (tid / (d_v/4)) + r * (256 /
// (d_v/4)).  Loads are coalesced (16 bytes per lane for float32 storage, 8 for
// bfloat16).
#include "decode.h"

namespace dla {

// Every state is read or written at most once per step, and the states of all
// heads (gigabytes) do not fit in the caches, so state traffic goes with the
// non-temporal hint.
typedef float f32x4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));

// NT: with the non-temporal hint.  (A template parameter, not a run-time
// choice: a select between a hinted and a plain load of one address is folded
// into one load without the hint.)
template <bool NT>
__device__ __forceinline__ float4 ld_group(const float* base, int g) {
  const f32x4v* p = reinterpret_cast<const f32x4v*>(base) + g;
  f32x4v x;
  if constexpr (NT)
    x = __builtin_nontemporal_load(p);
  else
    x = *p;
  return make_float4(x[0], x[1], x[2], x[3]);
}
template <bool NT>
__device__ __forceinline__ float4 ld_group(const bf16_t* base, int g) {
  const u32x2v* p = reinterpret_cast<const u32x2v*>(base) + g;
  u32x2v x;
  if constexpr (NT)
    x = __builtin_nontemporal_load(p);
  else
    x = *p;
  return make_float4(__uint_as_float(x[0] << 16), __uint_as_float(x[0] & 0xFFFF0000u),
                     __uint_as_float(x[1] << 16), __uint_as_float(x[1] & 0xFFFF0000u));
}
__device__ __forceinline__ void st_group(float* base, int g, const float4& v) {
  const f32x4v x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<f32x4v*>(base) + g);
}
__device__ __forceinline__ void st_group(bf16_t* base, int g, const float4& v) {
  // round to nearest even, as the pool copies and the outputs are rounded
  const uint32_t lo0 = from_f32<bf16_t>(v.x).x, hi0 = from_f32<bf16_t>(v.y).x;
  const uint32_t lo1 = from_f32<bf16_t>(v.z).x, hi1 = from_f32<bf16_t>(v.w).x;
  const u32x2v x = {lo0 | (hi0 << 16), lo1 | (hi1 << 16)};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x2v*>(base) + g);
}

template <int DK, int DV>
struct StateTile {
  static constexpr int CQ = DV / 4;      // 4-element groups per row
  static constexpr int RG = 256 / CQ;    // row groups
  static constexpr int RPT = DK / RG;    // rows per thread
  static constexpr int NV = RPT;         // groups per thread
};

// States [j0, j1) of split sp out of ns, over the m pre-merge states; a
// boundary that would fall between the merged pair (istar, istar + 1) moves one
// state on, so both sit in one range.
__device__ __forceinline__ void split_range(int m, int ns, int sp, int istar, int* j0, int* j1) {
  const int per = (m + ns - 1) / ns;
  int a0 = min(m, sp * per), a1 = min(m, (sp + 1) * per);
  if (istar >= 0) {
    if (a0 == istar + 1) ++a0;
    if (a1 == istar + 1) ++a1;
  }
  *j0 = a0;
  *j1 = a1;
}

// The decisions of a split step, handed to the finishing kernel.
struct DecodeRecord {
  int32_t b, istar;
  double I;
};

// The end of a step for head h, by one workgroup: the newest state
// (accumulated, or the new state k v^T in frame Gn, in the slot the merge
// freed or the first free slot; with bfloat16 storage in the open region),
// the output acc + lambda_{m'-1} (q.k) v, the exports and the metadata.
// open_at(r) gives the thread's r-th group of the newest state before the
// step (needed only when b = 0).
template <int DK, int DV, typename Tout, typename TS, typename OpenAt>
__device__ __forceinline__ void finish_step(const DecodeArgs& a, int h, int m, int b, int istar,
                                            double I, double Gn, float acc, float qk2,
                                            const float* sk, const float* sv, const double* sF,
                                            const double* sI, const int32_t* sN,
                                            const int32_t* sP, const float* sLam, Meta M,
                                            TS* states, float* open, OpenAt open_at) {
  using ST = StateTile<DK, DV>;
  constexpr int D = DK * DV;
  constexpr bool SB = sizeof(TS) == 2;
  const int tid = threadIdx.x;
  const int cq = tid % ST::CQ;
  const int rg = tid / ST::CQ;
  const int C = a.desc.C;
  const size_t ht = (size_t)h * a.hs;
  const int m_post = b ? (istar >= 0 ? m : m + 1) : m;
  // Delta rule (Gated DeltaNet form): the token writes beta k v^T, and an
  // accumulating newest state is first erased along k: with the true old
  // state f S~ (f = exp(Gn - F)) and u = S~^T k, the new state is
  //   f S~ + beta k (v - f u)^T.
  const bool delta = a.beta != nullptr;
  const float beta = delta ? a.beta[ht] : 1.f;
  const float fo = (!b && m > 0) ? __expf((float)(Gn - sF[m - 1])) : 0.f;
  __shared__ float sUp[ST::RG][DV];
  __shared__ float sU[DV];
  if (delta && !b) {
    float up[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < ST::NV; ++r) {
      const float kr = sk[rg + ST::RG * r];
      const float4 o = open_at(r);
      up[0] += kr * o.x;
      up[1] += kr * o.y;
      up[2] += kr * o.z;
      up[3] += kr * o.w;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) sUp[rg][4 * cq + c] = up[c];
    __syncthreads();
    if (tid < DV) {
      float u = 0.f;
#pragma unroll
      for (int g2 = 0; g2 < ST::RG; ++g2) u += sUp[g2][tid];
      sU[tid] = fo * u;   // (f u: the true state's S^T k)
    }
    __syncthreads();
  }
  {
    float* dst;
    if (SB)
      dst = open;
    else if (!b)
      dst = reinterpret_cast<float*>(states) + (size_t)sP[m - 1] * D;
    else
      dst = reinterpret_cast<float*>(states) + (size_t)((istar >= 0) ? sP[istar + 1] : sP[m]) * D;
    // the token's write beta (v - f u) (beta = 1, u = 0 in the gated form)
    float4 vq = reinterpret_cast<const float4*>(sv)[cq];
    if (delta) {
      const float4 uq = b ? make_float4(0.f, 0.f, 0.f, 0.f) : reinterpret_cast<const float4*>(sU)[cq];
      vq = make_float4(beta * (vq.x - uq.x), beta * (vq.y - uq.y), beta * (vq.z - uq.z),
                       beta * (vq.w - uq.w));
    }
    if (b) {
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) {
        const float kr = sk[rg + ST::RG * r];
        st_group(dst, tid + 256 * r, make_float4(kr * vq.x, kr * vq.y, kr * vq.z, kr * vq.w));
      }
    } else {
      const float f = fo;
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) {
        const float kr = sk[rg + ST::RG * r];
        const float4 o = open_at(r);
        float4 s;
        s.x = f * o.x + kr * vq.x;
        s.y = f * o.y + kr * vq.y;
        s.z = f * o.z + kr * vq.z;
        s.w = f * o.w + kr * vq.w;
        st_group(dst, tid + 256 * r, s);
      }
    }
  }
  // the new token's own contribution lambda_{m'-1} (q.k) times its write
  if (!a.skip_readout && tid < DV) {
    const float wv = delta ? beta * (sv[tid] - (b ? 0.f : sU[tid])) : sv[tid];
    acc += sLam[m_post - 1] * qk2 * wv;
    static_cast<Tout*>(a.out)[ht * DV + tid] = from_f32<Tout>(acc);
  }
  if (tid == 0) {
    if (a.b_out) a.b_out[ht] = (int8_t)b;
    if (a.merge_out) a.merge_out[ht] = istar;
    if (a.score_out) a.score_out[ht] = (float)I;
  }
  // metadata update (chronological arrays, parallel over slots)
  if (!b) {
    if (tid == 0) {
      M.F[m - 1] = Gn;
      M.n[m - 1] = sN[m - 1] + 1;
      M.ibar[m - 1] = sI[m - 1] + I;
    }
  } else {
    if (istar >= 0) {
      // merge istar, istar+1; shift later states down; freed slot goes to perm[m-1]
      for (int j = tid; j < C; j += 256) {
        if (j == istar) {
          M.F[j] = Gn;
          M.n[j] = sN[j] + sN[j + 1];
          M.ibar[j] = sI[j] + sI[j + 1];
        } else if (j > istar && j < m - 1) {
          M.F[j] = sF[j + 1];
          M.n[j] = sN[j + 1];
          M.ibar[j] = sI[j + 1];
          M.perm[j] = sP[j + 1];
        } else if (j == m - 1) {
          // the new state takes the freed slot
          M.perm[j] = sP[istar + 1];
          M.F[j] = Gn;
          M.n[j] = 1;
          M.ibar[j] = I;
        }
      }
    } else if (tid == 0) {
      M.F[m] = Gn;
      M.n[m] = 1;
      M.ibar[m] = I;
    }
    if (tid == 0) *M.m = m_post;
  }
  if (tid == 0) {
    *M.G = Gn;
    *M.tokens += 1;
  }
}

// SPLIT: one of NS workgroups of a head (partials to the metadata's scratch;
// decode_finish_kernel ends the step); otherwise the whole step of a head.
template <int DK, int DV, typename Tin, typename Tout, typename TS, bool SPLIT>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a) {
  using ST = StateTile<DK, DV>;
  constexpr int D = DK * DV;
  constexpr bool SB = sizeof(TS) == 2;  // bfloat16 closed states, float32 open region
  if (!cache_matches(a.cache, a.desc)) {  // refused: the descriptor is not the cache's
    flag_mismatch(a.cache);
    return;
  }
  const int ns = SPLIT ? a.nsplit : 1;
  const int h = blockIdx.x / ns;
  const int sp = blockIdx.x % ns;
  const int tid = threadIdx.x;
  const int C = a.desc.C;
  const int cq = tid % ST::CQ;
  const int rg = tid / ST::CQ;

  extern __shared__ double smem[];
  double* sF = smem;                                    // [C]
  double* sI = sF + C;                                  // [C]
  int32_t* sN = reinterpret_cast<int32_t*>(sI + C);     // [C]
  int32_t* sP = sN + C;                                 // [C]
  float* sLam = reinterpret_cast<float*>(sP + C);       // [C]
  __shared__ float sq[DK], sk[DK], sv[DV];
  __shared__ float red[8];
  __shared__ float sOut[ST::RG][DV];
  __shared__ double sArg[8];
  __shared__ int sArgI[8];
  __shared__ double sScal[4];
  __shared__ int sDec[4];

  const size_t ht = (size_t)h * a.hs;
  const Tin* q = static_cast<const Tin*>(a.q) + ht * DK;
  const Tin* k = static_cast<const Tin*>(a.k) + ht * DK;
  const Tin* v = static_cast<const Tin*>(a.v) + ht * DV;
  for (int i = tid; i < DK; i += 256) {
    sk[i] = to_f32(k[i]);
    sq[i] = a.skip_readout ? 0.f : to_f32(q[i]);
  }
  for (int i = tid; i < DV; i += 256) sv[i] = to_f32(v[i]);

  char* mbase = a.cache + a.meta_offset + (size_t)h * a.meta_stride;
  Meta M = meta_at(mbase, C);
  const int m = min(max(*M.m, 0), C);
  const double G0 = *M.G;
  for (int j = tid; j < C; j += 256) {
    sF[j] = M.F[j];
    sI[j] = M.ibar[j];
    sN[j] = M.n[j];
    sP[j] = min(max(M.perm[j], 0), C - 1);
    sLam[j] = a.lam ? to_f32(static_cast<const Tin*>(a.lam)[ht * C + j]) : 1.f;
  }
  __syncthreads();

  const double Gn = G0 + (double)a.g[ht];
  TS* states = reinterpret_cast<TS*>(a.cache + a.states_offset) + (size_t)h * C * D;
  float* open = SB ? reinterpret_cast<float*>(a.cache + a.open_offset) + (size_t)h * D : nullptr;
  // the newest state's storage: its slot, or the open region
  float* newest = SB ? open : reinterpret_cast<float*>(states) + (size_t)(m > 0 ? sP[m - 1] : 0) * D;

  // |k|^2, |v|^2, q.k
  float kk = 0.f, vv = 0.f, qk = 0.f;
  if (tid < 64) {
    for (int i = tid; i < DK; i += 64) {
      kk += sk[i] * sk[i];
      qk += sq[i] * sk[i];
    }
    for (int i = tid; i < DV; i += 64) vv += sv[i] * sv[i];
  }

  // newest state in registers, and the two scalars b = |S~|^2, c = k^T S~ v;
  // every workgroup of a split head reads it, so there it is read cacheable
  float4 Sopen[ST::NV];
  float ct = 0.f, bt = 0.f;
  if (m > 0) {
    const float4 vq = reinterpret_cast<const float4*>(sv)[cq];
#pragma unroll
    for (int r = 0; r < ST::NV; ++r) {
      Sopen[r] = ld_group<!SPLIT>(newest, tid + 256 * r);
      const float kr = sk[rg + ST::RG * r];
      const float4 s = Sopen[r];
      ct += kr * (s.x * vq.x + s.y * vq.y + s.z * vq.z + s.w * vq.w);
      bt += s.x * s.x + s.y * s.y + s.z * s.z + s.w * s.w;
    }
  }
  block_sum2_256(ct, bt, red);
  float kk2 = kk, vv2 = vv;
  block_sum2_256(kk2, vv2, red);
  float qk2 = qk, dummy = 0.f;
  block_sum2_256(qk2, dummy, red);

  // score and boundary decision (one thread, float64 scalars)
  if (tid == 0) {
    double I = 0.0;
    int b = 1;
    if (m > 0) {
      const double f = exp(Gn - sF[m - 1]);
      const double a2 = (double)kk2 * (double)vv2;
      I = info_score(a2, f * f * (double)bt, f * (double)ct, (double)D, a.eps, a.eps_rms);
      b = (I >= (double)a.tau) ? 1 : 0;
      if (a.b_ovr && a.b_ovr[ht] != -1) b = a.b_ovr[ht] ? 1 : 0;
      if (C == 1) b = 0;
    }
    sScal[0] = I;
    sDec[0] = b;
  }
  __syncthreads();
  const int b = sDec[0];
  const double I = sScal[0];

  // Alg. 2: lowest-density adjacent pair when a new state opens in a full cache
  int istar = -1;
  if (b && m == C) {
    double best = INFINITY;
    int bi = 0x7fffffff;
    for (int i = tid; i + 1 < C; i += 256) {
      const double d = (sI[i] + sI[i + 1]) / (double)(sN[i] + sN[i + 1]);
      if (d < best) {
        best = d;
        bi = i;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const double ob = __shfl_xor(best, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (ob < best || (ob == best && oi < bi)) {
        best = ob;
        bi = oi;
      }
    }
    if ((tid & 63) == 0) {
      sArg[tid >> 6] = best;
      sArgI[tid >> 6] = bi;
    }
    __syncthreads();
    if (tid == 0) {
      double bb = sArg[0];
      int ii = sArgI[0];
      for (int w = 1; w < 4; ++w)
        if (sArg[w] < bb || (sArg[w] == bb && sArgI[w] < ii)) {
          bb = sArg[w];
          ii = sArgI[w];
        }
      // NaN densities (scores from non-finite inputs) compare false, so a
      // sequential argmin that starts at pair 0 never moves to them, and stays
      // at pair 0 when pair 0's density is NaN or none is a number
      if (ii < 0 || ii > C - 2) ii = 0;
      if (__builtin_isnan((sI[0] + sI[1]) / (double)(sN[0] + sN[1]))) ii = 0;
      if (a.m_ovr && a.m_ovr[ht] != -1) {
        const int f = a.m_ovr[ht];
        if (f >= 0 && f <= C - 2)
          ii = f;
        else if (sp == 0)
          atomicOr(&reinterpret_cast<CacheHeader*>(a.cache)->flags, DLA_FLAG_BAD_MERGE_OVERRIDE);
      }
      sDec[1] = ii;
    }
    __syncthreads();
    istar = sDec[1];
  }
  const int m_post = b ? (istar >= 0 ? m : m + 1) : m;

  // stream this workgroup's states: readout partials and the state writes
  float o4[4] = {0.f, 0.f, 0.f, 0.f};
  float qr[ST::NV];
#pragma unroll
  for (int r = 0; r < ST::NV; ++r) qr[r] = sq[rg + ST::RG * r];
  int j0, j1;
  split_range(m, ns, sp, istar, &j0, &j1);

  for (int j = j0; j < j1; ++j) {
    const bool is_open = (j == m - 1);
    float4 X[ST::NV];
    if (is_open) {
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) X[r] = Sopen[r];
    } else {
      const TS* src = states + (size_t)sP[j] * D;
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) X[r] = ld_group<true>(src, tid + 256 * r);
    }
    const int post = (istar >= 0 && j > istar) ? j - 1 : j;
    const float w = a.skip_readout ? 0.f : sLam[post] * __expf((float)(Gn - sF[j]));
    float y0 = 0.f, y1 = 0.f, y2 = 0.f, y3 = 0.f;
#pragma unroll
    for (int r = 0; r < ST::NV; ++r) {
      y0 += qr[r] * X[r].x;
      y1 += qr[r] * X[r].y;
      y2 += qr[r] * X[r].z;
      y3 += qr[r] * X[r].w;
    }
    o4[0] += w * y0;
    o4[1] += w * y1;
    o4[2] += w * y2;
    o4[3] += w * y3;

    if (j == istar) {
      // merged pair, stored in this step's frame Gn:
      //   S~ = exp(Gn - F_i) S~_i + exp(Gn - F_{i+1}) S~_{i+1}.
      // Gn is at least as recent as either frame, so both factors are <= 1.
      // (The frame of the later state is not always the more recent one: the
      // left state may have been rewritten by a merge after its neighbour was
      // last written, and rebasing to the older frame can overflow.)
      const int j2 = j + 1;
      float4 Y[ST::NV];
      if (j2 == m - 1) {
#pragma unroll
        for (int r = 0; r < ST::NV; ++r) Y[r] = Sopen[r];
      } else {
        const TS* src = states + (size_t)sP[j2] * D;
#pragma unroll
        for (int r = 0; r < ST::NV; ++r) Y[r] = ld_group<true>(src, tid + 256 * r);
      }
      const float e2 = __expf((float)(Gn - sF[j2]));
      const float w2 = a.skip_readout ? 0.f : sLam[j] * e2;
      const float e1 = __expf((float)(Gn - sF[j]));
      float z0 = 0.f, z1 = 0.f, z2 = 0.f, z3 = 0.f;
      TS* dst = states + (size_t)sP[j] * D;
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) {
        z0 += qr[r] * Y[r].x;
        z1 += qr[r] * Y[r].y;
        z2 += qr[r] * Y[r].z;
        z3 += qr[r] * Y[r].w;
        float4 s;
        s.x = e1 * X[r].x + e2 * Y[r].x;
        s.y = e1 * X[r].y + e2 * Y[r].y;
        s.z = e1 * X[r].z + e2 * Y[r].z;
        s.w = e1 * X[r].w + e2 * Y[r].w;
        st_group(dst, tid + 256 * r, s);
      }
      o4[0] += w2 * z0;
      o4[1] += w2 * z1;
      o4[2] += w2 * z2;
      o4[3] += w2 * z3;
      ++j;  // the pair is done
    } else if (SB && is_open && b) {
      // the newest state closes: its bfloat16 copy goes to its slot, in its
      // own frame (a merge with its left neighbour is handled above)
      TS* dst = states + (size_t)sP[j] * D;
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) st_group(dst, tid + 256 * r, X[r]);
    }
  }

  // the workgroup's partial output
  if (!a.skip_readout) {
#pragma unroll
    for (int c = 0; c < 4; ++c) sOut[rg][4 * cq + c] = o4[c];
  }
  __syncthreads();
  float acc = 0.f;
  if (!a.skip_readout && tid < DV) {
#pragma unroll
    for (int g2 = 0; g2 < ST::RG; ++g2) acc += sOut[g2][tid];
  }
  if constexpr (SPLIT) {
    // for the finishing kernel: the partial, and (first workgroup) the decisions
    if (!a.skip_readout && tid < DV) decode_partials(mbase, C)[(size_t)sp * DV + tid] = acc;
    if (sp == 0 && tid == 0) {
      DecodeRecord* rec = reinterpret_cast<DecodeRecord*>(decode_record(mbase, C));
      rec->b = b;
      rec->istar = istar;
      rec->I = I;
    }
  } else {
    finish_step<DK, DV, Tout, TS>(a, h, m, b, istar, I, Gn, acc, qk2, sk, sv, sF, sI, sN, sP, sLam,
                                  M, states, open, [&](int r) { return Sopen[r]; });
  }
}

// The end of a split step, one workgroup per head: the partials of the NS
// workgroups summed in split order, then finish_step.
template <int DK, int DV, typename Tin, typename Tout, typename TS>
__global__ __launch_bounds__(256) void decode_finish_kernel(DecodeArgs a) {
  constexpr int D = DK * DV;
  constexpr bool SB = sizeof(TS) == 2;
  if (!cache_matches(a.cache, a.desc)) return;  // refused call (see decode_kernel)
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int C = a.desc.C;
  const int ns = a.nsplit;
  extern __shared__ double smem[];
  double* sF = smem;                                    // [C]
  double* sI = sF + C;                                  // [C]
  int32_t* sN = reinterpret_cast<int32_t*>(sI + C);     // [C]
  int32_t* sP = sN + C;                                 // [C]
  float* sLam = reinterpret_cast<float*>(sP + C);       // [C]
  __shared__ float sk[DK], sv[DV];
  __shared__ float red[8];
  const size_t ht = (size_t)h * a.hs;
  const Tin* q = static_cast<const Tin*>(a.q) + ht * DK;
  const Tin* k = static_cast<const Tin*>(a.k) + ht * DK;
  const Tin* v = static_cast<const Tin*>(a.v) + ht * DV;
  float qk = 0.f;
  for (int i = tid; i < DK; i += 256) {
    sk[i] = to_f32(k[i]);
    if (!a.skip_readout) qk += to_f32(q[i]) * sk[i];
  }
  for (int i = tid; i < DV; i += 256) sv[i] = to_f32(v[i]);
  char* mbase = a.cache + a.meta_offset + (size_t)h * a.meta_stride;
  Meta M = meta_at(mbase, C);
  const int m = min(max(*M.m, 0), C);
  const double Gn = *M.G + (double)a.g[ht];
  for (int j = tid; j < C; j += 256) {
    sF[j] = M.F[j];
    sI[j] = M.ibar[j];
    sN[j] = M.n[j];
    sP[j] = min(max(M.perm[j], 0), C - 1);
    sLam[j] = a.lam ? to_f32(static_cast<const Tin*>(a.lam)[ht * C + j]) : 1.f;
  }
  const DecodeRecord rec = *reinterpret_cast<const DecodeRecord*>(decode_record(mbase, C));
  float dummy = 0.f;
  block_sum2_256(qk, dummy, red);   // (its barriers also publish the LDS tables)
  float acc = 0.f;
  if (!a.skip_readout && tid < DV) {
    const float* part = decode_partials(mbase, C);
    for (int s2 = 0; s2 < ns; ++s2) acc += part[(size_t)s2 * DV + tid];
  }
  TS* states = reinterpret_cast<TS*>(a.cache + a.states_offset) + (size_t)h * C * D;
  float* open = SB ? reinterpret_cast<float*>(a.cache + a.open_offset) + (size_t)h * D : nullptr;
  const float* newest =
      SB ? open : reinterpret_cast<const float*>(states) + (size_t)(m > 0 ? sP[m - 1] : 0) * D;
  const int b = min(max(rec.b, 0), 1);
  const int istar = (b && m == C) ? min(max(rec.istar, 0), C - 2) : -1;
  finish_step<DK, DV, Tout, TS>(a, h, m, b, istar, rec.I, Gn, acc, qk, sk, sv, sF, sI, sN, sP,
                                sLam, M, states, open,
                                [&](int r) { return ld_group<true>(newest, threadIdx.x + 256 * r); });
}

// Workgroups per head: enough for about four per compute unit over all heads,
// at most kMaxSplit, and at least two states per workgroup.
int decode_splits(int nheads, int C) {
  int ns = (1024 + nheads - 1) / nheads;
  ns = ns < kMaxSplit ? ns : kMaxSplit;
  const int byc = C / 2 > 1 ? C / 2 : 1;
  ns = ns < byc ? ns : byc;
  return ns > 1 ? ns : 1;
}

template <int DK, int DV, typename Tin, typename Tout, typename TS>
static hipError_t launch_decode_t(const DecodeArgs& a, int nheads, hipStream_t s) {
  const size_t shm = (size_t)a.desc.C * (8 + 8 + 4 + 4 + 4);
  if (a.nsplit == 1) {
    hipLaunchKernelGGL((decode_kernel<DK, DV, Tin, Tout, TS, false>), dim3((unsigned)nheads),
                       dim3(256), shm, s, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((decode_kernel<DK, DV, Tin, Tout, TS, true>),
                     dim3((unsigned)(nheads * a.nsplit)), dim3(256), shm, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_finish_kernel<DK, DV, Tin, Tout, TS>), dim3((unsigned)nheads),
                     dim3(256), shm, s, a);
  return hipGetLastError();
}

template <int DK, int DV, typename TS>
static hipError_t launch_decode_dims(const DecodeArgs& a, int nheads, dla_dtype in, dla_dtype out,
                                     hipStream_t s) {
  if (in == DLA_F32 && out == DLA_F32) return launch_decode_t<DK, DV, float, float, TS>(a, nheads, s);
  if (in == DLA_F32 && out == DLA_BF16) return launch_decode_t<DK, DV, float, bf16_t, TS>(a, nheads, s);
  if (in == DLA_BF16 && out == DLA_F32) return launch_decode_t<DK, DV, bf16_t, float, TS>(a, nheads, s);
  return launch_decode_t<DK, DV, bf16_t, bf16_t, TS>(a, nheads, s);
}

template <int DK, int DV>
static hipError_t launch_decode_st(const DecodeArgs& a, int nheads, dla_dtype in, dla_dtype out,
                                   hipStream_t s) {
  if (a.desc.state_dtype == DLA_BF16) return launch_decode_dims<DK, DV, bf16_t>(a, nheads, in, out, s);
  return launch_decode_dims<DK, DV, float>(a, nheads, in, out, s);
}

hipError_t launch_decode(const DecodeArgs& a, int nheads, int dk, int dv, dla_dtype in,
                         dla_dtype out, hipStream_t s) {
  if (a.nsplit < 1 || a.nsplit > kMaxSplit) return hipErrorInvalidValue;
  if (dk == 128 && dv == 128) return launch_decode_st<128, 128>(a, nheads, in, out, s);
  if (dk == 64 && dv == 64) return launch_decode_st<64, 64>(a, nheads, in, out, s);
  if (dk == 128 && dv == 64) return launch_decode_st<128, 64>(a, nheads, in, out, s);
  return launch_decode_st<64, 128>(a, nheads, in, out, s);
}

}  // namespace dla
