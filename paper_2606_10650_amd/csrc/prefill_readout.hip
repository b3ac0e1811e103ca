// Prefill, stage 3: multi-state readout and state-cache maintenance.
//
// Readout (eq. capacity_bounded_output): o_t = sum_j lambda[t][j] q_t^T S_j over
// the states of the cache after token t.  The decisions of stage 2 fix, for
// every token, which states exist; this stage turns them into dense MFMA work.
//
// One workgroup per (head, 32 value columns), sequential over chunks of 128
// tokens; each of the 4 waves owns 32 tokens of a chunk.  For a chunk:
//   * inter-chunk part: every state S_j present at the chunk start contributes
//     lambda[t][x_j(t)] exp(G_t - F_j) q_t^T S~_j, where x_j(t) is its
//     chronological index at token t.  A state's index is the number of live
//     state leaders up to it, and a leader is live at t while its death token
//     (from stage 2) is later than t, so x_j(t) is a running count over j.  The
//     product S~_j^T Q^T is a 32 x 32 bf16 MFMA tile per (state, wave) with K =
//     d_k; S~_j is staged through LDS (double buffered) and the weight is a
//     per-lane scalar because each lane owns one token of the output tile.
//   * intra-chunk part: (Q K^T (.) M) V over the chunk's own tokens, with
//     M[t][s] = [s <= t] exp(G_t - G_s) lambda[t][slot_t(s)], slot_t(s) being
//     the index at token t of the state that holds token s.
//   * state update: the states alive after the chunk are the surviving leaders;
//     each new or changed one is the decayed sum of the old states it absorbed
//     plus sum_s exp(G_end - G_s) k_s v_s^T over its tokens in the chunk, stored
//     in the frame G_end.  Unchanged states are not touched (lazy decay).
#include <type_traits>

#include "mfma.h"
#include "prefill.h"

namespace dla {

constexpr int RL = 128;  // tokens per chunk (4 waves x 32)
constexpr int NC = 32;   // value columns per workgroup

template <int DK, typename Tin>
struct ReadoutSmem {
  static constexpr int SA = DK + 16 / (int)sizeof(Tin);  // padded row of a staged state slice
  static size_t bytes(int C) {
    size_t off = 2 * NC * SA * sizeof(Tin);  // sA
    off += (size_t)RL * DK * sizeof(Tin);    // sK
    off += (size_t)RL * NC * sizeof(Tin);    // sV
    off = round_up(off, 16);
    off += RL * 8 + RL * 4 + RL * 4;         // sG, sDec, sDeath
    off += (size_t)C * 8;                    // sF
    off += (size_t)C * 4 * 11;               // int arrays
    return off;
  }
};

template <int DK, int DV, typename Tin, typename Tout>
__global__ __launch_bounds__(256) void prefill_readout_kernel(PrefillArgs a, PrefillWS w) {
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using SM = ReadoutSmem<DK, Tin>;
  constexpr int D = DK * DV;
  constexpr int NCG = DV / NC;
  constexpr int KS = DK / 16;
  constexpr int SA = SM::SA;
  const int nh = a.desc.B * a.desc.H;
  // XCD-aware mapping: workgroups are dealt to the 8 XCDs round-robin by id, so
  // give all column groups of one head the same id modulo 8 (shared L2).
  const int bid = blockIdx.x;
  const int slotid = bid >> 3;
  const int cg = slotid % NCG;
  const int h = (slotid / NCG) * 8 + (bid & 7);
  if (h >= nh) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int C = a.desc.C;
  const int T = a.T;
  const bool do_out = !a.skip_readout;

  extern __shared__ __align__(16) char smem[];
  Tin* sA = reinterpret_cast<Tin*>(smem);
  Tin* sK = sA + 2 * NC * SA;
  Tin* sV = sK + RL * DK;
  char* p = reinterpret_cast<char*>(sV + RL * NC);
  p = smem + round_up((size_t)(p - smem), 16);
  double* sG = reinterpret_cast<double*>(p);
  float* sDec = reinterpret_cast<float*>(sG + RL);
  int32_t* sDeath = reinterpret_cast<int32_t*>(sDec + RL);
  double* sF = reinterpret_cast<double*>(sDeath + RL);
  int32_t* sPerm = reinterpret_cast<int32_t*>(sF + C);
  int32_t* sLead = sPerm + C;
  int32_t* sDt = sLead + C;
  int32_t* eJa = sDt + C;
  int32_t* eJb = eJa + C;
  int32_t* eR0 = eJb + C;
  int32_t* eR1 = eR0 + C;
  int32_t* ePhys = eR1 + C;
  int32_t* eLead = ePhys + C;
  int32_t* ePool = eLead + C;
  int32_t* eChg = ePool + C;
  __shared__ int sMend;

  InitView iv = init_at(w, h, C);
  const int m0 = min(max(*iv.m0, 0), C);
  int m = m0;
  for (int j = tid; j < C; j += 256) {
    sPerm[j] = min(max(iv.perm0[j], 0), C - 1);
    sF[j] = iv.F0[j];
    sLead[j] = j - m0;
  }

  float* states = reinterpret_cast<float*>(a.cache + a.states_offset) + (size_t)h * C * D;
  const double* Gtok = w.Gtok + (size_t)h * T;
  const int32_t* death = w.death + (size_t)h * T;
  const Tin* Kin = static_cast<const Tin*>(a.k) + (size_t)h * T * DK;
  const Tin* Vin = static_cast<const Tin*>(a.v) + (size_t)h * T * DV;
  const Tin* Qin = static_cast<const Tin*>(a.q) + (size_t)h * T * DK;
  const Tin* Lin = a.lam ? static_cast<const Tin*>(a.lam) + (size_t)h * T * C : nullptr;
  Tout* Out = a.out ? static_cast<Tout*>(a.out) + (size_t)h * T * DV : nullptr;

  // stage the 32-column slice of logical state j into sA[buf] as [column][k]
  auto stage = [&](int j, int buf) {
    const float* src = states + (size_t)sPerm[j] * D + cg * NC;
    const int c = tid & 31;
#pragma unroll
    for (int u = 0; u < DK / 64; ++u) {
      const int k0 = 8 * ((tid >> 5) + 8 * u);
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = src[(size_t)(k0 + e) * DV + c];
      Tin* dst = sA + (size_t)(buf * NC + c) * SA + k0;
#pragma unroll
      for (int e = 0; e < 8; ++e) dst[e] = from_f32<Tin>(x[e]);
    }
  };

  for (int c0 = 0; c0 < T; c0 += RL) {
    const int nrow = min(RL, T - c0);
    const int c1 = c0 + nrow;
    __syncthreads();
    for (int i = tid; i < RL; i += 256) {
      sG[i] = Gtok[c0 + min(i, nrow - 1)];
      sDeath[i] = (i < nrow) ? death[c0 + i] : -1;
    }
    for (int j = tid; j < m; j += 256) {
      const int ld = sLead[j];
      sDt[j] = (ld >= 0) ? death[ld] : iv.death0[ld + m0];
    }
    // K rows (all d_k) and V rows (this group's columns) of the chunk; rows past
    // the end of the sequence are zero
    for (int idx = tid; idx < RL * DK / 8; idx += 256) {
      const int r = idx / (DK / 8), k8 = idx % (DK / 8);
      Tin* dst = sK + r * DK + 8 * k8;
      if (r < nrow) {
        const Tin* src = Kin + (size_t)(c0 + r) * DK + 8 * k8;
#pragma unroll
        for (int e = 0; e < 8; ++e) dst[e] = src[e];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) dst[e] = from_f32<Tin>(0.f);
      }
    }
    for (int idx = tid; idx < RL * NC; idx += 256) {
      const int r = idx / NC, c = idx % NC;
      sV[idx] = (r < nrow) ? Vin[(size_t)(c0 + r) * DV + cg * NC + c] : from_f32<Tin>(0.f);
    }
    __syncthreads();
    const double Gend = sG[nrow - 1];
    for (int i = tid; i < RL; i += 256) sDec[i] = (i < nrow) ? (float)exp(Gend - sG[i]) : 0.f;

    // ------------------------------------------------------------- readout
    if (do_out) {
      const int tr = wv * 32 + l32;  // this lane's token within the chunk
      const bool rv = tr < nrow;
      const int trc = rv ? tr : nrow - 1;
      const double Gt = sG[trc];
      FT qf[KS];
      const Tin* qrow = Qin + (size_t)(c0 + trc) * DK;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = rv ? FR::load(qrow + 16 * ks + 8 * half) : FR::zero();
      const Tin* lrow = Lin ? Lin + (size_t)(c0 + trc) * C : nullptr;
      f32x16 acc = zero16();
      int cnt = 0;
      if (m > 0) stage(0, 0);
      __syncthreads();
      for (int j = 0; j < m; ++j) {
        const int buf = j & 1;
        if (j + 1 < m) stage(j + 1, buf ^ 1);
        f32x16 fr = zero16();
        const Tin* arow = sA + (size_t)(buf * NC + l32) * SA;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) FR::mma(fr, FR::load(arow + 16 * ks + 8 * half), qf[ks]);
        cnt += (sDt[j] > c0 + tr) ? 1 : 0;
        float wgt = 0.f;
        if (rv) {
          const float lam = lrow ? to_f32(lrow[max(cnt - 1, 0)]) : 1.f;
          wgt = lam * __expf((float)(Gt - sF[j]));
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] += wgt * fr[r];
        __syncthreads();
      }
      const int Aold = cnt;  // states from before the chunk still live at token t

      // live in-chunk leaders at token t as a bit mask over the chunk
      uint32_t am[RL / 32];
#pragma unroll
      for (int q = 0; q < RL / 32; ++q) am[q] = 0u;
      for (int u = 0; u < nrow; ++u)
        if (sDeath[u] > c0 + tr) am[u >> 5] |= 1u << (u & 31);

      for (int sb = 0; sb <= wv; ++sb) {
        if (32 * sb >= nrow) break;
        f32x16 pt = zero16();
        const Tin* krow = sK + (size_t)(32 * sb + l32) * DK;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) FR::mma(pt, FR::load(krow + 16 * ks + 8 * half), qf[ks]);
        float pw[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int s = 32 * sb + out_row(r, lane);
          float wt = 0.f;
          if (rv && s <= tr) {
            int cl = 0;
#pragma unroll
            for (int q = 0; q < RL / 32; ++q) {
              const uint32_t mk = (q < (s >> 5)) ? 0xFFFFFFFFu
                                 : (q == (s >> 5) ? (0xFFFFFFFFu >> (31 - (s & 31))) : 0u);
              cl += __popc(am[q] & mk);
            }
            const int idx = min(max(Aold + cl - 1, 0), C - 1);
            const float lam = lrow ? to_f32(lrow[idx]) : 1.f;
            wt = lam * __expf((float)(Gt - sG[s]));
          }
          pw[r] = pt[r] * wt;
        }
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          float va[8];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            va[e] = to_f32(sV[(32 * sb + 16 * st + 8 * (e >> 2) + 4 * half + (e & 3)) * NC + l32]);
          FR::mma(acc, FR::from_floats(va), FR::from_floats(pw + 8 * st));
        }
      }
      if (rv) {
        Tout* orow = Out + (size_t)(c0 + tr) * DV + cg * NC;
#pragma unroll
        for (int r = 0; r < 16; ++r) orow[out_row(r, lane)] = from_f32<Tout>(acc[r]);
      }
    }

    // ------------------------------------------------------- state update
    __syncthreads();
    if (tid == 0) {
      int ne = 0, lastOld = -1;
      for (int j = 0; j < m; ++j) {
        if (sDt[j] >= c1) {
          eJa[ne] = j;
          eJb[ne] = j;
          eR0[ne] = 0;
          eR1[ne] = -1;
          eLead[ne] = sLead[j];
          lastOld = ne;
          ++ne;
        } else if (ne > 0) {
          eJb[ne - 1] = j;  // merged into the live state on its left
        }
      }
      const int firstNew = ne;
      for (int i = 0; i < nrow; ++i) {
        if (sDeath[i] >= c1) {
          eJa[ne] = -1;
          eJb[ne] = -2;
          eR0[ne] = i;
          eR1[ne] = nrow - 1;
          eLead[ne] = c0 + i;
          if (ne > firstNew) {
            eR1[ne - 1] = i - 1;
          } else if (lastOld >= 0) {
            eR0[lastOld] = 0;
            eR1[lastOld] = i - 1;
          }
          ++ne;
        }
      }
      if (ne == firstNew && lastOld >= 0) {
        eR0[lastOld] = 0;
        eR1[lastOld] = nrow - 1;
      }
      int np = 0;
      for (int j = 0; j < m; ++j)
        if (sDt[j] < c1) ePool[np++] = sPerm[j];
      for (int j = m; j < C; ++j) ePool[np++] = sPerm[j];
      int pi = 0;
      for (int e = 0; e < ne; ++e) {
        ePhys[e] = (eJa[e] >= 0) ? sPerm[eJa[e]] : ePool[pi++];
        eChg[e] = (eJa[e] < 0 || eJb[e] > eJa[e] || eR1[e] >= eR0[e]) ? 1 : 0;
      }
      // remaining free slots keep their order after the live ones
      for (int x = 0; pi + x < np; ++x) ePool[x] = ePool[pi + x];
      sMend = ne;
    }
    __syncthreads();
    const int ne = sMend;
    for (int phase = 0; phase < 2; ++phase) {
      for (int e = 0; e < ne; ++e) {
        if (!eChg[e] || ((eJa[e] >= 0) != (phase == 0))) continue;
        const int c = tid & 31;
        float* dst = states + (size_t)ePhys[e] * D + cg * NC + c;
        const int ja = eJa[e], jb = eJb[e], r0 = eR0[e], r1 = eR1[e];
        const int i0 = tid >> 5;
        float val[DK / 8];
#pragma unroll
        for (int u = 0; u < DK / 8; ++u) val[u] = 0.f;
        for (int j = ja; j <= jb; ++j) {
          const float f = __expf((float)(Gend - sF[j]));
          const float* src = states + (size_t)sPerm[j] * D + cg * NC + c;
#pragma unroll
          for (int u = 0; u < DK / 8; ++u) val[u] += f * src[(size_t)(i0 + 8 * u) * DV];
        }
        for (int s = r0; s <= r1; ++s) {
          const float vs = sDec[s] * to_f32(sV[s * NC + c]);
#pragma unroll
          for (int u = 0; u < DK / 8; ++u) val[u] += vs * to_f32(sK[s * DK + i0 + 8 * u]);
        }
#pragma unroll
        for (int u = 0; u < DK / 8; ++u) dst[(size_t)(i0 + 8 * u) * DV] = val[u];
      }
      __syncthreads();
    }
    if (tid == 0) {
      int np_rest = C - ne;
      for (int e = 0; e < ne; ++e) {
        const int ja = eJa[e];
        const double f = eChg[e] ? Gend : sF[ja];
        sF[e] = f;  // ja >= e for states with an old part: read before overwritten
        sLead[e] = eLead[e];
      }
      for (int e = 0; e < ne; ++e) sPerm[e] = ePhys[e];
      for (int x = 0; x < np_rest; ++x) sPerm[ne + x] = ePool[x];
      sMend = ne;
    }
    __syncthreads();
    m = sMend;
  }

  if (cg == 0) {
    Meta M = meta_at(a.cache + a.meta_offset + (size_t)h * a.meta_stride, C);
    for (int j = tid; j < C; j += 256) {
      M.perm[j] = sPerm[j];
      if (j < m) M.F[j] = sF[j];
    }
    if (tid == 0) {
      *M.m = m;
      *M.G = Gtok[T - 1];
      *M.tokens += T;
    }
  }
}

template <int DK, int DV, typename Tin>
static hipError_t launch_readout_t(const PrefillArgs& a, const PrefillWS& w, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  const int grid = (int)round_up(nh, 8) * (DV / NC);
  const size_t shm = ReadoutSmem<DK, Tin>::bytes(a.desc.C);
  if (shm > 160 * 1024) return hipErrorInvalidValue;
  if (a.out_dtype == DLA_F32) {
    auto k = prefill_readout_kernel<DK, DV, Tin, float>;
    hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    hipLaunchKernelGGL(k, dim3(grid), dim3(256), shm, s, a, w);
  } else {
    auto k = prefill_readout_kernel<DK, DV, Tin, bf16_t>;
    hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    hipLaunchKernelGGL(k, dim3(grid), dim3(256), shm, s, a, w);
  }
  return hipGetLastError();
}

template <int DK, int DV>
static hipError_t launch_readout_dims(const PrefillArgs& a, const PrefillWS& w, hipStream_t s) {
  if (a.in_dtype == DLA_F32) return launch_readout_t<DK, DV, float>(a, w, s);
  return launch_readout_t<DK, DV, bf16_t>(a, w, s);
}

hipError_t launch_prefill_readout(const PrefillArgs& a, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C);
  const int dk = a.desc.d_k, dv = a.desc.d_v;
  if (dk == 128 && dv == 128) return launch_readout_dims<128, 128>(a, w, s);
  if (dk == 64 && dv == 64) return launch_readout_dims<64, 64>(a, w, s);
  if (dk == 128 && dv == 64) return launch_readout_dims<128, 64>(a, w, s);
  return launch_readout_dims<64, 128>(a, w, s);
}

}  // namespace dla
