// Prefill in the Gated DeltaNet form of the layer (Sec. 2.2, eq. delta_rule_rnn,
// with the decisions and merges of Sec. 3.1-3.2).
//
// With every state decayed by alpha_t = exp(g_t) first, a token that joins the
// newest state S takes the delta rule
//   S <- (I - beta_t k_t k_t^T) alpha_t S + beta_t k_t v_t^T
//      = alpha_t S + k_t u_t^T,   u_t = beta_t (v_t - (alpha_t S)^T k_t),
// and a token that opens a state starts it at beta_t k_t v_t^T, i.e. u_t =
// beta_t v_t.  So every state is the same decayed sum of rank-one terms k_s
// u_s^T over its tokens as the gated form with v_s replaced by u_s, and once the
// pseudo-values u_s are known the chunked update and readout stages apply
// unchanged.  The pseudo-values depend on the newest state before each token,
// which depends on every earlier decision, so they come from a sequential scan
// that keeps the newest state on chip: one 512-thread workgroup per head, each
// thread holding a (d_k / 8) x (d_v / 64) block of the state in registers.
// Per token it forms y = (alpha S)^T k and the score's three scalars (a =
// |k|^2 |v|^2, b = |alpha S|^2, c = y . v), decides (Alg. 1, with Alg. 2 at a
// full cache), and applies the rank-one step with u.  It emits the decisions,
// scores and merge indices, the death token of every state leader (the same
// bookkeeping as the gated scan), the cache's per-state counts and aggregated
// scores, and u as float32.
//
// The call then runs the chunked update and readout stages of the gated form
// over (q, k, u, lambda), on the gated prefill's schedule: with the scan in
// segments on a second stream, overlapped with the update and readout of the
// segments already scanned, unless the caller asks for serial stages.  For
// 16-bit inputs the update takes u in float32 (it stages every value as three
// bfloat16 terms, so the states stay float32 exact) and the readout a bfloat16
// copy of u (for its in-chunk part, which rounds values to bfloat16 in the
// gated form too); float32 inputs run the float32 stages on u.
#include "prefill.h"

namespace dla {

constexpr int DTHR = 512;        // threads of the delta scan
constexpr int DWAVE = DTHR / 64;
constexpr int DSL = 64;          // tokens staged in LDS per round

// Barrier for the per-token exchanges through LDS: waits for the wave's LDS
// operations only, so that the pseudo-values and exports stored to global
// memory stay in flight (a full __syncthreads would wait for those stores at
// every token).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt((63 & 15) | (7 << 4) | (0 << 8) | ((63 >> 4) << 14));
  __builtin_amdgcn_s_barrier();
}

template <int DK, int DV>
struct DeltaP {
  // wave w holds rows [w RB, (w + 1) RB) of the state, lane l columns
  // [l CB, (l + 1) CB): a wave's share of S^T k covers every column, so it
  // needs no exchange between lanes
  static constexpr int RB = DK / DWAVE;  // state rows per thread
  static constexpr int CB = DV / 64;     // state columns per thread
  static_assert(RB * DWAVE == DK && CB * 64 == DV, "state blocks");
  static size_t smem_bytes(int C) {
    size_t off = (size_t)DSL * (DK + DV) * 4;  // sK, sV
    off += (size_t)DSL * 4 * 5;                 // sAl, sBeta, sA, sBo, sMo
    off += (size_t)(DWAVE + 1) * DV * 4;        // sY, sU
    off += 2 * DWAVE * 4;                       // sRed
    off = round_up(off, 8);
    off += (size_t)C * 8;                       // sIb
    off += (size_t)C * 4 * 2;                   // sN, sLead
    return round_up(off, 16);
  }
};

template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(DTHR) void prefill_delta_scan_kernel(PrefillArgs a, PrefillWS w,
                                                                  int tb, int te,
                                                                  const float* __restrict__ beta,
                                                                  float* __restrict__ U,
                                                                  bf16_t* __restrict__ U16) {
  if (!cache_matches(a.cache, a.desc)) return;  // refused call (see the prep kernel)
  using P = DeltaP<DK, DV>;
  constexpr int RB = P::RB, CB = P::CB;
  constexpr int D = DK * DV;
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int rb = wv;    // row block of the thread's state block
  const int cb = lane;  // column block
  const int C = a.desc.C;
  const int T = a.T;
  const size_t tok0 = (size_t)h * T;

  extern __shared__ __align__(16) char smem[];
  float* sK = reinterpret_cast<float*>(smem);  // [DSL][DK]
  float* sV = sK + DSL * DK;                   // [DSL][DV]
  float* sAl = sV + DSL * DV;                  // alpha_t
  float* sBeta = sAl + DSL;
  float* sA = sBeta + DSL;                     // |k|^2 |v|^2
  int32_t* sBo = reinterpret_cast<int32_t*>(sA + DSL);
  int32_t* sMo = sBo + DSL;
  float* sY = reinterpret_cast<float*>(sMo + DSL);  // [waves][DV] partial y
  float* sU = sY + DWAVE * DV;                      // [DV] pseudo-values
  float* sRed = sU + DV;                            // [2 waves]
  double* sIb =
      reinterpret_cast<double*>(smem + round_up((size_t)((char*)(sRed + 2 * DWAVE) - smem), 8));
  int32_t* sN = reinterpret_cast<int32_t*>(sIb + C);
  int32_t* sLead = sN + C;

  Meta M = meta_at(a.cache + a.meta_offset + (size_t)h * a.meta_stride, C);
  InitView iv = init_at(w, h, C);
  // tokens [tb, te); a segment after the first resumes from the carry the
  // previous one left in the workspace (the bookkeeping, and the newest state
  // in this kernel's own thread order)
  ScarryView sv = scarry_at(w, h, C);
  const int m0 = min(max(*iv.m0, 0), C);
  for (int j = tid; j < C; j += DTHR) {
    if (tb == 0) {
      sIb[j] = j < m0 ? M.ibar[j] : 0.0;
      sN[j] = j < m0 ? M.n[j] : 0;
      sLead[j] = j - m0;  // states present before the call: negative leaders
    } else {
      sIb[j] = sv.ibar[j];
      sN[j] = sv.n[j];
      sLead[j] = sv.lead[j];
    }
  }
  // the newest state at the start of the call, true (decayed) values
  float S[RB][CB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) S[i][j] = 0.f;
  if (tb > 0) {
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) S[i][j] = sv.S[((size_t)tid * RB + i) * CB + j];
  } else if (m0 > 0) {
    const float* src =
        a.desc.state_dtype == DLA_BF16
            ? reinterpret_cast<const float*>(a.cache + a.open_offset) + (size_t)h * D
            : reinterpret_cast<const float*>(a.cache + a.states_offset) +
                  ((size_t)h * C + min(max(M.perm[m0 - 1], 0), C - 1)) * D;
    const float f = (float)exp(*M.G - M.F[m0 - 1]);
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) S[i][j] = f * src[(size_t)(rb * RB + i) * DV + cb * CB + j];
  }
  int m = tb > 0 ? min(max(*sv.m, 0), C) : m0;

  const Tin* Kin = static_cast<const Tin*>(a.k) + tok0 * DK;
  const Tin* Vin = static_cast<const Tin*>(a.v) + tok0 * DV;
  const float* g = a.g + tok0;
  const float* bt = beta + tok0;
  int32_t* death = w.death + tok0;
  float* Uh = U + tok0 * DV;
  bf16_t* U16h = U16 ? U16 + tok0 * DV : nullptr;  // bfloat16 copy (16-bit inputs)

  for (int c0 = tb; c0 < te; c0 += DSL) {
    const int nr = min(DSL, te - c0);
    __syncthreads();  // the previous round is done with the staged tokens
    for (int i = tid; i < nr * DK; i += DTHR) sK[i] = to_f32(Kin[(size_t)c0 * DK + i]);
    for (int i = tid; i < nr * DV; i += DTHR) sV[i] = to_f32(Vin[(size_t)c0 * DV + i]);
    for (int t = tid; t < nr; t += DTHR) {
      sAl[t] = __expf(g[c0 + t]);
      sBeta[t] = bt[c0 + t];
      sBo[t] = a.b_ovr ? (int)a.b_ovr[tok0 + c0 + t] : -1;
      sMo[t] = a.m_ovr ? a.m_ovr[tok0 + c0 + t] : -1;
    }
    __syncthreads();
    // a_t = |k_t|^2 |v_t|^2, one wave per token
    for (int t = wv; t < nr; t += DWAVE) {
      float kk = 0.f, vv = 0.f;
      for (int i = lane; i < DK; i += 64) kk += sK[t * DK + i] * sK[t * DK + i];
      for (int i = lane; i < DV; i += 64) vv += sV[t * DV + i] * sV[t * DV + i];
      kk = wave_sum(kk);
      vv = wave_sum(vv);
      if (lane == 0) sA[t] = kk * vv;
    }
    __syncthreads();

    for (int tt = 0; tt < nr; ++tt) {
      const int t = c0 + tt;
      const float al = sAl[tt];
      float kr[RB];
#pragma unroll
      for (int i = 0; i < RB; ++i) kr[i] = sK[tt * DK + rb * RB + i];
      // decay, and the block's shares of y = S^T k, |S|^2 and c = k^T S v
      float yp[CB];
#pragma unroll
      for (int j = 0; j < CB; ++j) yp[j] = 0.f;
      float bp = 0.f;
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < CB; ++j) {
          S[i][j] *= al;
          yp[j] += kr[i] * S[i][j];
          bp += S[i][j] * S[i][j];
        }
      float cp = 0.f;
#pragma unroll
      for (int j = 0; j < CB; ++j) cp += yp[j] * sV[tt * DV + cb * CB + j];
      // the waves' shares are added below; |S|^2 and c over the wave
      bp = wave_total_dpp(bp);
      cp = wave_total_dpp(cp);
#pragma unroll
      for (int j = 0; j < CB; ++j) sY[wv * DV + cb * CB + j] = yp[j];
      if (lane == 0) {
        sRed[wv] = bp;
        sRed[DWAVE + wv] = cp;
      }
      lds_barrier();
      float yj = 0.f;
      if (tid < DV) {
#pragma unroll
        for (int w2 = 0; w2 < DWAVE; ++w2) yj += sY[w2 * DV + tid];
      }
      double b = 0.0, c = 0.0;
#pragma unroll
      for (int w2 = 0; w2 < DWAVE; ++w2) {
        b += (double)sRed[w2];
        c += (double)sRed[DWAVE + w2];
      }
      // the decision, identical in every thread
      int bd;
      float It;
      if (m == 0) {  // the first token of an empty cache opens a state with score 0
        bd = 1;
        It = 0.f;
      } else {
        It = score_f(sA[tt], (float)b, (float)c, (float)D, a.eps, a.eps_rms);
        bd = (It >= a.tau) ? 1 : 0;
        if (sBo[tt] != -1) bd = sBo[tt] ? 1 : 0;
        if (C == 1) bd = 0;
      }
      if (bd) {
        int istar = -1;
        if (m == C) {
          // Alg. 2 on wave 0: the adjacent pair of lowest density, ties to the
          // lowest index (the gated scan's rules, overrides included)
          if (wv == 0) {
            double best = INFINITY;
            int bi = 0x7fffffff;
            for (int i = lane; i + 1 < C; i += 64) {
              const double d = (sIb[i] + sIb[i + 1]) / (double)(sN[i] + sN[i + 1]);
              if (d < best) {
                best = d;
                bi = i;
              }
            }
            wave_argmin_d(best, bi);
            istar = (bi >= 0 && bi <= C - 2) ? bi : 0;
            if (__builtin_isnan((sIb[0] + sIb[1]) / (double)(sN[0] + sN[1]))) istar = 0;
            const int fo = sMo[tt];
            if (fo != -1) {
              if (fo >= 0 && fo <= C - 2)
                istar = fo;
              else if (lane == 0)
                atomicOr(&reinterpret_cast<CacheHeader*>(a.cache)->flags,
                         DLA_FLAG_BAD_MERGE_OVERRIDE);
            }
            // the right state of the pair dies at token t
            const int ld = sLead[istar + 1];
            if (lane == 0) {
              if (ld >= 0)
                death[ld] = t;
              else
                iv.death0[ld + m0] = t;
            }
            for (int j0 = istar; j0 + 1 < m; j0 += 64) {
              const int j = j0 + lane;
              const bool act = j + 1 < m;
              double nI = 0.0;
              int nN = 0, nL = 0;
              if (act) {
                nI = (j == istar) ? sIb[j] + sIb[j + 1] : sIb[j + 1];
                nN = (j == istar) ? sN[j] + sN[j + 1] : sN[j + 1];
                nL = (j == istar) ? sLead[j] : sLead[j + 1];
              }
              __builtin_amdgcn_wave_barrier();
              if (act) {
                sIb[j] = nI;
                sN[j] = nN;
                sLead[j] = nL;
              }
              __builtin_amdgcn_wave_barrier();
            }
          }
          m -= 1;
        }
        if (tid == 0) {
          sN[m] = 1;
          sIb[m] = (double)It;
          sLead[m] = t;
          death[t] = T;
          if (a.b_out) a.b_out[tok0 + t] = 1;
          if (a.merge_out) a.merge_out[tok0 + t] = istar;
          if (a.score_out) a.score_out[tok0 + t] = It;
        }
        m += 1;
      } else {
        if (tid == 0) {
          sN[m - 1] += 1;
          sIb[m - 1] += (double)It;
          death[t] = -1;
          if (a.b_out) a.b_out[tok0 + t] = 0;
          if (a.merge_out) a.merge_out[tok0 + t] = -1;
          if (a.score_out) a.score_out[tok0 + t] = It;
        }
      }
      // pseudo-values, then the rank-one step (a new state starts from zero)
      if (tid < DV) {
        const float u = sBeta[tt] * (sV[tt * DV + tid] - (bd ? 0.f : yj));
        sU[tid] = u;
        Uh[(size_t)t * DV + tid] = u;
        if (U16h) U16h[(size_t)t * DV + tid] = from_f32<bf16_t>(u);
      }
      lds_barrier();
      float uc[CB];
#pragma unroll
      for (int j = 0; j < CB; ++j) uc[j] = sU[cb * CB + j];
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < CB; ++j) S[i][j] = (bd ? 0.f : S[i][j]) + kr[i] * uc[j];
    }
  }
  __syncthreads();
  if (te < T) {
    // the carry for the next segment
    for (int j = tid; j < C; j += DTHR) {
      sv.ibar[j] = sIb[j];
      sv.n[j] = sN[j];
      sv.lead[j] = sLead[j];
    }
    if (tid == 0) *sv.m = m;
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) sv.S[((size_t)tid * RB + i) * CB + j] = S[i][j];
    return;
  }
  for (int j = tid; j < m; j += DTHR) {
    M.n[j] = sN[j];
    M.ibar[j] = sIb[j];
  }
}

template <int DK, int DV>
static size_t delta_smem(int C) {
  return DeltaP<DK, DV>::smem_bytes(C);
}

size_t prefill_delta_scan_smem(const dla_cache_desc& d) {
  if (d.d_k == 128 && d.d_v == 128) return delta_smem<128, 128>(d.C);
  if (d.d_k == 64 && d.d_v == 64) return delta_smem<64, 64>(d.C);
  if (d.d_k == 128 && d.d_v == 64) return delta_smem<128, 64>(d.C);
  return delta_smem<64, 128>(d.C);
}

template <int DK, int DV, typename Tin>
static hipError_t launch_delta_scan_t(const PrefillArgs& a, const PrefillWS& w, int tb, int te,
                                      const float* beta, float* U, bf16_t* U16, hipStream_t s) {
  const size_t shm = DeltaP<DK, DV>::smem_bytes(a.desc.C);
  if (shm > 160 * 1024) return hipErrorInvalidValue;
  auto k = prefill_delta_scan_kernel<DK, DV, Tin>;
  if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
      hipSuccess)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3(a.desc.B * a.desc.H), dim3(DTHR), shm, s, a, w, tb, te, beta, U, U16);
  return hipGetLastError();
}

template <int DK, int DV>
static hipError_t launch_delta_scan_dims(const PrefillArgs& a, const PrefillWS& w, int tb, int te,
                                         const float* beta, float* U, bf16_t* U16,
                                         hipStream_t s) {
  if (a.in_dtype == DLA_F32) return launch_delta_scan_t<DK, DV, float>(a, w, tb, te, beta, U, U16, s);
  return launch_delta_scan_t<DK, DV, bf16_t>(a, w, tb, te, beta, U, U16, s);
}

static hipError_t launch_delta_scan(const PrefillArgs& a, const PrefillWS& w, int tb, int te,
                                    const float* beta, float* U, bf16_t* U16, hipStream_t s) {
  const int dk = a.desc.d_k, dv = a.desc.d_v;
  if (dk == 128 && dv == 128) return launch_delta_scan_dims<128, 128>(a, w, tb, te, beta, U, U16, s);
  if (dk == 64 && dv == 64) return launch_delta_scan_dims<64, 64>(a, w, tb, te, beta, U, U16, s);
  if (dk == 128 && dv == 64) return launch_delta_scan_dims<128, 64>(a, w, tb, te, beta, U, U16, s);
  return launch_delta_scan_dims<64, 128>(a, w, tb, te, beta, U, U16, s);
}

// Workspace of a delta-form prefill: the stages' workspace (for the serial or
// the pipelined plan; the float32 stages for float32 inputs), then the write
// vectors u (float32), and for 16-bit inputs a bfloat16 copy of them.
struct DeltaWS {
  size_t u, u16, total;
};

static DeltaWS delta_ws(const dla_cache_desc& d, int T, dla_dtype in, bool readout, bool serial,
                        size_t budget) {
  DeltaWS r;
  const size_t nh = (size_t)d.B * d.H;
  size_t off = round_up(prefill_workspace_bytes(d, T, in, readout, serial, budget), 256);
  r.u = off;
  off = round_up(off + nh * T * d.d_v * 4, 256);
  r.u16 = off;
  off = round_up(off + (in != DLA_F32 && readout ? nh * T * d.d_v * 2 : 0), 256);
  r.total = off;
  return r;
}

size_t prefill_delta_workspace_bytes(const dla_cache_desc& d, int T, dla_dtype in, bool readout,
                                     bool serial, size_t budget) {
  return delta_ws(d, T, in, readout, serial, budget).total;
}

// The stages of the gated prefill's schedule: serial (frames, the whole scan,
// then update and readout segment by segment, on s), or pipelined (the scan
// segment by segment on a second stream forked from s after the frames, and
// segment k's update and readout on s after scan segment k; the last
// segment's wait joins the second stream into s, and so does every error
// path after the fork).
hipError_t launch_prefill_delta(const PrefillArgs& a, const float* beta, hipStream_t s) {
  const bool readout = !a.skip_readout;
  const bool wide = a.in_dtype != DLA_F32;
  const bool serial = a.serial != 0;
  const DeltaWS L = delta_ws(a.desc, a.T, a.in_dtype, readout, serial, a.pool_budget);
  const size_t nh = (size_t)a.desc.B * a.desc.H;
  char* base = a.workspace;
  float* U = reinterpret_cast<float*>(base + L.u);
  bf16_t* U16 = wide && readout ? reinterpret_cast<bf16_t*>(base + L.u16) : nullptr;
  // the update takes u (float32), the readout u in the inputs' type
  PrefillArgs fu = a;
  fu.v = U;
  fu.v_f32 = wide ? 1 : 0;
  PrefillArgs fr = fu;
  fr.v_f32 = 0;
  if (wide) fr.v = U16;
  const bool pipe = pipelined(a.T, a.in_dtype, readout, serial);
  SegPlan p = seg_plan(a.desc, a.T, a.in_dtype, readout, serial, a.pool_budget);
  if (pipe && p.shared) {
    // Here the scan is the long stage (its sequential chain per token takes
    // about three times the update and readout), so the segments stay at the
    // ramp's first size instead of growing: what remains after the scan, the
    // last segment's update and readout, is then short.  The pool is shared,
    // so the segments change neither the workspace nor the results.
    p.fit = p.first;
    p.nseg = 0;
    p.nch_seg = 0;
    for (int b = 0; b < p.nch; ++p.nseg) {
      const int n = ramp_size(p.first, p.fit, p.nseg, p.nch - b);
      p.nch_seg = n > p.nch_seg ? n : p.nch_seg;
      b += n;
    }
  }
  const PrefillWS w = ws_layout(base, nh, a.T, a.desc.C, a.desc.d_k * a.desc.d_v, p.nch);
  hipError_t e;
  if ((e = launch_prefill_prep(fu, s)) != hipSuccess) return e;
  hipStream_t side = s;
  hipEvent_t* pev = nullptr;
  bool forked = false;
  auto fail = [&](hipError_t err) -> hipError_t {
    if (forked && hipEventRecord(pev[0], side) == hipSuccess) (void)hipStreamWaitEvent(s, pev[0], 0);
    return err;
  };
  if (pipe) {
    if ((e = pipe_resources(s, p.nseg + 1, &side, &pev)) != hipSuccess) return e;
    if ((e = hipEventRecord(pev[0], s)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(side, pev[0], 0)) != hipSuccess) return e;
    forked = true;
    for (int seg = 0; seg < p.nseg; ++seg) {
      int cs, ce;
      seg_range(p, seg, &cs, &ce);
      const int te = (seg + 1 == p.nseg) ? a.T : ce * p.RL;
      if ((e = launch_delta_scan(a, w, cs * p.RL, te, beta, U, U16, side)) != hipSuccess)
        return fail(e);
      if ((e = hipEventRecord(pev[1 + seg], side)) != hipSuccess) return fail(e);
    }
  } else if ((e = launch_delta_scan(a, w, 0, a.T, beta, U, U16, s)) != hipSuccess) {
    return e;
  }
  for (int seg = 0; seg < p.nseg; ++seg) {
    if (pipe && (e = hipStreamWaitEvent(s, pev[1 + seg], 0)) != hipSuccess) return fail(e);
    if ((e = launch_prefill_update(fu, p, seg, s)) != hipSuccess) return fail(e);
    if (readout && (e = launch_prefill_readout(fr, p, seg, s)) != hipSuccess) return fail(e);
  }
  // (the last segment's wait on pev[nseg] has joined the second stream)
  return hipSuccess;
}

}  // namespace dla
