// Prefill, stages 1 and 2: token frame preparation, and the sequential
// boundary scan with the capacity schedule (Alg. 1 and Alg. 2, Sec. 3.1-3.2).
//
// Stage 1 (prep, one workgroup per head): the cumulative log-decay of every
// token in float64, and a copy of the cache's per-head metadata as it was
// before the call (later stages overwrite the cache).
//
// Stage 2 (scan, one workgroup per head, sequential over tokens): the newest
// state lives in registers (float32, 64 values per thread for d = 128).  Per
// token: the two scalars b = |S|^2 and c = k^T S v (one block reduction), the
// score in float64 from its rank-one closed form, the boundary, and -- when a
// new state opens in a full cache -- the argmin over the C-1 adjacent pair
// densities kept in LDS.  Emits b_t, merge index and score per token, and the
// death token of every state leader (the token at which Alg. 2 merged that
// state into its left neighbour), from which the readout stage reconstructs the
// chronological index of every state at every token without a replay.
#include "prefill.h"

namespace dla {

// ---------------------------------------------------------------------------
// stage 1
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void prefill_prep_kernel(PrefillArgs a, PrefillWS w) {
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int C = a.desc.C;
  const int T = a.T;
  Meta M = meta_at(a.cache + a.meta_offset + (size_t)h * a.meta_stride, C);
  InitView iv = init_at(w, h, C);
  const int m0 = min(max(*M.m, 0), C);
  const double G0 = *M.G;
  if (tid == 0) {
    *iv.m0 = m0;
    *iv.G0 = G0;
  }
  for (int j = tid; j < C; j += 256) {
    iv.F0[j] = M.F[j];
    iv.perm0[j] = M.perm[j];
    iv.death0[j] = T;
  }
  __shared__ double part[256];
  const float* g = a.g + (size_t)h * T;
  const int per = (T + 255) / 256;
  const int t0 = min(T, tid * per);
  const int t1 = min(T, t0 + per);
  double s = 0.0;
  for (int t = t0; t < t1; ++t) s += (double)g[t];
  part[tid] = s;
  __syncthreads();
  // exclusive scan of the 256 partial sums (Hillis-Steele on a copy)
  for (int o = 1; o < 256; o <<= 1) {
    const double x = (tid >= o) ? part[tid - o] : 0.0;
    __syncthreads();
    part[tid] += x;
    __syncthreads();
  }
  double run = G0 + part[tid] - s;
  double* G = w.Gtok + (size_t)h * T;
  for (int t = t0; t < t1; ++t) {
    run += (double)g[t];
    G[t] = run;
  }
}

hipError_t launch_prefill_prep(const PrefillArgs& a, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C);
  hipLaunchKernelGGL(prefill_prep_kernel, dim3(nh), dim3(256), 0, s, a, w);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// stage 2
// ---------------------------------------------------------------------------
template <int DK, int DV>
struct ScanTile {
  static constexpr int CQ = DV / 4;
  static constexpr int RG = 256 / CQ;
  static constexpr int NV = DK / RG;
};

template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(256) void prefill_scan_kernel(PrefillArgs a, PrefillWS w) {
  using ST = ScanTile<DK, DV>;
  constexpr int D = DK * DV;
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int C = a.desc.C;
  const int T = a.T;
  const int cq = tid % ST::CQ;
  const int rg = tid / ST::CQ;

  extern __shared__ double smem[];
  double* sI = smem;                                     // [C] aggregated scores
  int32_t* sN = reinterpret_cast<int32_t*>(sI + C);      // [C] token counts
  int32_t* sLead = sN + C;                               // [C] leader token of each state
  __shared__ float sk[2][DK], sv[2][DV];
  __shared__ float red[16];
  __shared__ double sDecI;
  __shared__ int sDec[2];
  __shared__ double sArg[4];
  __shared__ int sArgI[4];

  Meta M = meta_at(a.cache + a.meta_offset + (size_t)h * a.meta_stride, C);
  InitView iv = init_at(w, h, C);
  const int m0 = min(max(*M.m, 0), C);
  int m = m0;
  for (int j = tid; j < C; j += 256) {
    sI[j] = M.ibar[j];
    sN[j] = M.n[j];
    sLead[j] = j - m0;
  }

  const float* states = reinterpret_cast<const float*>(a.cache + a.states_offset) +
                        (size_t)h * C * D;
  float4 S[ST::NV];
  double Fo = 0.0;
  if (m0 > 0) {
    const float4* src =
        reinterpret_cast<const float4*>(states + (size_t)min(max(M.perm[m0 - 1], 0), C - 1) * D);
#pragma unroll
    for (int r = 0; r < ST::NV; ++r) S[r] = src[tid + 256 * r];
    Fo = M.F[m0 - 1];
  } else {
#pragma unroll
    for (int r = 0; r < ST::NV; ++r) S[r] = make_float4(0.f, 0.f, 0.f, 0.f);
  }

  const Tin* kin = static_cast<const Tin*>(a.k) + (size_t)h * T * DK;
  const Tin* vin = static_cast<const Tin*>(a.v) + (size_t)h * T * DV;
  const double* Gt = w.Gtok + (size_t)h * T;
  int32_t* death = w.death + (size_t)h * T;
  const size_t tok0 = (size_t)h * T;

  // token 0 into LDS
  if (tid < DK) sk[0][tid] = to_f32(kin[tid]);
  if (tid >= 128 && tid - 128 < DV) sv[0][tid - 128] = to_f32(vin[tid - 128]);

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    // prefetch the next token
    float pk = 0.f, pv = 0.f;
    if (t + 1 < T) {
      if (tid < DK) pk = to_f32(kin[(size_t)(t + 1) * DK + tid]);
      if (tid >= 128 && tid - 128 < DV) pv = to_f32(vin[(size_t)(t + 1) * DV + tid - 128]);
    }
    const double G = Gt[t];
    __syncthreads();

    const float4 v4 = reinterpret_cast<const float4*>(sv[buf])[cq];
    float ct = 0.f, bt = 0.f;
#pragma unroll
    for (int r = 0; r < ST::NV; ++r) {
      const float kr = sk[buf][rg + ST::RG * r];
      const float4 s = S[r];
      ct += kr * (s.x * v4.x + s.y * v4.y + s.z * v4.z + s.w * v4.w);
      bt += s.x * s.x + s.y * s.y + s.z * s.z + s.w * s.w;
    }
    float kk = 0.f, vv = 0.f;
    if (tid < DK) kk = sk[buf][tid] * sk[buf][tid];
    if (tid < DV) vv = sv[buf][tid] * sv[buf][tid];
    ct = wave_sum(ct);
    bt = wave_sum(bt);
    kk = wave_sum(kk);
    vv = wave_sum(vv);
    if ((tid & 63) == 0) {
      red[(tid >> 6)] = ct;
      red[4 + (tid >> 6)] = bt;
      red[8 + (tid >> 6)] = kk;
      red[12 + (tid >> 6)] = vv;
    }
    __syncthreads();
    if (tid == 0) {
      double I = 0.0;
      int b = 1;
      if (m > 0) {
        const float c = (red[0] + red[1]) + (red[2] + red[3]);
        const float bb = (red[4] + red[5]) + (red[6] + red[7]);
        const float k2 = (red[8] + red[9]) + (red[10] + red[11]);
        const float v2 = (red[12] + red[13]) + (red[14] + red[15]);
        const double f = exp(G - Fo);
        I = info_score((double)k2 * (double)v2, f * f * (double)bb, f * (double)c, (double)D,
                       a.eps, a.eps_rms);
        b = (I >= (double)a.tau) ? 1 : 0;
        if (a.b_ovr && a.b_ovr[tok0 + t] != -1) b = a.b_ovr[tok0 + t] ? 1 : 0;
        if (C == 1) b = 0;
      }
      sDecI = I;
      sDec[0] = b;
    }
    __syncthreads();
    const int b = sDec[0];
    const double I = sDecI;

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
        for (int q = 1; q < 4; ++q)
          if (sArg[q] < bb || (sArg[q] == bb && sArgI[q] < ii)) {
            bb = sArg[q];
            ii = sArgI[q];
          }
        if (a.m_ovr && a.m_ovr[tok0 + t] != -1) {
          const int f = a.m_ovr[tok0 + t];
          if (f >= 0 && f <= C - 2)
            ii = f;
          else
            atomicOr(&reinterpret_cast<CacheHeader*>(a.cache)->flags,
                     DLA_FLAG_BAD_MERGE_OVERRIDE);
        }
        sDec[1] = ii;
        // the state right of the pair dies at token t
        const int lead = sLead[ii + 1];
        if (lead >= 0)
          death[lead] = t;
        else
          iv.death0[lead + m0] = t;
      }
      __syncthreads();
      istar = sDec[1];
      // merge istar and istar+1, shift the later states down (C <= 1024: at most
      // 4 entries per thread, all read before any is written)
      double nI[4];
      int nN[4], nL[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = tid + 256 * u;
        if (j >= istar && j + 1 < m) {
          nI[u] = (j == istar) ? sI[j] + sI[j + 1] : sI[j + 1];
          nN[u] = (j == istar) ? sN[j] + sN[j + 1] : sN[j + 1];
          nL[u] = (j == istar) ? sLead[j] : sLead[j + 1];
        }
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = tid + 256 * u;
        if (j >= istar && j + 1 < m) {
          sI[j] = nI[u];
          sN[j] = nN[u];
          sLead[j] = nL[u];
        }
      }
      __syncthreads();
      m -= 1;
    }

    const float4 vq = v4;
    if (!b) {
      const float f = (float)exp(G - Fo);
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) {
        const float kr = sk[buf][rg + ST::RG * r];
        S[r].x = f * S[r].x + kr * vq.x;
        S[r].y = f * S[r].y + kr * vq.y;
        S[r].z = f * S[r].z + kr * vq.z;
        S[r].w = f * S[r].w + kr * vq.w;
      }
      if (tid == 0) {
        sN[m - 1] += 1;
        sI[m - 1] += I;
        death[t] = -1;
      }
    } else {
#pragma unroll
      for (int r = 0; r < ST::NV; ++r) {
        const float kr = sk[buf][rg + ST::RG * r];
        S[r] = make_float4(kr * vq.x, kr * vq.y, kr * vq.z, kr * vq.w);
      }
      if (tid == 0) {
        sN[m] = 1;
        sI[m] = I;
        sLead[m] = t;
        death[t] = T;
      }
      m += 1;
    }
    Fo = G;
    if (tid == 0) {
      if (a.b_out) a.b_out[tok0 + t] = (int8_t)b;
      if (a.merge_out) a.merge_out[tok0 + t] = istar;
      if (a.score_out) a.score_out[tok0 + t] = (float)I;
    }
    // next token into the other buffer
    if (t + 1 < T) {
      if (tid < DK) sk[buf ^ 1][tid] = pk;
      if (tid >= 128 && tid - 128 < DV) sv[buf ^ 1][tid - 128] = pv;
    }
  }
  __syncthreads();
  for (int j = tid; j < m; j += 256) {
    M.n[j] = sN[j];
    M.ibar[j] = sI[j];
  }
}

template <int DK, int DV>
static void launch_scan_dims(const PrefillArgs& a, const PrefillWS& w, int nh, hipStream_t s) {
  const size_t shm = (size_t)a.desc.C * (8 + 4 + 4);
  if (a.in_dtype == DLA_F32)
    hipLaunchKernelGGL((prefill_scan_kernel<DK, DV, float>), dim3(nh), dim3(256), shm, s, a, w);
  else
    hipLaunchKernelGGL((prefill_scan_kernel<DK, DV, bf16_t>), dim3(nh), dim3(256), shm, s, a, w);
}

hipError_t launch_prefill_scan(const PrefillArgs& a, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C);
  const int dk = a.desc.d_k, dv = a.desc.d_v;
  if (dk == 128 && dv == 128)
    launch_scan_dims<128, 128>(a, w, nh, s);
  else if (dk == 64 && dv == 64)
    launch_scan_dims<64, 64>(a, w, nh, s);
  else if (dk == 128 && dv == 64)
    launch_scan_dims<128, 64>(a, w, nh, s);
  else
    launch_scan_dims<64, 128>(a, w, nh, s);
  return hipGetLastError();
}

}  // namespace dla
