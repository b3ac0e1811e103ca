// Prefill, stages 1 and 2: token frame preparation, and the sequential
// boundary scan with the capacity schedule (Alg. 1 and Alg. 2, Sec. 3.1-3.2).
//
// Stage 1 (prep, one workgroup per head): the cumulative log-decay of every
// token in float64, and a copy of the cache's per-head metadata as it was
// before the call (later stages overwrite the cache).
//
// Stage 2 (scan, one 8-wave workgroup per head, sequential over chunks of 64
// tokens).
// The decisions are sequential -- whether token t opens a state depends on the
// newest state, which depends on every earlier decision -- but within a chunk
// the score of token t against a newest state that started at position p has a
// closed form in a few chunk-wide tables, so each chunk costs a handful of
// dense MFMA products plus a short pointer chase:
//   * P[s][t] = (k_s . k_t)(v_s . v_t)  (Gram products, MFMA), a_t = P[t][t];
//   * c0[t] = k_t^T S_0 v_t against the newest state S_0 at the chunk start
//     (MFMA with S_0 split into three bf16 terms, exact to float32 rounding);
//   * R[p][t] = sum_{s=p}^{t-1} exp(G_t - G_s) P[t][s], so that k_t^T S v_t for
//     the state S of tokens p..t-1 is R[p][t] (plus the decayed c0 term when
//     the state began before the chunk);
//   * |S|^2 follows the recurrence b <- alpha^2 (b + 2c + a), evaluated for
//     all t at once as a wavefront scan of affine maps.
// The score (rank-one closed form of the RMS-normalised distance, Sec. 3.1)
// and the boundary test then hold for every token of a row at once; a ballot
// finds the first boundary, which starts the next row.  Each boundary runs the
// capacity schedule of Alg. 2 on the (count, score) pairs in LDS.  At the
// chunk end the newest state (float32 MFMA accumulators, 32 x 32 tiles spread
// over the waves) is advanced by the chunk's tokens.  Emits b_t, merge index and
// score per token, and the death token of every state leader (the token at
// which Alg. 2 merged that state into its left neighbour), from which the
// readout stage reconstructs the chronological index of every state at every
// token without a replay.
#include <type_traits>

#include "mfma.h"
#include "prefill.h"

namespace dla {

// ---------------------------------------------------------------------------
// stage 1
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void prefill_prep_kernel(PrefillArgs a, PrefillWS w) {
  if (!cache_matches(a.cache, a.desc)) {  // refused: the descriptor is not the cache's
    flag_mismatch(a.cache);
    return;
  }
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
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C, a.desc.d_k * a.desc.d_v,
                          seg_plan(a.desc, a.T, a.in_dtype, !a.skip_readout, a.serial != 0, a.pool_budget).nch);
  hipLaunchKernelGGL(prefill_prep_kernel, dim3(nh), dim3(256), 0, s, a, w);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// stage 2
// ---------------------------------------------------------------------------
constexpr int SL = 64;  // tokens per scan chunk (one per lane of a wavefront)
constexpr int SWAVE = 8;  // waves per scan workgroup
constexpr int STHR = 64 * SWAVE;

typedef u32x4 u32x4s;

template <int DK, int DV, typename Tin>
struct ScanP {
  static constexpr int E = (int)sizeof(Tin);
  static constexpr int EPP = 16 / E;                // elements per 16 bytes
  static constexpr int K16 = SL * DK * E / 16 / STHR;  // 16-byte K pieces per thread
  static constexpr int V16 = SL * DV * E / 16 / STHR;
  // LDS row strides (elements), padded by 16 bytes so that lanes reading
  // consecutive rows hit distinct banks
  static constexpr int KRS = DK + EPP;  // sK  [SL][KRS]
  static constexpr int VRS = DV + EPP;  // sV  [SL][VRS]
  static constexpr int TRS = SL + EPP;  // sKt [DK][TRS], sVt [DV][TRS] (transposed)
  // transposed copies for 16-bit inputs; float32 inputs (twice the bytes) read
  // the row-major copies element by element instead, to stay within LDS
  static constexpr bool TRANS = E == 2;
  static constexpr int NTERM = E == 2 ? 3 : 1;  // bf16 terms that carry a float32 value
  // sK, sV, sP and sVV are contiguous and dead once the tables are built; for
  // 16-bit inputs the decayed keys of the state advance (NTERM x [DK][TRS])
  // reuse their bytes (float32 inputs form them in the advance instead)
  static constexpr size_t DEAD_BYTES = (size_t)SL * (KRS + VRS) * E + 2 * (size_t)SL * (SL + 1) * 4;
  static_assert((size_t)NTERM * DK * TRS * E <= DEAD_BYTES, "decayed keys");
  static size_t smem_bytes(int C) {
    size_t off = DEAD_BYTES;                            // sK, sV, sP, sVV
    off += TRANS ? (size_t)(DK + DV) * TRS * E : 0;     // sKt, sVt
    off += (size_t)SL * (SL + 1) * 4;                   // sR
    off += (size_t)SWAVE * SL * 4;                      // sPart
    off += (size_t)SL * 4 * 8;                          // float rows
    off += (size_t)SL * 4 * 3 + SL * 2;                 // int rows, int8 rows
    off = round_up(off, 8);
    off += (size_t)C * (8 + 4 + 4) + 64;
    return round_up(off, 16);
  }
};

template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(STHR) void prefill_scan_kernel(PrefillArgs a, PrefillWS w, int tb,
                                                            int te) {
  if (!cache_matches(a.cache, a.desc)) return;  // refused call (see the prep kernel)
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using P = ScanP<DK, DV, Tin>;
  constexpr int D = DK * DV;
  constexpr int NB = DK / 32;  // 32-row bands of d_k
  constexpr int NJ = DV / 32;  // 32-column tiles of d_v
  // state tiles (band b, column tile j), tile i = b + NB j: wave w holds tiles
  // w, w + SWAVE, ... (all in band w % NB)
  constexpr int NTILE = NB * NJ;
  constexpr int NTW = (NTILE + SWAVE - 1) / SWAVE;
  constexpr int KSK = DK / 16, KSV = DV / 16;
  constexpr int K16 = P::K16, V16 = P::V16;
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int C = a.desc.C;
  const int T = a.T;
  const size_t tok0 = (size_t)h * T;
  const float Df = (float)D;

  extern __shared__ __align__(16) char smem[];
  constexpr int KRS = P::KRS, VRS = P::VRS;
  Tin* sK = reinterpret_cast<Tin*>(smem);  // keys of the chunk, row-major
  Tin* sV = sK + SL * KRS;                 // values, row-major
  float* sP = reinterpret_cast<float*>(sV + SL * VRS);  // [SL][SL+1], (K K^T) tiles
  float* sVV = sP + SL * (SL + 1);                      // [SL][SL+1], (V V^T) tiles
  Tin* sKd = reinterpret_cast<Tin*>(smem);  // [NTERM][DK][TRS] decayed keys (alias)
  Tin* sKt = reinterpret_cast<Tin*>(smem + P::DEAD_BYTES);  // keys, transposed [DK][TRS]
  Tin* sVt = sKt + DK * P::TRS;            // values, transposed [DV][TRS]
  float* sR = reinterpret_cast<float*>(P::TRANS ? sVt + DV * P::TRS : sKt);  // [SL][SL+1], R[p][t] at [t][p]
  float* sPart = sR + SL * (SL + 1);                    // [SWAVE][SL]
  float* sGc = sPart + SWAVE * SL;  // G_t - G(chunk start), float
  float* sA = sGc + SL;        // exp(sGc[t])
  float* sAl2 = sA + SL;       // alpha_t^2
  float* sDe = sAl2 + SL;      // exp(G_end - G_t)
  float* sa = sDe + SL;        // |k_t|^2 |v_t|^2
  float* sc0 = sa + SL;        // k_t^T S_0 v_t
  float* sIo = sc0 + SL;       // scores
  float* sRed = sIo + SL;      // reductions (8 floats used)
  int32_t* sMo = reinterpret_cast<int32_t*>(sRed + SL);  // merge overrides
  int32_t* sMout = sMo + SL;                             // merge indices
  int32_t* sDC = sMout + SL;                             // death tokens of the chunk's tokens
  int8_t* sBo = reinterpret_cast<int8_t*>(sDC + SL);     // boundary overrides
  int8_t* sBout = sBo + SL;                              // boundaries
  char* q8 = reinterpret_cast<char*>(sBout + SL);
  double* sIb = reinterpret_cast<double*>(smem + round_up((size_t)(q8 - smem), 8));  // [C]
  int32_t* sN = reinterpret_cast<int32_t*>(sIb + C);  // [C]
  int32_t* sLead = sN + C;                            // [C]
  int32_t* sMisc = sLead + C;                         // m, p_last
  __shared__ double sGlast[1];

  Meta M = meta_at(a.cache + a.meta_offset + (size_t)h * a.meta_stride, C);
  InitView iv = init_at(w, h, C);
  ScarryView sv = scarry_at(w, h, C);
  // states present before the call (copied from the cache by stage 1)
  const int m0 = *iv.m0;
  if (tb == 0) {
    for (int j = tid; j < C; j += STHR) {
      sIb[j] = M.ibar[j];
      sN[j] = M.n[j];
      sLead[j] = j - m0;
    }
    if (tid == 0) sMisc[0] = m0;
  } else {
    // resume where the previous segment stopped
    for (int j = tid; j < C; j += STHR) {
      sIb[j] = sv.ibar[j];
      sN[j] = sv.n[j];
      sLead[j] = sv.lead[j];
    }
    if (tid == 0) sMisc[0] = *sv.m;
  }

  // newest state at the start of the call, true (decayed) values, as MFMA
  // accumulators: S[k] is the wave's tile wv + SWAVE k (rows 32 band.. of d_k,
  // columns 32 tj(k)..)
  const int band = wv % NB;
  auto tj = [&](int k) { return (wv + SWAVE * k) / NB; };
  auto tok = [&](int k) { return wv + SWAVE * k < NTILE; };
  f32x16 S[NTW];
#pragma unroll
  for (int k = 0; k < NTW; ++k) S[k] = zero16();
  const double G0 = *M.G;
  if (tb > 0) {
#pragma unroll
    for (int k = 0; k < NTW; ++k)
      if (tok(k)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) S[k][r] = sv.S[((size_t)(wv + SWAVE * k) * 16 + r) * 64 + lane];
      }
  } else if (m0 > 0) {
    // the newest state: its float32 slot, or the open region with bfloat16 storage
    const float* src =
        a.desc.state_dtype == DLA_BF16
            ? reinterpret_cast<const float*>(a.cache + a.open_offset) + (size_t)h * D
            : reinterpret_cast<const float*>(a.cache + a.states_offset) +
                  ((size_t)h * C + min(max(M.perm[m0 - 1], 0), C - 1)) * D;
    const float f = (float)exp(G0 - M.F[m0 - 1]);
#pragma unroll
    for (int k = 0; k < NTW; ++k)
      if (tok(k)) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          S[k][r] = f * src[(size_t)(32 * band + out_row(r, lane)) * DV + 32 * tj(k) + l32];
      }
  }
  auto state_norm2 = [&]() -> float {  // |S|^2 over the block
    float x = 0.f;
#pragma unroll
    for (int k = 0; k < NTW; ++k)
      if (tok(k)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) x += S[k][r] * S[k][r];
      }
    x = wave_sum(x);
    // one barrier: between one call's reads of sRed and the next call's writes
    // lie the barriers of a whole chunk
    if (lane == 0) sRed[wv] = x;
    __syncthreads();
    float b = 0.f;
#pragma unroll
    for (int i = 0; i < SWAVE; ++i) b += sRed[i];
    return b;
  };
  float b0 = state_norm2();

  const Tin* Kin = static_cast<const Tin*>(a.k) + tok0 * DK;
  const Tin* Vin = static_cast<const Tin*>(a.v) + tok0 * DV;
  const double* Gtok = w.Gtok + tok0;
  int32_t* death = w.death + tok0;
  constexpr int KROW16 = DK * (int)sizeof(Tin) / 16;  // 16-byte pieces per key row
  constexpr int VROW16 = DV * (int)sizeof(Tin) / 16;
  // Next-chunk registers: lane tid % SL holds token row tid % SL, pieces
  // tid / SL + SWAVE u of its key and value rows (so the transposed copies are
  // written with consecutive lanes on consecutive tokens), and threads tid < SL
  // hold the token's cumulative log-decay and overrides.
  u32x4s pk[K16], pv[V16];
  double gpre = 0.0;
  int bpre = -1, mpre = -1;
  auto prefetch = [&](int c0n) __attribute__((always_inline)) {
    const int nr = min(SL, T - c0n);
#pragma unroll
    for (int u = 0; u < K16; ++u) {
      const int pi = tid + STHR * u;
      const int r = min(pi % SL, nr - 1);
      pk[u] = reinterpret_cast<const u32x4s*>(Kin + (size_t)(c0n + r) * DK)[pi / SL];
    }
#pragma unroll
    for (int u = 0; u < V16; ++u) {
      const int pi = tid + STHR * u;
      const int r = min(pi % SL, nr - 1);
      pv[u] = reinterpret_cast<const u32x4s*>(Vin + (size_t)(c0n + r) * DV)[pi / SL];
    }
    if (tid < SL) {
      const int t = min(tid, nr - 1);
      gpre = Gtok[c0n + t];
      bpre = (a.b_ovr && tid < nr) ? a.b_ovr[tok0 + c0n + tid] : (int8_t)-1;
      mpre = (a.m_ovr && tid < nr) ? a.m_ovr[tok0 + c0n + tid] : -1;
    }
  };
  prefetch(tb);
  double Gprev = tb > 0 ? Gtok[tb - 1] : G0;
  const float tau = a.tau;

  for (int c0 = tb; c0 < te; c0 += SL) {
    const int nrow = min(SL, T - c0);
    // ------------------------------------------------ stage the chunk
    // transposed copy of a 16-bit piece (8 columns of token r, r = lane): the
    // lane pair (2i, 2i + 1) swaps halves, so each lane writes 32-bit words
    // holding both tokens of the pair, 4 columns each
    auto put_t = [&](Tin* dst, int pc, int r, const u32x4s& val) __attribute__((always_inline)) {
      const bool odd = (r & 1) != 0;
      const uint32_t s0 = odd ? val[0] : val[2], s1 = odd ? val[1] : val[3];
      const uint32_t r0 = (uint32_t)__builtin_amdgcn_mov_dpp((int)s0, 0xB1, 0xF, 0xF, false);
      const uint32_t r1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)s1, 0xB1, 0xF, 0xF, false);
      // even lane: columns 0..3, own token first; odd lane: columns 4..7, the
      // partner's token (r - 1) first
      const uint32_t m0 = odd ? val[2] : val[0], m1 = odd ? val[3] : val[1];
      const uint32_t lo0 = odd ? r0 : m0, hi0 = odd ? m0 : r0;
      const uint32_t lo1 = odd ? r1 : m1, hi1 = odd ? m1 : r1;
      uint32_t* row = reinterpret_cast<uint32_t*>(dst + (pc * P::EPP + (odd ? 4 : 0)) * P::TRS + (r & ~1));
      row[0] = __builtin_amdgcn_perm(hi0, lo0, 0x05040100u);
      row[P::TRS / 2] = __builtin_amdgcn_perm(hi0, lo0, 0x07060302u);
      row[P::TRS] = __builtin_amdgcn_perm(hi1, lo1, 0x05040100u);
      row[3 * (P::TRS / 2)] = __builtin_amdgcn_perm(hi1, lo1, 0x07060302u);
    };
#pragma unroll
    for (int u = 0; u < K16; ++u) {
      const int pi = tid + STHR * u;
      const int r = pi % SL, pc = pi / SL;
      const u32x4s z = {0u, 0u, 0u, 0u};
      const u32x4s val = (r < nrow) ? pk[u] : z;
      *reinterpret_cast<u32x4s*>(sK + r * KRS + pc * P::EPP) = val;
      if constexpr (P::TRANS) put_t(sKt, pc, r, val);
    }
#pragma unroll
    for (int u = 0; u < V16; ++u) {
      const int pi = tid + STHR * u;
      const int r = pi % SL, pc = pi / SL;
      const u32x4s z = {0u, 0u, 0u, 0u};
      const u32x4s val = (r < nrow) ? pv[u] : z;
      *reinterpret_cast<u32x4s*>(sV + r * VRS + pc * P::EPP) = val;
      if constexpr (P::TRANS) put_t(sVt, pc, r, val);
    }
    if (tid < SL) {
      // log-decay offsets from the chunk start; the last token's G is the
      // next chunk's start
      const int t = tid;
      const double Gt = gpre;
      const double Glast = __shfl(gpre, nrow - 1, 64);
      const float gc = (float)(Gt - Gprev);
      const float gcp = __shfl_up(gc, 1, 64);  // token t - 1 (t >= 1)
      sGc[t] = gc;
      sA[t] = __expf(gc);
      // alpha_t^2 = exp(2 g_t); only tokens of the chunk read their predecessor
      sAl2[t] = (t < nrow) ? __expf(2.f * (t == 0 ? gc : gc - gcp)) : 0.f;
      sDe[t] = (t < nrow) ? __expf((float)(Glast - Gt)) : 0.f;
      sBo[t] = (int8_t)bpre;
      sMo[t] = mpre;
      sDC[t] = -1;
      sBout[t] = 0;
      sMout[t] = -1;
      sIo[t] = 0.f;
      if (t == 0) sGlast[0] = Glast;
    }
    __syncthreads();
    const double Gnext = sGlast[0];  // G after the chunk's last token
    if (c0 + SL < te) prefetch(c0 + SL);

    // ------------------------------------------------ Gram products and the carry term
    {
      // tile (tr, tc) of K K^T (waves 0..3, into sP) or of V V^T (waves 4..7,
      // into sVV); the product P = (K K^T) (.) (V V^T) is formed where it is read
      const int tq = wv & 3;
      const int tr = tq >> 1, tcl = tq & 1;
      f32x16 g = zero16();
      if (wv < 4) {
        const Tin* ka = sK + (32 * tr + l32) * KRS;
        const Tin* kb = sK + (32 * tcl + l32) * KRS;
#pragma unroll
        for (int ks = 0; ks < KSK; ++ks)
          FR::mma(g, FR::load(ka + 16 * ks + 8 * half), FR::load(kb + 16 * ks + 8 * half));
      } else {
        const Tin* va = sV + (32 * tr + l32) * VRS;
        const Tin* vb = sV + (32 * tcl + l32) * VRS;
#pragma unroll
        for (int ks = 0; ks < KSV; ++ks)
          FR::mma(g, FR::load(va + 16 * ks + 8 * half), FR::load(vb + 16 * ks + 8 * half));
      }
      float* dst = wv < 4 ? sP : sVV;
#pragma unroll
      for (int r = 0; r < 16; ++r) dst[(32 * tr + out_row(r, lane)) * (SL + 1) + 32 * tcl + l32] = g[r];
    }
    {
      // partial over this wave's state tiles: sum_i sum_j k_t[i] S0[i][j] v_t[j]
      float part[2] = {0.f, 0.f};
#pragma unroll
      for (int k = 0; k < NTW; ++k) {
        if (!tok(k)) continue;
        const int nj = tj(k);
        // A = S0^T (rows j, K = i) straight from the accumulator layout, in three
        // bf16 terms; B = K^T with the matching permutation of i
        FT ah[2], am[2], al[2];
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          float x[8], r1[8], r2[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = S[k][8 * st + e];
          ah[st] = FR::from_floats(x);
          if constexpr (sizeof(Tin) == 2) {
#pragma unroll
            for (int e = 0; e < 8; ++e) r1[e] = x[e] - (float)ah[st][e];
            am[st] = FR::from_floats(r1);
#pragma unroll
            for (int e = 0; e < 8; ++e) r2[e] = r1[e] - (float)am[st][e];
            al[st] = FR::from_floats(r2);
          }
        }
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) {
          f32x16 y = zero16();
          const Tin* krow = sK + (32 * tn + l32) * KRS + 32 * band + 4 * half;
#pragma unroll
          for (int st = 0; st < 2; ++st) {
            // k index 16 st + 8 (e / 4) + 4 h + e % 4 of the band, as in the
            // accumulator layout of S0
            const FT kb = load_4x2<Tin>(krow + 16 * st, krow + 16 * st + 8);
            if constexpr (sizeof(Tin) == 2) {
              FR::mma(y, al[st], kb);
              FR::mma(y, am[st], kb);
            }
            FR::mma(y, ah[st], kb);
          }
          // v_t[j] for the rows j = 8 q + 4 h + (0..3) of the tile held by the lane
          const Tin* vrow = sV + (32 * tn + l32) * VRS + 32 * nj + 4 * half;
          float sacc = 0.f;
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            float vx[4];
            load4f(vrow + 8 * q4, vx);
#pragma unroll
            for (int e = 0; e < 4; ++e) sacc += y[4 * q4 + e] * vx[e];
          }
          part[tn] += sacc;
        }
      }
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        const float tot = part[tn] + __shfl_xor(part[tn], 32, 64);
        if (half == 0) sPart[wv * SL + 32 * tn + l32] = tot;
      }
    }
    __syncthreads();

    // ------------------------------------------------ tables: a_t, c0[t], R[p][t]
    if (tid < SL) {
      float c = 0.f;
#pragma unroll
      for (int b = 0; b < SWAVE; ++b) c += sPart[b * SL + tid];
      sc0[tid] = c;
      sa[tid] = sP[tid * (SL + 1) + tid] * sVV[tid * (SL + 1) + tid];
    }
    {
      // row t of R: lane l holds s = SL - 1 - l, so the suffix sum over s is a
      // prefix sum over the lanes (DPP ladder); wave q takes rows t = q, q +
      // SWAVE, ...  R[p][t] is stored at sR[t (SL + 1) + p].
      const int s = SL - 1 - lane;
      const float gs = sGc[s];
#pragma unroll
      for (int t = wv; t < SL; t += SWAVE) {
        float x = (s < t) ? __expf(sGc[t] - gs) * (sP[t * (SL + 1) + s] * sVV[t * (SL + 1) + s]) : 0.f;
        x += dpp_f<0x111, 0xF>(0.f, x);
        x += dpp_f<0x112, 0xF>(0.f, x);
        x += dpp_f<0x114, 0xF>(0.f, x);
        x += dpp_f<0x118, 0xF>(0.f, x);
        x += dpp_f<0x142, 0xA>(0.f, x);
        x += dpp_f<0x143, 0xC>(0.f, x);
        sR[t * (SL + 1) + s] = x;
      }
    }
    __syncthreads();

    // ------------------------------------------------ decisions (wave 0)
    // Meanwhile the waves on the other SIMDs (wave 4 shares wave 0's) stage the
    // chunk's decayed keys exp(G_end - G_s) k_s for the state advance, split
    // into NTERM terms of the input type, transposed: item (i, g) covers row i of
    // d_k and tokens 8 g .. 8 g + 7 (zero past the chunk end, where sDe = 0).
    if (P::TRANS && wv != 0 && wv != 4) {
      constexpr int NITEM = DK * (SL / 8);
      const int hw = wv < 4 ? wv - 1 : wv - 2;  // 0 .. 5
      for (int it = hw * 64 + lane; it < NITEM; it += 6 * 64) {
        const int i = it / (SL / 8), g = it % (SL / 8);
        const FT kraw = FR::load(sKt + i * P::TRS + 8 * g);
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = sDe[8 * g + e] * (float)kraw[e];
        Tin* dst = sKd + i * P::TRS + 8 * g;
        const FT khi = FR::from_floats(x);
        *reinterpret_cast<FT*>(dst) = khi;
        if constexpr (sizeof(Tin) == 2) {
          float r1[8], r2[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) r1[e] = x[e] - (float)khi[e];
          const FT kmi = FR::from_floats(r1);
#pragma unroll
          for (int e = 0; e < 8; ++e) r2[e] = r1[e] - (float)kmi[e];
          *reinterpret_cast<FT*>(dst + DK * P::TRS) = kmi;
          *reinterpret_cast<FT*>(dst + 2 * DK * P::TRS) = FR::from_floats(r2);
        }
      }
    }
    if (wv == 0) {
      const int t = lane;
      const float at = sa[t];
      const float c0t = sc0[t];
      const float At = sA[t];
      const float al2n = (t + 1 < SL) ? sAl2[t + 1] : 0.f;  // alpha^2 of token t+1
      int mcur = sMisc[0];
      int p = -1;  // start of the newest state: -1 = before the chunk
      int plast = -1;
      if (mcur == 0) {
        // the first token of an empty cache opens a state with score 0
        if (lane == 0) {
          sBout[0] = 1;
          sIo[0] = 0.f;
          sMout[0] = -1;
          sN[0] = 1;
          sIb[0] = 0.0;
          sLead[0] = c0;
          sDC[0] = T;
        }
        mcur = 1;
        p = 0;
        plast = 0;
      }
      while (true) {
        const int first = p + 1;  // first token scored against this state
        float ct;
        if (p < 0)
          ct = At * c0t + sR[t * (SL + 1)];  // R[0][t]
        else
          ct = (t > p) ? sR[t * (SL + 1) + p] : 0.f;
        // |S|^2 before token t: b(t+1) = alpha_{t+1}^2 (b(t) + 2 c(t) + a_t), b(first) = binit
        const float binit = (p < 0) ? sA[0] * sA[0] * b0 : 0.f;
        const int ustart = (p < 0) ? 0 : p;
        float Am = 1.f, Bm = 0.f;
        if (t >= ustart) {
          Am = al2n;
          Bm = al2n * (2.f * ct + at);
        }
        // inclusive scan of the affine maps x -> Am x + Bm over lanes
        wave_scan_affine(Am, Bm);
        const float bnext = Am * binit + Bm;  // b(t+1)
        float bt = dpp_f<0x138, 0xF>(binit, bnext);  // lane t - 1
        if (t == ustart) bt = binit;
        if (p < 0 && t == 0) bt = binit;
        const bool valid = (t < nrow) && (t >= first);
        const float It = valid ? score_f(at, bt, ct, Df, a.eps, a.eps_rms) : 0.f;
        int bd = (It >= tau) ? 1 : 0;
        if (sBo[t] != -1) bd = sBo[t] ? 1 : 0;
        if (C == 1) bd = 0;
        const uint64_t mask = __ballot(valid && bd);
        const int tstar = mask ? (__ffsll((unsigned long long)mask) - 1) : nrow;
        // tokens first .. tstar-1 join the newest state
        const bool joins = valid && t < tstar;
        if (joins) sIo[t] = It;
        const double sI = wave_sum_d(joins ? (double)It : 0.0);
        if (lane == 0 && tstar > first) {
          sN[mcur - 1] += tstar - first;
          sIb[mcur - 1] += sI;
        }
        if (tstar >= nrow) break;
        // boundary at tstar: Alg. 2 when the cache is full, then a new state
        const float Istar = __shfl(It, tstar, 64);
        int istar = -1;
        if (mcur == C) {
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
          // NaN densities (scores from non-finite inputs) compare false, so a
          // sequential argmin that starts at pair 0 never moves to them, and
          // stays at pair 0 when pair 0's density is NaN or none is a number
          istar = (bi >= 0 && bi <= C - 2) ? bi : 0;
          if (__builtin_isnan((sIb[0] + sIb[1]) / (double)(sN[0] + sN[1]))) istar = 0;
          const int fo = sMo[tstar];
          if (fo != -1) {
            if (fo >= 0 && fo <= C - 2)
              istar = fo;
            else if (lane == 0)
              atomicOr(&reinterpret_cast<CacheHeader*>(a.cache)->flags, DLA_FLAG_BAD_MERGE_OVERRIDE);
          }
          // the state right of the pair dies at token c0 + tstar
          const int ld = sLead[istar + 1];
          if (lane == 0) {
            if (ld >= c0)
              sDC[ld - c0] = c0 + tstar;
            else if (ld >= 0)
              death[ld] = c0 + tstar;
            else
              iv.death0[ld + m0] = c0 + tstar;
          }
          // merge istar, istar+1 and shift the later states down, 64 entries at a
          // time in increasing order (a block's writes never touch entries that a
          // later block still has to read)
          for (int j0 = istar; j0 + 1 < mcur; j0 += 64) {
            const int j = j0 + lane;
            const bool act = j + 1 < mcur;
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
          mcur -= 1;
        }
        if (lane == 0) {
          sBout[tstar] = 1;
          sIo[tstar] = Istar;
          sMout[tstar] = istar;
          sN[mcur] = 1;
          sIb[mcur] = (double)Istar;
          sLead[mcur] = c0 + tstar;
          sDC[tstar] = T;
        }
        mcur += 1;
        p = tstar;
        plast = tstar;
      }
      if (lane == 0) {
        sMisc[0] = mcur;
        sMisc[1] = plast;
      }
    }
    __syncthreads();

    // ------------------------------------------------ advance the newest state
    const int plast = sMisc[1];
    {
      const float sc = (plast < 0) ? sA[nrow - 1] : 0.f;
#pragma unroll
      for (int k = 0; k < NTW; ++k)
#pragma unroll
        for (int r = 0; r < 16; ++r) S[k][r] *= sc;
      const int s0 = (plast < 0) ? 0 : plast;
#pragma unroll
      for (int st = 0; st < SL / 16; ++st) {
        if (16 * st + 15 < s0 || 16 * st >= nrow) continue;  // wave-uniform
        // element e of half h <-> token 16 st + 8 h + e; A = K~^T (rows of this
        // wave's band of d_k, the staged terms), B = V (32 columns per tile),
        // with the tokens before s0 masked out of V
        const int sb0 = 16 * st + 8 * half;
        FT ka[P::NTERM];
        if constexpr (P::TRANS) {
#pragma unroll
          for (int q = 0; q < P::NTERM; ++q) ka[q] = FR::load(sKd + (q * DK + 32 * band + l32) * P::TRS + sb0);
        } else {
          // float32: one term, formed here from the row-major keys
#pragma unroll
          for (int e = 0; e < 8; ++e) ka[0][e] = sDe[sb0 + e] * sK[(sb0 + e) * KRS + 32 * band + l32];
        }
        const bool part = 16 * st < s0;  // wave-uniform
        FT vb[NTW];
#pragma unroll
        for (int k = 0; k < NTW; ++k) {
          if constexpr (P::TRANS) {
            vb[k] = tok(k) ? FR::load(sVt + (32 * tj(k) + l32) * P::TRS + sb0) : FR::zero();
          } else {
            vb[k] = FR::zero();
            if (tok(k)) {
#pragma unroll
              for (int e = 0; e < 8; ++e) vb[k][e] = sV[(sb0 + e) * VRS + 32 * tj(k) + l32];
            }
          }
          if (part) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (sb0 + e < s0) vb[k][e] = FR::zero()[0];
          }
        }
        // smallest term first; each term runs over the column tiles before the
        // next, so no MFMA waits on its predecessor
#pragma unroll
        for (int q = P::NTERM - 1; q >= 0; --q)
#pragma unroll
          for (int k = 0; k < NTW; ++k)
            if (tok(k)) FR::mma(S[k], ka[q], vb[k]);
      }
    }
    b0 = state_norm2();  // (contains a barrier)
    if (tid < nrow) {
      const int t = tid;
      death[c0 + t] = sDC[t];
      if (a.b_out) a.b_out[tok0 + c0 + t] = sBout[t];
      if (a.merge_out) a.merge_out[tok0 + c0 + t] = sMout[t];
      if (a.score_out) a.score_out[tok0 + c0 + t] = sIo[t];
    }
    Gprev = Gnext;
  }
  __syncthreads();
  const int mfin = sMisc[0];
  if (te == T) {
    for (int j = tid; j < mfin; j += STHR) {
      M.n[j] = sN[j];
      M.ibar[j] = sIb[j];
    }
  } else {
    for (int j = tid; j < mfin; j += STHR) {
      sv.ibar[j] = sIb[j];
      sv.n[j] = sN[j];
      sv.lead[j] = sLead[j];
    }
    if (tid == 0) *sv.m = mfin;
#pragma unroll
    for (int k = 0; k < NTW; ++k)
      if (tok(k)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sv.S[((size_t)(wv + SWAVE * k) * 16 + r) * 64 + lane] = S[k][r];
      }
  }
}

// whether the scan's LDS working set fits for this shape
bool prefill_scan_supported(const dla_cache_desc& d, dla_dtype in_dtype) {
  auto fits = [&](auto dk_c, auto dv_c) {
    constexpr int DK = decltype(dk_c)::value, DV = decltype(dv_c)::value;
    const size_t b = in_dtype == DLA_F32 ? ScanP<DK, DV, float>::smem_bytes(d.C)
                                         : ScanP<DK, DV, bf16_t>::smem_bytes(d.C);
    return b <= 160 * 1024;
  };
  using I64 = std::integral_constant<int, 64>;
  using I128 = std::integral_constant<int, 128>;
  if (d.d_k == 128) return d.d_v == 128 ? fits(I128{}, I128{}) : fits(I128{}, I64{});
  return d.d_v == 128 ? fits(I64{}, I128{}) : fits(I64{}, I64{});
}

template <int DK, int DV>
static hipError_t launch_scan_dims(const PrefillArgs& a, const PrefillWS& w, int nh, int tb,
                                   int te, hipStream_t s) {
  if (a.in_dtype == DLA_F32) {
    auto k = prefill_scan_kernel<DK, DV, float>;
    const size_t shm = ScanP<DK, DV, float>::smem_bytes(a.desc.C);
    if (shm > 160 * 1024) return hipErrorInvalidValue;
    if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
        hipSuccess)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3(nh), dim3(STHR), shm, s, a, w, tb, te);
  } else {
    auto k = prefill_scan_kernel<DK, DV, bf16_t>;
    const size_t shm = ScanP<DK, DV, bf16_t>::smem_bytes(a.desc.C);
    if (shm > 160 * 1024) return hipErrorInvalidValue;
    if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
        hipSuccess)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3(nh), dim3(STHR), shm, s, a, w, tb, te);
  }
  return hipGetLastError();
}

hipError_t launch_prefill_scan(const PrefillArgs& a, int tb, int te, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  const int dk = a.desc.d_k, dv = a.desc.d_v;
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C, dk * dv,
                          seg_plan(a.desc, a.T, a.in_dtype, !a.skip_readout, a.serial != 0, a.pool_budget).nch);
  if (tb < 0 || te > a.T || tb >= te || tb % SL != 0) return hipErrorInvalidValue;
  if (dk == 128 && dv == 128) return launch_scan_dims<128, 128>(a, w, nh, tb, te, s);
  if (dk == 64 && dv == 64) return launch_scan_dims<64, 64>(a, w, nh, tb, te, s);
  if (dk == 128 && dv == 64) return launch_scan_dims<128, 64>(a, w, nh, tb, te, s);
  return launch_scan_dims<64, 128>(a, w, nh, tb, te, s);
}

}  // namespace dla
