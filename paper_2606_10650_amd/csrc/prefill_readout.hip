// Prefill, stage 3: multi-state readout and state-cache maintenance.
//
// Readout (eq. capacity_bounded_output): o_t = sum_j lambda[t][j] q_t^T S_j over
// the states of the cache after token t.  The decisions of stage 2 fix, for
// every token, which states exist; this stage turns them into dense MFMA work.
//
// One workgroup per (head, 32 value columns), sequential over chunks of
// 128 * NT tokens; wave w owns the 32-token tiles w, w + 4, ... of a chunk.
//   * inter-chunk part: every state S_j present at the chunk start contributes
//     lambda[t][x_j(t)] exp(G_t - F_j) q_t^T S~_j, x_j(t) being its chronological
//     index at token t: the number of live state leaders up to it, where a
//     leader lives while its death token (from stage 2) is later than t.  The
//     tile S~_j^T Q^T (32 columns x 32 tokens, K = d_k) is a bf16 MFMA chain;
//     each lane owns one token of the tile, so the weight is a per-lane scalar
//     applied to the tile's fresh accumulator.  States are streamed as a copy in
//     MFMA operand order (the shadow), 4 states ahead through registers and a
//     double-buffered LDS ring (one barrier per state).
//   * intra-chunk part: (Q K^T (.) M) V over the chunk's own tokens with
//     M[t][s] = [s <= t] exp(G_t - G_s) lambda[t][slot_t(s)]; slot_t(s) is
//     uniform over a 32-token block unless a live leader starts inside it, so
//     lambda is gathered once per (token, block) in the common case.
//   * state update: the states alive after the chunk are the surviving leaders.
//     A new or changed state is the decayed sum of the old states it absorbed
//     plus sum_s exp(G_end - G_s) k_s v_s^T over its tokens in the chunk, stored
//     in frame G_end (float32 master in the cache, plus its shadow).  The token
//     sum is an MFMA product K~^T V with K~ split into three bf16 terms, so it is
//     exact to float32 rounding.  Unchanged states are not touched (lazy decay).
#include "mfma.h"
#include "prefill.h"

namespace dla {

constexpr int NWAVE = 4;
constexpr int NC = 32;  // value columns per workgroup
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // 16 bytes, first-class

template <int DK, typename Tin, int NT>
struct RO {
  static constexpr int RL = 32 * NWAVE * NT;  // tokens per chunk
  static constexpr int KS = DK / 16;
  static constexpr int SLICE = DK * NC;                          // elements per (state, group)
  static constexpr int SLICE16 = SLICE * (int)sizeof(Tin) / 16;  // 16-byte pieces per slice
  static constexpr int V16 = SLICE16 / 256;                      // pieces per thread
  static_assert(SLICE16 % 256 == 0, "slice must split evenly over 256 threads");
  static size_t smem_bytes(int C) {
    size_t off = 2 * (size_t)SLICE16 * 16;            // ring
    off += (size_t)RL * NC * sizeof(Tin);             // sV
    off += (size_t)RL * (8 + 4 * 6);                  // sG sRf sBf sDecE sDeath sLeadU sLeadD
    off += (size_t)C * (8 + 4);                       // sF sSf
    off += (size_t)C * 4 * 11 + 64;                   // int arrays, reduction scratch
    return round_up(off, 16);
  }
};

// Exclusive prefix count over n <= 1024 flags in a block of 256 threads:
// out[i] = number of set flags before i.  Returns the total.  red: 4 ints.
template <typename F>
__device__ int block_excl_count(int n, F flag, int32_t* out, int32_t* red) {
  const int tid = threadIdx.x;
  int f[4];
  int local = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = 4 * tid + u;
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
  for (int u = 0; u < 4; ++u) {
    const int i = 4 * tid + u;
    if (i < n) out[i] = run;
    run += f[u];
  }
  const int total = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return total;
}

template <int DK, int DV, typename Tin, typename Tout, int NT>
__global__ __launch_bounds__(256) void prefill_readout_kernel(PrefillArgs a, PrefillWS w) {
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using P = RO<DK, Tin, NT>;
  constexpr int D = DK * DV;
  constexpr int NCG = DV / NC;
  constexpr int KS = P::KS;
  constexpr int RL = P::RL;
  constexpr int V16 = P::V16;
  constexpr int SLICE16 = P::SLICE16;
  const int nh = a.desc.B * a.desc.H;
  // XCD-aware mapping: workgroups are dealt to the 8 XCDs round-robin by id, so
  // the column groups of one head get the same id modulo 8 (one L2).
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
  u32x4* ring = reinterpret_cast<u32x4*>(smem);
  Tin* sV = reinterpret_cast<Tin*>(ring + 2 * SLICE16);
  double* sG = reinterpret_cast<double*>(sV + RL * NC);
  float* sRf = reinterpret_cast<float*>(sG + RL);  // exp(G_t - G_ref)
  float* sBf = sRf + RL;                            // exp(G_blockend - G_s)
  float* sDecE = sBf + RL;                          // exp(G_end - G_s)
  int32_t* sDeath = reinterpret_cast<int32_t*>(sDecE + RL);
  int32_t* sLeadU = sDeath + RL;  // in-chunk leaders: position in the chunk
  int32_t* sLeadD = sLeadU + RL;  //                   death token
  double* sF = reinterpret_cast<double*>(sLeadD + RL);
  float* sSf = reinterpret_cast<float*>(sF + C);  // exp(G_ref - F_j)
  int32_t* sPerm = reinterpret_cast<int32_t*>(sSf + C);
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
  int32_t* red = eChg + C;
  __shared__ int sCnt[4];
  __shared__ int sBlk[RL / 32 + 1];

  InitView iv = init_at(w, h, C);
  const int m0 = min(max(*iv.m0, 0), C);
  const double G0 = *iv.G0;
  int m = m0;
  for (int j = tid; j < C; j += 256) {
    sPerm[j] = min(max(iv.perm0[j], 0), C - 1);
    sF[j] = iv.F0[j];
    sLead[j] = j - m0;
  }

  float* states = reinterpret_cast<float*>(a.cache + a.states_offset) + (size_t)h * C * D;
  Tin* shadow = reinterpret_cast<Tin*>(w.shadow) + (size_t)h * C * D;
  const double* Gtok = w.Gtok + (size_t)h * T;
  const int32_t* death = w.death + (size_t)h * T;
  const Tin* Kin = static_cast<const Tin*>(a.k) + (size_t)h * T * DK;
  const Tin* Vin = static_cast<const Tin*>(a.v) + (size_t)h * T * DV;
  const Tin* Qin = static_cast<const Tin*>(a.q) + (size_t)h * T * DK;
  const Tin* Lin = a.lam ? static_cast<const Tin*>(a.lam) + (size_t)h * T * C : nullptr;
  Tout* Out = a.out ? static_cast<Tout*>(a.out) + (size_t)h * T * DV : nullptr;
  // shadow slice of (physical slot, this group): element (k, c) at
  // ((k / 16) * 2 + (k % 16) / 8) * 256 + c * 8 + k % 8
  auto slice_of = [&](int phys) -> Tin* { return shadow + ((size_t)phys * NCG + cg) * P::SLICE; };

  // shadows of the states present before the call
  __syncthreads();
  for (int j = 0; j < m; ++j) {
    const float* src = states + (size_t)sPerm[j] * D + cg * NC;
    Tin* dst = slice_of(sPerm[j]);
    const int c = tid & 31;
    for (int kg = tid >> 5; kg < DK / 8; kg += 8) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = src[(size_t)(8 * kg + e) * DV + c];
      Tin* d8 = dst + kg * 256 + c * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) d8[e] = from_f32<Tin>(x[e]);
    }
  }

  for (int c0 = 0; c0 < T; c0 += RL) {
    const int nrow = min(RL, T - c0);
    const int c1 = c0 + nrow;
    const double Gref = (c0 == 0) ? G0 : Gtok[c0 - 1];
    const double Gend = Gtok[c1 - 1];
    __syncthreads();
    for (int i = tid; i < RL; i += 256) {
      const int ic = min(i, nrow - 1);
      const double Gi = Gtok[c0 + ic];
      const int be = min(32 * (i >> 5) + 31, nrow - 1);
      sG[i] = Gi;
      sRf[i] = __expf((float)(Gi - Gref));
      sBf[i] = __expf((float)(Gtok[c0 + be] - Gi));
      sDecE[i] = (i < nrow) ? __expf((float)(Gend - Gi)) : 0.f;
      sDeath[i] = (i < nrow) ? death[c0 + i] : -1;
    }
    for (int j = tid; j < m; j += 256) {
      const int ld = sLead[j];
      sDt[j] = (ld >= 0) ? death[ld] : iv.death0[ld + m0];
      sSf[j] = __expf((float)(Gref - sF[j]));
    }
    // this group's value columns of the chunk
    {
      constexpr int PER_ROW16 = NC * (int)sizeof(Tin) / 16;
      for (int idx = tid; idx < RL * PER_ROW16; idx += 256) {
        const int r = idx / PER_ROW16, p = idx % PER_ROW16;
        uint4 val = make_uint4(0u, 0u, 0u, 0u);
        if (r < nrow) val = reinterpret_cast<const uint4*>(Vin + (size_t)(c0 + r) * DV + cg * NC)[p];
        reinterpret_cast<uint4*>(sV + r * NC)[p] = val;
      }
    }
    __syncthreads();
    // compact list of the chunk's state leaders (wave 0)
    if (wv == 0) {
      int n = 0;
      for (int base = 0; base < nrow; base += 64) {
        const int i = base + lane;
        const bool isl = (i < nrow) && (sDeath[i] >= 0);
        const uint64_t bal = __ballot(isl);
        const int pos = n + __popcll(bal & ((1ull << lane) - 1ull));
        if (isl) {
          sLeadU[pos] = i;
          sLeadD[pos] = sDeath[i];
        }
        n += __popcll(bal);
      }
      if (lane == 0) sCnt[0] = n;
    }
    __syncthreads();
    const int nLead = sCnt[0];
    // first leader of each 32-token block (the leader list is in token order)
    for (int sb = tid; sb <= RL / 32; sb += 256) {
      int lo = 0, hi = nLead;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (sLeadU[mid] < 32 * sb) lo = mid + 1; else hi = mid;
      }
      sBlk[sb] = lo;
    }
    __syncthreads();

    // ------------------------------------------------------------- readout
    if (do_out) {
      int tr[NT];
      bool rv[NT];
      float rf[NT];
      FT qf[NT][KS];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        tr[nt] = 32 * (wv + NWAVE * nt) + l32;
        rv[nt] = tr[nt] < nrow;
        rf[nt] = rv[nt] ? sRf[tr[nt]] : 0.f;
        const Tin* qrow = Qin + (size_t)(c0 + (rv[nt] ? tr[nt] : 0)) * DK;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          qf[nt][ks] = rv[nt] ? FR::load(qrow + 16 * ks + 8 * half) : FR::zero();
      }
      f32x16 acc[NT];
      int cnt[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[nt] = zero16();
        cnt[nt] = 0;
      }

      // inter-chunk part: stream the states present at the chunk start, three
      // ahead, each through its own named register buffer (constant indexing).
      // Load order per step: lambda of the next state, then the prefetch, so
      // that waiting for a lambda never waits for a prefetch.
      if (m > 0) {
      u32x4 preA[V16], preB[V16], preC[V16];
      auto prefetch = [&](int j, u32x4(&pr)[V16]) __attribute__((always_inline)) {
        const u32x4* src = reinterpret_cast<const u32x4*>(slice_of(sPerm[min(j, m - 1)]));
#pragma unroll
        for (int u = 0; u < V16; ++u) pr[u] = src[tid + 256 * u];
      };
      prefetch(0, preA);
      prefetch(1, preB);
      prefetch(2, preC);
      // lambda rows of this lane's tokens (clamped to a valid row; a missing
      // lambda reads the key tensor and is replaced by 1)
      const Tin* lp[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        lp[nt] = Lin ? Lin + (size_t)(c0 + (rv[nt] ? tr[nt] : 0)) * C : Kin;
      Tin lamC[NT];
      {
        const int d0 = sDt[0];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          cnt[nt] = (d0 > c0 + tr[nt]) ? 1 : 0;
          lamC[nt] = lp[nt][Lin ? max(cnt[nt] - 1, 0) : 0];
        }
      }
      auto scale = [&](f32x16& ac, const f32x16& fr, float wgt) __attribute__((always_inline)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) ac[r] += wgt * fr[r];
      };
      auto chain = [&](const Tin* A, int nt) __attribute__((always_inline)) -> f32x16 {
        f32x16 fr = zero16();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) FR::mma(fr, FR::load(A + ((ks * 2 + half) * 32 + l32) * 8), qf[nt][ks]);
        return fr;
      };
      auto step = [&](int j, u32x4(&pr)[V16]) __attribute__((always_inline)) {
        u32x4* rb = ring + (j & 1) * SLICE16;
#pragma unroll
        for (int u = 0; u < V16; ++u) rb[tid + 256 * u] = pr[u];
        // lambda of state j + 1: raw values, converted when used
        const int jn = min(j + 1, m - 1);
        const int dn = sDt[jn];
        int cntN[NT];
        Tin lamN[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          cntN[nt] = cnt[nt] + ((j + 1 < m && dn > c0 + tr[nt]) ? 1 : 0);
          lamN[nt] = lp[nt][Lin ? max(cntN[nt] - 1, 0) : 0];
        }
        prefetch(j + 3, pr);
        __syncthreads();
        const float sf = sSf[j];
        float wgt[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) wgt[nt] = (Lin ? to_f32(lamC[nt]) : 1.f) * rf[nt] * sf;
        const Tin* A = reinterpret_cast<const Tin*>(rb);
        // two fresh accumulators in flight: the MFMA chain of one token tile
        // runs while the previous tile is scaled into its accumulator
        f32x16 frA = chain(A, 0);
        if constexpr (NT == 1) {
          scale(acc[0], frA, wgt[0]);
        } else {
          f32x16 frB = chain(A, 1);
          scale(acc[0], frA, wgt[0]);
#pragma unroll
          for (int nt = 2; nt < NT; nt += 2) {
            frA = chain(A, nt);
            scale(acc[nt - 1], frB, wgt[nt - 1]);
            if (nt + 1 < NT) {
              frB = chain(A, nt + 1);
              scale(acc[nt], frA, wgt[nt]);
            } else {
              scale(acc[nt], frA, wgt[nt]);
            }
          }
          if (NT % 2 == 0) scale(acc[NT - 1], frB, wgt[NT - 1]);
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          cnt[nt] = cntN[nt];
          lamC[nt] = lamN[nt];
        }
      };
      for (int j0 = 0; j0 < m; j0 += 3) {
        step(j0, preA);
        if (j0 + 1 < m) step(j0 + 1, preB);
        if (j0 + 2 < m) step(j0 + 2, preC);
      }
      }

      // intra-chunk part
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int trn = tr[nt];
        const int tabs = c0 + trn;
        const int Aold = cnt[nt];
        const int blk_t = trn >> 5;
        const Tin* lrow = Lin ? Lin + (size_t)(c0 + (rv[nt] ? trn : 0)) * C : nullptr;
        int before = 0;  // leaders live at t in the blocks before sb
        const int nsb = min(wv + NWAVE * nt + 1, (nrow + 31) >> 5);
        for (int sb = 0; sb < nsb; ++sb) {
          // leaders inside block sb that are live at token t, as a bit mask
          uint32_t word = 0u;
          for (int k2 = sBlk[sb]; k2 < sBlk[sb + 1]; ++k2)
            if (sLeadD[k2] > tabs) word |= 1u << (sLeadU[k2] & 31);
          f32x16 pt = zero16();
          const int srow = 32 * sb + l32;
          const Tin* krow = Kin + (size_t)(c0 + min(srow, nrow - 1)) * DK;
          const bool svalid = srow < nrow;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            FR::mma(pt, svalid ? FR::load(krow + 16 * ks + 8 * half) : FR::zero(), qf[nt][ks]);
          float pw[16];
          if (sb < blk_t) {
            // the whole block precedes the token: one decay factor per lane, and
            // lambda uniform unless a live leader starts inside the block
            const float f1 = rv[nt] ? __expf((float)(sG[trn] - sG[32 * sb + 31])) : 0.f;
            if ((word & ~1u) == 0u) {
              const int idx = min(max(Aold + before + (int)(word & 1u) - 1, 0), C - 1);
              const float f = f1 * ((lrow && rv[nt]) ? to_f32(lrow[idx]) : 1.f);
#pragma unroll
              for (int r = 0; r < 16; ++r) pw[r] = pt[r] * f * sBf[32 * sb + out_row(r, lane)];
            } else {
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const int so = out_row(r, lane);
                const int cl = before + __popc(word & (0xFFFFFFFFu >> (31 - so)));
                const int idx = min(max(Aold + cl - 1, 0), C - 1);
                const float lam = (lrow && rv[nt]) ? to_f32(lrow[idx]) : 1.f;
                pw[r] = pt[r] * f1 * lam * sBf[32 * sb + so];
              }
            }
          } else {
            // the token's own block: causal mask and decay per element
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int so = out_row(r, lane);
              const int s = 32 * sb + so;
              float wgt = 0.f;
              if (rv[nt] && s <= trn) {
                const int cl = before + __popc(word & (0xFFFFFFFFu >> (31 - so)));
                const int idx = min(max(Aold + cl - 1, 0), C - 1);
                const float lam = lrow ? to_f32(lrow[idx]) : 1.f;
                wgt = lam * __expf((float)(sG[trn] - sG[s]));
              }
              pw[r] = pt[r] * wgt;
            }
          }
          before += __popc(word);
#pragma unroll
          for (int st = 0; st < 2; ++st) {
            float va[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
              va[e] = to_f32(sV[(32 * sb + 16 * st + 8 * (e >> 2) + 4 * half + (e & 3)) * NC + l32]);
            FR::mma(acc[nt], FR::from_floats(va), FR::from_floats(pw + 8 * st));
          }
        }
        if (rv[nt]) {
          Tout* orow = Out + (size_t)(c0 + trn) * DV + cg * NC;
#pragma unroll
          for (int r = 0; r < 16; ++r) orow[out_row(r, lane)] = from_f32<Tout>(acc[nt][r]);
        }
      }
    }

    // ------------------------------------------------------- state update
    __syncthreads();
    // live states after the chunk: the old leaders still alive, then the new
    // leaders still alive, in chronological order
    const int nAO = block_excl_count(m, [&](int j) { return sDt[j] >= c1; }, eJa, red);
    // (the chunk's sDeath row is no longer needed: it receives the leaders' counts)
    const int nAN = block_excl_count(nLead, [&](int k2) { return sLeadD[k2] >= c1; }, sDeath, red);
    const int ne = nAO + nAN;
    const int ndead = m - nAO;
    // eJa[j] / sDeath[k2] hold the prefix counts; ePhys temporarily receives the
    // first old index of each old group, eLead the position of each new leader
    for (int j = tid; j < m; j += 256) {
      const int pos = eJa[j];
      if (sDt[j] >= c1)
        ePhys[pos] = j;
      else
        ePool[j - pos] = sPerm[j];  // slots of states merged away, in order
    }
    for (int k2 = tid; k2 < nLead; k2 += 256)
      if (sLeadD[k2] >= c1) eLead[nAO + sDeath[k2]] = sLeadU[k2];
    for (int x = tid; x < C - m; x += 256) ePool[ndead + x] = sPerm[m + x];  // free slots
    __syncthreads();
    {
      int ja_[4], jb_[4], r0_[4], r1_[4], ld_[4], ph_[4], ch_[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = tid + 256 * u;
        if (e >= ne) continue;
        if (e < nAO) {
          ja_[u] = ePhys[e];
          jb_[u] = (e + 1 < nAO) ? ePhys[e + 1] - 1 : m - 1;
          r0_[u] = 0;
          r1_[u] = (e == nAO - 1) ? ((nAN > 0) ? eLead[nAO] - 1 : nrow - 1) : -1;
          ld_[u] = sLead[ja_[u]];
          ph_[u] = sPerm[ja_[u]];
          ch_[u] = (jb_[u] > ja_[u] || r1_[u] >= r0_[u]) ? 1 : 0;
        } else {
          ja_[u] = -1;
          jb_[u] = -2;
          r0_[u] = eLead[e];
          r1_[u] = (e + 1 < ne) ? eLead[e + 1] - 1 : nrow - 1;
          ld_[u] = c0 + r0_[u];
          ph_[u] = ePool[e - nAO];
          ch_[u] = 1;
        }
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = tid + 256 * u;
        if (e >= ne) continue;
        eJa[e] = ja_[u];
        eJb[e] = jb_[u];
        eR0[e] = r0_[u];
        eR1[e] = r1_[u];
        eLead[e] = ld_[u];
        ePhys[e] = ph_[u];
        eChg[e] = ch_[u];
      }
    }
    __syncthreads();

    // new states: first those with an old part (they read old slots), then the
    // purely new ones (which may reuse the slots of merged-away states)
    for (int phase = 0; phase < 2; ++phase) {
      for (int e = 0; e < ne; ++e) {
        if (!eChg[e] || ((eJa[e] >= 0) != (phase == 0))) continue;
        if (wv >= DK / 32) continue;  // one 32-row band of d_k per wave
        const int ja = eJa[e], jb = eJb[e], r0 = eR0[e], r1 = eR1[e];
        const int ib = 32 * wv;
        f32x16 acc16 = zero16();
        if (r1 >= r0) {
          for (int sg = r0 >> 4; sg <= (r1 >> 4); ++sg) {
            float kt[8], vb[8];
#pragma unroll
            for (int e8 = 0; e8 < 8; ++e8) {
              const int s = 16 * sg + 8 * half + e8;
              const bool in = (s >= r0) && (s <= r1);
              kt[e8] = in ? sDecE[s] * to_f32(Kin[(size_t)(c0 + s) * DK + ib + l32]) : 0.f;
              vb[e8] = in ? to_f32(sV[s * NC + l32]) : 0.f;
            }
            const FT bv = FR::from_floats(vb);
            if constexpr (sizeof(Tin) == 4) {
              FR::mma(acc16, FR::from_floats(kt), bv);
            } else {
              // three bf16 terms carry the float32 value of K~
              float q1[8], q2[8];
              const FT hi = FR::from_floats(kt);
#pragma unroll
              for (int e8 = 0; e8 < 8; ++e8) q1[e8] = kt[e8] - (float)hi[e8];
              const FT mid = FR::from_floats(q1);
#pragma unroll
              for (int e8 = 0; e8 < 8; ++e8) q2[e8] = q1[e8] - (float)mid[e8];
              const FT lo = FR::from_floats(q2);
              FR::mma(acc16, lo, bv);
              FR::mma(acc16, mid, bv);
              FR::mma(acc16, hi, bv);
            }
          }
        }
        for (int j = ja; j <= jb; ++j) {
          const float f = __expf((float)(Gend - sF[j]));
          const float* src = states + (size_t)sPerm[j] * D + cg * NC + l32;
#pragma unroll
          for (int r = 0; r < 16; ++r) acc16[r] += f * src[(size_t)(ib + out_row(r, lane)) * DV];
        }
        float* dst = states + (size_t)ePhys[e] * D + cg * NC + l32;
#pragma unroll
        for (int r = 0; r < 16; ++r) dst[(size_t)(ib + out_row(r, lane)) * DV] = acc16[r];
        Tin* sh = slice_of(ePhys[e]);
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int ks = (ib >> 4) + (g4 >> 1);
          Tin* d4 = sh + ((ks * 2 + (g4 & 1)) * 32 + l32) * 8 + 4 * half;
#pragma unroll
          for (int q = 0; q < 4; ++q) d4[q] = from_f32<Tin>(acc16[4 * g4 + q]);
        }
      }
      __syncthreads();
    }
    // bookkeeping for the next chunk
    {
      double f_[4];
      int ld_[4], ph_[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = tid + 256 * u;
        if (e < ne) {
          f_[u] = eChg[e] ? Gend : sF[eJa[e]];
          ld_[u] = eLead[e];
          ph_[u] = ePhys[e];
        } else if (e < C) {
          ph_[u] = ePool[nAN + (e - ne)];
        }
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = tid + 256 * u;
        if (e < ne) {
          sF[e] = f_[u];
          sLead[e] = ld_[u];
          sPerm[e] = ph_[u];
        } else if (e < C) {
          sPerm[e] = ph_[u];
        }
      }
    }
    m = ne;
  }
  __syncthreads();

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

template <int DK, int DV, typename Tin, int NT>
static hipError_t launch_readout_t(const PrefillArgs& a, const PrefillWS& w, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  const int grid = (int)round_up(nh, 8) * (DV / NC);
  const size_t shm = RO<DK, Tin, NT>::smem_bytes(a.desc.C);
  if (shm > 160 * 1024) return hipErrorInvalidValue;
  if (a.out_dtype == DLA_F32) {
    auto k = prefill_readout_kernel<DK, DV, Tin, float, NT>;
    hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    hipLaunchKernelGGL(k, dim3(grid), dim3(256), shm, s, a, w);
  } else {
    auto k = prefill_readout_kernel<DK, DV, Tin, bf16_t, NT>;
    hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    hipLaunchKernelGGL(k, dim3(grid), dim3(256), shm, s, a, w);
  }
  return hipGetLastError();
}

template <int DK, int DV>
static hipError_t launch_readout_dims(const PrefillArgs& a, const PrefillWS& w, hipStream_t s) {
  if (a.in_dtype == DLA_F32) return launch_readout_t<DK, DV, float, 2>(a, w, s);
  return launch_readout_t<DK, DV, bf16_t, 4>(a, w, s);
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
