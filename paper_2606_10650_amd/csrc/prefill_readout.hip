// Prefill, stage 3: multi-state readout and state-cache maintenance.
//
// Readout (eq. capacity_bounded_output): o_t = sum_j lambda[t][j] q_t^T S_j over
// the states of the cache after token t.  The decisions of stage 2 fix, for
// every token, which states exist; this stage turns them into dense MFMA work.
//
// One workgroup of 8 waves per (head, 32 value columns), sequential over chunks
// of 256 tokens; each wave owns one 32-token tile of a chunk.
//   * inter-chunk part: every state S_j present at the chunk start contributes
//     lambda[t][x_j(t)] exp(G_t - F_j) q_t^T S~_j, x_j(t) being its chronological
//     index at token t: the number of live state leaders up to it, where a
//     leader lives while its death token (from stage 2) is later than t.  The
//     tile S~_j^T Q^T (32 columns x 32 tokens, K = d_k) is a bf16 MFMA chain;
//     each lane owns one token of the tile, so the weight is a per-lane scalar
//     applied to the tile's fresh accumulator.  States are streamed as a copy
//     in MFMA operand order (the shadow), three states ahead through registers
//     and a double-buffered LDS ring (one barrier per state); each wave reads a
//     state's operand from LDS once.
//   * key-block loop: the chunk's keys are staged 32 tokens at a time in LDS
//     (double-buffered, the next block loaded while the current one is used),
//     row-major and transposed.  Each block serves two products:
//       - intra-chunk readout (Q K^T (.) M) V with M[t][s] = [s <= t]
//         exp(G_t - G_s) lambda[t][slot_t(s)]; slot_t(s) is uniform over a
//         block unless a live leader starts inside it, so lambda is gathered
//         once per (token, block) in the common case;
//       - the chunk's share of every changed state: the tokens of the chunk
//         form consecutive ranges, one per state alive after the chunk, and
//         each wave accumulates sum_s exp(G_end - G_s) k_s v_s^T over the
//         current range for its 32-row band of d_k (K~ split into three bf16
//         terms, so the MFMA product is exact to float32 rounding).  At the end
//         of a range the state is completed with the decayed old states it
//         absorbed and stored in frame G_end (float32 master in the cache plus
//         its shadow).
//     States changed by merges alone are rebuilt before the loop (they read old
//     slots that new states may reuse); unchanged states are not touched (lazy
//     decay).
#include "mfma.h"
#include "prefill.h"

namespace dla {

constexpr int NWAVE = 8;             // waves per workgroup (two per SIMD)
constexpr int NTHR = 64 * NWAVE;
constexpr int NC = 32;  // value columns per workgroup

// Token tile owned by wave wv (one 32-token tile per wave): waves p and
// p + NWAVE/2 own the tiles p and NWAVE - 1 - p, the pair they share in the
// inter-chunk readout.
__device__ __forceinline__ int tile_of(int wv, int) {
  return wv < NWAVE / 2 ? wv : 3 * NWAVE / 2 - 1 - wv;
}

template <int DK, typename Tin, int NT>
struct RO {
  static constexpr int RL = 32 * NWAVE * NT;  // tokens per chunk
  static constexpr int KS = DK / 16;
  static constexpr int E = (int)sizeof(Tin);
  static constexpr int EPP = 16 / E;                             // elements per 16 bytes
  static constexpr int SLICE = DK * NC;                          // elements per (state, group)
  // LDS row strides (elements), padded by 16 bytes so that lanes reading
  // consecutive rows hit distinct banks
  static constexpr int VTS = RL + EPP;       // transposed values  [NC][VTS]
  static constexpr int KRS = DK + EPP;       // key block, row-major [32][KRS]
  static constexpr int KBUF = 32 * KRS;
  static constexpr int KROW16 = DK * E / 16;  // 16-byte pieces per key row
  static constexpr int KPT = (32 * KROW16 + NTHR / 2 - 1) / (NTHR / 2);  // per staging thread
  // lambda window of lw entries per token, stored with lw + 1 stride
  static_assert(NT == 1, "one token tile per wave");
  static constexpr int SLICE16 = SLICE * E / 16;   // 16-byte pieces per slice
  static constexpr size_t RING_BYTES = 2 * (size_t)SLICE16 * 16;
  static size_t smem_bytes(int C, int lw) {
    size_t off = RING_BYTES;                          // ring
    off += (size_t)NC * VTS * E;                      // sVt
    off += 2 * (size_t)KBUF * E;                      // key blocks
    off += (size_t)RL * (lw > 0 ? lw + 1 : 0) * E;    // lambda window
    off = round_up(off, 16);
    off += (size_t)RL * (8 + 4 * 7);                  // sG sRf sBf sDecE sDeath sLeadU sLeadD sAold
    off += (size_t)C * 8 + (size_t)(C + 4) * 4;       // sF, sSf (zero past the last state)
    off += (size_t)C * 4 * 11 + 64;                   // int arrays, reduction scratch
    return round_up(off, 16);
  }
};

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

template <int DK, int DV, typename Tin, typename Tout, int NT>
__global__ __launch_bounds__(NTHR) void prefill_readout_kernel(PrefillArgs a, PrefillWS w, int lw) {
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using P = RO<DK, Tin, NT>;
  constexpr int D = DK * DV;
  constexpr int NCG = DV / NC;
  constexpr int KS = P::KS;
  constexpr int RL = P::RL;
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
  u32x4* ring = reinterpret_cast<u32x4*>(smem);            // 2 state slices
  Tin* sVt = reinterpret_cast<Tin*>(smem + P::RING_BYTES);  // [NC][VTS] values, transposed
  Tin* kbuf = sVt + NC * P::VTS;                          // 2 key blocks of KBUF elements
  Tin* sLamW = kbuf + 2 * P::KBUF;                        // [RL][lw + 1] lambda window
  const int lws = lw + 1;
  double* sG = reinterpret_cast<double*>(smem + round_up(
      P::RING_BYTES +
          ((size_t)NC * P::VTS + 2 * (size_t)P::KBUF + (size_t)RL * (lw > 0 ? lws : 0)) * P::E,
      16));
  float* sRf = reinterpret_cast<float*>(sG + RL);  // exp(G_t - G_ref)
  float* sBf = sRf + RL;                            // exp(G_blockend - G_s)
  float* sDecE = sBf + RL;                          // exp(G_end - G_s)
  int32_t* sDeath = reinterpret_cast<int32_t*>(sDecE + RL);
  int32_t* sLeadU = sDeath + RL;  // in-chunk leaders: position in the chunk
  int32_t* sLeadD = sLeadU + RL;  //                   death token
  int32_t* sAold = sLeadD + RL;   // old states alive at each token of the chunk
  double* sF = reinterpret_cast<double*>(sAold + RL);
  float* sSf = reinterpret_cast<float*>(sF + C);  // exp(G_ref - F_j); 0 for j in [m, m + 3)
  int32_t* sPerm = reinterpret_cast<int32_t*>(sSf + C + 4);
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
  for (int j = tid; j < C; j += NTHR) {
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
    for (int kg = tid >> 5; kg < DK / 8; kg += NTHR / 32) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = src[(size_t)(8 * kg + e) * DV + c];
      Tin* d8 = dst + kg * 256 + c * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) d8[e] = from_f32<Tin>(x[e]);
    }
  }

  // band of d_k rows owned by this wave in the state update; the waves form
  // NWAVE / NBAND groups that each cover all bands
  constexpr int NBAND = DK / 32;
  const int ib = 32 * (wv % NBAND);
  const int wgrp = wv / NBAND;
  const bool band = wgrp == 0;
  // decayed old states j = ja..jb (float32 masters) added to a band accumulator
  auto add_old = [&](f32x16& acc16, int ja, int jb, double Gend) __attribute__((always_inline)) {
    for (int j = ja; j <= jb; ++j) {
      const float* src = states + (size_t)sPerm[j] * D + cg * NC + l32;
      // all 16 loads in flight before the first use
      float x[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) x[r] = src[(size_t)(ib + out_row(r, lane)) * DV];
      const float f = __expf((float)(Gend - sF[j]));
#pragma unroll
      for (int r = 0; r < 16; ++r) acc16[r] += f * x[r];
    }
  };
  // store a band of a state: float32 master and its shadow
  auto store_state = [&](const f32x16& acc16, int phys) __attribute__((always_inline)) {
    float* dst = states + (size_t)phys * D + cg * NC + l32;
#pragma unroll
    for (int r = 0; r < 16; ++r) dst[(size_t)(ib + out_row(r, lane)) * DV] = acc16[r];
    Tin* sh = slice_of(phys);
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int ks = (ib >> 4) + (g4 >> 1);
      Tin* d4 = sh + ((ks * 2 + (g4 & 1)) * 32 + l32) * 8 + 4 * half;
#pragma unroll
      for (int q = 0; q < 4; ++q) d4[q] = from_f32<Tin>(acc16[4 * g4 + q]);
    }
  };

  for (int c0 = 0; c0 < T; c0 += RL) {
    const int nrow = min(RL, T - c0);
    const int c1 = c0 + nrow;
    const int nblk = (nrow + 31) >> 5;
    const double Gref = (c0 == 0) ? G0 : Gtok[c0 - 1];
    const double Gend = Gtok[c1 - 1];
    __syncthreads();
    for (int i = tid; i < RL; i += NTHR) {
      const int ic = min(i, nrow - 1);
      const double Gi = Gtok[c0 + ic];
      const int be = min(32 * (i >> 5) + 31, nrow - 1);
      sG[i] = Gi;
      sRf[i] = __expf((float)(Gi - Gref));
      sBf[i] = __expf((float)(Gtok[c0 + be] - Gi));
      sDecE[i] = (i < nrow) ? __expf((float)(Gend - Gi)) : 0.f;
      sDeath[i] = (i < nrow) ? death[c0 + i] : -1;
    }
    for (int j = tid; j < m + 3; j += NTHR) {
      if (j < m) {
        const int ld = sLead[j];
        sDt[j] = (ld >= 0) ? death[ld] : iv.death0[ld + m0];
      }
      sSf[j] = (j < m) ? __expf((float)(Gref - sF[j])) : 0.f;
    }
    // this group's value columns of the chunk, transposed (sVt[c][r])
    {
      constexpr int PER_ROW16 = NC * P::E / 16;
      for (int idx = tid; idx < RL * PER_ROW16; idx += NTHR) {
        const int r = idx / PER_ROW16, p = idx % PER_ROW16;
        u32x4 val = {0u, 0u, 0u, 0u};
        if (r < nrow)
          val = *reinterpret_cast<const u32x4*>(Vin + (size_t)(c0 + r) * DV + cg * NC + p * P::EPP);
#pragma unroll
        for (int e = 0; e < P::EPP; ++e) sVt[(p * P::EPP + e) * P::VTS + r] = piece_elem<Tin>(val, e);
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
    for (int sb = tid; sb <= RL / 32; sb += NTHR) {
      int lo = 0, hi = nLead;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (sLeadU[mid] < 32 * sb) lo = mid + 1; else hi = mid;
      }
      sBlk[sb] = lo;
    }

    // ------------------------------------------ states alive after the chunk
    // the old leaders still alive, then the new leaders still alive, in
    // chronological order
    const int nAO = block_excl_count(m, [&](int j) { return sDt[j] >= c1; }, eJa, red);
    // (the chunk's sDeath row is no longer needed: it receives the leaders' counts)
    const int nAN = block_excl_count(nLead, [&](int k2) { return sLeadD[k2] >= c1; }, sDeath, red);
    const int ne = nAO + nAN;
    const int ndead = m - nAO;
    // eJa[j] / sDeath[k2] hold the prefix counts; ePhys temporarily receives the
    // first old index of each old group, eLead the position of each new leader
    for (int j = tid; j < m; j += NTHR) {
      const int pos = eJa[j];
      if (sDt[j] >= c1)
        ePhys[pos] = j;
      else
        ePool[j - pos] = sPerm[j];  // slots of states merged away, in order
    }
    for (int k2 = tid; k2 < nLead; k2 += NTHR)
      if (sLeadD[k2] >= c1) eLead[nAO + sDeath[k2]] = sLeadU[k2];
    for (int x = tid; x < C - m; x += NTHR) ePool[ndead + x] = sPerm[m + x];  // free slots
    __syncthreads();
    {
      constexpr int PU = 1024 / NTHR;
      int ja_[PU], jb_[PU], r0_[PU], r1_[PU], ld_[PU], ph_[PU], ch_[PU];
#pragma unroll
      for (int u = 0; u < PU; ++u) {
        const int e = tid + NTHR * u;
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
      for (int u = 0; u < PU; ++u) {
        const int e = tid + NTHR * u;
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

    // this wave's token tile for the intra-chunk readout and the output
    int tr[NT];
    bool rv[NT];
    FT qf[NT][KS];
    f32x16 acc[NT];
    int cnt[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      tr[nt] = 32 * tile_of(wv, nt) + l32;
      rv[nt] = tr[nt] < nrow;
      acc[nt] = zero16();
      cnt[nt] = 0;
    }
    if (do_out) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const Tin* qrow = Qin + (size_t)(c0 + (rv[nt] ? tr[nt] : 0)) * DK;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          qf[nt][ks] = rv[nt] ? FR::load(qrow + 16 * ks + 8 * half) : FR::zero();
      }
    }

    // ------------------------------------------------ inter-chunk readout
    // Stream the states present at the chunk start through a double-buffered
    // LDS ring: each thread loads its share of a state's shadow slice three
    // states ahead (named register buffers, constant indexing), writes it to
    // the ring, and after one barrier every wave reads the state's operand from
    // LDS once for its token tile.  Per step the loads are issued in a fixed
    // order (lambda of the next state, then the prefetch), so waiting for one
    // never waits for the other.
    if (do_out && m > 0) {
      float rf[NT];
      const Tin* lp[NT];
      Tin lamC[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        rf[nt] = rv[nt] ? sRf[tr[nt]] : 0.f;
        // lambda row (clamped to a valid row; a missing lambda reads the key
        // tensor and is replaced by 1)
        lp[nt] = Lin ? Lin + (size_t)(c0 + (rv[nt] ? tr[nt] : 0)) * C : Kin;
      }
      constexpr int SL16 = P::SLICE16;
      constexpr int V16 = (SL16 + NTHR - 1) / NTHR;
      u32x4 preA[V16], preB[V16], preC[V16];
      auto prefetch = [&](int j, u32x4(&pr)[V16]) __attribute__((always_inline)) {
        const u32x4* src = reinterpret_cast<const u32x4*>(slice_of(sPerm[min(j, m - 1)]));
#pragma unroll
        for (int u = 0; u < V16; ++u) {
          const int pi = tid + NTHR * u;
          if (SL16 % NTHR == 0 || pi < SL16) pr[u] = src[pi];
        }
      };
      // first lambda, then the first three states: the steady-state order
      {
        const int d0 = sDt[0];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          cnt[nt] = (d0 > c0 + tr[nt]) ? 1 : 0;
          lamC[nt] = lp[nt][Lin ? max(cnt[nt] - 1, 0) : 0];
        }
      }
      prefetch(0, preA);
      prefetch(1, preB);
      prefetch(2, preC);
      auto step = [&](int j, u32x4(&pr)[V16]) __attribute__((always_inline)) {
        u32x4* rb = ring + (j & 1) * SL16;
#pragma unroll
        for (int u = 0; u < V16; ++u) {
          const int pi = tid + NTHR * u;
          if (SL16 % NTHR == 0 || pi < SL16) rb[pi] = pr[u];
        }
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
        __builtin_amdgcn_sched_barrier(0);
        prefetch(j + 3, pr);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        // weights of state j (a step past the last state has sSf = 0)
        const float sf = sSf[j];
        float wgt[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) wgt[nt] = (Lin ? to_f32(lamC[nt]) : 1.f) * rf[nt] * sf;
        // the state's operand, read from LDS once for all token tiles; each
        // tile's chain is split over two accumulators (even and odd K steps)
        const Tin* A = reinterpret_cast<const Tin*>(rb);
        FT sa[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) sa[ks] = FR::load(A + ((ks * 2 + half) * 32 + l32) * 8);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          f32x16 f0 = zero16(), f1 = zero16();
#pragma unroll
          for (int ks = 0; ks < KS; ks += 2) {
            FR::mma(f0, sa[ks], qf[nt][ks]);
            FR::mma(f1, sa[ks + 1], qf[nt][ks + 1]);
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[nt][r] += wgt[nt] * (f0[r] + f1[r]);
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          cnt[nt] = cntN[nt];
          lamC[nt] = lamN[nt];
        }
      };
      // whole triples: every step issues the same memory operations, so the
      // compiler keeps three prefetches in flight across iterations
      for (int j0 = 0; j0 < m; j0 += 3) {
        step(j0, preA);
        step(j0 + 1, preB);
        step(j0 + 2, preC);
      }
    }
    // old states alive at each of this wave's tokens (chronological index of
    // the first in-chunk state at that token)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      if (rv[nt]) sAold[tr[nt]] = cnt[nt];
    __syncthreads();  // the ring and the old shadows are no longer read

    // lambda window of every token: lambda[t][Aold_t - 1 + x] for x < lw, the
    // weights of the states that hold the chunk's own tokens
    if (do_out && Lin && lw > 0) {
      for (int idx = tid; idx < nrow * lw; idx += NTHR) {
        const int t = idx / lw, x = idx - t * lw;
        const int j = min(max(sAold[t] - 1 + x, 0), C - 1);
        sLamW[t * lws + x] = Lin[(size_t)(c0 + t) * C + j];
      }
    }

    // ------------------------------- states changed by merges of old states only
    if (band) {
      for (int e = 0; e < nAO; ++e) {
        if (!eChg[e] || eR1[e] >= eR0[e]) continue;
        f32x16 u16 = zero16();
        add_old(u16, eJa[e], eJb[e], Gend);
        store_state(u16, ePhys[e]);
      }
    }

    // ------------------------------------------------------- key-block loop
    // keys are staged by the upper half of the workgroup (waves that never
    // store to global memory inside the loop, so waiting for a prefetch never
    // waits for state stores)
    const bool kstager = tid >= NTHR / 2;
    const int ktid = tid - NTHR / 2;
    u32x4 kpre[P::KPT];
    auto kload = [&](int sb) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < P::KPT; ++u) {
        const int pi = ktid + (NTHR / 2) * u;
        const int r = pi / P::KROW16, pc = pi % P::KROW16;
        const int tok = 32 * sb + r;
        u32x4 z = {0u, 0u, 0u, 0u};
        if (r < 32 && tok < nrow)
          z = *reinterpret_cast<const u32x4*>(Kin + (size_t)(c0 + tok) * DK + pc * P::EPP);
        kpre[u] = z;
      }
    };
    auto kstore = [&](Tin* kb) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < P::KPT; ++u) {
        const int pi = ktid + (NTHR / 2) * u;
        const int r = pi / P::KROW16, pc = pi % P::KROW16;
        if (r < 32) *reinterpret_cast<u32x4*>(kb + r * P::KRS + pc * P::EPP) = kpre[u];
      }
    };
    // the first range of chunk tokens: the newest old state's, unless a new
    // leader that stays alive starts the chunk
    int rc = (nAO > 0 && eR1[nAO - 1] >= eR0[nAO - 1]) ? nAO - 1 : nAO;
    f32x16 uacc = zero16();
    int before[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) before[nt] = 0;
    // nothing issued before the loop is outstanding inside it (vmcnt(0)), so the
    // only memory operations a wave waits for there are its own
    __builtin_amdgcn_s_waitcnt(0x0F70);
    if (kstager) kload(0);
    for (int sb = 0; sb < nblk; ++sb) {
      Tin* kb = kbuf + (sb & 1) * P::KBUF;
      if (kstager) {
        kstore(kb);
        if (sb + 1 < nblk) kload(sb + 1);
      }
      __syncthreads();

      // intra-chunk readout
      if (do_out && sb <= max(tile_of(wv, 0), tile_of(wv, NT - 1))) {
        const Tin* krow = kb + l32 * P::KRS + 8 * half;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int ti = tile_of(wv, nt);
          if (sb > ti || 32 * ti >= nrow) continue;
          const int trn = tr[nt];
          const int tabs = c0 + trn;
          const int Aold = cnt[nt];
          const Tin* lrow = Lin ? Lin + (size_t)(c0 + (rv[nt] ? trn : 0)) * C : nullptr;
          const Tin* lwin = sLamW + trn * lws;
          // weight of the state at window position x (x = live in-chunk leaders
          // up to the key token): from the window, else from the lambda row
          auto lam_at = [&](int x) __attribute__((always_inline)) -> float {
            if (!lrow || !rv[nt]) return 1.f;
            if (x < lw) return to_f32(lwin[x]);
            return to_f32(lrow[min(max(Aold - 1 + x, 0), C - 1)]);
          };
          // leaders inside block sb that are live at token t, as a bit mask
          uint32_t word = 0u;
          for (int k2 = sBlk[sb]; k2 < sBlk[sb + 1]; ++k2)
            if (sLeadD[k2] > tabs) word |= 1u << (sLeadU[k2] & 31);
          // P^T tile: rows = the block's key tokens, columns = this tile's tokens
          f32x16 pt = zero16();
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) FR::mma(pt, FR::load(krow + 16 * ks), qf[nt][ks]);
          // weights, in place
          if (sb < ti) {
            // the whole block precedes the token: one decay factor per lane, and
            // lambda uniform unless a live leader starts inside the block
            const float f1 = rv[nt] ? __expf((float)(sG[trn] - sG[32 * sb + 31])) : 0.f;
            if ((word & ~1u) == 0u) {
              const float f = f1 * lam_at(before[nt] + (int)(word & 1u));
#pragma unroll
              for (int r = 0; r < 16; ++r) pt[r] *= f * sBf[32 * sb + out_row(r, lane)];
            } else {
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const int so = out_row(r, lane);
                const int cl = before[nt] + __popc(word & (0xFFFFFFFFu >> (31 - so)));
                pt[r] *= f1 * lam_at(cl) * sBf[32 * sb + so];
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
                const int cl = before[nt] + __popc(word & (0xFFFFFFFFu >> (31 - so)));
                wgt = lam_at(cl) * __expf((float)(sG[trn] - sG[s]));
              }
              pt[r] *= wgt;
            }
          }
          before[nt] += __popc(word);
          // values of the block's tokens in the permuted k order of the weights:
          // element e of half h <-> token 16 st + 8 (e / 4) + 4 h + e % 4
#pragma unroll
          for (int st = 0; st < 2; ++st) {
            float pw[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) pw[e] = pt[8 * st + e];
            const Tin* vp = sVt + l32 * P::VTS + 32 * sb + 16 * st + 4 * half;
            FR::mma(acc[nt], load_4x2<Tin>(vp, vp + 8), FR::from_floats(pw));
          }
        }
      }

      // the block's share of every changed state (this wave's band of d_k)
      if (band && rc < ne) {
        const int bs = 32 * sb, be = min(bs + 32, nrow);
        while (true) {
          const int r0 = max(eR0[rc], bs), r1 = min(eR1[rc], be - 1);
#pragma unroll
          for (int g = 0; g < 2; ++g) {
            const int gs = bs + 16 * g;
            if (gs > r1 || gs + 15 < r0) continue;
            // element e of half h <-> token gs + 8 h + e
            const int s0 = gs + 8 * half;
            const FT bv = FR::load(sVt + l32 * P::VTS + s0);
            // A = K~^T: column ib + l32 of the block's rows s0 .. s0 + 7 (the lanes
            // of a half read consecutive columns; the halves rows 8 apart, in
            // disjoint banks)
            const Tin* kc = kb + (s0 - bs) * P::KRS + ib + l32;
            float kx[8];
#pragma unroll
            for (int e8 = 0; e8 < 8; ++e8) {
              const int s = s0 + e8;
              kx[e8] = (s >= r0 && s <= r1) ? sDecE[s] * to_f32(kc[e8 * P::KRS]) : 0.f;
            }
            if constexpr (sizeof(Tin) == 4) {
              FR::mma(uacc, FR::from_floats(kx), bv);
            } else {
              // three bf16 terms carry the float32 value of K~
              float q1[8], q2[8];
              const FT hi = FR::from_floats(kx);
#pragma unroll
              for (int e8 = 0; e8 < 8; ++e8) q1[e8] = kx[e8] - (float)hi[e8];
              const FT mid = FR::from_floats(q1);
#pragma unroll
              for (int e8 = 0; e8 < 8; ++e8) q2[e8] = q1[e8] - (float)mid[e8];
              const FT lo = FR::from_floats(q2);
              FR::mma(uacc, lo, bv);
              FR::mma(uacc, mid, bv);
              FR::mma(uacc, hi, bv);
            }
          }
          if (eR1[rc] > be - 1) break;  // the range continues in the next block
          // the range ends here: complete the state and store it
          if (eJa[rc] >= 0) add_old(uacc, eJa[rc], eJb[rc], Gend);
          store_state(uacc, ePhys[rc]);
          uacc = zero16();
          ++rc;
          if (rc >= ne || eR0[rc] >= be) break;
        }
      }
    }

    // outputs
    if (do_out) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if (rv[nt]) {
          Tout* orow = Out + (size_t)(c0 + tr[nt]) * DV + cg * NC;
#pragma unroll
          for (int r = 0; r < 16; ++r) orow[out_row(r, lane)] = from_f32<Tout>(acc[nt][r]);
        }
      }
    }
    __syncthreads();

    // bookkeeping for the next chunk
    {
      constexpr int PU = 1024 / NTHR;
      double f_[PU];
      int ld_[PU], ph_[PU];
#pragma unroll
      for (int u = 0; u < PU; ++u) {
        const int e = tid + NTHR * u;
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
      for (int u = 0; u < PU; ++u) {
        const int e = tid + NTHR * u;
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
    for (int j = tid; j < C; j += NTHR) {
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

constexpr size_t kMaxLds = 160 * 1024;

// Largest lambda window (entries per token) that fits in LDS with chunk
// parameter NT, or -1 if none does.
template <int DK, typename Tin, int NT>
static int readout_window(int C) {
  for (int lw : {32, 16, 8, 0})
    if (RO<DK, Tin, NT>::smem_bytes(C, lw) <= kMaxLds) return lw;
  return -1;
}

template <int DK, int DV, typename Tin, int NT>
static hipError_t launch_readout_t(const PrefillArgs& a, const PrefillWS& w, int lw, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  const int grid = (int)round_up(nh, 8) * (DV / NC);
  const size_t shm = RO<DK, Tin, NT>::smem_bytes(a.desc.C, lw);
  if (shm > kMaxLds) return hipErrorInvalidValue;
  auto launch = [&](auto k) -> hipError_t {
    if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
        hipSuccess)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3(grid), dim3(NTHR), shm, s, a, w, lw);
    return hipGetLastError();
  };
  if (a.out_dtype == DLA_F32) return launch(prefill_readout_kernel<DK, DV, Tin, float, NT>);
  return launch(prefill_readout_kernel<DK, DV, Tin, bf16_t, NT>);
}

// 256-token chunks: one 32-token tile per wave, which keeps a wave's working
// set within the 256 registers it has at two waves per SIMD.
template <int DK, int DV>
static hipError_t launch_readout_dims(const PrefillArgs& a, const PrefillWS& w, hipStream_t s) {
  const int C = a.desc.C;
  if (a.in_dtype == DLA_F32) {
    const int lw = readout_window<DK, float, 1>(C);
    if (lw < 0) return hipErrorInvalidValue;
    return launch_readout_t<DK, DV, float, 1>(a, w, lw, s);
  }
  const int lw = readout_window<DK, bf16_t, 1>(C);
  if (lw < 0) return hipErrorInvalidValue;
  return launch_readout_t<DK, DV, bf16_t, 1>(a, w, lw, s);
}

bool prefill_readout_supported(const dla_cache_desc& d, dla_dtype in_dtype) {
  const int C = d.C;
  if (in_dtype == DLA_F32)
    return (d.d_k == 128 ? readout_window<128, float, 1>(C) : readout_window<64, float, 1>(C)) >= 0;
  return (d.d_k == 128 ? readout_window<128, bf16_t, 1>(C) : readout_window<64, bf16_t, 1>(C)) >= 0;
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
