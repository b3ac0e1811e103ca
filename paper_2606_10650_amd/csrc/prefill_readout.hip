// Prefill, stage 4: multi-state readout (eq. capacity_bounded_output),
//   o_t = sum_j lambda[t][j] q_t^T S_j   over the states of the cache after token t.
//
// Every chunk of RL tokens is independent here: the update stage recorded the
// states present at its start (a list of pool objects with their frames and
// death tokens), so one workgroup of 8 waves per (head, chunk, 32 value
// columns) computes the chunk's outputs with no sequential dependence.  Each
// wave owns NT token tiles of 32.
//   * inter-chunk part: every state S_j present at the chunk start contributes
//     lambda[t][x_j(t)] exp(G_t - F_j) q_t^T S~_j, x_j(t) being its chronological
//     index at token t: the number of live states up to it, a state living while
//     its death token is later than t.  The tile S~_j^T Q^T (32 columns x 32
//     tokens, K = d_k) is an MFMA chain; each lane owns one token of a tile, so
//     the weight is a per-lane scalar applied to the chain's result.  States
//     are streamed from the pool three ahead through registers and a
//     double-buffered LDS ring (one barrier per state); each wave reads a
//     state's operand from LDS once for all of its tiles.
//   * intra-chunk part: (Q K^T (.) M) V with M[t][s] = [s <= t] exp(G_t - G_s)
//     lambda[t][slot_t(s)] over the chunk's own keys, staged 32 tokens at a
//     time in LDS.  slot_t(s) is uniform over a key block unless a live state
//     leader starts inside it, so lambda is gathered once per (token, block) in
//     the common case.
// Workgroups are dealt to the 8 XCDs round-robin by id; the mapping puts the
// column groups and neighbouring chunks of one head on one XCD, so the chunk's
// queries, keys and lambda rows, and the state copies that neighbouring chunks
// share, are read from HBM once per L2.
#include "prefill_chunk.h"

namespace dla {

template <int DK, typename Tin>
struct RO : ChunkP<DK, Tin> {
  using B = ChunkP<DK, Tin>;
  static constexpr size_t RING_BYTES = 2 * (size_t)B::SLICE16 * 16;
  static constexpr size_t KB_BYTES = 2 * (size_t)B::KBUF * B::E;
  // the ring (inter part) and the key blocks (intra part) share LDS
  static constexpr size_t SHARED_BYTES = RING_BYTES > KB_BYTES ? RING_BYTES : KB_BYTES;
  static size_t smem_bytes(int C, int lw) {
    size_t off = round_up(SHARED_BYTES, 16);
    off += (size_t)NC * B::VTS * B::E;                    // sVt
    off += (size_t)B::RL * (lw > 0 ? lw + 1 : 0) * B::E;  // lambda window
    off = round_up(off, 16);
    off += (size_t)B::RL * (8 + 4 * 6);  // sG sRf sBf sDeath sLeadU sLeadD sAold
    off += (size_t)(C + 4) * 4 * 2;      // sSf, sObj (padded past the last state)
    off += (size_t)C * 4;                // sDt
    return round_up(off, 16);
  }
};

// Token tile of wave wv: with two tiles per wave, wave p owns tiles p and
// 2 NWAVE - 1 - p, so the causal intra-chunk work is the same for every wave.
template <int NT>
__device__ __forceinline__ int tile_of(int wv, int nt) {
  return nt == 0 ? wv : 2 * NWAVE - 1 - wv;
}

template <int DK, int DV, typename Tin, typename Tout>
__global__ __launch_bounds__(NTHR) void prefill_readout_kernel(PrefillArgs a, PrefillWS w,
                                                               SegPlan plan, int seg, int lw) {
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using P = RO<DK, Tin>;
  constexpr int NT = P::NT;
  constexpr int NCG = DV / NC;
  constexpr int KS = P::KS;
  constexpr int RL = P::RL;
  const int nh = a.desc.B * a.desc.H;
  const int cs = seg * plan.nch_seg;
  const int nchs = min(plan.nch, cs + plan.nch_seg) - cs;
  // id -> (XCD x, i); i -> (head group, chunk, column group), column group fastest
  const int bid = blockIdx.x;
  const int i = bid >> 3;
  const int cg = i % NCG;
  const int c = cs + (i / NCG) % nchs;
  const int h = (i / (NCG * nchs)) * 8 + (bid & 7);
  if (h >= nh) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int C = a.desc.C;
  const int T = a.T;

  extern __shared__ __align__(16) char smem[];
  u32x4* ring = reinterpret_cast<u32x4*>(smem);  // 2 state slices (inter part)
  Tin* kbuf = reinterpret_cast<Tin*>(smem);      // 2 key blocks (intra part)
  Tin* sVt = reinterpret_cast<Tin*>(smem + round_up(P::SHARED_BYTES, 16));  // [NC][VTS]
  Tin* sLamW = sVt + NC * P::VTS;  // [RL][lw + 1] lambda window
  const int lws = lw + 1;
  double* sG = reinterpret_cast<double*>(smem + round_up(
      round_up(P::SHARED_BYTES, 16) +
          ((size_t)NC * P::VTS + (size_t)RL * (lw > 0 ? lws : 0)) * P::E,
      16));
  float* sRf = reinterpret_cast<float*>(sG + RL);  // exp(G_t - G_ref)
  float* sBf = sRf + RL;                            // exp(G_blockend - G_s)
  int32_t* sDeath = reinterpret_cast<int32_t*>(sBf + RL);
  int32_t* sLeadU = sDeath + RL;  // in-chunk leaders: position in the chunk
  int32_t* sLeadD = sLeadU + RL;  //                   death token
  int32_t* sAold = sLeadD + RL;   // old states alive at each token of the chunk
  float* sSf = reinterpret_cast<float*>(sAold + RL);  // exp(G_ref - F_j); 0 for j >= m
  int32_t* sObj = reinterpret_cast<int32_t*>(sSf + C + 4);
  int32_t* sDt = sObj + C + 4;
  __shared__ int sCnt[2];
  __shared__ int sBlk[RL / 32 + 1];

  const double G0 = *init_at(w, h, C).G0;
  const double* Gtok = w.Gtok + (size_t)h * T;
  const int32_t* death = w.death + (size_t)h * T;
  const Tin* Kin = static_cast<const Tin*>(a.k) + (size_t)h * T * DK;
  const Tin* Vin = static_cast<const Tin*>(a.v) + (size_t)h * T * DV;
  const Tin* Qin = static_cast<const Tin*>(a.q) + (size_t)h * T * DK;
  const Tin* Lin = a.lam ? static_cast<const Tin*>(a.lam) + (size_t)h * T * C : nullptr;
  Tout* Out = static_cast<Tout*>(a.out) + (size_t)h * T * DV;

  const int c0 = c * RL;
  const int nrow = min(RL, T - c0);
  const int nblk = (nrow + 31) >> 5;
  const double Gref = (c0 == 0) ? G0 : Gtok[c0 - 1];

  // the chunk's state list
  const char* lst = list_at(w, h, c, plan.nch);
  const int m = min(max(*reinterpret_cast<const int32_t*>(lst), 0), C);
  {
    const ListEntry* ent = reinterpret_cast<const ListEntry*>(lst + 16);
    for (int j = tid; j < m + 4; j += NTHR) {
      if (j < m) {
        const ListEntry le = ent[j];
        sObj[j] = min(max(le.obj, 0), plan.P_cap - 1);
        sDt[j] = le.dt;
        sSf[j] = __expf((float)(Gref - le.F));
      } else {
        sObj[j] = 0;
        sSf[j] = 0.f;
      }
    }
  }
  for (int i2 = tid; i2 < RL; i2 += NTHR) {
    const int ic = min(i2, nrow - 1);
    const double Gi = Gtok[c0 + ic];
    const int be = min(32 * (i2 >> 5) + 31, nrow - 1);
    sG[i2] = Gi;
    sRf[i2] = __expf((float)(Gi - Gref));
    sBf[i2] = __expf((float)(Gtok[c0 + be] - Gi));
    sDeath[i2] = (i2 < nrow) ? death[c0 + i2] : -1;
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
      const int i2 = base + lane;
      const bool isl = (i2 < nrow) && (sDeath[i2] >= 0);
      const uint64_t bal = __ballot(isl);
      const int pos = n + __popcll(bal & ((1ull << lane) - 1ull));
      if (isl) {
        sLeadU[pos] = i2;
        sLeadD[pos] = sDeath[i2];
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

  // this wave's token tiles
  int tr[NT];
  bool rv[NT];
  FT qf[NT][KS];
  f32x16 acc[NT];
  int cnt[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    tr[nt] = 32 * tile_of<NT>(wv, nt) + l32;
    rv[nt] = tr[nt] < nrow;
    acc[nt] = zero16();
    cnt[nt] = 0;
    const Tin* qrow = Qin + (size_t)(c0 + (rv[nt] ? tr[nt] : 0)) * DK;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[nt][ks] = rv[nt] ? FR::load(qrow + 16 * ks + 8 * half) : FR::zero();
  }

  // ------------------------------------------------ inter-chunk readout
  // Each thread loads its share of a state's slice three states ahead (named
  // register buffers, constant indexing), writes it to the ring, and after one
  // barrier every wave reads the state's operand from LDS once for its tiles.
  // Per step the loads are issued in a fixed order (lambda of the next state,
  // then the prefetch), so waiting for one never waits for the other.
  if (m > 0) {
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
      const u32x4* src = reinterpret_cast<const u32x4*>(
          pool_slice<Tin>(w.pool, h, plan.P_cap, sObj[min(j, m - 1)], cg, NCG, P::SLICE));
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
      // the state's operand, read from LDS once for all token tiles
      const Tin* A = reinterpret_cast<const Tin*>(rb);
      FT sa[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) sa[ks] = FR::load(A + ((ks * 2 + half) * 32 + l32) * 8);
      f32x16 f[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) f[nt] = zero16();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) FR::mma(f[nt], sa[ks], qf[nt][ks]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[nt][r] += wgt[nt] * f[nt][r];
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
  __syncthreads();  // the ring is no longer read

  // lambda window of every token: lambda[t][Aold_t - 1 + x] for x < lw, the
  // weights of the states that hold the chunk's own tokens
  if (Lin && lw > 0) {
    for (int idx = tid; idx < nrow * lw; idx += NTHR) {
      const int t = idx / lw, x = idx - t * lw;
      const int j = min(max(sAold[t] - 1 + x, 0), C - 1);
      sLamW[t * lws + x] = Lin[(size_t)(c0 + t) * C + j];
    }
  }

  // ------------------------------------------------------- key-block loop
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
  int before[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) before[nt] = 0;
  int maxtile = 0;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) maxtile = max(maxtile, tile_of<NT>(wv, nt));
  if (kstager) kload(0);
  for (int sb = 0; sb < nblk; ++sb) {
    Tin* kb = kbuf + (sb & 1) * P::KBUF;
    if (kstager) {
      kstore(kb);
      if (sb + 1 < nblk) kload(sb + 1);
    }
    __syncthreads();
    if (sb > maxtile) continue;
    const Tin* krow = kb + l32 * P::KRS + 8 * half;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int ti = tile_of<NT>(wv, nt);
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

  // outputs
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    if (rv[nt]) {
      Tout* orow = Out + (size_t)(c0 + tr[nt]) * DV + cg * NC;
#pragma unroll
      for (int r = 0; r < 16; ++r) orow[out_row(r, lane)] = from_f32<Tout>(acc[nt][r]);
    }
  }
}

constexpr size_t kMaxLds = 160 * 1024;

// Largest lambda window (entries per token) that fits in LDS, or -1 if none does.
template <int DK, typename Tin>
static int readout_window(int C) {
  for (int lw : {32, 16, 8, 0})
    if (RO<DK, Tin>::smem_bytes(C, lw) <= kMaxLds) return lw;
  return -1;
}

template <int DK, int DV, typename Tin>
static hipError_t launch_readout_t(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C, p.nch);
  const int cs = seg * p.nch_seg;
  const int nchs = (p.nch < cs + p.nch_seg ? p.nch : cs + p.nch_seg) - cs;
  const long long grid = (long long)round_up(nh, 8) * nchs * (DV / NC);
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  const int lw = readout_window<DK, Tin>(a.desc.C);
  if (lw < 0) return hipErrorInvalidValue;
  const size_t shm = RO<DK, Tin>::smem_bytes(a.desc.C, lw);
  auto launch = [&](auto k) -> hipError_t {
    if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
        hipSuccess)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(NTHR), shm, s, a, w, p, seg, lw);
    return hipGetLastError();
  };
  if (a.out_dtype == DLA_F32) return launch(prefill_readout_kernel<DK, DV, Tin, float>);
  return launch(prefill_readout_kernel<DK, DV, Tin, bf16_t>);
}

template <int DK, int DV>
static hipError_t launch_readout_dims(const PrefillArgs& a, const SegPlan& p, int seg,
                                      hipStream_t s) {
  if (a.in_dtype == DLA_F32) return launch_readout_t<DK, DV, float>(a, p, seg, s);
  return launch_readout_t<DK, DV, bf16_t>(a, p, seg, s);
}

bool prefill_update_supported(const dla_cache_desc& d, dla_dtype in_dtype);

bool prefill_chunks_supported(const dla_cache_desc& d, dla_dtype in_dtype) {
  const bool f = in_dtype == DLA_F32;
  const int lw = d.d_k == 128 ? (f ? readout_window<128, float>(d.C) : readout_window<128, bf16_t>(d.C))
                              : (f ? readout_window<64, float>(d.C) : readout_window<64, bf16_t>(d.C));
  return lw >= 0 && prefill_update_supported(d, in_dtype);
}

hipError_t launch_prefill_readout(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s) {
  const int dk = a.desc.d_k, dv = a.desc.d_v;
  if (dk == 128 && dv == 128) return launch_readout_dims<128, 128>(a, p, seg, s);
  if (dk == 64 && dv == 64) return launch_readout_dims<64, 64>(a, p, seg, s);
  if (dk == 128 && dv == 64) return launch_readout_dims<128, 64>(a, p, seg, s);
  return launch_readout_dims<64, 128>(a, p, seg, s);
}

}  // namespace dla
