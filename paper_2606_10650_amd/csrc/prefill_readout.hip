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
//     its death token is later than t (a state merged away is weighted as the
//     state that absorbed it).  The tile S~_j^T Q^T (32 columns x 32 tokens,
//     K = d_k) is an MFMA chain; each lane owns one token of a tile, so the
//     weight is a per-lane scalar applied to the chain's result.  States are
//     streamed from the pool two per step through an LDS ring of state pairs,
//     loaded straight from memory into LDS a few steps ahead, with one barrier
//     per step; each wave reads a state's operand from LDS once for all of its
//     tiles.  The lambda entries of a state at the lane's tokens come the same
//     way into a small LDS ring, two steps ahead, and each lane forms the
//     weights of its own tokens.
//   * intra-chunk part: (Q K^T (.) M) V with M[t][s] = [s <= t] exp(G_t - G_s)
//     lambda[t][slot_t(s)] over the chunk's own keys.  The keys pass through
//     an LDS ring of 32-token blocks, KU blocks per barrier, requested one
//     barrier ahead.  slot_t(s) is uniform over a block unless a live state
//     leader starts inside it, so lambda is read once per (token, block) in the
//     common case, from a window of each token's lambda row staged in LDS.
// Workgroups are dealt to the 8 XCDs round-robin by id; the mapping puts the
// column groups and neighbouring chunks of one head on one XCD, so the chunk's
// queries, keys and lambda rows, and the state copies that neighbouring chunks
// share, are read from HBM once per L2.
#include <type_traits>

#include "prefill_chunk.h"

namespace dla {

// Readout weights of 1 for every chronological position, read in place of a
// missing lambda row (C <= 1024).
struct OnesTable {
  uint16_t b[1024];  // bfloat16 1.0
  float f[1024];
};
constexpr OnesTable make_ones() {
  OnesTable t{};
  for (int i = 0; i < 1024; ++i) {
    t.b[i] = 0x3F80u;
    t.f[i] = 1.f;
  }
  return t;
}
__device__ const OnesTable kOnes = make_ones();
template <typename Tin>
__device__ __forceinline__ const Tin* ones_row() {
  if constexpr (sizeof(Tin) == 2)
    return reinterpret_cast<const Tin*>(kOnes.b);
  else
    return reinterpret_cast<const Tin*>(kOnes.f);
}

template <int DK, typename Tin>
struct RO : ChunkP<DK, Tin> {
  using B = ChunkP<DK, Tin>;
  // 16-bit operands of the next state are read from LDS into registers while
  // the MFMA chains of the current state run (float32 operands take twice the
  // registers and are read at the start of their own state)
  static constexpr bool PREF = B::E == 2;
  static constexpr int PF = PREF ? 1 : 0;
  // inter phase: state ring of NPAIR steps of two states (four for 16-bit
  // inputs, two for float32 inputs, whose slices are twice the size); a
  // step's slices are requested LEAD steps ahead
  static constexpr int NPAIR = B::E == 2 ? 4 : 2;
  static constexpr int NSLOT = 2 * NPAIR;
  static constexpr int LEAD = NPAIR - 1;
  // then the lambda ring: NLAM states x waves x 64 lanes, one dword per lane
  // (a 16-bit entry lands zero-extended); lane l holds the entry of the token
  // of tile l / 32, column l % 32.  A step's entries are requested LAM_D steps
  // ahead.
  static constexpr int LAM_D = LEAD - PF;
  static constexpr int NLAM = 2 * (LAM_D + 1);
  static constexpr size_t RING_BYTES = NSLOT * (size_t)B::SLICE16 * 16;
  static constexpr size_t WRING_BYTES = (size_t)NLAM * RWAVE * 64 * 4;
  static constexpr size_t INTER_BYTES = RING_BYTES + WRING_BYTES;
  // intra phase: key ring, and the lambda window, which is written before the
  // inter phase and so lies past both the key ring and the inter region
  static constexpr int KU = B::E == 2 ? 4 : 2;  // key blocks per barrier
  static constexpr int KSLOT = 2 * KU;
  static constexpr size_t KRING_BYTES = (KSLOT * (size_t)B::KBUF * B::E + 15) / 16 * 16;
  static constexpr size_t WIN_OFF = KRING_BYTES > INTER_BYTES ? KRING_BYTES : INTER_BYTES;
  __host__ __device__ static size_t region_bytes(int lw) {
    return round_up(WIN_OFF + (size_t)B::RL * (lw > 0 ? lw + 1 : 0) * B::E, 16);
  }
  static size_t smem_bytes(int C, int lw) {
    size_t off = region_bytes(lw);
    off += (size_t)NC * B::VTS * B::E;  // sVt
    off = round_up(off, 16);
    off += (size_t)B::RL * 4 * 7;  // sGc sRf sBf sDeath sLeadU sLeadD sAold
    off += (size_t)(C + 8) * 4 * 3;      // sSf, sObj, sDt (padded past the last state)
    return round_up(off, 16);
  }
};

// Token tile of wave wv: tiles come in mirrored pairs, wave p owning tiles
// 2 RWAVE q + p and 2 RWAVE q + 2 RWAVE - 1 - p of pair q, so every wave has
// the same causal intra-chunk work, and at every key block the same number of
// tiles still to serve.
template <int NT>
__device__ __forceinline__ int tile_of(int wv, int nt) {
  const int base = 2 * RWAVE * (nt >> 1);
  return (nt & 1) ? base + 2 * RWAVE - 1 - wv : base + wv;
}

template <int DK, int DV, typename Tin, typename Tout>
__global__ __launch_bounds__(RTHR) void prefill_readout_kernel(PrefillArgs a, PrefillWS w,
                                                               SegPlan plan, int seg, int lw) {
  if (!cache_matches(a.cache, a.desc)) return;  // refused call (see the prep kernel)
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using P = RO<DK, Tin>;
  constexpr int NT = P::NT;
  constexpr int NCG = DV / NC;
  constexpr int KS = P::KS;
  constexpr int RL = P::RL;
  constexpr int EPP = P::EPP;
  const int nh = a.desc.B * a.desc.H;
  int cs, ce;
  seg_range(plan, seg, &cs, &ce);
  const int nchs = ce - cs;
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
  // inter phase
  u32x4* ring = reinterpret_cast<u32x4*>(smem);                   // NSLOT state slices
  // intra phase (same bytes)
  Tin* kring = reinterpret_cast<Tin*>(smem);                      // KSLOT x [32][KRS] keys
  Tin* sLamW = reinterpret_cast<Tin*>(smem + P::WIN_OFF);         // [RL][lw + 1] lambda
  const int lws = lw + 1;
  const size_t rgn = P::region_bytes(lw);
  Tin* sVt = reinterpret_cast<Tin*>(smem + rgn);                  // [NC][VTS] values
  float* sGc = reinterpret_cast<float*>(smem + round_up(rgn + (size_t)NC * P::VTS * P::E, 16));
  float* sRf = sGc + RL;                            // exp(G_t - G_ref)
  float* sBf = sRf + RL;                            // exp(G_blockend - G_s)
  int32_t* sDeath = reinterpret_cast<int32_t*>(sBf + RL);
  int32_t* sLeadU = sDeath + RL;  // in-chunk leaders: position in the chunk
  int32_t* sLeadD = sLeadU + RL;  //                   death token
  int32_t* sAold = sLeadD + RL;   // old states alive at each token of the chunk
  float* sSf = reinterpret_cast<float*>(sAold + RL);  // exp(G_ref - F_j); 0 for j >= m
  int32_t* sObj = reinterpret_cast<int32_t*>(sSf + C + 8);
  int32_t* sDt = sObj + C + 8;
  __shared__ int sCnt[2];
  __shared__ int sBlk[RL / 32 + 1];
  __shared__ int sWsum[RWAVE];

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

  // ------------------------------------------------ set-up: every load first
  const char* lst = list_at(w, h, c, plan.nch);
  const ListEntry* ent = reinterpret_cast<const ListEntry*>(lst + 16);
  constexpr int EPT = 1024 / RTHR;  // list entries per thread (C <= 1024)
  ListEntry le[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int j = tid + RTHR * u;
    if (j < C) le[u] = ent[j];  // entries past m are read but not used
  }
  const int m = min(max(*reinterpret_cast<const int32_t*>(lst), 0), C);
  const double Gref = (c0 == 0) ? *init_at(w, h, C).G0 : Gtok[c0 - 1];
  constexpr int TPT = (RL + RTHR - 1) / RTHR;
  double gi_[TPT], gb_[TPT];
  int dth_[TPT];
#pragma unroll
  for (int u = 0; u < TPT; ++u) {
    const int t = tid + RTHR * u;
    const int ic = min(t, nrow - 1);
    const int be = min(32 * (t >> 5) + 31, nrow - 1);
    gi_[u] = Gtok[c0 + ic];
    gb_[u] = Gtok[c0 + be];
    dth_[u] = (t < nrow) ? death[c0 + t] : -1;
  }
  constexpr int PER_ROW16 = NC * P::E / 16;
  constexpr int VPT = RL * PER_ROW16 / RTHR;
  u32x4 vp_[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int idx = tid + RTHR * u;
    const int r = idx / PER_ROW16, p = idx % PER_ROW16;
    const u32x4 z = {0u, 0u, 0u, 0u};
    vp_[u] = (r < nrow)
                 ? *reinterpret_cast<const u32x4*>(Vin + (size_t)(c0 + r) * DV + cg * NC + p * EPP)
                 : z;
  }
  int tr[NT];
  bool rv[NT];
  FT qf[NT][KS];
  f32x16 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    tr[nt] = 32 * tile_of<NT>(wv, nt) + l32;
    rv[nt] = tr[nt] < nrow;
    acc[nt] = zero16();
    const Tin* qrow = Qin + (size_t)(c0 + (rv[nt] ? tr[nt] : 0)) * DK;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[nt][ks] = rv[nt] ? FR::load(qrow + 16 * ks + 8 * half) : FR::zero();
  }
  // ... then the LDS tables
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int j = tid + RTHR * u;
    if (j < m) {
      sObj[j] = min(max(le[u].obj, 0), plan.P_cap - 1);
      sDt[j] = le[u].dt;
      sSf[j] = __expf((float)(Gref - le[u].F));
    } else if (j < C + 8) {
      sObj[j] = 0;
      sDt[j] = 0;
      sSf[j] = 0.f;
    }
  }
  for (int j = max(C, RTHR * EPT) + tid; j < C + 8; j += RTHR) {  // padding past RTHR * EPT
    sObj[j] = 0;
    sDt[j] = 0;
    sSf[j] = 0.f;
  }
#pragma unroll
  for (int u = 0; u < TPT; ++u) {
    const int t = tid + RTHR * u;
    if (t < RL) {
      sAold[t] = 0;                     // death counts first (see below)
      sGc[t] = (float)(gi_[u] - Gref);  // G_t - G_ref
      sRf[t] = __expf((float)(gi_[u] - Gref));
      sBf[t] = __expf((float)(gb_[u] - gi_[u]));
      sDeath[t] = dth_[u];
    }
  }
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int idx = tid + RTHR * u;
    const int r = idx / PER_ROW16, p = idx % PER_ROW16;
#pragma unroll
    for (int e = 0; e < EPP; ++e) sVt[(p * EPP + e) * P::VTS + r] = piece_elem<Tin>(vp_[u], e);
  }
  __syncthreads();
  // The inter phase's first requests (the lambda entries of states 0 .. 5 at
  // the lane's tokens, and the pool slices of states 0 .. 5) go out as soon as
  // the list tables are in LDS, so that their latency overlaps the rest of the
  // set-up.  Each lane forms the weights of its own tile tokens.
  // lambda rows: a buffer over the chunk's lambda rows (wave-uniform), the
  // row of tile token nt at byte offset loff[nt]; without lambda, the ones table
  const __amdgpu_buffer_rsrc_t lrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<Tin*>(Lin ? Lin + (size_t)c0 * C : ones_row<Tin>()), (short)0,
      Lin ? nrow * C * P::E : 1024 * P::E, 0x00020000);
  // The lane's lambda token: the token of tile min(l / 32, NT - 1), column
  // l % 32; its row at byte offset loff.  cm: live states up to the last state
  // whose entry was requested, minus one (states past the list read a death
  // token of 0 from the padding, so they never count).
  const int ltile = min(half, NT - 1);
  const int ltok = 32 * tile_of<NT>(wv, ltile) + l32;
  const int loff = Lin ? (ltok < nrow ? ltok : 0) * C * P::E : 0;
  const int ltokc = c0 + ltok;
  int cm = -1;
  // Lambda entries of state j, requested in state order straight into the
  // wave's slot of the LDS lambda ring (a wave reads back only what its own
  // request wrote).
  char* sLam = reinterpret_cast<char*>(smem) + P::RING_BYTES;
  auto lam_slot = [&](int j) __attribute__((always_inline)) -> char* {
    return sLam + (size_t)((j % P::NLAM) * RWAVE + wv) * 64 * 4;
  };
  auto lam_dt = [&](int j) __attribute__((always_inline)) -> int { return sDt[min(j, C + 7)]; };
  // (dt: the death token of state j, lam_dt(j))
  auto lam_dma = [&](int j, int dt) __attribute__((always_inline)) {
    cm += (int)(dt > ltokc);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        lrs, (__attribute__((address_space(3))) void*)lam_slot(j), P::E,
        loff + max(cm, 0) * P::E, 0, 0, 0);
  };
  // the entry of state j at the lane's token of tile nt
  auto lam_get = [&](int j, int nt) __attribute__((always_inline)) -> float {
    return to_f32(*reinterpret_cast<const Tin*>(lam_slot(j) + (32 * nt + l32) * 4));
  };
  constexpr int SL16 = P::SLICE16;
  constexpr int V16 = (SL16 + RTHR - 1) / RTHR;
  constexpr int LEAD = P::LEAD;  // steps between a slice's request and its chains
  // the pool slices of this head and column group: object obj at
  // pool_h + obj * NCG * SLICE (the object index is wave-uniform, so the
  // address is formed in scalar registers)
  const Tin* pool_h = pool_slice<Tin>(w.pool, h, plan.P_cap, 0, cg, NCG, P::SLICE);
  // pool object of state j (the last state's past the list)
  auto obj_of = [&](int j) __attribute__((always_inline)) -> int { return sObj[min(j, m - 1)]; };
  // slices of pool objects o0, o1 into ring pair pr, straight from memory into
  // LDS (each lane's 16 bytes land at the wave's base plus 16 bytes per lane)
  auto dma2 = [&](int pr, int o0, int o1) __attribute__((always_inline)) {
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int obj = __builtin_amdgcn_readfirstlane(s2 ? o1 : o0);
      const __amdgpu_buffer_rsrc_t src = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<Tin*>(pool_h + (size_t)obj * (NCG * P::SLICE)), (short)0, SL16 * 16,
          0x00020000);
#pragma unroll
      for (int u = 0; u < V16; ++u) {
        const int pi = tid + RTHR * u;
        // (SL16 is a multiple of 64, so the test is uniform over a wave)
        if (SL16 % RTHR == 0 || pi < SL16)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              src, (__attribute__((address_space(3))) void*)(ring + (pr * 2 + s2) * SL16 + (pi - lane)),
              16, pi * 16, 0, 0, 0);
      }
    }
  };
  if (m > 0) {
#pragma unroll
    for (int j = 0; j < 2 * P::LAM_D; ++j) lam_dma(j, lam_dt(j));
#pragma unroll
    for (int J = 0; J < LEAD; ++J) dma2(J, obj_of(2 * J), obj_of(2 * J + 1));
  }
  // old states alive at each token: m minus the states of the list whose death
  // token is at or before it (a state lives while its death token is later)
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int j = tid + RTHR * u;
    if (j < m) {
      const int d = le[u].dt - c0;
      if (d >= 0 && d < RL) atomicAdd(&sAold[d], 1);
    }
  }
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
  {
    // inclusive prefix of the death counts over the chunk's tokens
    constexpr int TPW = (RL + RTHR - 1) / RTHR;  // tokens per thread (1)
    static_assert(TPW == 1, "one token per thread");
    int hv = (tid < RL) ? sAold[tid] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(hv, o, 64);
      if (lane >= o) hv += y;
    }
    if (lane == 63) sWsum[wv] = hv;
    __syncthreads();
    int base = 0;
    for (int w2 = 0; w2 < wv; ++w2) base += sWsum[w2];
    if (tid < RL) sAold[tid] = m - (base + hv);
    __syncthreads();
  }
  // lambda window of every token: lambda[t][Aold_t - 1 + x] for x < lw, the
  // weights of the states that hold the chunk's own tokens.  Consecutive lanes
  // read consecutive entries of a row; every load is issued before the stores.
  // (The window lies past both the key ring and the inter region.)
  if (Lin && lw > 0) {
    // (lw is a power of two)
    const int lwl = __builtin_ctz((unsigned)lw);
    constexpr int WPT = RL * 32 / RTHR;
    Tin lv[WPT];
    const int nwin = nrow * lw;
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int idx = tid + RTHR * u;
      if (idx < nwin) {
        const int t = idx >> lwl, x = idx & (lw - 1);
        lv[u] = Lin[(size_t)(c0 + t) * C + min(max(sAold[t] - 1 + x, 0), C - 1)];
      }
    }
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int idx = tid + RTHR * u;
      if (idx < nwin) {
        const int t = idx >> lwl, x = idx & (lw - 1);
        sLamW[t * lws + x] = lv[u];
      }
    }
  }
  // first leader of each 32-token block (the leader list is in token order)
  for (int sb = tid; sb <= RL / 32; sb += RTHR) {
    int lo = 0, hi = nLead;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sLeadU[mid] < 32 * sb) lo = mid + 1; else hi = mid;
    }
    sBlk[sb] = lo;
  }

  // ------------------------------------------------ inter-chunk readout
  // Ring pair p of the LDS (NPAIR pairs) holds states 2J and 2J+1 for every
  // step J = p mod NPAIR.  Step J starts with a barrier and runs the MFMA
  // chains of states 2J and 2J+1 with their operands in registers; meanwhile
  // the operand of the state after each is read from LDS (for 16-bit inputs),
  // and the step requests, straight from memory into LDS, the slices of step
  // J + LEAD (into the pair that step J - 1 read, before this barrier) and the
  // lambda entries of step J + LAM_D.  Each lane forms the weights of its own
  // tokens from those entries.  Steps past the last state have sSf = 0.
  // The weight of state j at token t is lambda[t][x] exp(G_t - F_j), x = (live
  // states up to j) - 1 (a state merged away at or before t is weighted as the
  // live state that absorbed it).
  if (m > 0) {
    // The tiles are staggered: after the MFMA chain of tile k of state j comes
    // the weighting of tile k - 1 (of state j - 1 for k = 0), so every FMA runs
    // while the matrix core works on an independent chain.
    f32x16 f[NT];
    float wP = 0.f;  // weight of the last tile's pending chain result
    float rf[NT];    // exp(G_t - G_ref) of the lane's tile tokens
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f[nt] = zero16();
      rf[nt] = rv[nt] ? sRf[tr[nt]] : 0.f;
    }
    // sched_group_barrier masks: 0x008 MFMA, 0x002 VALU, 0x100 LDS read
    auto interleave = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
      }
    };
    // a wave's operand of the state slice at A
    auto opload = [&](const Tin* A, FT (&sa)[KS]) __attribute__((always_inline)) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) sa[ks] = FR::load(A + ((ks * 2 + half) * 32 + l32) * 8);
    };
    // The chains of state j with operand sa (slice Ac).  With PREF the operand
    // of the state after j (slice An) is read into sn meanwhile.  mid() runs
    // between the chains of the first and the second tile.
    auto sub = [&](int j, FT (&sa)[KS], const Tin* Ac, const Tin* An, FT (&sn)[KS],
                   auto&& mid) __attribute__((always_inline)) {
      // LDS reads first; their values are needed only after the first chain
      const float sf = sSf[j];
      float lv[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) lv[nt] = lam_get(j, nt);
      if constexpr (P::PREF)
        opload(An, sn);
      else
        opload(Ac, sa);
      float wg[NT];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        // f[nt] held tile nt of the previous state, weighted one tile ago; the
        // chain's MFMAs alternate with the FMAs of that weighting
        f[nt] = zero16();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) FR::mma(f[nt], sa[ks], qf[nt][ks]);
        const int pt = nt == 0 ? NT - 1 : nt - 1;
        const float wq = nt == 0 ? wP : wg[nt - 1];
        if (NT > 1 || nt > 0) {
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[pt][r] += wq * f[pt][r];
        }
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        if (nt == 0) {
#pragma unroll
          for (int n2 = 0; n2 < NT; ++n2) wg[n2] = lv[n2] * rf[n2] * sf;
          mid();
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if constexpr (NT == 1) {
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[0][r] += wg[0] * f[0][r];
      }
      wP = wg[NT - 1];
    };
    auto nothing = []() __attribute__((always_inline)) {};
    FT saX[KS], saY[KS];
    // Before the barrier of step J the slices of step J (and of step J+1, whose
    // first operand the step reads ahead with PREF) and the lambda entries of
    // step J must be in LDS.  Step J' requests, between the first and second
    // chains of its first state, the lambda entries of step J'+LAM_D and then
    // the slices of step J'+LEAD; so the wave waits for its requests up to
    // the slices of step J+PF-LEAD, and the later ones stay in flight: per
    // step two lambda requests and 2 V16 slice pieces.  The wave's LDS reads
    // are complete before the barrier, so a pair or lambda slot is rewritten
    // only after it was read.
    constexpr int VM_AFTER = (LEAD - 1 - P::PF) * (2 + 2 * V16);
    static_assert(VM_AFTER >= 0 && VM_AFTER < 64, "vmcnt range");
    static_assert(P::LAM_D >= LEAD - P::PF, "lambda requests precede the slices waited for");
    constexpr int WAIT = (VM_AFTER & 15) | (7 << 4) | (0 << 8) | ((VM_AFTER >> 4) << 14);
    __syncthreads();  // (waits for every request: the first LEAD steps' slices are in LDS)
    if constexpr (P::PREF) opload(reinterpret_cast<const Tin*>(ring), saX);
    for (int J = 0; 2 * J < m; ++J) {
      if (J > 0) {
        __builtin_amdgcn_s_waitcnt(WAIT);
        __builtin_amdgcn_s_barrier();
      }
      __builtin_amdgcn_sched_barrier(0);
      const Tin* A0 = reinterpret_cast<const Tin*>(ring + (J % P::NPAIR) * 2 * SL16);
      const Tin* A2 = reinterpret_cast<const Tin*>(ring + ((J + 1) % P::NPAIR) * 2 * SL16);
      const int jl = 2 * (J + P::LAM_D);
      const int dt0 = lam_dt(jl), dt1 = lam_dt(jl + 1);
      // (the object numbers are read here, so that the requests below need not
      // wait for an LDS read behind the operand reads)
      const int ob0 = obj_of(2 * (J + LEAD)), ob1 = obj_of(2 * (J + LEAD) + 1);
      sub(2 * J, saX, A0, A0 + P::SLICE, saY, [&]() __attribute__((always_inline)) {
        lam_dma(jl, dt0);
        lam_dma(jl + 1, dt1);
        dma2((J + LEAD) % P::NPAIR, ob0, ob1);
      });
      __builtin_amdgcn_sched_barrier(0);
      sub(2 * J + 1, saY, A0 + P::SLICE, A2, saX, nothing);
    }
    if constexpr (NT > 1) {
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[NT - 1][r] += wP * f[NT - 1][r];
    }
  }
  __syncthreads();  // the state ring and the lambda blocks are no longer read

  // The chunk's keys pass through a 2 KU-slot LDS ring, 32 tokens per block;
  // every thread loads its 16-byte pieces of a block (consecutive threads,
  // consecutive pieces of a row).
  constexpr int KPT = (32 * P::KROW16 + RTHR - 1) / RTHR;
  auto kload = [&](int sb, u32x4 (&kr)[KPT]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      const int pi = tid + RTHR * u;
      const int r = pi / P::KROW16, pc = pi % P::KROW16;
      const int tok = 32 * sb + r;
      const u32x4 z = {0u, 0u, 0u, 0u};
      kr[u] = (r < 32 && tok < nrow)
                  ? *reinterpret_cast<const u32x4*>(Kin + (size_t)(c0 + tok) * DK + pc * EPP)
                  : z;
    }
  };
  auto kstore = [&](int sb, const u32x4 (&kr)[KPT]) __attribute__((always_inline)) {
    Tin* kb = kring + (sb % P::KSLOT) * P::KBUF;
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      const int pi = tid + RTHR * u;
      const int r = pi / P::KROW16, pc = pi % P::KROW16;
      if (r < 32) *reinterpret_cast<u32x4*>(kb + r * P::KRS + pc * EPP) = kr[u];
    }
  };
  u32x4 kq[P::KU][KPT];
  // store blocks sb0 .. sb0 + KU - 1 (those in the chunk) from kq
  auto kput = [&](int sb0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < P::KU; ++u)
      if (sb0 + u < nblk) kstore(sb0 + u, kq[u]);
  };
  // the first KU blocks
#pragma unroll
  for (int u = 0; u < P::KU; ++u)
    if (u < nblk) kload(u, kq[u]);

  // ------------------------------------------------------- key-block loop
  int before[NT];  // live in-chunk leaders in the blocks before, at each tile token
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) before[nt] = 0;
  float gtok[NT];   // G_t - G_ref of each tile token
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) gtok[nt] = rv[nt] ? sGc[tr[nt]] : 0.f;
  // Key block sb against the active tiles N0 .. N0 + NA - 1 of this wave (a
  // uniform set: a tile is active while the block does not start after it).
  // The key operand, the value operand, the rows' decays and the block's
  // leaders are read once for all of them, and the tiles' MFMA chains are
  // interleaved.
  auto blockT = [&](auto n0_c, auto na_c, int sb) __attribute__((always_inline)) {
    constexpr int N0 = decltype(n0_c)::value;
    constexpr int NA = decltype(na_c)::value;
    const Tin* krow = kring + (sb % P::KSLOT) * P::KBUF + l32 * P::KRS + 8 * half;
    FT ka[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) ka[ks] = FR::load(krow + 16 * ks);
    // P^T tiles: rows = the block's key tokens, columns = the tile's tokens
    f32x16 pt[NA];
#pragma unroll
    for (int i = 0; i < NA; ++i) pt[i] = zero16();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int i = 0; i < NA; ++i) FR::mma(pt[i], ka[ks], qf[N0 + i][ks]);
    // values of the block's tokens in the permuted k order of the weights:
    // element e of half h <-> token 16 st + 8 (e / 4) + 4 h + e % 4
    FT va[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const Tin* vp = sVt + l32 * P::VTS + 32 * sb + 16 * st + 4 * half;
      va[st] = load_4x2<Tin>(vp, vp + 8);
    }
    float bf[16];  // exp(G_blockend - G_s) of each accumulator row
#pragma unroll
    for (int r = 0; r < 16; ++r) bf[r] = sBf[32 * sb + out_row(r, lane)];
    const float gend = sGc[32 * sb + 31];
    // leaders inside block sb that are live at each tile token, as bit masks
    uint32_t word[NA];
#pragma unroll
    for (int i = 0; i < NA; ++i) word[i] = 0u;
    for (int k2 = sBlk[sb]; k2 < sBlk[sb + 1]; ++k2) {
      const int ldd = sLeadD[k2];
      const uint32_t bit = 1u << (sLeadU[k2] & 31);
#pragma unroll
      for (int i = 0; i < NA; ++i)
        if (ldd > c0 + tr[N0 + i]) word[i] |= bit;
    }
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int nt = N0 + i;
      const int ti = tile_of<NT>(wv, nt);
      const int trn = tr[nt];
      const int Aold = sAold[trn];  // old states alive at the token
      const Tin* lrow = Lin ? Lin + (size_t)(c0 + (rv[nt] ? trn : 0)) * C : nullptr;
      const Tin* lwin = sLamW + trn * lws;
      // weight of the state at window position x (x = live in-chunk leaders up
      // to the key token): from the window, else from the lambda row
      // (the window read is unconditional and the row read separate, so the
      // two never merge into one generic-address load)
      auto lam_at = [&](int x) __attribute__((always_inline)) -> float {
        if (!lrow || !rv[nt]) return 1.f;
        float v = lw > 0 ? to_f32(lwin[min(x, lw - 1)]) : 0.f;
        if (x >= lw) v = to_f32(lrow[min(max(Aold - 1 + x, 0), C - 1)]);
        return v;
      };
      // live leaders at key rows <= so = rb + 4 half of the block, with rb =
      // 8 (r / 4) + r % 4 a constant per accumulator element: ww holds the mask
      // shifted so that the count is a popcount under a constant mask
      const uint32_t ww = half ? word[i] : (word[i] << 4);
      auto upto = [&](int r) __attribute__((always_inline)) -> int {
        const int rb = 8 * (r >> 2) + (r & 3);
        return __popc(ww & (0xFFFFFFFFu >> (27 - rb)));
      };
      // lambda is uniform over the block unless a live leader starts after its
      // first row
      const bool uni = (word[i] & ~1u) == 0u;
      const float lu = uni ? lam_at(before[nt] + (int)(word[i] & 1u)) : 0.f;
      if (sb < ti) {
        // the whole block precedes the token: decay exp(G_t - G_end) per lane
        // times exp(G_end - G_s) per row (both at most 1)
        const float f1 = rv[nt] ? __expf(gtok[nt] - gend) : 0.f;
        if (uni) {
          const float fw = f1 * lu;
#pragma unroll
          for (int r = 0; r < 16; ++r) pt[i][r] *= fw * bf[r];
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r) pt[i][r] *= f1 * lam_at(before[nt] + upto(r)) * bf[r];
        }
      } else {
        // the token's own block: causal mask, decay exp(G_t - G_s) per element
        // (the mask selects zero rather than multiplying by it, so that a
        // non-finite key later in the block cannot reach an earlier token)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int s = 32 * sb + out_row(r, lane);
          const float lr = uni ? lu : lam_at(before[nt] + upto(r));
          pt[i][r] = (rv[nt] && s <= trn) ? pt[i][r] * (lr * __expf(gtok[nt] - sGc[s])) : 0.f;
        }
      }
      before[nt] += __popc(word[i]);
    }
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        float pw[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) pw[e] = pt[i][8 * st + e];
        FR::mma(acc[N0 + i], va[st], FR::from_floats(pw));
      }
  };
  // the active tiles at block sb: tile nt is active while sb <= its index and
  // it starts inside the chunk; tiles are in increasing order
  auto block = [&](int sb) __attribute__((always_inline)) {
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    const int t0 = tile_of<NT>(wv, 0);
    const bool a0 = sb <= t0 && 32 * t0 < nrow;
    if constexpr (NT == 2) {
      const int t1 = tile_of<NT>(wv, 1);
      const bool a1 = sb <= t1 && 32 * t1 < nrow;
      if (a0 && a1)
        blockT(I0{}, I2{}, sb);
      else if (a1)
        blockT(I1{}, I1{}, sb);
      else if (a0)
        blockT(I0{}, I1{}, sb);
    } else {
      if (a0) blockT(I0{}, I1{}, sb);
    }
  };
  // Each iteration requests the next KU blocks at its start and stores them at
  // its end, after the arithmetic of its own KU blocks: no register buffer
  // lives across the loop's back-edge, and the loads stay in flight over KU
  // blocks of work.  The stores go to the slots of the previous iteration's
  // blocks, whose readers all passed this iteration's barrier.
  kput(0);
  for (int sb0 = 0; sb0 < nblk; sb0 += P::KU) {
#pragma unroll
    for (int u = 0; u < P::KU; ++u)
      if (sb0 + P::KU + u < nblk) kload(sb0 + P::KU + u, kq[u]);
    __syncthreads();
    for (int u = 0; u < P::KU && sb0 + u < nblk; ++u) block(sb0 + u);
    kput(sb0 + P::KU);
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
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C, a.desc.d_k * a.desc.d_v, p.nch);
  int cs, ce;
  seg_range(p, seg, &cs, &ce);
  const int nchs = ce - cs;
  const long long grid = (long long)round_up(nh, 8) * nchs * (DV / NC);
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  const int lw = readout_window<DK, Tin>(a.desc.C);
  if (lw < 0) return hipErrorInvalidValue;
  const size_t shm = RO<DK, Tin>::smem_bytes(a.desc.C, lw);
  auto launch = [&](auto k) -> hipError_t {
    if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
        hipSuccess)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(RTHR), shm, s, a, w, p, seg, lw);
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
bool prefill_scan_supported(const dla_cache_desc& d, dla_dtype in_dtype);

bool prefill_chunks_supported(const dla_cache_desc& d, dla_dtype in_dtype) {
  const bool f = in_dtype == DLA_F32;
  const int lw = d.d_k == 128 ? (f ? readout_window<128, float>(d.C) : readout_window<128, bf16_t>(d.C))
                              : (f ? readout_window<64, float>(d.C) : readout_window<64, bf16_t>(d.C));
  return lw >= 0 && prefill_update_supported(d, in_dtype) && prefill_scan_supported(d, in_dtype);
}

hipError_t launch_prefill_readout(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s) {
  const int dk = a.desc.d_k, dv = a.desc.d_v;
  if (dk == 128 && dv == 128) return launch_readout_dims<128, 128>(a, p, seg, s);
  if (dk == 64 && dv == 64) return launch_readout_dims<64, 64>(a, p, seg, s);
  if (dk == 128 && dv == 64) return launch_readout_dims<128, 64>(a, p, seg, s);
  return launch_readout_dims<64, 128>(a, p, seg, s);
}

}  // namespace dla
