// Prefill, stage 3: state-cache maintenance over the chunks of one segment.
//
// The decisions of the scan (boundaries, and the death token of every state
// leader: the token at which Alg. 2 merged its state into the left neighbour)
// fix which states exist after every token.  This stage walks the chunks of a
// segment in order, one workgroup of 8 waves per (head, 32 value columns):
//   * at each chunk start it records the chunk's state list (pool object,
//     death token and frame of every state present), which the readout stage
//     consumes;
//   * the states alive after the chunk are rebuilt from the old states they
//     absorbed (Alg. 2 merges: sums of adjacent states) plus, for states that
//     hold tokens of the chunk, sum_s exp(G_end - G_s) k_s v_s^T over their
//     consecutive token range (the update rule of Sec. 3.1 with the gated
//     decay of every state).  K~ = exp(G_end - G_s) k_s is split into three
//     bf16 terms so the MFMA product is exact to float32 rounding.  Each
//     rebuilt state is stored in frame G_end: the float32 master in its cache
//     slot, and a copy in MFMA operand order as a new pool object.  States
//     that nothing touched keep their slot, frame and object (lazy decay).
// Slots of states merged away, and free slots, are reused by new states; the
// per-head permutation maps chronological states to slots.
#include "prefill_chunk.h"

namespace dla {

template <int DK, typename Tin>
static size_t update_smem_bytes(int C) {
  using P = ChunkP<DK, Tin>;
  size_t off = (size_t)NC * P::VTS * P::E;   // sVt
  off += 2 * (size_t)P::KBUF * P::E;         // key blocks
  off = round_up(off, 16);
  off += (size_t)P::RL * 4 * 4;              // sDecE sDeath sLeadU sLeadD
  off += (size_t)C * 8;                      // sF
  off += (size_t)C * 4 * 14 + 64;            // int arrays, reduction scratch
  return round_up(off, 16);
}

template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(NTHR) void prefill_update_kernel(PrefillArgs a, PrefillWS w,
                                                              SegPlan plan, int seg) {
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using P = ChunkP<DK, Tin>;
  constexpr int D = DK * DV;
  constexpr int NCG = DV / NC;
  constexpr int RL = P::RL;
  const int nh = a.desc.B * a.desc.H;
  // XCD-aware mapping: workgroups are dealt to the 8 XCDs round-robin by id, so
  // the column groups of one head get the same id modulo 8 and share an L2 for
  // the chunk's keys, which all of them read.
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
  const int cs = seg * plan.nch_seg;
  const int ce = min(plan.nch, cs + plan.nch_seg);
  const bool last_seg = seg == plan.nseg - 1;
  const bool copies = plan.P_cap > 0;  // pool objects for a readout stage

  extern __shared__ __align__(16) char smem[];
  Tin* sVt = reinterpret_cast<Tin*>(smem);  // [NC][VTS] values, transposed
  Tin* kbuf = sVt + NC * P::VTS;            // 2 key blocks of KBUF elements
  float* sDecE = reinterpret_cast<float*>(
      smem + round_up(((size_t)NC * P::VTS + 2 * (size_t)P::KBUF) * P::E, 16));  // exp(G_end - G_s)
  int32_t* sDeath = reinterpret_cast<int32_t*>(sDecE + RL);
  int32_t* sLeadU = sDeath + RL;  // in-chunk leaders: position in the chunk
  int32_t* sLeadD = sLeadU + RL;  //                   death token
  double* sF = reinterpret_cast<double*>(sLeadD + RL);
  int32_t* sPerm = reinterpret_cast<int32_t*>(sF + C);
  int32_t* sLead = sPerm + C;
  int32_t* sDt = sLead + C;
  int32_t* sObj = sDt + C;
  int32_t* eJa = sObj + C;
  int32_t* eJb = eJa + C;
  int32_t* eR0 = eJb + C;
  int32_t* eR1 = eR0 + C;
  int32_t* ePhys = eR1 + C;
  int32_t* eLead = ePhys + C;
  int32_t* ePool = eLead + C;
  int32_t* eChg = ePool + C;
  int32_t* eObj = eChg + C;
  int32_t* eTmp = eObj + C;
  int32_t* red = eTmp + C;
  __shared__ int sCnt[2];

  InitView iv = init_at(w, h, C);
  CarryView cv = carry_at(w, h, C);
  const int m0 = min(max(*iv.m0, 0), C);
  int m;
  if (seg == 0) {
    m = m0;
    for (int j = tid; j < C; j += NTHR) {
      sPerm[j] = min(max(iv.perm0[j], 0), C - 1);
      sF[j] = iv.F0[j];
      sLead[j] = j - m0;
      sObj[j] = j;
    }
  } else {
    m = min(max(*cv.m, 0), C);
    for (int j = tid; j < C; j += NTHR) {
      sPerm[j] = min(max(cv.perm[j], 0), C - 1);
      sF[j] = cv.F[j];
      sLead[j] = cv.lead[j];
      sObj[j] = j;
    }
  }
  int next_obj = m;

  float* states = reinterpret_cast<float*>(a.cache + a.states_offset) + (size_t)h * C * D;
  const double* Gtok = w.Gtok + (size_t)h * T;
  const int32_t* death = w.death + (size_t)h * T;
  const Tin* Kin = static_cast<const Tin*>(a.k) + (size_t)h * T * DK;
  const Tin* Vin = static_cast<const Tin*>(a.v) + (size_t)h * T * DV;
  auto obj_slice = [&](int obj) -> Tin* {
    return pool_slice<Tin>(w.pool, h, plan.P_cap, obj, cg, NCG, P::SLICE);
  };

  // copies of the states present at the segment start
  __syncthreads();
  if (copies) {
    for (int j = 0; j < m; ++j) {
      const float* src = states + (size_t)sPerm[j] * D + cg * NC;
      Tin* dst = obj_slice(j);
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
  }

  // band of d_k rows owned by this wave; the waves form NWAVE / NBAND groups
  // and group 0 does the arithmetic
  constexpr int NBAND = DK / 32;
  const int ib = 32 * (wv % NBAND);
  const bool band = wv < NBAND;
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
  // store a band of a state: float32 master, and its copy when obj >= 0
  auto store_state = [&](const f32x16& acc16, int phys, int obj) __attribute__((always_inline)) {
    float* dst = states + (size_t)phys * D + cg * NC + l32;
#pragma unroll
    for (int r = 0; r < 16; ++r) dst[(size_t)(ib + out_row(r, lane)) * DV] = acc16[r];
    if (obj >= 0) {
      Tin* sh = obj_slice(obj);
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int ks = (ib >> 4) + (g4 >> 1);
        Tin* d4 = sh + ((ks * 2 + (g4 & 1)) * 32 + l32) * 8 + 4 * half;
#pragma unroll
        for (int q = 0; q < 4; ++q) d4[q] = from_f32<Tin>(acc16[4 * g4 + q]);
      }
    }
  };

  for (int c = cs; c < ce; ++c) {
    const int c0 = c * RL;
    const int nrow = min(RL, T - c0);
    const int c1 = c0 + nrow;
    const int nblk = (nrow + 31) >> 5;
    const double Gend = Gtok[c1 - 1];
    // copies of this chunk's rebuilt states are read by the next chunk of the
    // segment only
    const bool make_obj = copies && c + 1 < ce;
    __syncthreads();
    for (int i = tid; i < RL; i += NTHR) {
      sDecE[i] = (i < nrow) ? __expf((float)(Gend - Gtok[c0 + i])) : 0.f;
      sDeath[i] = (i < nrow) ? death[c0 + i] : -1;
    }
    for (int j = tid; j < m; j += NTHR) {
      const int ld = sLead[j];
      sDt[j] = (ld >= 0) ? death[ld] : iv.death0[ld + m0];
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
    // the chunk's state list, for the readout stage
    if (cg == 0 && copies) {
      char* lst = list_at(w, h, c, plan.nch);
      if (tid == 0) *reinterpret_cast<int32_t*>(lst) = m;
      ListEntry* ent = reinterpret_cast<ListEntry*>(lst + 16);
      for (int j = tid; j < m; j += NTHR) {
        ListEntry le;
        le.obj = sObj[j];
        le.dt = sDt[j];
        le.F = sF[j];
        ent[j] = le;
      }
    }
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
    // pool objects of the rebuilt states, in chronological order
    const int nchg = block_excl_count(ne, [&](int e) { return eChg[e] != 0; }, eTmp, red);
    // (next_obj + nchg <= P_cap: a segment starts with at most C objects and
    // each of its chunks but the last adds at most C)
    for (int e = tid; e < ne; e += NTHR)
      eObj[e] = (eChg[e] && make_obj && next_obj + eTmp[e] < plan.P_cap) ? next_obj + eTmp[e] : -1;
    __syncthreads();

    // ------------------------------- states changed by merges of old states only
    // (rebuilt first: they read old slots that new states may reuse)
    if (band) {
      for (int e = 0; e < nAO; ++e) {
        if (!eChg[e] || eR1[e] >= eR0[e]) continue;
        f32x16 u16 = zero16();
        add_old(u16, eJa[e], eJb[e], Gend);
        store_state(u16, ePhys[e], eObj[e]);
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
          store_state(uacc, ePhys[rc], eObj[rc]);
          uacc = zero16();
          ++rc;
          if (rc >= ne || eR0[rc] >= be) break;
        }
      }
    }
    __syncthreads();

    // bookkeeping for the next chunk
    {
      constexpr int PU = 1024 / NTHR;
      double f_[PU];
      int ld_[PU], ph_[PU], ob_[PU];
#pragma unroll
      for (int u = 0; u < PU; ++u) {
        const int e = tid + NTHR * u;
        if (e < ne) {
          f_[u] = eChg[e] ? Gend : sF[eJa[e]];
          ld_[u] = eLead[e];
          ph_[u] = ePhys[e];
          ob_[u] = eChg[e] ? eObj[e] : sObj[eJa[e]];
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
          sObj[e] = ob_[u];
        } else if (e < C) {
          sPerm[e] = ph_[u];
        }
      }
    }
    m = ne;
    next_obj += make_obj ? nchg : 0;
  }
  __syncthreads();

  if (cg == 0) {
    if (last_seg) {
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
    } else {
      for (int j = tid; j < C; j += NTHR) {
        cv.perm[j] = sPerm[j];
        cv.F[j] = sF[j];
        cv.lead[j] = sLead[j];
      }
      if (tid == 0) *cv.m = m;
    }
  }
}

template <int DK, int DV, typename Tin>
static hipError_t launch_update_t(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C, p.nch);
  const int grid = (int)round_up(nh, 8) * (DV / NC);
  const size_t shm = update_smem_bytes<DK, Tin>(a.desc.C);
  if (shm > 160 * 1024) return hipErrorInvalidValue;
  auto k = prefill_update_kernel<DK, DV, Tin>;
  if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
      hipSuccess)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3(grid), dim3(NTHR), shm, s, a, w, p, seg);
  return hipGetLastError();
}

template <int DK, int DV>
static hipError_t launch_update_dims(const PrefillArgs& a, const SegPlan& p, int seg,
                                     hipStream_t s) {
  if (a.in_dtype == DLA_F32) return launch_update_t<DK, DV, float>(a, p, seg, s);
  return launch_update_t<DK, DV, bf16_t>(a, p, seg, s);
}

bool prefill_update_supported(const dla_cache_desc& d, dla_dtype in_dtype) {
  const bool f = in_dtype == DLA_F32;
  const size_t b = d.d_k == 128 ? (f ? update_smem_bytes<128, float>(d.C)
                                     : update_smem_bytes<128, bf16_t>(d.C))
                                : (f ? update_smem_bytes<64, float>(d.C)
                                     : update_smem_bytes<64, bf16_t>(d.C));
  return b <= 160 * 1024;
}

hipError_t launch_prefill_update(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s) {
  const int dk = a.desc.d_k, dv = a.desc.d_v;
  if (dk == 128 && dv == 128) return launch_update_dims<128, 128>(a, p, seg, s);
  if (dk == 64 && dv == 64) return launch_update_dims<64, 64>(a, p, seg, s);
  if (dk == 128 && dv == 64) return launch_update_dims<128, 64>(a, p, seg, s);
  return launch_update_dims<64, 128>(a, p, seg, s);
}

}  // namespace dla
