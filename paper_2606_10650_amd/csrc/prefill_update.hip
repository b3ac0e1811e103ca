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
//     hold tokens of the chunk, sum_s k_s (exp(G_end - G_s) v_s)^T over their
//     consecutive token range (the update rule of Sec. 3.1 with the gated
//     decay of every state).  The decayed values are staged in LDS as three
//     bf16 terms whose sum is their float32 value, so the MFMA products with
//     the raw bf16 keys are exact to float32 rounding.  The waves split the
//     chunk's tokens into consecutive parts; each reads its keys straight from
//     global memory several 16-token groups ahead, with no barrier inside the
//     part.  Each rebuilt state is stored in frame G_end: the float32 master
//     in its cache slot, and a copy in MFMA operand order as a new pool
//     object.  States that nothing touched keep their slot, frame and object
//     (lazy decay).
// Slots of states merged away, and free slots, are reused by new states; the
// per-head permutation maps chronological states to slots.
#include "prefill_chunk.h"

namespace dla {

// Geometry of the update stage.  The workgroup's 8 waves form NSET sets of
// NBAND waves; wave (set, band) owns rows 32 band .. 32 band + 31 of d_k and the
// set-th of NSET consecutive parts of the chunk's tokens.
template <int DK, typename Tin>
struct UpdP {
  using CP = ChunkP<DK, Tin>;
  static constexpr int E = CP::E;
  static constexpr int RL = CP::RL;
  static constexpr int EPP = CP::EPP;
  static constexpr int VTS = CP::VTS;
  static constexpr int NTERM = E == 2 ? 3 : 1;   // bf16 terms that carry a float32 value
  static constexpr int TS = NC * VTS;            // elements per term
  static constexpr int NBAND = DK / 32;
  static constexpr int NSET = NWAVE / NBAND;
  static constexpr int PART = RL / NSET;         // tokens per part
  static constexpr int KD = E == 2 ? 8 : 4;      // key groups in flight per wave
  static constexpr int KW = E == 2 ? 4 : 8;      // 32-bit key loads per lane and group
  static constexpr int TPW = E == 2 ? 2 : 1;     // tokens per 32-bit word of staged values
  static constexpr int NPIECE = NC / EPP;        // 16-byte pieces of a token's 32 values
  static constexpr int VIPT = RL / TPW * NPIECE / NTHR;  // staging items per thread
  static constexpr size_t VBYTES = (size_t)NTERM * TS * E;
  static_assert(RL / TPW * NPIECE == VIPT * NTHR, "staging items");
  static_assert(PART % 16 == 0 && KD % 2 == 0, "part geometry");
  // the staged values' region also holds the chunk's leader tables before the
  // values are staged, and the partial sums of ranges that cross a part
  // boundary after the last use of the values
  static_assert(VBYTES >= (size_t)3 * RL * 4 && VBYTES >= (size_t)NWAVE * 64 * 16 * 4, "aliases");
};

// Key groups of the token-range loop in flight per wave when the keys come
// through LDS (KL): each group is the wave's 32 rows of d_k for 16 tokens, 1 KB
// of 16-bit keys.
constexpr int KDL = 4;

template <int DK, typename Tin>
__host__ __device__ static size_t update_smem_base(int C) {
  using U = UpdP<DK, Tin>;
  size_t off = round_up(U::VBYTES, 16);  // staged values (and their aliases)
  off += (size_t)C * 8;                  // sF
  off += (size_t)C * 4 * 13 + 64;        // int arrays, reduction scratch
  return round_up(off, 16);
}
template <int DK, typename Tin, bool KL>
static size_t update_smem_bytes(int C) {
  return update_smem_base<DK, Tin>(C) + (KL ? (size_t)NWAVE * KDL * 1024 : 0);  // key rings
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, int bytes) {
  // raw buffer: loads at byte offsets >= bytes return zero
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}

// KL: the token-range loop reads its keys from a per-wave LDS ring that the
// loads fill directly (16-bit inputs), with explicit waits; else straight from
// global memory into registers.
// VF: float32 values with 16-bit keys (a.v_f32), staged through the same three
// bfloat16 terms.
template <int DK, int DV, typename Tin, typename TS, bool KL, bool VF>
__global__ __launch_bounds__(NTHR) void prefill_update_kernel(PrefillArgs a, PrefillWS w,
                                                              SegPlan plan, int seg) {
  if (!cache_matches(a.cache, a.desc)) return;  // refused call (see the prep kernel)
  using FR = Frag<Tin>;
  using FT = typename FR::T;
  using U = UpdP<DK, Tin>;
  constexpr int D = DK * DV;
  constexpr int NCG = DV / NC;
  constexpr int RL = U::RL;
  constexpr int E = U::E;
  constexpr int VTS = U::VTS;
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
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int C = a.desc.C;
  const int T = a.T;
  int cs, ce;
  seg_range(plan, seg, &cs, &ce);
  const bool last_seg = seg == plan.nseg - 1;
  const bool copies = plan.P_cap > 0;  // pool objects for a readout stage

  extern __shared__ __align__(16) char smem[];
  // [NTERM][NC][VTS]: exp(G_end - G_s) v_s of the group's columns, transposed
  // (for 16-bit inputs as three bf16 terms, largest first)
  Tin* sV = reinterpret_cast<Tin*>(smem);
  int32_t* sDeath = reinterpret_cast<int32_t*>(smem);  // aliases, see UpdP
  int32_t* sLeadU = sDeath + RL;  // in-chunk leaders: position in the chunk
  int32_t* sLeadD = sLeadU + RL;  //                   death token
  float* xbuf = reinterpret_cast<float*>(smem);
  double* sF = reinterpret_cast<double*>(smem + round_up(U::VBYTES, 16));
  int32_t* sPerm = reinterpret_cast<int32_t*>(sF + C);
  int32_t* sLead = sPerm + C;
  int32_t* sObj = sLead + C;
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
  int32_t* sDt = eTmp;  // death token of each state present (until the alive sets)
  int32_t* eMO = eTmp;  // states rebuilt from old states only (after the pool objects)
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
      sObj[j] = plan.shared ? min(max(cv.obj[j], 0), plan.P_cap - 1) : j;
    }
  }
  // with a shared pool, a later segment continues the object numbering and
  // its states already have copies (made by the chunk before the segment)
  int next_obj = (plan.shared && seg > 0) ? min(max(*cv.next_obj, 0), plan.P_cap) : m;
  const bool fresh = !(plan.shared && seg > 0);

  // masters: float32 slots, or bfloat16 slots for closed states with the
  // newest state of the head in the float32 open region
  constexpr bool SB = sizeof(TS) == 2;
  constexpr int ES = (int)sizeof(TS);
  TS* states = reinterpret_cast<TS*>(a.cache + a.states_offset) + (size_t)h * C * D;
  float* open = SB ? reinterpret_cast<float*>(a.cache + a.open_offset) + (size_t)h * D : nullptr;
  const double* Gtok = w.Gtok + (size_t)h * T;
  const int32_t* death = w.death + (size_t)h * T;
  const Tin* Kin = static_cast<const Tin*>(a.k) + (size_t)h * T * DK;
  const Tin* Vin = static_cast<const Tin*>(a.v) + (size_t)h * T * DV;
  const float* Vf = static_cast<const float*>(a.v) + (size_t)h * T * DV;  // (VF)
  static_assert(!VF || E == 2, "float32 values go with 16-bit keys");
  auto obj_slice = [&](int obj) -> Tin* {
    return pool_slice<Tin>(w.pool, h, plan.P_cap, obj, cg, NCG, U::CP::SLICE);
  };

  // copies of the states present at the segment start
  __syncthreads();
  if (copies && fresh) {
    for (int j = 0; j < m; ++j) {
      const bool from_open = SB && j == m - 1;  // (wave-uniform)
      const TS* src = states + (size_t)sPerm[j] * D + cg * NC;
      const float* srco = from_open ? open + cg * NC : nullptr;
      Tin* dst = obj_slice(j);
      const int c = tid & 31;
      for (int kg = tid >> 5; kg < DK / 8; kg += NTHR / 32) {
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const size_t idx = (size_t)(8 * kg + e) * DV + c;
          x[e] = from_open ? srco[idx] : to_f32(src[idx]);
        }
        Tin* d8 = dst + kg * 256 + c * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) d8[e] = from_f32<Tin>(x[e]);
      }
    }
  }

  constexpr int NBAND = U::NBAND;
  constexpr int NSET = U::NSET;
  const int band = wv % NBAND;
  const int ib = 32 * band;
  const int set = wv / NBAND;
  // Band accesses of a master go through a buffer resource based at the band's
  // first element: lane offset (4 half d_v + l32) elements, element r at row
  // 8 (r / 4) + r % 4 further (the 8 (r / 4) rows in the scalar offset)
  // (slot and object numbers are wave-uniform: read them into scalars so the
  // resources live in scalar registers)
  auto band_rsrc = [&](int phys) __attribute__((always_inline)) {
    phys = __builtin_amdgcn_readfirstlane(phys);
    return buffer_rsrc(states + (size_t)phys * D + (size_t)ib * DV + cg * NC, 32 * DV * ES);
  };
  auto open_rsrc = [&]() __attribute__((always_inline)) {
    return buffer_rsrc(open + (size_t)ib * DV + cg * NC, 32 * DV * 4);
  };
  // a band of master j of the states present at the chunk start (the newest of
  // them, j = m - 1, is in the open region with bfloat16 storage)
  auto load_band = [&](int j, float (&x)[16]) __attribute__((always_inline)) {
    if (SB && j == m - 1) {
      const __amdgpu_buffer_rsrc_t r0 = open_rsrc();
#pragma unroll
      for (int r = 0; r < 16; ++r)
        x[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
            r0, (4 * half * DV + l32 + (r & 3) * DV) * 4, (r >> 2) * 8 * DV * 4, 0));
    } else {
      const __amdgpu_buffer_rsrc_t r0 = band_rsrc(sPerm[j]);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int vo = (4 * half * DV + l32 + (r & 3) * DV) * ES, so = (r >> 2) * 8 * DV * ES;
        if constexpr (ES == 4)
          x[r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r0, vo, so, 0));
        else
          x[r] = __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r0, vo, so, 0) << 16);
      }
    }
  };
  // decayed old states j = ja..jb added to a band accumulator, two states'
  // loads in flight at a time
  auto add_old = [&](f32x16& acc16, int ja, int jb, double Gend) __attribute__((always_inline)) {
    for (int j = ja; j <= jb; j += 2) {
      const bool two = j + 1 <= jb;
      float x[16], y[16];
      load_band(j, x);
      load_band(two ? j + 1 : j, y);
      const float f0 = __expf((float)(Gend - sF[j]));
      const float f1 = two ? __expf((float)(Gend - sF[j + 1])) : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc16[r] += f0 * x[r];
#pragma unroll
      for (int r = 0; r < 16; ++r) acc16[r] += f1 * y[r];
    }
  };
  // store a band of a state: the master (in the open region for the newest
  // state after the chunk with bfloat16 storage), and its copy when obj >= 0
  // (the copy's 8-byte pieces at ((ib / 8 + g4) * 256 + l32 * 8 + 4 half)
  // elements).  The stores carry the non-temporal hint (cache policy 2): the
  // states of a call (gigabytes) are not re-read before they have left the
  // caches.
  auto store_state = [&](const f32x16& acc16, int phys, int obj, bool to_open)
      __attribute__((always_inline)) {
    if (SB && to_open) {
      const __amdgpu_buffer_rsrc_t rs = open_rsrc();
#pragma unroll
      for (int r = 0; r < 16; ++r)
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc16[r]), rs,
                                              (4 * half * DV + l32 + (r & 3) * DV) * 4,
                                              (r >> 2) * 8 * DV * 4, 2);
    } else {
      const __amdgpu_buffer_rsrc_t rs = band_rsrc(phys);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int vo = (4 * half * DV + l32 + (r & 3) * DV) * ES, so = (r >> 2) * 8 * DV * ES;
        if constexpr (ES == 4)
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc16[r]), rs, vo, so, 2);
        else
          __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(acc16[r]).x, rs, vo, so, 2);
      }
    }
    obj = __builtin_amdgcn_readfirstlane(obj);
    if (obj >= 0) {
      const __amdgpu_buffer_rsrc_t ro = buffer_rsrc(obj_slice(obj), U::CP::SLICE * E);
      const int voff = (l32 * 8 + 4 * half) * E;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int soff = ((ib >> 3) + g4) * 256 * E;
        if constexpr (E == 2) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          const bf16x4 v4 = {(__bf16)acc16[4 * g4], (__bf16)acc16[4 * g4 + 1], (__bf16)acc16[4 * g4 + 2],
                             (__bf16)acc16[4 * g4 + 3]};
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v4), ro, voff, soff, 2);
        } else {
          const u32x4 v4 = {__float_as_uint(acc16[4 * g4]), __float_as_uint(acc16[4 * g4 + 1]),
                            __float_as_uint(acc16[4 * g4 + 2]), __float_as_uint(acc16[4 * g4 + 3])};
          __builtin_amdgcn_raw_buffer_store_b128(v4, ro, voff, soff, 2);
        }
      }
    }
  };

  for (int c = cs; c < ce; ++c) {
    const int c0 = c * RL;
    const int nrow = min(RL, T - c0);
    const int c1 = c0 + nrow;
    const double Gend = Gtok[c1 - 1];
    // copies of this chunk's rebuilt states are read by the next chunk: of the
    // segment only, or of the call with a shared pool
    const bool make_obj = copies && c + 1 < (plan.shared ? plan.nch : ce);
    __syncthreads();
    for (int i = tid; i < RL; i += NTHR) sDeath[i] = (i < nrow) ? death[c0 + i] : -1;
    for (int j = tid; j < m; j += NTHR) {
      const int ld = sLead[j];
      sDt[j] = (ld >= 0) ? death[ld] : iv.death0[ld + m0];
    }
    // the chunk's values (this group's columns) and log-decays: loads issued
    // now, staged in LDS once the leader tables no longer need the region.
    // Item i covers TPW consecutive tokens and one 16-byte piece.
    u32x4 vraw[U::VIPT][U::TPW];
    u32x4 vhi[VF ? U::VIPT : 1][VF ? U::TPW : 1];  // (VF) the piece's last four values
    double vg[U::VIPT][U::TPW];
    {
      const __amdgpu_buffer_rsrc_t vr =
          VF ? buffer_rsrc(Vf + (size_t)c0 * DV, nrow * DV * 4)
             : buffer_rsrc(Vin + (size_t)c0 * DV, nrow * DV * E);
#pragma unroll
      for (int u = 0; u < U::VIPT; ++u) {
        const int item = tid + NTHR * u;
        const int tp = item % (RL / U::TPW), p = item / (RL / U::TPW);
#pragma unroll
        for (int t = 0; t < U::TPW; ++t) {
          const int tok = U::TPW * tp + t;
          if constexpr (VF) {
            const int off = (tok * DV + cg * NC + p * U::EPP) * 4;
            vraw[u][t] = __builtin_amdgcn_raw_buffer_load_b128(vr, off, 0, 0);
            vhi[u][t] = __builtin_amdgcn_raw_buffer_load_b128(vr, off + 16, 0, 0);
          } else {
            vraw[u][t] = __builtin_amdgcn_raw_buffer_load_b128(
                vr, (tok * DV + cg * NC + p * U::EPP) * E, 0, 0);
          }
          vg[u][t] = Gtok[c0 + min(tok, nrow - 1)];
        }
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
          // with bfloat16 storage the newest state at the chunk start lives
          // in the open region: when it closes untouched, it is written to
          // its slot (rebuilt from itself)
          if (SB && ja_[u] == m - 1 && e != ne - 1) ch_[u] = 1;
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

    // ------------------------------------------------------ staged values
    // exp(G_end - G_s) v_s, rounded to the input type's terms (three bf16 terms
    // whose sum is the float32 product, so the MFMA products below are those of
    // float32 values); tokens past the chunk end hold zero
#pragma unroll
    for (int u = 0; u < U::VIPT; ++u) {
      const int item = tid + NTHR * u;
      const int tp = item % (RL / U::TPW), p = item / (RL / U::TPW);
      float ef[U::TPW];
#pragma unroll
      for (int t = 0; t < U::TPW; ++t)
        ef[t] = (U::TPW * tp + t < nrow) ? __expf((float)(Gend - vg[u][t])) : 0.f;
      if constexpr (E == 2) {
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        uint32_t* row = reinterpret_cast<uint32_t*>(sV + (p * U::EPP) * VTS) + tp;
#pragma unroll
        for (int q = 0; q < U::EPP; ++q) {
          // element q of the token's piece (float32 values: four per 16 bytes)
          auto val = [&](int t) __attribute__((always_inline)) -> float {
            if constexpr (VF)
              return __uint_as_float(q < 4 ? vraw[u][t][q & 3] : vhi[u][t][q & 3]);
            else
              return to_f32(piece_elem<bf16_t>(vraw[u][t], q));
          };
          const float x0 = ef[0] * val(0);
          const float x1 = ef[1] * val(1);
          const bf16x2 hi = {(__bf16)x0, (__bf16)x1};
          const float y0 = x0 - (float)hi[0], y1 = x1 - (float)hi[1];
          const bf16x2 mid = {(__bf16)y0, (__bf16)y1};
          const bf16x2 lo = {(__bf16)(y0 - (float)mid[0]), (__bf16)(y1 - (float)mid[1])};
          uint32_t* r = row + q * (VTS / 2);
          r[0] = __builtin_bit_cast(uint32_t, hi);
          r[U::TS / 2] = __builtin_bit_cast(uint32_t, mid);
          r[U::TS] = __builtin_bit_cast(uint32_t, lo);
        }
      } else {
#pragma unroll
        for (int q = 0; q < U::EPP; ++q)
          sV[(p * U::EPP + q) * VTS + tp] = ef[0] * piece_elem<float>(vraw[u][0], q);
      }
    }

    // pool objects of the rebuilt states, in chronological order
    const int nchg = block_excl_count(ne, [&](int e) { return eChg[e] != 0; }, eTmp, red);
    // (next_obj + nchg <= P_cap: a segment starts with at most C objects and
    // each of its chunks but the last adds at most C)
    for (int e = tid; e < ne; e += NTHR)
      eObj[e] = (eChg[e] && make_obj && next_obj + eTmp[e] < plan.P_cap) ? next_obj + eTmp[e] : -1;
    __syncthreads();
    // the token ranges: the newest old state's (when it takes chunk tokens),
    // then the new leaders', tiling the chunk
    const int rfirst = (nAO > 0 && eR1[nAO - 1] >= eR0[nAO - 1]) ? nAO - 1 : nAO;
    const int ncont = rfirst < nAO ? 1 : 0;
    // states changed by merges of old states only (wave 0)
    if (wv == 0) {
      int n = 0;
      for (int base = 0; base < nAO; base += 64) {
        const int e = base + lane;
        const bool f = e < nAO && eChg[e] != 0 && eR1[e] < eR0[e];
        const uint64_t bal = __ballot(f);
        if (f) eMO[n + __popcll(bal & ((1ull << lane) - 1ull))] = e;
        n += __popcll(bal);
      }
      if (lane == 0) sCnt[1] = n;
    }
    __syncthreads();
    const int nMO = sCnt[1];

    // -------------------------------------- sums of old states (Alg. 2 merges)
    // Item 0 is the newest old group when it takes chunk tokens: its decayed
    // old states start the accumulator of the set that owns token 0.  The
    // other items are the states rebuilt from old states only, stored here.
    // Every read of an old slot completes before the barrier below, so slots
    // of merged-away states can take new states afterwards.
    f32x16 acc = zero16();
    for (int i = set; i < ncont + nMO; i += NSET) {
      const int e = i < ncont ? rfirst : eMO[i - ncont];
      f32x16 u16 = zero16();
      add_old(u16, eJa[e], eJb[e], Gend);
      if (i < ncont)
        acc = u16;
      else
        store_state(u16, ePhys[e], eObj[e], e == ne - 1);
    }
    __syncthreads();

    // ------------------------------------------------------- token ranges
    // Each set walks the 16-token groups of its part.  The MFMA A operand is
    // K^T (32 rows of d_k by 16 tokens, zero outside the current range), read
    // from global memory KD groups ahead; B is the staged values.  A range
    // that ends in the part is stored when it ends; a range that reaches past
    // the part is finished by the set where it started, with the partial sums
    // of the later sets.
    const int ps = set * U::PART;
    const int pe = min(ps + U::PART, nrow);
    int inR = -1, outR = -1;
    f32x16 xacc = zero16();
    if (ps < nrow && rfirst < ne) {
      // the range holding token ps: the last one starting at or before it
      int cnt = 0;
      for (int base = rfirst; base < ne; base += 64) {
        const int e = base + lane;
        const uint64_t bal = __ballot(e < ne && eR0[e] <= ps);
        cnt += __popcll(bal);
        if (bal != ~0ull) break;
      }
      int rc = max(rfirst + cnt - 1, rfirst);
      int r0c = __builtin_amdgcn_readfirstlane(eR0[rc]);
      int r1c = __builtin_amdgcn_readfirstlane(eR1[rc]);
      if (r0c < ps) inR = rc;

      const __amdgpu_buffer_rsrc_t kr = buffer_rsrc(Kin + (size_t)c0 * DK, nrow * DK * E);
      const bool odd = (l32 & 1) != 0;
      // 16-bit keys: lane pair (2i, 2i + 1) of a half reads the 32-bit words
      // holding rows ib + 2i, ib + 2i + 1 of tokens s0 .. s0 + 3 (even lane) and
      // s0 + 4 .. s0 + 7 (odd lane), and the pair swaps halves; float32 keys:
      // the lane reads its row of the 8 tokens
      auto kload = [&](int g, uint32_t (&dst)[U::KW]) __attribute__((always_inline)) {
        const int s0 = 16 * g + 8 * half;
        if constexpr (E == 2) {
          const int off = ((s0 + (odd ? 4 : 0)) * DK + ib + (l32 & ~1)) * 2;
#pragma unroll
          for (int u = 0; u < 4; ++u) dst[u] = __builtin_amdgcn_raw_buffer_load_b32(kr, off + u * DK * 2, 0, 0);
        } else {
          const int off = (s0 * DK + ib + l32) * 4;
#pragma unroll
          for (int u = 0; u < 8; ++u) dst[u] = __builtin_amdgcn_raw_buffer_load_b32(kr, off + u * DK * 4, 0, 0);
        }
      };
      auto kfrag = [&](const uint32_t (&r)[U::KW]) __attribute__((always_inline)) -> FT {
        if constexpr (E == 2) {
          const uint32_t L0 = __builtin_amdgcn_perm(r[1], r[0], 0x05040100u);  // low halves
          const uint32_t L1 = __builtin_amdgcn_perm(r[3], r[2], 0x05040100u);
          const uint32_t H0 = __builtin_amdgcn_perm(r[1], r[0], 0x07060302u);  // high halves
          const uint32_t H1 = __builtin_amdgcn_perm(r[3], r[2], 0x07060302u);
          // quad_perm [1, 0, 3, 2]: swap with the pair's other lane
          const uint32_t R0 = (uint32_t)__builtin_amdgcn_mov_dpp((int)(odd ? L0 : H0), 0xB1, 0xF, 0xF, false);
          const uint32_t R1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)(odd ? L1 : H1), 0xB1, 0xF, 0xF, false);
          u32x4 wq;
          wq[0] = odd ? R0 : L0;
          wq[1] = odd ? R1 : L1;
          wq[2] = odd ? H0 : R0;
          wq[3] = odd ? H1 : R1;
          return __builtin_bit_cast(FT, wq);
        } else {
          FT out;
#pragma unroll
          for (int e = 0; e < 8; ++e) out[e] = __uint_as_float(r[e]);
          return out;
        }
      };
      // zero the A elements of tokens outside [r0, r1] (element e <-> token s0 + e)
      auto kmask = [&](FT av, int s0, int r0, int r1) __attribute__((always_inline)) -> FT {
        if constexpr (E == 2) {
          u32x4 wq = __builtin_bit_cast(u32x4, av);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int t = s0 + 2 * q;
            const uint32_t mk = ((t >= r0 && t <= r1) ? 0x0000FFFFu : 0u) |
                                ((t + 1 >= r0 && t + 1 <= r1) ? 0xFFFF0000u : 0u);
            wq[q] &= mk;
          }
          return __builtin_bit_cast(FT, wq);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (s0 + e < r0 || s0 + e > r1) av[e] = 0.f;
          return av;
        }
      };
      struct BOp {
        FT t[U::NTERM];
      };
      auto bload = [&](int g, BOp& b) __attribute__((always_inline)) {
        const Tin* p = sV + l32 * VTS + 16 * g + 8 * half;
#pragma unroll
        for (int q = 0; q < U::NTERM; ++q) b.t[q] = FR::load(p + q * U::TS);
      };
      auto mma_all = [&](const FT& av, const BOp& b) __attribute__((always_inline)) {
#pragma unroll
        for (int q = U::NTERM - 1; q >= 0; --q) FR::mma(acc, av, b.t[q]);  // smallest term first
      };
      auto group = [&](int g, const FT& av, const BOp& b) __attribute__((always_inline)) {
        const int gs = 16 * g, ge = gs + 15;
        const int s0 = gs + 8 * half;
        while (true) {
          if (r0c > gs || r1c < ge)
            mma_all(kmask(av, s0, r0c, r1c), b);
          else
            mma_all(av, b);
          if (r1c > ge) break;  // the range continues in the next group
          // the range ends here
          if (rc == inR)
            xacc = acc;
          else
            store_state(acc, ePhys[rc], eObj[rc], rc == ne - 1);
          acc = zero16();
          ++rc;
          if (rc >= ne) break;
          r0c = __builtin_amdgcn_readfirstlane(eR0[rc]);
          r1c = __builtin_amdgcn_readfirstlane(eR1[rc]);
          if (r0c > ge) break;
        }
      };

      const int g0 = ps >> 4, g1 = (pe + 15) >> 4;
      BOp bb[2];
      if constexpr (KL) {
        // The wave's keys pass through its ring of KDL groups in LDS, each
        // loaded straight from memory (lane i brings 16 bytes: token i / 4 of
        // the group, piece (i % 4) ^ (token / 4 % 4) of the band's 32 rows, so
        // that the reads below spread over the banks).  A range end inside the
        // loop stores a state, so the number of memory operations between a
        // group's request and its use varies: the waits count only the later
        // key requests, which are a lower bound.
        char* kring = smem + update_smem_base<DK, Tin>(C) + (size_t)wv * KDL * 1024;
        auto kdma = [&](int g) __attribute__((always_inline)) {
          const int t = lane >> 2, pc = (lane & 3) ^ ((t >> 2) & 3);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              kr, (__attribute__((address_space(3))) void*)(kring + (g % KDL) * 1024), 16,
              ((16 * g + t) * DK + ib + 8 * pc) * 2, 0, 0, 0);
        };
        // the 32-bit words kload would read for group g, from the ring
        auto kread = [&](int g, uint32_t (&dst)[U::KW]) __attribute__((always_inline)) {
          const char* slot = kring + (g % KDL) * 1024;
          const int r = l32 & ~1;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int tk = 8 * half + (odd ? 4 : 0) + u;
            const int pos = 4 * tk + ((r >> 3) ^ ((tk >> 2) & 3));
            dst[u] = *reinterpret_cast<const uint32_t*>(slot + pos * 16 + (r & 7) * 2);
          }
        };
        // wait until the request of group g has landed: the requests issued
        // after it, up to group e - 1, are a lower bound on those in flight
        static_assert(KDL == 4, "wait counts");
        auto kwait = [&](int later) __attribute__((always_inline)) {
          if (later >= 3)
            __builtin_amdgcn_s_waitcnt((3 & 15) | (7 << 4) | (15 << 8) | ((3 >> 4) << 14));
          else if (later == 2)
            __builtin_amdgcn_s_waitcnt((2 & 15) | (7 << 4) | (15 << 8) | ((2 >> 4) << 14));
          else if (later == 1)
            __builtin_amdgcn_s_waitcnt((1 & 15) | (7 << 4) | (15 << 8) | ((1 >> 4) << 14));
          else
            __builtin_amdgcn_s_waitcnt((0 & 15) | (7 << 4) | (15 << 8) | ((0 >> 4) << 14));
        };
        for (int u = 0; u < KDL; ++u)
          if (g0 + u < g1) kdma(g0 + u);
        bload(g0, bb[0]);
        uint32_t kwa[U::KW], kwb[U::KW];
        kwait(min(KDL - 1, g1 - 1 - g0));
        kread(g0, kwa);
        // Group g with its staged values in cur and its key words in kc; the
        // next group's values and key words are read into nxt and kn.  The
        // request of group g + KDL reuses group g's slot, whose reads have
        // returned (their words are in av).
        auto step = [&](int g, BOp& cur, BOp& nxt, uint32_t (&kc)[U::KW], uint32_t (&kn)[U::KW])
            __attribute__((always_inline)) {
          const FT av = kfrag(kc);
          if (g + KDL < g1) kdma(g + KDL);
          if (g + 1 < g1) {
            bload(g + 1, nxt);
            kwait(min(KDL - 1, g1 - 2 - g));
            kread(g + 1, kn);
          }
          group(g, av, cur);
        };
        for (int g = g0; g < g1; g += 2) {
          step(g, bb[0], bb[1], kwa, kwb);
          if (g + 1 < g1) step(g + 1, bb[1], bb[0], kwb, kwa);
        }
      } else {
        uint32_t kw[U::KD][U::KW];
#pragma unroll
        for (int u = 0; u < U::KD; ++u)
          if (g0 + u < g1) kload(g0 + u, kw[u]);
        bload(g0, bb[0]);
        for (int gb = g0; gb < g1; gb += U::KD) {
#pragma unroll
          for (int u = 0; u < U::KD; ++u) {
            const int g = gb + u;
            if (g < g1) {
              if (g + 1 < g1) bload(g + 1, bb[(u + 1) & 1]);
              const FT av = kfrag(kw[u]);
              if (g + U::KD < g1) kload(g + U::KD, kw[u]);
              group(g, av, bb[u & 1]);
            }
          }
        }
      }
      if (rc < ne && r0c < pe && r1c >= pe) {  // the range reaches past the part
        if (rc == inR)
          xacc = acc;
        else
          outR = rc;
      }
    }
    __syncthreads();  // every set is done with the staged values
    if (inR >= 0) {
      float4* xb = reinterpret_cast<float4*>(xbuf + wv * 1024);
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        xb[r4 * 64 + lane] = make_float4(xacc[4 * r4], xacc[4 * r4 + 1], xacc[4 * r4 + 2], xacc[4 * r4 + 3]);
    }
    __syncthreads();
    if (outR >= 0) {
      const int r1o = eR1[outR];
      for (int q = set + 1; q < NSET && q * U::PART <= r1o; ++q) {
        const float4* xb = reinterpret_cast<const float4*>(xbuf + (q * NBAND + band) * 1024);
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const float4 x = xb[r4 * 64 + lane];
          acc[4 * r4] += x.x;
          acc[4 * r4 + 1] += x.y;
          acc[4 * r4 + 2] += x.z;
          acc[4 * r4 + 3] += x.w;
        }
      }
      store_state(acc, ePhys[outR], eObj[outR], outR == ne - 1);
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
        cv.obj[j] = sObj[j];
      }
      if (tid == 0) {
        *cv.m = m;
        *cv.next_obj = next_obj;
      }
    }
  }
}

template <int DK, int DV, typename Tin, typename TS>
static hipError_t launch_update_t(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s) {
  const int nh = a.desc.B * a.desc.H;
  PrefillWS w = ws_layout(a.workspace, nh, a.T, a.desc.C, a.desc.d_k * a.desc.d_v, p.nch);
  const int grid = (int)round_up(nh, 8) * (DV / NC);
  auto launch = [&](auto k, size_t shm) -> hipError_t {
    if (shm > 160 * 1024) return hipErrorInvalidValue;
    if (hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm) !=
        hipSuccess)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3(grid), dim3(NTHR), shm, s, a, w, p, seg);
    return hipGetLastError();
  };
  // keys through LDS for 16-bit inputs when the rings fit beside the rest
  constexpr bool E2 = sizeof(Tin) == 2;
  const size_t shm_kl = update_smem_bytes<DK, Tin, E2>(a.desc.C);
  const size_t shm = update_smem_bytes<DK, Tin, false>(a.desc.C);
  if (E2 && a.v_f32) {
    if (shm_kl <= 160 * 1024) return launch(prefill_update_kernel<DK, DV, Tin, TS, E2, E2>, shm_kl);
    return launch(prefill_update_kernel<DK, DV, Tin, TS, false, E2>, shm);
  }
  if (a.v_f32) return hipErrorInvalidValue;  // (float32 values go with 16-bit keys)
  if (E2 && shm_kl <= 160 * 1024) return launch(prefill_update_kernel<DK, DV, Tin, TS, E2, false>, shm_kl);
  return launch(prefill_update_kernel<DK, DV, Tin, TS, false, false>, shm);
}

template <int DK, int DV>
static hipError_t launch_update_dims(const PrefillArgs& a, const SegPlan& p, int seg,
                                     hipStream_t s) {
  const bool sb = a.desc.state_dtype == DLA_BF16;
  if (a.in_dtype == DLA_F32)
    return sb ? launch_update_t<DK, DV, float, bf16_t>(a, p, seg, s)
              : launch_update_t<DK, DV, float, float>(a, p, seg, s);
  return sb ? launch_update_t<DK, DV, bf16_t, bf16_t>(a, p, seg, s)
            : launch_update_t<DK, DV, bf16_t, float>(a, p, seg, s);
}

bool prefill_update_supported(const dla_cache_desc& d, dla_dtype in_dtype) {
  const bool f = in_dtype == DLA_F32;
  const size_t b = d.d_k == 128 ? (f ? update_smem_bytes<128, float, false>(d.C)
                                     : update_smem_bytes<128, bf16_t, false>(d.C))
                                : (f ? update_smem_bytes<64, float, false>(d.C)
                                     : update_smem_bytes<64, bf16_t, false>(d.C));
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
