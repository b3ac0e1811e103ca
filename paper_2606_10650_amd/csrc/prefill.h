// Prefill entry (internal): arguments, workspace layout, segment plan and
// launchers.
#pragma once
#include "dla_common.h"

namespace dla {

struct PrefillArgs {
  dla_cache_desc desc;
  char* cache;
  size_t meta_offset, meta_stride, states_offset, open_offset;
  const void* q;
  const void* k;
  const void* v;
  const float* g;
  const void* lam;
  void* out;
  int8_t* b_out;
  int32_t* merge_out;
  float* score_out;
  const int8_t* b_ovr;
  const int32_t* m_ovr;
  int T;
  float tau, eps, eps_rms;
  int skip_readout;
  dla_dtype in_dtype, out_dtype;
  int serial;  // stages one after another on the caller's stream
  size_t pool_budget;  // bytes of state copies per call (pool_budget_of)
  char* workspace;
  // values given as float32 with 16-bit keys (the update stage of the Gated
  // DeltaNet form, whose values are the delta rule's write vectors)
  int v_f32;
};

// ---------------------------------------------------------------------------
// Readout chunks and segments.
//
// Stages 3 (state update) and 4 (readout) work on chunks of RL tokens.  The
// update stage walks the chunks in order and records, for every chunk, the
// list of states present at its start; every state it rebuilds gets a fresh
// object in a per-head pool holding a bfloat16 (or float32) copy of the state
// in MFMA operand order.  The readout stage then runs every chunk in parallel
// against the pool.  A chunk creates at most C objects, so the pool holds up to
// C objects per chunk; to bound its size the call is split into segments of at
// most nch_seg chunks (update, then readout, per segment), and each segment
// starts its pool afresh with copies of the states present at its start.
// ---------------------------------------------------------------------------
constexpr int NWAVE = 8;  // waves per workgroup of the update stage
constexpr int NTHR = 64 * NWAVE;
constexpr int RWAVE = 8;  // waves per workgroup of the readout stage (two per SIMD)
constexpr int RTHR = 64 * RWAVE;
constexpr int NC = 32;    // value columns per workgroup
constexpr size_t kPoolBudget = (size_t)8 << 30;  // default bytes of state copies per call

// The budget of state copies that the flags select (bits 8..15: log2 of the
// bytes, 0 for the default), or 0 when the field is out of range.
inline size_t pool_budget_of(uint32_t flags) {
  const uint32_t k = (flags & DLA_POOL_BUDGET_MASK) >> DLA_POOL_BUDGET_SHIFT;
  if (k == 0) return kPoolBudget;
  if (k < 20 || k > 40) return 0;
  return (size_t)1 << k;
}
// A pipelined call runs the scan segment by segment on a second stream while
// the first stream updates and reads out the segments already scanned, so only
// the first segment's scan is exposed; its segments grow as a ramp (seg_range).

// token tiles of 32 per readout wave: two for 16-bit inputs, one for float32
// inputs (whose operands take twice the registers and LDS)
__host__ __device__ constexpr int readout_nt(int elem_bytes) { return elem_bytes == 2 ? 2 : 1; }
__host__ __device__ constexpr int chunk_len(int elem_bytes) {
  return 32 * RWAVE * readout_nt(elem_bytes);
}

struct SegPlan {
  int RL;       // tokens per chunk
  int nch;      // chunks in the call
  int nch_seg;  // chunks per segment (the largest segment of a ramp)
  int nseg;     // segments
  int P_cap;    // pool objects per head (0 without a readout)
  int first;    // 0: segments of nch_seg chunks; else a ramp starting at `first`
  int fit;      // largest segment of a ramp (pool budget)
  int shared;   // 1: one pool for the whole call, objects numbered across segments
};

// Segment sizes of a ramp: each segment is half again as long as the one
// before (first, then growing, at most fit), and a segment takes everything
// left when that is at most twice its size.  The update and readout of a
// segment cost about twice the scan's time per chunk, so while they run the
// scan of the next, longer segment finishes, and the caller's stream rarely
// waits for the scan after the first, short, segment.
__host__ __device__ inline int ramp_size(int first, int fit, int k, int rem) {
  int sz = first;
  for (int i = 0; i < k && sz < fit; ++i) sz += (sz + 1) / 2;
  sz = sz < fit ? sz : fit;
  int n = rem <= 2 * sz ? rem : sz;
  return n < fit ? n : fit;
}

// chunks [cs, ce) of segment seg
__host__ __device__ inline void seg_range(const SegPlan& p, int seg, int* cs, int* ce) {
  if (p.first == 0) {
    *cs = seg * p.nch_seg;
    *ce = p.nch < *cs + p.nch_seg ? p.nch : *cs + p.nch_seg;
    return;
  }
  int b = 0;
  for (int k = 0; k < seg; ++k) b += ramp_size(p.first, p.fit, k, p.nch - b);
  *cs = b;
  *ce = b + ramp_size(p.first, p.fit, seg, p.nch - b);
}

inline size_t dtype_bytes(dla_dtype t) { return t == DLA_F32 ? 4 : 2; }

// Whether a call overlaps the scan with the later stages: with a readout, at
// least two chunks, and unless the caller asked for serial stages.
inline bool pipelined(int T, dla_dtype in, bool readout, bool serial) {
  const int RL = chunk_len((int)(in == DLA_F32 ? 4 : 2));
  return readout && !serial && T > RL;
}

inline SegPlan seg_plan(const dla_cache_desc& d, int T, dla_dtype in, bool readout,
                        bool serial, size_t budget) {
  SegPlan p;
  const int E = (int)dtype_bytes(in);
  p.RL = chunk_len(E);
  p.nch = T > 0 ? (T + p.RL - 1) / p.RL : 0;
  p.first = 0;
  p.fit = 0;
  p.shared = 0;
  if (!readout || p.nch == 0) {
    p.nch_seg = p.nch > 0 ? p.nch : 1;
    p.nseg = 1;
    p.P_cap = 0;
    return p;
  }
  const size_t per_chunk = (size_t)d.B * d.H * d.C * d.d_k * d.d_v * E;
  const size_t fit_z = budget / per_chunk;
  int fit = fit_z > (size_t)p.nch ? p.nch : (int)fit_z;
  if (fit < 1) fit = 1;
  if (pipelined(T, in, readout, serial)) {
    p.first = p.nch / 16 > 1 ? p.nch / 16 : 1;
    p.fit = fit;
    p.nseg = 0;
    p.nch_seg = 0;
    for (int b = 0; b < p.nch; ++p.nseg) {
      const int n = ramp_size(p.first, fit, p.nseg, p.nch - b);
      p.nch_seg = n > p.nch_seg ? n : p.nch_seg;
      b += n;
    }
  } else {
    p.nseg = (p.nch + fit - 1) / fit;
    p.nch_seg = (p.nch + p.nseg - 1) / p.nseg;
    p.nseg = (p.nch + p.nch_seg - 1) / p.nch_seg;  // no empty segment
  }
  // a pipelined call whose copies all fit the budget keeps one pool, so that
  // no segment starts with copies of the states already present
  p.shared = (p.first > 0 && p.nch <= fit) ? 1 : 0;
  p.P_cap = d.C * (p.shared ? p.nch : p.nch_seg);
  return p;
}

// Workspace regions (per head, 256-byte aligned):
//   Gtok   double [nh][T]   cumulative log-decay after each token (global frame)
//   death  int32  [nh][T]   -1: token t is not the first token of a state;
//                           T: it starts a state that is never merged away;
//                           t' in (t, T): its state was merged into its left
//                           neighbour at token t' (Alg. 2)
//   init   per head: int32 m0, int32 pad, double G0, double F0[C], int32 perm0[C],
//          int32 death0[C] (the cache's metadata before the call, and the death
//          token of the states present before the call)
//   carry  per head: int32 m, int32 next_obj, double F[C], int32 perm[C],
//          int32 lead[C], int32 obj[C] (update-stage bookkeeping handed from one
//          segment to the next; next_obj and obj only with a shared pool)
//   scarry per head: int32 m, int32 pad, double Ibar[C], int32 n[C], int32 lead[C],
//          then from a 16-byte boundary float S[d_k d_v] (the scan's bookkeeping
//          and its newest state, in accumulator order, handed from one scan
//          segment to the next)
//   lists  [nh][nch] chunk lists: int32 m at offset 0, then from offset 16 one
//          ListEntry per state present at the chunk start, in chronological order
//   pool   [nh][P_cap] state copies, each [d_v/32][d_k/16][2][32][8] elements of
//          the input dtype: the per-lane order of the MFMA A operand for one
//          32-column group, so a lane reads its operand with 16-byte loads
struct ListEntry {
  int32_t obj;  // pool object holding the state's copy
  int32_t dt;   // token at which Alg. 2 merges the state away (T: never)
  double F;     // frame: the true state is exp(G - F) times the stored one
};

struct PrefillWS {
  double* Gtok;
  int32_t* death;
  char* init;
  size_t init_stride;
  char* carry;
  size_t carry_stride;
  char* scarry;
  size_t scarry_stride;
  char* lists;
  size_t list_stride;
  char* pool;
};

__host__ __device__ inline size_t ws_init_stride(int C) { return round_up(16 + 16 * (size_t)C, 256); }
__host__ __device__ inline size_t ws_carry_stride(int C) { return round_up(8 + 20 * (size_t)C, 256); }
__host__ __device__ inline size_t ws_scarry_stride(int C, int D) {
  return round_up(round_up(16 + 16 * (size_t)C, 16) + 4 * (size_t)D, 256);
}
__host__ __device__ inline size_t ws_list_stride(int C) {
  return round_up(16 + sizeof(ListEntry) * (size_t)C, 256);
}

__host__ __device__ inline PrefillWS ws_layout(char* base, int nh, int T, int C, int D, int nch) {
  PrefillWS w;
  size_t off = 0;
  w.Gtok = reinterpret_cast<double*>(base + off);
  off = round_up(off + (size_t)nh * T * sizeof(double), 256);
  w.death = reinterpret_cast<int32_t*>(base + off);
  off = round_up(off + (size_t)nh * T * sizeof(int32_t), 256);
  w.init = base + off;
  w.init_stride = ws_init_stride(C);
  off = round_up(off + (size_t)nh * w.init_stride, 256);
  w.carry = base + off;
  w.carry_stride = ws_carry_stride(C);
  off = round_up(off + (size_t)nh * w.carry_stride, 256);
  w.scarry = base + off;
  w.scarry_stride = ws_scarry_stride(C, D);
  off = round_up(off + (size_t)nh * w.scarry_stride, 256);
  w.lists = base + off;
  w.list_stride = ws_list_stride(C);
  off = round_up(off + (size_t)nh * nch * w.list_stride, 256);
  w.pool = base + off;
  return w;
}

inline size_t prefill_workspace_bytes(const dla_cache_desc& d, int T, dla_dtype in, bool readout,
                                      bool serial, size_t budget) {
  const size_t nh = (size_t)d.B * d.H;
  const SegPlan p = seg_plan(d, T, in, readout, serial, budget);
  size_t off = round_up(nh * T * sizeof(double), 256);
  off = round_up(off + nh * T * sizeof(int32_t), 256);
  off = round_up(off + nh * ws_init_stride(d.C), 256);
  off = round_up(off + nh * ws_carry_stride(d.C), 256);
  off = round_up(off + nh * ws_scarry_stride(d.C, d.d_k * d.d_v), 256);
  off = round_up(off + nh * (size_t)p.nch * ws_list_stride(d.C), 256);
  off += nh * (size_t)p.P_cap * d.d_k * d.d_v * dtype_bytes(in);
  return off;
}

struct InitView {
  int32_t* m0;
  double* G0;
  double* F0;
  int32_t* perm0;
  int32_t* death0;
};

__host__ __device__ inline InitView init_at(const PrefillWS& w, int h, int C) {
  char* p = w.init + (size_t)h * w.init_stride;
  InitView v;
  v.m0 = reinterpret_cast<int32_t*>(p);
  v.G0 = reinterpret_cast<double*>(p + 8);
  v.F0 = reinterpret_cast<double*>(p + 16);
  v.perm0 = reinterpret_cast<int32_t*>(p + 16 + 8 * (size_t)C);
  v.death0 = v.perm0 + C;
  return v;
}

struct CarryView {
  int32_t* m;
  int32_t* next_obj;
  double* F;
  int32_t* perm;
  int32_t* lead;
  int32_t* obj;
};

__host__ __device__ inline CarryView carry_at(const PrefillWS& w, int h, int C) {
  char* p = w.carry + (size_t)h * w.carry_stride;
  CarryView v;
  v.m = reinterpret_cast<int32_t*>(p);
  v.next_obj = v.m + 1;
  v.F = reinterpret_cast<double*>(p + 8);
  v.perm = reinterpret_cast<int32_t*>(p + 8 + 8 * (size_t)C);
  v.lead = v.perm + C;
  v.obj = v.lead + C;
  return v;
}

struct ScarryView {
  int32_t* m;
  double* ibar;
  int32_t* n;
  int32_t* lead;
  float* S;
};

__host__ __device__ inline ScarryView scarry_at(const PrefillWS& w, int h, int C) {
  char* p = w.scarry + (size_t)h * w.scarry_stride;
  ScarryView v;
  v.m = reinterpret_cast<int32_t*>(p);
  v.ibar = reinterpret_cast<double*>(p + 16);
  v.n = reinterpret_cast<int32_t*>(p + 16 + 8 * (size_t)C);
  v.lead = v.n + C;
  v.S = reinterpret_cast<float*>(p + round_up(16 + 16 * (size_t)C, 16));
  return v;
}

__host__ __device__ inline char* list_at(const PrefillWS& w, int h, int c, int nch) {
  return w.lists + ((size_t)h * nch + c) * w.list_stride;
}

hipError_t launch_prefill_prep(const PrefillArgs& a, hipStream_t s);
// the scan over tokens [tb, te) (chunk-aligned); a segment after the first
// resumes from the scan carry that the previous one left in the workspace
hipError_t launch_prefill_scan(const PrefillArgs& a, int tb, int te, hipStream_t s);
hipError_t launch_prefill_update(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s);
hipError_t launch_prefill_readout(const PrefillArgs& a, const SegPlan& p, int seg, hipStream_t s);
// whether the scan, update and readout stages' working sets fit in LDS for this
// shape
bool prefill_chunks_supported(const dla_cache_desc& d, dla_dtype in_dtype);

// Gated DeltaNet form (prefill_delta.hip): the sequential scan that yields the
// pseudo-values, then the update and readout stages over them (pipelined
// unless a.serial).
hipError_t launch_prefill_delta(const PrefillArgs& a, const float* beta, hipStream_t s);
size_t prefill_delta_workspace_bytes(const dla_cache_desc& d, int T, dla_dtype in, bool readout,
                                     bool serial, size_t budget);
size_t prefill_delta_scan_smem(const dla_cache_desc& d);

// The second stream of a pipelined call on the device of the caller's stream,
// and n events for ordering the two streams (owned by the library, one set per
// host thread and device; created on first use).
hipError_t pipe_resources(hipStream_t caller, int n, hipStream_t* side, hipEvent_t** evs);

// Event hooks of a call: ev (nullable) receives an event before the first
// stage and after the token frames, the scan, the state updates and the
// readouts; rev (nullable, nrev entries) receives one event before and one
// after each segment's readout launch, for segments s < nrev / 2.
struct StageEvents {
  void* const* ev;
  void* const* rev;
  int nrev;
};

// Stages in order.  Serial: frames, the whole scan, then update and readout
// segment by segment, all on s.  Pipelined: the scan segments run on a second
// stream, forked from s after the token frames, and segment k's update and
// readout on s wait for segment k's scan; s waits for the whole scan before
// its last update, so the call joins on s.
inline hipError_t launch_prefill(const PrefillArgs& a, hipStream_t s, const StageEvents& se) {
  const bool pipe = pipelined(a.T, a.in_dtype, !a.skip_readout, a.serial != 0);
  const SegPlan p = seg_plan(a.desc, a.T, a.in_dtype, !a.skip_readout, a.serial != 0,
                             a.pool_budget);
  auto rec = [&](int i, hipStream_t st) -> hipError_t {
    if (se.ev && hipEventRecord((hipEvent_t)se.ev[i], st) != hipSuccess) return hipErrorInvalidValue;
    return hipSuccess;
  };
  auto rrec = [&](int seg, int end) -> hipError_t {
    if (se.rev && 2 * seg + 1 < se.nrev &&
        hipEventRecord((hipEvent_t)se.rev[2 * seg + end], s) != hipSuccess)
      return hipErrorInvalidValue;
    return hipSuccess;
  };
  hipError_t e;
  if ((e = rec(0, s)) != hipSuccess) return e;
  if ((e = launch_prefill_prep(a, s)) != hipSuccess) return e;
  if ((e = rec(1, s)) != hipSuccess) return e;
  hipStream_t side = s;
  hipEvent_t* pev = nullptr;
  bool forked = false;
  // After the fork, an error still joins the second stream into s before it
  // is returned, so that nothing enqueued on the second stream can outlive the
  // call's ordering on s (the caller may free the workspace once s is done).
  auto fail = [&](hipError_t err) -> hipError_t {
    if (forked && hipEventRecord(pev[0], side) == hipSuccess) (void)hipStreamWaitEvent(s, pev[0], 0);
    return err;
  };
  if (pipe) {
    // event 0 forks the side stream after the frames; event 1 + k marks the
    // end of scan segment k
    if ((e = pipe_resources(s, p.nseg + 1, &side, &pev)) != hipSuccess) return e;
    if ((e = hipEventRecord(pev[0], s)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(side, pev[0], 0)) != hipSuccess) return e;
    forked = true;
    for (int seg = 0; seg < p.nseg; ++seg) {
      int cs, ce;
      seg_range(p, seg, &cs, &ce);
      const int tb = cs * p.RL;
      const int te = (seg + 1 == p.nseg) ? a.T : ce * p.RL;
      if ((e = launch_prefill_scan(a, tb, te, side)) != hipSuccess) return fail(e);
      if ((e = hipEventRecord(pev[1 + seg], side)) != hipSuccess) return fail(e);
    }
    if ((e = rec(2, side)) != hipSuccess) return fail(e);
  } else {
    if ((e = launch_prefill_scan(a, 0, a.T, s)) != hipSuccess) return e;
    if ((e = rec(2, s)) != hipSuccess) return e;
  }
  for (int seg = 0; seg < p.nseg; ++seg) {
    if (pipe && (e = hipStreamWaitEvent(s, pev[1 + seg], 0)) != hipSuccess) return fail(e);
    if ((e = launch_prefill_update(a, p, seg, s)) != hipSuccess) return fail(e);
    if (seg == p.nseg - 1 && (e = rec(3, s)) != hipSuccess) return fail(e);
    if (!a.skip_readout) {
      if ((e = rrec(seg, 0)) != hipSuccess) return fail(e);
      if ((e = launch_prefill_readout(a, p, seg, s)) != hipSuccess) return fail(e);
      if ((e = rrec(seg, 1)) != hipSuccess) return fail(e);
    }
  }
  // (the last segment's wait on pev[nseg] has joined the second stream)
  return rec(4, s);
}

}  // namespace dla
