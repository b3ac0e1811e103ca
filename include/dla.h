/*
 * dla.h -- C ABI of libdla, the MI355X (gfx950) implementation of the Dynamic
 * Linear Attention (DLA) layer forward of arXiv 2606.10650: information-aware
 * dynamic state merging (Sec. 3.1, Alg. 1) and capacity-bounded memory with a
 * multi-state readout (Sec. 3.2, Alg. 2, eq. capacity_bounded_output).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Plain pointers and sizes only.  Every array argument is DEVICE memory owned
 *   by the caller; the library never allocates, frees or keeps a pointer after a
 *   call returns.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All work
 *   is enqueued on it; calls return after enqueueing.
 * - Synchronous argument errors return a status and enqueue nothing.  A launch
 *   failure returns DLA_ERR_HIP.  dla_get_last_error() returns the status of the
 *   calling thread's last call.  Nothing is thrown across the ABI.
 * - Calls on different caches may run concurrently; calls on one cache must be
 *   ordered (same stream, or synchronised by the caller).
 * - Shapes come from the cache descriptor: batch B, heads H, capacity C, key
 *   and value head dimensions d_k, d_v, and the storage type of the states.
 *   Supported: d_k, d_v in {64, 128}, 1 <= C <= 1024, B*H >= 1.  dla_prefill
 *   returns DLA_ERR_UNSUPPORTED when a stage's per-workgroup working set would
 *   not fit in 160 KiB of LDS; every shape of the supported set, in either
 *   input type, fits.
 * - The cache remembers the descriptor it was made with (its header, see
 *   below).  dla_prefill and dla_decode_step cannot read device memory on the
 *   host without synchronising, so every kernel they enqueue first compares
 *   the header with the descriptor it was given; on any difference (magic,
 *   version, B, H, C, d_k, d_v, state type) no kernel reads or writes a state,
 *   a metadata entry, an output, an export or the workspace, and the first
 *   kernel of the call sets DLA_FLAG_CACHE_MISMATCH in the header's device
 *   flags.  The outputs of such a call are left as they were.  The caller
 *   learns of it from dla_cache_flags (or dla_cache_header_check on a host
 *   copy of the header).  The cache buffer must hold at least its 256-byte
 *   header for this check to be safe.
 * - Token tensors are row-major [B][H][T][d] (d fastest); log_gate is
 *   [B][H][T] float32 (the per-token log-decay g_t <= 0 of the base model:
 *   every state decays by exp(g_t) at token t, the caller owns g_t <= 0);
 *   lambda is [B][H][T][C] in the input dtype, lambda[t][j] weights the state
 *   at chronological position j (0 = oldest) of the cache after token t is
 *   absorbed (eq. capacity_bounded_output; entries j >= m_t are ignored), NULL
 *   means lambda = 1.
 * - Per-token exports (each nullable): boundary int8 in {0,1} (b_t of Sec. 3.1;
 *   1 at the first token of an empty cache), merge_idx int32 (the chronological
 *   index i* in the pre-merge cache of the left state of the adjacent pair
 *   merged at token t by Alg. 2, or -1), score float32 (the State Information
 *   Score I_t of eq. importance_score; 0 at the first token of an empty cache).
 * - Overrides (each nullable, [B][H][T]): boundary_override -1 = decide, 0/1 =
 *   force b_t; merge_override -1 = decide, else force i* in [0, C-2].  An
 *   out-of-range merge override is ignored (the merge is decided) and sets
 *   DLA_FLAG_BAD_MERGE_OVERRIDE in the cache's device flags.  Overrides do not
 *   apply to the first token of an empty cache, and C = 1 forces b_t = 0 after
 *   it (no adjacent pair exists).
 */
#ifndef DLA_H
#define DLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DLA_OK = 0,
  DLA_ERR_INVALID_ARG = 1,    /* null pointer, bad size, bad dtype, T < 0 */
  DLA_ERR_UNSUPPORTED = 2,    /* head dimension, capacity or state type outside the supported set */
  DLA_ERR_CACHE_MISMATCH = 3, /* descriptor differs from the one the cache was made with
                                 (dla_cache_flags, dla_cache_header_check) */
  DLA_ERR_HIP = 4,            /* a HIP runtime call or kernel launch failed */
  DLA_ERR_WORKSPACE = 5       /* workspace missing or smaller than required */
} dla_status;

typedef enum { DLA_F32 = 0, DLA_BF16 = 1 } dla_dtype;

/* Shape of a state cache.  state_dtype is the storage type of the states:
 * DLA_F32 keeps every state in float32; DLA_BF16 keeps the states that no
 * token joins any more (every state but the newest of a head) in bfloat16 and
 * the newest state of each head in float32.  A closed state changes only when
 * Alg. 2 merges it with a neighbour, and each such merge is computed in
 * float32 from the stored values and rounded once to bfloat16, so bfloat16
 * storage halves the bytes a decode step streams at the cost of one rounding
 * (relative 2^-9) per closing and per merge.  The newest state, which the
 * State Information Score compares against (Sec. 3.1), stays float32, so the
 * boundary and merge decisions do not depend on the storage type. */
typedef struct {
  int32_t B, H, C, d_k, d_v;
  int32_t state_dtype; /* dla_dtype: DLA_F32 or DLA_BF16 */
} dla_cache_desc;

/* Layer parameters.  tau: boundary threshold (b_t = [I_t >= tau], Sec. 3.1);
 * eps: the epsilon of the score's denominator (eq. importance_score);
 * eps_rms: the epsilon of the RMSNorm applied to both states before scoring
 * (unit weight, over all d_k*d_v entries).
 * flags: DLA_SKIP_READOUT builds the cache and the exports but computes no
 * output (out may be NULL).  DLA_SERIAL_STAGES runs every stage of a prefill
 * on the caller's stream, one after another.  Without it, a prefill with a
 * readout and more than one chunk (512 tokens; 256 for float32 inputs) is
 * pipelined: it splits into segments of whole chunks and runs the sequential
 * boundary scan (Sec. 3.1-3.2), segment after segment, on a second stream
 * that the library forks from the caller's stream and joins back into it
 * before the call's last stage, while the caller's stream updates and reads
 * out the segments already scanned.  Results are identical either way; only
 * the workspace size differs (dla_prefill_workspace_size takes the flags).
 * The second stream and its events are created on a host thread's first
 * pipelined call on a device and kept, per thread and device, until the
 * process ends.
 * stage_events: NULL, or DLA_PREFILL_STAGES + 1 hipEvent_t handles (created by
 * the caller) that dla_prefill records before its first stage and after each
 * stage (token frames, boundary scan, state update, readout), for timing the
 * stages; dla_decode_step ignores it.  All are recorded on the caller's stream
 * except, in a pipelined call, the scan's, which is recorded on the second
 * stream after the last scan segment.  A call split into segments (pipelined,
 * or whose state copies exceed the workspace budget, see
 * dla_prefill_workspace_size) alternates the update and readout stages segment
 * by segment; the last two events then follow the last update and the last
 * readout.
 * readout_events, n_readout_events: NULL and 0, or n_readout_events hipEvent_t
 * handles; the readout launch of segment s is bracketed by events 2s (before)
 * and 2s + 1 (after), recorded on the caller's stream, for s <
 * n_readout_events / 2. */
typedef struct {
  float tau;
  float eps;
  float eps_rms;
  uint32_t flags;
  void* const* stage_events;
  void* const* readout_events;
  int32_t n_readout_events;
} dla_params;

#define DLA_PREFILL_STAGES 4

#define DLA_SKIP_READOUT 1u
#define DLA_SERIAL_STAGES 2u
/* Bits 8..15 of the flags set the budget of the readout's state copies (see
 * dla_prefill_workspace_size): DLA_POOL_BUDGET_LOG2(k) bounds them to 2^k
 * bytes per call, 20 <= k <= 40 (1 MiB .. 1 TiB); 0 keeps the default of
 * 8 GiB.  A smaller budget splits the call into more segments of whole
 * chunks (at least one chunk each, whatever the budget); results are
 * identical.  The same flags must reach dla_prefill_workspace_size,
 * dla_prefill_segment_count, dla_prefill_segment_starts and dla_prefill.
 * Any other k is DLA_ERR_INVALID_ARG. */
#define DLA_POOL_BUDGET_SHIFT 8
#define DLA_POOL_BUDGET_MASK 0xFF00u
#define DLA_POOL_BUDGET_LOG2(k) (((uint32_t)(k) << DLA_POOL_BUDGET_SHIFT) & DLA_POOL_BUDGET_MASK)

/* Device flags kept in the cache header (read with dla_cache_flags).
 * DLA_FLAG_BAD_MERGE_OVERRIDE: a merge override outside [0, C-2] was ignored.
 * DLA_FLAG_CACHE_MISMATCH: a prefill or decode step was given a descriptor
 * that differs from the cache's header, and did nothing. */
#define DLA_FLAG_BAD_MERGE_OVERRIDE 1u
#define DLA_FLAG_CACHE_MISMATCH 2u

/*
 * State cache (Sec. 3.2: chronological states with token counts n_i and
 * aggregated scores I_i, at most C of them), one per head.
 *
 * Layout of the cache buffer (all offsets in bytes, see dla_cache_layout):
 *   header  [0, 256): uint32 magic 0x31414C44 ('DLA1'), uint32 version (2),
 *           int32 B, H, C, d_k, d_v, uint32 device flags, int32 state_dtype,
 *           zero padding.
 *   per-head metadata at meta_offset + h * meta_stride, h = b*H + head:
 *           int32 m (live states), int32 0, double G (sum of all absorbed
 *           log-decays), int64 tokens absorbed, int64 0,
 *           double F[C] (frame of each live state), double Ibar[C] (aggregated
 *           score), int32 n[C] (token count), int32 perm[C] (physical slot of
 *           each logical state; entries m..C-1 list the free slots),
 *           then from a 64-byte boundary 64 bytes and float [16][d_v]:
 *           scratch for the decisions and the partial outputs of a decode step
 *           split over several workgroups.
 *           Arrays are in chronological order (index 0 = oldest).
 *   states  at states_offset: [B*H][C][d_k][d_v] by physical slot, in the
 *           state type.  The true state of logical state j is
 *           exp(G - F[j]) * stored slot perm[j] (states decay lazily: a slot is
 *           rescaled only when written).
 *   open    bfloat16 storage only, at open_offset: float32 [B*H][d_k][d_v],
 *           the newest state m-1 of each head, which then takes the place of
 *           its slot perm[m-1] (that slot is written when the state closes).
 *           open_offset is 0 for float32 storage.
 */
typedef struct {
  size_t meta_offset;
  size_t meta_stride;
  size_t states_offset;
  size_t open_offset;
  size_t total_bytes;
} dla_cache_layout;

/* Fill *layout for a descriptor.  Host only, no device work. */
dla_status dla_cache_layout_of(const dla_cache_desc* desc, dla_cache_layout* layout);

/* Two-call cache set-up.  With dev_buf == NULL: write the required size to
 * *bytes.  With a device buffer of at least *bytes bytes: enqueue its
 * initialisation to an empty cache (m = 0 for every head) on `stream`. */
dla_status dla_state_cache_alloc(const dla_cache_desc* desc, void* dev_buf, size_t* bytes,
                                 void* stream);

/* Copy the cache's device flags to *flags and clear them.  Synchronises
 * `stream`.  Returns DLA_ERR_CACHE_MISMATCH (and leaves the flags) when the
 * cache's header does not match desc. */
dla_status dla_cache_flags(const dla_cache_desc* desc, void* cache, uint32_t* flags,
                           void* stream);

/* Check a HOST copy of a cache header (its first 256 bytes, e.g. from a
 * checkpoint) against desc: DLA_OK and the device flags in *flags (nullable)
 * when magic, version, B, H, C, d_k, d_v and the state type all match,
 * DLA_ERR_CACHE_MISMATCH otherwise.  No device work. */
dla_status dla_cache_header_check(const dla_cache_desc* desc, const void* header,
                                  uint32_t* flags);

/* Workspace that dla_prefill needs for T tokens of the given input dtype and
 * params flags (DLA_SKIP_READOUT needs less: no state copies).  Besides O(T)
 * bytes per head (token frames, death tokens) and O(C) per head and chunk of
 * 512 tokens (256 for float32 inputs; the state list of every chunk), the
 * readout needs copies of the states in the input dtype: up to C per head and
 * chunk, d_k*d_v elements each.  They are bounded to 8 GiB per call (or the
 * budget set in the flags, DLA_POOL_BUDGET_LOG2): above that the call is split
 * into segments of whole chunks that reuse the space.
 * A pipelined call (see dla_params) splits into segments that grow by half
 * from one sixteenth of the chunks (2, 3, 5, 8 and 14 chunks at 16384 tokens).
 * Its segments share one pool when all its copies fit the budget; otherwise
 * none is larger than the budget allows and each reuses the space.  It also
 * keeps the scan's newest state (d_k*d_v floats per head) between segments. */
dla_status dla_prefill_workspace_size(const dla_cache_desc* desc, int32_t T, dla_dtype in_dtype,
                                      uint32_t flags, size_t* bytes);

/* Number of segments that dla_prefill splits T tokens of the given input
 * dtype and params flags into (see dla_params and dla_prefill_workspace_size),
 * written to *nseg; 1 when T is 0.  The readout then runs as that many
 * launches, which readout_events can bracket. */
dla_status dla_prefill_segment_count(const dla_cache_desc* desc, int32_t T, dla_dtype in_dtype,
                                     uint32_t flags, int32_t* nseg);

/* First token of each of those segments, in order: writes min(n, nseg)
 * entries to the HOST array starts (starts[0] = 0).  Host only. */
dla_status dla_prefill_segment_starts(const dla_cache_desc* desc, int32_t T, dla_dtype in_dtype,
                                      uint32_t flags, int32_t* starts, int32_t n);

/*
 * Prefill: absorb T tokens per head into the cache, in order, computing for
 * each token the score, the boundary decision, any capacity merge, and the
 * readout o_t = sum_j lambda[t][j] q_t^T S_j over the cache after token t
 * (eq. capacity_bounded_output; the first token of an empty cache opens a
 * state).  Continues from whatever the cache holds: prefill of T1 tokens
 * followed by prefill of T2 tokens equals prefill of T1 + T2 tokens.
 *
 * q (nullable with DLA_SKIP_READOUT), k: [B][H][T][d_k] in_dtype;
 * v: [B][H][T][d_v] in_dtype; log_gate: [B][H][T] float32; lambda: see above;
 * out: [B][H][T][d_v] out_dtype (nullable with DLA_SKIP_READOUT);
 * exports and overrides: see above.  workspace: at least
 * dla_prefill_workspace_size() bytes of device memory, 256-byte aligned.
 * T = 0 is a no-op.
 */
dla_status dla_prefill(const dla_cache_desc* desc, void* cache, const void* q, const void* k,
                       const void* v, const float* log_gate, const void* lambda, int32_t T,
                       dla_dtype in_dtype, const dla_params* params, void* out,
                       dla_dtype out_dtype, int8_t* boundary, int32_t* merge_idx, float* score,
                       const int8_t* boundary_override, const int32_t* merge_override,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * dla_prefill for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, results and errors as dla_prefill, without the workspace.
 * Its workspace is a static device array of DLA_STATIC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends; nothing is
 * allocated by the call.  The stages always run serially on `stream` (no
 * second stream or event is created; DLA_SERIAL_STAGES is implied).  A call
 * whose workspace (dla_prefill_workspace_size with DLA_SERIAL_STAGES) exceeds
 * DLA_STATIC_SCRATCH_BYTES returns DLA_ERR_WORKSPACE and enqueues nothing.
 * Every call on a device shares that device's array, and no part of it needs
 * clearing between calls: calls that overlap on one device race (order them on
 * one stream).
 */
#define DLA_STATIC_SCRATCH_BYTES ((size_t)128 << 20)
dla_status dla_prefill_static(const dla_cache_desc* desc, void* cache, const void* q,
                              const void* k, const void* v, const float* log_gate,
                              const void* lambda, int32_t T, dla_dtype in_dtype,
                              const dla_params* params, void* out, dla_dtype out_dtype,
                              int8_t* boundary, int32_t* merge_idx, float* score,
                              const int8_t* boundary_override, const int32_t* merge_override,
                              void* stream);

/*
 * Decode step: absorb one token per head (the prefill semantics with T = 1),
 * streaming every live state once.  With few heads the step splits each head's
 * states over up to 16 workgroups, which leave partial outputs in the scratch
 * area of the head's metadata; a second kernel on the same stream sums them in
 * a fixed order (results are deterministic) and ends the step.  q, k: [B][H][d_k]; v, out: [B][H][d_v];
 * log_gate: [B][H]; lambda: [B][H][C] (nullable); exports and overrides:
 * [B][H] (nullable).  Needs no workspace.
 */
dla_status dla_decode_step(const dla_cache_desc* desc, void* cache, const void* q, const void* k,
                           const void* v, const float* log_gate, const void* lambda,
                           dla_dtype in_dtype, const dla_params* params, void* out,
                           dla_dtype out_dtype, int8_t* boundary, int32_t* merge_idx,
                           float* score, const int8_t* boundary_override,
                           const int32_t* merge_override, void* stream);

/*
 * Gated DeltaNet form of the layer (Sec. 2.2, eq. delta_rule_rnn; the paper
 * applies DLA to that backbone as well).  beta: float32 step sizes, [B][H] for
 * a decode step, [B][H][T] for a sequence, not null.  The newest state follows
 * the delta rule while tokens accumulate into it (Sec. 3.1 update rule, b_t =
 * 0): with every state first decayed by exp(g_t),
 *   S <- (I - beta_t k_t k_t^T) S + beta_t k_t v_t^T,
 * and a boundary opens the new state beta_t k_t v_t^T (b_t = 1).  Closed states
 * are summaries and only decay; merges (Alg. 2), scores, decisions and the
 * readout are those of dla_decode_step (the score compares k_t v_t^T with the
 * newest state before the token's update; it is scale-invariant, so beta does
 * not enter it).  With C = 1 the layer is the Gated DeltaNet recurrence.
 * Same cache as dla_prefill / dla_decode_step (either may continue a cache
 * the other built, in the same form).
 */
dla_status dla_decode_step_delta(const dla_cache_desc* desc, void* cache, const void* q,
                                 const void* k, const void* v, const float* log_gate,
                                 const float* beta, const void* lambda, dla_dtype in_dtype,
                                 const dla_params* params, void* out, dla_dtype out_dtype,
                                 int8_t* boundary, int32_t* merge_idx, float* score,
                                 const int8_t* boundary_override, const int32_t* merge_override,
                                 void* stream);

/*
 * Workspace of dla_prefill_delta for T tokens per head (same meaning of flags
 * as dla_prefill_workspace_size: DLA_SKIP_READOUT, DLA_SERIAL_STAGES,
 * DLA_POOL_BUDGET_LOG2).
 */
dla_status dla_prefill_delta_workspace_size(const dla_cache_desc* desc, int32_t T,
                                            dla_dtype in_dtype, uint32_t flags, size_t* bytes);

/*
 * T tokens per head in the Gated DeltaNet form (the rule of
 * dla_decode_step_delta), with the arrays of dla_prefill ([B][H][T][d] tokens,
 * [B][H][T] log_gate, beta, exports and overrides, [B][H][T][C] lambda).
 * A token that joins the newest state adds k_t u_t^T to the decayed state,
 * with pseudo-value u_t = beta_t (v_t - (alpha_t S)^T k_t); a token that opens
 * one starts it at k_t (beta_t v_t)^T.  Every state is therefore the decayed
 * sum of k_s u_s^T over its tokens: a sequential scan (one workgroup per head,
 * the newest state on chip) makes the decisions and the pseudo-values, and the
 * chunked update and readout stages of dla_prefill run on (q, k, u, lambda)
 * (u kept in float32 for the states; a bfloat16 copy for the readout of
 * 16-bit inputs).  The stages follow dla_prefill's schedule: pipelined (the
 * scan in segments on the library's second stream, joined back into `stream`
 * before the call's last stage), or in order on `stream` with
 * DLA_SERIAL_STAGES; results are identical either way.  The workspace
 * (dla_prefill_delta_workspace_size bytes for the same flags, 256-byte
 * aligned, caller-owned) must not be used by another call until the stream
 * has passed this one.  Errors as dla_prefill; DLA_ERR_UNSUPPORTED where the
 * stages do not fit.
 */
dla_status dla_prefill_delta(const dla_cache_desc* desc, void* cache, const void* q, const void* k,
                             const void* v, const float* log_gate, const float* beta,
                             const void* lambda, int32_t T, dla_dtype in_dtype,
                             const dla_params* params, void* out, dla_dtype out_dtype,
                             int8_t* boundary, int32_t* merge_idx, float* score,
                             const int8_t* boundary_override, const int32_t* merge_override,
                             void* workspace, size_t workspace_bytes, void* stream);

const char* dla_status_string(dla_status s);
dla_status dla_get_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DLA_H */
