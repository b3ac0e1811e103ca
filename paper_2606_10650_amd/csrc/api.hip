// Host side of libdla: argument validation, cache set-up and the launch
// sequence of each entry point.  Every entry point enqueues on the caller's
// stream and never allocates device memory.
#include <string.h>

#include <mutex>
#include <vector>

#include "dla_common.h"
#include "prefill.h"
#include "decode.h"

namespace dla {

// Pipelined prefills fork a second stream from the caller's.  Each host thread
// gets its own stream and events per device, so concurrent calls from several
// threads never share an event; they live until the process ends.
hipError_t pipe_resources(hipStream_t caller, int n, hipStream_t* side, hipEvent_t** evs) {
  struct PerDevice {
    hipStream_t side = nullptr;
    std::vector<hipEvent_t> ev;
  };
  static thread_local std::vector<PerDevice> per;
  // the device of the caller's stream (the current device for the null
  // stream); the second stream and the events are made on it
  int dev = 0, cur = 0;
  hipError_t e = hipStreamGetDevice(caller, &dev);
  if (e != hipSuccess) return e;
  if (dev < 0) return hipErrorInvalidDevice;
  if ((int)per.size() <= dev) per.resize(dev + 1);
  PerDevice& pd = per[dev];
  if (!pd.side || (int)pd.ev.size() < n) {
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    if (!pd.side && (e = hipStreamCreateWithFlags(&pd.side, hipStreamNonBlocking)) != hipSuccess)
      pd.side = nullptr;
    while (e == hipSuccess && (int)pd.ev.size() < n) {
      hipEvent_t x;
      if ((e = hipEventCreateWithFlags(&x, hipEventDisableTiming)) == hipSuccess) pd.ev.push_back(x);
    }
    const hipError_t r = (cur != dev) ? hipSetDevice(cur) : hipSuccess;
    if (e != hipSuccess) return e;
    if (r != hipSuccess) return r;
  }
  *side = pd.side;
  *evs = pd.ev.data();
  return hipSuccess;
}


// Workspace of dla_prefill_static: a file-scope device array, one copy per
// device the library runs on, kept until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in for
// the symbol): the device address of this device's copy comes from
// hipGetSymbolAddress, taken once per device with that device current.
static __device__ __align__(256) char scratch[DLA_STATIC_SCRATCH_BYTES];

hipError_t static_scratch(hipStream_t caller, void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0, cur = 0;
  hipError_t e = hipStreamGetDevice(caller, &dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    const hipError_t r = (cur != dev) ? hipSetDevice(cur) : hipSuccess;
    if (e != hipSuccess) return e;
    if (r != hipSuccess) return r;
    if (!p || ((uintptr_t)p & 255u)) return hipErrorInvalidValue;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

__global__ void cache_init_kernel(char* cache, dla_cache_desc d, size_t meta_offset,
                                  size_t meta_stride) {
  const int h = blockIdx.x;
  if (h == 0 && threadIdx.x == 0) {
    CacheHeader* hd = reinterpret_cast<CacheHeader*>(cache);
    hd->magic = kMagic;
    hd->version = kVersion;
    hd->B = d.B;
    hd->H = d.H;
    hd->C = d.C;
    hd->dk = d.d_k;
    hd->dv = d.d_v;
    hd->flags = 0u;
    hd->state_dtype = d.state_dtype;
  }
  Meta M = meta_at(cache + meta_offset + (size_t)h * meta_stride, d.C);
  if (threadIdx.x == 0) {
    *M.m = 0;
    *reinterpret_cast<int32_t*>(cache + meta_offset + (size_t)h * meta_stride + 4) = 0;
    *M.G = 0.0;
    *M.tokens = 0;
    *reinterpret_cast<int64_t*>(cache + meta_offset + (size_t)h * meta_stride + 24) = 0;
  }
  for (int j = threadIdx.x; j < d.C; j += blockDim.x) {
    M.F[j] = 0.0;
    M.ibar[j] = 0.0;
    M.n[j] = 0;
    M.perm[j] = j;
  }
}

__global__ void flags_clear_kernel(char* cache) {
  if (threadIdx.x == 0) reinterpret_cast<CacheHeader*>(cache)->flags = 0u;
}

}  // namespace dla

using namespace dla;

static thread_local dla_status g_last = DLA_OK;

static dla_status ret(dla_status s) {
  g_last = s;
  return s;
}

static dla_status check_desc(const dla_cache_desc* d) {
  if (!d) return DLA_ERR_INVALID_ARG;
  if (d->B < 1 || d->H < 1 || d->C < 1) return DLA_ERR_INVALID_ARG;
  if (d->C > 1024) return DLA_ERR_UNSUPPORTED;
  if ((d->d_k != 64 && d->d_k != 128) || (d->d_v != 64 && d->d_v != 128))
    return DLA_ERR_UNSUPPORTED;
  if ((int64_t)d->B * d->H > (int64_t)1 << 24) return DLA_ERR_UNSUPPORTED;
  if (d->state_dtype != DLA_F32 && d->state_dtype != DLA_BF16) return DLA_ERR_INVALID_ARG;
  return DLA_OK;
}

static bool dtype_ok(dla_dtype t) { return t == DLA_F32 || t == DLA_BF16; }

extern "C" {

const char* dla_status_string(dla_status s) {
  switch (s) {
    case DLA_OK: return "ok";
    case DLA_ERR_INVALID_ARG: return "invalid argument";
    case DLA_ERR_UNSUPPORTED: return "unsupported shape";
    case DLA_ERR_CACHE_MISMATCH: return "cache does not match the descriptor";
    case DLA_ERR_HIP: return "HIP runtime error";
    case DLA_ERR_WORKSPACE: return "workspace missing or too small";
  }
  return "unknown status";
}

dla_status dla_get_last_error(void) { return g_last; }

dla_status dla_cache_layout_of(const dla_cache_desc* desc, dla_cache_layout* layout) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  if (!layout) return ret(DLA_ERR_INVALID_ARG);
  *layout = layout_of(*desc);
  return ret(DLA_OK);
}

dla_status dla_state_cache_alloc(const dla_cache_desc* desc, void* dev_buf, size_t* bytes,
                                 void* stream) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  if (!bytes) return ret(DLA_ERR_INVALID_ARG);
  const dla_cache_layout L = layout_of(*desc);
  if (!dev_buf) {
    *bytes = L.total_bytes;
    return ret(DLA_OK);
  }
  if (*bytes < L.total_bytes) return ret(DLA_ERR_INVALID_ARG);
  const int nh = desc->B * desc->H;
  hipLaunchKernelGGL(cache_init_kernel, dim3(nh), dim3(256), 0, (hipStream_t)stream,
                     (char*)dev_buf, *desc, L.meta_offset, L.meta_stride);
  if (hipGetLastError() != hipSuccess) return ret(DLA_ERR_HIP);
  return ret(DLA_OK);
}

dla_status dla_cache_flags(const dla_cache_desc* desc, void* cache, uint32_t* flags,
                           void* stream) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  if (!cache || !flags) return ret(DLA_ERR_INVALID_ARG);
  CacheHeader hd;
  hipStream_t st = (hipStream_t)stream;
  if (hipMemcpyAsync(&hd, cache, sizeof(hd), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return ret(DLA_ERR_HIP);
  if (!header_matches(hd, *desc)) return ret(DLA_ERR_CACHE_MISMATCH);
  *flags = hd.flags;
  hipLaunchKernelGGL(flags_clear_kernel, dim3(1), dim3(64), 0, st, (char*)cache);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(st) != hipSuccess)
    return ret(DLA_ERR_HIP);
  return ret(DLA_OK);
}

dla_status dla_cache_header_check(const dla_cache_desc* desc, const void* header,
                                  uint32_t* flags) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  if (!header) return ret(DLA_ERR_INVALID_ARG);
  CacheHeader hd;
  memcpy(&hd, header, sizeof(hd));
  if (!header_matches(hd, *desc)) return ret(DLA_ERR_CACHE_MISMATCH);
  if (flags) *flags = hd.flags;
  return ret(DLA_OK);
}

dla_status dla_prefill_workspace_size(const dla_cache_desc* desc, int32_t T, dla_dtype in_dtype,
                                      uint32_t flags, size_t* bytes) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  const size_t budget = pool_budget_of(flags);
  if (!bytes || T < 0 || !dtype_ok(in_dtype) || !budget) return ret(DLA_ERR_INVALID_ARG);
  *bytes = prefill_workspace_bytes(*desc, T, in_dtype, (flags & DLA_SKIP_READOUT) == 0,
                                   (flags & DLA_SERIAL_STAGES) != 0, budget);
  return ret(DLA_OK);
}

dla_status dla_prefill_segment_count(const dla_cache_desc* desc, int32_t T, dla_dtype in_dtype,
                                     uint32_t flags, int32_t* nseg) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  const size_t budget = pool_budget_of(flags);
  if (!nseg || T < 0 || !dtype_ok(in_dtype) || !budget) return ret(DLA_ERR_INVALID_ARG);
  *nseg = seg_plan(*desc, T, in_dtype, (flags & DLA_SKIP_READOUT) == 0,
                   (flags & DLA_SERIAL_STAGES) != 0, budget).nseg;
  return ret(DLA_OK);
}

dla_status dla_prefill_segment_starts(const dla_cache_desc* desc, int32_t T, dla_dtype in_dtype,
                                      uint32_t flags, int32_t* starts, int32_t n) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  const size_t budget = pool_budget_of(flags);
  if (!starts || n < 0 || T < 0 || !dtype_ok(in_dtype) || !budget) return ret(DLA_ERR_INVALID_ARG);
  const SegPlan p = seg_plan(*desc, T, in_dtype, (flags & DLA_SKIP_READOUT) == 0,
                             (flags & DLA_SERIAL_STAGES) != 0, budget);
  for (int seg = 0; seg < p.nseg && seg < n; ++seg) {
    int cs, ce;
    seg_range(p, seg, &cs, &ce);
    starts[seg] = cs * p.RL < T ? cs * p.RL : T;
  }
  return ret(DLA_OK);
}

// The body of dla_prefill and dla_prefill_static.  static_ws: the workspace
// is this device's static scratch (stages forced serial, so that no stream or
// event is ever created; the workspace arguments are ignored).
static dla_status prefill_impl(const dla_cache_desc* desc, void* cache, const void* q,
                               const void* k, const void* v, const float* log_gate,
                               const void* lambda, int32_t T, dla_dtype in_dtype,
                               const dla_params* params, void* out, dla_dtype out_dtype,
                               int8_t* boundary, int32_t* merge_idx, float* score,
                               const int8_t* boundary_override, const int32_t* merge_override,
                               void* workspace, size_t workspace_bytes, void* stream,
                               bool static_ws) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  if (!params || T < 0 || !dtype_ok(in_dtype) || !dtype_ok(out_dtype)) return ret(DLA_ERR_INVALID_ARG);
  const bool skip = (params->flags & DLA_SKIP_READOUT) != 0;
  if (!cache || !k || !v || !log_gate) return ret(DLA_ERR_INVALID_ARG);
  if (!skip && (!q || !out)) return ret(DLA_ERR_INVALID_ARG);
  if (T == 0) return ret(DLA_OK);
  if (!prefill_chunks_supported(*desc, in_dtype)) return ret(DLA_ERR_UNSUPPORTED);
  if ((int64_t)desc->B * desc->H * (int64_t)T * (desc->C > 128 ? desc->C : 128) >
      ((int64_t)1 << 40))
    return ret(DLA_ERR_UNSUPPORTED);
  const bool serial = static_ws || (params->flags & DLA_SERIAL_STAGES) != 0;
  const size_t budget = pool_budget_of(params->flags);
  if (!budget) return ret(DLA_ERR_INVALID_ARG);
  if (params->n_readout_events < 0 || (params->n_readout_events > 0 && !params->readout_events))
    return ret(DLA_ERR_INVALID_ARG);
  const size_t need = prefill_workspace_bytes(*desc, T, in_dtype, !skip, serial, budget);
  if (static_ws) {
    if (need > DLA_STATIC_SCRATCH_BYTES) return ret(DLA_ERR_WORKSPACE);
    if (static_scratch((hipStream_t)stream, &workspace) != hipSuccess) return ret(DLA_ERR_HIP);
    workspace_bytes = DLA_STATIC_SCRATCH_BYTES;
  }
  if (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 255u))
    return ret(DLA_ERR_WORKSPACE);
  PrefillArgs a;
  memset(&a, 0, sizeof(a));
  const dla_cache_layout L = layout_of(*desc);
  a.desc = *desc;
  a.cache = (char*)cache;
  a.meta_offset = L.meta_offset;
  a.meta_stride = L.meta_stride;
  a.states_offset = L.states_offset;
  a.open_offset = L.open_offset;
  a.q = q;
  a.k = k;
  a.v = v;
  a.g = log_gate;
  a.lam = lambda;
  a.out = skip ? nullptr : out;
  a.b_out = boundary;
  a.merge_out = merge_idx;
  a.score_out = score;
  a.b_ovr = boundary_override;
  a.m_ovr = merge_override;
  a.T = T;
  a.tau = params->tau;
  a.eps = params->eps;
  a.eps_rms = params->eps_rms;
  a.skip_readout = skip ? 1 : 0;
  a.in_dtype = in_dtype;
  a.out_dtype = out_dtype;
  a.serial = serial ? 1 : 0;
  a.pool_budget = budget;
  a.workspace = (char*)workspace;
  StageEvents se;
  se.ev = params->stage_events;
  se.rev = params->readout_events;
  se.nrev = params->n_readout_events;
  if (launch_prefill(a, (hipStream_t)stream, se) != hipSuccess)
    return ret(DLA_ERR_HIP);
  return ret(DLA_OK);
}

dla_status dla_prefill(const dla_cache_desc* desc, void* cache, const void* q, const void* k,
                       const void* v, const float* log_gate, const void* lambda, int32_t T,
                       dla_dtype in_dtype, const dla_params* params, void* out,
                       dla_dtype out_dtype, int8_t* boundary, int32_t* merge_idx, float* score,
                       const int8_t* boundary_override, const int32_t* merge_override,
                       void* workspace, size_t workspace_bytes, void* stream) {
  return prefill_impl(desc, cache, q, k, v, log_gate, lambda, T, in_dtype, params, out, out_dtype,
                      boundary, merge_idx, score, boundary_override, merge_override, workspace,
                      workspace_bytes, stream, false);
}

dla_status dla_prefill_static(const dla_cache_desc* desc, void* cache, const void* q,
                              const void* k, const void* v, const float* log_gate,
                              const void* lambda, int32_t T, dla_dtype in_dtype,
                              const dla_params* params, void* out, dla_dtype out_dtype,
                              int8_t* boundary, int32_t* merge_idx, float* score,
                              const int8_t* boundary_override, const int32_t* merge_override,
                              void* stream) {
  return prefill_impl(desc, cache, q, k, v, log_gate, lambda, T, in_dtype, params, out, out_dtype,
                      boundary, merge_idx, score, boundary_override, merge_override, nullptr, 0,
                      stream, true);
}

}  // extern "C"

// One decode step for every head, or step t of a sequence (hs = T): the
// per-token arrays are passed already offset to the step's token.
static dla_status decode_impl(const dla_cache_desc* desc, void* cache, const void* q, const void* k,
                              const void* v, const float* log_gate, const float* beta,
                              const void* lambda, dla_dtype in_dtype, const dla_params* params,
                              void* out, dla_dtype out_dtype, int8_t* boundary, int32_t* merge_idx,
                              float* score, const int8_t* boundary_override,
                              const int32_t* merge_override, long long hs, void* stream) {
  const bool skip = (params->flags & DLA_SKIP_READOUT) != 0;
  const dla_cache_layout L = layout_of(*desc);
  DecodeArgs a;
  memset(&a, 0, sizeof(a));
  a.desc = *desc;
  a.cache = (char*)cache;
  a.meta_offset = L.meta_offset;
  a.meta_stride = L.meta_stride;
  a.states_offset = L.states_offset;
  a.open_offset = L.open_offset;
  a.nsplit = decode_splits(desc->B * desc->H, desc->C);
  a.q = q;
  a.k = k;
  a.v = v;
  a.g = log_gate;
  a.lam = lambda;
  a.out = out;
  a.b_out = boundary;
  a.merge_out = merge_idx;
  a.score_out = score;
  a.b_ovr = boundary_override;
  a.m_ovr = merge_override;
  a.beta = beta;
  a.hs = hs;
  a.tau = params->tau;
  a.eps = params->eps;
  a.eps_rms = params->eps_rms;
  a.skip_readout = skip ? 1 : 0;
  if (launch_decode(a, desc->B * desc->H, desc->d_k, desc->d_v, in_dtype, out_dtype,
                    (hipStream_t)stream) != hipSuccess)
    return DLA_ERR_HIP;
  return DLA_OK;
}

static dla_status decode_check(const dla_cache_desc* desc, void* cache, const void* q,
                               const void* k, const void* v, const float* log_gate,
                               dla_dtype in_dtype, const dla_params* params, void* out,
                               dla_dtype out_dtype) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return s;
  if (!params || !dtype_ok(in_dtype) || !dtype_ok(out_dtype)) return DLA_ERR_INVALID_ARG;
  const bool skip = (params->flags & DLA_SKIP_READOUT) != 0;
  if (!cache || !k || !v || !log_gate) return DLA_ERR_INVALID_ARG;
  if (!skip && (!q || !out)) return DLA_ERR_INVALID_ARG;
  return DLA_OK;
}

extern "C" {

dla_status dla_decode_step(const dla_cache_desc* desc, void* cache, const void* q, const void* k,
                           const void* v, const float* log_gate, const void* lambda,
                           dla_dtype in_dtype, const dla_params* params, void* out,
                           dla_dtype out_dtype, int8_t* boundary, int32_t* merge_idx,
                           float* score, const int8_t* boundary_override,
                           const int32_t* merge_override, void* stream) {
  dla_status s = decode_check(desc, cache, q, k, v, log_gate, in_dtype, params, out, out_dtype);
  if (s != DLA_OK) return ret(s);
  return ret(decode_impl(desc, cache, q, k, v, log_gate, nullptr, lambda, in_dtype, params, out,
                         out_dtype, boundary, merge_idx, score, boundary_override, merge_override,
                         1, stream));
}

dla_status dla_decode_step_delta(const dla_cache_desc* desc, void* cache, const void* q,
                                 const void* k, const void* v, const float* log_gate,
                                 const float* beta, const void* lambda, dla_dtype in_dtype,
                                 const dla_params* params, void* out, dla_dtype out_dtype,
                                 int8_t* boundary, int32_t* merge_idx, float* score,
                                 const int8_t* boundary_override, const int32_t* merge_override,
                                 void* stream) {
  dla_status s = decode_check(desc, cache, q, k, v, log_gate, in_dtype, params, out, out_dtype);
  if (s != DLA_OK) return ret(s);
  if (!beta) return ret(DLA_ERR_INVALID_ARG);
  return ret(decode_impl(desc, cache, q, k, v, log_gate, beta, lambda, in_dtype, params, out,
                         out_dtype, boundary, merge_idx, score, boundary_override, merge_override,
                         1, stream));
}

dla_status dla_prefill_delta_workspace_size(const dla_cache_desc* desc, int32_t T,
                                            dla_dtype in_dtype, uint32_t flags, size_t* bytes) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  const size_t budget = pool_budget_of(flags);
  if (!bytes || T < 0 || !dtype_ok(in_dtype) || !budget) return ret(DLA_ERR_INVALID_ARG);
  *bytes = prefill_delta_workspace_bytes(*desc, T, in_dtype, (flags & DLA_SKIP_READOUT) == 0,
                                         (flags & DLA_SERIAL_STAGES) != 0, budget);
  return ret(DLA_OK);
}

dla_status dla_prefill_delta(const dla_cache_desc* desc, void* cache, const void* q, const void* k,
                             const void* v, const float* log_gate, const float* beta,
                             const void* lambda, int32_t T, dla_dtype in_dtype,
                             const dla_params* params, void* out, dla_dtype out_dtype,
                             int8_t* boundary, int32_t* merge_idx, float* score,
                             const int8_t* boundary_override, const int32_t* merge_override,
                             void* workspace, size_t workspace_bytes, void* stream) {
  dla_status s = check_desc(desc);
  if (s != DLA_OK) return ret(s);
  if (!params || T < 0 || !dtype_ok(in_dtype) || !dtype_ok(out_dtype)) return ret(DLA_ERR_INVALID_ARG);
  const bool skip = (params->flags & DLA_SKIP_READOUT) != 0;
  if (!cache || !k || !v || !log_gate || !beta) return ret(DLA_ERR_INVALID_ARG);
  if (!skip && (!q || !out)) return ret(DLA_ERR_INVALID_ARG);
  if (T == 0) return ret(DLA_OK);
  // the update and readout stages in the inputs' type, and the sequential scan's LDS
  if (!prefill_chunks_supported(*desc, in_dtype) || prefill_delta_scan_smem(*desc) > 160 * 1024)
    return ret(DLA_ERR_UNSUPPORTED);
  if ((int64_t)desc->B * desc->H * (int64_t)T * (desc->C > 128 ? desc->C : 128) >
      ((int64_t)1 << 40))
    return ret(DLA_ERR_UNSUPPORTED);
  const size_t budget = pool_budget_of(params->flags);
  if (!budget) return ret(DLA_ERR_INVALID_ARG);
  const bool serial = (params->flags & DLA_SERIAL_STAGES) != 0;
  const size_t need = prefill_delta_workspace_bytes(*desc, T, in_dtype, !skip, serial, budget);
  if (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 255u))
    return ret(DLA_ERR_WORKSPACE);
  PrefillArgs a;
  memset(&a, 0, sizeof(a));
  const dla_cache_layout L = layout_of(*desc);
  a.desc = *desc;
  a.cache = (char*)cache;
  a.meta_offset = L.meta_offset;
  a.meta_stride = L.meta_stride;
  a.states_offset = L.states_offset;
  a.open_offset = L.open_offset;
  a.q = q;
  a.k = k;
  a.v = v;
  a.g = log_gate;
  a.lam = lambda;
  a.out = skip ? nullptr : out;
  a.b_out = boundary;
  a.merge_out = merge_idx;
  a.score_out = score;
  a.b_ovr = boundary_override;
  a.m_ovr = merge_override;
  a.T = T;
  a.tau = params->tau;
  a.eps = params->eps;
  a.eps_rms = params->eps_rms;
  a.skip_readout = skip ? 1 : 0;
  a.in_dtype = in_dtype;
  a.out_dtype = out_dtype;
  a.serial = serial ? 1 : 0;
  a.pool_budget = budget;
  a.workspace = (char*)workspace;
  if (launch_prefill_delta(a, beta, (hipStream_t)stream) != hipSuccess) return ret(DLA_ERR_HIP);
  return ret(DLA_OK);
}

}  // extern "C"
