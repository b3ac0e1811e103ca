// Measurement kernels: the dense bfloat16 MFMA rate and the HBM read bandwidth
// of the device (roofline denominators).  They compute nothing of the method.
#include "dla_peak.h"
#include "mfma.h"

namespace dla {

// Four waves per workgroup, four independent accumulator chains per wave, so
// that every SIMD always has an MFMA ready to issue.
__global__ __launch_bounds__(256) void peak_mfma_kernel(int iters, float* sink) {
  const int tid = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (float)((tid + e) & 7));
    b[e] = (__bf16)(0.002f * (float)((tid * 3 + e) & 7));
  }
  f32x16 c0 = zero16(), c1 = zero16(), c2 = zero16(), c3 = zero16();
  for (int i = 0; i < iters; ++i) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
  sink[(size_t)blockIdx.x * 256 + tid] = s;
}

// Grid-stride read of the buffer, four 16-byte non-temporal loads in flight
// per thread.
__global__ __launch_bounds__(256) void peak_read_kernel(const u32x4* p, size_t n16, float* sink) {
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 x0 = __builtin_nontemporal_load(p + i);
    const u32x4 x1 = __builtin_nontemporal_load(p + i + stride);
    const u32x4 x2 = __builtin_nontemporal_load(p + i + 2 * stride);
    const u32x4 x3 = __builtin_nontemporal_load(p + i + 3 * stride);
    acc ^= x0[0] ^ x1[1] ^ x2[2] ^ x3[3] ^ x0[3] ^ x1[2] ^ x2[1] ^ x3[0];
  }
  for (; i < n16; i += stride) {
    const u32x4 x = __builtin_nontemporal_load(p + i);
    acc ^= x[0] ^ x[1] ^ x[2] ^ x[3];
  }
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = __uint_as_float(acc & 0x3FFFFFFFu);
}

}  // namespace dla

using namespace dla;

extern "C" {

dla_status dla_peak_mfma_bf16(int32_t blocks, int32_t iters, float* sink, void* stream) {
  if (blocks <= 0 || iters <= 0 || !sink) return DLA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(peak_mfma_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters,
                     sink);
  return hipGetLastError() == hipSuccess ? DLA_OK : DLA_ERR_HIP;
}

dla_status dla_peak_hbm_read(const void* buf, size_t bytes, int32_t blocks, float* sink,
                             void* stream) {
  if (!buf || !sink || blocks <= 0 || bytes == 0 || (bytes & 4095u)) return DLA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(peak_read_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                     static_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? DLA_OK : DLA_ERR_HIP;
}

}  // extern "C"
