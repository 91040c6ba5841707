// Measurement hook of the GPU library: the packed 16-bit VALU issue rate
// this device sustains, against which the search kernels' roofline
// fractions can also be read (the datasheet figure assumes every CU issues
// one wave64 instruction per clock at the peak engine clock).  The public
// entry point, hmm_probe_pk16, is in hmm_host.cpp.
//
// Every lane runs 16 independent chains of the MSV recurrence's two
// instructions (v_pk_add_f16, then a packed fp16 maximum), 32 waves per CU,
// so issue, not latency, bounds the kernel.  Each wave64 packed instruction
// counts 128 element-ops (64 lanes x 2 halves).
#include <hip/hip_runtime.h>

#include "hmm_internal.h"

namespace hmmgpu {
namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr int kChains = 16;

__global__ void __launch_bounds__(1024) pk16_probe_kernel(uint32_t *out, int iters, uint32_t seed) {
  h2 v[kChains];
  const uint32_t t = threadIdx.x + blockIdx.x * blockDim.x;
#pragma unroll
  for (int c = 0; c < kChains; c++) {
    const _Float16 x = (_Float16)(float)((t + c * 7 + seed) & 63);
    v[c] = h2{x, -x};
  }
  const h2 a = h2{(_Float16)1.0f, (_Float16)-1.0f}, b = h2{(_Float16)-2.0f, (_Float16)3.0f};
  for (int i = 0; i < iters; i++) {
#pragma unroll
    for (int c = 0; c < kChains; c++) v[c] = __builtin_elementwise_maximum(v[c] + a, b);
  }
  uint32_t acc = 0;
#pragma unroll
  for (int c = 0; c < kChains; c++) acc ^= __builtin_bit_cast(uint32_t, v[c]);
  out[t] = acc;
}

}  // namespace
}  // namespace hmmgpu

namespace hmmgpu {

hipError_t probe_pk16(uint32_t *scratch, int64_t scratch_words, hipStream_t s, double *ops_per_s, float *ms_out) {
  int dev = 0, ncu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int threads = 1024, iters = 4096;
  const int blocks = 2 * (ncu > 0 ? ncu : 256);
  if (scratch_words < (int64_t)threads * blocks) return hipErrorInvalidValue;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  // a warm-up launch, then the timed one
  if (e == hipSuccess) {
    hipLaunchKernelGGL(pk16_probe_kernel, dim3(blocks), dim3(threads), 0, s, scratch, iters, 1u);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(pk16_probe_kernel, dim3(blocks), dim3(threads), 0, s, scratch, iters, 2u);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.0f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (e != hipSuccess) return e;
  if (!(ms > 0.0f)) return hipErrorUnknown;
  const double instr = (double)blocks * (threads / 64) * iters * kChains * 2.0;   // wave64 instructions
  *ops_per_s = instr * 128.0 / (ms * 1e-3);
  if (ms_out) *ms_out = ms;
  return hipSuccess;
}

}  // namespace hmmgpu
