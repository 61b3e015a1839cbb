// Matrix-core rate probe: every wave runs kProbeChains independent chains of
// v_mfma_f32_32x32x16_bf16 on operands held in registers, so that the launch
// time is the matrix cores' alone.  The operands come from the workgroup index
// (unknown to the compiler) and the accumulated sum is stored only if it equals
// a value it cannot take, so no product is folded away.
#include "probe.h"

namespace mla {

__global__ __launch_bounds__(kProbeWaves * 64) void probe_mfma_kernel(int iters, float* sink) {
  const float x = 1.0f / (float)(blockIdx.x + 3);
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(x * (float)(e + 1));
    b[e] = (__bf16)(x * (float)(8 - e));
  }
  f32x16 c[kProbeChains];
#pragma unroll
  for (int k = 0; k < kProbeChains; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) c[k][e] = 0.f;
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int k = 0; k < kProbeChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[k], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kProbeChains; ++k) s += c[k][0] + c[k][15];
  if (s == -1.0f) sink[0] = s;   // the products are all positive
}

hipError_t launch_probe_mfma(int iters, int n_wg, float* sink, hipStream_t s) {
  probe_mfma_kernel<<<dim3((unsigned)n_wg), dim3(kProbeWaves * 64), 0, s>>>(iters, sink);
  return hipGetLastError();
}

}  // namespace mla
