// Segmented log-sum-exp merge of per-segment attention partials (Alg. 2,
// SegmentedLSEMerge).  Bandwidth-bound: each slot's partials are streamed once
// with 16-byte loads and the merged row is written once.
#include "common.h"

namespace mla {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// One 64-lane wave per slot, 4 slots per 256-thread block.  Lane l owns the
// float4 columns l, l+64, ... of the head-output row (d_c wide, or d_c + d_r
// with a rotary value: the merge is linear, so both parts merge alike).
// n_slots_dev, if set, holds the slot count (n_slots is then the bound of the grid).
template <int DC, bool OUT_BF16>
__global__ __launch_bounds__(256) void merge_kernel(int64_t n_slots, const int64_t* __restrict__ n_slots_dev,
                                                    const float* __restrict__ part_o,
                                                    const float* __restrict__ part_lse,
                                                    const int64_t* __restrict__ part_ptr,
                                                    void* __restrict__ out_o, float* __restrict__ out_lse) {
  constexpr int NV = DC / 4;                  // float4 per row
  constexpr int PER = (NV + 63) / 64;         // float4 per lane
  const int lane = threadIdx.x & 63;
  const int64_t slot = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (slot >= (n_slots_dev != nullptr ? *n_slots_dev : n_slots)) return;
  const int64_t p0 = part_ptr[slot];
  const int n = (int)(part_ptr[slot + 1] - p0);

  f32x4 acc[PER];
  float m = -INFINITY, wsum = 0.f;
  if (n == 1) {
#pragma unroll
    for (int v = 0; v < PER; ++v) {
      const int c = lane + 64 * v;
      if (c < NV) acc[v] = *(const f32x4*)(part_o + p0 * DC + 4 * c);
    }
    m = part_lse[p0];
    wsum = 1.f;
  } else {
    for (int i = lane; i < n; i += 64) m = fmaxf(m, part_lse[p0 + i]);
    m = wave_max(m);
#pragma unroll
    for (int v = 0; v < PER; ++v) acc[v] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int i = 0; i < n; ++i) {
      const float w = expf(part_lse[p0 + i] - m);
      wsum += w;
      const float* src = part_o + (p0 + i) * DC;
#pragma unroll
      for (int v = 0; v < PER; ++v) {
        const int c = lane + 64 * v;
        if (c < NV) {
          const f32x4 x = *(const f32x4*)(src + 4 * c);
          acc[v] += w * x;
        }
      }
    }
    const float inv = 1.f / wsum;
#pragma unroll
    for (int v = 0; v < PER; ++v) acc[v] *= inv;
  }
#pragma unroll
  for (int v = 0; v < PER; ++v) {
    const int c = lane + 64 * v;
    if (c >= NV) continue;
    if constexpr (OUT_BF16) {
      u32x2 pk;
      pk[0] = pack_bf16x2(acc[v][0], acc[v][1]);
      pk[1] = pack_bf16x2(acc[v][2], acc[v][3]);
      *(u32x2*)((uint16_t*)out_o + slot * DC + 4 * c) = pk;
    } else {
      *(f32x4*)((float*)out_o + slot * DC + 4 * c) = acc[v];
    }
  }
  if (out_lse != nullptr && lane == 0) out_lse[slot] = m + logf(wsum);
}

hipError_t launch_merge(int64_t n_slots, int32_t d_latent, const float* part_o, const float* part_lse,
                        const int64_t* part_ptr, int32_t out_dtype, void* out_o, float* out_lse,
                        hipStream_t s, const int64_t* n_slots_dev) {
  if (n_slots == 0) return hipSuccess;
  const dim3 grid((unsigned)((n_slots + 3) / 4)), block(256);
  const bool bf = out_dtype == MLA_BF16;
#define MLA_MERGE(DC)                                                                                     \
  (bf ? merge_kernel<DC, true><<<grid, block, 0, s>>>(n_slots, n_slots_dev, part_o, part_lse, part_ptr,  \
                                                      out_o, out_lse)                                    \
      : merge_kernel<DC, false><<<grid, block, 0, s>>>(n_slots, n_slots_dev, part_o, part_lse, part_ptr, \
                                                       out_o, out_lse))
  if (d_latent == 512)
    MLA_MERGE(512);
  else if (d_latent == 576)   // rotary value: latent and RoPE dims
    MLA_MERGE(576);
  else
    MLA_MERGE(64);
#undef MLA_MERGE
  return hipGetLastError();
}

}  // namespace mla
