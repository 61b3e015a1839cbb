// Adaptive MoE fanout (Sec. 2.4, eq:moe).  For each token row the router's
// top_k experts (the paper's Top-6) are ranked by weight, their weights are
// normalized only to choose the fanout
//   K = min{k in [min_k, top_k] : sum_{j<=k} p_(j) / sum_{r<=top_k} p_(r) >= tau}
// (top_k when no k qualifies), and the executed experts keep their original
// weights.  The integer K is decided in float32, in rank order: the sum of the
// top_k weights left to right, each share a correctly rounded division, the
// shares accumulated left to right.
//
// Grid-stride over rows.  Ranking keys are 64-bit: the
// weight's IEEE-754 totalOrder bits above the inverted expert index, so keys are
// unique, larger weights rank first and equal weights go to the lower expert.
// Up to 256 experts a row is held by 16 lanes (four rows per wave), above that
// by a whole wave; lane l of a row holds experts l, l+16, ... (or l, l+64, ...)
// in registers, loaded with coalesced 64- or 256-byte requests, the next row
// while this one is ranked.  Each of the top_k rounds takes every lane's best
// remaining key, the row's maximum (DPP inside 16-lane rows, row swaps across
// them; no LDS), and the owner drops the winner.  A second
// kernel over a few blocks counts the rows that execute each expert (per-block
// LDS histograms added into expert_count).
#include "moe.h"

#include <algorithm>

namespace mla {
namespace {

__device__ __forceinline__ uint32_t total_order_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u >> 31) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_total_order_bits(uint32_t t) {
  return __uint_as_float((t >> 31) ? (t & 0x7FFFFFFFu) : ~t);
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

__device__ __forceinline__ uint64_t join(uint32_t lo, uint32_t hi) { return ((uint64_t)hi << 32) | lo; }

// maximum over each group of LPR consecutive lanes (16 or 64), in every lane of
// the group: quad butterflies and row mirrors (DPP) inside each 16-lane row,
// then, for 64-lane groups, the gfx950 row swaps across 16 and 32 lanes
template <int LPR>
__device__ __forceinline__ uint64_t group_max_u64(uint64_t v) {
  static_assert(LPR == 16 || LPR == 64, "lanes per row");
  uint64_t o;
  o = join(dpp<0xB1>((uint32_t)v), dpp<0xB1>((uint32_t)(v >> 32)));     // lane ^ 1
  v = o > v ? o : v;
  o = join(dpp<0x4E>((uint32_t)v), dpp<0x4E>((uint32_t)(v >> 32)));     // lane ^ 2
  v = o > v ? o : v;
  o = join(dpp<0x141>((uint32_t)v), dpp<0x141>((uint32_t)(v >> 32)));   // mirror in 8 lanes: quad pairs
  v = o > v ? o : v;
  o = join(dpp<0x140>((uint32_t)v), dpp<0x140>((uint32_t)(v >> 32)));   // mirror in 16 lanes: halves
  v = o > v ? o : v;
  if (LPR == 64) {
    {
      const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
      const auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(v >> 32), (uint32_t)(v >> 32), false, false);
      const uint64_t a = join(lo[0], hi[0]), b = join(lo[1], hi[1]);       // rows r and r ^ 1
      v = a > b ? a : b;
    }
    {
      const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
      const auto hi = __builtin_amdgcn_permlane32_swap((uint32_t)(v >> 32), (uint32_t)(v >> 32), false, false);
      const uint64_t a = join(lo[0], hi[0]), b = join(lo[1], hi[1]);       // halves of the wave
      v = a > b ? a : b;
    }
  }
  return v;
}

template <int LPR, int NV>
__device__ __forceinline__ void load_row(const MoeArgs& a, int64_t r, int sl, float (&v)[NV]) {
  const float* p = a.router + r * a.n_experts;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int e = LPR * i + sl;
    v[i] = p[e < a.n_experts ? e : a.n_experts - 1];   // clamped: no branch; masked below
  }
}

// LPR lanes per row (64 / LPR rows per wave); lane sl of a row holds experts
// sl, sl + LPR, ..., sl + LPR (NV - 1)
template <int LPR, int NV>
__global__ __launch_bounds__(256) void moe_fanout_kernel(MoeArgs a) {
  constexpr int RPW = 64 / LPR;                      // rows per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sl = lane % LPR, slot = lane / LPR;
  const int E = a.n_experts, TK = a.top_k;
  const int64_t stride = (int64_t)gridDim.x * 4 * RPW;
  int64_t r = ((int64_t)blockIdx.x * 4 + wave) * RPW + slot;
  // every lane runs the same number of iterations (rows past the end compute on
  // a clamped copy and write nothing), so the DPP exchanges see whole groups
  const int64_t last = a.n_rows - 1;
  const int64_t r_first_of_wave = r - slot;
  if (r_first_of_wave > last) return;
  float cur[NV];
  load_row<LPR, NV>(a, r < last ? r : last, sl, cur);
  for (; r - slot <= last; r += stride) {
    float nxt[NV];
    const bool more = r - slot + stride <= last;     // uniform in the wave
    if (more) {
      const int64_t rn = r + stride;
      load_row<LPR, NV>(a, rn < last ? rn : last, sl, nxt);
    }
    // totalOrder codes of the lane's weights; a taken mask marks experts already
    // ranked (and the lane's slots past E)
    uint32_t tob[NV];
    uint32_t taken = 0;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      tob[i] = total_order_bits(cur[i]);
      if (LPR * i + sl >= E) taken |= 1u << i;
    }
    // top_k rounds: the lane's best remaining expert (ascending i keeps the lower
    // expert on equal codes), the row maximum of the 64-bit keys, the owner marks it
    int32_t id[kMoeMaxTopK];
    float w[kMoeMaxTopK];
#pragma unroll
    for (int j = 0; j < kMoeMaxTopK; ++j) {
      id[j] = 0;
      w[j] = 0.0f;
      if (j < TK) {
        uint32_t bt = 0;
        int bi = -1;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const bool better = !((taken >> i) & 1u) && (bi < 0 || tob[i] > bt);
          bt = better ? tob[i] : bt;
          bi = better ? i : bi;
        }
        const uint64_t mine =
            bi < 0 ? 0ull : ((uint64_t)bt << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)(LPR * bi + sl));
        const uint64_t m = group_max_u64<LPR>(mine);
        if (bi >= 0 && mine == m) taken |= 1u << bi;                     // keys are unique
        id[j] = (int32_t)(0xFFFFFFFFu - (uint32_t)m);
        w[j] = from_total_order_bits((uint32_t)(m >> 32));
      }
    }
    // fanout, decided in float32 in rank order
    float S = w[0];
#pragma unroll
    for (int j = 1; j < kMoeMaxTopK; ++j)
      if (j < TK) S = S + w[j];
    float cum = 0.0f;
    int K = TK;
    bool done = false;
#pragma unroll
    for (int j = 0; j < kMoeMaxTopK; ++j) {
      if (j < TK) {
        cum = cum + w[j] / S;
        if (!done && j + 1 >= a.min_k && cum >= a.tau) {
          K = j + 1;
          done = true;
        }
      }
    }
    // lane sl < top_k of the row writes rank sl; lane 0 of the row the fanout
    int32_t my_id = 0;
    float my_w = 0.0f;
#pragma unroll
    for (int j = 0; j < kMoeMaxTopK; ++j)
      if (sl == j) {
        my_id = id[j];
        my_w = w[j];
      }
    if (r <= last) {
      if (sl < TK) {
        a.expert_idx[r * TK + sl] = my_id;
        a.expert_w[r * TK + sl] = my_w;
      }
      if (sl == 0) a.fanout[r] = K;
    }
    if (more) {
#pragma unroll
      for (int i = 0; i < NV; ++i) cur[i] = nxt[i];
    }
  }
}

// rows that execute each expert: per-block LDS histograms over a few blocks,
// added into expert_count (zeroed by the previous kernel)
__global__ __launch_bounds__(256) void moe_count_kernel(MoeArgs a) {
  __shared__ uint32_t hist[kMoeMaxExperts];
  const int E = a.n_experts, TK = a.top_k;
  for (int i = threadIdx.x; i < E; i += 256) hist[i] = 0;
  __syncthreads();
  for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < a.n_rows; r += (int64_t)gridDim.x * 256) {
    const int K = a.fanout[r];
    for (int j = 0; j < TK; ++j) {
      const int32_t e = a.expert_idx[r * TK + j];
      if (j < K && (uint32_t)e < (uint32_t)E) atomicAdd(&hist[e], 1u);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < E; i += 256) {
    const uint32_t h = hist[i];
    if (h) atomicAdd((uint32_t*)&a.expert_count[i], h);
  }
}

__global__ __launch_bounds__(256) void moe_zero_counts_kernel(int32_t* c, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) c[i] = 0;
}

}  // namespace

hipError_t launch_moe_fanout(const MoeArgs& a, hipStream_t s) {
  hipError_t e;
  if (a.expert_count != nullptr) {
    moe_zero_counts_kernel<<<dim3((unsigned)((a.n_experts + 255) / 256)), dim3(256), 0, s>>>(a.expert_count,
                                                                                        a.n_experts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.n_rows == 0) return hipSuccess;
  const dim3 blk(256);
  const int E = a.n_experts;
  auto grid = [&](int rows_per_wave) {
    // a few row groups per wave, so that each wave's next row loads while it ranks one
    return dim3((unsigned)std::min<int64_t>((a.n_rows + 4 * rows_per_wave - 1) / (4 * rows_per_wave), 2048));
  };
  if (E <= 16) moe_fanout_kernel<16, 1><<<grid(4), blk, 0, s>>>(a);
  else if (E <= 32) moe_fanout_kernel<16, 2><<<grid(4), blk, 0, s>>>(a);
  else if (E <= 64) moe_fanout_kernel<16, 4><<<grid(4), blk, 0, s>>>(a);
  else if (E <= 128) moe_fanout_kernel<16, 8><<<grid(4), blk, 0, s>>>(a);
  else if (E <= 256) moe_fanout_kernel<16, 16><<<grid(4), blk, 0, s>>>(a);
  else if (E <= 512) moe_fanout_kernel<64, 8><<<grid(1), blk, 0, s>>>(a);
  else moe_fanout_kernel<64, 16><<<grid(1), blk, 0, s>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.expert_count != nullptr) {
    const unsigned cblocks = (unsigned)std::min<int64_t>((a.n_rows + 1023) / 1024, 256);
    moe_count_kernel<<<dim3(cblocks), dim3(256), 0, s>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace mla
