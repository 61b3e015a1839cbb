// Shared second output projection y = W_b z (Sec. 2.1 eq:factorization; Alg. 2
// returns W_b z): every row's group-sliced state z [N, d_in] meets the one
// dense W_b, stored as a linear layer's weight [d_out, d_in].  Both operands are
// K-contiguous, so this is C = A B^T with A = z, B = W_b, on bf16 MFMA with fp32
// accumulation; y is written in fp32 or bf16.
//
// Tiles of 256 rows x 256 channels per workgroup of 8 waves (2 x 4), each wave
// 128 x 64 (4 x 2 MFMA 32x32x16 blocks).  K advances 64 at a time; the A and B
// slices of a step (32 KB each) are staged into LDS with 16-byte direct
// global->LDS loads, double-buffered, and each wave reads the fragments of the
// next 16-wide substep while the MFMAs of the current one run.  A wave is held
// at issue while the load path takes each direct load, so only waves 0-3 (one
// per SIMD) issue them, 8 KB of each operand apiece: on every SIMD the partner
// wave's MFMAs run meanwhile.  In LDS a row of
// a slice is 8 chunks of 16 bytes, chunk c of row r stored at slot
// c ^ ((r >> 1) & 7), so the 16-lane quarter-waves of a 16-byte fragment read
// hit 16 distinct bank groups.  Tile order: workgroups go to the 8 XCDs
// round-robin, so XCD x takes a contiguous range of tiles, and inside it tiles
// walk 4 row panels per column panel, so tiles resident together on an XCD share
// A and B panels in its L2.
#include "wb.h"

#include <algorithm>

namespace mla {
namespace {

constexpr int WB_BM = 256, WB_BN = 256, WB_BK = 64;
constexpr int WB_WAVES = 8;
constexpr int WB_DMA_WAVES = 4;                       // waves that issue the direct loads
constexpr int WB_ROWB = WB_BK * 2;                    // bytes of one row of a slice
constexpr int WB_SLICE = WB_BM * WB_ROWB;             // bytes of one A (or B) slice: 32 KB
constexpr int WB_STAGE = 2 * WB_SLICE;                // A then B
constexpr int WB_LOADS = WB_SLICE / 1024 / WB_DMA_WAVES;  // 1 KB direct loads per issuing wave and slice
constexpr int WB_RPL = 1024 / WB_ROWB;                // rows per 1 KB load
constexpr int WB_GM = 4;                              // row panels per column panel in the tile walk

__device__ __forceinline__ void wb_dma16(const void* base, uint32_t voff, const unsigned char MLA_LDS* dst) {
  const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(uintptr_t)dst);
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(b >> 32));
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  const uint64_t bs = ((uint64_t)hi << 32) | (uint64_t)lo;
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(bs), "s"(m0) : "memory", "m0");
}

// this wave's direct loads have landed and its LDS reads are done; then all
// waves meet (the slice just loaded is complete, the other buffer is free)
__device__ __forceinline__ void wb_barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

template <bool OUT_BF16>
__global__ __launch_bounds__(WB_WAVES * 64) void wb_gemm_kernel(WbArgs a, int m_tiles, int n_tiles) {
  constexpr int MI = 4, NI = 2, KS = WB_BK / 16;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[2 * WB_STAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // XCD-aware, grouped tile walk (batches one after another)
  const int per_batch = m_tiles * n_tiles;
  const int total = per_batch * a.batch;
  const int per = (total + 7) / 8;
  const int tb = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
  if (tb >= total) return;
  const int bt = tb / per_batch, t = tb % per_batch;
  const int group = t / (WB_GM * n_tiles), rem = t % (WB_GM * n_tiles);
  const int gm = std::min(WB_GM, m_tiles - group * WB_GM);
  const int mt = group * WB_GM + rem % gm, nt = rem / gm;
  const int64_t m0 = (int64_t)mt * WB_BM;
  const int n0 = nt * WB_BN;

  // Direct loads: load j of issuing wave w fills LDS bytes [1024 (L w + j), +1024)
  // of a slice (L loads per wave), i.e. rows 8 (L w + j) + lane/8 of the tile at
  // slot lane%8, whose source is chunk (lane%8) ^ swz(row).  The load takes a
  // wave-uniform base (the wave's first row) plus a 32-bit lane offset; a wave's
  // rows span 64 rows, so the offsets stay below 2^32 for row strides up to
  // 2^25 elements (the host checks).  Rows past the end are clamped to the last
  // row (their results are not stored).
  const int K = a.d_in;
  const int64_t ldz = a.ldz, ldw = a.ldw;
  const int wr0 = WB_LOADS * WB_RPL * (wave % WB_DMA_WAVES);
  const int64_t a_base_row = std::min<int64_t>(m0 + wr0, a.n_rows - 1);
  const int64_t b_base_row = std::min<int64_t>((int64_t)n0 + wr0, (int64_t)a.d_out - 1);
  uint32_t a_lo[WB_LOADS], b_lo[WB_LOADS];
#pragma unroll
  for (int j = 0; j < WB_LOADS; ++j) {
    const int r = WB_RPL * (WB_LOADS * (wave % WB_DMA_WAVES) + j) + (lane >> 3);
    const int c = (lane & 7) ^ swz(r);
    const int64_t m = std::min<int64_t>(m0 + r, a.n_rows - 1);
    const int64_t n = std::min<int64_t>((int64_t)n0 + r, (int64_t)a.d_out - 1);
    a_lo[j] = (uint32_t)((m - a_base_row) * ldz * 2 + c * 16);
    b_lo[j] = (uint32_t)((n - b_base_row) * ldw * 2 + c * 16);
  }
  const unsigned char* Abase = (const unsigned char*)(a.z + bt * a.z_batch) + a_base_row * ldz * 2;
  const unsigned char* Bbase = (const unsigned char*)(a.w_b + bt * a.w_batch) + b_base_row * ldw * 2;

  auto load_slice = [&](int kt) {
    if (wave >= WB_DMA_WAVES) return;
    unsigned char* st = lds + (kt & 1) * WB_STAGE;
    const unsigned char* ak = Abase + (int64_t)kt * WB_ROWB;
    const unsigned char* bk = Bbase + (int64_t)kt * WB_ROWB;
#pragma unroll
    for (int j = 0; j < WB_LOADS; ++j)
      wb_dma16(ak, a_lo[j], (const unsigned char MLA_LDS*)(st + 1024 * (WB_LOADS * wave + j)));
#pragma unroll
    for (int j = 0; j < WB_LOADS; ++j)
      wb_dma16(bk, b_lo[j], (const unsigned char MLA_LDS*)(st + WB_SLICE + 1024 * (WB_LOADS * wave + j)));
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int wm = wave >> 2, wn = wave & 3;
  const int l32 = lane & 31, hk = lane >> 5;
  // fragment byte offsets inside a stage for substep ks: row*ROWB + 16*((2ks+hk) ^ swz(row))
  int a_fr[MI][KS], b_fr[NI][KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const int ra = wm * 128 + i * 32 + l32;
      a_fr[i][ks] = ra * WB_ROWB + 16 * ((2 * ks + hk) ^ swz(ra));
    }
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int rb = wn * 64 + j * 32 + l32;
      b_fr[j][ks] = WB_SLICE + rb * WB_ROWB + 16 * ((2 * ks + hk) ^ swz(rb));
    }
  }

  const int nk = K / WB_BK;
  load_slice(0);
  for (int kt = 0; kt < nk; ++kt) {
    wb_barrier();                              // slice kt is in; buffer (kt+1)&1 was read at kt-1
    if (kt + 1 < nk) load_slice(kt + 1);
    const unsigned char* st = lds + (kt & 1) * WB_STAGE;
    bf16x8 af[2][MI], bfr[2][NI];
#pragma unroll
    for (int i = 0; i < MI; ++i) af[0][i] = *(const bf16x8*)(st + a_fr[i][0]);
#pragma unroll
    for (int j = 0; j < NI; ++j) bfr[0][j] = *(const bf16x8*)(st + b_fr[j][0]);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int c = ks & 1, nx = c ^ 1;
      if (ks + 1 < KS) {
#pragma unroll
        for (int i = 0; i < MI; ++i) af[nx][i] = *(const bf16x8*)(st + a_fr[i][ks + 1]);
#pragma unroll
        for (int j = 0; j < NI; ++j) bfr[nx][j] = *(const bf16x8*)(st + b_fr[j][ks + 1]);
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[c][i], bfr[c][j], acc[i][j], 0, 0, 0);
    }
  }

  // epilogue: lane holds column l32 of each 32x32 block, rows hk*4 + 8(e/4) + e%4
  const int64_t ybase = bt * a.y_batch;
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int n = n0 + wn * 64 + j * 32 + l32;
      if (n >= a.d_out) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t m = m0 + wm * 128 + i * 32 + hk * 4 + (e >> 2) * 8 + (e & 3);
        if (m >= a.n_rows) continue;
        if (OUT_BF16)
          ((__bf16*)a.y)[ybase + m * a.ldy + n] = (__bf16)acc[i][j][e];
        else
          ((float*)a.y)[ybase + m * a.ldy + n] = acc[i][j][e];
      }
    }
}

}  // namespace

hipError_t launch_wb(const WbArgs& a, hipStream_t s) {
  if (a.n_rows == 0) return hipSuccess;
  const int m_tiles = (int)((a.n_rows + WB_BM - 1) / WB_BM);
  const int n_tiles = (a.d_out + WB_BN - 1) / WB_BN;
  const int total = m_tiles * n_tiles * a.batch;
  const dim3 grid((unsigned)(8 * ((total + 7) / 8)));
  if (a.y_bf16)
    wb_gemm_kernel<true><<<grid, dim3(WB_WAVES * 64), 0, s>>>(a, m_tiles, n_tiles);
  else
    wb_gemm_kernel<false><<<grid, dim3(WB_WAVES * 64), 0, s>>>(a, m_tiles, n_tiles);
  return hipGetLastError();
}

}  // namespace mla
