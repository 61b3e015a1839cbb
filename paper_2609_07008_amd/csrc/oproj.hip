// Group-aligned sliced first output projection with artifact restore-and-replace
// (eq:offonline, eq:factorization, Alg. 2: z_online = W_{a,G} O_G + W_{a,L} O_{L,A};
// z = z_online + z_off on unprotected rows, z = z_online on protected rows).
//
// Two bf16 MFMA GEMM passes per projection group pg, both on the caller's stream:
//   pass G: every row, K = the Global heads of pg's groups; the epilogue adds
//           z_off[r] on unprotected rows and nothing on protected rows, so
//           z_off is never read for protected rows (the replace);
//   pass L: rows a of the protected set, K = the Local heads of pg's groups;
//           the result is added to the pass-G value in z[prot_rows[a]] (or, for
//           the offline producer, which runs pass L alone, written there).
// An epilogue loads the values it adds a 32-row block at a time, before the
// block's first store, so that their latencies overlap.
// Each head's weight rows are a d_c-row block of w_o[pg]; a K tile of 64 never
// straddles two heads, so the B operand is gathered per tile by head.  The MFMAs
// compute the transposed tile (W^T O^T), so that each lane holds one output row
// and runs of 4 consecutive channels: the epilogue reads z_off and writes z 8 and
// 16 bytes at a time.
#include "oproj.h"

#include <algorithm>

namespace mla {

// Tile shapes: BM rows x BN channels per workgroup of WM x WN waves (wave tiles
// of multiples of 32), K in steps of 64.
constexpr int OP_BK = 64;
constexpr int OP_ALD = OP_BK + 8;     // padded A row (bf16): 144 B, conflict-free 16-byte row reads

template <int PASS, int BM, int BN, int WM, int WN>   // PASS 0 = Local over protected rows, 1 = Global
// at most 128 registers per wave, so that two workgroups of 8 waves share a CU
__global__ __launch_bounds__(WM * WN * 64) __attribute__((amdgpu_waves_per_eu(4)))
void oproj_kernel(OprojArgs a, int m_tiles, int n_tiles, int local_add) {
  constexpr int NT = WM * WN * 64;
  // padded B row: 2*BLD = 64 mod 256 bytes, so the four k-rows that each half-wave
  // of a transposing read touches land on disjoint 16-bank groups (all 64 banks)
  constexpr int OP_BLD = BN + 32;
  constexpr int TM = BM / WM, TN = BN / WN;    // wave tile
  constexpr int MI = TM / 32, NI = TN / 32;     // 32x32 MFMA blocks per wave
  constexpr int A_CH = BM * OP_BK / 8 / NT;     // 16-byte chunks per thread and K step
  constexpr int B_CH = OP_BK * BN / 8 / NT;
  static_assert(TM % 32 == 0 && TN % 32 == 0 && A_CH >= 1 && B_CH >= 1, "tile shape");
  static_assert(((2 * OP_BLD) % 256) == 64, "B row padding");
  constexpr int OP_BM = BM, OP_BN = BN;
  // one LDS buffer per operand: the next K step waits in registers, and two
  // workgroups fit a CU, one's epilogue running beside the other's K loop
  __shared__ __attribute__((aligned(16))) uint16_t As[OP_BM * OP_ALD];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[OP_BK * OP_BLD];
  __shared__ int row_flag[OP_BM];
  __shared__ int row_out[OP_BM];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hpg = a.n_heads / a.n_groups;
  const int gpp = a.n_groups / a.n_pg;              // output groups per projection group
  const int cw = a.d_model / a.n_pg;                // channels per projection group
  const int heads_pp = a.n_heads / a.n_pg;
  const int DC = a.d_latent;

  // XCD-aware tile order: workgroups go to the 8 XCDs round-robin by id, so XCD x
  // takes the contiguous tile range [x*per, (x+1)*per); the n_tiles column tiles
  // of one row block are consecutive and share that row block in the XCD's L2
  const int total = n_tiles * m_tiles * a.n_pg;
  const int per = (total + 7) / 8;
  int bid = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
  if (bid >= total) return;
  const int nt = bid % n_tiles;
  bid /= n_tiles;
  const int mt = bid % m_tiles;
  const int pg = bid / m_tiles;
  const int m0 = mt * OP_BM, n0 = nt * OP_BN;

  // protected rows in use: the host count, or the device count clamped to the capacity
  int n_prot = a.n_prot;
  if (a.n_prot_dev != nullptr) {
    const int d = *a.n_prot_dev;
    n_prot = d < 0 ? 0 : (d < a.n_prot ? d : a.n_prot);
  }
  const int64_t M = PASS == 0 ? (int64_t)n_prot : a.n_rows;
  if (m0 >= M) return;   // a tile past the device count of protected rows
  const int heads_k = PASS == 0 ? gpp * (hpg - 1) : gpp;   // d_c-wide K blocks
  const int K = heads_k * DC;
  const uint16_t* A = (const uint16_t*)(PASS == 0 ? a.o_loc : a.o_glob);
  const int64_t lda = PASS == 0 ? (int64_t)a.n_groups * (hpg - 1) * DC : (int64_t)a.n_groups * DC;
  const int64_t acol = PASS == 0 ? (int64_t)pg * gpp * (hpg - 1) * DC : (int64_t)pg * gpp * DC;
  const uint16_t* W = (const uint16_t*)a.w_o + (int64_t)pg * heads_pp * DC * cw;

  if (PASS == 0) {
    for (int i = tid; i < OP_BM; i += NT) {
      const int64_t m = m0 + i;
      int orow = -1;
      if (m < M) {
        orow = a.prot_rows[m];
        if (orow < 0 || orow >= a.n_rows) orow = -1;   // outside z: the row is skipped
      }
      row_flag[i] = 1;
      row_out[i] = orow;
    }
  } else {
    // the tile's rows are [m0, m0 + BM): the protected ones are the run of the
    // sorted list between two lower bounds, found once per workgroup
    __shared__ int run[2];
    if (tid < 2) {
      const int64_t key = tid == 0 ? (int64_t)m0 : (int64_t)m0 + OP_BM;
      int lo = 0, hi = n_prot;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if ((int64_t)a.prot_rows[mid] < key) lo = mid + 1; else hi = mid;
      }
      run[tid] = lo;
    }
    for (int i = tid; i < OP_BM; i += NT) {
      row_flag[i] = 0;
      row_out[i] = m0 + i < M ? m0 + i : -1;
    }
    __syncthreads();
    for (int k = run[0] + tid; k < run[1]; k += NT) {
      const int64_t r = (int64_t)a.prot_rows[k] - m0;
      if (r >= 0 && r < OP_BM) row_flag[r] = 1;   // in range for any list, sorted or not
    }
  }

  // weight row of K index k (k is a multiple of 32 inside one head block)
  auto w_row = [&](int k) -> int64_t {
    const int kb = k / DC, d = k - kb * DC;
    int hl;   // head index inside the projection group
    if (PASS == 0) {
      const int gl = kb / (hpg - 1), j = kb - gl * (hpg - 1);
      const int gh = a.glob_head[pg * gpp + gl];
      hl = gl * hpg + (j < gh ? j : j + 1);
    } else {
      hl = kb * hpg + a.glob_head[pg * gpp + kb];
    }
    return (int64_t)hl * DC + d;
  };

  u32x4 ra[A_CH], rb[B_CH];
  auto load_tiles = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + NT * i;
      const int r = c / (OP_BK / 8), cc = c % (OP_BK / 8);
      int64_t m = m0 + r;
      if (m >= M) m = M - 1;
      ra[i] = *(const u32x4*)(A + m * lda + acol + k0 + cc * 8);
    }
    const int64_t wr = w_row(k0);
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + NT * i;
      const int kr = c / (OP_BN / 8), cc = c % (OP_BN / 8);
      const int n = n0 + cc * 8;
      if (n < cw)
        rb[i] = *(const u32x4*)(W + (wr + kr) * cw + n);
      else
        rb[i] = u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_tiles = [&]() {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + NT * i;
      *(u32x4*)(&As[(c / (OP_BK / 8)) * OP_ALD + (c % (OP_BK / 8)) * 8]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + NT * i;
      *(u32x4*)(&Bs[(c / (OP_BN / 8)) * OP_BLD + (c % (OP_BN / 8)) * 8]) = rb[i];
    }
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int wm = wave / WN, wn = wave % WN;
  const int half = lane >> 5, l32 = lane & 31;
  const int q = lane >> 4, j16 = lane & 15;

  load_tiles(0);
  store_tiles();
  __syncthreads();
  const int nk = K / OP_BK;
  for (int it = 0; it < nk; ++it) {
    if (it + 1 < nk) load_tiles((it + 1) * OP_BK);
#pragma unroll
    for (int ks = 0; ks < OP_BK / 16; ++ks) {
      bf16x8 af[MI], bfr[NI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
        af[mi] = *(const bf16x8*)(&As[(wm * TM + mi * 32 + l32) * OP_ALD + ks * 16 + half * 8]);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        // transposed LDS reads: lane (r*4+cb) of each 16-lane group addresses
        // k-row kb+r, columns n+cb*4..; lane j then holds column n+j of rows kb..kb+3
        const int r = j16 >> 2, cb = j16 & 3;
        const int kb = ks * 16 + (q >> 1) * 8;
        const int n = wn * TN + ni * 32 + (q & 1) * 16 + cb * 4;
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (MLA_LDS bf16x4*)(&Bs[(kb + r) * OP_BLD + n]));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (MLA_LDS bf16x4*)(&Bs[(kb + 4 + r) * OP_BLD + n]));
        bfr[ni] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[ni], af[mi], acc[mi][ni], 0, 0, 0);
    }
    __syncthreads();
    if (it + 1 < nk) {
      store_tiles();
      __syncthreads();
    }
  }

  // epilogue: the accumulators hold the transposed blocks, so a lane holds output
  // row l32 of each 32-row block and channels half*4 + 8i .. +3 of each
  // 32-channel block.  Each 32 x 32 block goes through this wave's part of the
  // (now idle) A buffer and comes back row-contiguous: 8 lanes cover one row's
  // 32 channels, so every z store instruction writes eight whole 128-byte lines
  // of f32 z (and each z_off read takes eight 64-byte runs).
  constexpr int SLD = 36;   // staged row: 32 floats + 4 of padding
  static_assert(NT / 64 * 32 * SLD * 4 <= OP_BM * OP_ALD * 2, "epilogue staging fits the A buffer");
  // lane quantities recomputed here rather than kept live across the K loop
  const int elane = (int)__lane_id();
  float MLA_LDS* stage = (float MLA_LDS*)As + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * (32 * SLD);
  const uint16_t* zoff = (const uint16_t*)a.z_off;
  const int prow = elane >> 3, pc4 = (elane & 7) * 4;   // read-back: row prow + 8p, channels pc4 .. +3
  // the values this block adds: pass G, bf16 z_off of the unprotected rows (none
  // on protected rows); pass L after pass G, the row's z (f32 bits, or bf16)
  const bool add_any = PASS == 1 || local_add != 0;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    u32x4 addv[NI][4];
    f32x4 addf[NI][4];
    if (add_any) {
      // every lane loads (element 0 where nothing is added) and the unused
      // values are zeroed after: no branch around the loads, so each later wait
      // counts exactly the loads still ahead of it
      auto add_off = [&](int ni, int p, bool& use) -> int64_t {
        const int n = n0 + wn * TN + ni * 32 + pc4;
        const int r = wm * TM + mi * 32 + p * 8 + prow;
        const int64_t orow = m0 + r < M && n < cw ? (int64_t)row_out[r] : -1;
        use = orow >= 0 && (PASS == 0 || !row_flag[r]);
        return use ? orow * a.d_model + (int64_t)pg * cw + n : 0;
      };
      if (PASS == 1 || a.z_bf16) {
        const uint16_t* src = PASS == 1 ? zoff : (const uint16_t*)a.z;
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            bool use;
            const u32x2 zz = *(const u32x2*)(src + add_off(ni, p, use));
            addv[ni][p] = use ? u32x4{zz[0], zz[1], 0u, 0u} : u32x4{0u, 0u, 0u, 0u};
          }
      } else {
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            bool use;
            const u32x4 w = *(const u32x4*)(a.z + add_off(ni, p, use));
            addv[ni][p] = use ? w : u32x4{0u, 0u, 0u, 0u};
          }
      }
      // widened to f32 here, so that the block's one wait for its loads comes
      // before any of its stores (later waits would count those stores too)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const u32x4 w = addv[ni][p];
          addf[ni][p] = PASS == 1 || a.z_bf16
                            ? f32x4{bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])}
                            : f32x4{__uint_as_float(w[0]), __uint_as_float(w[1]), __uint_as_float(w[2]),
                                    __uint_as_float(w[3])};
        }
    }
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *(f32x4 MLA_LDS*)(stage + (elane & 31) * SLD + (elane >> 5) * 4 + 8 * i) =
            f32x4{acc[mi][ni][4 * i], acc[mi][ni][4 * i + 1], acc[mi][ni][4 * i + 2], acc[mi][ni][4 * i + 3]};
      const int n = n0 + wn * TN + ni * 32 + pc4;   // 4 consecutive channels; cw is a multiple of 32
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int rr = p * 8 + prow;
        f32x4 v = *(const f32x4 MLA_LDS*)(stage + rr * SLD + pc4);
        const int r = wm * TM + mi * 32 + rr;       // tile row
        if (m0 + r >= M || n >= cw) continue;
        const int64_t orow = row_out[r];
        if (orow < 0) continue;
        const int64_t off = orow * a.d_model + (int64_t)pg * cw + n;
        if (add_any) v += addf[ni][p];
        if (a.z_bf16)
          *(u32x2*)((uint16_t*)a.z + off) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        else
          *(f32x4*)(a.z + off) = v;
      }
    }
  }
}

// W_{a,L}^T of each projection group, for the producer's Local projection as a
// plain K-contiguous GEMM: wt[pg][n][k] = w_o[pg][row(k)][n], k running over the
// Local heads of pg's groups in the order of the head outputs' columns (ascending
// head index, the group's Global head skipped).  64 x 64 tiles through LDS, so
// that both the reads (along n) and the writes (along k) are row-contiguous.
__global__ __launch_bounds__(256) void local_wt_kernel(OprojArgs a, uint16_t* wt, int n_ktiles, int n_ntiles) {
  __shared__ uint16_t tile[64][65];
  const int hpg = a.n_heads / a.n_groups, gpp = a.n_groups / a.n_pg;
  const int cw = a.d_model / a.n_pg, DC = a.d_latent;
  const int heads_pp = a.n_heads / a.n_pg;
  const int64_t KL = (int64_t)gpp * (hpg - 1) * DC;
  int b = blockIdx.x;
  const int kt = b % n_ktiles;
  b /= n_ktiles;
  const int nt = b % n_ntiles;
  const int pg = b / n_ntiles;
  const uint16_t* W = (const uint16_t*)a.w_o + (int64_t)pg * heads_pp * DC * cw;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int r = ty; r < 64; r += 4) {   // read: tile row r = k, column tx = n
    const int64_t k = (int64_t)kt * 64 + r;
    const int n = nt * 64 + tx;
    uint16_t v = 0;
    if (k < KL && n < cw) {
      const int kb = (int)(k / DC), d = (int)(k - (int64_t)kb * DC);
      const int gl = kb / (hpg - 1), j = kb - gl * (hpg - 1);
      const int gh = a.glob_head[pg * gpp + gl];
      const int hl = gl * hpg + (j < gh ? j : j + 1);
      v = W[((int64_t)hl * DC + d) * cw + n];
    }
    tile[r][tx] = v;
  }
  __syncthreads();
  for (int r = ty; r < 64; r += 4) {   // write: row n, column k
    const int n = nt * 64 + r;
    const int64_t k = (int64_t)kt * 64 + tx;
    if (n < cw && k < KL) wt[((int64_t)pg * cw + n) * KL + k] = tile[tx][r];
  }
}

hipError_t launch_local_wt(const OprojArgs& a, uint16_t* wt, hipStream_t s) {
  const int hpg = a.n_heads / a.n_groups, gpp = a.n_groups / a.n_pg;
  const int64_t KL = (int64_t)gpp * (hpg - 1) * a.d_latent;
  const int cw = a.d_model / a.n_pg;
  const int n_ktiles = (int)((KL + 63) / 64), n_ntiles = (cw + 63) / 64;
  const int64_t blocks = (int64_t)n_ktiles * n_ntiles * a.n_pg;
  if (blocks == 0) return hipSuccess;
  local_wt_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a, wt, n_ktiles, n_ntiles);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void fill_zero_kernel(u32x4* p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = u32x4{0u, 0u, 0u, 0u};
}

// zero fill with a kernel (no memset node, so the call can be graph-captured);
// p is 16-byte aligned and bytes a multiple of 16
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<int64_t>((n16 + 255) / 256, 16384);
  fill_zero_kernel<<<dim3(blocks), dim3(256), 0, s>>>((u32x4*)p, n16);
  return hipGetLastError();
}

// 256 x 128 tiles, 8 waves (4 x 2 wave tiles of 64 x 64): 58 KB of LDS and up to
// 128 registers per wave, two workgroups per CU.  Same per-element K order as any
// other tile shape, so the results do not depend on it.  At 256K the step's two
// passes take 3.16 ms (128 x 256 the same; 256 x 256 with one workgroup per CU
// 3.58, 64 x 256 with three 3.39, 128 x 128 with four 4.03 ms).
constexpr int kOpBM = 256, kOpBN = 128, kOpWM = 4, kOpWN = 2;

int64_t oproj_workgroups(int64_t M, int d_model, int n_pg) {
  const int64_t tiles = (M + kOpBM - 1) / kOpBM * ((d_model / n_pg + kOpBN - 1) / kOpBN) * n_pg;
  return 8 * ((tiles + 7) / 8);
}

template <int PASS>
hipError_t launch_pass(const OprojArgs& a, int64_t M, int local_add, hipStream_t s) {
  constexpr int BM = kOpBM, BN = kOpBN, WM = kOpWM, WN = kOpWN;
  const int cw = a.d_model / a.n_pg;
  const int n_tiles = (cw + BN - 1) / BN;
  const int m_tiles = (int)((M + BM - 1) / BM);
  const int total = m_tiles * n_tiles * a.n_pg;
  oproj_kernel<PASS, BM, BN, WM, WN><<<dim3((unsigned)(8 * ((total + 7) / 8))), dim3(WM * WN * 64), 0, s>>>(
      a, m_tiles, n_tiles, local_add);
  return hipGetLastError();
}

hipError_t launch_oproj(const OprojArgs& a, int passes, hipStream_t s) {
  const int hpg = a.n_heads / a.n_groups;
  if ((passes & 2) && a.n_rows > 0) {
    const hipError_t e = launch_pass<1>(a, a.n_rows, 0, s);
    if (e != hipSuccess) return e;
  }
  // after pass G the Local values add to z; alone (the producer) they are written
  if ((passes & 1) && a.n_prot > 0 && hpg > 1) return launch_pass<0>(a, a.n_prot, (passes & 2) ? 1 : 0, s);
  return hipSuccess;
}

}  // namespace mla
