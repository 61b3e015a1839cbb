// Query-side RoPE relocation and segment-wise absorbed-MLA attention over the
// packed latent stream (Sec. 2.3 eq:rope, Alg. 2 SelectiveMLA), plus the
// device half of the plan (partial index, segment bookkeeping, protected flags).
//
// Work item = up to 128 head-rows (query rows x heads) that share every key of
// the single latent stream (the latent is never split per head, Sec. 2.1).
// One 256-thread workgroup (4 waves x 32 head-rows) walks the item's visible
// segments in request order; for each segment it rotates the RoPE part of its
// queries by R(t - p_s) into the segment's canonical frame, then streams the
// segment's 64-key latent tiles through LDS:
//   S^T = K Q^T      (keys x head-rows, MFMA 32x32x16 bf16, K tile from LDS,
//                     Q resident in registers)
//   online softmax   (one head-row per lane pair, lazy rescaling)
//   O^T += V^T P^T   (latent dims x head-rows, V = the same LDS tile read with
//                     transposing LDS loads)
// and emits one normalized partial and one log-sum-exp per (slot, chunk).
// Tiles are fetched with 16-byte direct-to-LDS loads, double-buffered, with the
// 16-byte chunks of a key row XOR-swizzled so column reads hit distinct banks.
#include "common.h"

namespace mla {

template <int DC, int DR>
struct Cfg {
  static constexpr int D = DC + DR;
  static constexpr int KS = D / 16;          // 16-wide K steps of Q.K
  static constexpr int CS = DC / 16;         // latent K steps
  static constexpr int RS = DR / 16;         // RoPE K steps
  static constexpr int CH = D / 8;           // 16-byte chunks per key row
  static constexpr int CG = (CH + 7) / 8;    // groups of 8 chunks
  static constexpr int CGF = CH / 8;         // full groups (swizzled)
  static constexpr int BK = 64;              // keys per tile
  // LDS tile: 8 key-blocks of 8 keys; block kb8 starts at kb8*KB8 and holds CG
  // 1 KB sub-blocks (one per chunk group).  Inside a sub-block key k%8 sits at
  // (k%8)*128 and chunk c%8 at slot (c%8) ^ rotl3(k%8) (full groups only), so
  // both the row reads of K and the transposing column reads of V hit distinct
  // banks.  KB8 = 128 mod 256 keeps 16-lane 16-byte reads conflict-free on 64 banks.
  static constexpr int KB8 = CG * 1024 + 128;
  static constexpr int TILE_BYTES = 8 * KB8;
  static constexpr int LOADS = 2 * CG;       // direct loads per wave per tile (key-blocks 2w, 2w+1)
  static constexpr int OB = DC / 32;         // 32-wide output blocks
  static constexpr int OBH = OB / 2;         // output blocks owned by one wave
  static constexpr int HR = 64;              // head-rows per work item
  static_assert(DR == 16 || DR % 32 == 0, "d_rope must be 16 or a multiple of 32");
  static_assert(DC % 64 == 0, "d_latent must be a multiple of 64");
};

__device__ __forceinline__ int rotl3(int k) { return ((k << 1) | (k >> 2)) & 7; }

// 16-byte direct global->LDS load: lane i writes LDS bytes [dst + 16 i, +16) of
// the wave-uniform destination `dst`.  Issued through inline asm so that the
// compiler's wait-count pass does not treat every later LDS read as a possible
// alias (it would wait for the prefetch of the next tile); the tile loop waits
// for these loads explicitly (s_waitcnt vmcnt + barrier).
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, const unsigned char MLA_LDS* dst) {
  const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(uintptr_t)dst);
  // the base is wave-uniform; make that explicit so it is held in scalar registers.
  // readfirstlane returns a signed int: zero-extend each half through uint32_t.
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(b >> 32));
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  const uint64_t bs = ((uint64_t)hi << 32) | (uint64_t)lo;
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(bs), "s"(m0) : "memory", "m0");
}

__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const int w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  return v;
}

// Work item = up to 64 head-rows as two blocks of 32.  Wave w serves head-row
// block hb = w>>1 and half kh = w&1: it scores keys kh*32..kh*32+31 of each
// 64-key tile and accumulates latent dims [kh*d_c/2, (kh+1)*d_c/2) of O for
// all 64 keys, taking the other key half's softmax weights from its partner
// wave w^1 through LDS.  Both waves of a pair see identical row maxima, so
// they take identical rescaling decisions.
template <int DC, int DR>
__global__ __launch_bounds__(256, 1) void attend_kernel(AttendArgs a) {
  using C = Cfg<DC, DR>;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * C::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) bf16x8 pex[4][2][64];   // softmax weights for the partner
  __shared__ float stat[4][32];                                    // row maxima / sums for the partner
  __shared__ int restart_vote[4];

  unsigned char MLA_LDS* L = (unsigned char MLA_LDS*)lds;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hb = wave >> 1, kh = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;

  // XCD-aware item order: blocks are dispatched round-robin over the 8 XCDs;
  // give each XCD 32 consecutive items (similar key ranges) per group of 256.
  const int b = blockIdx.x;
  const int xcd = b & 7, kx = b >> 3;
  const int item_id = (kx >> 5) * 256 + xcd * 32 + (kx & 31);
  if (item_id >= a.n_items) return;

  const unsigned char* ws = a.ws;
  const SegInfo* segs = (const SegInfo*)(ws + a.hdr.off_segs);
  const int32_t* rank_seg = (const int32_t*)(ws + a.hdr.off_rank);
  const ChunkInfo* chunks = (const ChunkInfo*)(ws + a.hdr.off_chunks);
  const WorkItem it = ((const WorkItem*)(ws + a.hdr.off_items))[item_id];
  const int32_t* prot = (const int32_t*)(ws + a.hdr.off_prot);
  const double* theta_rev = (const double*)(ws + a.hdr.off_theta);
  const SegInfo own = segs[it.seg];
  const ChunkInfo chk = chunks[own.chunk_off + it.chunk];

  // ---- this lane's head-row ----
  const int hr_local = hb * 32 + l32;
  const bool valid = hr_local < it.count;
  const bool pair_active = hb * 32 < it.count;
  const int64_t hr = it.hr_begin + (valid ? hr_local : 0);
  int64_t row;
  const uint16_t* qsrc;
  int64_t slot;
  if (it.kind == 0) {
    row = hr / a.n_groups;
    qsrc = (const uint16_t*)a.q_glob + hr * C::D;
    slot = hr;
  } else {
    row = prot[hr / a.n_local];
    qsrc = (const uint16_t*)a.q_loc + hr * C::D;
    slot = a.n_rows * a.n_groups + hr;
  }
  const int64_t t_pos = own.req_offset + (row - own.kv_start);

  // ---- Q fragments (B operand of S^T = K Q^T): step ks holds dims ks*16 + half*8 .. +8;
  // for DR == 16 the RoPE step holds rope dims {half*4..+4} and {8+half*4..+4}, so that
  // every rotation pair (j, j + d_r/2) stays inside one lane.
  bf16x8 qf[C::KS];
#pragma unroll
  for (int ks = 0; ks < C::KS; ++ks) {
    if (DR == 16 && ks == C::CS) {
      const u32x2 lo = *(const u32x2*)(qsrc + DC + half * 4);
      const u32x2 hi = *(const u32x2*)(qsrc + DC + 8 + half * 4);
      qf[ks] = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
    } else {
      qf[ks] = *(const bf16x8*)(qsrc + ks * 16 + half * 8);
    }
    if (!valid) qf[ks] = bf16x8{};
  }

  f32x16 o[C::OBH];
  float m_run = -1e30f, l_run = 0.f;

  // ---- per-lane LDS address bases (everything else is an immediate offset) ----
  // K as the A operand: key kh*32 + l32, chunk ks*2 + half
  int abase[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4)
    abase[s4] = (kh * 4 + (l32 >> 3)) * C::KB8 + (l32 & 7) * 128 + (((2 * s4 + half) ^ rotl3(l32 & 7)) * 16);
  // V^T via transposing reads: in each 16-lane group q4 = lane/16, lane j = rr*4 + cb
  // addresses key (q4>>1)*4 + rr of an 8-key block and latent dims (q4&1)*16 + cb*4 of
  // a 32-dim block; lane j then receives dim j of those four keys.
  const int q4 = lane >> 4, rr = (lane >> 2) & 3, cb = lane & 3;
  const int vkey = (q4 >> 1) * 4 + rr;
  // This wave owns output blocks x .. x+OBH-1 with x = kh*OBH; block x+d covers
  // chunk group (x+d)>>1 at chunk offset ((x+d)&1)*4.  vb[d&1][j] is the base for
  // local block parity d&1 and the key block of this wave (j = 0) or of its
  // partner (j = 1); local block d adds (d>>1)*1024.
  const int xb = kh * C::OBH;
  int vb[2][2];
#pragma unroll
  for (int dl = 0; dl < 2; ++dl)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      vb[dl][j] = vkey * 128 + (((((xb + dl) & 1) * 4 + (q4 & 1) * 2 + (cb >> 1)) ^ rotl3(vkey)) * 16) +
                  (cb & 1) * 8 + (kh ^ j) * 4 * C::KB8 + ((xb + dl) >> 1) * 1024;
  // direct loads: lane l fills key l>>3 of an 8-key block, physical slot l&7
  const int lkey = lane >> 3;
  const int lchunk_full = (lane & 7) ^ rotl3(lkey);
  const int lchunk_part = (lane & 7) < (C::CH - C::CGF * 8) ? (lane & 7) : 0;

  auto seg_keys = [&](const SegInfo& s, bool is_own) -> int64_t {
    return is_own ? (int64_t)it.max_u + 1 : s.length;
  };

  // direct-to-LDS loads of tile `tile` of segment `s`: wave w fills key-blocks 2w, 2w+1
  auto issue = [&](unsigned char MLA_LDS* dbuf, const SegInfo& s, int64_t n_keys, int64_t tile) {
    const int64_t k0 = tile * C::BK;
    const int last = (int)(n_keys - 1 - k0);   // rows past the segment repeat its last row
    const bool full = last >= C::BK - 1;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int kb8 = 2 * wave + h;
      // uniform base: first row of the 8-key block; lane offset: its key row and chunk
      int64_t brow = k0 + kb8 * 8;
      int kr = lkey;
      if (!full) {
        const int lb = last - kb8 * 8;   // last valid key of this block, relative to its first
        if (lb < 0) {                    // whole block past the end: repeat the segment's last row
          brow = k0 + last;
          kr = 0;
        } else if (kr > lb) {
          kr = lb;
        }
      }
      const unsigned char* base = (const unsigned char*)a.kv + (s.kv_start + brow) * (C::D * 2);
      const uint32_t roff = (uint32_t)(kr * (C::D * 2));   // never negative
#pragma unroll
      for (int cg = 0; cg < C::CG; ++cg) {
        const int ch = cg * 8 + (cg < C::CGF ? lchunk_full : lchunk_part);
        dma16(base, roff + ch * 16, dbuf + kb8 * C::KB8 + cg * 1024);
      }
    }
  };

  // ---- tile cursor over the chunk's segments (request order) ----
  int c_rank;
  SegInfo cs;
  int64_t c_tile;
  int n_rank;
  SegInfo ns;
  int64_t n_keys, n_ntiles, n_tile;

  int lim = 0x7fffffff;        // largest visible canonical offset for this lane in segment cs
  int wave_lim = 0x7fffffff;   // smallest lim over the wave's valid lanes

  // relocation for a new segment: rotate the RoPE part of this lane's query by
  // R(t - p_s); the angle is reduced in double precision (in revolutions) and
  // fed to the hardware sin/cos
  auto relocate = [&](const SegInfo& s) {
    const int64_t delta = t_pos - s.req_offset;
    const int64_t lm = delta < s.length - 1 ? delta : s.length - 1;
    lim = valid ? (int)lm : 0x7fffffff;
    wave_lim = wave_min_i(lim);
    bf16x8 raw[C::RS];
#pragma unroll
    for (int rs = 0; rs < C::RS; ++rs) {
      if (DR == 16) {
        const u32x2 lo = *(const u32x2*)(qsrc + DC + half * 4);
        const u32x2 hi = *(const u32x2*)(qsrc + DC + 8 + half * 4);
        raw[rs] = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
      } else {
        raw[rs] = *(const bf16x8*)(qsrc + DC + rs * 16 + half * 8);
      }
    }
    const double dd = (double)delta;
#pragma unroll
    for (int rs = 0; rs < (DR == 16 ? 1 : C::RS / 2); ++rs) {
#pragma unroll
      for (int i = 0; i < (DR == 16 ? 4 : 8); ++i) {
        // pair (j, j + d_r/2): first element at (rs, slot i), partner at (prs, ps)
        const int j0 = DR == 16 ? i : rs * 16 + i;
        const int jstep = DR == 16 ? 4 : 8;       // frequency offset of the upper lane half
        const int prs = DR == 16 ? rs : rs + DR / 32;
        const int ps = DR == 16 ? i + 4 : i;
        const double rev = dd * theta_rev[j0 + half * jstep];
        const float r = (float)(rev - rint(rev));
        const float sn = __builtin_amdgcn_sinf(r), cn = __builtin_amdgcn_cosf(r);
        const float x1 = (float)raw[rs][i], x2 = (float)raw[prs][ps];
        qf[C::CS + rs][i] = valid ? (__bf16)(x1 * cn - x2 * sn) : (__bf16)0.f;
        qf[C::CS + prs][ps] = valid ? (__bf16)(x1 * sn + x2 * cn) : (__bf16)0.f;
      }
    }
  };

  // advance the "next" cursor by one tile; returns false at the end of the chunk
  auto advance = [&]() -> bool {
    if (n_tile + 1 < n_ntiles) {
      ++n_tile;
      return true;
    }
    if (n_rank >= chk.last_rank) return false;
    ++n_rank;
    const int sidx = rank_seg[n_rank];
    ns = segs[sidx];
    n_keys = seg_keys(ns, sidx == it.seg);
    n_ntiles = (n_keys + C::BK - 1) / C::BK;
    n_tile = 0;
    return true;
  };

  // The softmax reference max m_run is taken from the first tile.  A later tile
  // whose max exceeds it by more than 2^64 (weights stay below 2^64: fp32 and
  // bf16 hold them exactly enough) restarts the whole item from the larger
  // reference; the decision is shared by the workgroup so every wave meets the
  // same barriers.  The tile loop thus never applies vector ALU work to the O
  // accumulators, which stay in the matrix-core registers.
  const float sl2 = a.scale_log2;
  float m_init = -1e30f;
  bool restarted = false;
  for (;;) {
#pragma unroll
    for (int d = 0; d < C::OBH; ++d)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[d][e] = 0.f;
    m_run = m_init;
    l_run = 0.f;
    c_rank = chk.first_rank;
    cs = segs[rank_seg[c_rank]];
    c_tile = 0;
    n_rank = c_rank;
    ns = cs;
    n_keys = seg_keys(cs, rank_seg[c_rank] == it.seg);
    n_ntiles = (n_keys + C::BK - 1) / C::BK;
    n_tile = 0;
    relocate(cs);
    issue(L, cs, n_keys, 0);

    bool restart = false;
    bool first_tile = !restarted;   // uniform over the workgroup
    float mt = 0.f;   // this wave's row max of the current tile (log2 units)
    // One tile.  Barrier A: the tile in `cb` has landed in LDS and every wave has
    // finished the previous tile, so `nb` is free for the next prefetch.  Barrier C:
    // softmax weights and restart votes are visible to the partner waves.
    // Returns 0 = continue, 1 = chunk done, 2 = restart with a larger reference max.
    auto step = [&](const unsigned char MLA_LDS* cb, unsigned char MLA_LDS* nb) -> int {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __builtin_amdgcn_s_barrier();
      const bool more = advance();
      if (more) issue(nb, ns, n_keys, n_tile);
      const unsigned char MLA_LDS* buf = cb;
      // ---- S^T = K Q^T for this wave's 32 keys ----
      f32x16 sc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
      if (pair_active) {
        auto kfrag = [&](int ks) -> bf16x8 {
          if (DR == 16 && ks == C::CS) {
            // rope chunks 2*CS, 2*CS+1 sit in the partial (unswizzled) group: 8 bytes each
            const int base0 = (kh * 4 + (l32 >> 3)) * C::KB8 + (l32 & 7) * 128 + C::CGF * 1024 + half * 8;
            const u32x2 x0 = *(const u32x2 MLA_LDS*)(buf + base0);
            const u32x2 y0 = *(const u32x2 MLA_LDS*)(buf + base0 + 16);
            return __builtin_bit_cast(bf16x8, u32x4{x0[0], x0[1], y0[0], y0[1]});
          }
          return *(const bf16x8 MLA_LDS*)(buf + abase[ks & 3] + (ks >> 2) * 1024);
        };
        bf16x8 ka[3];
        ka[0] = kfrag(0);
        if (C::KS > 1) ka[1] = kfrag(1);
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) {
          if (ks + 2 < C::KS) ka[(ks + 2) % 3] = kfrag(ks + 2);
          sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[ks % 3], qf[ks], sc, 0, 0, 0);
        }
        // register e holds key kh*32 + half*4 + (e/4)*8 + e%4 of the tile, in log2 units
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[e] *= sl2;
        const int tk0 = (int)(c_tile * C::BK) + kh * 32;
        if (tk0 + 31 > wave_lim) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = tk0 + half * 4 + (e >> 2) * 8 + (e & 3);
            if (key > lim) sc[e] = -INFINITY;
          }
        }
        float m = sc[0];
#pragma unroll
        for (int e = 1; e < 16; ++e) m = fmaxf(m, sc[e]);
        mt = fmaxf(m, __shfl_xor(m, 32, 64));
      }
      if (first_tile) {
        // first tile of the item (workgroup-uniform): the pair fixes its common
        // reference max
        if (pair_active && half == 0) stat[wave][l32] = mt;
        __builtin_amdgcn_s_barrier();
        if (pair_active) m_run = fmaxf(stat[wave][l32], stat[wave ^ 1][l32]);
        first_tile = false;
      }

      bool up = false;
      if (pair_active) {
        up = __builtin_amdgcn_ballot_w64(mt > m_run + 64.f) != 0;
        // ---- softmax weights against the pair's common reference max ----
        float rsum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          sc[e] = __builtin_amdgcn_exp2f(sc[e] - m_run);
          rsum += sc[e];
        }
        l_run += rsum + __shfl_xor(rsum, 32, 64);          // this wave's 32 keys only
        bf16x8 pown[2];
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
          for (int i = 0; i < 8; ++i) pown[k2][i] = (__bf16)sc[k2 * 8 + i];
        pex[wave][0][lane] = pown[0];
        pex[wave][1][lane] = pown[1];
      }
      if (lane == 0) restart_vote[wave] = up ? 1 : 0;
      __builtin_amdgcn_s_barrier();
      // a row whose tile max passed the reference by 2^64: the whole workgroup
      // discards this tile and restarts (l_run is reset with the restart)
      restart = (restart_vote[0] | restart_vote[1] | restart_vote[2] | restart_vote[3]) != 0;
      if (restart) return 2;

      if (pair_active) {
        // ---- O^T[dims of half kh] += V^T P^T over all 64 keys ----
        // contraction order: this wave's key block, then the partner's
        bf16x8 pf[2][2];   // [own, partner][k step]
        pf[0][0] = pex[wave][0][lane];
        pf[0][1] = pex[wave][1][lane];
        pf[1][0] = pex[wave ^ 1][0][lane];
        pf[1][1] = pex[wave ^ 1][1][lane];
        constexpr int NPV = C::OBH * 4;
        auto vfrag = [&](int st) -> bf16x8 {
          const int d = st >> 2, j = (st >> 1) & 1, k2 = st & 1;
          const int off = vb[d & 1][j] + (d >> 1) * 1024 + k2 * 2 * C::KB8;
          const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((MLA_LDS bf16x4*)(buf + off));
          const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((MLA_LDS bf16x4*)(buf + off + C::KB8));
          return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        };
        bf16x8 vt[3];
        vt[0] = vfrag(0);
        if (NPV > 1) vt[1] = vfrag(1);
#pragma unroll
        for (int st = 0; st < NPV; ++st) {
          if (st + 2 < NPV) vt[(st + 2) % 3] = vfrag(st + 2);
          const int d = st >> 2, j = (st >> 1) & 1, k2 = st & 1;
          o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vt[st % 3], pf[j][k2], o[d], 0, 0, 0);
        }
      }
      if (!more) return 1;
      if (n_rank != c_rank) {   // the next tile opens a new segment
        c_rank = n_rank;
        cs = ns;
        relocate(cs);
      }
      c_tile = n_tile;
      return 0;
    };
    int cur = 0;
    for (;;) {
      const int r = step(L + cur, L + (C::TILE_BYTES - cur));
      if (r != 0) break;
      cur = C::TILE_BYTES - cur;
    }
    if (!restart) break;
    // drain the prefetch in flight; the pair agrees on its tile max and starts
    // over from the larger reference
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (pair_active && half == 0) stat[wave][l32] = mt;
    __builtin_amdgcn_s_barrier();
    m_init = pair_active ? fmaxf(m_run, fmaxf(stat[wave][l32], stat[wave ^ 1][l32])) : 0.f;
    restarted = true;
    __builtin_amdgcn_s_barrier();
  }

  // ---- epilogue: combine the pair's row sums, store normalized partial and lse ----
  if (pair_active && half == 0) stat[wave][l32] = l_run;
  __syncthreads();
  if (!valid) return;
  const float l_tot = l_run + stat[wave ^ 1][l32];
  const int64_t pidx = a.part_ptr[slot] + it.chunk;
  const float inv = 1.f / l_tot;
  float* dst = a.part_o + pidx * DC + kh * (DC / 2);
#pragma unroll
  for (int d = 0; d < C::OBH; ++d)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 v = {o[d][4 * i] * inv, o[d][4 * i + 1] * inv, o[d][4 * i + 2] * inv, o[d][4 * i + 3] * inv};
      *(f32x4*)(dst + d * 32 + half * 4 + 8 * i) = v;
    }
  if (kh == 0 && half == 0) a.part_lse[pidx] = (m_run + __log2f(l_tot)) * 0.6931471805599453f;
}

// ----------------------------------------------------------------------------
// device half of the plan
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(256) void plan_slots_kernel(AttendArgs a) {
  const unsigned char* ws = a.ws;
  const SegInfo* segs = (const SegInfo*)(ws + a.hdr.off_segs);
  const int32_t* rank_seg = (const int32_t*)(ws + a.hdr.off_rank);
  const int32_t* storage = (const int32_t*)(ws + a.hdr.off_storage);
  const ChunkInfo* chunks = (const ChunkInfo*)(ws + a.hdr.off_chunks);
  const int32_t* prot_seg = (const int32_t*)(ws + a.hdr.off_prot_seg);
  const int64_t* cum_local = (const int64_t*)(ws + a.hdr.off_cum_local);
  const int64_t nglob = a.n_rows * a.n_groups;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i <= a.n_slots;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i == a.n_slots) {
      a.part_ptr[i] = a.hdr.n_parts;
      continue;
    }
    int s;
    int64_t base;
    if (i < nglob) {
      const int64_t r = i / a.n_groups, g = i - r * a.n_groups;
      int lo = 0, hi = a.hdr.n_segs - 1;    // last segment (storage order) with kv_start <= r
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (segs[storage[mid]].kv_start <= r) lo = mid; else hi = mid - 1;
      }
      s = storage[lo];
      const SegInfo si = segs[s];
      base = si.cum_global + ((r - si.kv_start) * a.n_groups + g) * si.n_chunks;
    } else {
      const int64_t k = i - nglob;
      const int64_t ai = k / a.n_local, jj = k - ai * a.n_local;
      s = prot_seg[ai];
      base = a.hdr.global_parts + cum_local[ai] + jj * segs[s].n_chunks;
    }
    a.part_ptr[i] = base;
    if (a.part_seg != nullptr) {
      const SegInfo si = segs[s];
      for (int c = 0; c < si.n_chunks; ++c) {
        const ChunkInfo ch = chunks[si.chunk_off + c];
        a.part_seg[2 * (base + c)] = rank_seg[ch.first_rank];
        a.part_seg[2 * (base + c) + 1] = rank_seg[ch.last_rank];
      }
    }
  }
}

__global__ __launch_bounds__(256) void row_src_kernel(AttendArgs a) {
  const int32_t* prot = (const int32_t*)(a.ws + a.hdr.off_prot);
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < a.n_rows;
       r += (int64_t)gridDim.x * blockDim.x) {
    int lo = 0, hi = a.n_prot;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (prot[mid] < r) lo = mid + 1; else hi = mid;
    }
    a.row_src[r] = (lo < a.n_prot && prot[lo] == r) ? 1 : 0;
  }
}

hipError_t launch_plan(const AttendArgs& a, hipStream_t s) {
  const int64_t n = a.n_slots + 1;
  const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 8192);
  plan_slots_kernel<<<dim3(blocks), dim3(256), 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.row_src == nullptr) return e;
  const unsigned rb = (unsigned)std::min<int64_t>((a.n_rows + 255) / 256, 4096);
  row_src_kernel<<<dim3(rb), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  const unsigned grid = (unsigned)(((int64_t)a.n_items + 255) / 256 * 256);
  if (a.d_latent == 512 && a.d_rope == 64)
    attend_kernel<512, 64><<<dim3(grid), dim3(256), 0, s>>>(a);
  else if (a.d_latent == 64 && a.d_rope == 16)
    attend_kernel<64, 16><<<dim3(grid), dim3(256), 0, s>>>(a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace mla
