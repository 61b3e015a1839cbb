// Query-side RoPE relocation and segment-wise absorbed-MLA attention over the
// packed latent stream (Sec. 2.3 eq:rope, Alg. 2 SelectiveMLA), plus the
// device half of the plan (partial index, segment bookkeeping, protected flags).
//
// Work item = up to 128 head-rows (query rows x heads) that share every key of
// the single latent stream (the latent is never split per head, Sec. 2.1).
// One 256-thread workgroup walks the item's visible segments in request order
// and streams each segment's 64-key latent tiles through LDS once for all its
// head-rows.  Each of the 4 waves owns 32 head-rows outright:
//   relocation      rotate the RoPE part of its queries by R(t - p_s) into the
//                   segment's canonical frame when a new segment starts
//   S^T = K Q^T     64 keys x 32 head-rows (MFMA 32x32x16 bf16; K read from
//                   LDS, the d_c + d_r query dims resident in registers)
//   softmax         one head-row per lane pair, against a fixed reference max
//   O^T += V^T P^T  d_c latent dims x 32 head-rows; V is the same LDS tile read
//                   with transposing LDS loads, P^T is the S^T accumulator
//                   rounded to bf16 in place (its lane layout is already the
//                   MFMA operand layout once the keys are taken in the order
//                   the V reads use); with a rotary value (the whole latent row
//                   is the value) also the d_r RoPE dims, whose sums live in the
//                   workspace and are rotated back per segment (RestorePhase,
//                   R^-1: Alg. 2, eq:offonline)
// and emits one normalized partial and one log-sum-exp per (slot, chunk), or,
// with one chunk per slot, the merged head output itself.
// Tiles are fetched with 16-byte direct-to-LDS loads, double-buffered; the
// 16-byte chunks of a key row are XOR-swizzled so row and column reads hit
// distinct banks.
#include "common.h"
#include "restart.h"

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
  static constexpr int OB = DC / 32;         // 32-dim output blocks of O^T
  static constexpr int PS = BK / 16;         // 16-key contraction steps of P.V per tile
  static_assert(DR == 16 || DR % 32 == 0, "d_rope must be 16 or a multiple of 32");
  static_assert(DC % 64 == 0, "d_latent must be a multiple of 64");
  static_assert(kTileRows == 128, "one work item is 4 waves x 32 head-rows");
};

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

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

// S^T accumulation on the matrix cores with the accumulators pinned to
// architectural VGPRs: the O^T accumulators of the tile loop fill the whole
// accumulation register file, so S^T is kept out of it.  Back-to-back
// accumulation into the same registers needs no wait states; a vector ALU read
// of the result does (s_acc_ready), and so does an MFMA read of a register that
// a vector ALU op has just written (the leading s_nop of s_acc_first).
__device__ __forceinline__ void s_acc_first(f32x16& s0, f32x16& s1, const bf16x8& k0, const bf16x8& k1,
                                            const bf16x8& q) {
  asm("s_nop 4\n\t"
      "v_mfma_f32_32x32x16_bf16 %0, %2, %4, 0\n\t"
      "v_mfma_f32_32x32x16_bf16 %1, %3, %4, 0"
      : "=&v"(s0), "=&v"(s1)
      : "v"(k0), "v"(k1), "v"(q));
}
__device__ __forceinline__ void s_acc(f32x16& s0, f32x16& s1, const bf16x8& k0, const bf16x8& k1,
                                      const bf16x8& q) {
  asm("v_mfma_f32_32x32x16_bf16 %0, %2, %4, %0\n\t"
      "v_mfma_f32_32x32x16_bf16 %1, %3, %4, %1"
      : "+v"(s0), "+v"(s1)
      : "v"(k0), "v"(k1), "v"(q));
}
// A rotary value's RoPE output block: r += V P for one 16-key step, in
// architectural VGPRs for the same reason.  The compiler does not see an MFMA
// here, so the asm carries the wait states itself: the leading s_nop covers a
// vector ALU write of P just before (the compiler packs P's bf16 pairs lazily,
// next to their first use), r_acc_ready a memory or vector ALU read of r after.
__device__ __forceinline__ void r_acc1(f32x16& r, const bf16x8& v, const bf16x8& p) {
  asm("s_nop 4\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(r) : "v"(v), "v"(p));
}
__device__ __forceinline__ void r_acc_ready(f32x16& r) { asm("s_nop 15\n\ts_nop 7" : "+v"(r)); }
// 24 wait states: more than an XDL result needs before a vector ALU read
__device__ __forceinline__ void s_acc_ready(f32x16& s0, f32x16& s1) {
  asm("s_nop 15\n\ts_nop 7" : "+v"(s0), "+v"(s1));
}

// Tile barrier: this wave's direct-to-LDS loads and LDS accesses are complete,
// then all waves meet.  One asm statement with a memory clobber, so the
// compiler moves no LDS access across it.
__device__ __forceinline__ void tile_barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// value of lane l%32 and of lane l%32 + 32, in every lane (one permlane swap)
__device__ __forceinline__ void lane_halves(float v, float& x, float& y) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  x = __uint_as_float(r[0]);
  y = __uint_as_float(r[1]);
}

// What a work item's waves take from the plan: the tables, the item, and this
// lane's head-row (its storage row, query, output slot and request position).
// Blocks are dispatched round-robin over the 8 XCDs; each XCD gets 32
// consecutive items (similar key ranges) per group of 256.
struct ItemView {
  const SegInfo* segs;
  const int32_t* rank_seg;
  const double* theta_rev;
  WorkItem it;
  SegInfo own;
  ChunkInfo chk;
  bool valid;    // this lane has a head-row
  bool active;   // wave-uniform: the wave has head-rows
  int64_t row, slot, t_pos;
  const uint16_t* qsrc;
};

__device__ __forceinline__ int xcd_item_id(int b) {
  const int xcd = b & 7, kx = b >> 3;
  return (kx >> 5) * 256 + xcd * 32 + (kx & 31);
}

// work items of this launch: the host plan's count, or the device plan's
__device__ __forceinline__ int item_count(const AttendArgs& a) {
  return a.dyn != nullptr ? a.dyn->n_items : a.n_items;
}

template <class C>
__device__ __forceinline__ ItemView item_view(const AttendArgs& a, int item_id, int wave, int l32) {
  ItemView v;
  v.segs = a.segs;
  v.rank_seg = a.rank_seg;
  v.theta_rev = a.theta_rev;
  const int32_t* prot = a.prot;
  v.it = a.items[item_id];
  v.own = v.segs[v.it.seg];
  v.chk = a.chunks[v.own.chunk_off + v.it.chunk];
  const int hr_local = wave * 32 + l32;
  v.valid = hr_local < v.it.count;
  v.active = wave * 32 < v.it.count;
  const int64_t hr = v.it.hr_begin + (v.valid ? hr_local : 0);
  if (v.it.kind == 0) {
    v.row = hr / a.n_groups;
    v.qsrc = (const uint16_t*)a.q_glob + hr * C::D;
    v.slot = hr;
  } else {
    v.row = prot[hr / a.n_local];
    v.qsrc = (const uint16_t*)a.q_loc + hr * C::D;
    v.slot = a.local_slot_base + hr;
  }
  v.t_pos = v.own.req_offset + (v.row - v.own.kv_start);
  return v;
}

// visible keys of segment s for the item: its own segment up to the item's last row
__device__ __forceinline__ int64_t seg_keys(const ItemView& v, const SegInfo& s, bool is_own) {
  return is_own ? (int64_t)v.it.max_u + 1 : s.length;
}

// Direct-to-LDS loads of tile `tile` of segment `s` (n_keys visible keys) into
// dbuf: wave w fills key-blocks 2w, 2w+1; lane l loads key l>>3 of a block, the
// 16-byte chunk at physical slot l&7 of each 8-chunk group.  Rows past the
// segment's end repeat its last row.
template <class C>
__device__ __forceinline__ void issue_tile(const void* kv, const SegInfo& s, int64_t n_keys, int64_t tile,
                                           unsigned char MLA_LDS* dbuf, int wave, int lkey, int lchunk_full,
                                           int lchunk_part) {
  const int64_t k0 = tile * C::BK;
  const int last = (int)(n_keys - 1 - k0);
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
    const unsigned char* base = (const unsigned char*)kv + (s.kv_start + brow) * (C::D * 2);
    const uint32_t roff = (uint32_t)(kr * (C::D * 2));   // never negative
#pragma unroll
    for (int cg = 0; cg < C::CG; ++cg) {
      const int ch = cg * 8 + (cg < C::CGF ? lchunk_full : lchunk_part);
      dma16(base, roff + ch * 16, dbuf + kb8 * C::KB8 + cg * 1024);
    }
  }
}

// Relocation for a new segment s (Sec. 2.3 eq:rope): rotate the RoPE part of
// this lane's query by R(t - p_s) into qf's RoPE steps; the angle is reduced in
// double precision (in revolutions) and fed to the hardware sin/cos.  Returns
// the lane's largest visible canonical offset in s (INT_MAX without a head-row).
template <class C, int DC, int DR, bool RELOAD = true>
__device__ __forceinline__ int relocate_query(bf16x8 (&qf)[C::KS], const ItemView& v, const SegInfo& s, int half) {
  const int64_t delta = v.t_pos - s.req_offset;
  const int64_t lm = delta < s.length - 1 ? delta : s.length - 1;
  bf16x8 raw[C::RS];
#pragma unroll
  for (int rs = 0; rs < C::RS; ++rs) {
    if (!RELOAD) {
      raw[rs] = qf[C::CS + rs];   // still the unrotated query
    } else if (DR == 16) {
      const u32x2 lo = *(const u32x2*)(v.qsrc + DC + half * 4);
      const u32x2 hi = *(const u32x2*)(v.qsrc + DC + 8 + half * 4);
      raw[rs] = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
    } else {
      raw[rs] = *(const bf16x8*)(v.qsrc + DC + rs * 16 + half * 8);
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
      const double rev = dd * v.theta_rev[j0 + half * jstep];
      const float r = (float)(rev - rint(rev));
      const float sn = __builtin_amdgcn_sinf(r), cn = __builtin_amdgcn_cosf(r);
      const float x1 = (float)raw[rs][i], x2 = (float)raw[prs][ps];
      qf[C::CS + rs][i] = v.valid ? (__bf16)(x1 * cn - x2 * sn) : (__bf16)0.f;
      qf[C::CS + prs][ps] = v.valid ? (__bf16)(x1 * sn + x2 * cn) : (__bf16)0.f;
    }
  }
  return v.valid ? (int)lm : 0x7fffffff;
}

// A lane's share of a 64-dim RoPE output row held as two 32-dim MFMA output
// blocks: register 4i + j of block dd is dim dd*32 + half*4 + 8i + j, so each
// rotation pair (k, k + 32) sits in one register of the two blocks.
__device__ __forceinline__ void rot_store(float* p, int half, const f32x16 (&r)[2]) {
#pragma unroll
  for (int dd = 0; dd < 2; ++dd)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *(f32x4*)(p + dd * 32 + half * 4 + 8 * i) = f32x4{r[dd][4 * i], r[dd][4 * i + 1], r[dd][4 * i + 2], r[dd][4 * i + 3]};
}
// tot += R(-dd*theta) acc, pair by pair: the angle reduced in double precision
// (revolutions) and fed to the hardware sin/cos
__device__ __forceinline__ void rot_accumulate(f32x16 (&tot)[2], const f32x16 (&acc)[2], double dd,
                                               const double* theta_rev, int half) {
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int k = half * 4 + (e >> 2) * 8 + (e & 3);
    const double rev = dd * theta_rev[k];
    const float r = (float)(rev - rint(rev));
    const float sn = __builtin_amdgcn_sinf(r), cn = __builtin_amdgcn_cosf(r);
    const float x = acc[0][e], y = acc[1][e];
    tot[0][e] += x * cn + y * sn;
    tot[1][e] += y * cn - x * sn;
  }
}

// Rotary-value accumulators of one wave in device memory, lane-major: four
// 32-dim blocks (0, 1: the current segment's RoPE output sum, canonical frame;
// 2, 3: the row's total, query frame), each 4 KB = four 1 KB runs, run i holding
// registers 4i..4i+3 of every lane at 16 bytes per lane, so that each 16-byte
// load or store of a wave is one contiguous kilobyte.  The wave's base is
// uniform and the lane's byte offset is recomputed at each use (an opaque asm,
// so that no 64-bit per-lane pointer is hoisted out of the tile loop and held in
// registers): the loads and stores take the scalar-base + 32-bit offset form.
__device__ __forceinline__ uint32_t lane_x16() {
  uint32_t v;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0\n\tv_lshlrev_b32 %0, 4, %0" : "=v"(v));
  return v;
}
__device__ __forceinline__ float* rot_run(float* w, int b, int i, uint32_t lo) {
  return (float*)((char*)w + (uint32_t)(b * 4096 + i * 1024) + lo);
}
__device__ __forceinline__ float* rot_run(float* w, int b, int i) { return rot_run(w, b, i, lane_x16()); }
__device__ __forceinline__ void rot_blk_load(float* w, int b, f32x16& r) {
  const uint32_t lo = lane_x16();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f32x4 x = *(const f32x4*)rot_run(w, b, i, lo);
#pragma unroll
    for (int j = 0; j < 4; ++j) r[4 * i + j] = x[j];
  }
}
__device__ __forceinline__ void rot_blk_store(float* w, int b, const f32x16& r) {
  const uint32_t lo = lane_x16();
#pragma unroll
  for (int i = 0; i < 4; ++i)
    *(f32x4*)rot_run(w, b, i, lo) = f32x4{r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]};
}
// all four blocks cleared
__device__ __forceinline__ void rot_clear(float* w) {
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) *(f32x4*)rot_run(w, b, i) = f32x4{0.f, 0.f, 0.f, 0.f};
}
// Close a segment: its sum, rotated by R(-dd*theta), added into the row's
// total, and the sum cleared for the next segment; one run at a time, so that
// few registers are live.  The register 4i + j of block 0 is dim
// half*4 + 8i + j and its rotation partner (+32) the same register of block 1.
__device__ __forceinline__ void rot_close(float* w, double dd, const double* theta_rev) {
  const int half = (int)(__lane_id() >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f32x4 x = *(const f32x4*)rot_run(w, 0, i), y = *(const f32x4*)rot_run(w, 1, i);
    f32x4 tx = *(const f32x4*)rot_run(w, 2, i), ty = *(const f32x4*)rot_run(w, 3, i);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const double rev = dd * theta_rev[half * 4 + 8 * i + j];
      const float r = (float)(rev - rint(rev));
      const float sn = __builtin_amdgcn_sinf(r), cn = __builtin_amdgcn_cosf(r);
      tx[j] += x[j] * cn + y[j] * sn;
      ty[j] += y[j] * cn - x[j] * sn;
    }
    *(f32x4*)rot_run(w, 2, i) = tx;
    *(f32x4*)rot_run(w, 3, i) = ty;
    *(f32x4*)rot_run(w, 0, i) = f32x4{0.f, 0.f, 0.f, 0.f};
    *(f32x4*)rot_run(w, 1, i) = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// Order of a tile's P.V MFMAs with a rotary value: the n_lat latent MFMAs in
// order, and the 8 RoPE-block MFMAs (block b, 16-key step j) placed after latent
// MFMA kRopeAfter[b] + 3j.  Each block's 16 accumulators are then loaded ~14
// latent MFMAs before their first use and stored ~16 before the tile's end, and
// only one block is in registers at a time.  code[st] of sequence step st: the
// latent index, or -1 - (4b + j) for a RoPE step.
constexpr int kRopeAfter[2] = {13, 37};
template <int NLAT, bool ROT>
struct PvOrder {
  static constexpr int n = NLAT + (ROT ? 8 : 0);
  int code[n];
  constexpr PvOrder() : code() {
    int l = 0, r = 0;
    for (int k = 0; k < n; ++k) {
      const bool rope = ROT && r < 8 && l == kRopeAfter[r >> 2] + 3 * (r & 3) + 1;
      code[k] = rope ? -1 - r : l;
      if (rope) ++r; else ++l;
    }
  }
};

template <int DC, int DR, bool ROT>
__global__ __launch_bounds__(256, 1) void attend_kernel(AttendArgs a) {
  using C = Cfg<DC, DR>;
  static_assert(!ROT || DR == 64, "rotation pairs (j, j + 32) sit in one lane of the two RoPE output blocks");
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * C::TILE_BYTES];
  __shared__ unsigned restart_at;

  unsigned char MLA_LDS* L = (unsigned char MLA_LDS*)lds;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, l32 = lane & 31;

  const int item_id = xcd_item_id(blockIdx.x);
  if (item_id >= item_count(a)) return;
  const ItemView v = item_view<C>(a, item_id, wave, l32);
  const SegInfo* segs = v.segs;
  const int32_t* rank_seg = v.rank_seg;
  const WorkItem& it = v.it;
  const ChunkInfo& chk = v.chk;
  const bool valid = v.valid, active = v.active;
  const int64_t slot = v.slot;
  const uint16_t* qsrc = v.qsrc;
  // rotary value: the wave's accumulators in device memory (the registers are
  // full), 16 KB per wave (rot_run); the address is recomputed from the item and
  // wave at each use, so that it holds no register across the tile loop
  auto rot = [&]() -> float* { return a.rot + ((int64_t)item_id * 4 + wave) * 4096; };

  // ---- Q fragments (B operand of S^T = K Q^T), loaded once the first tile's loads
  // are out: step ks holds dims ks*16 + half*8 .. +8; for DR == 16 the RoPE step
  // holds rope dims {half*4..+4} and {8+half*4..+4}, so that every rotation pair
  // (j, j + d_r/2) stays inside one lane.
  bf16x8 qf[C::KS];

  f32x16 o[C::OB];
  float m_run = -1e30f, l_run = 0.f;

  // ---- per-lane LDS address bases (everything else is an immediate offset) ----
  // K as the A operand: key kt*32 + l32 of the tile (kt adds 4 key-blocks), chunk
  // 2*(ks&3) + half of chunk group ks>>2
  int abase[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4)
    abase[s4] = (l32 >> 3) * C::KB8 + (l32 & 7) * 128 + (((2 * s4 + half) ^ rotl3(l32 & 7)) * 16);
  // V^T via transposing reads.  P.V step s2 contracts tile keys 16*s2 .. 16*s2+15 in
  // the order the S^T accumulator holds them: lane half h takes keys 16*s2 + h*4 + 0..3
  // (8-key block 2*s2) and 16*s2 + 8 + h*4 + 0..3 (block 2*s2 + 1).  In each 16-lane
  // group q4 = lane/16, lane j = rr*4 + cb addresses key h*4 + rr of the block and
  // latent dims (q4&1)*16 + cb*4 .. +3 of a 32-dim output block; lane j then receives
  // dim (q4&1)*16 + j of those four keys.  Output block d covers chunk group d>>1 at
  // chunk offset (d&1)*4; vb[d&1][s2>>1] is the base for block parity d&1 and key
  // half s2>>1 of the tile, block d adds (d>>1)*1024 and step s2 adds (s2&1)*2*KB8.
  const int q4 = lane >> 4, rr = (lane >> 2) & 3, cb = lane & 3;
  const int vkey = (q4 >> 1) * 4 + rr;
  int vb[2][2];
#pragma unroll
  for (int dp = 0; dp < 2; ++dp)
#pragma unroll
    for (int kq = 0; kq < 2; ++kq)
      vb[dp][kq] = vkey * 128 + (((dp * 4 + (q4 & 1) * 2 + (cb >> 1)) ^ rotl3(vkey)) * 16) + (cb & 1) * 8 +
                   kq * 4 * C::KB8;
  // direct loads: lane l fills key l>>3 of an 8-key block, physical slot l&7
  const int lkey = lane >> 3;
  const int lchunk_full = (lane & 7) ^ rotl3(lkey);
  const int lchunk_part = (lane & 7) < (C::CH - C::CGF * 8) ? (lane & 7) : 0;


  auto issue = [&](unsigned char MLA_LDS* dbuf, const SegInfo& s, int64_t n_keys, int64_t tile) {
    issue_tile<C>(a.kv, s, n_keys, tile, dbuf, wave, lkey, lchunk_full, lchunk_part);
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

  // relocation for a new segment: this lane's query in the segment's canonical
  // frame, and the visibility limits of the lane and of the wave
  auto relocate = [&](const SegInfo& s) {
    lim = relocate_query<C, DC, DR>(qf, v, s, half);
    wave_lim = wave_min_i(lim);
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
    n_keys = seg_keys(v, ns, sidx == it.seg);
    n_ntiles = (n_keys + C::BK - 1) / C::BK;
    n_tile = 0;
    return true;
  };

  // The softmax reference m_run is the first tile's row max (log2 units), so a
  // later tile's weights 2^(s - m_run) are not bounded by 1.  A tile in which a
  // lane's weights sum to 2^64 or more (fp32 sums and bf16 weights hold every
  // weight below that without loss) restarts the whole item with that row's
  // reference raised to m_run + log2 of the larger sum of its two lanes: less
  // than 6 above the row's max over the tile (32 keys per lane), at least 64 above
  // m_run, so a reference that is still too low is raised again by 64 or more on
  // the next attempt (by 128 when a weight overflowed fp32).  A NaN sum never
  // votes, and the item's last permitted attempt casts no vote at all, so the
  // number of passes is bounded (restart.h).  A wave that sees
  // such a tile records its index (1-based) with an LDS atomic min in
  // restart_at; after the barrier that opens tile t every wave tests restart_at
  // <= t, which only votes cast before that barrier can satisfy, so all waves
  // leave the tile loop at the same tile (the tiles computed in between are
  // discarded with the rest).  The tile loop thus never applies vector ALU work
  // to the O accumulators, which stay in the matrix-core accumulation registers.
  // the first tile's loads go out before the queries are read, so that the two
  // latencies overlap at the start of an item
  {
    const SegInfo s0 = segs[rank_seg[chk.first_rank]];
    issue(L, s0, seg_keys(v, s0, rank_seg[chk.first_rank] == it.seg), 0);
  }
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
  const float sl2 = a.scale_log2;
  float m_init = -1e30f;
  bool restarted = false;
  int attempt = 0;                  // passes made over the item (workgroup-uniform)
  if (tid == 0) restart_at = ~0u;   // ordered before any access by the first tile barrier
  // the first attempt's relocation for the chunk's first segment, from the
  // unrotated RoPE part still in qf
  {
    const SegInfo s0 = segs[rank_seg[chk.first_rank]];
    lim = relocate_query<C, DC, DR, false>(qf, v, s0, half);
    wave_lim = wave_min_i(lim);
  }
  for (;;) {
#pragma unroll
    for (int d = 0; d < C::OB; ++d)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[d][e] = 0.f;
    m_run = m_init;
    l_run = 0.f;
    float m_seen = m_init;
    c_rank = chk.first_rank;
    cs = segs[rank_seg[c_rank]];
    c_tile = 0;
    n_rank = c_rank;
    ns = cs;
    n_keys = seg_keys(v, cs, rank_seg[c_rank] == it.seg);
    n_ntiles = (n_keys + C::BK - 1) / C::BK;
    n_tile = 0;
    if (restarted) {
      relocate(cs);
      issue(L, cs, n_keys, 0);   // the first attempt's went out before the queries
    }

    if (ROT && active) rot_clear(rot());
    bool restart = false;
    const bool may_vote = restart_allowed(attempt);   // uniform: the last attempt never votes
    bool first_tile = !restarted;   // uniform over the workgroup
    unsigned ti = 0;                 // tile index within the attempt (uniform)
    int cur = 0;
    for (;;) {
      // The tile in buffer `cur` has landed (this wave's loads: vmcnt; the other
      // waves' loads: the barrier), every wave has finished reading the other
      // buffer, and the restart votes cast during the previous tile are visible.
      tile_barrier();
      if (*(volatile unsigned MLA_LDS*)&restart_at <= ti) {
        restart = true;
        break;
      }
      const bool more = advance();
      if (more) issue(L + (C::TILE_BYTES - cur), ns, n_keys, n_tile);
      const unsigned char MLA_LDS* buf = L + cur;
      if (active) {
        // ---- S^T = K Q^T: keys 0..31 into s[0], keys 32..63 into s[1] ----
        f32x16 s[2];
        auto kfrag = [&](int kt, int ks) -> bf16x8 {
          if (DR == 16 && ks == C::CS) {
            // rope chunks 2*CS, 2*CS+1 sit in the partial (unswizzled) group: 8 bytes each
            const int base0 = (kt * 4 + (l32 >> 3)) * C::KB8 + (l32 & 7) * 128 + C::CGF * 1024 + half * 8;
            const u32x2 x0 = *(const u32x2 MLA_LDS*)(buf + base0);
            const u32x2 y0 = *(const u32x2 MLA_LDS*)(buf + base0 + 16);
            return __builtin_bit_cast(bf16x8, u32x4{x0[0], x0[1], y0[0], y0[1]});
          }
          return *(const bf16x8 MLA_LDS*)(buf + abase[ks & 3] + (ks >> 2) * 1024 + kt * 4 * C::KB8);
        };
        // K fragments are read two steps ahead of their MFMAs; the scheduling
        // barriers keep the compiler from sinking the reads next to their use
        bf16x8 ka[3][2];
        ka[0][0] = kfrag(0, 0);
        ka[0][1] = kfrag(1, 0);
        ka[1][0] = kfrag(0, 1);
        ka[1][1] = kfrag(1, 1);
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) {
          if (ks + 2 < C::KS) {
            ka[(ks + 2) % 3][0] = kfrag(0, ks + 2);
            ka[(ks + 2) % 3][1] = kfrag(1, ks + 2);
          }
          __builtin_amdgcn_sched_barrier(0);
          if (ks == 0)
            s_acc_first(s[0], s[1], ka[0][0], ka[0][1], qf[0]);
          else
            s_acc(s[0], s[1], ka[ks % 3][0], ka[ks % 3][1], qf[ks]);
          __builtin_amdgcn_sched_barrier(0);
        }
        // the first V^T fragments of P.V do not depend on the softmax: read them now
        constexpr int NPV = C::PS * C::OB;
        // rotary value: K_r^T P^T into the two RoPE output blocks, placed by pv_code
        constexpr int NRV = ROT ? 2 * C::PS : 0;
        constexpr int VD = 3;   // V^T fragments in flight ahead of their MFMA
        constexpr PvOrder<NPV, ROT> order{};
        auto vfrag = [&](int st) -> bf16x8 {
          int s2 = st / C::OB, d = st % C::OB;
          if constexpr (ROT) {
            const int code = order.code[st];
            s2 = code >= 0 ? code / C::OB : (-1 - code) & 3;
            d = code >= 0 ? code % C::OB : C::OB + ((-1 - code) >> 2);
          }
          const int off = vb[d & 1][s2 >> 1] + (d >> 1) * 1024 + (s2 & 1) * 2 * C::KB8;
          const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((MLA_LDS bf16x4*)(buf + off));
          const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((MLA_LDS bf16x4*)(buf + off + C::KB8));
          return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        };
        bf16x8 vt[VD + 1];
#pragma unroll
        for (int j = 0; j < VD; ++j) vt[j] = vfrag(j);
        __builtin_amdgcn_sched_barrier(0);
        s_acc_ready(s[0], s[1]);
        // register e of s[kt] holds tile key kt*32 + half*4 + (e/4)*8 + e%4 (raw Q.K)
        const int tk0 = (int)(c_tile * C::BK);
        if (tk0 + C::BK - 1 > wave_lim) {
          // visible iff (e/4)*8 + e%4 (+32 for s[1]) <= lim - tk0 - half*4; the lane
          // half is recomputed from the lane id rather than kept live across the loop
          const int rel = lim - tk0 - ((int)(__lane_id() >> 5) << 2);
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = (e >> 2) * 8 + (e & 3);
            if (key > rel) s[0][e] = -INFINITY;
            if (key + 32 > rel) s[1][e] = -INFINITY;
          }
        }
        // the row max only where it sets the reference: the first tile of an item
        auto row_max = [&]() -> float {
          float m = fmaxf(s[0][0], s[1][0]);
#pragma unroll
          for (int e = 1; e < 16; ++e) m = fmaxf(m, fmaxf(s[0][e], s[1][e]));
          float mx, my;
          lane_halves(m, mx, my);
          return fmaxf(mx, my) * sl2;   // row max of the tile, log2 units (sl2 > 0)
        };
        if (first_tile) {
          m_run = row_max();
          m_seen = fmaxf(m_seen, m_run);
        }
        // ---- softmax weights 2^(s*scale*log2e - m_run), rounded to bf16 in place:
        // pf[s2] is the B operand (P^T) of P.V step s2 ----
        bf16x8 pf[C::PS];
        const float nm = -m_run;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            pf[kt * 2 + (e >> 3)][e & 7] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][e], sl2, nm));
        // this lane's share of the row sum: the rounded weights that P.V uses, two per dot product
        float rsum;
        {
          const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
          float r0 = 0.f, r1 = 0.f;
#pragma unroll
          for (int s2 = 0; s2 < C::PS; ++s2) {
            // constant-index shuffles (a bit_cast of a vector element would read element 0)
            const bf16x8 w = pf[s2];
            r0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 0, 1), one2, r0, false);
            r1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 2, 3), one2, r1, false);
            r0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 4, 5), one2, r0, false);
            r1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 6, 7), one2, r1, false);
          }
          rsum = r0 + r1;
        }
        if (__builtin_amdgcn_ballot_w64(may_vote && restart_vote(rsum)) != 0) {   // rare: restart vote
          float ax, ay;
          lane_halves(restart_raise(rsum), ax, ay);
          m_seen = raised_reference(m_seen, m_run, ax, ay);
          if (lane == 0) atomicMin(&restart_at, ti + 1);
        }
        l_run += rsum;   // this lane's keys only; the two halves are combined at the end

        // rotary value: the segment's running RoPE output sum, one 32-dim block at a time
        f32x16 racc;
        if (ROT) rot_blk_load(rot(), 0, racc);

        // ---- O^T += V^T P^T over the 64 keys: 16-key steps outer, output blocks inner ----
#pragma unroll
        for (int st = 0; st < NPV + NRV; ++st) {
          if (st + VD < NPV + NRV) vt[(st + VD) % (VD + 1)] = vfrag(st + VD);
          __builtin_amdgcn_sched_barrier(0);
          const int code = ROT ? order.code[st] : st;
          if (code >= 0) {
            const int s2 = code / C::OB, d = code % C::OB;
            o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vt[st % (VD + 1)], pf[s2], o[d], 0, 0, 0);
          } else {
            const int b = (-1 - code) >> 2, j = (-1 - code) & 3;
            r_acc1(racc, vt[st % (VD + 1)], pf[j]);
            if (j == 3) {
              // block b is complete: store it; block 1 is loaded into the same registers
              r_acc_ready(racc);
              rot_blk_store(rot(), b, racc);
              if (b == 0) rot_blk_load(rot(), 1, racc);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      first_tile = false;
      ++ti;
      if (!more) break;
      if (n_rank != c_rank) {   // the next tile opens a new segment
        if (ROT) {
          // the closing segment's sum, rotated by R(-(t - p_s)), into the row's total
          if (active) rot_close(rot(), (double)(v.t_pos - cs.req_offset), v.theta_rev);
        }
        c_rank = n_rank;
        cs = ns;
        relocate(cs);
      }
      c_tile = n_tile;
      cur = C::TILE_BYTES - cur;
    }
    if (!restart) {
      // votes cast during the last tile
      tile_barrier();
      restart = *(volatile unsigned MLA_LDS*)&restart_at != ~0u;
      if (!restart) break;
    }
    // every wave has seen the vote: drain the loads in flight, clear the vote
    // (ordered before the next votes by the next attempt's first tile barrier)
    // and start over from the largest row max seen
    tile_barrier();
    if (tid == 0) restart_at = ~0u;
    m_init = m_seen;
    restarted = true;
    ++attempt;
  }

  // ---- epilogue: combine the two lane halves' row sums, store normalized partial and lse ----
  float lx, ly;
  lane_halves(l_run, lx, ly);
  // bf16 head outputs go through LDS, where every lane of the wave helps
  const bool staged = a.out_direct != nullptr && a.out_direct_bf16;
  if (!valid && !staged) return;
  const float l_tot = lx + ly;
  const float inv = 1.f / l_tot;
  // rotary value: the last segment's sum into the row's total, normalized
  f32x16 vr[2];
  if (ROT) {
    f32x16 acc[2];
    rot_blk_load(rot(), 0, acc[0]);
    rot_blk_load(rot(), 1, acc[1]);
    rot_blk_load(rot(), 2, vr[0]);
    rot_blk_load(rot(), 3, vr[1]);
    rot_accumulate(vr, acc, (double)(v.t_pos - cs.req_offset), v.theta_rev, half);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      vr[0][e] *= inv;
      vr[1][e] *= inv;
    }
  }
  if (a.out_direct != nullptr) {
    // one chunk per slot (the merge done here by online rescaling, or the
    // offline producer): the head output itself, and its lse when asked for
    if (valid && a.part_lse != nullptr && half == 0)
      a.part_lse[slot] = (m_run + __log2f(l_tot)) * 0.6931471805599453f;
    if (a.out_direct_bf16) {
      // The wave's 32 head-rows own consecutive slots.  Their latent dims go
      // through the wave's part of the tile buffers (idle since the last tile
      // barrier): written in the accumulator layout (lane: row l32, dims half*4 +
      // 8i of each block), read back row-contiguous (lane: 8 consecutive dims;
      // DC/8 lanes a row), so each global store writes whole rows (one contiguous
      // kilobyte for d_c = 512).  Rows are padded by 8 bytes (1032 for d_c = 512),
      // so the 32 lanes of a half-wave write 64 distinct banks.
      constexpr int SROW = DC + 4;   // staged row, bf16 elements
      constexpr int LPR = DC / 8;    // lanes per row on the way out
      static_assert(4 * 32 * SROW * 2 <= 2 * C::TILE_BYTES && 64 % LPR == 0, "staging fits the tile buffers");
      uint16_t MLA_LDS* srow = (uint16_t MLA_LDS*)L + wave * 32 * SROW;
#pragma unroll
      for (int d = 0; d < C::OB; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          *(u32x2 MLA_LDS*)(srow + l32 * SROW + d * 32 + half * 4 + 8 * i) =
              u32x2{pack_bf16x2(o[d][4 * i] * inv, o[d][4 * i + 1] * inv),
                    pack_bf16x2(o[d][4 * i + 2] * inv, o[d][4 * i + 3] * inv)};
      const int nrow = it.count - wave * 32 < 32 ? it.count - wave * 32 : 32;   // valid rows of the wave
      const int64_t slot0 = (it.kind == 0 ? 0 : a.local_slot_base) + it.hr_begin + wave * 32;
      uint16_t* ob0 = (uint16_t*)a.out_direct + slot0 * a.dv;
      // rows of the wave in passes of 64 / LPR rows, eight passes' reads issued before
      // their stores (rows past nrow read stale staging bytes and store nothing)
      constexpr int RPI = 64 / LPR, NP = 32 / RPI, UB = NP < 8 ? NP : 8;
      const int rl = lane / LPR, cl = lane % LPR;
#pragma unroll
      for (int p0 = 0; p0 < NP; p0 += UB) {
        u32x4 t[UB];
#pragma unroll
        for (int j = 0; j < UB; ++j) t[j] = *(const u32x4 MLA_LDS*)(srow + ((p0 + j) * RPI + rl) * SROW + cl * 8);
#pragma unroll
        for (int j = 0; j < UB; ++j) {
          const int r = (p0 + j) * RPI + rl;
          if (r < nrow) *(u32x4*)(ob0 + (int64_t)r * a.dv + cl * 8) = t[j];
        }
      }
      if (!valid) return;
      uint16_t* ob = (uint16_t*)a.out_direct + slot * a.dv;
      if (ROT)
#pragma unroll
        for (int d = 0; d < 2; ++d)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            *(u32x2*)(ob + DC + d * 32 + half * 4 + 8 * i) = u32x2{pack_bf16x2(vr[d][4 * i], vr[d][4 * i + 1]),
                                                                   pack_bf16x2(vr[d][4 * i + 2], vr[d][4 * i + 3])};
    } else {
      float* of = (float*)a.out_direct + slot * a.dv;
#pragma unroll
      for (int d = 0; d < C::OB; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          *(f32x4*)(of + d * 32 + half * 4 + 8 * i) =
              f32x4{o[d][4 * i] * inv, o[d][4 * i + 1] * inv, o[d][4 * i + 2] * inv, o[d][4 * i + 3] * inv};
      if (ROT) rot_store(of + DC, half, vr);
    }
    return;
  }
  const int64_t pidx = a.part_ptr[slot] + it.chunk;
  float* dst = a.part_o + pidx * a.dv;
#pragma unroll
  for (int d = 0; d < C::OB; ++d)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 v = {o[d][4 * i] * inv, o[d][4 * i + 1] * inv, o[d][4 * i + 2] * inv, o[d][4 * i + 3] * inv};
      *(f32x4*)(dst + d * 32 + half * 4 + 8 * i) = v;
    }
  if (ROT) rot_store(dst + DC, half, vr);
  if (half == 0) a.part_lse[pidx] = (m_run + __log2f(l_tot)) * 0.6931471805599453f;
}


// ----------------------------------------------------------------------------
// device half of the plan
// ----------------------------------------------------------------------------
// segment (storage order) holding storage row r: the last one whose kv_start <= r
__device__ __forceinline__ int segment_of_row(const AttendArgs& a, int64_t r) {
  int lo = 0, hi = a.n_segs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[a.storage[mid]].kv_start <= r) lo = mid; else hi = mid - 1;
  }
  return a.storage[lo];
}

__global__ __launch_bounds__(256) void plan_slots_kernel(AttendArgs a) {
  const SegInfo* segs = a.segs;
  const int64_t n_slots = a.dyn != nullptr ? a.dyn->n_slots : a.n_slots;
  const int64_t n_parts = a.dyn != nullptr ? a.dyn->n_parts : a.n_parts;
  const int64_t nglob = a.n_rows * a.n_groups;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i <= n_slots;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i == n_slots) {
      a.part_ptr[i] = n_parts;
      continue;
    }
    int s;
    int64_t base;
    if (i < nglob) {
      const int64_t r = i / a.n_groups, g = i - r * a.n_groups;
      s = segment_of_row(a, r);
      const SegInfo si = segs[s];
      base = si.cum_global + ((r - si.kv_start) * a.n_groups + g) * si.n_chunks;
    } else {
      const int64_t k = i - nglob;
      const int64_t ai = k / a.n_local, jj = k - ai * a.n_local;
      if (a.dyn == nullptr) {
        s = a.prot_seg[ai];
        base = a.global_parts + a.cum_local[ai] + jj * segs[s].n_chunks;
      } else {
        s = segment_of_row(a, a.prot[ai]);
        const int64_t nch = segs[s].n_chunks;
        base = a.global_parts + a.seg_local_base[s] + ((ai - a.seg_prot_lo[s]) * a.n_local + jj) * nch;
      }
    }
    a.part_ptr[i] = base;
    if (a.part_seg != nullptr) {
      const SegInfo si = segs[s];
      for (int c = 0; c < si.n_chunks; ++c) {
        const ChunkInfo ch = a.chunks[si.chunk_off + c];
        a.part_seg[2 * (base + c)] = a.rank_seg[ch.first_rank];
        a.part_seg[2 * (base + c) + 1] = a.rank_seg[ch.last_rank];
      }
    }
  }
}

__global__ __launch_bounds__(256) void row_src_kernel(AttendArgs a) {
  const int32_t* prot = a.prot;
  const int n_prot = a.dyn != nullptr ? a.dyn->n_prot : a.n_prot;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < a.n_rows;
       r += (int64_t)gridDim.x * blockDim.x) {
    int lo = 0, hi = n_prot;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (prot[mid] < r) lo = mid + 1; else hi = mid;
    }
    a.row_src[r] = (lo < n_prot && prot[lo] == r) ? 1 : 0;
  }
}

// part_ptr / part_seg (when part_ptr is set) and row_src (when set); grids cover
// the host count of slots and rows (for a device plan, the capacity bound)
hipError_t launch_plan(const AttendArgs& a, hipStream_t s) {
  if (a.part_ptr != nullptr) {
    const int64_t n = a.n_slots + 1;
    const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 8192);
    plan_slots_kernel<<<dim3(blocks), dim3(256), 0, s>>>(a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.row_src == nullptr) return hipSuccess;
  const unsigned rb = (unsigned)std::min<int64_t>((a.n_rows + 255) / 256, 4096);
  row_src_kernel<<<dim3(rb), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  const unsigned grid = (unsigned)(((int64_t)a.n_items + 255) / 256 * 256);
  const bool rot = a.dv != a.d_latent;   // rotary value: the RoPE dims too (needs a.rot)
  if (rot && (a.d_latent != 512 || a.d_rope != 64 || a.rot == nullptr)) return hipErrorInvalidValue;
  if (a.d_latent == 512 && a.d_rope == 64) {
    if (rot)
      attend_kernel<512, 64, true><<<dim3(grid), dim3(256), 0, s>>>(a);
    else
      attend_kernel<512, 64, false><<<dim3(grid), dim3(256), 0, s>>>(a);
  } else if (a.d_latent == 64 && a.d_rope == 16) {
    attend_kernel<64, 16, false><<<dim3(grid), dim3(256), 0, s>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mla
