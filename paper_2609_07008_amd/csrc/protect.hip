// Protected token-row set (Sec. 2.3, eq:protected):
//   A = Q u N u D u B_edge u I_top u T_tail
// Q query rows, N new rows, D dirty rows, B_edge the first and last rows of every
// relocated segment, T_tail the most recent rows in request order, and I_top the
// rows the Indexer ranks highest, which top the protected share of the candidate
// rows (rows that have an artifact: neither query nor new rows) up to the
// controller's budget.
//
// Every row that I_top may take gets a unique 64-bit key: the score's IEEE-754
// totalOrder bits above the inverted row index, so the largest keys are the
// highest scores, equal scores going to the lower row.  I_top is then "the k
// largest keys", and the k-th largest key kth decides every row by one compare.
//
// Six kernels on the caller's stream (back-to-back launches; the workspace's
// control words and 4096-bin histogram arrive zeroed with the table upload, or,
// when the table comes from a plan image, are zeroed by a fill kernel first):
//   classify  (grid)  per row: its segment (binary search in the storage-ordered
//                     table, held in LDS when it has at most 1024 segments, then
//                     a forward walk over a thread's 8 consecutive rows), the
//                     flags and the key; per block: counts of candidate, fixed-set
//                     and eligible rows and a histogram of the top 12 key bits of
//                     the eligible rows, added into the global copies.
//   gather    (grid)  every block derives k from the counts and the budget, and
//                     the histogram bucket holding the k-th largest key; appends
//                     that bucket's keys to a list (staged in LDS, one device
//                     atomic per block).
//   select    (1 WG)  radix select of kth inside the list: 8-bit digits over the
//                     remaining 52 bits, per-wave LDS histograms, the digit found
//                     by a 64-lane scan.
//   count     (grid)  selected rows per 2048-row block;
//   scan      (1 WG)  exclusive offsets of the blocks and |A|;
//   write     (grid)  each block writes its selected rows at its offset, ascending.
#include "protect.h"

#include <algorithm>

namespace mla {
namespace {

constexpr int kBits1 = 12;                   // key bits resolved by the histogram
constexpr int kBins = 1 << kBits1;
constexpr int kRowsPerBlock = 2048;          // classify / count / write blocks: 256 threads x 8 rows
constexpr int kLdsSegs = 1024;               // tables up to this size are searched in LDS
constexpr int kSelectThreads = 1024;

struct ProtectCtl {                          // zero at entry (uploaded)
  unsigned long long n_cand, n_base, n_elig;  // classify
  unsigned long long n_list;                 // gather: keys appended
  long long k;                               // bucket: I_top size
  long long k_rem;                           // bucket: rank of kth inside its bucket (1-based)
  unsigned long long bucket;                 // bucket: top 12 bits of kth
  unsigned long long kth;                    // select
};

__device__ __forceinline__ uint32_t total_order_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u >> 31) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ ProtectCtl* ctl_of(const ProtectArgs& a) { return (ProtectCtl*)(a.ws + a.off_ctl); }

// Block-wide inclusive scan of one value per thread (NT threads, LDS scratch of NT).
template <int NT>
__device__ __forceinline__ unsigned long long block_scan(unsigned long long v, unsigned long long* sh) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int off = 1; off < NT; off <<= 1) {
    const unsigned long long x = tid >= off ? sh[tid - off] : 0ull;
    __syncthreads();
    sh[tid] += x;
    __syncthreads();
  }
  const unsigned long long r = sh[tid];
  __syncthreads();
  return r;
}

struct RowCounts {
  uint32_t cand = 0, base = 0, elig = 0;
};

// Flags and keys of the rows r0 .. r0+7 (r0 a multiple of 8): one binary search for
// r0's segment, then a forward walk.  kv_start / length / req / orig point at the
// table in LDS or in the workspace (the caller's branch decides, so each instance
// keeps one address space).
__device__ __forceinline__ void classify8(const ProtectArgs& a, int64_t r0, const int64_t* kv_start,
                                          const int64_t* length, const int64_t* req, const int32_t* orig,
                                          uint32_t* hist, RowCounts& c) {
  const int64_t n = a.n_rows;
  const int nr = (int)(n - r0 < 8 ? n - r0 : 8);
  float sc[8];
  uint8_t rf[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {   // issue every load before the search
    sc[j] = (a.scores && j < nr) ? a.scores[r0 + j] : 0.0f;
    rf[j] = (a.row_flags && j < nr) ? a.row_flags[r0 + j] : (uint8_t)0;
  }
  int lo = 0, hi = a.n_segs - 1;   // last segment (storage order) with kv_start <= r0
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (kv_start[mid] <= r0) lo = mid; else hi = mid - 1;
  }
  uint64_t f8 = 0;
  uint64_t* key = (uint64_t*)(a.ws + a.off_key);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (j >= nr) break;
    const int64_t r = r0 + j;
    while (lo + 1 < a.n_segs && kv_start[lo + 1] <= r) ++lo;
    const int64_t u = r - kv_start[lo];
    const int64_t pos = req[lo] + u;
    const bool q = orig[lo] == a.query_seg;
    const bool is_new = (rf[j] & 1) != 0, dirty = (rf[j] & 2) != 0;
    const bool relocated = req[lo] != 0 && !q;
    const bool edge = relocated && (u < a.edge_rows || u >= length[lo] - a.edge_rows);
    const bool recent = pos >= n - a.tail_rows;
    const bool base = q || is_new || dirty || edge || recent;
    const bool cand = !q && !is_new;
    const bool elig = cand && !base;
    // bit 0: in the fixed sets; bit 1: candidate row; bit 2: eligible for I_top
    f8 |= (uint64_t)((base ? 1 : 0) | (cand ? 2 : 0) | (elig ? 4 : 0)) << (8 * j);
    const uint32_t sb = a.scores ? total_order_bits(sc[j]) : 0u;
    const uint64_t k = ((uint64_t)sb << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)r);
    key[r] = k;
    c.cand += cand;
    c.base += cand && base;
    c.elig += elig;
    if (elig) atomicAdd(&hist[k >> (64 - kBits1)], 1u);
  }
  uint8_t* fl = (uint8_t*)(a.ws + a.off_flag);
  if (nr == 8) {
    *(uint64_t*)(fl + r0) = f8;
  } else {
    for (int j = 0; j < nr; ++j) fl[r0 + j] = (uint8_t)(f8 >> (8 * j));
  }
}

__global__ __launch_bounds__(256) void protect_classify_kernel(ProtectArgs a) {
  __shared__ uint32_t hist[kBins];
  __shared__ int64_t s_kv[kLdsSegs], s_len[kLdsSegs], s_req[kLdsSegs];
  __shared__ int32_t s_orig[kLdsSegs];
  __shared__ unsigned long long cnt[3];
  const int64_t* g_kv = (const int64_t*)(a.table + a.off_kv);
  const int64_t* g_len = (const int64_t*)(a.table + a.off_len);
  const int64_t* g_req = (const int64_t*)(a.table + a.off_req);
  const int32_t* g_orig = (const int32_t*)(a.table + a.off_orig);
  const bool in_lds = a.n_segs <= kLdsSegs;
  for (int i = threadIdx.x; i < kBins; i += 256) hist[i] = 0;
  if (in_lds) {
    for (int i = threadIdx.x; i < a.n_segs; i += 256) {
      s_kv[i] = g_kv[i];
      s_len[i] = g_len[i];
      s_req[i] = g_req[i];
      s_orig[i] = g_orig[i];
    }
  }
  if (threadIdx.x < 3) cnt[threadIdx.x] = 0;
  __syncthreads();
  RowCounts c;
  const int64_t stride = (int64_t)gridDim.x * kRowsPerBlock;
  const int64_t first = (int64_t)blockIdx.x * kRowsPerBlock + threadIdx.x * 8;
  if (in_lds) {
    for (int64_t r0 = first; r0 < a.n_rows; r0 += stride) classify8(a, r0, s_kv, s_len, s_req, s_orig, hist, c);
  } else {
    for (int64_t r0 = first; r0 < a.n_rows; r0 += stride) classify8(a, r0, g_kv, g_len, g_req, g_orig, hist, c);
  }
  atomicAdd(&cnt[0], (unsigned long long)c.cand);
  atomicAdd(&cnt[1], (unsigned long long)c.base);
  atomicAdd(&cnt[2], (unsigned long long)c.elig);
  __syncthreads();
  ProtectCtl* ctl = ctl_of(a);
  if (threadIdx.x == 0) {
    atomicAdd(&ctl->n_cand, cnt[0]);
    atomicAdd(&ctl->n_base, cnt[1]);
    atomicAdd(&ctl->n_elig, cnt[2]);
  }
  uint32_t* g_hist = (uint32_t*)(a.ws + a.off_hist);
  for (int i = threadIdx.x; i < kBins; i += 256) {
    const uint32_t h = hist[i];
    if (h) atomicAdd(&g_hist[i], h);
  }
}

// k, the bucket of the k-th largest eligible key and kth's rank inside it, from
// the counts and the histogram; every gather block derives the same values.
__global__ __launch_bounds__(256) void protect_gather_kernel(ProtectArgs a) {
  constexpr int BPT = kBins / 256;           // histogram bins per thread
  __shared__ unsigned long long sh[256];
  __shared__ uint64_t buf[kRowsPerBlock];    // this block's keys of the bucket
  __shared__ long long s_k, s_krem;
  __shared__ unsigned long long s_bucket, s_base;
  __shared__ uint32_t s_n;
  ProtectCtl* ctl = ctl_of(a);
  const int tid = threadIdx.x;
  if (tid == 0) {
    long long k = (long long)floor(a.budget * (double)ctl->n_cand + 0.5) - (long long)ctl->n_base;
    if (k < 0) k = 0;
    if (k > (long long)ctl->n_elig) k = (long long)ctl->n_elig;
    s_k = k;
    if (blockIdx.x == 0) ctl->k = k;
  }
  __syncthreads();
  const long long k = s_k;
  if (k == 0) return;
  // thread t owns bins [kBins-BPT(t+1), kBins-BPT t), taken in descending order
  const uint32_t* g_hist = (const uint32_t*)(a.ws + a.off_hist);
  uint32_t h[BPT];
  unsigned long long mine = 0;
#pragma unroll
  for (int j = 0; j < BPT; ++j) {
    h[j] = g_hist[kBins - 1 - BPT * tid - j];
    mine += h[j];
  }
  const unsigned long long incl = block_scan<256>(mine, sh);
  const long long excl = (long long)(incl - mine);
  if (excl < k && k <= (long long)incl) {   // exactly one thread
    long long cum = excl;
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      if (cum + (long long)h[j] >= k) {
        s_bucket = (unsigned long long)(kBins - 1 - BPT * tid - j);
        s_krem = k - cum;
        break;
      }
      cum += h[j];
    }
  }
  __syncthreads();
  const uint64_t bucket = s_bucket;
  if (blockIdx.x == 0 && tid == 0) {
    ctl->k_rem = s_krem;
    ctl->bucket = bucket;
  }
  // append the bucket's keys: staged in LDS, one device atomic per block and chunk
  const uint64_t* key = (const uint64_t*)(a.ws + a.off_key);
  const uint8_t* fl = (const uint8_t*)(a.ws + a.off_flag);
  uint64_t* list = (uint64_t*)(a.ws + a.off_list);
  for (int64_t c0 = (int64_t)blockIdx.x * kRowsPerBlock; c0 < a.n_rows; c0 += (int64_t)gridDim.x * kRowsPerBlock) {
    if (tid == 0) s_n = 0;
    __syncthreads();
    const int64_t r0 = c0 + tid * 8;
    uint64_t f8 = 0;
    if (r0 + 8 <= a.n_rows) {
      f8 = *(const uint64_t*)(fl + r0);
    } else {
      for (int64_t r = r0; r < a.n_rows; ++r) f8 |= (uint64_t)fl[r] << (8 * (r - r0));
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if ((f8 >> (8 * j)) & 4) {
        const uint64_t kk = key[r0 + j];
        if ((kk >> (64 - kBits1)) == bucket) buf[atomicAdd(&s_n, 1u)] = kk;
      }
    }
    __syncthreads();
    const uint32_t nb = s_n;
    if (tid == 0 && nb > 0) s_base = atomicAdd(&ctl->n_list, (unsigned long long)nb);
    __syncthreads();
    for (uint32_t i = tid; i < nb; i += 256) list[s_base + i] = buf[i];
    __syncthreads();
  }
}

__global__ __launch_bounds__(kSelectThreads) void protect_select_kernel(ProtectArgs a) {
  constexpr int NT = kSelectThreads;
  __shared__ uint32_t dh[NT / 64][256];      // per-wave digit histograms
  __shared__ long long s_krem;
  __shared__ unsigned long long s_pre;
  ProtectCtl* ctl = ctl_of(a);
  if (ctl->k == 0) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t M = (int64_t)ctl->n_list;
  const uint64_t* list = (const uint64_t*)(a.ws + a.off_list);
  if (tid == 0) {
    s_pre = ctl->bucket << (64 - kBits1);
    s_krem = ctl->k_rem;
  }
  for (int lo = 64 - kBits1; lo > 0;) {      // bits >= lo of kth are known
    const int w = lo >= 8 ? 8 : lo;
    const int shift = lo - w;
    for (int i = tid; i < (NT / 64) * 256; i += NT) (&dh[0][0])[i] = 0;
    __syncthreads();
    const uint64_t pre = s_pre;
    for (int64_t i = tid; i < M; i += NT) {
      const uint64_t kk = list[i];
      if ((kk >> lo) == (pre >> lo)) atomicAdd(&dh[wave][(kk >> shift) & ((1u << w) - 1u)], 1u);
    }
    __syncthreads();
    if (tid < 256) {
      uint32_t t = 0;
#pragma unroll
      for (int v = 0; v < NT / 64; ++v) t += dh[v][tid];
      dh[0][tid] = t;
    }
    __syncthreads();
    if (wave == 0) {
      // lane L holds digits 255-4L .. 252-4L (descending); scan across the lanes
      uint32_t c4[4], sum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c4[j] = dh[0][255 - 4 * lane - j];
        sum += c4[j];
      }
      uint32_t incl = sum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
      }
      const long long rem = s_krem;
      const long long excl = (long long)(incl - sum);
      if (excl < rem && rem <= (long long)incl) {   // exactly one lane
        long long cum = excl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (cum + (long long)c4[j] >= rem) {
            s_krem = rem - cum;
            s_pre = pre | ((uint64_t)(255 - 4 * lane - j) << shift);
            break;
          }
          cum += c4[j];
        }
      }
    }
    __syncthreads();
    lo = shift;
  }
  if (tid == 0) ctl->kth = s_pre;
}

// selection mask of the 8 rows r0 .. r0+7 (r0 a multiple of 8)
__device__ __forceinline__ uint32_t selected8(const ProtectArgs& a, int64_t r0, bool sel_top, uint64_t kth) {
  const uint64_t* key = (const uint64_t*)(a.ws + a.off_key);
  const uint8_t* fl = (const uint8_t*)(a.ws + a.off_flag);
  uint64_t f8 = 0;
  if (r0 + 8 <= a.n_rows) {
    f8 = *(const uint64_t*)(fl + r0);
  } else {
    for (int64_t r = r0; r < a.n_rows; ++r) f8 |= (uint64_t)fl[r] << (8 * (r - r0));
  }
  uint32_t m = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t f = (uint32_t)(f8 >> (8 * j)) & 0xFFu;
    const bool s = (f & 1) || (sel_top && (f & 4) && key[r0 + j] >= kth);
    m |= (s ? 1u : 0u) << j;
  }
  return m;
}

__global__ __launch_bounds__(256) void protect_count_kernel(ProtectArgs a) {
  __shared__ unsigned long long sh[256];
  const ProtectCtl* ctl = ctl_of(a);
  const uint32_t m = selected8(a, (int64_t)blockIdx.x * kRowsPerBlock + threadIdx.x * 8, ctl->k > 0, ctl->kth);
  const unsigned long long tot = block_scan<256>((unsigned long long)__popc(m), sh);
  if (threadIdx.x == 255) ((uint64_t*)(a.ws + a.off_bcnt))[blockIdx.x] = tot;
}

__global__ __launch_bounds__(256) void protect_scan_kernel(ProtectArgs a, int64_t n_blocks) {
  __shared__ unsigned long long sh[256];
  uint64_t* bcnt = (uint64_t*)(a.ws + a.off_bcnt);
  const int tid = threadIdx.x;
  // thread t turns a contiguous run of the block counts into exclusive offsets
  const int64_t per = (n_blocks + 255) / 256;
  const int64_t i0 = std::min<int64_t>(tid * per, n_blocks), i1 = std::min<int64_t>(i0 + per, n_blocks);
  unsigned long long run = 0;
  for (int64_t i = i0; i < i1; ++i) run += bcnt[i];
  const unsigned long long incl = block_scan<256>(run, sh);
  unsigned long long at = incl - run;
  for (int64_t i = i0; i < i1; ++i) {
    const unsigned long long v = bcnt[i];
    bcnt[i] = at;
    at += v;
  }
  if (tid == 255) *a.n_prot = (int32_t)incl;
}

__global__ __launch_bounds__(256) void protect_write_kernel(ProtectArgs a) {
  __shared__ unsigned long long sh[256];
  const ProtectCtl* ctl = ctl_of(a);
  const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock + threadIdx.x * 8;
  uint32_t m = selected8(a, r0, ctl->k > 0, ctl->kth);
  const uint32_t c = (uint32_t)__popc(m);
  const unsigned long long incl = block_scan<256>(c, sh);
  unsigned long long at = ((const uint64_t*)(a.ws + a.off_bcnt))[blockIdx.x] + incl - c;
  while (m) {
    const int j = __ffs(m) - 1;
    m &= m - 1;
    a.prot_rows[at++] = (int32_t)(r0 + j);
  }
}

}  // namespace

int64_t protect_count_blocks(int64_t n_rows) { return std::max<int64_t>(1, (n_rows + kRowsPerBlock - 1) / kRowsPerBlock); }

__global__ __launch_bounds__(256) void protect_zero_kernel(ProtectArgs a) {
  // the control words (kProtectCtlBytes) and the histogram (kProtectHistBytes), 4 bytes a thread
  uint32_t* ctl = (uint32_t*)(a.ws + a.off_ctl);
  uint32_t* hist = (uint32_t*)(a.ws + a.off_hist);
  for (int i = blockIdx.x * 256 + threadIdx.x; i < (int)(kProtectCtlBytes / 4); i += gridDim.x * 256) ctl[i] = 0u;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < (int)(kProtectHistBytes / 4); i += gridDim.x * 256) hist[i] = 0u;
}

hipError_t launch_protect(const ProtectArgs& a, hipStream_t s) {
  hipError_t e;
  const int64_t n = a.n_rows;
  if (a.zero_ctl) {
    protect_zero_kernel<<<dim3(16), dim3(256), 0, s>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int64_t nb = protect_count_blocks(n);
  const unsigned grid = (unsigned)std::min<int64_t>(nb, 1024);
  protect_classify_kernel<<<dim3(grid), dim3(256), 0, s>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  protect_gather_kernel<<<dim3(grid), dim3(256), 0, s>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  protect_select_kernel<<<dim3(1), dim3(kSelectThreads), 0, s>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  protect_count_kernel<<<dim3((unsigned)nb), dim3(256), 0, s>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  protect_scan_kernel<<<dim3(1), dim3(256), 0, s>>>(a, nb);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  protect_write_kernel<<<dim3((unsigned)nb), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace mla
