// Protected token-row set (Sec. 2.3, eq:protected):
//   A = Q u N u D u B_edge u I_top u T_tail
// Q query rows, N new rows, D dirty rows, B_edge the first and last rows of every
// relocated segment, T_tail the most recent rows in request order, and I_top the
// rows the Indexer ranks highest, which top the protected share of the candidate
// rows (rows that have an artifact: neither query nor new rows) up to the
// controller's budget.
//
// Two kernels on the caller's stream:
//   classify  (grid)  one thread per row: its segment (binary search in the
//                     storage-ordered table), the flags above, and for rows that
//                     I_top may take a 64-bit key: the score's IEEE-754
//                     totalOrder bits above the inverted row index, so keys are
//                     unique and the largest keys are the highest scores, equal
//                     scores going to the lower row.
//   select    (one    counts the candidates, derives k, finds the k-th largest
//             1024-   key by an 8-bit radix select over the key bits, then writes
//             thread  the selected rows in ascending order (per-thread runs and a
//             group)  block-wide prefix sum) and their count.
#include "common.h"

#include <algorithm>

namespace mla {

constexpr int kSelThreads = 1024;

__device__ __forceinline__ uint32_t total_order_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u >> 31) ? ~u : (u | 0x80000000u);
}

__global__ __launch_bounds__(256) void protect_classify_kernel(ProtectArgs a) {
  const int64_t* kv_start = (const int64_t*)(a.ws + a.off_kv);
  const int64_t* length = (const int64_t*)(a.ws + a.off_len);
  const int64_t* req = (const int64_t*)(a.ws + a.off_req);
  const int32_t* orig = (const int32_t*)(a.ws + a.off_orig);
  uint64_t* key = (uint64_t*)(a.ws + a.off_key);
  uint8_t* fl = (uint8_t*)(a.ws + a.off_flag);
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < a.n_rows;
       r += (int64_t)gridDim.x * blockDim.x) {
    int lo = 0, hi = a.n_segs - 1;   // last segment (storage order) with kv_start <= r
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (kv_start[mid] <= r) lo = mid; else hi = mid - 1;
    }
    const int64_t u = r - kv_start[lo];
    const int64_t pos = req[lo] + u;
    const uint8_t rf = a.row_flags ? a.row_flags[r] : (uint8_t)0;
    const bool q = orig[lo] == a.query_seg;
    const bool is_new = (rf & 1) != 0, dirty = (rf & 2) != 0;
    const bool relocated = req[lo] != 0 && !q;
    const bool edge = relocated && (u < a.edge_rows || u >= length[lo] - a.edge_rows);
    const bool recent = pos >= a.n_rows - a.tail_rows;
    const bool base = q || is_new || dirty || edge || recent;
    const bool cand = !q && !is_new;
    // bit 0: in the fixed sets; bit 1: candidate row; bit 2: eligible for I_top
    fl[r] = (uint8_t)((base ? 1 : 0) | (cand ? 2 : 0) | (cand && !base ? 4 : 0));
    const uint32_t sb = a.scores ? total_order_bits(a.scores[r]) : 0u;
    key[r] = ((uint64_t)sb << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)r);
  }
}

__global__ __launch_bounds__(kSelThreads) void protect_select_kernel(ProtectArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t scan[kSelThreads];
  __shared__ unsigned long long s_cnt[3];
  __shared__ unsigned long long s_prefix;
  __shared__ long long s_krem;
  const uint64_t* key = (const uint64_t*)(a.ws + a.off_key);
  const uint8_t* fl = (const uint8_t*)(a.ws + a.off_flag);
  const int tid = threadIdx.x;
  const int64_t n = a.n_rows;

  // counts: candidates, candidates in the fixed sets, rows eligible for I_top
  if (tid < 3) s_cnt[tid] = 0;
  __syncthreads();
  unsigned long long c_cand = 0, c_base = 0, c_elig = 0;
  for (int64_t r = tid; r < n; r += kSelThreads) {
    const uint8_t f = fl[r];
    c_cand += (f >> 1) & 1;
    c_base += ((f & 3) == 3) ? 1 : 0;
    c_elig += (f >> 2) & 1;
  }
  atomicAdd(&s_cnt[0], c_cand);
  atomicAdd(&s_cnt[1], c_base);
  atomicAdd(&s_cnt[2], c_elig);
  __syncthreads();
  if (tid == 0) {
    const long long target = (long long)floor(a.budget * (double)s_cnt[0] + 0.5);
    long long k = target - (long long)s_cnt[1];
    if (k < 0) k = 0;
    if (k > (long long)s_cnt[2]) k = (long long)s_cnt[2];
    s_krem = k;
    s_prefix = 0;
  }
  __syncthreads();
  const long long k = s_krem;

  // radix select of the k-th largest key among the eligible rows (keys are unique)
  if (k > 0) {
    for (int shift = 56; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += kSelThreads) hist[i] = 0;
      __syncthreads();
      const uint64_t pre = s_prefix;
      const int hs = shift + 8;   // bits at and above hs are fixed by earlier passes
      for (int64_t r = tid; r < n; r += kSelThreads) {
        if (!(fl[r] & 4)) continue;
        const uint64_t kk = key[r];
        if (hs < 64 && (kk >> hs) != (pre >> hs)) continue;
        atomicAdd(&hist[(kk >> shift) & 255], 1u);
      }
      __syncthreads();
      if (tid == 0) {
        long long rem = s_krem, cum = 0;
        int d = 255;
        for (; d > 0; --d) {
          if (cum + (long long)hist[d] >= rem) break;
          cum += hist[d];
        }
        s_krem = rem - cum;
        s_prefix = pre | ((uint64_t)d << shift);
      }
      __syncthreads();
    }
  }
  const uint64_t kth = s_prefix;   // the k-th largest eligible key (unused when k == 0)

  // ascending compaction: thread t owns rows [t*run, (t+1)*run)
  const int64_t run = (n + kSelThreads - 1) / kSelThreads;
  const int64_t r0 = (int64_t)tid * run, r1 = r0 + run < n ? r0 + run : n;
  auto selected = [&](int64_t r) -> bool {
    const uint8_t f = fl[r];
    return (f & 1) || (k > 0 && (f & 4) && key[r] >= kth);
  };
  uint32_t mine = 0;
  for (int64_t r = r0; r < r1; ++r) mine += selected(r) ? 1u : 0u;
  scan[tid] = mine;
  __syncthreads();
  for (int off = 1; off < kSelThreads; off <<= 1) {   // inclusive Hillis-Steele scan
    const uint32_t v = tid >= off ? scan[tid - off] : 0u;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  uint32_t at = scan[tid] - mine;
  for (int64_t r = r0; r < r1; ++r)
    if (selected(r)) a.prot_rows[at++] = (int32_t)r;
  if (tid == kSelThreads - 1) *a.n_prot = (int32_t)scan[tid];
}

hipError_t launch_protect(const ProtectArgs& a, hipStream_t s) {
  if (a.n_rows > 0) {
    const unsigned blocks = (unsigned)std::min<int64_t>((a.n_rows + 255) / 256, 16384);
    protect_classify_kernel<<<dim3(blocks), dim3(256), 0, s>>>(a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  protect_select_kernel<<<dim3(1), dim3(kSelThreads), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace mla
