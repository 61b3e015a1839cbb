// Device half of a device-built plan (Alg. 2: ProtectedRows feeding
// SelectiveMLA in the same layer without a trip through the host).
//
// The host fixes, once per request, everything that depends only on the segment
// table: segment visibility in request order, the chunking of each visible list,
// the Global partial index and the launch order of the item groups (one group
// per kind, segment and chunk, largest upper-bound cost first).  Per call, the
// protected rows A and |A| are read from device memory and two kernels finish
// the plan:
//   dplan_count_kernel (one workgroup)  validates A (ascending, in range, at most
//     the capacity the plan was built for), finds each segment's run of
//     protected rows by binary search (A is sorted and segments are contiguous
//     in storage), the Local partial base of each segment (a scan in storage
//     order), each group's item count and their prefix (a scan in launch order),
//     and the call's counts;
//   dplan_items_kernel (one thread per item bound)  writes each work item: its
//     group by binary search in the prefix, then its head-row range.  Inside a
//     group items run from the segment's last head-rows down, so that the
//     costliest items of the group start first.
// A rejected A leaves zero items, zero slots and status MLA_ERR_ROWS: the
// attention kernels then do nothing.
#include "common.h"

namespace mla {

constexpr int kPlanThreads = 1024;

// exclusive prefix of v over the workgroup's threads (in thread order); *total
// receives the sum.  Every thread of the workgroup calls it.
__device__ int64_t block_exclusive_scan(int64_t v, int64_t* total) {
  __shared__ int64_t wsum[kPlanThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int64_t before = 0, all = 0;
  for (int i = 0; i < kPlanThreads / 64; ++i) {
    before += i < w ? wsum[i] : 0;
    all += wsum[i];
  }
  __syncthreads();   // wsum may be rewritten by the next call
  *total = all;
  return before + x - v;
}

// first index in prot[0, n) whose value is >= r
__device__ __forceinline__ int lower_bound_i32(const int32_t* prot, int n, int64_t r) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)prot[mid] < r) lo = mid + 1; else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(kPlanThreads) void dplan_count_kernel(DPlanArgs a) {
  __shared__ int s_ok;
  __shared__ int s_np;
  const int tid = threadIdx.x;
  if (tid == 0) {
    const int np = *a.n_prot_dev;
    s_np = np;
    s_ok = (np >= 0 && np <= a.prot_cap) ? 1 : 0;
  }
  __syncthreads();
  const int np = s_ok ? s_np : 0;
  // validation: rows in range and strictly increasing
  int bad = 0;
  for (int i = tid; i < np; i += kPlanThreads) {
    const int32_t r = a.prot[i];
    if (r < 0 || (int64_t)r >= a.n_rows || (i > 0 && a.prot[i - 1] >= r)) bad = 1;
  }
  if (__syncthreads_or(bad) || !s_ok) {
    if (tid == 0) {
      a.dyn->n_slots = 0;
      a.dyn->n_parts = 0;
      a.dyn->n_items = 0;
      a.dyn->n_prot = 0;
      a.dyn->status = MLA_ERR_ROWS;
      if (a.status_out != nullptr) *a.status_out = MLA_ERR_ROWS;
    }
    return;
  }
  // each segment's run of protected rows, and its Local partial base in storage order
  int64_t carry = 0;
  for (int base = 0; base < a.n_segs; base += kPlanThreads) {
    const int i = base + tid;
    int64_t parts = 0;
    if (i < a.n_segs) {
      const int s = a.storage[i];
      const SegInfo si = a.segs[s];
      const int lo = lower_bound_i32(a.prot, np, si.kv_start);
      const int hi = lower_bound_i32(a.prot, np, si.kv_start + si.length);
      a.seg_prot_lo[s] = lo;
      a.seg_prot_cnt[s] = hi - lo;
      parts = (int64_t)(hi - lo) * a.n_local * si.n_chunks;
    }
    int64_t total;
    const int64_t ex = block_exclusive_scan(parts, &total);
    if (i < a.n_segs) a.seg_local_base[a.storage[i]] = carry + ex;
    carry += total;
  }
  const int64_t local_parts = carry;
  __syncthreads();   // seg_prot_cnt of every segment is written
  // item counts of the groups in launch order, and their prefix
  int64_t items = 0;
  for (int base = 0; base < a.n_item_groups; base += kPlanThreads) {
    const int i = base + tid;
    int64_t cnt = 0;
    if (i < a.n_item_groups) {
      const ItemGroup g = a.groups[i];
      cnt = g.kind == 0 ? g.n_items
                        : ((int64_t)a.seg_prot_cnt[g.seg] * a.n_local + kTileRows - 1) / kTileRows;
    }
    int64_t total;
    const int64_t ex = block_exclusive_scan(cnt, &total);
    if (i < a.n_item_groups) a.group_base[i] = (int32_t)(items + ex);
    items += total;
  }
  if (tid == 0) {
    // the host's bounds hold for every list of at most prot_cap rows; should one
    // not hold, nothing runs rather than anything being written out of range
    const bool fits = items <= a.max_items && a.global_parts + local_parts <= a.max_parts;
    a.group_base[a.n_item_groups] = (int32_t)items;
    a.dyn->n_slots = fits ? a.n_rows * a.n_groups + (int64_t)np * a.n_local : 0;
    a.dyn->n_parts = fits ? a.global_parts + local_parts : 0;
    a.dyn->n_items = fits ? (int32_t)items : 0;
    a.dyn->n_prot = fits ? np : 0;
    a.dyn->status = fits ? MLA_OK : MLA_ERR_WORKSPACE;
    if (a.status_out != nullptr) *a.status_out = a.dyn->status;
  }
}

__global__ __launch_bounds__(256) void dplan_items_kernel(DPlanArgs a) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= a.dyn->n_items) return;
  // the group holding item i: the last g with group_base[g] <= i
  int lo = 0, hi = a.n_item_groups - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.group_base[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const ItemGroup g = a.groups[lo];
  const int k = i - a.group_base[lo];
  const SegInfo si = a.segs[g.seg];
  int64_t h0, h1;   // head-row range of the group
  if (g.kind == 0) {
    h0 = si.kv_start * a.n_groups;
    h1 = (si.kv_start + si.length) * a.n_groups;
  } else {
    h0 = (int64_t)a.seg_prot_lo[g.seg] * a.n_local;
    h1 = h0 + (int64_t)a.seg_prot_cnt[g.seg] * a.n_local;
  }
  const int64_t end = h1 - (int64_t)k * kTileRows;
  const int64_t begin = end - kTileRows > h0 ? end - kTileRows : h0;
  const int64_t last_row = g.kind == 0 ? (end - 1) / a.n_groups : (int64_t)a.prot[(end - 1) / a.n_local];
  WorkItem w;
  w.hr_begin = begin;
  w.count = (int32_t)(end - begin);
  w.kind = g.kind;
  w.seg = g.seg;
  w.chunk = g.chunk;
  w.max_u = (int32_t)(last_row - si.kv_start);
  w.pad = 0;
  a.items[i] = w;
}

hipError_t launch_dplan(const DPlanArgs& a, hipStream_t s) {
  dplan_count_kernel<<<dim3(1), dim3(kPlanThreads), 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.max_items == 0) return e;
  dplan_items_kernel<<<dim3((unsigned)((a.max_items + 255) / 256)), dim3(256), 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace mla
