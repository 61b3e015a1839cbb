// Host side of the MLA-Online C ABI: argument validation, the plan (segment
// visibility in request order, chunking of each row's visible-segment list,
// the partial index and the longest-first work list), and kernel dispatch.
#include <algorithm>
#include <cstdarg>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <numeric>
#include <string>
#include <vector>

#include "common.h"
#include "mla_probe.h"
#include "moe.h"
#include "oproj.h"
#include "probe.h"
#include "protect.h"
#include "wb.h"

// Device scratch of mla_online_attend_planned_noalloc (one copy per GPU, for the
// life of the process); host code reaches it only through scratch_address().
static __device__ __align__(256) unsigned char scratch[MLA_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_detail;

mla_status fail(mla_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
mla_status fail(mla_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_detail = buf;
  return s;
}

mla_status hip_fail(hipError_t e, const char* what) {
  return fail(MLA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------------------
// validation
// ---------------------------------------------------------------------------
// width of one head output: the latent, plus the RoPE dims when the value is rotary
int32_t head_dv(const mla_geom* g) { return g->d_latent + (g->value_rope ? g->d_rope : 0); }

mla_status check_geom(const mla_geom* g, bool for_oproj) {
  if (g == nullptr) return fail(MLA_ERR_NULL, "geom is NULL");
  if (g->n_heads < 1 || g->n_groups < 1 || g->n_heads % g->n_groups != 0)
    return fail(MLA_ERR_SHAPE, "n_heads (%d) must be a positive multiple of n_groups (%d)", g->n_heads,
                g->n_groups);
  if (g->n_groups > mla::kMaxGroups)
    return fail(MLA_ERR_UNSUPPORTED, "n_groups %d exceeds %d", g->n_groups, mla::kMaxGroups);
  if (!((g->d_latent == 512 && g->d_rope == 64) || (g->d_latent == 64 && g->d_rope == 16)))
    return fail(MLA_ERR_UNSUPPORTED, "(d_latent, d_rope) = (%d, %d); built: (512, 64), (64, 16)", g->d_latent,
                g->d_rope);
  if (!(g->softmax_scale > 0.f) || !std::isfinite(g->softmax_scale))
    return fail(MLA_ERR_SHAPE, "softmax_scale must be finite and > 0");
  if (!(g->rope_base > 1.0) || !std::isfinite(g->rope_base))
    return fail(MLA_ERR_SHAPE, "rope_base must be finite and > 1");
  if (g->value_rope != 0 && g->value_rope != 1) return fail(MLA_ERR_SHAPE, "value_rope = %d", g->value_rope);
  if (g->value_rope && !(g->d_latent == 512 && g->d_rope == 64))
    return fail(MLA_ERR_UNSUPPORTED, "a rotary value is built for (d_latent, d_rope) = (512, 64)");
  if (for_oproj) {
    if (g->d_model < 1 || g->n_proj_groups < 1 || g->n_groups % g->n_proj_groups != 0 ||
        g->d_model % g->n_proj_groups != 0)
      return fail(MLA_ERR_SHAPE, "n_proj_groups (%d) must divide n_groups (%d) and d_model (%d)",
                  g->n_proj_groups, g->n_groups, g->d_model);
    if ((g->d_model / g->n_proj_groups) % 32 != 0)
      return fail(MLA_ERR_UNSUPPORTED, "d_model / n_proj_groups = %d is not a multiple of 32",
                  g->d_model / g->n_proj_groups);
  }
  return MLA_OK;
}

// Segments: lengths >= 1; storage and request intervals both tile [0, N).
mla_status check_segments(const mla_segment* segs, int32_t n, int64_t* n_rows) {
  if (segs == nullptr) return fail(MLA_ERR_NULL, "segs is NULL");
  if (n < 1) return fail(MLA_ERR_SEGMENTS, "n_segs = %d, need at least one segment", n);
  int64_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (segs[i].length < 1) return fail(MLA_ERR_SEGMENTS, "segment %d has length %lld", i, (long long)segs[i].length);
    if (segs[i].kv_start < 0 || segs[i].req_offset < 0)
      return fail(MLA_ERR_SEGMENTS, "segment %d has a negative start", i);
    if (segs[i].length > INT32_MAX - total) return fail(MLA_ERR_UNSUPPORTED, "more than 2^31-1 rows");
    total += segs[i].length;
  }
  for (int pass = 0; pass < 2; ++pass) {
    std::vector<int32_t> idx(n);
    std::iota(idx.begin(), idx.end(), 0);
    auto key = [&](int32_t i) { return pass == 0 ? segs[i].kv_start : segs[i].req_offset; };
    std::sort(idx.begin(), idx.end(), [&](int32_t x, int32_t y) { return key(x) < key(y); });
    int64_t at = 0;
    for (int32_t i : idx) {
      if (key(i) != at)
        return fail(MLA_ERR_SEGMENTS, "segments do not tile [0, %lld) in %s space at %lld (segment %d)",
                    (long long)total, pass == 0 ? "storage" : "request", (long long)at, i);
      at += segs[i].length;
    }
  }
  *n_rows = total;
  return MLA_OK;
}

mla_status check_prot(const int32_t* prot, int32_t n_prot, int64_t n_rows) {
  if (n_prot < 0) return fail(MLA_ERR_ROWS, "n_prot = %d", n_prot);
  if (n_prot > 0 && prot == nullptr) return fail(MLA_ERR_NULL, "prot_rows is NULL");
  if (n_prot > n_rows) return fail(MLA_ERR_ROWS, "n_prot %d exceeds n_rows %lld", n_prot, (long long)n_rows);
  for (int32_t a = 0; a < n_prot; ++a) {
    if (prot[a] < 0 || prot[a] >= n_rows) return fail(MLA_ERR_ROWS, "prot_rows[%d] = %d out of range", a, prot[a]);
    if (a > 0 && prot[a] <= prot[a - 1])
      return fail(MLA_ERR_ROWS, "prot_rows not strictly increasing at %d", a);
  }
  return MLA_OK;
}

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------
struct Plan {
  mla::PlanHeader hdr{};
  std::vector<unsigned char> blob;   // exact workspace image
};

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// rotary value: bytes of the attention kernel's accumulators, 128 f32 per
// head-row of each of n_items work items
int64_t rot_bytes(int64_t n_items) { return std::max<int64_t>(n_items, 1) * mla::kTileRows * 128 * 4; }

// What depends only on the segment table: request order, storage order, the
// chunking of each segment's visible list (ranks 0 .. rank(s)) and the Global
// partial index.  offline: every segment sees only itself (Alg. 1).
struct SegTables {
  std::vector<int32_t> rank_seg, storage, rank_of;
  std::vector<mla::SegInfo> info;
  std::vector<mla::ChunkInfo> chunks;
  int64_t global_parts = 0;
};

void segment_tables(const mla_geom* g, const mla_segment* segs, int32_t n_segs, int64_t split_keys, bool offline,
                    SegTables* T) {
  const int G = g->n_groups;
  T->rank_seg.resize(n_segs);
  T->storage.resize(n_segs);
  T->rank_of.resize(n_segs);
  std::iota(T->rank_seg.begin(), T->rank_seg.end(), 0);
  std::sort(T->rank_seg.begin(), T->rank_seg.end(),
            [&](int32_t x, int32_t y) { return segs[x].req_offset < segs[y].req_offset; });
  for (int32_t r = 0; r < n_segs; ++r) T->rank_of[T->rank_seg[r]] = r;
  std::iota(T->storage.begin(), T->storage.end(), 0);
  std::sort(T->storage.begin(), T->storage.end(),
            [&](int32_t x, int32_t y) { return segs[x].kv_start < segs[y].kv_start; });
  T->info.assign(n_segs, mla::SegInfo{});
  T->chunks.clear();
  for (int32_t s = 0; s < n_segs; ++s) {
    mla::SegInfo& in = T->info[s];
    in.kv_start = segs[s].kv_start;
    in.length = segs[s].length;
    in.req_offset = segs[s].req_offset;
    in.rank = T->rank_of[s];
    in.chunk_off = (int32_t)T->chunks.size();
    if (offline) {
      T->chunks.push_back({T->rank_of[s], T->rank_of[s]});
      in.n_chunks = 1;
      continue;
    }
    int32_t first = 0;
    int64_t keys = 0;
    for (int32_t r = 0; r <= T->rank_of[s]; ++r) {
      const int64_t len = segs[T->rank_seg[r]].length;
      const bool close = split_keys == 0 ? (r > first) : (r > first && keys + len > split_keys);
      if (close) {
        T->chunks.push_back({first, r - 1});
        first = r;
        keys = 0;
      }
      keys += len;
    }
    T->chunks.push_back({first, T->rank_of[s]});
    in.n_chunks = (int32_t)T->chunks.size() - in.chunk_off;
  }
  // partial counts: global slots in storage order (none offline)
  int64_t cum = 0;
  for (int32_t i : T->storage) {
    T->info[i].cum_global = cum;
    if (!offline) cum += (int64_t)G * T->info[i].length * T->info[i].n_chunks;
  }
  T->global_parts = cum;
}

// RoPE frequencies in revolutions: base^(-2j/d_r) / (2 pi)
void rope_theta_rev(const mla_geom* g, double* th) {
  const double two_pi = 6.283185307179586476925286766559;
  for (int j = 0; j < g->d_rope / 2; ++j) th[j] = std::pow(g->rope_base, -2.0 * j / g->d_rope) / two_pi;
}

// offline: the producer's plan (Alg. 1) -- every segment sees only itself, and
// only Local heads run (every row is listed in prot, no Global slots exist).
mla_status build_plan(const mla_geom* g, const mla_segment* segs, int32_t n_segs, const int32_t* prot,
                      int32_t n_prot, int64_t split_keys, bool want_blob, Plan* out, bool offline = false) {
  mla_status st = check_geom(g, false);
  if (st != MLA_OK) return st;
  int64_t N = 0;
  if ((st = check_segments(segs, n_segs, &N)) != MLA_OK) return st;
  if ((st = check_prot(prot, n_prot, N)) != MLA_OK) return st;
  if (split_keys < 0) return fail(MLA_ERR_SHAPE, "split_keys = %lld must be >= 0", (long long)split_keys);

  const int G = g->n_groups, hpg = g->n_heads / g->n_groups;
  const int64_t Lh = (int64_t)G * (hpg - 1);
  SegTables T;
  segment_tables(g, segs, n_segs, split_keys, offline, &T);
  const std::vector<int32_t>& rank_seg = T.rank_seg;
  const std::vector<int32_t>& storage = T.storage;
  std::vector<mla::SegInfo>& info = T.info;
  const std::vector<mla::ChunkInfo>& chunks = T.chunks;
  const int64_t global_parts = T.global_parts;
  std::vector<int32_t> prot_seg(n_prot);
  std::vector<int64_t> cum_local(n_prot + 1, 0);
  {
    int32_t si = 0;
    for (int32_t a = 0; a < n_prot; ++a) {
      while (segs[storage[si]].kv_start + segs[storage[si]].length <= prot[a]) ++si;
      prot_seg[a] = storage[si];
      cum_local[a + 1] = cum_local[a] + Lh * info[storage[si]].n_chunks;
    }
  }
  const int64_t n_slots = (offline ? 0 : N * G) + (int64_t)n_prot * Lh;
  const int64_t n_parts = global_parts + cum_local[n_prot];

  // work items: per segment, its rows' head-rows in runs of kTileRows, times its chunks
  struct Cand {
    mla::WorkItem w;
    int64_t cost;
  };
  std::vector<Cand> items;
  auto add_items = [&](int kind, int32_t s, int64_t hr_lo, int64_t hr_hi, auto row_of) {
    for (int64_t h = hr_lo; h < hr_hi; h += mla::kTileRows) {
      const int64_t cnt = std::min<int64_t>(mla::kTileRows, hr_hi - h);
      const int64_t max_u = row_of(h + cnt - 1) - segs[s].kv_start;
      for (int32_t c = 0; c < info[s].n_chunks; ++c) {
        const mla::ChunkInfo ch = chunks[info[s].chunk_off + c];
        int64_t tiles = 0;
        for (int32_t r = ch.first_rank; r <= ch.last_rank; ++r) {
          const int32_t t = rank_seg[r];
          const int64_t keys = t == s ? max_u + 1 : segs[t].length;
          tiles += (keys + 63) / 64;
        }
        Cand cd;
        cd.w.hr_begin = h;
        cd.w.count = (int32_t)cnt;
        cd.w.kind = kind;
        cd.w.seg = s;
        cd.w.chunk = c;
        cd.w.max_u = (int32_t)max_u;
        cd.w.pad = 0;
        cd.cost = tiles * ((cnt + 31) / 32);
        items.push_back(cd);
      }
    }
  };
  if (!offline)
    for (int32_t s = 0; s < n_segs; ++s)
      add_items(0, s, segs[s].kv_start * G, (segs[s].kv_start + segs[s].length) * G,
                [&](int64_t hr) { return hr / G; });
  if (Lh > 0) {
    int32_t a = 0;
    while (a < n_prot) {
      const int32_t s = prot_seg[a];
      int32_t b = a;
      while (b < n_prot && prot_seg[b] == s) ++b;
      add_items(1, s, a * Lh, (int64_t)b * Lh, [&](int64_t hr) { return (int64_t)prot[hr / Lh]; });
      a = b;
    }
  }
  // longest first; ties in a fixed order
  std::stable_sort(items.begin(), items.end(), [](const Cand& x, const Cand& y) { return x.cost > y.cost; });
  if (items.size() > (size_t)INT32_MAX - 256) return fail(MLA_ERR_UNSUPPORTED, "too many work items");

  // layout of the workspace image
  mla::PlanHeader& h = out->hdr;
  h = mla::PlanHeader{};
  h.n_rows = N;
  h.n_slots = n_slots;
  h.n_parts = n_parts;
  h.global_parts = global_parts;
  h.n_segs = n_segs;
  h.n_items = (int32_t)items.size();
  h.n_prot = n_prot;
  size_t off = align_up(sizeof(mla::PlanHeader), 256);
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return (int64_t)o;
  };
  h.off_segs = take(sizeof(mla::SegInfo) * n_segs);
  h.off_rank = take(sizeof(int32_t) * n_segs);
  h.off_storage = take(sizeof(int32_t) * n_segs);
  h.off_chunks = take(sizeof(mla::ChunkInfo) * chunks.size());
  h.off_items = take(sizeof(mla::WorkItem) * items.size());
  h.off_prot = take(sizeof(int32_t) * std::max<int32_t>(n_prot, 1));
  h.off_prot_seg = take(sizeof(int32_t) * std::max<int32_t>(n_prot, 1));
  h.off_cum_local = take(sizeof(int64_t) * (n_prot + 1));
  h.off_theta = take(sizeof(double) * mla::kMaxRopePairs);
  h.total_bytes = (int64_t)off;
  // rotary value: the attention kernel's per-item accumulators, after the image
  h.off_rot = g->value_rope ? (int64_t)off : -1;
  h.ws_bytes = (int64_t)off + (g->value_rope ? rot_bytes((int64_t)items.size()) : 0);
  if (!want_blob) return MLA_OK;

  out->blob.assign(off, 0);
  unsigned char* B = out->blob.data();
  std::memcpy(B, &h, sizeof h);
  std::memcpy(B + h.off_segs, info.data(), sizeof(mla::SegInfo) * n_segs);
  std::memcpy(B + h.off_rank, rank_seg.data(), sizeof(int32_t) * n_segs);
  std::memcpy(B + h.off_storage, storage.data(), sizeof(int32_t) * n_segs);
  std::memcpy(B + h.off_chunks, chunks.data(), sizeof(mla::ChunkInfo) * chunks.size());
  mla::WorkItem* wi = reinterpret_cast<mla::WorkItem*>(B + h.off_items);
  for (size_t i = 0; i < items.size(); ++i) wi[i] = items[i].w;
  if (n_prot > 0) {
    std::memcpy(B + h.off_prot, prot, sizeof(int32_t) * n_prot);
    std::memcpy(B + h.off_prot_seg, prot_seg.data(), sizeof(int32_t) * n_prot);
  }
  std::memcpy(B + h.off_cum_local, cum_local.data(), sizeof(int64_t) * (n_prot + 1));
  rope_theta_rev(g, reinterpret_cast<double*>(B + h.off_theta));
  return MLA_OK;
}

// device pointers of a host plan's tables inside the workspace it was uploaded to
void host_plan_tables(mla::AttendArgs& a, const mla::PlanHeader& h, const unsigned char* ws) {
  a.segs = reinterpret_cast<const mla::SegInfo*>(ws + h.off_segs);
  a.rank_seg = reinterpret_cast<const int32_t*>(ws + h.off_rank);
  a.storage = reinterpret_cast<const int32_t*>(ws + h.off_storage);
  a.chunks = reinterpret_cast<const mla::ChunkInfo*>(ws + h.off_chunks);
  a.items = reinterpret_cast<const mla::WorkItem*>(ws + h.off_items);
  a.prot = reinterpret_cast<const int32_t*>(ws + h.off_prot);
  a.theta_rev = reinterpret_cast<const double*>(ws + h.off_theta);
  a.prot_seg = reinterpret_cast<const int32_t*>(ws + h.off_prot_seg);
  a.cum_local = reinterpret_cast<const int64_t*>(ws + h.off_cum_local);
  a.dyn = nullptr;
  a.n_rows = h.n_rows;
  a.n_slots = h.n_slots;
  a.n_parts = h.n_parts;
  a.global_parts = h.global_parts;
  a.n_items = h.n_items;
  a.n_prot = h.n_prot;
  a.n_segs = h.n_segs;
}

// ---------------------------------------------------------------------------
// pinned staging for the plan upload: two slots per device, each reused only
// after the copy that last read it has completed
// ---------------------------------------------------------------------------
struct Staging {
  void* host[2] = {nullptr, nullptr};
  size_t cap[2] = {0, 0};
  hipEvent_t done[2] = {nullptr, nullptr};
  int next = 0;
};
std::mutex g_stage_mu;
std::map<int, Staging> g_stage;

mla_status upload_plan(const Plan& plan, void* ws, hipStream_t stream) {
  // a captured copy would replay from a staging slot that later calls rewrite
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cap);
  if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
  if (cap != hipStreamCaptureStatusNone)
    return fail(MLA_ERR_UNSUPPORTED, "the stream is capturing a graph; this call uploads its plan from a "
                "reused host staging buffer, so it runs outside capture only");
  int dev = 0;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lk(g_stage_mu);
  Staging& st = g_stage[dev];
  const int k = st.next;
  st.next ^= 1;
  if (st.done[k] == nullptr) {
    if ((e = hipEventCreateWithFlags(&st.done[k], hipEventDisableTiming)) != hipSuccess)
      return hip_fail(e, "hipEventCreateWithFlags");
  } else if ((e = hipEventSynchronize(st.done[k])) != hipSuccess) {
    return hip_fail(e, "hipEventSynchronize (staging)");
  }
  const size_t bytes = plan.blob.size();
  if (st.cap[k] < bytes) {
    if (st.host[k] != nullptr) (void)hipHostFree(st.host[k]);
    st.host[k] = nullptr;
    st.cap[k] = 0;
    const size_t cap = std::max<size_t>(bytes, 1 << 20);
    if ((e = hipHostMalloc(&st.host[k], cap, hipHostMallocDefault)) != hipSuccess)
      return hip_fail(e, "hipHostMalloc (plan staging)");
    st.cap[k] = cap;
  }
  std::memcpy(st.host[k], plan.blob.data(), bytes);
  if ((e = hipMemcpyAsync(ws, st.host[k], bytes, hipMemcpyHostToDevice, stream)) != hipSuccess)
    return hip_fail(e, "hipMemcpyAsync (plan upload)");
  if ((e = hipEventRecord(st.done[k], stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  return MLA_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* mla_status_str(mla_status s) {
  switch (s) {
    case MLA_OK: return "MLA_OK";
    case MLA_ERR_NULL: return "MLA_ERR_NULL: a required pointer is NULL";
    case MLA_ERR_SHAPE: return "MLA_ERR_SHAPE: inconsistent sizes, alignment or geometry";
    case MLA_ERR_UNSUPPORTED: return "MLA_ERR_UNSUPPORTED: configuration not built";
    case MLA_ERR_SEGMENTS: return "MLA_ERR_SEGMENTS: segment table does not tile the rows";
    case MLA_ERR_ROWS: return "MLA_ERR_ROWS: protected rows unsorted, duplicated or out of range";
    case MLA_ERR_WORKSPACE: return "MLA_ERR_WORKSPACE: workspace too small";
    case MLA_ERR_HIP: return "MLA_ERR_HIP: HIP runtime error";
  }
  return "unknown mla_status";
}

const char* mla_last_error_detail(void) { return g_detail.c_str(); }

const char* mla_version(void) { return "mla_online 0.1 (gfx950)"; }

mla_status mla_online_attend_query(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                                   const int32_t* prot_rows, int32_t n_prot, int64_t split_keys,
                                   int64_t* n_slots, int64_t* n_parts, size_t* ws_bytes) {
  g_detail.clear();
  if (n_slots == nullptr || n_parts == nullptr || ws_bytes == nullptr)
    return fail(MLA_ERR_NULL, "output pointer is NULL");
  Plan p;
  const mla_status st = build_plan(geom, segs, n_segs, prot_rows, n_prot, split_keys, false, &p);
  if (st != MLA_OK) return st;
  *n_slots = p.hdr.n_slots;
  *n_parts = p.hdr.n_parts;
  *ws_bytes = (size_t)p.hdr.ws_bytes;
  return MLA_OK;
}

mla_status mla_online_attend(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                             const int32_t* prot_rows, int32_t n_prot, int64_t split_keys, const void* kv,
                             const void* q_glob, const void* q_loc, float* part_o, float* part_lse,
                             int64_t* part_ptr, int32_t* part_seg, uint8_t* row_src, void* workspace,
                             size_t ws_bytes, void* stream) {
  g_detail.clear();
  Plan p;
  mla_status st = build_plan(geom, segs, n_segs, prot_rows, n_prot, split_keys, true, &p);
  if (st != MLA_OK) return st;
  const int hpg = geom->n_heads / geom->n_groups;
  if (kv == nullptr || q_glob == nullptr || part_o == nullptr || part_lse == nullptr || part_ptr == nullptr ||
      workspace == nullptr)
    return fail(MLA_ERR_NULL, "kv, q_glob, part_o, part_lse, part_ptr and workspace are required");
  if (n_prot > 0 && hpg > 1 && q_loc == nullptr) return fail(MLA_ERR_NULL, "q_loc is NULL but Local heads exist");
  if (!aligned16(kv) || !aligned16(q_glob) || (q_loc && !aligned16(q_loc)) || !aligned16(part_o))
    return fail(MLA_ERR_SHAPE, "kv, q_glob, q_loc and part_o must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return fail(MLA_ERR_SHAPE, "workspace must be 256-byte aligned");
  if (ws_bytes < (size_t)p.hdr.ws_bytes)
    return fail(MLA_ERR_WORKSPACE, "workspace %zu bytes < required %lld", ws_bytes, (long long)p.hdr.ws_bytes);

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if ((st = upload_plan(p, workspace, s)) != MLA_OK) return st;

  mla::AttendArgs a{};
  a.kv = kv;
  a.q_glob = q_glob;
  a.q_loc = q_loc;
  a.part_o = part_o;
  a.part_lse = part_lse;
  a.part_ptr = part_ptr;
  a.part_seg = part_seg;
  a.row_src = row_src;
  host_plan_tables(a, p.hdr, reinterpret_cast<const unsigned char*>(workspace));
  a.n_groups = geom->n_groups;
  a.n_local = geom->n_groups * (hpg - 1);
  a.d_latent = geom->d_latent;
  a.d_rope = geom->d_rope;
  a.dv = head_dv(geom);
  a.scale_log2 = geom->softmax_scale * 1.4426950408889634f;
  a.local_slot_base = p.hdr.n_rows * geom->n_groups;
  a.out_direct = nullptr;
  a.rot = p.hdr.off_rot >= 0 ? reinterpret_cast<float*>(reinterpret_cast<unsigned char*>(workspace) + p.hdr.off_rot)
                             : nullptr;
  hipError_t e = mla::launch_plan(a, s);
  if (e != hipSuccess) return hip_fail(e, "plan kernels");
  e = mla::launch_attend(a, s);
  if (e != hipSuccess) return hip_fail(e, "attention kernel");
  return MLA_OK;
}

mla_status mla_segment_merge(int64_t n_slots, int32_t d_latent, const float* part_o, const float* part_lse,
                             const int64_t* part_ptr, int32_t out_dtype, void* out_o, float* out_lse,
                             void* stream) {
  g_detail.clear();
  if (n_slots < 0) return fail(MLA_ERR_SHAPE, "n_slots = %lld", (long long)n_slots);
  if (d_latent != 512 && d_latent != 64 && d_latent != 576)
    return fail(MLA_ERR_UNSUPPORTED, "head output width %d; built: 64, 512, 576", d_latent);
  if (out_dtype != MLA_BF16 && out_dtype != MLA_F32) return fail(MLA_ERR_SHAPE, "out_dtype %d", out_dtype);
  if (n_slots == 0) return MLA_OK;
  if (part_o == nullptr || part_lse == nullptr || part_ptr == nullptr || out_o == nullptr)
    return fail(MLA_ERR_NULL, "part_o, part_lse, part_ptr and out_o are required");
  if (!aligned16(part_o) || !aligned16(out_o)) return fail(MLA_ERR_SHAPE, "part_o and out_o must be 16-byte aligned");
  hipError_t e = mla::launch_merge(n_slots, d_latent, part_o, part_lse, part_ptr, out_dtype, out_o, out_lse,
                                   reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "merge kernel");
  return MLA_OK;
}

mla_status mla_sliced_oproj_add(const mla_geom* geom, int64_t n_rows, const void* o_glob, const void* o_loc,
                                const int32_t* glob_head, const int32_t* prot_rows, int32_t n_prot,
                                const void* w_o, const void* z_off, float* z, void* stream) {
  g_detail.clear();
  mla_status st = check_geom(geom, true);
  if (st != MLA_OK) return st;
  if (n_rows < 1 || n_rows > INT32_MAX) return fail(MLA_ERR_SHAPE, "n_rows = %lld", (long long)n_rows);
  if (n_prot < 0 || n_prot > n_rows) return fail(MLA_ERR_ROWS, "n_prot = %d with n_rows = %lld", n_prot, (long long)n_rows);
  const int hpg = geom->n_heads / geom->n_groups;
  if (glob_head == nullptr) return fail(MLA_ERR_NULL, "glob_head is NULL");
  for (int g = 0; g < geom->n_groups; ++g)
    if (glob_head[g] < 0 || glob_head[g] >= hpg)
      return fail(MLA_ERR_SHAPE, "glob_head[%d] = %d outside [0, %d)", g, glob_head[g], hpg);
  if (o_glob == nullptr || w_o == nullptr || z == nullptr) return fail(MLA_ERR_NULL, "o_glob, w_o and z are required");
  if (n_prot > 0 && prot_rows == nullptr) return fail(MLA_ERR_NULL, "prot_rows is NULL");
  if (n_prot > 0 && hpg > 1 && o_loc == nullptr) return fail(MLA_ERR_NULL, "o_loc is NULL but Local heads exist");
  if (n_prot < n_rows && z_off == nullptr) return fail(MLA_ERR_NULL, "z_off is NULL but unprotected rows exist");
  if (!aligned16(o_glob) || (o_loc && !aligned16(o_loc)) || !aligned16(w_o) || !aligned16(z) ||
      (z_off && !aligned16(z_off)))
    return fail(MLA_ERR_SHAPE, "o_glob, o_loc, w_o, z_off and z must be 16-byte aligned");
  if (mla::oproj_workgroups(n_rows, geom->d_model, geom->n_proj_groups) > INT32_MAX)
    return fail(MLA_ERR_UNSUPPORTED, "%lld rows x d_model %d is more o-proj tiles than one launch takes",
                (long long)n_rows, geom->d_model);
  mla::OprojArgs a{};
  a.o_glob = o_glob;
  a.o_loc = o_loc;
  a.prot_rows = prot_rows;
  a.w_o = w_o;
  a.z_off = z_off;
  a.z = z;
  a.n_rows = n_rows;
  a.n_prot = n_prot;
  a.n_heads = geom->n_heads;
  a.n_groups = geom->n_groups;
  a.d_latent = head_dv(geom);
  a.d_model = geom->d_model;
  a.n_pg = geom->n_proj_groups;
  for (int g = 0; g < geom->n_groups; ++g) a.glob_head[g] = glob_head[g];
  a.z_bf16 = 0;
  hipError_t e = mla::launch_oproj(a, 3, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "o-proj kernels");
  return MLA_OK;
}

// ---------------------------------------------------------------------------
// plan once per request; attend and project with the protected set on the device
// ---------------------------------------------------------------------------
namespace {

// indices into mla_plan_info::layout: byte offsets in the plan image (P_*) and
// in the workspace (W_*), and two counts
enum {
  P_SEGS, P_RANK, P_STORAGE, P_CHUNKS, P_THETA, P_GROUPS, N_ITEM_GROUPS, GLOBAL_PARTS,
  W_DYN, W_SEG_LO, W_SEG_CNT, W_SEG_BASE, W_GROUP_BASE, W_ITEMS, W_PART_PTR, W_PART_O, W_PART_LSE, W_ROT,
  P_TKV, P_TLEN, P_TREQ, P_TORIG,   // the segment table in storage order, for the protected set
  LAYOUT_USED
};
static_assert(LAYOUT_USED <= 24, "mla_plan_info::layout holds 24 entries");

uint64_t mix(uint64_t h, uint64_t v) {
  for (int i = 0; i < 8; ++i) {   // FNV-1a over the little-endian bytes of v
    h ^= (v >> (8 * i)) & 0xffu;
    h *= 1099511628211ull;
  }
  return h;
}

uint64_t info_checksum(const mla_plan_info* p) {
  uint64_t h = 1469598103934665603ull;
  const mla_geom& g = p->geom;
  const int64_t gv[] = {g.n_heads, g.n_groups, g.d_latent, g.d_rope, g.d_model, g.n_proj_groups, g.value_rope};
  for (int64_t v : gv) h = mix(h, (uint64_t)v);
  uint32_t sc;
  std::memcpy(&sc, &g.softmax_scale, 4);
  uint64_t rb;
  std::memcpy(&rb, &g.rope_base, 8);
  h = mix(mix(h, sc), rb);
  const int64_t v[] = {p->n_rows, p->split_keys, p->max_slots, p->max_parts, p->n_segs, p->prot_cap,
                       p->max_items, p->one_chunk, (int64_t)p->plan_bytes, (int64_t)p->ws_bytes};
  for (int64_t x : v) h = mix(h, (uint64_t)x);
  for (int i = 0; i < 24; ++i) h = mix(h, (uint64_t)p->layout[i]);
  return h;
}

bool same_geom(const mla_geom& a, const mla_geom& b) {
  return a.n_heads == b.n_heads && a.n_groups == b.n_groups && a.d_latent == b.d_latent && a.d_rope == b.d_rope &&
         a.d_model == b.d_model && a.n_proj_groups == b.n_proj_groups && a.value_rope == b.value_rope &&
         std::memcmp(&a.softmax_scale, &b.softmax_scale, 4) == 0 && std::memcmp(&a.rope_base, &b.rope_base, 8) == 0;
}

struct StaticPlan {
  SegTables T;
  std::vector<mla::ItemGroup> groups;
  std::vector<unsigned char> blob;
};

// The static plan and its sizes.  Item groups: one per (kind, segment, chunk),
// in launch order: largest upper bound of an item's cost first (the chunk's
// key tiles with the segment's own keys all visible), stable.
mla_status static_plan(const mla_geom* g, const mla_segment* segs, int32_t n_segs, int64_t split_keys,
                       int32_t prot_cap, bool want_blob, mla_plan_info* info, StaticPlan* out) {
  if (info == nullptr) return fail(MLA_ERR_NULL, "info is NULL");
  mla_status st = check_geom(g, false);
  if (st != MLA_OK) return st;
  int64_t N = 0;
  if ((st = check_segments(segs, n_segs, &N)) != MLA_OK) return st;
  if (split_keys < 0) return fail(MLA_ERR_SHAPE, "split_keys = %lld must be >= 0", (long long)split_keys);
  if (prot_cap < 0 || prot_cap > N) return fail(MLA_ERR_SHAPE, "prot_cap = %d outside [0, %lld]", prot_cap, (long long)N);
  const int G = g->n_groups, hpg = g->n_heads / g->n_groups;
  const int64_t Lh = (int64_t)G * (hpg - 1);
  SegTables& T = out->T;
  segment_tables(g, segs, n_segs, split_keys, false, &T);

  struct Cand {
    mla::ItemGroup grp;
    int64_t ub;
  };
  std::vector<Cand> cands;
  int64_t global_items = 0, local_terms = 0;
  int32_t max_chunks = 0;
  for (int32_t s = 0; s < n_segs; ++s) {
    const mla::SegInfo& in = T.info[s];
    max_chunks = std::max(max_chunks, in.n_chunks);
    for (int32_t c = 0; c < in.n_chunks; ++c) {
      const mla::ChunkInfo ch = T.chunks[in.chunk_off + c];
      int64_t tiles = 0;
      for (int32_t r = ch.first_rank; r <= ch.last_rank; ++r) tiles += (segs[T.rank_seg[r]].length + 63) / 64;
      const int64_t n_glob = (in.length * G + mla::kTileRows - 1) / mla::kTileRows;
      cands.push_back({{0, s, c, (int32_t)n_glob}, tiles});
      global_items += n_glob;
      if (Lh > 0) {
        cands.push_back({{1, s, c, 0}, tiles});
        ++local_terms;
      }
    }
  }
  std::stable_sort(cands.begin(), cands.end(), [](const Cand& x, const Cand& y) { return x.ub > y.ub; });
  out->groups.resize(cands.size());
  for (size_t i = 0; i < cands.size(); ++i) out->groups[i] = cands[i].grp;

  // bounds over every protected set of at most prot_cap rows: the most
  // chunk-weighted placement fills the segments with the most chunks first
  int64_t weighted = 0;   // max over A of sum_a n_chunks(seg(a))
  if (Lh > 0) {
    std::vector<int32_t> by_chunks(T.storage);
    std::stable_sort(by_chunks.begin(), by_chunks.end(),
                     [&](int32_t x, int32_t y) { return T.info[x].n_chunks > T.info[y].n_chunks; });
    int64_t left = prot_cap;
    for (int32_t sidx : by_chunks) {
      const int64_t take = std::min<int64_t>(left, T.info[sidx].length);
      weighted += take * T.info[sidx].n_chunks;
      left -= take;
      if (left == 0) break;
    }
  }
  const int64_t local_items = Lh > 0 ? weighted * Lh / mla::kTileRows + local_terms : 0;
  if (global_items + local_items > (int64_t)INT32_MAX - 256)
    return fail(MLA_ERR_UNSUPPORTED, "too many work items for one launch");

  std::memset(info, 0, sizeof *info);
  info->geom = *g;
  info->n_rows = N;
  info->split_keys = split_keys;
  info->max_slots = N * G + (int64_t)prot_cap * Lh;
  info->max_parts = T.global_parts + weighted * Lh;
  info->n_segs = n_segs;
  info->prot_cap = prot_cap;
  info->max_items = (int32_t)(global_items + local_items);
  info->one_chunk = max_chunks == 1 ? 1 : 0;
  int64_t* L = info->layout;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return (int64_t)o;
  };
  L[P_SEGS] = take(sizeof(mla::SegInfo) * n_segs);
  L[P_RANK] = take(sizeof(int32_t) * n_segs);
  L[P_STORAGE] = take(sizeof(int32_t) * n_segs);
  L[P_CHUNKS] = take(sizeof(mla::ChunkInfo) * T.chunks.size());
  L[P_THETA] = take(sizeof(double) * mla::kMaxRopePairs);
  L[P_GROUPS] = take(sizeof(mla::ItemGroup) * std::max<size_t>(out->groups.size(), 1));
  L[P_TKV] = take(sizeof(int64_t) * n_segs);
  L[P_TLEN] = take(sizeof(int64_t) * n_segs);
  L[P_TREQ] = take(sizeof(int64_t) * n_segs);
  L[P_TORIG] = take(sizeof(int32_t) * n_segs);
  L[N_ITEM_GROUPS] = (int64_t)out->groups.size();
  L[GLOBAL_PARTS] = T.global_parts;
  info->plan_bytes = off;
  off = 0;
  const int dv = head_dv(g);
  L[W_DYN] = take(sizeof(mla::DynPlan));
  L[W_SEG_LO] = take(sizeof(int32_t) * n_segs);
  L[W_SEG_CNT] = take(sizeof(int32_t) * n_segs);
  L[W_SEG_BASE] = take(sizeof(int64_t) * n_segs);
  L[W_GROUP_BASE] = take(sizeof(int32_t) * (out->groups.size() + 1));
  L[W_ITEMS] = take(sizeof(mla::WorkItem) * std::max<int64_t>(info->max_items, 1));
  if (info->one_chunk) {
    L[W_PART_PTR] = L[W_PART_O] = L[W_PART_LSE] = -1;
  } else {
    L[W_PART_PTR] = take(sizeof(int64_t) * (size_t)(info->max_slots + 1));
    L[W_PART_O] = take(sizeof(float) * (size_t)info->max_parts * dv);
    L[W_PART_LSE] = take(sizeof(float) * (size_t)info->max_parts);
  }
  L[W_ROT] = g->value_rope ? take((size_t)rot_bytes(info->max_items)) : -1;
  info->ws_bytes = off;
  info->check = info_checksum(info);
  if (!want_blob) return MLA_OK;

  out->blob.assign(info->plan_bytes, 0);
  unsigned char* B = out->blob.data();
  std::memcpy(B + L[P_SEGS], T.info.data(), sizeof(mla::SegInfo) * n_segs);
  std::memcpy(B + L[P_RANK], T.rank_seg.data(), sizeof(int32_t) * n_segs);
  std::memcpy(B + L[P_STORAGE], T.storage.data(), sizeof(int32_t) * n_segs);
  std::memcpy(B + L[P_CHUNKS], T.chunks.data(), sizeof(mla::ChunkInfo) * T.chunks.size());
  rope_theta_rev(g, reinterpret_cast<double*>(B + L[P_THETA]));
  if (!out->groups.empty())
    std::memcpy(B + L[P_GROUPS], out->groups.data(), sizeof(mla::ItemGroup) * out->groups.size());
  for (int32_t i = 0; i < n_segs; ++i) {
    const mla_segment& sg = segs[T.storage[i]];
    reinterpret_cast<int64_t*>(B + L[P_TKV])[i] = sg.kv_start;
    reinterpret_cast<int64_t*>(B + L[P_TLEN])[i] = sg.length;
    reinterpret_cast<int64_t*>(B + L[P_TREQ])[i] = sg.req_offset;
    reinterpret_cast<int32_t*>(B + L[P_TORIG])[i] = T.storage[i];
  }
  return MLA_OK;
}

// Scratch of the allocation-free attend entry point: one array per GPU, held
// until the process ends.  In host code `scratch` names a host-side stand-in,
// not device memory, so kernels get the device address that
// hipGetSymbolAddress returns for the current device (looked up once per
// device, then kept).  Every call on a GPU shares that GPU's array, and the
// plan kernels write each entry before it is read, so nothing needs clearing.
constexpr size_t kScratchBytes = MLA_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// device address of this GPU's scratch array (looked up on the first call on
// each device, with that device current)
mla_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(MLA_ERR_UNSUPPORTED, "device %d: the scratch table holds %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (scratch)");
    if (p == nullptr || (reinterpret_cast<uintptr_t>(p) & 255u) != 0)
      return fail(MLA_ERR_HIP, "scratch array at %p is not 256-byte aligned", p);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MLA_OK;
}

// the checks shared by the two planned calls
mla_status check_planned(const mla_geom* geom, const mla_plan_info* info) {
  if (geom == nullptr || info == nullptr) return fail(MLA_ERR_NULL, "geom and info are required");
  if (info->check != info_checksum(info))
    return fail(MLA_ERR_SHAPE, "info was not written by mla_online_plan (or was changed since)");
  if (!same_geom(*geom, info->geom)) return fail(MLA_ERR_SHAPE, "geom differs from the geometry of the plan");
  return check_geom(geom, false);
}

}  // namespace

mla_status mla_online_plan_query(const mla_geom* geom, const mla_segment* segs, int32_t n_segs, int64_t split_keys,
                                 int32_t prot_cap, mla_plan_info* info) {
  g_detail.clear();
  StaticPlan sp;
  return static_plan(geom, segs, n_segs, split_keys, prot_cap, false, info, &sp);
}

mla_status mla_online_plan(const mla_geom* geom, const mla_segment* segs, int32_t n_segs, int64_t split_keys,
                           int32_t prot_cap, mla_plan_info* info, void* plan, size_t plan_bytes, void* stream) {
  g_detail.clear();
  StaticPlan sp;
  mla_status st = static_plan(geom, segs, n_segs, split_keys, prot_cap, true, info, &sp);
  if (st != MLA_OK) return st;
  if (plan == nullptr) return fail(MLA_ERR_NULL, "plan is NULL");
  if ((reinterpret_cast<uintptr_t>(plan) & 255u) != 0) return fail(MLA_ERR_SHAPE, "plan must be 256-byte aligned");
  if (plan_bytes < info->plan_bytes)
    return fail(MLA_ERR_WORKSPACE, "plan buffer %zu bytes < required %zu", plan_bytes, info->plan_bytes);
  Plan p;
  p.blob = std::move(sp.blob);
  return upload_plan(p, plan, reinterpret_cast<hipStream_t>(stream));
}

namespace {

// The body of both planned attend entry points.  use_scratch: the workspace is
// the library's per-device scratch array (workspace / ws_bytes are ignored).
mla_status attend_planned_impl(const mla_geom* geom, const mla_plan_info* info, const void* plan,
                               const int32_t* prot_rows, const int32_t* n_prot, const void* kv, const void* q_glob,
                               const void* q_loc, int32_t out_dtype, void* out_o, float* out_lse, int64_t* part_ptr,
                               int32_t* part_seg, uint8_t* row_src, int32_t* status, void* workspace,
                               size_t ws_bytes, void* stream, bool use_scratch) {
  mla_status st = check_planned(geom, info);
  if (st != MLA_OK) return st;
  const int G = geom->n_groups, hpg = geom->n_heads / geom->n_groups;
  const int64_t* L = info->layout;
  if (plan == nullptr || n_prot == nullptr || kv == nullptr || q_glob == nullptr || out_o == nullptr ||
      (!use_scratch && workspace == nullptr))
    return fail(MLA_ERR_NULL, "plan, n_prot, kv, q_glob, out_o and workspace are required");
  if (info->prot_cap > 0 && prot_rows == nullptr) return fail(MLA_ERR_NULL, "prot_rows is NULL");
  if (info->prot_cap > 0 && hpg > 1 && q_loc == nullptr) return fail(MLA_ERR_NULL, "q_loc is NULL but Local heads exist");
  if (part_seg != nullptr && part_ptr == nullptr) return fail(MLA_ERR_NULL, "part_seg needs part_ptr");
  if (out_dtype != MLA_BF16 && out_dtype != MLA_F32) return fail(MLA_ERR_SHAPE, "out_dtype %d", out_dtype);
  if (!aligned16(kv) || !aligned16(q_glob) || (q_loc && !aligned16(q_loc)) || !aligned16(out_o))
    return fail(MLA_ERR_SHAPE, "kv, q_glob, q_loc and out_o must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(plan) & 255u) != 0) return fail(MLA_ERR_SHAPE, "plan must be 256-byte aligned");
  if (use_scratch) {
    const size_t need = info->ws_bytes;
    if (need > kScratchBytes)
      return fail(MLA_ERR_WORKSPACE, "this plan needs %zu bytes of scratch; the library's scratch array holds %zu",
                  need, kScratchBytes);
    if ((st = scratch_address(&workspace)) != MLA_OK) return st;
  } else {
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return fail(MLA_ERR_SHAPE, "workspace must be 256-byte aligned");
    if (ws_bytes < info->ws_bytes)
      return fail(MLA_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, info->ws_bytes);
  }

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const unsigned char* P = reinterpret_cast<const unsigned char*>(plan);
  unsigned char* W = reinterpret_cast<unsigned char*>(workspace);
  const int32_t n_local = G * (hpg - 1);

  mla::DPlanArgs d{};
  d.segs = reinterpret_cast<const mla::SegInfo*>(P + L[P_SEGS]);
  d.storage = reinterpret_cast<const int32_t*>(P + L[P_STORAGE]);
  d.groups = reinterpret_cast<const mla::ItemGroup*>(P + L[P_GROUPS]);
  d.prot = prot_rows;
  d.n_prot_dev = n_prot;
  d.prot_cap = info->prot_cap;
  d.n_rows = info->n_rows;
  d.n_segs = info->n_segs;
  d.n_item_groups = (int32_t)L[N_ITEM_GROUPS];
  d.n_groups = G;
  d.n_local = n_local;
  d.global_parts = L[GLOBAL_PARTS];
  d.max_parts = info->max_parts;
  d.max_items = info->max_items;
  d.dyn = reinterpret_cast<mla::DynPlan*>(W + L[W_DYN]);
  d.seg_prot_lo = reinterpret_cast<int32_t*>(W + L[W_SEG_LO]);
  d.seg_prot_cnt = reinterpret_cast<int32_t*>(W + L[W_SEG_CNT]);
  d.seg_local_base = reinterpret_cast<int64_t*>(W + L[W_SEG_BASE]);
  d.group_base = reinterpret_cast<int32_t*>(W + L[W_GROUP_BASE]);
  d.items = reinterpret_cast<mla::WorkItem*>(W + L[W_ITEMS]);
  d.status_out = status;
  hipError_t e = mla::launch_dplan(d, s);
  if (e != hipSuccess) return hip_fail(e, "plan kernels");

  mla::AttendArgs a{};
  a.kv = kv;
  a.q_glob = q_glob;
  a.q_loc = q_loc;
  a.part_seg = part_seg;
  a.row_src = row_src;
  a.segs = d.segs;
  a.rank_seg = reinterpret_cast<const int32_t*>(P + L[P_RANK]);
  a.storage = d.storage;
  a.chunks = reinterpret_cast<const mla::ChunkInfo*>(P + L[P_CHUNKS]);
  a.items = d.items;
  a.prot = prot_rows;
  a.theta_rev = reinterpret_cast<const double*>(P + L[P_THETA]);
  a.seg_prot_lo = d.seg_prot_lo;
  a.seg_local_base = d.seg_local_base;
  a.dyn = d.dyn;
  a.n_rows = info->n_rows;
  a.n_slots = info->max_slots;
  a.n_parts = info->max_parts;
  a.global_parts = L[GLOBAL_PARTS];
  a.n_items = info->max_items;
  a.n_prot = info->prot_cap;
  a.n_segs = info->n_segs;
  a.n_groups = G;
  a.n_local = n_local;
  a.d_latent = geom->d_latent;
  a.d_rope = geom->d_rope;
  a.dv = head_dv(geom);
  a.scale_log2 = geom->softmax_scale * 1.4426950408889634f;
  a.local_slot_base = info->n_rows * G;
  if (info->one_chunk) {
    a.part_ptr = part_ptr;
    a.out_direct = out_o;
    a.out_direct_bf16 = out_dtype == MLA_BF16 ? 1 : 0;
    a.part_lse = out_lse;
  } else {
    a.part_ptr = part_ptr != nullptr ? part_ptr : reinterpret_cast<int64_t*>(W + L[W_PART_PTR]);
    a.part_o = reinterpret_cast<float*>(W + L[W_PART_O]);
    a.part_lse = reinterpret_cast<float*>(W + L[W_PART_LSE]);
  }
  a.rot = L[W_ROT] >= 0 ? reinterpret_cast<float*>(W + L[W_ROT]) : nullptr;
  if ((e = mla::launch_plan(a, s)) != hipSuccess) return hip_fail(e, "plan kernels");
  if ((e = mla::launch_attend(a, s)) != hipSuccess) return hip_fail(e, "attention kernel");
  if (!info->one_chunk) {
    e = mla::launch_merge(info->max_slots, a.dv, a.part_o, a.part_lse, a.part_ptr, out_dtype, out_o, out_lse, s,
                          &d.dyn->n_slots);
    if (e != hipSuccess) return hip_fail(e, "merge kernel");
  }
  return MLA_OK;
}

}  // namespace

mla_status mla_online_attend_planned(const mla_geom* geom, const mla_plan_info* info, const void* plan,
                                     const int32_t* prot_rows, const int32_t* n_prot, const void* kv,
                                     const void* q_glob, const void* q_loc, int32_t out_dtype, void* out_o,
                                     float* out_lse, int64_t* part_ptr, int32_t* part_seg, uint8_t* row_src,
                                     int32_t* status, void* workspace, size_t ws_bytes, void* stream) {
  g_detail.clear();
  return attend_planned_impl(geom, info, plan, prot_rows, n_prot, kv, q_glob, q_loc, out_dtype, out_o, out_lse,
                             part_ptr, part_seg, row_src, status, workspace, ws_bytes, stream, false);
}

mla_status mla_online_attend_planned_noalloc(const mla_geom* geom, const mla_plan_info* info, const void* plan,
                                             const int32_t* prot_rows, const int32_t* n_prot, const void* kv,
                                             const void* q_glob, const void* q_loc, int32_t out_dtype, void* out_o,
                                             float* out_lse, int64_t* part_ptr, int32_t* part_seg,
                                             uint8_t* row_src, int32_t* status, void* stream) {
  g_detail.clear();
  return attend_planned_impl(geom, info, plan, prot_rows, n_prot, kv, q_glob, q_loc, out_dtype, out_o, out_lse,
                             part_ptr, part_seg, row_src, status, nullptr, 0, stream, true);
}

mla_status mla_sliced_oproj_add_planned(const mla_geom* geom, const mla_plan_info* info, const void* o_glob,
                                        const void* o_loc, const int32_t* glob_head, const int32_t* prot_rows,
                                        const int32_t* n_prot, const void* w_o, const void* z_off, int32_t z_dtype,
                                        void* z, void* stream) {
  g_detail.clear();
  mla_status st = check_planned(geom, info);
  if (st != MLA_OK) return st;
  if ((st = check_geom(geom, true)) != MLA_OK) return st;
  const int64_t N = info->n_rows;
  const int hpg = geom->n_heads / geom->n_groups;
  if (glob_head == nullptr) return fail(MLA_ERR_NULL, "glob_head is NULL");
  for (int g = 0; g < geom->n_groups; ++g)
    if (glob_head[g] < 0 || glob_head[g] >= hpg)
      return fail(MLA_ERR_SHAPE, "glob_head[%d] = %d outside [0, %d)", g, glob_head[g], hpg);
  if (o_glob == nullptr || w_o == nullptr || z == nullptr || z_off == nullptr || n_prot == nullptr)
    return fail(MLA_ERR_NULL, "o_glob, w_o, z_off, z and n_prot are required");
  if (info->prot_cap > 0 && prot_rows == nullptr) return fail(MLA_ERR_NULL, "prot_rows is NULL");
  if (info->prot_cap > 0 && hpg > 1 && o_loc == nullptr) return fail(MLA_ERR_NULL, "o_loc is NULL but Local heads exist");
  if (z_dtype != MLA_BF16 && z_dtype != MLA_F32) return fail(MLA_ERR_SHAPE, "z_dtype %d", z_dtype);
  if (!aligned16(o_glob) || (o_loc && !aligned16(o_loc)) || !aligned16(w_o) || !aligned16(z) || !aligned16(z_off))
    return fail(MLA_ERR_SHAPE, "o_glob, o_loc, w_o, z_off and z must be 16-byte aligned");
  if (mla::oproj_workgroups(N, geom->d_model, geom->n_proj_groups) > INT32_MAX)
    return fail(MLA_ERR_UNSUPPORTED, "%lld rows x d_model %d is more o-proj tiles than one launch takes",
                (long long)N, geom->d_model);
  mla::OprojArgs a{};
  a.o_glob = o_glob;
  a.o_loc = o_loc;
  a.prot_rows = prot_rows;
  a.w_o = w_o;
  a.z_off = z_off;
  a.z = reinterpret_cast<float*>(z);
  a.n_rows = N;
  a.n_prot = info->prot_cap;
  a.n_prot_dev = n_prot;
  a.n_heads = geom->n_heads;
  a.n_groups = geom->n_groups;
  a.d_latent = head_dv(geom);
  a.d_model = geom->d_model;
  a.n_pg = geom->n_proj_groups;
  a.z_bf16 = z_dtype == MLA_BF16 ? 1 : 0;
  for (int g = 0; g < geom->n_groups; ++g) a.glob_head[g] = glob_head[g];
  const hipError_t e = mla::launch_oproj(a, 3, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "o-proj kernels");
  return MLA_OK;
}

// ---------------------------------------------------------------------------
// MLA-Off producer (Alg. 1 NativeProducer)
// ---------------------------------------------------------------------------
namespace {

struct OfflineLayout {
  Plan plan;
  std::vector<int32_t> rows;   // identity row list: every row computes its Local heads
  size_t off_o = 0;            // bf16 head outputs [N, G, hpg-1, dv]
  size_t off_wt = 0;           // W_{a,L}^T per projection group [n_pg, d_model/n_pg, K_L] bf16
  size_t total = 0;
};

mla_status offline_layout(const mla_geom* geom, const mla_segment* segs, int32_t n_segs, bool want_blob,
                          OfflineLayout* L) {
  mla_status st = check_geom(geom, true);
  if (st != MLA_OK) return st;
  int64_t N = 0;
  if ((st = check_segments(segs, n_segs, &N)) != MLA_OK) return st;
  L->rows.resize((size_t)N);
  std::iota(L->rows.begin(), L->rows.end(), 0);
  if ((st = build_plan(geom, segs, n_segs, L->rows.data(), (int32_t)N, 0, want_blob, &L->plan, true)) != MLA_OK)
    return st;
  const int hpg = geom->n_heads / geom->n_groups;
  const size_t n_out = (size_t)N * geom->n_groups * (hpg - 1);
  const size_t o_bytes = n_out * head_dv(geom) * 2;
  L->off_o = align_up((size_t)L->plan.hdr.ws_bytes, 256);
  L->off_wt = L->off_o + align_up(o_bytes, 256);
  const size_t kl = (size_t)(geom->n_groups / geom->n_proj_groups) * (hpg - 1) * head_dv(geom);
  L->total = L->off_wt + align_up((size_t)geom->d_model * kl * 2, 256);
  return MLA_OK;
}

}  // namespace

mla_status mla_offline_produce_query(const mla_geom* geom, const mla_segment* segs, int32_t n_segs,
                                     size_t* ws_bytes) {
  g_detail.clear();
  if (ws_bytes == nullptr) return fail(MLA_ERR_NULL, "ws_bytes is NULL");
  OfflineLayout L;
  const mla_status st = offline_layout(geom, segs, n_segs, false, &L);
  if (st != MLA_OK) return st;
  *ws_bytes = L.total;
  return MLA_OK;
}

mla_status mla_offline_produce(const mla_geom* geom, const mla_segment* segs, int32_t n_segs, const void* kv,
                               const void* q_loc, const int32_t* glob_head, const void* w_o, int32_t out_dtype,
                               void* z_off, void* workspace, size_t ws_bytes, void* stream) {
  g_detail.clear();
  OfflineLayout L;
  mla_status st = offline_layout(geom, segs, n_segs, true, &L);
  if (st != MLA_OK) return st;
  const int hpg = geom->n_heads / geom->n_groups;
  const int64_t N = L.plan.hdr.n_rows;
  if (out_dtype != MLA_BF16 && out_dtype != MLA_F32) return fail(MLA_ERR_SHAPE, "out_dtype %d", out_dtype);
  if (glob_head == nullptr) return fail(MLA_ERR_NULL, "glob_head is NULL");
  for (int g = 0; g < geom->n_groups; ++g)
    if (glob_head[g] < 0 || glob_head[g] >= hpg)
      return fail(MLA_ERR_SHAPE, "glob_head[%d] = %d outside [0, %d)", g, glob_head[g], hpg);
  if (z_off == nullptr || workspace == nullptr) return fail(MLA_ERR_NULL, "z_off and workspace are required");
  if (!aligned16(z_off)) return fail(MLA_ERR_SHAPE, "z_off must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return fail(MLA_ERR_SHAPE, "workspace must be 256-byte aligned");
  if (ws_bytes < L.total)
    return fail(MLA_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, L.total);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const size_t z_bytes = (size_t)N * geom->d_model * (out_dtype == MLA_BF16 ? 2 : 4);
  if (hpg == 1) {   // no Local heads: the artifact is zero
    const hipError_t e = mla::launch_fill_zero(z_off, z_bytes, s);
    return e == hipSuccess ? MLA_OK : hip_fail(e, "fill kernel");
  }
  if (kv == nullptr || q_loc == nullptr || w_o == nullptr) return fail(MLA_ERR_NULL, "kv, q_loc and w_o are required");
  if (!aligned16(kv) || !aligned16(q_loc) || !aligned16(w_o))
    return fail(MLA_ERR_SHAPE, "kv, q_loc and w_o must be 16-byte aligned");
  if (mla::oproj_workgroups(N, geom->d_model, geom->n_proj_groups) > INT32_MAX)
    return fail(MLA_ERR_UNSUPPORTED, "%lld rows x d_model %d is more o-proj tiles than one launch takes",
                (long long)N, geom->d_model);
  {
    // the Local projection's direct loads address a wave's 64 rows with 32-bit offsets
    const int64_t ldz = (int64_t)geom->n_groups * (hpg - 1) * head_dv(geom);
    if (64 * ldz * 2 >= ((int64_t)1 << 32))
      return fail(MLA_ERR_UNSUPPORTED, "Local head outputs of %lld elements a row", (long long)ldz);
  }
  if ((st = upload_plan(L.plan, workspace, s)) != MLA_OK) return st;

  unsigned char* ws = reinterpret_cast<unsigned char*>(workspace);
  mla::AttendArgs a{};
  a.kv = kv;
  a.q_glob = q_loc;   // unused: the plan holds no Global items
  a.q_loc = q_loc;
  host_plan_tables(a, L.plan.hdr, ws);
  a.n_groups = geom->n_groups;
  a.n_local = geom->n_groups * (hpg - 1);
  a.d_latent = geom->d_latent;
  a.d_rope = geom->d_rope;
  a.dv = head_dv(geom);
  a.scale_log2 = geom->softmax_scale * 1.4426950408889634f;
  a.local_slot_base = 0;
  a.out_direct = ws + L.off_o;
  a.out_direct_bf16 = 1;
  a.part_lse = nullptr;
  a.rot = L.plan.hdr.off_rot >= 0 ? reinterpret_cast<float*>(ws + L.plan.hdr.off_rot) : nullptr;
  hipError_t e = mla::launch_attend(a, s);
  if (e != hipSuccess) return hip_fail(e, "attention kernel");

  mla::OprojArgs op{};
  op.o_glob = nullptr;
  op.o_loc = ws + L.off_o;
  op.prot_rows = reinterpret_cast<const int32_t*>(ws + L.plan.hdr.off_prot);   // identity row list
  op.w_o = w_o;
  op.z_off = nullptr;
  op.z = reinterpret_cast<float*>(z_off);
  op.n_rows = N;
  op.n_prot = (int32_t)N;
  op.n_heads = geom->n_heads;
  op.n_groups = geom->n_groups;
  op.d_latent = head_dv(geom);
  op.d_model = geom->d_model;
  op.n_pg = geom->n_proj_groups;
  op.z_bf16 = out_dtype == MLA_BF16 ? 1 : 0;
  for (int g = 0; g < geom->n_groups; ++g) op.glob_head[g] = glob_head[g];
  // z_off = W_{a,L} O_L per projection group as one batched K-contiguous GEMM on
  // the shared-W_b kernel: O_L's columns of the group against its Local weights,
  // transposed once per call into the workspace
  uint16_t* wt = reinterpret_cast<uint16_t*>(ws + L.off_wt);
  if ((e = mla::launch_local_wt(op, wt, s)) != hipSuccess) return hip_fail(e, "weight transpose kernel");
  const int gpp = geom->n_groups / geom->n_proj_groups;
  const int dv = head_dv(geom);
  const int cw = geom->d_model / geom->n_proj_groups;
  mla::WbArgs g{};
  g.z = reinterpret_cast<const uint16_t*>(ws + L.off_o);
  g.w_b = wt;
  g.y = z_off;
  g.n_rows = N;
  g.d_in = gpp * (hpg - 1) * dv;
  g.d_out = cw;
  g.y_bf16 = out_dtype == MLA_BF16 ? 1 : 0;
  g.batch = geom->n_proj_groups;
  g.ldz = (int64_t)geom->n_groups * (hpg - 1) * dv;
  g.ldw = g.d_in;
  g.ldy = geom->d_model;
  g.z_batch = (int64_t)gpp * (hpg - 1) * dv;
  g.w_batch = (int64_t)cw * g.d_in;
  g.y_batch = cw;
  if ((e = mla::launch_wb(g, s)) != hipSuccess) return hip_fail(e, "Local projection kernel");
  return MLA_OK;
}

// ---------------------------------------------------------------------------
// protected token-row set (eq:protected)
// ---------------------------------------------------------------------------
namespace {

struct ProtectLayout {
  Plan table;   // storage-ordered segment table, uploaded like a plan
  int64_t n_rows = 0;
  int64_t off_kv = 0, off_len = 0, off_req = 0, off_orig = 0, off_ctl = 0, off_hist = 0;
  int64_t off_key = 0, off_flag = 0, off_list = 0, off_bcnt = 0;
  size_t total = 0;
};

mla_status protect_layout(const mla_segment* segs, int32_t n_segs, bool want_blob, ProtectLayout* L) {
  int64_t N = 0;
  const mla_status st = check_segments(segs, n_segs, &N);
  if (st != MLA_OK) return st;
  L->n_rows = N;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return (int64_t)o;
  };
  L->off_kv = take(sizeof(int64_t) * n_segs);
  L->off_len = take(sizeof(int64_t) * n_segs);
  L->off_req = take(sizeof(int64_t) * n_segs);
  L->off_orig = take(sizeof(int32_t) * n_segs);
  L->off_ctl = take(mla::kProtectCtlBytes);
  L->off_hist = take(mla::kProtectHistBytes);
  const size_t table_bytes = off;   // uploaded: the table, then zeroed control words and histogram
  L->off_key = take(sizeof(uint64_t) * (size_t)N);
  L->off_flag = take((size_t)N);
  L->off_list = take(sizeof(uint64_t) * (size_t)N);
  L->off_bcnt = take(sizeof(uint64_t) * (size_t)std::max<int64_t>(1, mla::protect_count_blocks(N)));
  L->total = off;
  if (!want_blob) return MLA_OK;
  std::vector<int32_t> storage(n_segs);
  std::iota(storage.begin(), storage.end(), 0);
  std::sort(storage.begin(), storage.end(), [&](int32_t x, int32_t y) { return segs[x].kv_start < segs[y].kv_start; });
  L->table.blob.assign(table_bytes, 0);
  unsigned char* B = L->table.blob.data();
  for (int32_t i = 0; i < n_segs; ++i) {
    const mla_segment& sg = segs[storage[i]];
    reinterpret_cast<int64_t*>(B + L->off_kv)[i] = sg.kv_start;
    reinterpret_cast<int64_t*>(B + L->off_len)[i] = sg.length;
    reinterpret_cast<int64_t*>(B + L->off_req)[i] = sg.req_offset;
    reinterpret_cast<int32_t*>(B + L->off_orig)[i] = storage[i];
  }
  return MLA_OK;
}

}  // namespace

mla_status mla_protected_rows_query(const mla_segment* segs, int32_t n_segs, size_t* ws_bytes) {
  g_detail.clear();
  if (ws_bytes == nullptr) return fail(MLA_ERR_NULL, "ws_bytes is NULL");
  ProtectLayout L;
  const mla_status st = protect_layout(segs, n_segs, false, &L);
  if (st != MLA_OK) return st;
  *ws_bytes = L.total;
  return MLA_OK;
}

mla_status mla_protected_rows(const mla_segment* segs, int32_t n_segs, const mla_protect_cfg* cfg,
                              const uint8_t* row_flags, const float* index_scores, int32_t* prot_rows,
                              int32_t* n_prot, void* workspace, size_t ws_bytes, void* stream) {
  g_detail.clear();
  if (cfg == nullptr) return fail(MLA_ERR_NULL, "cfg is NULL");
  ProtectLayout L;
  mla_status st = protect_layout(segs, n_segs, true, &L);
  if (st != MLA_OK) return st;
  if (cfg->query_seg < -1 || cfg->query_seg >= n_segs)
    return fail(MLA_ERR_SHAPE, "query_seg %d outside [-1, %d)", cfg->query_seg, n_segs);
  if (cfg->edge_rows < 0 || cfg->tail_rows < 0)
    return fail(MLA_ERR_SHAPE, "edge_rows %d and tail_rows %lld must be >= 0", cfg->edge_rows,
                (long long)cfg->tail_rows);
  if (!(cfg->budget >= 0.0 && cfg->budget <= 1.0)) return fail(MLA_ERR_SHAPE, "budget must lie in [0, 1]");
  if (prot_rows == nullptr || n_prot == nullptr || workspace == nullptr)
    return fail(MLA_ERR_NULL, "prot_rows, n_prot and workspace are required");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return fail(MLA_ERR_SHAPE, "workspace must be 256-byte aligned");
  if (ws_bytes < L.total) return fail(MLA_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, L.total);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if ((st = upload_plan(L.table, workspace, s)) != MLA_OK) return st;
  mla::ProtectArgs a{};
  a.ws = reinterpret_cast<unsigned char*>(workspace);
  a.table = a.ws;
  a.zero_ctl = 0;
  a.row_flags = row_flags;
  a.scores = index_scores;
  a.prot_rows = prot_rows;
  a.n_prot = n_prot;
  a.n_rows = L.n_rows;
  a.tail_rows = cfg->tail_rows;
  a.off_kv = L.off_kv;
  a.off_len = L.off_len;
  a.off_req = L.off_req;
  a.off_orig = L.off_orig;
  a.off_ctl = L.off_ctl;
  a.off_hist = L.off_hist;
  a.off_key = L.off_key;
  a.off_flag = L.off_flag;
  a.off_list = L.off_list;
  a.off_bcnt = L.off_bcnt;
  a.n_segs = n_segs;
  a.query_seg = cfg->query_seg;
  a.edge_rows = cfg->edge_rows;
  a.budget = cfg->budget;
  const hipError_t e = mla::launch_protect(a, s);
  if (e != hipSuccess) return hip_fail(e, "protected-row kernels");
  return MLA_OK;
}

namespace {

// workspace of the planned protected-set call: control words, histogram, keys,
// flags, the gather list and the block counts (the table stays in the plan)
size_t protect_planned_layout(int64_t N, int64_t* off_ctl, int64_t* off_hist, int64_t* off_key,
                              int64_t* off_flag, int64_t* off_list, int64_t* off_bcnt) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return (int64_t)o;
  };
  *off_ctl = take(mla::kProtectCtlBytes);
  *off_hist = take(mla::kProtectHistBytes);
  *off_key = take(sizeof(uint64_t) * (size_t)N);
  *off_flag = take((size_t)N);
  *off_list = take(sizeof(uint64_t) * (size_t)N);
  *off_bcnt = take(sizeof(uint64_t) * (size_t)std::max<int64_t>(1, mla::protect_count_blocks(N)));
  return off;
}

mla_status check_plan_info(const mla_plan_info* info) {
  if (info == nullptr) return fail(MLA_ERR_NULL, "info is NULL");
  if (info->check != info_checksum(info))
    return fail(MLA_ERR_SHAPE, "info was not written by mla_online_plan (or was changed since)");
  return MLA_OK;
}

}  // namespace

mla_status mla_protected_rows_planned_query(const mla_plan_info* info, size_t* ws_bytes) {
  g_detail.clear();
  const mla_status st = check_plan_info(info);
  if (st != MLA_OK) return st;
  if (ws_bytes == nullptr) return fail(MLA_ERR_NULL, "ws_bytes is NULL");
  int64_t o[6];
  *ws_bytes = protect_planned_layout(info->n_rows, &o[0], &o[1], &o[2], &o[3], &o[4], &o[5]);
  return MLA_OK;
}

mla_status mla_protected_rows_planned(const mla_plan_info* info, const void* plan, const mla_protect_cfg* cfg,
                                      const uint8_t* row_flags, const float* index_scores, int32_t* prot_rows,
                                      int32_t* n_prot, void* workspace, size_t ws_bytes, void* stream) {
  g_detail.clear();
  mla_status st = check_plan_info(info);
  if (st != MLA_OK) return st;
  if (cfg == nullptr) return fail(MLA_ERR_NULL, "cfg is NULL");
  if (cfg->query_seg < -1 || cfg->query_seg >= info->n_segs)
    return fail(MLA_ERR_SHAPE, "query_seg %d outside [-1, %d)", cfg->query_seg, info->n_segs);
  if (cfg->edge_rows < 0 || cfg->tail_rows < 0)
    return fail(MLA_ERR_SHAPE, "edge_rows %d and tail_rows %lld must be >= 0", cfg->edge_rows,
                (long long)cfg->tail_rows);
  if (!(cfg->budget >= 0.0 && cfg->budget <= 1.0)) return fail(MLA_ERR_SHAPE, "budget must lie in [0, 1]");
  if (plan == nullptr || prot_rows == nullptr || n_prot == nullptr || workspace == nullptr)
    return fail(MLA_ERR_NULL, "plan, prot_rows, n_prot and workspace are required");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0 || (reinterpret_cast<uintptr_t>(plan) & 255u) != 0)
    return fail(MLA_ERR_SHAPE, "plan and workspace must be 256-byte aligned");
  mla::ProtectArgs a{};
  const size_t need = protect_planned_layout(info->n_rows, &a.off_ctl, &a.off_hist, &a.off_key, &a.off_flag,
                                             &a.off_list, &a.off_bcnt);
  if (ws_bytes < need) return fail(MLA_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);
  const int64_t* L = info->layout;
  a.ws = reinterpret_cast<unsigned char*>(workspace);
  a.table = reinterpret_cast<const unsigned char*>(plan);
  a.zero_ctl = 1;
  a.off_kv = L[P_TKV];
  a.off_len = L[P_TLEN];
  a.off_req = L[P_TREQ];
  a.off_orig = L[P_TORIG];
  a.row_flags = row_flags;
  a.scores = index_scores;
  a.prot_rows = prot_rows;
  a.n_prot = n_prot;
  a.n_rows = info->n_rows;
  a.tail_rows = cfg->tail_rows;
  a.n_segs = info->n_segs;
  a.query_seg = cfg->query_seg;
  a.edge_rows = cfg->edge_rows;
  a.budget = cfg->budget;
  const hipError_t e = mla::launch_protect(a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "protected-row kernels");
  return MLA_OK;
}

mla_status mla_moe_fanout(int64_t n_rows, int32_t n_experts, const float* router, int32_t top_k, int32_t min_k,
                          float tau, int32_t* expert_idx, float* expert_w, int32_t* fanout, int32_t* expert_count,
                          void* stream) {
  g_detail.clear();
  if (n_rows < 0) return fail(MLA_ERR_SHAPE, "n_rows = %lld", (long long)n_rows);
  if (top_k < 1 || top_k > mla::kMoeMaxTopK)
    return fail(MLA_ERR_UNSUPPORTED, "top_k = %d; built: 1 .. %d", top_k, mla::kMoeMaxTopK);
  if (min_k < 1 || min_k > top_k) return fail(MLA_ERR_SHAPE, "min_k = %d outside [1, top_k = %d]", min_k, top_k);
  if (n_experts < top_k) return fail(MLA_ERR_SHAPE, "n_experts = %d < top_k = %d", n_experts, top_k);
  if (n_experts > mla::kMoeMaxExperts)
    return fail(MLA_ERR_UNSUPPORTED, "n_experts = %d; built: up to %d", n_experts, mla::kMoeMaxExperts);
  if (std::isnan(tau)) return fail(MLA_ERR_SHAPE, "tau is NaN");
  if (n_rows > INT64_MAX / n_experts) return fail(MLA_ERR_SHAPE, "n_rows * n_experts overflows");
  if (n_rows > 0 && (router == nullptr || expert_idx == nullptr || expert_w == nullptr || fanout == nullptr))
    return fail(MLA_ERR_NULL, "router, expert_idx, expert_w and fanout are required");
  const void* ptrs[] = {router, expert_idx, expert_w, fanout, expert_count};
  for (const void* q : ptrs)
    if ((reinterpret_cast<uintptr_t>(q) & 3u) != 0) return fail(MLA_ERR_SHAPE, "arrays must be 4-byte aligned");
  mla::MoeArgs a{};
  a.router = router;
  a.expert_idx = expert_idx;
  a.expert_w = expert_w;
  a.fanout = fanout;
  a.expert_count = expert_count;
  a.n_rows = n_rows;
  a.n_experts = n_experts;
  a.top_k = top_k;
  a.min_k = min_k;
  a.tau = tau;
  const hipError_t e = mla::launch_moe_fanout(a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "MoE fanout kernel");
  return MLA_OK;
}

mla_status mla_shared_wb(int64_t n_rows, int32_t d_in, int32_t d_out, const void* z, const void* w_b,
                         int32_t out_dtype, void* y, void* stream) {
  g_detail.clear();
  if (n_rows < 0) return fail(MLA_ERR_SHAPE, "n_rows = %lld", (long long)n_rows);
  if (d_in < 64 || d_in % 64 != 0) return fail(MLA_ERR_SHAPE, "d_in = %d must be a positive multiple of 64", d_in);
  if (d_in > mla::kWbMaxDin) return fail(MLA_ERR_UNSUPPORTED, "d_in = %d; built: up to %d", d_in, mla::kWbMaxDin);
  if (d_out < 1) return fail(MLA_ERR_SHAPE, "d_out = %d", d_out);
  if (out_dtype != MLA_BF16 && out_dtype != MLA_F32) return fail(MLA_ERR_SHAPE, "out_dtype %d", out_dtype);
  const int64_t n_tiles = (d_out - 1) / 256 + 1, m_tiles = n_rows / 256 + (n_rows % 256 != 0);
  if (m_tiles > ((int64_t)INT32_MAX - 8) / n_tiles)
    return fail(MLA_ERR_UNSUPPORTED, "n_rows = %lld: too many tiles", (long long)n_rows);
  if (n_rows == 0) return MLA_OK;
  if (z == nullptr || w_b == nullptr || y == nullptr) return fail(MLA_ERR_NULL, "z, w_b and y are required");
  if (!aligned16(z) || !aligned16(w_b) || !aligned16(y)) return fail(MLA_ERR_SHAPE, "z, w_b and y must be 16-byte aligned");
  mla::WbArgs a{};
  a.z = reinterpret_cast<const uint16_t*>(z);
  a.w_b = reinterpret_cast<const uint16_t*>(w_b);
  a.y = y;
  a.n_rows = n_rows;
  a.d_in = d_in;
  a.d_out = d_out;
  a.y_bf16 = out_dtype == MLA_BF16 ? 1 : 0;
  a.batch = 1;
  a.ldz = a.ldw = d_in;
  a.ldy = d_out;
  const hipError_t e = mla::launch_wb(a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "shared W_b kernel");
  return MLA_OK;
}

// ---------------------------------------------------------------------------
// diagnostic: the on-device bf16 matrix-core rate
// ---------------------------------------------------------------------------
mla_status mla_probe_mfma_bf16(int32_t iters, double* flop, float* sink, void* stream) {
  g_detail.clear();
  if (flop == nullptr || sink == nullptr) return fail(MLA_ERR_NULL, "flop and sink are required");
  if (iters < 1 || iters > (1 << 24)) return fail(MLA_ERR_SHAPE, "iters = %d outside [1, 2^24]", iters);
  int dev = 0, n_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if ((e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
    return hip_fail(e, "hipDeviceGetAttribute");
  const int n_wg = 2 * n_cu;   // two workgroups of 4 waves per compute unit: two waves per SIMD
  *flop = (double)n_wg * mla::kProbeWaves * mla::kProbeChains * (double)iters * 32768.0;
  if ((e = mla::launch_probe_mfma(iters, n_wg, sink, reinterpret_cast<hipStream_t>(stream))) != hipSuccess)
    return hip_fail(e, "probe kernel");
  return MLA_OK;
}

}  // extern "C"
