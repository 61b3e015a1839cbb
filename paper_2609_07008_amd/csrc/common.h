// Internal declarations shared by the MLA-Online HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mla_online.h"

namespace mla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define MLA_LDS __attribute__((address_space(3)))

constexpr int kMaxRopePairs = 32;   // d_rope <= 64
constexpr int kTileRows = 128;      // head-rows per attention work item (4 waves x 32)
constexpr int kMaxGroups = 128;

// ----------------------------------------------------------------------------
// Plan written by the host into the attend workspace (all offsets in bytes from
// the workspace base).  Segment "rank" = position in request order.
// ----------------------------------------------------------------------------
struct SegInfo {
  int64_t kv_start;
  int64_t length;
  int64_t req_offset;
  int64_t cum_global;   // global-slot partials before this segment's first row
  int32_t rank;         // request-order rank
  int32_t n_chunks;     // chunks of this segment's visible list
  int32_t chunk_off;    // first entry in the chunk table
  int32_t pad;
};

struct ChunkInfo {
  int32_t first_rank;   // first / last segment rank covered (request order)
  int32_t last_rank;
};

// One attention work item: up to 128 consecutive head-rows of q_glob (kind 0,
// head-row = r*G + g) or of q_loc (kind 1, head-row = a*L_h + k), all of them
// belonging to rows of segment `seg`, attending to chunk `chunk` of that
// segment's visible-segment list.
struct WorkItem {
  int64_t hr_begin;
  int32_t count;
  int32_t kind;
  int32_t seg;
  int32_t chunk;
  int32_t max_u;        // largest canonical offset of the item's rows in `seg`
  int32_t pad;
};

struct PlanHeader {
  int64_t n_rows;
  int64_t n_slots;
  int64_t n_parts;
  int64_t global_parts;   // partials of all Global slots
  int32_t n_segs;
  int32_t n_items;
  int32_t n_prot;
  int32_t pad;
  // byte offsets inside the workspace
  int64_t off_segs;        // SegInfo[n_segs] by segment index
  int64_t off_rank;        // int32[n_segs]: segment index of each rank
  int64_t off_storage;     // int32[n_segs]: segment indices sorted by kv_start
  int64_t off_chunks;      // ChunkInfo[total chunks]
  int64_t off_items;       // WorkItem[n_items], in launch order
  int64_t off_prot;        // int32[n_prot]: protected rows
  int64_t off_prot_seg;    // int32[n_prot]: segment of each protected row
  int64_t off_cum_local;   // int64[n_prot + 1]: local-slot partials before row a
  int64_t off_theta;       // double[d_r/2]: base^(-2j/d_r) / (2 pi), RoPE frequency in revolutions
  int64_t total_bytes;     // bytes of the image (the part uploaded)
  int64_t off_rot;         // rotary value: f32[n_items * 128 * 128] accumulators after the image, else -1
  int64_t ws_bytes;        // image and accumulators
};

// Device-built plan (the protected set comes from device memory): the work
// items of one (kind, segment, chunk) form a group; the groups are listed in a
// launch order fixed on the host (largest upper-bound cost first), and the
// device counts each group's items and lays them out in that order.
struct ItemGroup {
  int32_t kind;      // 0: Global head-rows of every row; 1: Local head-rows of protected rows
  int32_t seg;
  int32_t chunk;
  int32_t n_items;   // kind 0: ceil(length * G / kTileRows); kind 1: counted on the device
};

// Counts of one device-planned call, written by the plan kernel before the
// attention kernels read them.
struct DynPlan {
  int64_t n_slots;
  int64_t n_parts;
  int32_t n_items;
  int32_t n_prot;
  int32_t status;    // MLA_OK, or MLA_ERR_ROWS when the protected list was rejected
  int32_t pad;
};

// ----------------------------------------------------------------------------
// launchers (defined in the .hip files); all return hipError_t of the launch
// ----------------------------------------------------------------------------
struct AttendArgs {
  const void* kv;
  const void* q_glob;
  const void* q_loc;
  float* part_o;             // [n_parts, dv] normalized partials (unused with out_direct)
  float* part_lse;           // [n_parts] natural-log lse; with out_direct [slots] (may be NULL then)
  int64_t* part_ptr;         // [n_slots + 1] CSR offsets of each slot's partials
  int32_t* part_seg;         // [n_parts, 2] or NULL
  uint8_t* row_src;          // [n_rows] or NULL
  // plan tables in device memory
  const SegInfo* segs;           // by segment index
  const int32_t* rank_seg;       // segment index of each request-order rank
  const int32_t* storage;        // segment indices by kv_start
  const ChunkInfo* chunks;
  const WorkItem* items;         // in launch order
  const int32_t* prot;           // protected rows, ascending
  const double* theta_rev;       // RoPE frequencies in revolutions
  const int32_t* prot_seg;       // host plan: segment of each protected row
  const int64_t* cum_local;      // host plan: Local partials before protected row a
  const int32_t* seg_prot_lo;    // device plan: first protected-list index of each segment
  const int64_t* seg_local_base; // device plan: Local partials before that segment's first protected row
  const DynPlan* dyn;            // device plan: this call's counts (NULL: a host plan, counts below)
  int64_t n_rows;
  int64_t n_slots;
  int64_t n_parts;
  int64_t global_parts;
  int32_t n_items;           // host plan: work items; device plan: the bound the grid covers
  int32_t n_prot;
  int32_t n_segs;
  int32_t n_groups;
  int32_t n_local;           // L_h = G*(hpg-1)
  int32_t d_latent;
  int32_t d_rope;
  int32_t dv;                // head output width: d_latent, or d_latent + d_rope (rotary value)
  float scale_log2;          // softmax_scale * log2(e)
  int64_t local_slot_base;   // slot of Local head-row 0: n_rows * n_groups, or 0 without Global slots
  void* out_direct;          // if set: one chunk per slot, the normalized O written here [slots, dv]
                             // (part_o unused)
  int32_t out_direct_bf16;   // element type of out_direct: 1 bf16, 0 f32
  float* rot;                // rotary value: [slots (out_direct) or n_parts, 128] f32 accumulators
};

hipError_t launch_plan(const AttendArgs& a, hipStream_t s);
hipError_t launch_attend(const AttendArgs& a, hipStream_t s);

// n_slots_dev: if set, the device count of slots (n_slots is then the bound the grid covers)
hipError_t launch_merge(int64_t n_slots, int32_t d_latent, const float* part_o,
                        const float* part_lse, const int64_t* part_ptr, int32_t out_dtype,
                        void* out_o, float* out_lse, hipStream_t s, const int64_t* n_slots_dev = nullptr);

// device half of a device-built plan: protected-row ranges per segment, the
// partial bases, the item counts and the work list (dplan.hip)
struct DPlanArgs {
  const SegInfo* segs;
  const int32_t* storage;
  const ItemGroup* groups;   // [n_item_groups] in launch order
  const int32_t* prot;       // device protected rows
  const int32_t* n_prot_dev; // device |A|
  int32_t prot_cap;
  int64_t n_rows;
  int32_t n_segs;
  int32_t n_item_groups;
  int32_t n_groups;          // G
  int32_t n_local;           // L_h
  int64_t global_parts;
  int64_t max_parts;         // the workspace's room for partials (chunked mode)
  int32_t max_items;
  DynPlan* dyn;
  int32_t* seg_prot_lo;      // [n_segs]
  int32_t* seg_prot_cnt;     // [n_segs]
  int64_t* seg_local_base;   // [n_segs]
  int32_t* group_base;       // [n_item_groups + 1]
  WorkItem* items;           // [max_items]
  int32_t* status_out;       // device int32 or NULL
};
hipError_t launch_dplan(const DPlanArgs& a, hipStream_t s);

// ----------------------------------------------------------------------------
// device helpers
// ----------------------------------------------------------------------------
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  // round-to-nearest-even conversion of two floats into packed bf16
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

}  // namespace mla
