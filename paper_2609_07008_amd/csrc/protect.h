// Arguments of the protected token-row set kernels (Sec. 2.3, eq:protected).
#pragma once

#include "common.h"

namespace mla {

struct ProtectArgs {
  unsigned char* ws;
  const unsigned char* table;  // base of the off_kv .. off_orig arrays: the workspace (uploaded
                               // with the call) or a plan image (mla_online_plan)
  int32_t zero_ctl;            // 1: the control words and histogram are zeroed by a kernel first
  const uint8_t* row_flags;    // [N] bit 0 new, bit 1 dirty (may be null)
  const float* scores;         // [N] Indexer scores (may be null: all equal)
  int32_t* prot_rows;          // [N] out: protected rows, ascending
  int32_t* n_prot;             // [1] out
  int64_t n_rows;
  int64_t tail_rows;
  int64_t off_kv, off_len, off_req, off_orig;   // segment table, storage order (from `table`)
  int64_t off_ctl, off_hist;                     // control words, 4096-bin histogram (zero at entry)
  int64_t off_key, off_flag, off_list, off_bcnt;  // [N] u64, [N] u8, [N] u64, [count blocks] u64
  int32_t n_segs;
  int32_t query_seg;
  int32_t edge_rows;
  int32_t pad;
  double budget;
};

hipError_t launch_protect(const ProtectArgs& a, hipStream_t s);
int64_t protect_count_blocks(int64_t n_rows);
constexpr size_t kProtectCtlBytes = 256;
constexpr size_t kProtectHistBytes = 4096 * 4;

}  // namespace mla
