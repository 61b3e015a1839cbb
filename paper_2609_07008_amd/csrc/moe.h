// Arguments of the adaptive MoE fanout kernel (Sec. 2.4, eq:moe).
#pragma once

#include "common.h"

namespace mla {

constexpr int kMoeMaxTopK = 8;
constexpr int kMoeMaxExperts = 1024;  // 16 register values per lane

struct MoeArgs {
  const float* router;     // [N, E] router weights
  int32_t* expert_idx;     // [N, top_k] out: experts by weight, descending
  float* expert_w;         // [N, top_k] out: their original weights
  int32_t* fanout;         // [N] out: K
  int32_t* expert_count;   // [E] out (may be null): rows that execute each expert
  int64_t n_rows;
  int32_t n_experts;
  int32_t top_k;
  int32_t min_k;
  float tau;
};

hipError_t launch_moe_fanout(const MoeArgs& a, hipStream_t s);

}  // namespace mla
