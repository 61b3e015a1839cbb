// Arguments of the group-sliced first output projection with the artifact add.
#pragma once

#include "common.h"

namespace mla {

struct OprojArgs {
  const void* o_glob;
  const void* o_loc;
  const int32_t* prot_rows;
  const void* w_o;
  const void* z_off;
  float* z;
  int64_t n_rows;
  int32_t n_prot;
  int32_t n_heads;
  int32_t n_groups;
  int32_t d_latent;
  int32_t d_model;
  int32_t n_pg;
  int32_t z_bf16;            // 1: z is bf16, 0: f32
  const int32_t* n_prot_dev; // if set: |A| in device memory, at most n_prot (the capacity the grid covers)
  int32_t glob_head[kMaxGroups];
};

// passes: bit 0 = Local heads over the protected rows, bit 1 = Global heads over all rows
hipError_t launch_oproj(const OprojArgs& a, int passes, hipStream_t s);
// grid size of one o-proj pass over M rows (the kernel indexes its tiles with int)
int64_t oproj_workgroups(int64_t M, int d_model, int n_pg);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
// the producer's Local weights transposed: wt [n_pg, d_model/n_pg, K_L] bf16, K_L =
// (G/n_pg)(hpg-1)d_v (a.d_latent is the head output width)
hipError_t launch_local_wt(const OprojArgs& a, uint16_t* wt, hipStream_t s);

}  // namespace mla
