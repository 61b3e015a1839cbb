// Arguments of the shared second output projection y = W_b z.
#pragma once

#include "common.h"

namespace mla {

constexpr int kWbMaxDin = 16384;

struct WbArgs {
  const uint16_t* z;     // [N, d_in] bf16
  const uint16_t* w_b;   // [d_out, d_in] bf16 (a linear layer's weight)
  void* y;               // [N, d_out] f32 or bf16
  int64_t n_rows;
  int32_t d_in;          // multiple of 64, <= kWbMaxDin
  int32_t d_out;
  int32_t y_bf16;
};

hipError_t launch_wb(const WbArgs& a, hipStream_t s);

}  // namespace mla
