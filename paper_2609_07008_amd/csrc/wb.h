// Arguments of the shared second output projection y = W_b z.
#pragma once

#include "common.h"

namespace mla {

constexpr int kWbMaxDin = 16384;

// C = A B^T with both operands K-contiguous: batch b computes
// y[b*y_batch + m*ldy + n] = sum_k z[b*z_batch + m*ldz + k] * w_b[b*w_batch + n*ldw + k]
// (element strides and offsets); the shared W_b is batch 1 with ldz = ldw = d_in, ldy = d_out.
struct WbArgs {
  const uint16_t* z;     // [N, d_in] bf16 rows of stride ldz
  const uint16_t* w_b;   // [d_out, d_in] bf16 rows of stride ldw (a linear layer's weight)
  void* y;               // [N, d_out] f32 or bf16 rows of stride ldy
  int64_t n_rows;
  int32_t d_in;          // multiple of 64, <= kWbMaxDin
  int32_t d_out;
  int32_t y_bf16;
  int32_t batch;         // independent products, 1 or more
  int64_t ldz, ldw, ldy;
  int64_t z_batch, w_batch, y_batch;
};

hipError_t launch_wb(const WbArgs& a, hipStream_t s);

}  // namespace mla
