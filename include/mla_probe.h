/* Diagnostic of libmla_online.so: an on-device measurement of the dense bf16
 * matrix-core rate, the peak that the measured attention and projection rates
 * are set against beside the data-sheet figure.  Not an operation of the
 * method; nothing else in the library calls it.
 */
#ifndef MLA_PROBE_H
#define MLA_PROBE_H

#include <stdint.h>

#include "mla_online.h"

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------------------
 * mla_probe_mfma_bf16: enqueue one kernel whose waves do nothing but bf16
 * matrix-core products (v_mfma_f32_32x32x16_bf16, 32,768 flop each): two
 * workgroups of 4 waves per compute unit of the current device, four
 * independent accumulation chains per wave, `iters` products per chain.
 *   iters   in [1, 2^24]
 *   flop    host, out: the kernel's total flop (time the launch on `stream`
 *           with events and divide)
 *   sink    device, at least 4 bytes; written only if the accumulated sum
 *           takes one impossible value (it keeps the products from being
 *           optimised away); never read
 *   stream  hipStream_t, or NULL for the default stream
 * Errors: MLA_ERR_NULL (flop or sink), MLA_ERR_SHAPE (iters), MLA_ERR_HIP
 * (device query or launch).  Nothing is synchronized.
 * ------------------------------------------------------------------------- */
mla_status mla_probe_mfma_bf16(int32_t iters, double* flop, float* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MLA_PROBE_H */
