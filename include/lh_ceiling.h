/*
 * lh_ceiling.h -- measurement probe beside the Lighthouse library (libceiling.so): the rate at
 * which this chip actually issues dense bf16 matrix-core work, the achievable ceiling reported
 * next to the nominal MI355X peak (2.5166 PFLOP/s = 256 CUs x 4096 FLOP per clock x 2.4 GHz).
 * It is not part of the attention path and touches none of its buffers.
 */
#ifndef LH_CEILING_H_
#define LH_CEILING_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Enqueues `blocks` workgroups of 4 waves on `stream` (a hipStream_t as void*, NULL = null
   stream). Every wave runs `iters` rounds of 4 independent v_mfma_f32_32x32x16_bf16 chains
   (32,768 FLOP per instruction) on register operands and writes one float per lane to
   out[blocks * 256] (device memory owned by the caller). Returns the FLOPs enqueued, or -1 if
   out is NULL or blocks / iters < 1; a launch error reported by the runtime gives -2. */
int64_t lh_ceiling_mfma_bf16(float* out, int32_t blocks, int32_t iters, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LH_CEILING_H_ */
