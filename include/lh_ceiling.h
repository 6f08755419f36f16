/*
 * lh_ceiling.h -- measurement probes beside the Lighthouse library (libceiling.so): the rate at
 * which this chip actually issues dense bf16 matrix-core work, the achievable ceiling reported
 * next to the nominal MI355X peak (2.5166 PFLOP/s = 256 CUs x 4096 FLOP per clock x 2.4 GHz),
 * and the cost of accumulating dQ with atomics in a single-pass attention backward. They are
 * not part of the attention path and touch none of its buffers.
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

/* The dQ accumulation a single-pass SDPA backward would need, without the rest of the kernel:
   blocks laid out as the dK/dV kernel's (256 keys per 512-thread workgroup, longest first
   across `heads` heads, query tiles of 64 rows swept from the last one down to the block's
   diagonal), each adding one 64 x 128 fp32 tile per visited query tile into dq
   [heads, S, 128] (caller-owned device memory of heads * S * 128 floats), in the MFMA output
   layout (each instruction covers two 128-byte row segments). mode 0: relaxed device-scope
   float atomic adds; mode 1: plain stores of the same tiles (the traffic without atomics).
   `mfma_per_tile` > 0 adds that many 32x32x16 bf16 MFMAs per wave and tile (the compute it
   would overlap). Returns the bytes of tile payload enqueued, -1 on a bad argument, -2 on a
   launch error. */
int64_t lh_probe_dq_sweep(float* dq, int32_t S, int32_t heads, int32_t mode, int32_t mfma_per_tile, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LH_CEILING_H_ */
