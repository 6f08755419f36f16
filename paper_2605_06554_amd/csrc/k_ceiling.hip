// k_ceiling.hip -- the achievable bf16 matrix-core rate of this chip (include/lh_ceiling.h).
// Each wave keeps 4 independent accumulator chains of 32x32x16 bf16 MFMAs busy with operands in
// registers: no memory traffic and no other instructions in the loop, so its rate is the
// issue ceiling at the clock the chip holds under this load.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/lh_ceiling.h"

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

__global__ void __launch_bounds__(256) mfma_loop(float* out, int iters) {
  // operands that differ per lane (random-looking bits, as real tiles are) and are unknown to
  // the compiler
  bf16x8 a, b;
  uint32_t h = (blockIdx.x * 256u + threadIdx.x) * 2654435761u;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    h ^= h << 13, h ^= h >> 17, h ^= h << 5;
    a[i] = (__bf16)((float)(h & 0xffff) * (1.0f / 32768.0f) - 1.0f);
    b[i] = (__bf16)((float)(h >> 16) * (1.0f / 32768.0f) - 1.0f);
  }
  f32x16 acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[c][i];
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

extern "C" int64_t lh_ceiling_mfma_bf16(float* out, int32_t blocks, int32_t iters, void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(mfma_loop, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, out, iters);
  if (hipGetLastError() != hipSuccess) return -2;
  return (int64_t)blocks * 4 * (int64_t)iters * 4 * 32768;
}
