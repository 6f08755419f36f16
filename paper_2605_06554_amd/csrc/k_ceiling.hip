// k_ceiling.hip -- measurement probes (include/lh_ceiling.h). The MFMA loop: each wave keeps 4
// independent accumulator chains of 32x32x16 bf16 MFMAs busy with operands in registers, no
// memory traffic and no other instructions, so its rate is the issue ceiling at the clock the
// chip holds under this load. The dQ sweep: the atomic dQ accumulation of a single-pass
// attention backward, alone or beside a given amount of MFMA work.
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

// dQ sweep of a single-pass backward (include/lh_ceiling.h): the dK/dV kernel's block order
// (linear id = rank * heads + head, rank 0 the head's first 256 keys) and query sweep.
constexpr int kCK = 256, kCQ = 64, kD = 128;

template <int MODE>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
dq_sweep(float* dq, int S, int nmfma) {
  const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
  const int rank = (int)(lin / gridDim.y);
  const int64_t head = lin % gridDim.y;
  const int k0 = rank * kCK;
  const int qstart = (k0 / kCQ) * kCQ;
  const int nqt = (S - qstart + kCQ - 1) / kCQ;
  const int qlast = qstart + (nqt - 1) * kCQ;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // wave w adds rows 32 (w & 1) .. +31, columns 32 (w >> 1) .. +31 of the 64 x 128 tile; element
  // i of lane l is row 8 (i / 4) + 4 (l / 32) + i % 4, column l % 32 (MFMA 32x32 output)
  const int rb = 32 * (w & 1) + 4 * (lane >> 5), col = 32 * (w >> 1) + (lane & 31);
  float* base = dq + head * (int64_t)S * kD;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = (__bf16)(0.001f * (lane + i)), b[i] = (__bf16)(0.002f * (i - lane));
  f32x16 acc[4] = {};
  for (int it = 0; it < nqt; ++it) {
    const int qt0 = qlast - it * kCQ;
    for (int m = 0; m < nmfma; m += 4) {
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int q = qt0 + rb + 8 * (j >> 2) + (j & 3);
      const float v = 1.0f + acc[j & 3][j];
      if (q < S) {
        float* p = base + (int64_t)q * kD + col;
        if (MODE == 0) __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else *p = v;
      }
    }
  }
}

}  // namespace

extern "C" int64_t lh_probe_dq_sweep(float* dq, int32_t S, int32_t heads, int32_t mode, int32_t mfma_per_tile,
                                     void* stream) {
  if (!dq || S < 1 || heads < 1 || (mode != 0 && mode != 1) || mfma_per_tile < 0) return -1;
  const dim3 grid((unsigned)((S + kCK - 1) / kCK), (unsigned)heads);
  if (mode == 0) hipLaunchKernelGGL(dq_sweep<0>, grid, dim3(512), 0, (hipStream_t)stream, dq, S, mfma_per_tile);
  else hipLaunchKernelGGL(dq_sweep<1>, grid, dim3(512), 0, (hipStream_t)stream, dq, S, mfma_per_tile);
  if (hipGetLastError() != hipSuccess) return -2;
  int64_t tiles = 0;
  for (int r = 0; r < (int)grid.x; ++r) tiles += (S - (r * kCK / kCQ) * kCQ + kCQ - 1) / kCQ;
  return tiles * heads * kCQ * kD * 4;
}

extern "C" int64_t lh_ceiling_mfma_bf16(float* out, int32_t blocks, int32_t iters, void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(mfma_loop, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, out, iters);
  if (hipGetLastError() != hipSuccess) return -2;
  return (int64_t)blocks * 4 * (int64_t)iters * 4 * 32768;
}
