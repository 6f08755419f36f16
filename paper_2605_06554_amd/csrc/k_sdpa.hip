// k_sdpa.hip -- dense causal SDPA on the gathered sub-sequence (Sec. 3.5, Eq. attn-sub with
// Eq. sdpa): dispatch, the Delta = rowsum(dO * O) kernel of the backward, and the fp32 path
// (plain per-row kernels, a thread per row, used for fp32 problems). The bf16 MFMA kernels are
// in k_sdpa_mfma.hip.
#include <mutex>

#include "lh_common.h"

hipError_t lh_launch_sdpa_fwd_bf16(const LhShape& s, const void* qs, const void* ks, const void* vs, void* os,
                                   float* lse, hipStream_t st);
hipError_t lh_launch_sdpa_bwd_bf16(const LhShape& s, const void* qs, const void* ks, const void* vs,
                                   const void* dos, const float* lse, const float* delta, void* dqs,
                                   void* dks, void* dvs, hipStream_t st);
hipError_t lh_launch_sdpa_fwd_idx(const LhShape& s, const void* q, const void* k, const void* v, const void* qp,
                                  const void* kp, const void* vp, const int32_t* idx, void* os, float* lse,
                                  hipStream_t st);
hipError_t lh_launch_sdpa_bwd_idx(const LhShape& s, const void* q, const void* k, const void* v, const void* qp,
                                  const void* kp, const void* vp, const int32_t* idx, const void* dos,
                                  const float* lse, const float* delta, void* dqs, void* dks, void* dvs,
                                  hipStream_t st);

namespace lh {

// ------------------------------------------------------------------ Delta = rowsum(dO * O)
template <typename T>
__global__ void __launch_bounds__(256) sdpa_delta(const T* __restrict__ O, const T* __restrict__ dO,
                                                  float* __restrict__ delta, int64_t rows, int D) {
  constexpr int CH = 16 / sizeof(T);
  const int CPR = D / CH;  // 16 or 8 or 32 threads per row
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = t / CPR;
  const int cc = (int)(t % CPR);
  float acc = 0.0f;
  if (row < rows) {
    float a[CH], b[CH];
    load_chunk<T>(O + row * D + cc * CH, a);
    load_chunk<T>(dO + row * D + cc * CH, b);
#pragma unroll
    for (int c = 0; c < CH; ++c) acc += a[c] * b[c];
  }
  for (int d = 1; d < CPR; d <<= 1) acc += __shfl_xor(acc, d, 64);
  if (row < rows && cc == 0) delta[row] = acc;
}

// ------------------------------------------------------------------ fp32 kernels (a thread per row)
constexpr int RT = 64;  // rows per workgroup
constexpr int TT = 32;  // rows per LDS tile

template <int D>
__global__ void __launch_bounds__(RT) sdpa_fwd_f32(const float* __restrict__ Q, const float* __restrict__ K,
                                                   const float* __restrict__ V, float* __restrict__ O,
                                                   float* __restrict__ LSE, int64_t S, float scale, int Hq,
                                                   int Hs, int Gq) {
  __shared__ float Ks[TT][D];
  __shared__ float Vs[TT][D];
  const int64_t bh = blockIdx.y;
  const int64_t kvh = (bh / Hq) * Hs + (bh % Hq) / Gq;  // selection head: rows of ks, vs
  const int64_t nqt = (S + RT - 1) / RT;
  const int64_t q0 = (nqt - 1 - (int64_t)blockIdx.x) * RT;
  const int64_t myq = q0 + threadIdx.x;
  const float* Qh = Q + bh * S * D;
  float q[D], o[D];
  for (int c = 0; c < D; ++c) {
    q[c] = myq < S ? Qh[myq * D + c] : 0.0f;
    o[c] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  int64_t kend = q0 + RT;
  if (kend > S) kend = S;
  for (int64_t k0 = 0; k0 < kend; k0 += TT) {
    for (int e = threadIdx.x; e < TT * D; e += RT) {
      const int64_t key = k0 + e / D;
      Ks[e / D][e % D] = key < S ? K[(kvh * S + key) * D + e % D] : 0.0f;
      Vs[e / D][e % D] = key < S ? V[(kvh * S + key) * D + e % D] : 0.0f;
    }
    __syncthreads();
    for (int t = 0; t < TT; ++t) {
      const int64_t key = k0 + t;
      if (key > myq || key >= S) break;
      float s = 0.0f;
      for (int c = 0; c < D; ++c) s += q[c] * Ks[t][c];
      s *= scale;
      const float mn = fmaxf(m, s);
      const float al = expf(m - mn), pv = expf(s - mn);
      l = l * al + pv;
      for (int c = 0; c < D; ++c) o[c] = o[c] * al + pv * Vs[t][c];
      m = mn;
    }
    __syncthreads();
  }
  if (myq < S) {
    for (int c = 0; c < D; ++c) O[(bh * S + myq) * D + c] = o[c] / l;
    LSE[bh * S + myq] = m + logf(l);
  }
}

template <int D>
__global__ void __launch_bounds__(RT) sdpa_bwd_dq_f32(const float* __restrict__ Q, const float* __restrict__ K,
                                                      const float* __restrict__ V, const float* __restrict__ dO,
                                                      const float* __restrict__ LSE, const float* __restrict__ DELTA,
                                                      float* __restrict__ dQ, int64_t S, float scale, int Hq,
                                                      int Hs, int Gq) {
  __shared__ float Ks[TT][D];
  __shared__ float Vs[TT][D];
  const int64_t bh = blockIdx.y;
  const int64_t kvh = (bh / Hq) * Hs + (bh % Hq) / Gq;
  const int64_t nqt = (S + RT - 1) / RT;
  const int64_t q0 = (nqt - 1 - (int64_t)blockIdx.x) * RT;
  const int64_t myq = q0 + threadIdx.x;
  float q[D], go[D], dq[D];
  for (int c = 0; c < D; ++c) {
    q[c] = myq < S ? Q[(bh * S + myq) * D + c] : 0.0f;
    go[c] = myq < S ? dO[(bh * S + myq) * D + c] : 0.0f;
    dq[c] = 0.0f;
  }
  const float lse = myq < S ? LSE[bh * S + myq] : 0.0f;
  const float dl = myq < S ? DELTA[bh * S + myq] : 0.0f;
  int64_t kend = q0 + RT;
  if (kend > S) kend = S;
  for (int64_t k0 = 0; k0 < kend; k0 += TT) {
    for (int e = threadIdx.x; e < TT * D; e += RT) {
      const int64_t key = k0 + e / D;
      Ks[e / D][e % D] = key < S ? K[(kvh * S + key) * D + e % D] : 0.0f;
      Vs[e / D][e % D] = key < S ? V[(kvh * S + key) * D + e % D] : 0.0f;
    }
    __syncthreads();
    for (int t = 0; t < TT; ++t) {
      const int64_t key = k0 + t;
      if (key > myq || key >= S) break;
      float s = 0.0f, dp = 0.0f;
      for (int c = 0; c < D; ++c) {
        s += q[c] * Ks[t][c];
        dp += go[c] * Vs[t][c];
      }
      const float pv = expf(s * scale - lse);
      const float ds = pv * (dp - dl);
      for (int c = 0; c < D; ++c) dq[c] += ds * Ks[t][c];
    }
    __syncthreads();
  }
  if (myq < S)
    for (int c = 0; c < D; ++c) dQ[(bh * S + myq) * D + c] = dq[c] * scale;
}

template <int D>
__global__ void __launch_bounds__(RT) sdpa_bwd_dkdv_f32(const float* __restrict__ Q, const float* __restrict__ K,
                                                        const float* __restrict__ V, const float* __restrict__ dO,
                                                        const float* __restrict__ LSE, const float* __restrict__ DELTA,
                                                        float* __restrict__ dK, float* __restrict__ dV, int64_t S,
                                                        float scale, int Hq, int Hs, int Gq) {
  __shared__ float Qs[TT][D];
  __shared__ float dOs[TT][D];
  __shared__ float ls[TT], dls[TT];
  const int64_t bs = blockIdx.y;  // selection head: its keys gather the gradients of its Gq query heads
  const int64_t bh = bs;
  const int64_t k0 = (int64_t)blockIdx.x * RT;
  const int64_t myk = k0 + threadIdx.x;
  float kr[D], vr[D], dk[D], dv[D];
  for (int c = 0; c < D; ++c) {
    kr[c] = myk < S ? K[(bh * S + myk) * D + c] : 0.0f;
    vr[c] = myk < S ? V[(bh * S + myk) * D + c] : 0.0f;
    dk[c] = dv[c] = 0.0f;
  }
  for (int mq = 0; mq < Gq; ++mq)
  for (int64_t qt = k0; qt < S; qt += TT) {
    const int64_t bq = (bs / Hs) * Hq + (bs % Hs) * Gq + mq;  // member query head
    for (int e = threadIdx.x; e < TT * D; e += RT) {
      const int64_t q = qt + e / D;
      Qs[e / D][e % D] = q < S ? Q[(bq * S + q) * D + e % D] : 0.0f;
      dOs[e / D][e % D] = q < S ? dO[(bq * S + q) * D + e % D] : 0.0f;
    }
    for (int e = threadIdx.x; e < TT; e += RT) {
      ls[e] = qt + e < S ? LSE[bq * S + qt + e] : 0.0f;
      dls[e] = qt + e < S ? DELTA[bq * S + qt + e] : 0.0f;
    }
    __syncthreads();
    for (int t = 0; t < TT; ++t) {
      const int64_t q = qt + t;
      if (q >= S) break;
      if (q < myk) continue;
      float s = 0.0f, dp = 0.0f;
      for (int c = 0; c < D; ++c) {
        s += Qs[t][c] * kr[c];
        dp += dOs[t][c] * vr[c];
      }
      const float pv = expf(s * scale - ls[t]);
      const float ds = pv * (dp - dls[t]);
      for (int c = 0; c < D; ++c) {
        dk[c] += ds * Qs[t][c];
        dv[c] += pv * dOs[t][c];
      }
    }
    __syncthreads();
  }
  if (myk < S)
    for (int c = 0; c < D; ++c) {
      dK[(bh * S + myk) * D + c] = dk[c] * scale;
      dV[(bh * S + myk) * D + c] = dv[c];
    }
}

}  // namespace lh

using namespace lh;

hipError_t lh_launch_sdpa_fwd(const LhShape& s, const void* qs, const void* ks, const void* vs,
                              void* os, float* lse, hipStream_t st) {
  if (s.S == 0) return hipSuccess;
  if (s.dtype == LH_BF16) return lh_launch_sdpa_fwd_bf16(s, qs, ks, vs, os, lse, st);
  const int64_t BH = s.B * s.Hq;
  dim3 grid((unsigned)((s.S + RT - 1) / RT), (unsigned)BH);
  auto q = (const float*)qs;
  auto k = (const float*)ks;
  auto v = (const float*)vs;
  if (s.D == 128)
    hipLaunchKernelGGL(sdpa_fwd_f32<128>, grid, dim3(RT), 0, st, q, k, v, (float*)os, lse, s.S, s.scale, s.Hq, s.Hs, s.Gq);
  else
    hipLaunchKernelGGL(sdpa_fwd_f32<64>, grid, dim3(RT), 0, st, q, k, v, (float*)os, lse, s.S, s.scale, s.Hq, s.Hs, s.Gq);
  return hipGetLastError();
}

static hipError_t launch_delta(const LhShape& s, const void* os, const void* dos, float* delta, hipStream_t st) {
  const int64_t rows = s.B * s.Hq * s.S;
  const int CPR = s.D / (s.dtype == LH_BF16 ? 8 : 4);
  dim3 grid((unsigned)((rows * CPR + 255) / 256));
  if (s.dtype == LH_BF16)
    hipLaunchKernelGGL(sdpa_delta<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)os, (const bf16_t*)dos, delta, rows, s.D);
  else
    hipLaunchKernelGGL(sdpa_delta<float>, grid, dim3(256), 0, st, (const float*)os, (const float*)dos, delta, rows, s.D);
  return hipGetLastError();
}

hipError_t lh_launch_sdpa_fwd_indexed(const LhShape& s, const void* q, const void* k, const void* v,
                                      const void* qpyr, const void* kpyr, const void* vpyr,
                                      const int32_t* idx, void* os, float* lse, hipStream_t st) {
  if (s.S == 0) return hipSuccess;
  return lh_launch_sdpa_fwd_idx(s, q, k, v, qpyr, kpyr, vpyr, idx, os, lse, st);
}

hipError_t lh_launch_sdpa_bwd_indexed(const LhShape& s, const void* q, const void* k, const void* v,
                                      const void* qpyr, const void* kpyr, const void* vpyr,
                                      const int32_t* idx, const void* os, const float* lse,
                                      const void* dos, void* dqs, void* dks, void* dvs, float* delta,
                                      hipStream_t st) {
  if (s.S == 0) return hipSuccess;
  hipError_t e = launch_delta(s, os, dos, delta, st);
  if (e != hipSuccess) return e;
  return lh_launch_sdpa_bwd_idx(s, q, k, v, qpyr, kpyr, vpyr, idx, dos, lse, delta, dqs, dks, dvs, st);
}

hipError_t lh_launch_sdpa_bwd(const LhShape& s, const void* qs, const void* ks, const void* vs,
                              const void* os, const float* lse, const void* dos, void* dqs,
                              void* dks, void* dvs, float* delta, hipStream_t st) {
  const int64_t BH = s.B * s.Hq;
  if (s.S == 0) return hipSuccess;
  {
    hipError_t e = launch_delta(s, os, dos, delta, st);
    if (e != hipSuccess) return e;
  }
  if (s.dtype == LH_BF16) return lh_launch_sdpa_bwd_bf16(s, qs, ks, vs, dos, lse, delta, dqs, dks, dvs, st);
  auto q = (const float*)qs;
  auto k = (const float*)ks;
  auto v = (const float*)vs;
  auto g = (const float*)dos;
  dim3 gq((unsigned)((s.S + RT - 1) / RT), (unsigned)BH);
  dim3 gk((unsigned)((s.S + RT - 1) / RT), (unsigned)(s.B * s.Hs));  // per selection head
  if (s.D == 128) {
    hipLaunchKernelGGL(sdpa_bwd_dkdv_f32<128>, gk, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dks, (float*)dvs,
                       s.S, s.scale, s.Hq, s.Hs, s.Gq);
    hipLaunchKernelGGL(sdpa_bwd_dq_f32<128>, gq, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dqs, s.S, s.scale,
                       s.Hq, s.Hs, s.Gq);
  } else {
    hipLaunchKernelGGL(sdpa_bwd_dkdv_f32<64>, gk, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dks, (float*)dvs,
                       s.S, s.scale, s.Hq, s.Hs, s.Gq);
    hipLaunchKernelGGL(sdpa_bwd_dq_f32<64>, gq, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dqs, s.S, s.scale,
                       s.Hq, s.Hs, s.Gq);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ scratch of lh_sdpa_bwd_noalloc
// Delta of the backward (B * Hq * S floats) for callers that cannot allocate: a file-scope
// device array, one copy per GPU, held until the process ends. Its address on the current
// device is looked up once per device with hipGetSymbolAddress; host code never passes the
// array's name itself to a kernel. sdpa_delta overwrites every element a call reads, so
// nothing needs clearing between calls; calls that overlap on one GPU share the array and race.
static constexpr size_t kSdpaScratchBytes = (size_t)16 << 20;
static constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kSdpaScratchBytes];
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

size_t lh_sdpa_scratch_bytes() { return kSdpaScratchBytes; }

hipError_t lh_sdpa_scratch(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = reinterpret_cast<float*>(g_scratch_ptr[dev]);
  return hipSuccess;
}
