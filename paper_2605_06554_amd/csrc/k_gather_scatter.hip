// k_gather_scatter.hip -- the data-movement stages of the layer and their adjoints.
//
//   gather       (Sec. 3.5, gather equation): row m of qs/ks/vs is the pyramid row idx[m].
//   scatter      (Sec. 3.6, Eqs. fanout and scatter): o[j] = sum over levels l of
//                os[slot(l, floor((j+1)/p^l) - 1)], the entries whose shifted range holds j.
//   scatter_bwd  adjoint of scatter: dos[m] = sum of dout over R(l_m, i_m) (clipped at N-1).
//   gather_bwd   adjoint of gather + pooling: dq[j] = sum_l dqs[slot(l, floor(j/p^l))] / p^l,
//                dk/dv also summed over the query heads of the KV group.
//
// All accumulate in fp32 in a fixed order and round once; every thread owns a 16-byte column
// chunk so that rows are read and written with full 16-byte vector accesses.
#include "lh_common.h"

namespace lh {

struct GatherArgs {
  const void *q, *k, *v, *qp, *kp, *vp;
  const int32_t* idx;
  void *qs, *ks, *vs;
  int64_t N, R, S;
  int32_t Hq, Hkv, G, D;
};

template <typename T>
__global__ void __launch_bounds__(256) gather_kernel(GatherArgs a) {
  constexpr int CH = 16 / sizeof(T);
  const int CPR = a.D / CH;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.S * CPR) return;
  const int64_t m = t / CPR;
  const int cc = (int)(t % CPR);
  const int64_t bh = blockIdx.y;
  const int hq = (int)(bh % a.Hq);
  const int64_t b = bh / a.Hq;
  const int g = hq / a.G;
  const int64_t id = a.idx[bh * a.S + m];
  const int64_t o = (bh * a.S + m) * a.D + cc * CH;
  if (id < 0 || id >= a.N + a.R) {  // not a pyramid id: zero row, never an out-of-range read
    const u32x4 z{0, 0, 0, 0};
    *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(a.qs) + o) = z;
    *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(a.ks) + o) = z;
    *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(a.vs) + o) = z;
    return;
  }
  const T *sq, *sk, *sv;
  if (id < a.N) {
    sq = reinterpret_cast<const T*>(a.q) + ((b * a.N + id) * a.Hq + hq) * a.D;
    sk = reinterpret_cast<const T*>(a.k) + ((b * a.N + id) * a.Hkv + g) * a.D;
    sv = reinterpret_cast<const T*>(a.v) + ((b * a.N + id) * a.Hkv + g) * a.D;
  } else {
    const int64_t r = id - a.N;
    sq = reinterpret_cast<const T*>(a.qp) + ((b * a.R + r) * a.Hq + hq) * a.D;
    sk = reinterpret_cast<const T*>(a.kp) + ((b * a.R + r) * a.Hkv + g) * a.D;
    sv = reinterpret_cast<const T*>(a.vp) + ((b * a.R + r) * a.Hkv + g) * a.D;
  }
  const u32x4 xq = *reinterpret_cast<const u32x4*>(sq + cc * CH);
  const u32x4 xk = *reinterpret_cast<const u32x4*>(sk + cc * CH);
  const u32x4 xv = *reinterpret_cast<const u32x4*>(sv + cc * CH);
  *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(a.qs) + o) = xq;
  *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(a.ks) + o) = xk;
  *reinterpret_cast<u32x4*>(reinterpret_cast<T*>(a.vs) + o) = xv;
}

struct ScatterArgs {
  const void* os;
  const int32_t* slot;
  void* o;
  int64_t N, S, Ptot;
  int32_t Hq, D, L;
  int64_t pw[16];
  int64_t off[17];
};

// o[b, j, hq, :]: consecutive threads cover consecutive (hq, chunk) of one base row, so the
// [B, N, Hq, D] output is written contiguously. The L slot lookups are issued together, then
// the L row loads, so a thread waits for two memory latencies rather than 2 L.
template <typename T, int L>
__global__ void __launch_bounds__(256) scatter_kernel(ScatterArgs a) {
  constexpr int CH = 16 / sizeof(T);
  const int CPR = a.D / CH;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_row = (int64_t)a.Hq * CPR;
  const int64_t j = t / per_row;
  if (j >= a.N) return;
  const int64_t rem = t % per_row;
  const int hq = (int)(rem / CPR), cc = (int)(rem % CPR);
  const int64_t b = blockIdx.y;
  const int64_t bh = b * a.Hq + hq;
  const int32_t* sl = a.slot + bh * a.Ptot;
  const T* src = reinterpret_cast<const T*>(a.os) + bh * a.S * a.D + cc * CH;
  int32_t m[L];
#pragma unroll
  for (int l = L - 1; l >= 0; --l) {
    const int64_t i = (j + 1) / a.pw[l] - 1;
    m[l] = i < 0 ? -1 : sl[a.off[l] + i];
  }
  float v[L][CH];
#pragma unroll
  for (int l = L - 1; l >= 0; --l) {
    if (m[l] >= 0 && m[l] < a.S) load_chunk<T>(src + (int64_t)m[l] * a.D, v[l]);
    else {
#pragma unroll
      for (int c = 0; c < CH; ++c) v[l][c] = 0.0f;
    }
  }
  float acc[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) acc[c] = 0.0f;
#pragma unroll
  for (int l = L - 1; l >= 0; --l)
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] += v[l][c];
  store_chunk<T>(reinterpret_cast<T*>(a.o) + ((b * a.N + j) * a.Hq + hq) * a.D + cc * CH, acc);
}

struct ScatterBwdArgs {
  const void* dout;  // [B, N, Hq, D]
  const int32_t* slot;
  void* dos;  // [B, Hq, S, D]
  int64_t N, S, Ptot, WR, U;  // U = N + P: positions of the shifted sequence
  int32_t Hq, D, HW;
  int64_t pw[16];
  int64_t off[17];
  int64_t nrows[16];
};

// Shifted window sums. With x[u] = dout[u - 1] (zero for u = 0 and u > N), the range of entry
// (l, i) is exactly the level-l window a = i + 1 of x: [a p^l, (a+1) p^l - 1]. A workgroup walks
// a range of u that is a multiple of p^(L-1) with fp32 running sums per level (as in pooling)
// and writes the sum of every closed window whose entry was gathered. dout is read once.
template <typename T, int L>
__global__ void __launch_bounds__(1024) scatter_bwd_kernel(ScatterBwdArgs a) {
  constexpr int CH = 16 / sizeof(T);
  const int CPR = a.D / CH;
  const int tid = threadIdx.x;
  const int hc = tid / CPR, cc = tid % CPR;
  const int hq = blockIdx.y * a.HW + hc;
  if (hq >= a.Hq) return;
  const int64_t b = blockIdx.z;
  const int64_t bh = b * a.Hq + hq;
  const int32_t* sl = a.slot + bh * a.Ptot;
  T* dos = reinterpret_cast<T*>(a.dos) + bh * a.S * a.D + cc * CH;
  const T* src = reinterpret_cast<const T*>(a.dout);
  const int64_t u0 = (int64_t)blockIdx.x * a.WR;
  int64_t u1 = u0 + a.WR;
  if (u1 > a.U) u1 = a.U;
  float acc[L > 1 ? L : 2][CH];
#pragma unroll
  for (int l = 0; l < (L > 1 ? L : 2); ++l)
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[l][c] = 0.0f;
  constexpr int RB = 4;
  for (int64_t ub = u0; ub < u1; ub += RB) {
    float v[RB][CH];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int64_t u = ub + r;
      if (u < u1 && u >= 1 && u <= a.N) {
        load_chunk<T>(src + ((b * a.N + (u - 1)) * a.Hq + hq) * a.D + cc * CH, v[r]);
      } else {
#pragma unroll
        for (int c = 0; c < CH; ++c) v[r][c] = 0.0f;
      }
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int64_t u = ub + r;
      if (u >= u1) break;
      // level 0: entry i = u - 1 takes x[u] = dout[u - 1]
      if (u >= 1 && u <= a.N) {
        const int32_t m = sl[u - 1];
        if (m >= 0 && m < a.S) store_chunk<T>(dos + (int64_t)m * a.D, v[r]);
      }
      if (L > 1) {
#pragma unroll
        for (int c = 0; c < CH; ++c) acc[1][c] += v[r][c];
#pragma unroll
        for (int l = 1; l < L; ++l) {
          if ((u + 1) % a.pw[l] != 0) break;
          const int64_t i = (u + 1) / a.pw[l] - 2;  // window a = i + 1 closed
          if (i >= 0 && i < a.nrows[l]) {
            const int32_t m = sl[a.off[l] + i];
            if (m >= 0 && m < a.S) store_chunk<T>(dos + (int64_t)m * a.D, acc[l]);
          }
          if (l + 1 < L) {
#pragma unroll
            for (int c = 0; c < CH; ++c) acc[l + 1 < L ? l + 1 : l][c] += acc[l][c];
          }
#pragma unroll
          for (int c = 0; c < CH; ++c) acc[l][c] = 0.0f;
        }
      }
    }
  }
}

struct GatherBwdArgs {
  const void* src;  // [B, Hq, S, D]
  const int32_t* slot;
  void* dst;  // [B, N, H, D]
  int64_t N, S, Ptot;
  int32_t Hq, H, Gs, D, L;  // output heads H; output head h sums query heads h*Gs .. h*Gs+Gs-1
  int64_t pw[16];
  int64_t off[17];
  float inv[16];
};

// Output head h sums query heads h Gs .. h Gs + Gs - 1 (Gs = G for dK/dV, 1 for dQ) over the
// levels, in the order (query head ascending, level L-1 first). For each query head the L slot
// lookups are issued together, then the L row loads; with GS > 0 (compile-time group size) the
// lookups of all heads go out first.
template <typename T, int L>
__device__ __forceinline__ void gather_bwd_head(const GatherBwdArgs& a, const int32_t* m, int64_t bhq, int cc,
                                                float* acc) {
  constexpr int CH = 16 / sizeof(T);
  const T* src = reinterpret_cast<const T*>(a.src) + bhq * a.S * a.D + cc * CH;
  float v[L][CH];
#pragma unroll
  for (int l = L - 1; l >= 0; --l) {
    if (m[l] >= 0 && m[l] < a.S) load_chunk<T>(src + (int64_t)m[l] * a.D, v[l]);
    else {
#pragma unroll
      for (int c = 0; c < CH; ++c) v[l][c] = 0.0f;
    }
  }
#pragma unroll
  for (int l = L - 1; l >= 0; --l)
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] += v[l][c] * a.inv[l];
}

template <typename T, int L, int GS>
__global__ void __launch_bounds__(256) gather_bwd_kernel(GatherBwdArgs a) {
  constexpr int CH = 16 / sizeof(T);
  const int CPR = a.D / CH;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_row = (int64_t)a.H * CPR;
  const int64_t j = t / per_row;
  if (j >= a.N) return;
  const int64_t rem = t % per_row;
  const int h = (int)(rem / CPR), cc = (int)(rem % CPR);
  const int64_t b = blockIdx.y;
  float acc[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) acc[c] = 0.0f;
  if constexpr (GS > 0) {
    int32_t m[GS][L];
#pragma unroll
    for (int g = 0; g < GS; ++g) {
      const int32_t* sl = a.slot + (b * a.Hq + (int64_t)h * GS + g) * a.Ptot;
#pragma unroll
      for (int l = L - 1; l >= 0; --l) m[g][l] = sl[a.off[l] + j / a.pw[l]];
    }
#pragma unroll
    for (int g = 0; g < GS; ++g) gather_bwd_head<T, L>(a, m[g], b * a.Hq + (int64_t)h * GS + g, cc, acc);
  } else {
    for (int g = 0; g < a.Gs; ++g) {
      const int64_t bhq = b * a.Hq + (int64_t)h * a.Gs + g;
      const int32_t* sl = a.slot + bhq * a.Ptot;
      int32_t m[L];
#pragma unroll
      for (int l = L - 1; l >= 0; --l) m[l] = sl[a.off[l] + j / a.pw[l]];
      gather_bwd_head<T, L>(a, m, bhq, cc, acc);
    }
  }
  store_chunk<T>(reinterpret_cast<T*>(a.dst) + ((b * a.N + j) * a.H + h) * a.D + cc * CH, acc);
}

template <typename T, int L>
static void launch_gather_bwd_G(const GatherBwdArgs& a, dim3 grid, hipStream_t st) {
  switch (a.Gs) {
    case 1: hipLaunchKernelGGL((gather_bwd_kernel<T, L, 1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gather_bwd_kernel<T, L, 2>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((gather_bwd_kernel<T, L, 4>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((gather_bwd_kernel<T, L, 8>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((gather_bwd_kernel<T, L, 0>), grid, dim3(256), 0, st, a); break;
  }
}

template <typename T>
static void launch_gather_bwd_L(const GatherBwdArgs& a, dim3 grid, hipStream_t st) {
  switch (a.L) {
    case 1: launch_gather_bwd_G<T, 1>(a, grid, st); break;
    case 2: launch_gather_bwd_G<T, 2>(a, grid, st); break;
    case 3: launch_gather_bwd_G<T, 3>(a, grid, st); break;
    case 4: launch_gather_bwd_G<T, 4>(a, grid, st); break;
    case 5: launch_gather_bwd_G<T, 5>(a, grid, st); break;
    case 6: launch_gather_bwd_G<T, 6>(a, grid, st); break;
    case 7: launch_gather_bwd_G<T, 7>(a, grid, st); break;
    default: launch_gather_bwd_G<T, 8>(a, grid, st); break;
  }
}

template <typename T>
static void launch_scatter_L(const ScatterArgs& a, dim3 grid, hipStream_t st) {
  switch (a.L) {
    case 1: hipLaunchKernelGGL((scatter_kernel<T, 1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((scatter_kernel<T, 2>), grid, dim3(256), 0, st, a); break;
    case 3: hipLaunchKernelGGL((scatter_kernel<T, 3>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((scatter_kernel<T, 4>), grid, dim3(256), 0, st, a); break;
    case 5: hipLaunchKernelGGL((scatter_kernel<T, 5>), grid, dim3(256), 0, st, a); break;
    case 6: hipLaunchKernelGGL((scatter_kernel<T, 6>), grid, dim3(256), 0, st, a); break;
    case 7: hipLaunchKernelGGL((scatter_kernel<T, 7>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((scatter_kernel<T, 8>), grid, dim3(256), 0, st, a); break;
  }
}

template <typename T, int L>
static hipError_t launch_scatter_bwd_T(const LhShape& s, const void* dout, const int32_t* slot,
                                       void* dos, hipStream_t st) {
  ScatterBwdArgs a;
  a.dout = dout;
  a.slot = slot;
  a.dos = dos;
  a.N = s.N;
  a.S = s.S;
  a.Ptot = s.Ptot;
  a.U = s.N + s.P;
  a.Hq = s.Hq;
  a.D = s.D;
  const int CPR = s.D / (16 / (int)sizeof(T));
  a.HW = s.Hq < 256 / CPR ? s.Hq : 256 / CPR;
  a.WR = s.P >= 64 ? s.P : s.P * ((64 + s.P - 1) / s.P);
  for (int l = 0; l < 16; ++l) a.pw[l] = s.pw[l], a.nrows[l] = l < s.L ? s.N / s.pw[l] : 0;
  for (int l = 0; l < 17; ++l) a.off[l] = s.off[l];
  dim3 grid((unsigned)((a.U + a.WR - 1) / a.WR), (unsigned)((s.Hq + a.HW - 1) / a.HW), (unsigned)s.B);
  hipLaunchKernelGGL((scatter_bwd_kernel<T, L>), grid, dim3((unsigned)(a.HW * CPR)), 0, st, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_scatter_bwd_L(const LhShape& s, const void* dout, const int32_t* slot,
                                       void* dos, hipStream_t st) {
  switch (s.L) {
    case 1: return launch_scatter_bwd_T<T, 1>(s, dout, slot, dos, st);
    case 2: return launch_scatter_bwd_T<T, 2>(s, dout, slot, dos, st);
    case 3: return launch_scatter_bwd_T<T, 3>(s, dout, slot, dos, st);
    case 4: return launch_scatter_bwd_T<T, 4>(s, dout, slot, dos, st);
    case 5: return launch_scatter_bwd_T<T, 5>(s, dout, slot, dos, st);
    case 6: return launch_scatter_bwd_T<T, 6>(s, dout, slot, dos, st);
    case 7: return launch_scatter_bwd_T<T, 7>(s, dout, slot, dos, st);
    case 8: return launch_scatter_bwd_T<T, 8>(s, dout, slot, dos, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace lh

using namespace lh;

hipError_t lh_launch_gather(const LhShape& s, const void* q, const void* k, const void* v,
                            const void* qpyr, const void* kpyr, const void* vpyr,
                            const int32_t* idx, void* qs, void* ks, void* vs, hipStream_t st) {
  GatherArgs a{q, k, v, qpyr, kpyr, vpyr, idx, qs, ks, vs, s.N, s.R, s.S, s.Hq, s.Hkv, s.G, s.D};
  const int CH = s.dtype == LH_BF16 ? 8 : 4;
  const int64_t n = s.S * (s.D / CH);
  dim3 grid((unsigned)((n + 255) / 256), (unsigned)(s.B * s.Hq));
  if (s.dtype == LH_BF16) hipLaunchKernelGGL(gather_kernel<bf16_t>, grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL(gather_kernel<float>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t lh_launch_scatter(const LhShape& s, const void* os, const int32_t* slot, void* o,
                             hipStream_t st) {
  ScatterArgs a;
  a.os = os;
  a.slot = slot;
  a.o = o;
  a.N = s.N;
  a.S = s.S;
  a.Ptot = s.Ptot;
  a.Hq = s.Hq;
  a.D = s.D;
  a.L = s.L;
  for (int l = 0; l < 16; ++l) a.pw[l] = s.pw[l];
  for (int l = 0; l < 17; ++l) a.off[l] = s.off[l];
  const int CH = s.dtype == LH_BF16 ? 8 : 4;
  const int64_t n = s.N * s.Hq * (s.D / CH);
  dim3 grid((unsigned)((n + 255) / 256), (unsigned)s.B);
  if (s.dtype == LH_BF16) launch_scatter_L<bf16_t>(a, grid, st);
  else launch_scatter_L<float>(a, grid, st);
  return hipGetLastError();
}

hipError_t lh_launch_scatter_bwd(const LhShape& s, const void* dout, const int32_t* slot,
                                 void* dos, hipStream_t st) {
  if (s.dtype == LH_BF16) return launch_scatter_bwd_L<bf16_t>(s, dout, slot, dos, st);
  return launch_scatter_bwd_L<float>(s, dout, slot, dos, st);
}

hipError_t lh_launch_gather_bwd(const LhShape& s, const void* dqs, const void* dks,
                                const void* dvs, const int32_t* slot, void* dq, void* dk,
                                void* dv, hipStream_t st) {
  const void* srcs[3] = {dqs, dks, dvs};
  void* dsts[3] = {dq, dk, dv};
  for (int which = 0; which < 3; ++which) {
    GatherBwdArgs a;
    a.src = srcs[which];
    a.slot = slot;
    a.dst = dsts[which];
    a.N = s.N;
    a.S = s.S;
    a.Ptot = s.Ptot;
    a.Hq = s.Hq;
    a.H = which == 0 ? s.Hq : s.Hkv;
    a.Gs = which == 0 ? 1 : s.G;
    a.D = s.D;
    a.L = s.L;
    for (int l = 0; l < 16; ++l) {
      a.pw[l] = s.pw[l];
      a.inv[l] = l < s.L ? 1.0f / (float)s.pw[l] : 0.0f;
    }
    for (int l = 0; l < 17; ++l) a.off[l] = s.off[l];
    const int CH = s.dtype == LH_BF16 ? 8 : 4;
    const int64_t n = s.N * a.H * (s.D / CH);
    dim3 grid((unsigned)((n + 255) / 256), (unsigned)s.B);
    if (s.dtype == LH_BF16) launch_gather_bwd_L<bf16_t>(a, grid, st);
    else launch_gather_bwd_L<float>(a, grid, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
