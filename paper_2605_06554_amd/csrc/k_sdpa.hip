// k_sdpa.hip -- dense causal SDPA on the gathered sub-sequence (Sec. 3.5, Eq. attn-sub with
// Eq. sdpa), forward and backward, per (b, hq) over [S, D] rows.
//
// bf16 path (MFMA, gfx950): v_mfma_f32_32x32x16_bf16 tiles, fp32 accumulation, online softmax
// in the exp2 domain with the scale folded in.
//   * Forward computes S^T = K Q^T so each lane owns one query row (its softmax statistics are
//     per-lane scalars) and O^T += V^T P^T; the transposed V operand is read straight from the
//     row-major LDS tile with ds_read_b64_tr_b16, and the key order inside each 16-key MFMA
//     step follows the accumulator layout of S^T so that P^T needs no data movement.
//   * Backward is deterministic (no atomics): a dK/dV kernel (each wave owns 32 keys and
//     streams query tiles) and a dQ kernel (each wave owns 32 queries and streams key tiles),
//     after a small kernel computing Delta = rowsum(dO * O).
// fp32 path: plain per-row kernels (a thread per row) used for fp32 problems.
//
// MFMA 32x32x16 lane layouts (lane l, h = l / 32): A[m = l % 32][k = 8h + 0..7],
// B[k = 8h + 0..7][n = l % 32], C[m = 8(i/4) + 4h + i%4][n = l % 32] for i = 0..15.
#include "lh_common.h"

namespace lh {

typedef short __attribute__((address_space(3))) lds_short;
typedef s16x4 __attribute__((address_space(3))) lds_s16x4;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Transposed read of a 4x16 block of a row-major bf16 LDS matrix: within each 16-lane group,
// lane i receives Mat[r0 + j][c0 + i] for j = 0..3 when every lane s passes the address of
// Mat[r0 + s / 4][c0 + 4 (s % 4)].
__device__ __forceinline__ s16x4 tr_read(const bf16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
}

__device__ __forceinline__ bf16x8 cat8(s16x4 lo, s16x4 hi) {
  typedef __attribute__((__vector_size__(8 * sizeof(short)))) short s16x8;
  s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x8 pack8(const float* f) {
  typedef __attribute__((__vector_size__(8 * sizeof(short)))) short s16x8;
  s16x8 v;
#pragma unroll
  for (int t = 0; t < 8; ++t) v[t] = (short)f2bf(f[t]);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x8 ld8(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

// A (or B) operand of a k-step over 16 rows of a row-major LDS matrix Mat[row][col] whose
// 16 rows are ordered like the C layout of a 32-row accumulator: slots 0-3 are rows
// 4h + 0..3 and slots 4-7 are rows 8 + 4h + 0..3 of the 16-row group starting at r16;
// column = c32 + lane % 32.
__device__ __forceinline__ bf16x8 tr_operand(const bf16_t* mat, int stride, int r16, int c32, int lane) {
  const int h = lane >> 5;
  const int row = r16 + 4 * h + ((lane & 15) >> 2);
  const int col = c32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const s16x4 lo = tr_read(mat + row * stride + col);
  const s16x4 hi = tr_read(mat + (row + 8) * stride + col);
  return cat8(lo, hi);
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ------------------------------------------------------------------ bf16 forward
constexpr int FQ = 128;  // query rows per workgroup (4 waves x 32)
constexpr int FK = 64;   // keys per tile

template <int D>
__global__ void __launch_bounds__(256) sdpa_fwd_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K,
                                                     const bf16_t* __restrict__ V, bf16_t* __restrict__ O,
                                                     float* __restrict__ LSE, int64_t S, float sl2) {
  constexpr int KST = D + 8, VST = D + 16;
  __shared__ __align__(16) bf16_t Ks[FK * KST];
  __shared__ __align__(16) bf16_t Vs[FK * VST];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = lane >> 5, r32 = lane & 31;
  const int64_t bh = blockIdx.y;
  const int64_t nqt = (S + FQ - 1) / FQ;
  const int64_t q0 = (nqt - 1 - (int64_t)blockIdx.x) * FQ;  // longest rows first
  const int64_t qw = q0 + 32 * w;
  const int64_t myq = qw + r32;
  const bf16_t* Qh = Q + bh * S * D;
  const bf16_t* Kh = K + bh * S * D;
  const bf16_t* Vh = V + bh * S * D;

  bf16x8 qreg[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    if (myq < S) qreg[kk] = ld8(Qh + myq * D + 16 * kk + 8 * h);
    else qreg[kk] = bf16x8{};
  }
  f32x16 oacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) oacc[d] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;

  int64_t kend = q0 + FQ;
  if (kend > S) kend = S;
  const int nkt = (int)((kend + FK - 1) / FK);
  for (int kt = 0; kt < nkt; ++kt) {
    const int64_t k0 = (int64_t)kt * FK;
    for (int c = tid; c < FK * (D / 8); c += 256) {
      const int r = c / (D / 8), cc = c % (D / 8);
      const int64_t key = k0 + r;
      u32x4 kv{0, 0, 0, 0}, vv{0, 0, 0, 0};
      if (key < S) {
        kv = *reinterpret_cast<const u32x4*>(Kh + key * D + cc * 8);
        vv = *reinterpret_cast<const u32x4*>(Vh + key * D + cc * 8);
      }
      *reinterpret_cast<u32x4*>(Ks + r * KST + cc * 8) = kv;
      *reinterpret_cast<u32x4*>(Vs + r * VST + cc * 8) = vv;
    }
    __syncthreads();
    if (qw + 31 >= k0) {
      f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
          sacc[kb] = mfma32(ld8(Ks + (kb * 32 + r32) * KST + 16 * kk + 8 * h), qreg[kk], sacc[kb]);
      const bool diag = k0 + FK - 1 > qw;
      float mloc = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float s = sacc[kb][i] * sl2;
          const int64_t key = k0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          if (diag && key > myq) s = -INFINITY;
          sacc[kb][i] = s;
          mloc = fmaxf(mloc, s);
        }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
      const float m_new = fmaxf(m_run, mloc);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float rs = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float pv = __builtin_amdgcn_exp2f(sacc[kb][i] - m_new);
          sacc[kb][i] = pv;
          rs += pv;
        }
      rs += __shfl_xor(rs, 32, 64);
      l_run = l_run * alpha + rs;
      m_run = m_new;
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[d][i] *= alpha;
      bf16x8 pb[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        float f[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) f[t] = sacc[s >> 1][8 * (s & 1) + t];
        pb[s] = pack8(f);
      }
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          oacc[d] = mfma32(tr_operand(Vs, VST, 16 * s, 32 * d, lane), pb[s], oacc[d]);
    }
    __syncthreads();
  }
  if (myq < S) {
    const float inv = 1.0f / l_run;
    bf16_t* Oh = O + bh * S * D + myq * D;
#pragma unroll
    for (int d = 0; d < D / 32; ++d)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int col = 32 * d + 8 * g4 + 4 * h;
        uint32_t w0 = (uint32_t)f2bf(oacc[d][4 * g4 + 0] * inv) | ((uint32_t)f2bf(oacc[d][4 * g4 + 1] * inv) << 16);
        uint32_t w1 = (uint32_t)f2bf(oacc[d][4 * g4 + 2] * inv) | ((uint32_t)f2bf(oacc[d][4 * g4 + 3] * inv) << 16);
        *reinterpret_cast<uint2*>(Oh + col) = make_uint2(w0, w1);
      }
    if (h == 0) LSE[bh * S + myq] = (m_run + __log2f(l_run)) * kLn2;
  }
}

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

// ------------------------------------------------------------------ bf16 backward: dQ
constexpr int BQ = 128;  // queries per workgroup in the dQ kernel
constexpr int BK = 64;   // keys per tile in the dQ kernel

template <int D>
__global__ void __launch_bounds__(256) sdpa_bwd_dq_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K,
                                                        const bf16_t* __restrict__ V, const bf16_t* __restrict__ dO,
                                                        const float* __restrict__ LSE, const float* __restrict__ DELTA,
                                                        bf16_t* __restrict__ dQ, int64_t S, float sl2, float scale) {
  constexpr int ST = D + 8;
  __shared__ __align__(16) bf16_t Ks[BK * ST];
  __shared__ __align__(16) bf16_t Vs[BK * ST];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = lane >> 5, r32 = lane & 31;
  const int64_t bh = blockIdx.y;
  const int64_t nqt = (S + BQ - 1) / BQ;
  const int64_t q0 = (nqt - 1 - (int64_t)blockIdx.x) * BQ;
  const int64_t qw = q0 + 32 * w;
  const int64_t myq = qw + r32;
  const bf16_t* Qh = Q + bh * S * D;
  const bf16_t* Kh = K + bh * S * D;
  const bf16_t* Vh = V + bh * S * D;
  const bf16_t* dOh = dO + bh * S * D;

  bf16x8 qreg[D / 16], doreg[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    if (myq < S) {
      qreg[kk] = ld8(Qh + myq * D + 16 * kk + 8 * h);
      doreg[kk] = ld8(dOh + myq * D + 16 * kk + 8 * h);
    } else {
      qreg[kk] = bf16x8{};
      doreg[kk] = bf16x8{};
    }
  }
  const float lse2 = myq < S ? LSE[bh * S + myq] * kLog2e : INFINITY;
  const float dlt = myq < S ? DELTA[bh * S + myq] : 0.0f;
  f32x16 dqacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) dqacc[d] = f32x16{};

  int64_t kend = q0 + BQ;
  if (kend > S) kend = S;
  const int nkt = (int)((kend + BK - 1) / BK);
  for (int kt = 0; kt < nkt; ++kt) {
    const int64_t k0 = (int64_t)kt * BK;
    for (int c = tid; c < BK * (D / 8); c += 256) {
      const int r = c / (D / 8), cc = c % (D / 8);
      const int64_t key = k0 + r;
      u32x4 kv{0, 0, 0, 0}, vv{0, 0, 0, 0};
      if (key < S) {
        kv = *reinterpret_cast<const u32x4*>(Kh + key * D + cc * 8);
        vv = *reinterpret_cast<const u32x4*>(Vh + key * D + cc * 8);
      }
      *reinterpret_cast<u32x4*>(Ks + r * ST + cc * 8) = kv;
      *reinterpret_cast<u32x4*>(Vs + r * ST + cc * 8) = vv;
    }
    __syncthreads();
    if (qw + 31 >= k0) {
      f32x16 sacc[2] = {f32x16{}, f32x16{}}, pacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          sacc[kb] = mfma32(ld8(Ks + (kb * 32 + r32) * ST + 16 * kk + 8 * h), qreg[kk], sacc[kb]);
          pacc[kb] = mfma32(ld8(Vs + (kb * 32 + r32) * ST + 16 * kk + 8 * h), doreg[kk], pacc[kb]);
        }
      const bool diag = k0 + BK - 1 > qw;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t key = k0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          float pv = __builtin_amdgcn_exp2f(sacc[kb][i] * sl2 - lse2);
          if (diag && key > myq) pv = 0.0f;
          sacc[kb][i] = pv * (pacc[kb][i] - dlt);  // dS^T
        }
      bf16x8 db[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        float f[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) f[t] = sacc[s >> 1][8 * (s & 1) + t];
        db[s] = pack8(f);
      }
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          dqacc[d] = mfma32(tr_operand(Ks, ST, 16 * s, 32 * d, lane), db[s], dqacc[d]);
    }
    __syncthreads();
  }
  if (myq < S) {
    bf16_t* o = dQ + bh * S * D + myq * D;
#pragma unroll
    for (int d = 0; d < D / 32; ++d)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int col = 32 * d + 8 * g4 + 4 * h;
        uint32_t w0 = (uint32_t)f2bf(dqacc[d][4 * g4 + 0] * scale) | ((uint32_t)f2bf(dqacc[d][4 * g4 + 1] * scale) << 16);
        uint32_t w1 = (uint32_t)f2bf(dqacc[d][4 * g4 + 2] * scale) | ((uint32_t)f2bf(dqacc[d][4 * g4 + 3] * scale) << 16);
        *reinterpret_cast<uint2*>(o + col) = make_uint2(w0, w1);
      }
  }
}

// ------------------------------------------------------------------ bf16 backward: dK, dV
constexpr int CK = 128;  // keys per workgroup (4 waves x 32)
constexpr int CQ = 64;   // queries per tile

template <int D>
__global__ void __launch_bounds__(256) sdpa_bwd_dkdv_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K,
                                                          const bf16_t* __restrict__ V, const bf16_t* __restrict__ dO,
                                                          const float* __restrict__ LSE, const float* __restrict__ DELTA,
                                                          bf16_t* __restrict__ dK, bf16_t* __restrict__ dV, int64_t S,
                                                          float sl2, float scale) {
  constexpr int ST = D + 8;
  __shared__ __align__(16) bf16_t Qs[CQ * ST];
  __shared__ __align__(16) bf16_t dOs[CQ * ST];
  __shared__ float lse_s[CQ];
  __shared__ float dlt_s[CQ];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = lane >> 5, r32 = lane & 31;
  const int64_t bh = blockIdx.y;
  const int64_t k0 = (int64_t)blockIdx.x * CK;  // short key tiles (late keys) do little work
  const int64_t kw = k0 + 32 * w;
  const int64_t mykey = kw + r32;
  const bf16_t* Qh = Q + bh * S * D;
  const bf16_t* Kh = K + bh * S * D;
  const bf16_t* Vh = V + bh * S * D;
  const bf16_t* dOh = dO + bh * S * D;

  bf16x8 kreg[D / 16], vreg[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    if (mykey < S) {
      kreg[kk] = ld8(Kh + mykey * D + 16 * kk + 8 * h);
      vreg[kk] = ld8(Vh + mykey * D + 16 * kk + 8 * h);
    } else {
      kreg[kk] = bf16x8{};
      vreg[kk] = bf16x8{};
    }
  }
  f32x16 dkacc[D / 32], dvacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) dkacc[d] = dvacc[d] = f32x16{};

  const int64_t qstart = (k0 / CQ) * CQ;
  for (int64_t qt0 = qstart; qt0 < S; qt0 += CQ) {
    for (int c = tid; c < CQ * (D / 8); c += 256) {
      const int r = c / (D / 8), cc = c % (D / 8);
      const int64_t q = qt0 + r;
      u32x4 qv{0, 0, 0, 0}, dv{0, 0, 0, 0};
      if (q < S) {
        qv = *reinterpret_cast<const u32x4*>(Qh + q * D + cc * 8);
        dv = *reinterpret_cast<const u32x4*>(dOh + q * D + cc * 8);
      }
      *reinterpret_cast<u32x4*>(Qs + r * ST + cc * 8) = qv;
      *reinterpret_cast<u32x4*>(dOs + r * ST + cc * 8) = dv;
    }
    for (int c = tid; c < CQ; c += 256) {
      const int64_t q = qt0 + c;
      lse_s[c] = q < S ? LSE[bh * S + q] * kLog2e : INFINITY;
      dlt_s[c] = q < S ? DELTA[bh * S + q] : 0.0f;
    }
    __syncthreads();
    if (qt0 + CQ - 1 >= kw && kw < S) {
      f32x16 sacc[2] = {f32x16{}, f32x16{}}, pacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          sacc[qb] = mfma32(ld8(Qs + (qb * 32 + r32) * ST + 16 * kk + 8 * h), kreg[kk], sacc[qb]);
          pacc[qb] = mfma32(ld8(dOs + (qb * 32 + r32) * ST + 16 * kk + 8 * h), vreg[kk], pacc[qb]);
        }
      const bool diag = qt0 < kw + 31;
      bf16x8 pb[4], db[4];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        float pf[16], df[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int ql = qb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          float pv = __builtin_amdgcn_exp2f(sacc[qb][i] * sl2 - lse_s[ql]);
          if (diag && mykey > qt0 + ql) pv = 0.0f;
          pf[i] = pv;
          df[i] = pv * (pacc[qb][i] - dlt_s[ql]);
        }
        pb[2 * qb] = pack8(pf);
        pb[2 * qb + 1] = pack8(pf + 8);
        db[2 * qb] = pack8(df);
        db[2 * qb + 1] = pack8(df + 8);
      }
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          dvacc[d] = mfma32(pb[s], tr_operand(dOs, ST, 16 * s, 32 * d, lane), dvacc[d]);
          dkacc[d] = mfma32(db[s], tr_operand(Qs, ST, 16 * s, 32 * d, lane), dkacc[d]);
        }
    }
    __syncthreads();
  }
  // C layout: row = key kw + 8(i/4) + 4h + i%4, column d = 32 dblk + lane % 32
#pragma unroll
  for (int d = 0; d < D / 32; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t key = kw + 8 * (i >> 2) + 4 * h + (i & 3);
      if (key < S) {
        dK[(bh * S + key) * D + 32 * d + r32] = f2bf(dkacc[d][i] * scale);
        dV[(bh * S + key) * D + 32 * d + r32] = f2bf(dvacc[d][i]);
      }
    }
}

// ------------------------------------------------------------------ fp32 kernels (a thread per row)
constexpr int RT = 64;  // rows per workgroup
constexpr int TT = 32;  // rows per LDS tile

template <int D>
__global__ void __launch_bounds__(RT) sdpa_fwd_f32(const float* __restrict__ Q, const float* __restrict__ K,
                                                   const float* __restrict__ V, float* __restrict__ O,
                                                   float* __restrict__ LSE, int64_t S, float scale) {
  __shared__ float Ks[TT][D];
  __shared__ float Vs[TT][D];
  const int64_t bh = blockIdx.y;
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
      Ks[e / D][e % D] = key < S ? K[(bh * S + key) * D + e % D] : 0.0f;
      Vs[e / D][e % D] = key < S ? V[(bh * S + key) * D + e % D] : 0.0f;
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
                                                      float* __restrict__ dQ, int64_t S, float scale) {
  __shared__ float Ks[TT][D];
  __shared__ float Vs[TT][D];
  const int64_t bh = blockIdx.y;
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
      Ks[e / D][e % D] = key < S ? K[(bh * S + key) * D + e % D] : 0.0f;
      Vs[e / D][e % D] = key < S ? V[(bh * S + key) * D + e % D] : 0.0f;
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
                                                        float scale) {
  __shared__ float Qs[TT][D];
  __shared__ float dOs[TT][D];
  __shared__ float ls[TT], dls[TT];
  const int64_t bh = blockIdx.y;
  const int64_t k0 = (int64_t)blockIdx.x * RT;
  const int64_t myk = k0 + threadIdx.x;
  float kr[D], vr[D], dk[D], dv[D];
  for (int c = 0; c < D; ++c) {
    kr[c] = myk < S ? K[(bh * S + myk) * D + c] : 0.0f;
    vr[c] = myk < S ? V[(bh * S + myk) * D + c] : 0.0f;
    dk[c] = dv[c] = 0.0f;
  }
  for (int64_t qt = k0; qt < S; qt += TT) {
    for (int e = threadIdx.x; e < TT * D; e += RT) {
      const int64_t q = qt + e / D;
      Qs[e / D][e % D] = q < S ? Q[(bh * S + q) * D + e % D] : 0.0f;
      dOs[e / D][e % D] = q < S ? dO[(bh * S + q) * D + e % D] : 0.0f;
    }
    for (int e = threadIdx.x; e < TT; e += RT) {
      ls[e] = qt + e < S ? LSE[bh * S + qt + e] : 0.0f;
      dls[e] = qt + e < S ? DELTA[bh * S + qt + e] : 0.0f;
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
  const int64_t BH = s.B * s.Hq;
  if (s.S == 0) return hipSuccess;
  if (s.dtype == LH_BF16) {
    dim3 grid((unsigned)((s.S + FQ - 1) / FQ), (unsigned)BH);
    const float sl2 = s.scale * kLog2e;
    auto q = (const bf16_t*)qs;
    auto k = (const bf16_t*)ks;
    auto v = (const bf16_t*)vs;
    if (s.D == 128) hipLaunchKernelGGL(sdpa_fwd_bf16<128>, grid, dim3(256), 0, st, q, k, v, (bf16_t*)os, lse, s.S, sl2);
    else hipLaunchKernelGGL(sdpa_fwd_bf16<64>, grid, dim3(256), 0, st, q, k, v, (bf16_t*)os, lse, s.S, sl2);
  } else {
    dim3 grid((unsigned)((s.S + RT - 1) / RT), (unsigned)BH);
    auto q = (const float*)qs;
    auto k = (const float*)ks;
    auto v = (const float*)vs;
    if (s.D == 128) hipLaunchKernelGGL(sdpa_fwd_f32<128>, grid, dim3(RT), 0, st, q, k, v, (float*)os, lse, s.S, s.scale);
    else hipLaunchKernelGGL(sdpa_fwd_f32<64>, grid, dim3(RT), 0, st, q, k, v, (float*)os, lse, s.S, s.scale);
  }
  return hipGetLastError();
}

hipError_t lh_launch_sdpa_bwd(const LhShape& s, const void* qs, const void* ks, const void* vs,
                              const void* os, const float* lse, const void* dos, void* dqs,
                              void* dks, void* dvs, float* delta, hipStream_t st) {
  const int64_t BH = s.B * s.Hq;
  if (s.S == 0) return hipSuccess;
  const int64_t rows = BH * s.S;
  const int CPR = s.D / (s.dtype == LH_BF16 ? 8 : 4);
  {
    dim3 grid((unsigned)((rows * CPR + 255) / 256));
    if (s.dtype == LH_BF16)
      hipLaunchKernelGGL(sdpa_delta<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)os, (const bf16_t*)dos, delta, rows, s.D);
    else
      hipLaunchKernelGGL(sdpa_delta<float>, grid, dim3(256), 0, st, (const float*)os, (const float*)dos, delta, rows, s.D);
  }
  if (s.dtype == LH_BF16) {
    const float sl2 = s.scale * kLog2e;
    auto q = (const bf16_t*)qs;
    auto k = (const bf16_t*)ks;
    auto v = (const bf16_t*)vs;
    auto g = (const bf16_t*)dos;
    dim3 gk((unsigned)((s.S + CK - 1) / CK), (unsigned)BH);
    dim3 gq((unsigned)((s.S + BQ - 1) / BQ), (unsigned)BH);
    if (s.D == 128) {
      hipLaunchKernelGGL(sdpa_bwd_dkdv_bf16<128>, gk, dim3(256), 0, st, q, k, v, g, lse, delta, (bf16_t*)dks, (bf16_t*)dvs, s.S, sl2, s.scale);
      hipLaunchKernelGGL(sdpa_bwd_dq_bf16<128>, gq, dim3(256), 0, st, q, k, v, g, lse, delta, (bf16_t*)dqs, s.S, sl2, s.scale);
    } else {
      hipLaunchKernelGGL(sdpa_bwd_dkdv_bf16<64>, gk, dim3(256), 0, st, q, k, v, g, lse, delta, (bf16_t*)dks, (bf16_t*)dvs, s.S, sl2, s.scale);
      hipLaunchKernelGGL(sdpa_bwd_dq_bf16<64>, gq, dim3(256), 0, st, q, k, v, g, lse, delta, (bf16_t*)dqs, s.S, sl2, s.scale);
    }
  } else {
    auto q = (const float*)qs;
    auto k = (const float*)ks;
    auto v = (const float*)vs;
    auto g = (const float*)dos;
    dim3 gk((unsigned)((s.S + RT - 1) / RT), (unsigned)BH);
    if (s.D == 128) {
      hipLaunchKernelGGL(sdpa_bwd_dkdv_f32<128>, gk, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dks, (float*)dvs, s.S, s.scale);
      hipLaunchKernelGGL(sdpa_bwd_dq_f32<128>, gk, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dqs, s.S, s.scale);
    } else {
      hipLaunchKernelGGL(sdpa_bwd_dkdv_f32<64>, gk, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dks, (float*)dvs, s.S, s.scale);
      hipLaunchKernelGGL(sdpa_bwd_dq_f32<64>, gk, dim3(RT), 0, st, q, k, v, g, lse, delta, (float*)dqs, s.S, s.scale);
    }
  }
  return hipGetLastError();
}
