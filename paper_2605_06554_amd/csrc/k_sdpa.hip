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

// ------------------------------------------------------------------ tiles in LDS
// A tile is TR rows of D bf16 values (D * 2 bytes per row, no padding). 16-byte chunk c of
// row r is stored at chunk position c ^ swz(r), swz(r) = 2 (r % 8) masked to the D / 8 chunks
// of a row: consecutive rows reading the same logical chunk hit different chunk positions (no
// bank conflicts for b128 reads), and the XOR with an even value keeps chunk pairs (2m, 2m+1)
// adjacent and in order, so the 32-byte row segments of the transposed loads stay intact.
template <int D>
__device__ __forceinline__ int swz(int r) { return ((r & 7) << 1) & (D / 8 - 1); }

template <int D>
__device__ __forceinline__ int tile_off(int r, int col) {  // element offset of (row, col)
  return r * D + ((((col >> 3) ^ swz<D>(r))) << 3) + (col & 7);
}

// Direct global -> LDS copy of TR rows starting at row r0 of a [S, D] bf16 matrix into a
// swizzled tile, by the NW waves of the block. Each wave instruction writes 1 KB of LDS
// contiguously (lane i -> byte 16 i), so every lane fetches the logical chunk that belongs at
// its physical position. Rows past S are clamped to row S - 1 (callers mask them).
template <int D, int TR, int NW>
__device__ __forceinline__ void load_tile_lds(bf16_t* tile, const bf16_t* src, int64_t r0, int64_t S, int w, int lane) {
  constexpr int CPR = D / 8;                 // chunks per row
  constexpr int PER_WAVE = TR * CPR / 64;    // wave instructions per tile
  static_assert(TR * CPR % (64 * NW) == 0, "tile must split evenly over the waves");
#pragma unroll
  for (int j = 0; j < PER_WAVE / NW; ++j) {
    const int blk = w * (PER_WAVE / NW) + j;   // 1 KB block of the tile
    const int pos = blk * 64 + lane;           // physical chunk index in the tile
    const int r = pos / CPR, pc = pos % CPR;
    const int c = pc ^ swz<D>(r);
    int64_t gr = r0 + r;
    if (gr > S - 1) gr = S - 1;
    const bf16_t* g = src + gr * D + c * 8;
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                     (__attribute__((address_space(3))) void*)(tile + blk * 512), 16, 0, 0);
  }
}

// MFMA operand: 8 consecutive columns (16 bytes) of one tile row.
template <int D>
__device__ __forceinline__ bf16x8 tile_row8(const bf16_t* tile, int r, int col) {
  return *reinterpret_cast<const bf16x8*>(tile + tile_off<D>(r, col));
}

// Transposed operand from a swizzled tile: slots 0-3 are rows r16 + 4h + 0..3 and slots 4-7 are
// rows r16 + 8 + 4h + 0..3; column c32 + lane % 32 (see tr_read).
template <int D>
__device__ __forceinline__ bf16x8 tile_tr8(const bf16_t* tile, int r16, int c32, int lane) {
  const int h = lane >> 5;
  const int row = r16 + 4 * h + ((lane & 15) >> 2);
  const int col = c32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const s16x4 lo = tr_read(tile + tile_off<D>(row, col));
  const s16x4 hi = tr_read(tile + tile_off<D>(row + 8, col));
  return cat8(lo, hi);
}

__device__ __forceinline__ bf16x8 cvt8(const float* f) {
  typedef __attribute__((__vector_size__(8 * sizeof(float)))) float f32x8;
  f32x8 v = {f[0], f[1], f[2], f[3], f[4], f[5], f[6], f[7]};
  return __builtin_convertvector(v, bf16x8);
}

// ------------------------------------------------------------------ bf16 forward
constexpr int FW = 8;         // waves per workgroup
constexpr int FQ = 32 * FW;   // query rows per workgroup
constexpr int FK = 64;        // keys per tile
constexpr float kRescale = 8.0f;  // lazy rescaling threshold (log2 units)

template <int D>
__global__ void __launch_bounds__(64 * FW) __attribute__((amdgpu_waves_per_eu(2, 2)))
sdpa_fwd_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
              bf16_t* __restrict__ O, float* __restrict__ LSE, int64_t S, float sl2) {
  __shared__ __align__(16) bf16_t Ks[2][FK * D];
  __shared__ __align__(16) bf16_t Vs[2][FK * D];
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

  int64_t kend = q0 + FQ;
  if (kend > S) kend = S;
  const int nkt = (int)((kend + FK - 1) / FK);
  load_tile_lds<D, FK, FW>(Ks[0], Kh, 0, S, w, lane);
  load_tile_lds<D, FK, FW>(Vs[0], Vh, 0, S, w, lane);

  bf16x8 qreg[D / 16];
  const int64_t qrow = myq < S ? myq : S - 1;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) qreg[kk] = ld8(Qh + qrow * D + 16 * kk + 8 * h);
  f32x16 oacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) oacc[d] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;

  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    __syncthreads();  // tile kt landed (the wait precedes the barrier); buffer buf^1 is free
    if (kt + 1 < nkt) {
      load_tile_lds<D, FK, FW>(Ks[buf ^ 1], Kh, (int64_t)(kt + 1) * FK, S, w, lane);
      load_tile_lds<D, FK, FW>(Vs[buf ^ 1], Vh, (int64_t)(kt + 1) * FK, S, w, lane);
    }
    const int64_t k0 = (int64_t)kt * FK;
    if (qw + 31 < k0) continue;  // every key of this tile is in the future of this wave's rows
    const bf16_t* Kt = Ks[buf];
    const bf16_t* Vt = Vs[buf];
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        sacc[kb] = mfma32(tile_row8<D>(Kt, kb * 32 + r32, 16 * kk + 8 * h), qreg[kk], sacc[kb]);
    if (k0 + FK - 1 > qw) {  // diagonal tile: mask keys after the row
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t key = k0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          if (key > myq) sacc[kb][i] = -INFINITY;
        }
    }
    float mloc = sacc[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mloc = fmaxf(mloc, sacc[kb][i]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * sl2;
    if (mloc > m_run + kRescale) {  // new running max: rescale what was accumulated so far
      const float alpha = __builtin_amdgcn_exp2f(m_run - mloc);
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[d][i] *= alpha;
      m_run = mloc;
    }
    bf16x8 pb[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      float f[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        f[t] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[s >> 1][8 * (s & 1) + t], sl2, -m_run));
        l_run += f[t];
      }
      pb[s] = cvt8(f);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
        oacc[d] = mfma32(tile_tr8<D>(Vt, 16 * s, 32 * d, lane), pb[s], oacc[d]);
  }
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (myq < S) {
    const float inv = 1.0f / l_tot;
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
    if (h == 0) LSE[bh * S + myq] = (m_run + __log2f(l_tot)) * kLn2;
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
// Each wave owns 32 query rows (its Q and dO rows stay in registers) and streams double-
// buffered K/V tiles: S^T = K Q^T and dP^T = V dO^T give, per lane, one query row's
// P = exp2(S scale log2e - lse log2e) and dS = P (dP - Delta); dQ^T += K^T dS^T with the
// transposed K operand read from the same LDS tile.
constexpr int QW = 8;        // waves per workgroup (dQ)
constexpr int BQ = 32 * QW;  // query rows per workgroup
constexpr int BK = 64;       // keys per tile

template <int D>
__global__ void __launch_bounds__(64 * QW) __attribute__((amdgpu_waves_per_eu(2, 2)))
sdpa_bwd_dq_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
                 const bf16_t* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ DELTA,
                 bf16_t* __restrict__ dQ, int64_t S, float sl2, float scale) {
  __shared__ __align__(16) bf16_t Ks[2][BK * D];
  __shared__ __align__(16) bf16_t Vs[2][BK * D];
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

  int64_t kend = q0 + BQ;
  if (kend > S) kend = S;
  const int nkt = (int)((kend + BK - 1) / BK);
  load_tile_lds<D, BK, QW>(Ks[0], Kh, 0, S, w, lane);
  load_tile_lds<D, BK, QW>(Vs[0], Vh, 0, S, w, lane);

  const int64_t qrow = myq < S ? myq : S - 1;
  bf16x8 qreg[D / 16], doreg[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    qreg[kk] = ld8(Qh + qrow * D + 16 * kk + 8 * h);
    doreg[kk] = ld8(dOh + qrow * D + 16 * kk + 8 * h);
  }
  const float lse2 = myq < S ? LSE[bh * S + myq] * kLog2e : INFINITY;
  const float dlt = myq < S ? DELTA[bh * S + myq] : 0.0f;
  f32x16 dqacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) dqacc[d] = f32x16{};

  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    __syncthreads();
    if (kt + 1 < nkt) {
      load_tile_lds<D, BK, QW>(Ks[buf ^ 1], Kh, (int64_t)(kt + 1) * BK, S, w, lane);
      load_tile_lds<D, BK, QW>(Vs[buf ^ 1], Vh, (int64_t)(kt + 1) * BK, S, w, lane);
    }
    const int64_t k0 = (int64_t)kt * BK;
    if (qw + 31 < k0) continue;
    const bf16_t* Kt = Ks[buf];
    const bf16_t* Vt = Vs[buf];
    const bool diag = k0 + BK - 1 > qw;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x16 sacc = f32x16{}, pacc = f32x16{};
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        sacc = mfma32(tile_row8<D>(Kt, kb * 32 + r32, 16 * kk + 8 * h), qreg[kk], sacc);
        pacc = mfma32(tile_row8<D>(Vt, kb * 32 + r32, 16 * kk + 8 * h), doreg[kk], pacc);
      }
      bf16x8 db[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float f[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int i = 8 * u + t;
          float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[i], sl2, -lse2));
          if (diag && k0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3) > myq) pv = 0.0f;
          f[t] = pv * (pacc[i] - dlt);
        }
        db[u] = cvt8(f);
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int d = 0; d < D / 32; ++d)
          dqacc[d] = mfma32(tile_tr8<D>(Kt, kb * 32 + 16 * u, 32 * d, lane), db[u], dqacc[d]);
    }
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
// Each wave owns 32 keys (their V rows stay in registers; the workgroup's K rows sit in LDS for
// the whole kernel) and streams double-buffered Q/dO tiles with their lse and Delta:
// S = Q K^T and dP = dO V^T (per lane: one key, 16 queries), then dV += P^T dO and
// dK += dS^T Q with the transposed dO/Q operands read from the same LDS tiles. Query tiles are
// processed in two 32-row halves to bound live registers.
constexpr int KWV = 4;        // waves per workgroup (dK/dV)
constexpr int CK = 32 * KWV;  // keys per workgroup
constexpr int CQ = 64;        // queries per tile

template <int D>
__global__ void __launch_bounds__(64 * KWV) __attribute__((amdgpu_waves_per_eu(1, 1)))
sdpa_bwd_dkdv_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
                   const bf16_t* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ DELTA,
                   bf16_t* __restrict__ dK, bf16_t* __restrict__ dV, int64_t S, float sl2, float scale) {
  __shared__ __align__(16) bf16_t Qs[2][CQ * D];
  __shared__ __align__(16) bf16_t dOs[2][CQ * D];
  __shared__ __align__(16) float lse_s[2][CQ];
  __shared__ __align__(16) float dlt_s[2][CQ];
  __shared__ __align__(16) bf16_t Kw[CK * D];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = lane >> 5, r32 = lane & 31;
  const int64_t bh = blockIdx.y;
  const int64_t k0 = (int64_t)blockIdx.x * CK;  // early keys see the most queries: launched first
  const int64_t kw = k0 + 32 * w;
  const int64_t mykey = kw + r32;
  const bf16_t* Qh = Q + bh * S * D;
  const bf16_t* Kh = K + bh * S * D;
  const bf16_t* Vh = V + bh * S * D;
  const bf16_t* dOh = dO + bh * S * D;
  const float* Lh = LSE + bh * S;
  const float* Dh = DELTA + bh * S;

  const int64_t qstart = (k0 / CQ) * CQ;
  const int nqt = (int)((S - qstart + CQ - 1) / CQ);
  auto stage = [&](int b, int64_t qt0) {
    load_tile_lds<D, CQ, KWV>(Qs[b], Qh, qt0, S, w, lane);
    load_tile_lds<D, CQ, KWV>(dOs[b], dOh, qt0, S, w, lane);
    if (tid < CQ) {
      const int64_t q = qt0 + tid;
      lse_s[b][tid] = q < S ? Lh[q] * kLog2e : INFINITY;
      dlt_s[b][tid] = q < S ? Dh[q] : 0.0f;
    }
  };
  load_tile_lds<D, CK, KWV>(Kw, Kh, k0, S, w, lane);
  stage(0, qstart);

  const int64_t krow = mykey < S ? mykey : S - 1;
  bf16x8 vreg[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) vreg[kk] = ld8(Vh + krow * D + 16 * kk + 8 * h);
  f32x16 dkacc[D / 32], dvacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) dkacc[d] = dvacc[d] = f32x16{};

  for (int it = 0; it < nqt; ++it) {
    const int buf = it & 1;
    const int64_t qt0 = qstart + (int64_t)it * CQ;
    __syncthreads();
    if (it + 1 < nqt) stage(buf ^ 1, qt0 + CQ);
    if (qt0 + CQ - 1 < kw || kw >= S) continue;  // every query of the tile precedes this wave's keys
    const bf16_t* Qt = Qs[buf];
    const bf16_t* dOt = dOs[buf];
    const bool diag = qt0 < kw + 31;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      f32x16 sacc = f32x16{}, pacc = f32x16{};
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        sacc = mfma32(tile_row8<D>(Qt, qb * 32 + r32, 16 * kk + 8 * h),
                      tile_row8<D>(Kw, 32 * w + r32, 16 * kk + 8 * h), sacc);
        pacc = mfma32(tile_row8<D>(dOt, qb * 32 + r32, 16 * kk + 8 * h), vreg[kk], pacc);
        if (kk % 4 == 3) __builtin_amdgcn_sched_barrier(0);  // bound the operand loads in flight
      }
      bf16x8 pb[2], db[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float pf[8], df[8];
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const int qg = qb * 32 + 16 * u + 8 * g + 4 * h;  // rows qg .. qg + 3 in the tile
          const float4 l4 = *reinterpret_cast<const float4*>(&lse_s[buf][qg]);
          const float4 d4 = *reinterpret_cast<const float4*>(&dlt_s[buf][qg]);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
          const float dv4[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int i = 8 * u + 4 * g + j;
            float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[i], sl2, -lv[j]));
            if (diag && mykey > qt0 + qg + j) pv = 0.0f;
            pf[4 * g + j] = pv;
            df[4 * g + j] = pv * (pacc[i] - dv4[j]);
          }
        }
        pb[u] = cvt8(pf);
        db[u] = cvt8(df);
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the operand loads of each phase together
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int d = 0; d < D / 32; ++d) {
          dvacc[d] = mfma32(pb[u], tile_tr8<D>(dOt, qb * 32 + 16 * u, 32 * d, lane), dvacc[d]);
          dkacc[d] = mfma32(db[u], tile_tr8<D>(Qt, qb * 32 + 16 * u, 32 * d, lane), dkacc[d]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
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
    if (s.D == 128) hipLaunchKernelGGL(sdpa_fwd_bf16<128>, grid, dim3(64 * FW), 0, st, q, k, v, (bf16_t*)os, lse, s.S, sl2);
    else hipLaunchKernelGGL(sdpa_fwd_bf16<64>, grid, dim3(64 * FW), 0, st, q, k, v, (bf16_t*)os, lse, s.S, sl2);
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
      hipLaunchKernelGGL(sdpa_bwd_dkdv_bf16<128>, gk, dim3(64 * KWV), 0, st, q, k, v, g, lse, delta, (bf16_t*)dks, (bf16_t*)dvs, s.S, sl2, s.scale);
      hipLaunchKernelGGL(sdpa_bwd_dq_bf16<128>, gq, dim3(64 * QW), 0, st, q, k, v, g, lse, delta, (bf16_t*)dqs, s.S, sl2, s.scale);
    } else {
      hipLaunchKernelGGL(sdpa_bwd_dkdv_bf16<64>, gk, dim3(64 * KWV), 0, st, q, k, v, g, lse, delta, (bf16_t*)dks, (bf16_t*)dvs, s.S, sl2, s.scale);
      hipLaunchKernelGGL(sdpa_bwd_dq_bf16<64>, gq, dim3(64 * QW), 0, st, q, k, v, g, lse, delta, (bf16_t*)dqs, s.S, sl2, s.scale);
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
