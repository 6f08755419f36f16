// k_pool_score.hip -- pyramid pooling (Sec. 3.3, Eq. pool) and norm scores (Sec. 3.4,
// Eqs. score-base and score-pool) in one streaming pass over a [B, N, H, D] tensor.
//
// One workgroup owns a range of base rows (a multiple of p^(L-1), so every pyramid window lies
// inside it) for a chunk of heads. Each thread owns one 16-byte column chunk of one head and
// walks the rows in order, keeping an fp64 running sum per level: when a level-l window
// closes, its sum is divided by p^l, rounded once to the storage dtype and written, and then
// added into the level-(l+1) sum. Sums of bf16 (or fp32) values in fp64 are exact for the
// data this path sees, so the stored mean is the correctly rounded exact mean.
//
// Scores: rows are staged through LDS so that one thread computes one row's squared norm
// sequentially (c ascending, fp64), takes the correctly rounded fp64 sqrt and rounds to fp32.
// One thread per head then max-pools the level-0 scores up the levels, in row order.
#include "lh_common.h"

namespace lh {

constexpr int kPoolRB = 8;  // rows staged per step

struct PoolArgs {
  const void* x;  // [B, N, H, D]
  void* pyr;      // [B, R, H, D] or null
  float* s;       // [B, H, Ptot] or null
  int64_t N, R, Ptot, WR;
  int32_t H, D, HW;
  int64_t pw[16];
  int64_t off[17];
  double inv[16];  // 1 / p^l, used only when it is exact (p a power of two)
  int32_t pow2;
};

template <typename T, int L>
__global__ void __launch_bounds__(1024) pool_score_kernel(PoolArgs a) {
  constexpr int CH = 16 / sizeof(T);  // elements per 16-byte chunk
  extern __shared__ __align__(16) unsigned char smem[];
  const int D = a.D;
  const int CPR = D / CH;
  const int tid = threadIdx.x;
  const int hc = tid / CPR, cc = tid % CPR;
  const int h = blockIdx.y * a.HW + hc;
  const bool active = h < a.H;
  const int64_t b = blockIdx.z;
  const int64_t j0 = (int64_t)blockIdx.x * a.WR;
  int64_t j1 = j0 + a.WR;
  if (j1 > a.N) j1 = a.N;
  const T* x = reinterpret_cast<const T*>(a.x);
  T* pyr = reinterpret_cast<T*>(a.pyr);
  const bool do_pool = (pyr != nullptr) && L > 1;
  const bool do_score = a.s != nullptr;

  // LDS: staged rows [RB][HW][D + pad] of T, then level-0 scores [RB][HW].
  const int rowT = D + 8 / (int)sizeof(T);  // +8 bytes keeps the per-row norm reads conflict-free
  T* tile = reinterpret_cast<T*>(smem);
  float* nrm = reinterpret_cast<float*>(smem + (size_t)kPoolRB * a.HW * rowT * sizeof(T));

  double acc[L > 1 ? L : 2][CH];
#pragma unroll
  for (int l = 0; l < (L > 1 ? L : 2); ++l)
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[l][c] = 0.0;
  float mx[L > 1 ? L : 2];
#pragma unroll
  for (int l = 0; l < (L > 1 ? L : 2); ++l) mx[l] = 0.0f;

  for (int64_t jb = j0; jb < j1; jb += kPoolRB) {
    const int nr = (int)((j1 - jb) < kPoolRB ? (j1 - jb) : kPoolRB);
    float v[kPoolRB][CH];
#pragma unroll
    for (int r = 0; r < kPoolRB; ++r) {
      if (r < nr && active) {
        load_chunk<T>(x + ((b * a.N + jb + r) * a.H + h) * D + cc * CH, v[r]);
      } else {
#pragma unroll
        for (int c = 0; c < CH; ++c) v[r][c] = 0.0f;
      }
    }
    if (do_score) {
#pragma unroll
      for (int r = 0; r < kPoolRB; ++r) {
        if (r < nr && active) {
          T* dst = tile + ((size_t)r * a.HW + hc) * rowT + cc * CH;
          // re-store the raw values (exact: they came from T)
          store_chunk<T>(dst, v[r]);
        }
      }
    }
    if (do_pool && active) {
#pragma unroll
      for (int r = 0; r < kPoolRB; ++r) {
        if (r < nr) {
          const int64_t j = jb + r;
#pragma unroll
          for (int c = 0; c < CH; ++c) acc[1][c] += (double)v[r][c];
#pragma unroll
          for (int l = 1; l < L; ++l) {
            if ((j + 1) % a.pw[l] != 0) break;
            const int64_t i = (j + 1) / a.pw[l] - 1;
            const double w = (double)a.pw[l], inv = a.inv[l];
            // mean = sum / p^l, rounded once; the reciprocal is exact when p is a power of two
            auto mean = [&](double x) { return a.pow2 ? x * inv : x / w; };
            T* dst = pyr + ((b * a.R + (a.off[l] - a.N) + i) * a.H + h) * D + cc * CH;
            if constexpr (sizeof(T) == 2) {
              uint32_t wd[4];
#pragma unroll
              for (int c = 0; c < 4; ++c)
                wd[c] = (uint32_t)f64_to_bf16(mean(acc[l][2 * c])) |
                       ((uint32_t)f64_to_bf16(mean(acc[l][2 * c + 1])) << 16);
              u32x4 o;
              o.x = wd[0], o.y = wd[1], o.z = wd[2], o.w = wd[3];
              *reinterpret_cast<u32x4*>(dst) = o;
            } else {
              float o[CH];
#pragma unroll
              for (int c = 0; c < CH; ++c) o[c] = (float)mean(acc[l][c]);
              store_chunk_f32(reinterpret_cast<float*>(dst), o);
            }
            if (l + 1 < L) {
#pragma unroll
              for (int c = 0; c < CH; ++c) acc[l + 1 < L ? l + 1 : l][c] += acc[l][c];
            }
#pragma unroll
            for (int c = 0; c < CH; ++c) acc[l][c] = 0.0;
          }
        }
      }
    }
    if (do_score) {
      __syncthreads();
      // one thread per (row, head): sequential fp64 sum of squares, c ascending
      for (int e = tid; e < nr * a.HW; e += blockDim.x) {
        const int r = e / a.HW, hh = e % a.HW;
        if (blockIdx.y * a.HW + hh >= a.H) continue;
        const T* row = tile + ((size_t)r * a.HW + hh) * rowT;
        double s2 = 0.0;
        for (int c = 0; c < D; ++c) {
          const double t = (double)Elem<T>::load(row + c);
          s2 += t * t;
        }
        const float sc = (float)sqrt(s2);
        nrm[r * a.HW + hh] = sc;
        a.s[((int64_t)b * a.H + blockIdx.y * a.HW + hh) * a.Ptot + jb + r] = sc;
      }
      __syncthreads();
      // max-pool cascade: one thread per head, rows in order
      if (tid < a.HW && L > 1 && blockIdx.y * a.HW + tid < a.H) {
        const int hh = tid;
        float* srow = a.s + ((int64_t)b * a.H + blockIdx.y * a.HW + hh) * a.Ptot;
        for (int r = 0; r < nr; ++r) {
          const int64_t j = jb + r;
          const float s0 = nrm[r * a.HW + hh];
          mx[1] = mx[1] > s0 ? mx[1] : s0;
#pragma unroll
          for (int l = 1; l < L; ++l) {
            if ((j + 1) % a.pw[l] != 0) break;
            const int64_t i = (j + 1) / a.pw[l] - 1;
            srow[a.off[l] + i] = mx[l];
            if (l + 1 < L) {
              const int ln = l + 1 < L ? l + 1 : l;
              mx[ln] = mx[ln] > mx[l] ? mx[ln] : mx[l];
            }
            mx[l] = 0.0f;
          }
        }
      }
      // the next step rewrites `tile` only after every thread passed the barrier above, and
      // `nrm` only after the next step's first barrier, which the cascade thread reaches last
    }
  }
}

template <typename T, int L>
static hipError_t launch_one(const LhShape& s, const void* x, void* pyr, float* sc, int H,
                             hipStream_t st) {
  PoolArgs a;
  a.x = x;
  a.pyr = pyr;
  a.s = sc;
  a.N = s.N;
  a.R = s.R;
  a.Ptot = s.Ptot;
  a.H = H;
  a.D = s.D;
  const int CH = 16 / sizeof(T);
  const int CPR = s.D / CH;
  a.HW = H < 256 / CPR ? H : 256 / CPR;
  if (a.HW < 1) a.HW = 1;
  int64_t P = s.P;
  a.WR = P >= 64 ? P : P * ((64 + P - 1) / P);
  for (int l = 0; l < 16; ++l) {
    a.pw[l] = s.pw[l];
    a.inv[l] = l < s.L ? 1.0 / (double)s.pw[l] : 0.0;
  }
  a.pow2 = (s.p & (s.p - 1)) == 0;
  for (int l = 0; l < 17; ++l) a.off[l] = s.off[l];
  dim3 grid((unsigned)((s.N + a.WR - 1) / a.WR), (unsigned)((H + a.HW - 1) / a.HW), (unsigned)s.B);
  dim3 block((unsigned)(a.HW * CPR));
  const int rowT = s.D + 8 / (int)sizeof(T);
  size_t shm = sc ? (size_t)kPoolRB * a.HW * rowT * sizeof(T) + (size_t)kPoolRB * a.HW * sizeof(float) : 0;
  hipLaunchKernelGGL((pool_score_kernel<T, L>), grid, block, shm, st, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_T(const LhShape& s, const void* x, void* pyr, float* sc, int H, hipStream_t st) {
  switch (s.L) {
    case 1: return launch_one<T, 1>(s, x, pyr, sc, H, st);
    case 2: return launch_one<T, 2>(s, x, pyr, sc, H, st);
    case 3: return launch_one<T, 3>(s, x, pyr, sc, H, st);
    case 4: return launch_one<T, 4>(s, x, pyr, sc, H, st);
    case 5: return launch_one<T, 5>(s, x, pyr, sc, H, st);
    case 6: return launch_one<T, 6>(s, x, pyr, sc, H, st);
    case 7: return launch_one<T, 7>(s, x, pyr, sc, H, st);
    case 8: return launch_one<T, 8>(s, x, pyr, sc, H, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace lh

using namespace lh;

hipError_t lh_launch_pool_score(const LhShape& s, const void* q, const void* k, const void* v,
                                void* qpyr, void* kpyr, void* vpyr, float* s_qk, float* s_kq,
                                hipStream_t st) {
  hipError_t e = hipSuccess;
  const bool bf = s.dtype == LH_BF16;
  struct Job {
    const void* x;
    void* pyr;
    float* sc;
    int H;
  } jobs[3] = {{q, qpyr, s_qk, s.Hq}, {k, kpyr, s_kq, s.Hkv}, {v, vpyr, nullptr, s.Hkv}};
  for (const Job& j : jobs) {
    if (!j.x || (!j.pyr && !j.sc)) continue;
    void* pyr = s.L > 1 ? j.pyr : nullptr;
    if (!pyr && !j.sc) continue;
    e = bf ? launch_T<bf16_t>(s, j.x, pyr, j.sc, j.H, st) : launch_T<float>(s, j.x, pyr, j.sc, j.H, st);
    if (e != hipSuccess) return e;
  }
  return e;
}
