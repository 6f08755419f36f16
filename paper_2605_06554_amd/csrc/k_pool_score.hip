// k_pool_score.hip -- pyramid pooling (Sec. 3.3, Eq. pool) and norm scores (Sec. 3.4,
// Eqs. score-base and score-pool) in one streaming pass over Q, K and V.
//
// One launch covers the three tensors: the head slots of Q (Hq), K (Hkv) and V (Hkv) form one
// list, and a workgroup owns a range of base rows for a chunk of that list. The range is a
// multiple of p^(L-1), so every pyramid window lies inside it. Each thread owns one 16-byte
// column chunk of one head and walks the rows in order with an fp64 running sum per level.
// When a level-l window closes, its sum times 1/p^l (exact for p a power of two; otherwise a
// division) is rounded once to the storage dtype and written, then added into the level-(l+1)
// sum. Window closings are tracked with per-level counters, which are the same for the whole
// workgroup, so no per-row division is needed. Sums of bf16 (or fp32) values in fp64 are exact
// for the data this path sees, so the stored mean is the correctly rounded exact mean.
//
// Scores (Q and K only): rows are staged through LDS so that one thread computes one row's
// squared norm sequentially (c ascending, fp64; 16-byte LDS reads), takes the correctly rounded
// fp64 sqrt and rounds to fp32. One thread per head slot (the block's last threads) max-pools
// the level-0 scores up the levels, one step behind: a step's cascade runs while the next
// step's norms are computed (two LDS score buffers).
#include "lh_common.h"

namespace lh {

constexpr int kPoolRB = 8;  // rows staged per step

struct PoolTensor {
  const void* x;  // [B, N, H, D]
  void* pyr;      // [B, R, H, D] or null
  float* s;       // [B, H, Ptot] or null
  int32_t H;
};

struct PoolArgs {
  PoolTensor t[3];
  int32_t slot1, slot2, nslots;  // head slots: [0, slot1) tensor 0, [slot1, slot2) tensor 1, rest 2
  int64_t N, R, Ptot;
  int32_t D, HW, WR, p, cpr_shift;
  int32_t epb[16];  // WR / p^l: level-l windows per workgroup
  int64_t off[17];
  double inv[16];  // 1 / p^l (exact when p is a power of two)
  double pwd[16];  // p^l
  int32_t pow2;
};

template <typename T>
__device__ __forceinline__ void store_mean(T* dst, const double* acc, double inv, double w, bool pow2) {
  constexpr int CH = 16 / sizeof(T);
  if constexpr (sizeof(T) == 2) {
    uint32_t wd[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const double lo = pow2 ? acc[2 * c] * inv : acc[2 * c] / w;
      const double hi = pow2 ? acc[2 * c + 1] * inv : acc[2 * c + 1] / w;
      wd[c] = (uint32_t)f64_to_bf16(lo) | ((uint32_t)f64_to_bf16(hi) << 16);
    }
    u32x4 o;
    o.x = wd[0], o.y = wd[1], o.z = wd[2], o.w = wd[3];
    store16_nt(dst, o);
  } else {
    float o[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) o[c] = (float)(pow2 ? acc[c] * inv : acc[c] / w);
    store_chunk_f32(reinterpret_cast<float*>(dst), o);
  }
}

// Max-pool cascade of nrc level-0 scores (rows in order) of head slot g2 of the block: the
// level-l window that a score completes is written, and its max carried one level up. The
// running state (mx, scnt, sent) carries over between calls.
template <int L, int LA>
__device__ __forceinline__ void cascade_rows(const PoolArgs& a, const float* nrm, int nrc, int col, int g2,
                                             int64_t b, float (&mx)[LA], int (&scnt)[LA + 1], int (&sent)[LA]) {
  const int t2i = g2 < a.slot1 ? 0 : g2 < a.slot2 ? 1 : 2;
  float* sb = a.t[t2i].s;
  if (!sb) return;
  const int h2 = g2 - (t2i == 0 ? 0 : t2i == 1 ? a.slot1 : a.slot2);
  float* srow = sb + (b * a.t[t2i].H + h2) * a.Ptot;
  for (int r = 0; r < nrc; ++r) {
    const float s0 = nrm[r * a.HW + col];
    mx[1] = mx[1] > s0 ? mx[1] : s0;
    ++scnt[1];
#pragma unroll
    for (int l = 1; l < L; ++l) {
      if (scnt[l] != a.p) break;
      scnt[l] = 0;
      srow[a.off[l] + (int64_t)blockIdx.x * a.epb[l] + sent[l]] = mx[l];
      ++sent[l];
      if (l + 1 < L) {
        const int ln = l + 1 < L ? l + 1 : l;
        mx[ln] = mx[ln] > mx[l] ? mx[ln] : mx[l];
        ++scnt[ln];
      }
      mx[l] = 0.0f;
    }
  }
}

// PF > 0: p == PF is known at compile time and kPoolRB is a multiple of it, so level-1
// windows close at fixed positions of every step. PF == 0: any p, checked row by row.
template <typename T, int L, int PF>
__global__ void __launch_bounds__(256) pool_score_kernel(PoolArgs a) {
  constexpr int CH = 16 / sizeof(T);
  constexpr int LA = L > 1 ? L : 2;
  static_assert(PF == 0 || kPoolRB % PF == 0, "steps must hold whole level-1 windows");
  extern __shared__ __align__(16) unsigned char smem[];
  const int D = a.D;
  const int tid = threadIdx.x;
  const int hs = tid >> a.cpr_shift, cc = tid & ((1 << a.cpr_shift) - 1);
  const int gs = blockIdx.y * a.HW + hs;  // global head slot
  const bool active = gs < a.nslots;
  const int ti = gs < a.slot1 ? 0 : gs < a.slot2 ? 1 : 2;
  const int h = gs - (ti == 0 ? 0 : ti == 1 ? a.slot1 : a.slot2);
  const PoolTensor& t0 = a.t[0];
  const PoolTensor& t1 = a.t[1];
  const PoolTensor& t2 = a.t[2];
  const T* x = reinterpret_cast<const T*>(ti == 0 ? t0.x : ti == 1 ? t1.x : t2.x);
  T* pyr = reinterpret_cast<T*>(ti == 0 ? t0.pyr : ti == 1 ? t1.pyr : t2.pyr);
  float* srow_base = ti == 0 ? t0.s : ti == 1 ? t1.s : t2.s;
  const int H = ti == 0 ? t0.H : ti == 1 ? t1.H : t2.H;
  const int64_t b = blockIdx.z;
  const int64_t j0 = (int64_t)blockIdx.x * a.WR;
  const int nrows = (int)((a.N - j0) < a.WR ? (a.N - j0) : a.WR);
  const bool do_pool = L > 1 && active && pyr != nullptr;
  const bool any_score = a.t[0].s != nullptr || a.t[1].s != nullptr || a.t[2].s != nullptr;

  // LDS: staged rows [RB][HW][D + pad] of T, then two buffers of level-0 scores [RB][HW].
  // rows padded by 16 bytes: 16-byte aligned, and the norm threads (one row each, consecutive
  // rows) read 16-byte chunks without bank conflicts
  const int rowT = D + 16 / (int)sizeof(T);
  T* tile = reinterpret_cast<T*>(smem);
  float* nrm_buf = reinterpret_cast<float*>(smem + (size_t)kPoolRB * a.HW * rowT * sizeof(T));
  // the cascade threads: the block's last HW threads, one per head slot
  const int ct = tid - ((int)blockDim.x - a.HW);
  const bool cthread = L > 1 && ct >= 0 && (int)blockIdx.y * a.HW + ct < a.nslots;
  int step = 0, nr_prev = 0;

  const T* xrow = x + ((b * a.N + j0) * H + h) * D + cc * CH;
  const int64_t xstride = (int64_t)H * D;
  T* prow[LA];
#pragma unroll
  for (int l = 1; l < L; ++l)
    prow[l] = pyr ? pyr + ((b * a.R + (a.off[l] - a.N) + (int64_t)blockIdx.x * a.epb[l]) * H + h) * D + cc * CH
                  : nullptr;
  const int64_t pstride = (int64_t)H * D;

  double acc[LA][CH];
#pragma unroll
  for (int l = 0; l < LA; ++l)
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[l][c] = 0.0;
  int cnt[LA + 1];  // rows (level 1) or closed windows (level l > 1) in the open level-l window
#pragma unroll
  for (int l = 0; l <= LA; ++l) cnt[l] = 0;
  // cascade state (used by the cascade threads)
  float mx[LA];
#pragma unroll
  for (int l = 0; l < LA; ++l) mx[l] = 0.0f;
  int scnt[LA + 1];
#pragma unroll
  for (int l = 0; l <= LA; ++l) scnt[l] = 0;
  int sent[LA];  // next entry index (within the workgroup) per level, for the scores
#pragma unroll
  for (int l = 0; l < LA; ++l) sent[l] = 0;

  // closes the level-1 window that just received its last row, and every window above it
  // that closes with it
  auto close_windows = [&]() {
#pragma unroll
    for (int l = 1; l < L; ++l) {
      if (l > 1 && cnt[l] != a.p) break;
      cnt[l] = 0;
      if (do_pool) {
        store_mean<T>(prow[l], acc[l], a.inv[l], a.pwd[l], a.pow2);
        prow[l] += pstride;
      }
      if (l + 1 < L) {
#pragma unroll
        for (int c = 0; c < CH; ++c) acc[l + 1 < L ? l + 1 : l][c] += acc[l][c];
        ++cnt[l + 1];
      }
#pragma unroll
      for (int c = 0; c < CH; ++c) acc[l][c] = 0.0;
    }
  };

  for (int rb = 0; rb < nrows; rb += kPoolRB) {
    const int nr = nrows - rb < kPoolRB ? nrows - rb : kPoolRB;
    // raw 16-byte chunks: converted to fp64 as they are summed (fewer live registers)
    u32x4 v[kPoolRB];
#pragma unroll
    for (int r = 0; r < kPoolRB; ++r) {
      if (r < nr && active) v[r] = load16_nt(xrow + (int64_t)(rb + r) * xstride);
      else v[r] = u32x4{0, 0, 0, 0};
    }
    if (any_score && active && srow_base) {
#pragma unroll
      for (int r = 0; r < kPoolRB; ++r)
        if (r < nr) *reinterpret_cast<u32x4*>(tile + ((size_t)r * a.HW + hs) * rowT + cc * CH) = v[r];
    }
    auto add_row = [&](const u32x4& w) {
      const uint32_t u[4] = {w.x, w.y, w.z, w.w};
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[1][2 * i] += (double)__uint_as_float(u[i] << 16);
          acc[1][2 * i + 1] += (double)__uint_as_float(u[i] & 0xffff0000u);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[1][i] += (double)__uint_as_float(u[i]);
      }
    };
    if (L > 1) {
      if constexpr (PF > 0) {
        // nr is a multiple of p here (rows per workgroup are a multiple of p^(L-1))
#pragma unroll
        for (int r = 0; r < kPoolRB; ++r) {
          if (r >= nr) break;
          add_row(v[r]);
          if (r % PF == PF - 1) close_windows();
        }
      } else {
#pragma unroll
        for (int r = 0; r < kPoolRB; ++r) {
          if (r >= nr) break;
          add_row(v[r]);
          if (++cnt[1] == a.p) close_windows();
        }
      }
    }
    if (any_score) {
      float* nrm = nrm_buf + (step & 1) * kPoolRB * a.HW;
      __syncthreads();
      // the previous step's cascade runs on the last threads while the first ones compute
      // this step's norms
      if (step > 0 && cthread)
        cascade_rows<L, LA>(a, nrm_buf + ((step - 1) & 1) * kPoolRB * a.HW, nr_prev, ct,
                            (int)blockIdx.y * a.HW + ct, b, mx, scnt, sent);
      // one thread per (row, head slot): sequential fp64 sum of squares, c ascending
      for (int e = tid; e < nr * a.HW; e += blockDim.x) {
        const int r = e / a.HW, hh = e - r * a.HW;
        const int g2 = blockIdx.y * a.HW + hh;
        if (g2 >= a.nslots) continue;
        const int t2i = g2 < a.slot1 ? 0 : g2 < a.slot2 ? 1 : 2;
        float* sb = t2i == 0 ? t0.s : t2i == 1 ? t1.s : t2.s;
        if (!sb) continue;
        const int h2 = g2 - (t2i == 0 ? 0 : t2i == 1 ? a.slot1 : a.slot2);
        const int H2 = t2i == 0 ? t0.H : t2i == 1 ? t1.H : t2.H;
        const T* row = tile + ((size_t)r * a.HW + hh) * rowT;
        double s2 = 0.0;
        for (int c = 0; c < D; c += CH) {  // 16-byte reads, elements in ascending order
          const u32x4 w4 = *reinterpret_cast<const u32x4*>(row + c);
          const uint32_t u[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if constexpr (sizeof(T) == 2) {
              const double lo = (double)__uint_as_float(u[e] << 16);
              const double hi = (double)__uint_as_float(u[e] & 0xffff0000u);
              s2 += lo * lo;  // squares of bf16 values are exact in fp64
              s2 += hi * hi;
            } else {
              const double x = (double)__uint_as_float(u[e]);
              s2 += x * x;  // squares of fp32 values are exact in fp64
            }
          }
        }
        const float sc = (float)sqrt(s2);
        nrm[r * a.HW + hh] = sc;
        sb[(b * H2 + h2) * a.Ptot + j0 + rb + r] = sc;
      }
      // this step's scores are complete and the previous cascade is done; `tile` may be
      // rewritten, and the next step's cascade reads this step's score buffer
      __syncthreads();
      nr_prev = nr;
    }
    ++step;
  }
  if (any_score && step > 0 && cthread)
    cascade_rows<L, LA>(a, nrm_buf + ((step - 1) & 1) * kPoolRB * a.HW, nr_prev, ct, (int)blockIdx.y * a.HW + ct,
                        b, mx, scnt, sent);
}

template <typename T, int L>
static void launch_L(const PoolArgs& a, dim3 grid, dim3 block, size_t shm, hipStream_t st) {
  if (a.p == 4 && L > 1) hipLaunchKernelGGL((pool_score_kernel<T, L, 4>), grid, block, shm, st, a);
  else if (a.p == 2 && L > 1) hipLaunchKernelGGL((pool_score_kernel<T, L, 2>), grid, block, shm, st, a);
  else hipLaunchKernelGGL((pool_score_kernel<T, L, 0>), grid, block, shm, st, a);
}

template <typename T>
static hipError_t launch_T(const LhShape& s, PoolArgs& a, hipStream_t st) {
  const int CH = 16 / sizeof(T);
  const int CPR = s.D / CH;
  int cs = 0;
  while ((1 << cs) < CPR) ++cs;
  a.cpr_shift = cs;
  a.HW = a.nslots < 256 / CPR ? a.nslots : 256 / CPR;
  if (a.HW < 1) a.HW = 1;
  // rows per workgroup: the smallest multiple of p^(L-1) that is >= 64
  int64_t W = s.P;
  while (W < 64) W += s.P;
  a.WR = (int32_t)W;
  for (int l = 0; l < 16; ++l) a.epb[l] = l < s.L ? (int32_t)(W / s.pw[l]) : 0;
  dim3 grid((unsigned)((s.N + W - 1) / W), (unsigned)((a.nslots + a.HW - 1) / a.HW), (unsigned)s.B);
  dim3 block((unsigned)(a.HW * CPR));
  const bool score = a.t[0].s || a.t[1].s || a.t[2].s;
  const int rowT = s.D + 16 / (int)sizeof(T);
  size_t shm = score ? (size_t)kPoolRB * a.HW * rowT * sizeof(T) + 2 * (size_t)kPoolRB * a.HW * sizeof(float) : 0;
  switch (s.L) {
    case 1: launch_L<T, 1>(a, grid, block, shm, st); break;
    case 2: launch_L<T, 2>(a, grid, block, shm, st); break;
    case 3: launch_L<T, 3>(a, grid, block, shm, st); break;
    case 4: launch_L<T, 4>(a, grid, block, shm, st); break;
    case 5: launch_L<T, 5>(a, grid, block, shm, st); break;
    case 6: launch_L<T, 6>(a, grid, block, shm, st); break;
    case 7: launch_L<T, 7>(a, grid, block, shm, st); break;
    case 8: launch_L<T, 8>(a, grid, block, shm, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace lh

using namespace lh;

hipError_t lh_launch_pool_score(const LhShape& s, const void* q, const void* k, const void* v,
                                void* qpyr, void* kpyr, void* vpyr, float* s_qk, float* s_kq,
                                hipStream_t st) {
  PoolArgs a = {};
  const PoolTensor jobs[3] = {{q, qpyr, s_qk, s.Hq}, {k, kpyr, s_kq, s.Hkv}, {v, vpyr, nullptr, s.Hkv}};
  int n = 0;
  for (const PoolTensor& j : jobs) {
    PoolTensor t = j;
    if (s.L == 1) t.pyr = nullptr;
    if (!t.x || (!t.pyr && !t.s)) continue;
    a.t[n++] = t;
  }
  if (n == 0) return hipSuccess;
  for (int i = n; i < 3; ++i) a.t[i] = PoolTensor{nullptr, nullptr, nullptr, 0};
  a.slot1 = a.t[0].H;
  a.slot2 = a.slot1 + a.t[1].H;
  a.nslots = a.slot2 + a.t[2].H;
  a.N = s.N;
  a.R = s.R;
  a.Ptot = s.Ptot;
  a.D = s.D;
  a.p = s.p;
  for (int l = 0; l < 16; ++l) {
    a.inv[l] = l < s.L ? 1.0 / (double)s.pw[l] : 0.0;
    a.pwd[l] = l < s.L ? (double)s.pw[l] : 1.0;
  }
  a.pow2 = (s.p & (s.p - 1)) == 0;
  for (int l = 0; l < 17; ++l) a.off[l] = s.off[l];
  return s.dtype == LH_BF16 ? launch_T<bf16_t>(s, a, st) : launch_T<float>(s, a, st);
}
