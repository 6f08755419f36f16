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
// chunk so that rows are read and written with full 16-byte vector accesses. Row and entry
// indices are 32-bit (the library rejects pyramids of 2^31 entries or more); element offsets
// are 64-bit.
//
// Runs (scatter, gather_bwd). A thread handles a run of p consecutive base positions. The run
// is aligned to p and p^l is a multiple of p, so the level-l entry (l >= 1) is the same for the
// whole run: its row is read once per run, and only level 0 is looked up per position. Run c
// covers j = c p + r - 1 (scatter, whose ranges are shifted by one) or j = c p + r
// (gather_bwd), r = 0..p-1, and its level-l entry index is floor(c / p^(l-1)), minus one for
// the scatter.
//
// XCD-aware order. Workgroups go round-robin to the 8 XCDs, each with its own L2, in order of
// their linear id. Neighbouring runs share their coarse rows, so the run index is remapped to
// give every XCD one contiguous eighth of the runs.
#include "lh_common.h"

#ifndef LH_RUN_BS
// Threads per workgroup of the run kernels (scatter, gather adjoint): up to 512, so that at
// D = 128 in bf16 one workgroup writes whole 8 KB output rows of 32 heads. Measured against
// 256 at N = 262,144 with 32 query heads: scatter 0.551 -> 0.513 ms, the dQ adjoint -2.5%; the
// scatter adjoint (its own launcher) was slower with 512 and keeps 256.
#define LH_RUN_BS 512
#endif
#ifndef LH_GBWD_GB
#define LH_GBWD_GB 4  // gather+pool adjoint: query heads whose loads are issued together
#endif

namespace lh {

// With gridDim.x a multiple of 8, blockIdx.x % 8 is the XCD of the workgroup; XCD x gets the
// x-th contiguous eighth of [0, nx).
__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t bx, uint32_t nx) {
  return (bx & 7u) * (nx >> 3) + (bx >> 3);
}

template <typename T>
__device__ __forceinline__ void add_chunk(float* acc, const u32x4& w) {
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += __uint_as_float(u[i] << 16);
      acc[2 * i + 1] += __uint_as_float(u[i] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] += __uint_as_float(u[i]);
  }
}

template <typename T>
__device__ __forceinline__ void add_chunk_scaled(float* acc, const u32x4& w, float s) {
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += __uint_as_float(u[i] << 16) * s;
      acc[2 * i + 1] += __uint_as_float(u[i] & 0xffff0000u) * s;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] += __uint_as_float(u[i]) * s;
  }
}

__device__ __forceinline__ u32x4 load_raw(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// ---------------------------------------------------------------- gather

struct GatherArgs {
  const void *q, *k, *v, *qp, *kp, *vp;
  const int32_t* idx;
  void *qs, *ks, *vs;
  int64_t N, R, S;
  int32_t Hq, Hkv, G, D, cpr_shift, rows_per_block;
  int32_t Hs, Gq;  // selection heads, query heads per selection head
};

template <typename T>
__global__ void __launch_bounds__(256) gather_kernel(GatherArgs a) {
  constexpr int CH = 16 / sizeof(T);
  const int cc = threadIdx.x & ((1 << a.cpr_shift) - 1);
  const int64_t m = (int64_t)blockIdx.x * a.rows_per_block + (threadIdx.x >> a.cpr_shift);
  if (m >= a.S) return;
  const int64_t bh = blockIdx.y;
  const int hq = (int)(bh % a.Hq);
  const int64_t b = bh / a.Hq;
  const int g = hq / a.G;
  // rows of the selection head of hq; K~ and V~ are written once per selection head (by its
  // first query head), Q~ per query head
  const int64_t bs = b * a.Hs + hq / a.Gq;
  const bool kv_out = hq % a.Gq == 0;
  const int64_t id = a.idx[bs * a.S + m];
  const int64_t o = (bh * a.S + m) * a.D + cc * CH;
  const int64_t okv = (bs * a.S + m) * a.D + cc * CH;
  if (id < 0 || id >= a.N + a.R) {  // not a pyramid id: zero row, never an out-of-range read
    const u32x4 z{0, 0, 0, 0};
    store16_nt(reinterpret_cast<T*>(a.qs) + o, z);
    if (kv_out) {
      store16_nt(reinterpret_cast<T*>(a.ks) + okv, z);
      store16_nt(reinterpret_cast<T*>(a.vs) + okv, z);
    }
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
  const u32x4 xq = load16_nt(sq + cc * CH);  // a query row is gathered once; K, V rows by every head of the group
  store16_nt(reinterpret_cast<T*>(a.qs) + o, xq);
  if (kv_out) {
    const u32x4 xk = load_raw(sk + cc * CH);
    const u32x4 xv = load_raw(sv + cc * CH);
    store16_nt(reinterpret_cast<T*>(a.ks) + okv, xk);
    store16_nt(reinterpret_cast<T*>(a.vs) + okv, xv);
  }
}

// ---------------------------------------------------------------- scatter and gather_bwd

struct RunArgs {
  const void* src;      // [B, Hq, S, D] gathered rows
  const int32_t* slot;  // [B, Hq, Ptot]
  void* dst;            // [B, N, H, D]
  int64_t Ptot;
  int32_t N, S, D, nruns, run;        // run = positions per run: p (1 when L = 1)
  int32_t Hq, H, Gs, HC, cpr_shift;   // output head h sums source heads h Gs .. h Gs + Gs - 1
  int32_t Hsrc, Hslot, sdiv;          // heads of src and of slot; source head x uses slot head x / sdiv
  int32_t pshift;                     // log2 p when p is a power of two, else -1
  int32_t pw[16];                     // p^l
  int32_t off[17];                    // flattened id of entry (l, 0)
  int32_t nrow[16];                   // N / p^l
  int32_t vec_slots;                  // Ptot % 4 == 0: a head's slot row is 16-byte aligned
  float inv[16];                      // 1 / p^l
  int32_t rpb;                        // runs per workgroup of a packed launch (else 1)
};

// Row 0 of source head x of batch b in src, and its slot row.
__device__ __forceinline__ int64_t src_head(const RunArgs& a, int64_t b, int x) { return b * a.Hsrc + x; }
__device__ __forceinline__ const int32_t* slot_row(const RunArgs& a, int64_t b, int x) {
  return a.slot + (b * a.Hslot + x / a.sdiv) * a.Ptot;
}

// Level-l entry (l >= 1) shared by every position of run c: floor(c / p^(l-1)).
__device__ __forceinline__ int32_t run_entry(const RunArgs& a, uint32_t c, int l) {
  return (int32_t)(a.pshift >= 0 ? (c >> (a.pshift * (l - 1))) : (c / (uint32_t)a.pw[l - 1]));
}

// o[b, j, hq, :]. Sum order: levels L-1 .. 1, then level 0; one rounding.
// PU > 0: runs of at most PU positions, all lookups and loads of a run issued together.
template <typename T, int L, int PU>
__global__ void __launch_bounds__(LH_RUN_BS) scatter_kernel(RunArgs a) {
  constexpr int CH = 16 / sizeof(T);
  const uint32_t c = xcd_contiguous(blockIdx.x, gridDim.x);
  const int hc = blockIdx.y * blockDim.x + threadIdx.x;
  if (c >= (uint32_t)a.nruns || hc >= a.HC) return;
  const int hq = hc >> a.cpr_shift, cc = hc & ((1 << a.cpr_shift) - 1);
  const int64_t b = blockIdx.z;
  const int32_t* sl = slot_row(a, b, hq);
  const T* src = reinterpret_cast<const T*>(a.src) + src_head(a, b, hq) * a.S * a.D + cc * CH;
  float acc[CH];
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = 0.0f;
  if constexpr (L > 1) {
    int32_t m[L];
#pragma unroll
    for (int l = L - 1; l >= 1; --l) {
      const int32_t i = run_entry(a, c, l) - 1;
      m[l] = i >= 0 ? sl[a.off[l] + i] : -1;
    }
    u32x4 v[L];
#pragma unroll
    for (int l = L - 1; l >= 1; --l)
      v[l] = (uint32_t)m[l] < (uint32_t)a.S ? load_raw(src + (int64_t)m[l] * a.D) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int l = L - 1; l >= 1; --l) add_chunk<T>(acc, v[l]);
  }
  // level 0: position j takes entry (0, j)
  T* dst = reinterpret_cast<T*>(a.dst) + ((b * a.N) * a.H + hq) * (int64_t)a.D + cc * CH;
  const int64_t dstride = (int64_t)a.H * a.D;
  const int32_t jbase = (int32_t)(c * (uint32_t)a.run) - 1;
  if constexpr (PU > 0) {
    int32_t m0[PU];
#pragma unroll
    for (int r = 0; r < PU; ++r) {
      const int32_t j = jbase + r;
      m0[r] = (r < a.run && j >= 0 && j < a.N) ? sl[j] : -1;
    }
    u32x4 v0[PU];
#pragma unroll
    for (int r = 0; r < PU; ++r)
      v0[r] = (uint32_t)m0[r] < (uint32_t)a.S ? load_raw(src + (int64_t)m0[r] * a.D) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int r = 0; r < PU; ++r) {
      const int32_t j = jbase + r;
      if (r < a.run && j >= 0 && j < a.N) {
        float o[CH];
#pragma unroll
        for (int e = 0; e < CH; ++e) o[e] = acc[e];
        add_chunk<T>(o, v0[r]);
        store_chunk<T>(dst + (int64_t)j * dstride, o);
      }
    }
  } else {
    for (int r = 0; r < a.run; ++r) {
      const int32_t j = jbase + r;
      if (j < 0 || j >= a.N) continue;
      const int32_t m0 = sl[j];
      float o[CH];
#pragma unroll
      for (int e = 0; e < CH; ++e) o[e] = acc[e];
      if ((uint32_t)m0 < (uint32_t)a.S) add_chunk<T>(o, load_raw(src + (int64_t)m0 * a.D));
      store_chunk<T>(dst + (int64_t)j * dstride, o);
    }
  }
}

// dst[b, j, h, :] = sum over the Gs query heads g of the group and the levels l of
// src_g[slot_g(l, floor(j/p^l))] / p^l. Sum order: levels L-1 .. 1 of every head in turn, then
// level 0 of every head in turn; one rounding.
template <typename T, int L, int PU>
__global__ void __launch_bounds__(LH_RUN_BS) gather_bwd_kernel(RunArgs a) {
  constexpr int CH = 16 / sizeof(T);
  constexpr int NP = PU > 0 ? PU : 1;
  const uint32_t c = xcd_contiguous(blockIdx.x, gridDim.x);
  const int hc = blockIdx.y * blockDim.x + threadIdx.x;
  if (c >= (uint32_t)a.nruns || hc >= a.HC) return;
  const int h = hc >> a.cpr_shift, cc = hc & ((1 << a.cpr_shift) - 1);
  const int64_t b = blockIdx.z;
  const int32_t jbase = (int32_t)(c * (uint32_t)a.run);
  int32_t ent[L > 1 ? L : 2];
#pragma unroll
  for (int l = 1; l < L; ++l) ent[l] = a.off[l] + run_entry(a, c, l);
  float acc[CH];
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = 0.0f;
  float fine[NP][CH];
#pragma unroll
  for (int r = 0; r < NP; ++r)
#pragma unroll
    for (int e = 0; e < CH; ++e) fine[r][e] = 0.0f;
  T* dst = reinterpret_cast<T*>(a.dst) + ((b * a.N) * a.H + h) * (int64_t)a.D + cc * CH;
  const int64_t dstride = (int64_t)a.H * a.D;
  for (int g = 0; g < a.Gs; ++g) {
    const int x = h * a.Gs + g;
    const int32_t* sl = slot_row(a, b, x);
    const T* src = reinterpret_cast<const T*>(a.src) + src_head(a, b, x) * a.S * a.D + cc * CH;
    int32_t m[L > 1 ? L : 2];
#pragma unroll
    for (int l = L - 1; l >= 1; --l) m[l] = sl[ent[l]];
    int32_t m0[NP];
    if constexpr (PU > 0) {
#pragma unroll
      for (int r = 0; r < PU; ++r) m0[r] = r < a.run ? sl[jbase + r] : -1;
    }
    u32x4 v[L > 1 ? L : 2];
#pragma unroll
    for (int l = L - 1; l >= 1; --l)
      v[l] = (uint32_t)m[l] < (uint32_t)a.S ? load_raw(src + (int64_t)m[l] * a.D) : u32x4{0, 0, 0, 0};
    if constexpr (PU > 0) {
      u32x4 v0[PU];
#pragma unroll
      for (int r = 0; r < PU; ++r)
        v0[r] = (uint32_t)m0[r] < (uint32_t)a.S ? load_raw(src + (int64_t)m0[r] * a.D) : u32x4{0, 0, 0, 0};
#pragma unroll
      for (int l = L - 1; l >= 1; --l) add_chunk_scaled<T>(acc, v[l], a.inv[l]);
#pragma unroll
      for (int r = 0; r < PU; ++r) add_chunk<T>(fine[r], v0[r]);
    } else {
#pragma unroll
      for (int l = L - 1; l >= 1; --l) add_chunk_scaled<T>(acc, v[l], a.inv[l]);
    }
  }
  if constexpr (PU > 0) {
#pragma unroll
    for (int r = 0; r < PU; ++r) {
      if (r < a.run) {
        float o[CH];
#pragma unroll
        for (int e = 0; e < CH; ++e) o[e] = acc[e] + fine[r][e];
        store_chunk<T>(dst + (int64_t)(jbase + r) * dstride, o);
      }
    }
  } else {
    for (int r = 0; r < a.run; ++r) {
      float o[CH];
#pragma unroll
      for (int e = 0; e < CH; ++e) o[e] = 0.0f;
      for (int g = 0; g < a.Gs; ++g) {
        const int x = h * a.Gs + g;
        const int32_t m0 = slot_row(a, b, x)[jbase + r];
        if ((uint32_t)m0 < (uint32_t)a.S)
          add_chunk<T>(o, load_raw(reinterpret_cast<const T*>(a.src) + (src_head(a, b, x) * a.S + m0) * a.D +
                                   cc * CH));
      }
#pragma unroll
      for (int e = 0; e < CH; ++e) o[e] = acc[e] + o[e];
      store_chunk<T>(dst + (int64_t)(jbase + r) * dstride, o);
    }
  }
}

// ---------------------------------------------------------------- long runs (p = 2, 4)
// A thread handles RL = P^TT positions (16 for p = 4, 8 for p = 2). Levels l >= TT have one
// entry per run, levels 1 <= l < TT one entry per sub-run of p^l positions, level 0 one per
// position. When the run lies inside level 0, its level-0 slots are read as 16-byte vectors.
// Every slot and then every row of the run is loaded before the sums, which keep the order of
// the runs of p above (levels L-1 .. 1, then level 0), so the results are the same bits.
constexpr int ipow(int p, int e) { return e == 0 ? 1 : p * ipow(p, e - 1); }
// index of the first level-l sub-run entry in the flattened list of levels 1 .. l-1
constexpr int sub_off(int P, int TT, int l) {
  int s = 0;
  for (int x = 1; x < l; ++x) s += ipow(P, TT - x);
  return s;
}

// Level-0 slots of positions j0 .. j0 + RL - 1 (-1 outside [0, N)). Positions j0 + SH .. start
// at a multiple of 4 (SH = 1 for the scatter's shifted runs). When the 4-aligned block
// [j0 + SH, j0 + SH + RL) lies inside level 0 it is read as RL / 4 16-byte vectors (the last SH
// values unused) and the first SH positions one by one.
template <int RL, int SH>
__device__ __forceinline__ void load_level0_slots(const RunArgs& a, const int32_t* sl, int32_t j0, int32_t* m0) {
  const int32_t base = j0 + SH;
  if (a.vec_slots && j0 >= 0 && base + RL <= a.N) {
    int32_t t[RL];
#pragma unroll
    for (int q = 0; q < RL / 4; ++q) {
      const int4 w = *reinterpret_cast<const int4*>(sl + base + 4 * q);
      t[4 * q] = w.x, t[4 * q + 1] = w.y, t[4 * q + 2] = w.z, t[4 * q + 3] = w.w;
    }
#pragma unroll
    for (int r = 0; r < SH; ++r) m0[r] = sl[j0 + r];
#pragma unroll
    for (int r = SH; r < RL; ++r) m0[r] = t[r - SH];
  } else {
#pragma unroll
    for (int r = 0; r < RL; ++r) {
      const int32_t j = j0 + r;
      m0[r] = (j >= 0 && j < a.N) ? sl[j] : -1;
    }
  }
}

__device__ __forceinline__ u32x4 load_entry_row(const void* src, int32_t m, int32_t S, int D, int esz) {
  return (uint32_t)m < (uint32_t)S
             ? load_raw(reinterpret_cast<const char*>(src) + (int64_t)m * D * esz)
             : u32x4{0, 0, 0, 0};
}

// Scatter over runs c of RL positions j = c RL + r - 1.
template <typename T, int L, int P, int TT>
__global__ void __launch_bounds__(LH_RUN_BS) scatter_long_kernel(RunArgs a) {
  constexpr int CH = 16 / sizeof(T);
  constexpr int RL = ipow(P, TT);
  constexpr int LS = TT < L ? TT : L;  // levels 1 .. LS-1 change inside the run
  constexpr int NSUB = sub_off(P, TT, LS);
  constexpr int NSH = L - LS;  // levels LS .. L-1: one entry per run
  const uint32_t c = xcd_contiguous(blockIdx.x, gridDim.x);
  const int hc = blockIdx.y * blockDim.x + threadIdx.x;
  if (c >= (uint32_t)a.nruns || hc >= a.HC) return;
  const int hq = hc >> a.cpr_shift, cc = hc & ((1 << a.cpr_shift) - 1);
  const int64_t b = blockIdx.z;
  const int32_t* sl = slot_row(a, b, hq);
  const T* src = reinterpret_cast<const T*>(a.src) + src_head(a, b, hq) * a.S * a.D + cc * CH;
  const int32_t j0 = (int32_t)(c * RL) - 1;
  int32_t msh[NSH > 0 ? NSH : 1], msub[NSUB > 0 ? NSUB : 1], m0[RL];
#pragma unroll
  for (int l = LS; l < L; ++l) {  // entry floor((j + 1) / p^l) - 1 = floor(c / p^(l - TT)) - 1
    const int32_t i = (int32_t)(c / (uint32_t)ipow(P, l - TT)) - 1;
    msh[l - LS] = (i >= 0 && i < a.nrow[l]) ? sl[a.off[l] + i] : -1;
  }
#pragma unroll
  for (int l = 1; l < LS; ++l)  // sub-run s: entry c p^(TT-l) + s - 1
#pragma unroll
    for (int s2 = 0; s2 < ipow(P, TT - l); ++s2) {
      const int32_t i = (int32_t)(c * ipow(P, TT - l)) + s2 - 1;
      msub[sub_off(P, TT, l) + s2] = (i >= 0 && i < a.nrow[l]) ? sl[a.off[l] + i] : -1;
    }
  load_level0_slots<RL, 1>(a, sl, j0, m0);
  u32x4 vsh[NSH > 0 ? NSH : 1], vsub[NSUB > 0 ? NSUB : 1], v0[RL];
#pragma unroll
  for (int x = 0; x < NSH; ++x) vsh[x] = load_entry_row(src, msh[x], a.S, a.D, sizeof(T));
#pragma unroll
  for (int x = 0; x < NSUB; ++x) vsub[x] = load_entry_row(src, msub[x], a.S, a.D, sizeof(T));
#pragma unroll
  for (int r = 0; r < RL; ++r) v0[r] = load_entry_row(src, m0[r], a.S, a.D, sizeof(T));
  float acc[CH];
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = 0.0f;
#pragma unroll
  for (int l = L - 1; l >= LS; --l) add_chunk<T>(acc, vsh[l - LS]);
  T* dst = reinterpret_cast<T*>(a.dst) + ((b * a.N) * a.H + hq) * (int64_t)a.D + cc * CH;
  const int64_t dstride = (int64_t)a.H * a.D;
#pragma unroll
  for (int r = 0; r < RL; ++r) {
    const int32_t j = j0 + r;
    if (j < 0 || j >= a.N) continue;
    float o[CH];
#pragma unroll
    for (int e = 0; e < CH; ++e) o[e] = acc[e];
#pragma unroll
    for (int l = LS - 1; l >= 1; --l) add_chunk<T>(o, vsub[sub_off(P, TT, l) + r / ipow(P, l)]);
    add_chunk<T>(o, v0[r]);
    store_chunk<T>(dst + (int64_t)j * dstride, o);
  }
}

// Gather + pool adjoint of one query head per output head (dQ) over runs c of RL positions
// j = c RL + r.
template <typename T, int L, int P, int TT>
__global__ void __launch_bounds__(LH_RUN_BS) gather_bwd_long_kernel(RunArgs a) {
  constexpr int CH = 16 / sizeof(T);
  constexpr int RL = ipow(P, TT);
  constexpr int LS = TT < L ? TT : L;
  constexpr int NSUB = sub_off(P, TT, LS);
  constexpr int NSH = L - LS;
  const uint32_t c = xcd_contiguous(blockIdx.x, gridDim.x);
  const int hc = blockIdx.y * blockDim.x + threadIdx.x;
  if (c >= (uint32_t)a.nruns || hc >= a.HC) return;
  const int h = hc >> a.cpr_shift, cc = hc & ((1 << a.cpr_shift) - 1);
  const int64_t b = blockIdx.z;
  const int32_t* sl = slot_row(a, b, h);
  const T* src = reinterpret_cast<const T*>(a.src) + src_head(a, b, h) * a.S * a.D + cc * CH;
  const int32_t j0 = (int32_t)(c * RL);
  int32_t msh[NSH > 0 ? NSH : 1], msub[NSUB > 0 ? NSUB : 1], m0[RL];
#pragma unroll
  for (int l = LS; l < L; ++l) {  // entry floor(j / p^l) = floor(c / p^(l - TT))
    const int32_t i = (int32_t)(c / (uint32_t)ipow(P, l - TT));
    msh[l - LS] = i < a.nrow[l] ? sl[a.off[l] + i] : -1;
  }
#pragma unroll
  for (int l = 1; l < LS; ++l)
#pragma unroll
    for (int s2 = 0; s2 < ipow(P, TT - l); ++s2) {
      const int32_t i = (int32_t)(c * ipow(P, TT - l)) + s2;
      msub[sub_off(P, TT, l) + s2] = i < a.nrow[l] ? sl[a.off[l] + i] : -1;
    }
  load_level0_slots<RL, 0>(a, sl, j0, m0);
  u32x4 vsh[NSH > 0 ? NSH : 1], vsub[NSUB > 0 ? NSUB : 1], v0[RL];
#pragma unroll
  for (int x = 0; x < NSH; ++x) vsh[x] = load_entry_row(src, msh[x], a.S, a.D, sizeof(T));
#pragma unroll
  for (int x = 0; x < NSUB; ++x) vsub[x] = load_entry_row(src, msub[x], a.S, a.D, sizeof(T));
#pragma unroll
  for (int r = 0; r < RL; ++r) v0[r] = load_entry_row(src, m0[r], a.S, a.D, sizeof(T));
  float acc[CH];
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = 0.0f;
#pragma unroll
  for (int l = L - 1; l >= LS; --l) add_chunk_scaled<T>(acc, vsh[l - LS], a.inv[l]);
  T* dst = reinterpret_cast<T*>(a.dst) + ((b * a.N) * a.H + h) * (int64_t)a.D + cc * CH;
  const int64_t dstride = (int64_t)a.H * a.D;
#pragma unroll
  for (int r = 0; r < RL; ++r) {
    const int32_t j = j0 + r;
    if (j >= a.N) continue;
    float o[CH], fine[CH];
#pragma unroll
    for (int e = 0; e < CH; ++e) o[e] = acc[e], fine[e] = 0.0f;
#pragma unroll
    for (int l = LS - 1; l >= 1; --l) add_chunk_scaled<T>(o, vsub[sub_off(P, TT, l) + r / ipow(P, l)], a.inv[l]);
    add_chunk<T>(fine, v0[r]);
#pragma unroll
    for (int e = 0; e < CH; ++e) o[e] = o[e] + fine[e];
    store_chunk<T>(dst + (int64_t)j * dstride, o);
  }
}

// Gather + pool adjoint summed over the Gs query heads of a group (dK, dV), runs of p <= 4
// positions: the slots and then the rows of GB heads at a time are loaded before their sums,
// which keep the order of gather_bwd_kernel.
template <typename T, int L, int GB>
__global__ void __launch_bounds__(LH_RUN_BS) gather_bwd_group_kernel(RunArgs a) {
  constexpr int CH = 16 / sizeof(T);
  constexpr int PU = 4;
  constexpr int LA = L > 1 ? L : 2;
  const uint32_t c = xcd_contiguous(blockIdx.x, gridDim.x);
  const int hc = blockIdx.y * blockDim.x + threadIdx.x;
  if (c >= (uint32_t)a.nruns || hc >= a.HC) return;
  const int h = hc >> a.cpr_shift, cc = hc & ((1 << a.cpr_shift) - 1);
  const int64_t b = blockIdx.z;
  const int32_t jbase = (int32_t)(c * (uint32_t)a.run);
  int32_t ent[LA];
#pragma unroll
  for (int l = 1; l < L; ++l) ent[l] = a.off[l] + run_entry(a, c, l);
  float acc[CH], fine[PU][CH];
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = 0.0f;
#pragma unroll
  for (int r = 0; r < PU; ++r)
#pragma unroll
    for (int e = 0; e < CH; ++e) fine[r][e] = 0.0f;
  for (int g0 = 0; g0 < a.Gs; g0 += GB) {
    int32_t m[GB][LA], m0[GB][PU];
#pragma unroll
    for (int gg = 0; gg < GB; ++gg) {
      const bool live = g0 + gg < a.Gs;
      const int32_t* sl = slot_row(a, b, h * a.Gs + g0 + gg);
#pragma unroll
      for (int l = L - 1; l >= 1; --l) m[gg][l] = live ? sl[ent[l]] : -1;
#pragma unroll
      for (int r = 0; r < PU; ++r) m0[gg][r] = (live && r < a.run) ? sl[jbase + r] : -1;
    }
    u32x4 v[GB][LA], v0[GB][PU];
#pragma unroll
    for (int gg = 0; gg < GB; ++gg) {
      const T* src = reinterpret_cast<const T*>(a.src) + src_head(a, b, h * a.Gs + g0 + gg) * a.S * a.D + cc * CH;
#pragma unroll
      for (int l = L - 1; l >= 1; --l) v[gg][l] = load_entry_row(src, m[gg][l], a.S, a.D, sizeof(T));
#pragma unroll
      for (int r = 0; r < PU; ++r) v0[gg][r] = load_entry_row(src, m0[gg][r], a.S, a.D, sizeof(T));
    }
#pragma unroll
    for (int gg = 0; gg < GB; ++gg) {
      if (g0 + gg >= a.Gs) break;
#pragma unroll
      for (int l = L - 1; l >= 1; --l) add_chunk_scaled<T>(acc, v[gg][l], a.inv[l]);
#pragma unroll
      for (int r = 0; r < PU; ++r) add_chunk<T>(fine[r], v0[gg][r]);
    }
  }
  T* dst = reinterpret_cast<T*>(a.dst) + ((b * a.N) * a.H + h) * (int64_t)a.D + cc * CH;
  const int64_t dstride = (int64_t)a.H * a.D;
#pragma unroll
  for (int r = 0; r < PU; ++r) {
    if (r < a.run) {
      float o[CH];
#pragma unroll
      for (int e = 0; e < CH; ++e) o[e] = acc[e] + fine[r][e];
      store_chunk<T>(dst + (int64_t)(jbase + r) * dstride, o);
    }
  }
}

// Gather + pool adjoint summed over the Gs query heads of a group (dK, dV) for p a power of two:
// a thread handles RH = 2^RHL positions j = c RH + r (RH a multiple of p). A level-l entry is
// shared by the run when p^l >= RH; otherwise the run holds RH / p^l of them. Heads are visited
// in order with the next head's slots loaded while the current head's rows are in flight. The
// sums keep the order of gather_bwd_kernel: for each window of p positions, levels L-1 .. 1 of
// every head in turn; per position, level 0 of every head in turn; one rounding.
template <int PL, int RHL, int L>
struct GroupRun {
  static constexpr int RH = 1 << RHL;
  static constexpr int P = 1 << PL;
  static constexpr int NW = RH / P;  // level-1 windows per run
  // entries of level l in the run (1 when shared)
  static constexpr int cnt(int l) { return l * PL >= RHL ? 1 : 1 << (RHL - l * PL); }
  static constexpr int base(int l) {  // index of level l's first entry in the flattened list
    int s = 0;
    for (int x = 1; x < l; ++x) s += cnt(x);
    return s;
  }
  static constexpr int NE = base(L) + RH;  // coarse entries, then RH level-0 entries
};

// PACK: one run has fewer threads of work than a wave (few KV heads), so a workgroup covers
// a.rpb consecutive runs; the run index then differs between lanes (a separate instantiation,
// so that the common case keeps a workgroup-uniform run index).
template <typename T, int L, int PL, int RHL, bool PACK>
__global__ void __launch_bounds__(LH_RUN_BS) gather_bwd_group_long_kernel(RunArgs a) {
  using G = GroupRun<PL, RHL, L>;
  constexpr int CH = 16 / sizeof(T);
  constexpr int RH = G::RH, NW = G::NW, NE = G::NE, NC = G::base(L);
  uint32_t c = xcd_contiguous(blockIdx.x, gridDim.x);
  int hc = blockIdx.y * blockDim.x + threadIdx.x;
  if constexpr (PACK) {
    const int sub = (int)threadIdx.x / a.HC;
    c = c * (uint32_t)a.rpb + (uint32_t)sub;
    hc = (int)threadIdx.x - sub * a.HC;
  }
  if (c >= (uint32_t)a.nruns || hc >= a.HC) return;
  const int h = hc >> a.cpr_shift, cc = hc & ((1 << a.cpr_shift) - 1);
  const int64_t b = blockIdx.z;
  const int32_t j0 = (int32_t)(c * RH);
  // flattened slot indices (into one head's slot row) of the run's entries; -1: none
  int32_t sidx[NE];
#pragma unroll
  for (int l = 1; l < L; ++l)
#pragma unroll
    for (int e = 0; e < G::cnt(l); ++e) {
      // entry floor(j / p^l) for the first position of sub-run e
      const int32_t i = G::cnt(l) == 1 ? (int32_t)((uint32_t)j0 >> (l * PL)) : (j0 >> (l * PL)) + e;
      sidx[G::base(l) + e] = i < a.nrow[l] ? a.off[l] + i : -1;
    }
#pragma unroll
  for (int r = 0; r < RH; ++r) sidx[NC + r] = j0 + r < a.N ? j0 + r : -1;
  auto load_slots = [&](int g, int32_t* m) __attribute__((always_inline)) {
    const int32_t* sl = slot_row(a, b, h * a.Gs + g);
#pragma unroll
    for (int e = 0; e < NE; ++e) m[e] = sidx[e] >= 0 ? sl[sidx[e]] : -1;
  };
  float acc[NW][CH], fine[RH][CH];
#pragma unroll
  for (int w = 0; w < NW; ++w)
#pragma unroll
    for (int e = 0; e < CH; ++e) acc[w][e] = 0.0f;
#pragma unroll
  for (int r = 0; r < RH; ++r)
#pragma unroll
    for (int e = 0; e < CH; ++e) fine[r][e] = 0.0f;
  int32_t m[NE], mn[NE];
  load_slots(0, m);
  for (int g = 0; g < a.Gs; ++g) {
    const T* src = reinterpret_cast<const T*>(a.src) + src_head(a, b, h * a.Gs + g) * a.S * a.D + cc * CH;
    u32x4 v[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) v[e] = load_entry_row(src, m[e], a.S, a.D, sizeof(T));
    if (g + 1 < a.Gs) load_slots(g + 1, mn);
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
      for (int l = L - 1; l >= 1; --l) {
        // the level-l entry of window w (windows of p positions nest in sub-runs of p^l)
        const int e = G::cnt(l) == 1 ? 0 : (w * G::P) >> (l * PL);
        add_chunk_scaled<T>(acc[w], v[G::base(l) + e], a.inv[l]);
      }
#pragma unroll
    for (int r = 0; r < RH; ++r) add_chunk<T>(fine[r], v[NC + r]);
#pragma unroll
    for (int e = 0; e < NE; ++e) m[e] = mn[e];
  }
  T* dst = reinterpret_cast<T*>(a.dst) + ((b * a.N) * a.H + h) * (int64_t)a.D + cc * CH;
  const int64_t dstride = (int64_t)a.H * a.D;
#pragma unroll
  for (int r = 0; r < RH; ++r) {
    if (j0 + r >= a.N) continue;
    float o[CH];
#pragma unroll
    for (int e = 0; e < CH; ++e) o[e] = acc[r / G::P][e] + fine[r][e];
    store_chunk<T>(dst + (int64_t)(j0 + r) * dstride, o);
  }
}

// ---------------------------------------------------------------- scatter_bwd

struct ScatterBwdArgs {
  const void* dout;  // [B, N, Hq, D]
  const int32_t* slot;
  void* dos;  // [B, Hq, S, D]
  int64_t Ptot;
  int32_t N, S, U, WR, Hq, D, HW, cpr_shift, p;  // U = N + p^(L-1): positions of the shifted sequence
  int32_t Hs, Gq;  // query head hq reads the slot row of selection head hq / Gq
  int32_t off[17];
  int32_t nrows[16];  // N / p^l
  int32_t epb[16];    // WR / p^l: level-l windows per workgroup
};

constexpr int kScatterBwdRB = 8;  // rows loaded per step

// Shifted window sums. With x[u] = dout[u - 1] (zero for u = 0 and u > N), the range of entry
// (l, i) is exactly the level-l window a = i + 1 of x: [a p^l, (a+1) p^l - 1]. A workgroup walks
// a range of u that is a multiple of p^(L-1) with fp32 running sums per level (as in pooling)
// and writes the sum of every closed window whose entry was gathered; level-0 entries are a
// plain copy. dout is read once. Window closings are tracked with counters, and the slot of a
// window's entry is fetched when the window opens, so it has arrived when the window closes.
template <typename T, int L>
__global__ void __launch_bounds__(256) scatter_bwd_kernel(ScatterBwdArgs a) {
  constexpr int CH = 16 / sizeof(T);
  constexpr int LA = L > 1 ? L : 2;
  constexpr int RB = kScatterBwdRB;
  const int tid = threadIdx.x;
  const int hc = tid >> a.cpr_shift, cc = tid & ((1 << a.cpr_shift) - 1);
  const int hq = blockIdx.y * a.HW + hc;
  if (hq >= a.Hq) return;  // no barriers below
  const int64_t b = blockIdx.z;
  const int64_t bh = b * a.Hq + hq;
  const int32_t* sl = a.slot + (b * a.Hs + hq / a.Gq) * a.Ptot;
  T* dos = reinterpret_cast<T*>(a.dos) + bh * a.S * a.D + cc * CH;
  const T* src = reinterpret_cast<const T*>(a.dout) + (b * a.N * a.Hq + hq) * (int64_t)a.D + cc * CH;
  const int64_t sstride = (int64_t)a.Hq * a.D;
  const int32_t u0 = (int32_t)blockIdx.x * a.WR;
  const int32_t nu = a.U - u0 < a.WR ? a.U - u0 : a.WR;

  float acc[LA][CH];
#pragma unroll
  for (int l = 0; l < LA; ++l)
#pragma unroll
    for (int e = 0; e < CH; ++e) acc[l][e] = 0.0f;
  int cnt[LA + 1];
#pragma unroll
  for (int l = 0; l <= LA; ++l) cnt[l] = 0;
  int32_t win[LA];  // index a of the open level-l window; its entry is i = a - 1
  int32_t ms[LA];   // slot of that entry, or -1
  auto entry_slot = [&](int l, int32_t i) -> int32_t {
    return (i >= 0 && i < a.nrows[l]) ? sl[a.off[l] + i] : -1;
  };
#pragma unroll
  for (int l = 1; l < L; ++l) {
    win[l] = (int32_t)blockIdx.x * a.epb[l];
    ms[l] = entry_slot(l, win[l] - 1);
  }

  for (int ub = 0; ub < nu; ub += RB) {
    u32x4 v[RB];
    int32_t m0[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int32_t u = u0 + ub + r;
      const bool valid = ub + r < nu && u >= 1 && u <= a.N;
      v[r] = valid ? load16_nt(src + (int64_t)(u - 1) * sstride) : u32x4{0, 0, 0, 0};  // dout: read once
      m0[r] = valid ? sl[u - 1] : -1;
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      if (ub + r >= nu) break;
      // level 0: entry i = u - 1 takes x[u] = dout[u - 1] unchanged
      if ((uint32_t)m0[r] < (uint32_t)a.S) store16_nt(dos + (int64_t)m0[r] * a.D, v[r]);
      if constexpr (L > 1) {
        add_chunk<T>(acc[1], v[r]);
        if (++cnt[1] == a.p) {
#pragma unroll
          for (int l = 1; l < L; ++l) {
            if (l > 1 && cnt[l] != a.p) break;
            cnt[l] = 0;
            if ((uint32_t)ms[l] < (uint32_t)a.S) store_chunk<T>(dos + (int64_t)ms[l] * a.D, acc[l]);
            if (l + 1 < L) {
#pragma unroll
              for (int e = 0; e < CH; ++e) acc[l + 1 < L ? l + 1 : l][e] += acc[l][e];
              ++cnt[l + 1 < L ? l + 1 : l];
            }
#pragma unroll
            for (int e = 0; e < CH; ++e) acc[l][e] = 0.0f;
            ++win[l];
            ms[l] = entry_slot(l, win[l] - 1);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------- host launchers

static int cpr_shift_of(int D, int esize) {
  const int cpr = D * esize / 16;
  int s = 0;
  while ((1 << s) < cpr) ++s;
  return s;
}

// Long runs of p^2 (p = 4) or p^3 (p = 2) positions for the scatter and for adjoints with one
// query head per output head; runs of p otherwise.
static int long_run_tt(const LhShape& s) {
  if (s.L < 2) return 0;
  if (s.p == 4) return 2;
  if (s.p == 2) return 3;
  return 0;
}

template <typename T, int L>
static void launch_scatter_P(const LhShape& s, RunArgs a, dim3 grid, dim3 block, hipStream_t st) {
  const int tt = long_run_tt(s);
  if (tt) {
    const int rl = tt == 2 ? 16 : 8;
    a.nruns = (int32_t)((s.N + rl) / rl);  // j = c rl + r - 1 up to N - 1
    grid.x = (unsigned)((a.nruns + 7) / 8 * 8);
    if (tt == 2) hipLaunchKernelGGL((scatter_long_kernel<T, L, 4, 2>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((scatter_long_kernel<T, L, 2, 3>), grid, block, 0, st, a);
  } else if (a.run <= 4) {
    hipLaunchKernelGGL((scatter_kernel<T, L, 4>), grid, block, 0, st, a);
  } else {
    hipLaunchKernelGGL((scatter_kernel<T, L, 0>), grid, block, 0, st, a);
  }
}

template <typename T, int L>
static void launch_gather_bwd_P(const LhShape& s, RunArgs a, dim3 grid, dim3 block, hipStream_t st) {
  const int tt = long_run_tt(s);
  if (a.Gs == 1 && tt) {
    const int rl = tt == 2 ? 16 : 8;
    a.nruns = (int32_t)((s.N + rl - 1) / rl);
    grid.x = (unsigned)((a.nruns + 7) / 8 * 8);
    if (tt == 2) hipLaunchKernelGGL((gather_bwd_long_kernel<T, L, 4, 2>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((gather_bwd_long_kernel<T, L, 2, 3>), grid, block, 0, st, a);
  } else if (a.Gs > 1 && L > 1 && (s.p == 2 || s.p == 4)) {
    constexpr int RHL = 3;  // runs of 8 positions
    a.nruns = (int32_t)((s.N + 7) / 8);
    // under a wave of threads per run: pack runs into one 64-thread workgroup
    a.rpb = a.HC < 64 ? 64 / a.HC : 1;
    grid.x = (unsigned)(((a.nruns + a.rpb - 1) / a.rpb + 7) / 8 * 8);
    if (a.rpb > 1) {
      block.x = (unsigned)(a.rpb * a.HC);
      if (s.p == 4) hipLaunchKernelGGL((gather_bwd_group_long_kernel<T, L, 2, RHL, true>), grid, block, 0, st, a);
      else hipLaunchKernelGGL((gather_bwd_group_long_kernel<T, L, 1, RHL, true>), grid, block, 0, st, a);
    } else {
      if (s.p == 4) hipLaunchKernelGGL((gather_bwd_group_long_kernel<T, L, 2, RHL, false>), grid, block, 0, st, a);
      else hipLaunchKernelGGL((gather_bwd_group_long_kernel<T, L, 1, RHL, false>), grid, block, 0, st, a);
    }
  } else if (a.Gs > 1 && a.run <= 4) {
    hipLaunchKernelGGL((gather_bwd_group_kernel<T, L, LH_GBWD_GB>), grid, block, 0, st, a);
  } else if (a.run <= 4) {
    hipLaunchKernelGGL((gather_bwd_kernel<T, L, 4>), grid, block, 0, st, a);
  } else {
    hipLaunchKernelGGL((gather_bwd_kernel<T, L, 0>), grid, block, 0, st, a);
  }
}

template <typename T>
static void launch_run_kernel(bool scatter, const LhShape& s, const RunArgs& a, dim3 grid, dim3 block,
                              hipStream_t st) {
#define LH_RUN_CASE(LL)                                            \
  case LL:                                                         \
    if (scatter) launch_scatter_P<T, LL>(s, a, grid, block, st);   \
    else launch_gather_bwd_P<T, LL>(s, a, grid, block, st);        \
    break;
  switch (s.L) {
    LH_RUN_CASE(1)
    LH_RUN_CASE(2)
    LH_RUN_CASE(3)
    LH_RUN_CASE(4)
    LH_RUN_CASE(5)
    LH_RUN_CASE(6)
    LH_RUN_CASE(7)
    default: LH_RUN_CASE(8)
  }
#undef LH_RUN_CASE
}

// H output heads, each summing Gs consecutive source heads of the Hsrc in src; source head x
// reads slot row x / sdiv (of the s.Hs selection heads).
static RunArgs run_args(const LhShape& s, const void* src, const int32_t* slot, void* dst, int H, int Gs,
                        int Hsrc, int sdiv, bool scatter) {
  RunArgs a = {};
  a.src = src;
  a.slot = slot;
  a.dst = dst;
  a.Ptot = s.Ptot;
  a.N = (int32_t)s.N;
  a.S = (int32_t)s.S;
  a.D = s.D;
  a.run = s.L > 1 ? s.p : 1;
  a.nruns = (int32_t)(s.N / a.run) + (scatter ? 1 : 0);
  a.Hq = s.Hq;
  a.H = H;
  a.Gs = Gs;
  a.Hsrc = Hsrc;
  a.Hslot = s.Hs;
  a.sdiv = sdiv;
  const int es = s.dtype == LH_BF16 ? 2 : 4;
  a.cpr_shift = cpr_shift_of(s.D, es);
  a.HC = H << a.cpr_shift;
  a.pshift = -1;
  if (s.L > 1 && (s.p & (s.p - 1)) == 0) {
    a.pshift = 0;
    while ((1 << a.pshift) < s.p) ++a.pshift;
  }
  for (int l = 0; l < 16; ++l) {
    a.pw[l] = l < s.L ? (int32_t)s.pw[l] : 1;
    a.inv[l] = l < s.L ? 1.0f / (float)s.pw[l] : 0.0f;
  }
  for (int l = 0; l < 17; ++l) a.off[l] = (int32_t)s.off[l];
  for (int l = 0; l < 16; ++l) a.nrow[l] = l < s.L ? (int32_t)(s.N / s.pw[l]) : 0;
  a.vec_slots = (s.Ptot % 4) == 0;
  a.rpb = 1;
  return a;
}

static void run_grid(const RunArgs& a, int B, dim3* grid, dim3* block) {
  const int bs = a.HC < LH_RUN_BS ? a.HC : LH_RUN_BS;
  const unsigned nx = (unsigned)((a.nruns + 7) / 8 * 8);  // a multiple of 8 for the XCD mapping
  *grid = dim3(nx, (unsigned)((a.HC + bs - 1) / bs), (unsigned)B);
  *block = dim3((unsigned)bs);
}

template <typename T, int L>
static hipError_t launch_scatter_bwd_T(const LhShape& s, const void* dout, const int32_t* slot,
                                       void* dos, hipStream_t st) {
  ScatterBwdArgs a = {};
  a.dout = dout;
  a.slot = slot;
  a.dos = dos;
  a.Ptot = s.Ptot;
  a.N = (int32_t)s.N;
  a.S = (int32_t)s.S;
  a.U = (int32_t)(s.N + s.P);
  a.Hq = s.Hq;
  a.Hs = s.Hs;
  a.Gq = s.Gq;
  a.D = s.D;
  a.p = s.p;
  a.cpr_shift = cpr_shift_of(s.D, (int)sizeof(T));
  const int CPR = 1 << a.cpr_shift;
  a.HW = s.Hq < 256 / CPR ? s.Hq : 256 / CPR;
  int64_t W = s.P;
  while (W < 64) W += s.P;
  a.WR = (int32_t)W;
  for (int l = 0; l < 16; ++l) {
    a.nrows[l] = l < s.L ? (int32_t)(s.N / s.pw[l]) : 0;
    a.epb[l] = l < s.L ? (int32_t)(W / s.pw[l]) : 0;
  }
  for (int l = 0; l < 17; ++l) a.off[l] = (int32_t)s.off[l];
  dim3 grid((unsigned)((a.U + W - 1) / W), (unsigned)((s.Hq + a.HW - 1) / a.HW), (unsigned)s.B);
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
  GatherArgs a{q, k, v, qpyr, kpyr, vpyr, idx, qs, ks, vs, s.N, s.R, s.S, s.Hq, s.Hkv, s.G, s.D, 0, 0, s.Hs, s.Gq};
  const int es = s.dtype == LH_BF16 ? 2 : 4;
  a.cpr_shift = cpr_shift_of(s.D, es);
  a.rows_per_block = 256 >> a.cpr_shift;
  dim3 grid((unsigned)((s.S + a.rows_per_block - 1) / a.rows_per_block), (unsigned)(s.B * s.Hq));
  if (s.dtype == LH_BF16) hipLaunchKernelGGL(gather_kernel<bf16_t>, grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL(gather_kernel<float>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t lh_launch_scatter(const LhShape& s, const void* os, const int32_t* slot, void* o,
                             hipStream_t st) {
  const RunArgs a = run_args(s, os, slot, o, s.Hq, 1, s.Hq, s.Gq, true);
  dim3 grid, block;
  run_grid(a, (int)s.B, &grid, &block);
  if (s.dtype == LH_BF16) launch_run_kernel<bf16_t>(true, s, a, grid, block, st);
  else launch_run_kernel<float>(true, s, a, grid, block, st);
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
    // dQ: per query head, from dqs [B,Hq,S,D]. dK, dV: per KV head, summing the gradients of
    // its G / Gq selection heads in dks, dvs [B,Hs,S,D] (its query heads, or the group itself).
    const RunArgs a = which == 0 ? run_args(s, srcs[0], slot, dsts[0], s.Hq, 1, s.Hq, s.Gq, false)
                                 : run_args(s, srcs[which], slot, dsts[which], s.Hkv, s.G / s.Gq, s.Hs, 1, false);
    dim3 grid, block;
    run_grid(a, (int)s.B, &grid, &block);
    if (s.dtype == LH_BF16) launch_run_kernel<bf16_t>(false, s, a, grid, block, st);
    else launch_run_kernel<float>(false, s, a, grid, block, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
