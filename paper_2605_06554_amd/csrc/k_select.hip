// k_select.hip -- hierarchical selection (Sec. 3.4, Eq. topk with Fig. 2 panel 3) and causal
// ordering of the selected entries (Sec. 3.5, mask paragraph).
//
// select_kernel: one workgroup of 1024 threads per (b, hq). Per level l = L-1 .. 1 it ranks the
// level's candidates (a sorted list of level-local indices) by the 32-bit key
// bits(max(s_QK, s_KQ)) -- non-negative floats, so the bit pattern orders them -- and finds the
// exact threshold of the k best by an MSB-first radix select (four 8-bit digits, LDS
// histograms with integer atomics). A stable compaction in candidate order then takes every
// key above the threshold and the first (lower-index) ties, and writes the p children of each
// parent -- which are the next level's candidates, already sorted -- into the workspace.
// With LH_FLAG_STRATIFIED (App. D.2) the same select and compaction run on every chunk of 2048
// consecutive candidates, each keeping its proportional share of the k parents.
// No floating-point atomics: the result is bitwise deterministic.
//
// order_kernel: one thread per candidate. Emitted entries are sorted by
// key = e * L + (L - 1 - l), e = (i + 1) p^l - 1 (window end, coarser level first on ties).
// Each level's list is sorted by i, hence by key, so an entry's rank is the sum over levels of
// a binary search (merge by rank, no general sort). It writes idx[rank] and slot[id] = rank.
#include "lh_common.h"

namespace lh {

constexpr int kSelThreads = 1024;
// Stratified mode (App. D.2): candidates of a ranking level are cut into chunks of this many.
constexpr int64_t kStratChunk = 2048;
constexpr int kSelWaves = kSelThreads / 64;

struct SelArgs {
  const float* s_qk;
  const float* s_kq;
  int32_t* ws;  // [B, Hq, Scand] candidate lists, level-major
  int64_t Ptot, Scand;
  int32_t Hq, Hkv, G, L, p;
  int32_t Hs, Gq;  // selection heads; query heads whose scores one selection ranks
  int64_t off[17];
  int64_t cand[16];
  int64_t npar[16];
  int64_t coff[17];
  int32_t stratified;  // LH_FLAG_STRATIFIED: per-chunk shares instead of one top-k per level
};

// Exclusive prefix sum over the 1024 threads of the block; returns the exclusive value and
// writes the block total. `sh` holds kSelWaves ints.
__device__ __forceinline__ int block_exclusive_scan(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int t = __shfl_up(inc, d, 64);
    if (lane >= d) inc += t;
  }
  if (lane == 63) sh[w] = inc;
  __syncthreads();
  int wsum = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelWaves; ++i) {
    const int x = sh[i];
    if (i < w) wsum += x;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return wsum + inc - v;
}

__global__ void __launch_bounds__(kSelThreads) select_kernel(SelArgs a) {
  extern __shared__ uint32_t keys[];  // candidate keys of the current level
  __shared__ int hist[256];
  __shared__ int scan_sh[kSelWaves];
  __shared__ uint32_t sel_state[2];  // prefix, remaining

  const int tid = threadIdx.x;
  const int bs = blockIdx.x;  // b * Hs + hs
  const int hs = bs % a.Hs;
  const int64_t b = bs / a.Hs;
  const int g = hs * a.Gq / a.G;  // KV head
  // query score rows of the selection: query heads hs Gq .. hs Gq + Gq - 1
  const float* sq = a.s_qk + (b * a.Hq + (int64_t)hs * a.Gq) * a.Ptot;
  const float* sk = a.s_kq + (b * a.Hkv + g) * a.Ptot;
  int32_t* C = a.ws + (int64_t)bs * a.Scand;
  const int L = a.L, p = a.p;

  // top level: every entry is a candidate
  for (int64_t u = tid; u < a.cand[L - 1]; u += kSelThreads) C[a.coff[L - 1] + u] = (int32_t)u;
  __threadfence_block();
  __syncthreads();

  for (int l = L - 1; l >= 1; --l) {
    const int64_t n = a.cand[l];
    const int64_t kk = a.npar[l];
    const int32_t* Cl = C + a.coff[l];
    int32_t* Cn = C + a.coff[l - 1];
    const float* sql = sq + a.off[l];
    const float* skl = sk + a.off[l];
    if (kk == n) {
      // every candidate is a parent
      for (int64_t j = tid; j < n * p; j += kSelThreads) Cn[j] = Cl[j / p] * p + (int32_t)(j % p);
      __threadfence_block();
      __syncthreads();
      continue;
    }
    if (kk == 0) continue;
    for (int64_t u = tid; u < n; u += kSelThreads) {
      const int32_t i = Cl[u];
      float x = sql[i];
      for (int t = 1; t < a.Gq; ++t) {  // the max over the query heads of a shared selection
        const float z = sql[(int64_t)t * a.Ptot + i];
        x = x > z ? x : z;
      }
      const float y = skl[i];
      keys[u] = __float_as_uint(x > y ? x : y);
    }
    __syncthreads();
    // One chunk covers the whole level in the exact mode. In the stratified mode chunk [s0, e0)
    // keeps its best floor(kk e0 / n) - floor(kk s0 / n) candidates, written after the
    // floor(kk s0 / n) parents of the chunks before it (candidate order is kept).
    const int64_t chunk = a.stratified ? kStratChunk : n;
    for (int64_t s0 = 0; s0 < n; s0 += chunk) {
      const int64_t e0 = s0 + chunk < n ? s0 + chunk : n;
      const int64_t first = a.stratified ? (kk * s0) / n : 0;
      const int64_t quota = a.stratified ? (kk * e0) / n - first : kk;
      if (quota == 0) continue;
      if (tid == 0) {
        sel_state[0] = 0u;
        sel_state[1] = (uint32_t)quota;
      }
      __syncthreads();
      // MSB-first radix select of the quota-th largest key of the chunk
      for (int shift = 24; shift >= 0; shift -= 8) {
        for (int t = tid; t < 256; t += kSelThreads) hist[t] = 0;
        __syncthreads();
        const uint32_t prefix = sel_state[0];
        const uint32_t himask = shift == 24 ? 0u : (0xffffffffu << (shift + 8));
        for (int64_t u = s0 + tid; u < e0; u += kSelThreads) {
          const uint32_t key = keys[u];
          if ((key & himask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
        __syncthreads();
        if (tid == 0) {
          uint32_t rem = sel_state[1];
          int bin = 255;
          for (; bin > 0; --bin) {
            const uint32_t c = (uint32_t)hist[bin];
            if (c >= rem) break;
            rem -= c;
          }
          sel_state[0] = prefix | ((uint32_t)bin << shift);
          sel_state[1] = rem;
        }
        __syncthreads();
      }
      const uint32_t T = sel_state[0];
      const int need = (int)sel_state[1];  // ties at T to take, lowest candidate positions first
      // stable compaction in candidate order (rounds of 1024 consecutive candidates)
      int gt_before = 0, eq_before = 0;
      for (int64_t base = s0; base < e0; base += kSelThreads) {
        const int64_t u = base + tid;
        uint32_t key = 0;
        if (u < e0) key = keys[u];
        const int gt = (u < e0 && key > T) ? 1 : 0;
        const int eq = (u < e0 && key == T) ? 1 : 0;
        int tot;
        const int packed = block_exclusive_scan((gt << 16) | eq, scan_sh, &tot);
        const int gt_rank = gt_before + (packed >> 16);
        const int eq_rank = eq_before + (packed & 0xffff);
        const bool take = gt || (eq && eq_rank < need);
        if (take) {
          const int64_t pos = first + gt_rank + (eq_rank < need ? eq_rank : need);
          const int32_t i = Cl[u];
          for (int r = 0; r < p; ++r) Cn[pos * p + r] = i * p + r;
        }
        gt_before += tot >> 16;
        eq_before += tot & 0xffff;
      }
      __syncthreads();  // sel_state and hist are reused by the next chunk
    }
    __threadfence_block();
    __syncthreads();
  }
}

struct OrdArgs {
  const int32_t* ws;
  int32_t* idx;   // [B, Hq, S]
  int32_t* slot;  // [B, Hq, Ptot]
  int64_t Ptot, Scand, S;
  int32_t L, p, replace;
  int64_t off[17];
  int64_t pw[16];
  int64_t cand[16];
  int64_t coff[17];
  int64_t nrows[16];  // N / p^l
};

__device__ __forceinline__ int64_t order_key(int64_t i, int l, const OrdArgs& a) {
  return ((i + 1) * a.pw[l] - 1) * a.L + (a.L - 1 - l);
}

// number of entries of the sorted list c[0, n) at level l whose key is below K
__device__ __forceinline__ int64_t count_below(const int32_t* c, int64_t n, int l, int64_t K,
                                               const OrdArgs& a) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (order_key(c[mid], l, a) < K) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// number of entries of the sorted int list c[0, n) below value x
__device__ __forceinline__ int64_t lower_bound_val(const int32_t* c, int64_t n, int64_t x) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (c[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__global__ void __launch_bounds__(256) order_kernel(OrdArgs a) {
  const int64_t gpos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gpos >= a.Scand) return;
  const int64_t bh = blockIdx.y;
  const int32_t* C = a.ws + bh * a.Scand;
  int l = 0;
  while (l + 1 < a.L && gpos >= a.coff[l + 1]) ++l;
  const int64_t i = C[gpos];
  if (a.replace && l >= 1) {
    // a parent's children are in the next finer candidate list; parents are not emitted
    const int64_t c = lower_bound_val(C + a.coff[l - 1], a.cand[l - 1], i * a.p);
    if (c < a.cand[l - 1] && C[a.coff[l - 1] + c] == i * a.p) return;
  }
  const int64_t K = order_key(i, l, a);
  int64_t rank = 0;
  for (int l2 = 0; l2 < a.L; ++l2) {
    const int32_t* c2 = C + a.coff[l2];
    const int64_t lb = count_below(c2, a.cand[l2], l2, K, a);
    int64_t cnt = lb;
    if (a.replace && l2 >= 1) {
      const int64_t x = lb < a.cand[l2] ? (int64_t)c2[lb] : a.nrows[l2];
      cnt -= lower_bound_val(C + a.coff[l2 - 1], a.cand[l2 - 1], x * a.p) / a.p;
    }
    rank += cnt;
  }
  if (rank < 0 || rank >= a.S) return;  // cannot happen for lists written by select_kernel
  a.idx[bh * a.S + rank] = (int32_t)(a.off[l] + i);
  a.slot[bh * a.Ptot + a.off[l] + i] = (int32_t)rank;
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x)
    p[t] = v;
}

}  // namespace lh

using namespace lh;

hipError_t lh_launch_select(const LhShape& s, const float* s_qk, const float* s_kq, int32_t* idx,
                            int32_t* slot, int32_t* ws, hipStream_t st) {
  const int64_t BH = s.B * s.Hs;  // one selection per (b, selection head)
  // slot = -1 everywhere (a fill kernel, so the sequence can be captured in a graph)
  {
    const int64_t n = BH * s.Ptot;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)blocks), dim3(256), 0, st, slot, n, -1);
  }
  SelArgs a;
  a.s_qk = s_qk;
  a.s_kq = s_kq;
  a.ws = ws;
  a.Ptot = s.Ptot;
  a.Scand = s.Scand;
  a.Hq = s.Hq;
  a.Hkv = s.Hkv;
  a.G = s.G;
  a.Hs = s.Hs;
  a.Gq = s.Gq;
  a.L = s.L;
  a.p = s.p;
  for (int l = 0; l < 17; ++l) a.off[l] = s.off[l], a.coff[l] = s.coff[l];
  for (int l = 0; l < 16; ++l) a.cand[l] = s.cand[l], a.npar[l] = s.npar[l];
  a.stratified = (s.flags & LH_FLAG_STRATIFIED) ? 1 : 0;
  const size_t shm = (size_t)(s.maxsel > 0 ? s.maxsel : 1) * sizeof(uint32_t);
  hipLaunchKernelGGL(select_kernel, dim3((unsigned)BH), dim3(kSelThreads), shm, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  OrdArgs o;
  o.ws = ws;
  o.idx = idx;
  o.slot = slot;
  o.Ptot = s.Ptot;
  o.Scand = s.Scand;
  o.S = s.S;
  o.L = s.L;
  o.p = s.p;
  o.replace = (s.flags & LH_FLAG_REPLACE_PARENTS) ? 1 : 0;
  for (int l = 0; l < 17; ++l) o.off[l] = s.off[l], o.coff[l] = s.coff[l];
  for (int l = 0; l < 16; ++l) o.pw[l] = s.pw[l], o.cand[l] = s.cand[l], o.nrows[l] = l < s.L ? s.N / s.pw[l] : 0;
  dim3 grid((unsigned)((s.Scand + 255) / 256), (unsigned)BH);
  hipLaunchKernelGGL(order_kernel, grid, dim3(256), 0, st, o);
  return hipGetLastError();
}
