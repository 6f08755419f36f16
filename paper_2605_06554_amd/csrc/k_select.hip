// k_select.hip -- hierarchical selection (Sec. 3.4, Eq. topk with Fig. 2 panel 3) and causal
// ordering of the selected entries (Sec. 3.5, mask paragraph).
//
// select_kernel: one workgroup of 1024 threads per (b, selection head). Per level l = L-1 .. 1
// it ranks the level's candidates (a sorted list of level-local indices; their keys in LDS, or in
// a global workspace row when a level has more than 32,768 candidates) by the 32-bit key
// bits(max(s_QK, s_KQ)) -- non-negative floats, so the bit pattern orders them -- and finds the
// exact threshold of the k best by an MSB-first radix select (11-bit digits below the bits all
// keys share, LDS histograms with integer atomics; one wave reads each digit off the histogram
// with a suffix scan). A stable compaction in candidate order then takes every key above the threshold and
// the first (lower-index) ties, and writes the p children of each parent -- which are the next
// level's candidates, already sorted -- into the workspace. In the compaction each wave walks
// a contiguous range of candidates and ranks them with ballots.
// With LH_FLAG_STRATIFIED (App. D.2) the same select and compaction run on every chunk of 2048
// consecutive candidates, each keeping its proportional share of the k parents.
// No floating-point atomics: the result is bitwise deterministic.
//
// order_kernel: emitted entries are sorted by key = e * L + (L - 1 - l), e = (i + 1) p^l - 1
// (window end, coarser level first on ties). A workgroup owns a range of window ends: its
// entries are a contiguous part of each level's sorted list, the emitted entries before the
// range are counted by lower bounds in those lists, and a scan over the range's (end, level)
// flags orders the rest. It writes idx[rank], and slot for every pyramid entry (-1 for those
// not gathered), so slot needs no separate fill.
#include "lh_common.h"

namespace lh {

constexpr int kSelThreads = 1024;
// Stratified mode (App. D.2): candidates of a ranking level are cut into chunks of this many.
constexpr int64_t kStratChunk = 2048;
constexpr int kSelWaves = kSelThreads / 64;

// Levels of at most this many candidates keep their keys in LDS (128 KB); larger levels keep
// them in a global workspace region of their own (one row of maxsel keys per selection), which
// the radix passes stream through L2.
constexpr int64_t kSelLdsKeys = 32768;
// Candidate lists of levels >= 1 of at most this many entries stay in LDS beside the keys
// (LL mode: 2 x 64 KB).
constexpr int64_t kSelLdsList = 16384;

struct SelArgs {
  const float* s_qk;
  const float* s_kq;
  int32_t* ws;  // [B, Hq, Scand] candidate lists, level-major
  uint32_t* gkeys;  // [B, Hs, maxsel] keys when maxsel > kSelLdsKeys, else null
  int64_t maxsel;
  int64_t Ptot, Scand;
  int32_t Hq, Hkv, G, L, p;
  int32_t Hs, Gq;  // selection heads; query heads whose scores one selection ranks
  int64_t off[17];
  int64_t cand[16];
  int64_t npar[16];
  int64_t coff[17];
  int32_t stratified;  // LH_FLAG_STRATIFIED: per-chunk shares instead of one top-k per level
  int32_t coff_aligned4;  // every coff[l] is a multiple of 4
};

// Radix digits of kDigitBits bits: kBins histogram bins.
constexpr int kDigitBits = 11;
constexpr int kBins = 1 << kDigitBits;
constexpr int kBinsPerLane = kBins / 64;

// One wave picks the digit of the quota-th largest key from the histogram: the highest bin
// whose count, added to the counts of every higher bin, reaches the remaining quota. The
// remaining quota drops by the count of the higher bins. Lane l holds bins kBinsPerLane l ..
// kBinsPerLane (l + 1) - 1; a suffix sum over the lanes finds the one lane where the running
// count crosses the quota, and that lane walks its bins from the top.
__device__ __forceinline__ void select_bin(const int* hist, uint32_t* sel_state, uint32_t prefix, int shift,
                                           int lane) {
  const uint32_t rem = sel_state[1];
  uint32_t c[kBinsPerLane];
#pragma unroll
  for (int q = 0; q < kBinsPerLane / 4; ++q) {
    const int4 hb = *reinterpret_cast<const int4*>(hist + kBinsPerLane * lane + 4 * q);
    c[4 * q] = (uint32_t)hb.x, c[4 * q + 1] = (uint32_t)hb.y, c[4 * q + 2] = (uint32_t)hb.z, c[4 * q + 3] = (uint32_t)hb.w;
  }
  uint32_t lsum = 0;
#pragma unroll
  for (int j = 0; j < kBinsPerLane; ++j) lsum += c[j];
  uint32_t suf = lsum;  // counts of this lane's bins and every higher one
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t t = __shfl_down(suf, d, 64);
    if (lane + d < 64) suf += t;
  }
  const uint32_t above = suf - lsum;  // counts of the bins above this lane's
  if (above < rem && above + lsum >= rem) {
    uint32_t acc = above;
    int j = kBinsPerLane - 1;
    for (; j > 0; --j) {
      if (acc + c[j] >= rem) break;
      acc += c[j];
    }
    sel_state[0] = prefix | ((uint32_t)(kBinsPerLane * lane + j) << shift);
    sel_state[1] = rem - acc;
  } else if (lane == 0 && suf < rem) {  // fewer keys than the quota (not reached): bin 0
    sel_state[0] = prefix;
    sel_state[1] = rem - (suf - c[0]);
  }
}

// GK: the level's keys live in the global rows a.gkeys (levels above kSelLdsKeys candidates)
// instead of LDS; the algorithm is the same.
// LL (lists in LDS, when every list of levels >= 1 has at most kSelLdsList entries): the
// candidate list of the current level is also kept in LDS, after the keys, so the id reads of
// the key load and of the compaction make no global round trip. The lists are still written to
// the workspace, where the order kernel reads them.
template <bool GK, bool LL>
__global__ void __launch_bounds__(kSelThreads) select_kernel(SelArgs a) {
  static_assert(!(GK && LL), "lists in LDS go with keys in LDS");
  extern __shared__ __align__(16) uint32_t keys_lds[];  // candidate keys of the current level (LL: then its list)
  __shared__ __align__(16) int hist[kBins];
  __shared__ uint32_t sel_state[2];  // prefix, remaining
  __shared__ int wave_gt[kSelWaves], wave_eq[kSelWaves];  // counts of each wave's candidates
  __shared__ uint32_t key_and[kSelWaves], key_or[kSelWaves];  // per-wave AND / OR of the keys

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int bs = blockIdx.x;  // b * Hs + hs
  const int hs = bs % a.Hs;
  const int64_t b = bs / a.Hs;
  const int g = hs * a.Gq / a.G;  // KV head
  // query score rows of the selection: query heads hs Gq .. hs Gq + Gq - 1
  const float* sq = a.s_qk + (b * a.Hq + (int64_t)hs * a.Gq) * a.Ptot;
  const float* sk = a.s_kq + (b * a.Hkv + g) * a.Ptot;
  int32_t* C = a.ws + (int64_t)bs * a.Scand;
  uint32_t* keys = GK ? a.gkeys + (int64_t)bs * a.maxsel : keys_lds;
  int32_t* list = reinterpret_cast<int32_t*>(keys_lds) + kSelLdsList;  // LL only
  // children of a parent as one 16-byte store: every list of this selection's workspace row
  // starts 16-byte aligned
  const bool vec4 = ((reinterpret_cast<uintptr_t>(C) & 15) == 0) && a.coff_aligned4;
  const int L = a.L, p = a.p;

  // Top level: every entry is a candidate. With LL the lists written to the workspace are read
  // only after the kernel (by the order kernel), so no level waits for its global writes.
  for (int64_t u = tid; u < a.cand[L - 1]; u += kSelThreads) {
    C[a.coff[L - 1] + u] = (int32_t)u;
    if (LL && L > 1) list[u] = (int32_t)u;
  }
  if (!LL) __threadfence_block();
  __syncthreads();

  for (int l = L - 1; l >= 1; --l) {
    const int64_t n = a.cand[l];
    const int64_t kk = a.npar[l];
    const int32_t* Cl = LL ? list : C + a.coff[l];
    int32_t* Cn = C + a.coff[l - 1];
    const bool ln = LL && l - 1 >= 1;  // the next level's list is kept in LDS too
    const float* sql = sq + a.off[l];
    const float* skl = sk + a.off[l];
    if (kk == n) {
      // every candidate is a parent
      if (LL) {
        // the list is expanded in place: copy it to the (unused) key buffer first
        for (int64_t u = tid; u < n; u += kSelThreads) keys[u] = (uint32_t)list[u];
        __syncthreads();
        if (p == 4 && vec4) {  // one parent per thread: its 4 children as one 16-byte store
          for (int64_t u = tid; u < n; u += kSelThreads) {
            const int32_t c0 = (int32_t)keys[u] * 4;
            const u32x4 v = {(uint32_t)c0, (uint32_t)c0 + 1u, (uint32_t)c0 + 2u, (uint32_t)c0 + 3u};
            *reinterpret_cast<u32x4*>(Cn + 4 * u) = v;
            if (ln) *reinterpret_cast<u32x4*>(list + 4 * u) = v;
          }
        } else {
          for (int64_t j = tid; j < n * p; j += kSelThreads) {
            const int32_t v = (int32_t)keys[j / p] * p + (int32_t)(j % p);
            Cn[j] = v;
            if (ln) list[j] = v;
          }
        }
      } else {
        for (int64_t j = tid; j < n * p; j += kSelThreads) Cn[j] = Cl[j / p] * p + (int32_t)(j % p);
      }
      if (!LL) __threadfence_block();
      __syncthreads();
      continue;
    }
    if (kk == 0) continue;
    // keys of the level, kB candidates per thread at a time: the id loads, then the score
    // loads, are each in flight together
    constexpr int kB = 8;
    for (int64_t u0 = tid; u0 < n; u0 += (int64_t)kSelThreads * kB) {
      int32_t ids[kB];
      float x[kB], y[kB];
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        const int64_t u = u0 + (int64_t)j * kSelThreads;
        ids[j] = u < n ? Cl[u] : 0;
      }
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        x[j] = sql[ids[j]];
        y[j] = skl[ids[j]];
      }
      for (int t = 1; t < a.Gq; ++t) {  // the max over the query heads of a shared selection
#pragma unroll
        for (int j = 0; j < kB; ++j) {
          const float z = sql[(int64_t)t * a.Ptot + ids[j]];
          x[j] = x[j] > z ? x[j] : z;
        }
      }
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        const int64_t u = u0 + (int64_t)j * kSelThreads;
        if (u < n) keys[u] = __float_as_uint(x[j] > y[j] ? x[j] : y[j]);
      }
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
      // The bits every key of the chunk shares need no radix pass: a block AND / OR of the keys
      // gives them, and the digits start at the highest bit that varies.
      uint32_t kand = 0xffffffffu, kor = 0u;
      for (int64_t u = s0 + tid; u < e0; u += kSelThreads) {
        const uint32_t key = keys[u];
        kand &= key;
        kor |= key;
      }
#pragma unroll
      for (int d = 32; d >= 1; d >>= 1) {
        kand &= __shfl_xor(kand, d, 64);
        kor |= __shfl_xor(kor, d, 64);
      }
      if (lane == 0) {
        key_and[wv] = kand;
        key_or[wv] = kor;
      }
      __syncthreads();
      kand = 0xffffffffu;
      kor = 0u;
      for (int i = 0; i < kSelWaves; ++i) {
        kand &= key_and[i];
        kor |= key_or[i];
      }
      const int nb = (kand ^ kor) ? 32 - __clz(kand ^ kor) : 0;  // low bits that vary
      if (tid == 0) {
        sel_state[0] = nb == 32 ? 0u : (kor & ~((1u << nb) - 1u));
        sel_state[1] = (uint32_t)quota;
      }
      __syncthreads();
      // MSB-first radix select of the quota-th largest key of the chunk, kDigitBits a pass
      for (int hi = nb; hi > 0; hi -= kDigitBits) {
        const int shift = hi > kDigitBits ? hi - kDigitBits : 0;
        for (int t = tid; t < kBins; t += kSelThreads) hist[t] = 0;
        __syncthreads();
        const uint32_t prefix = sel_state[0];
        const uint32_t himask = hi == 32 ? 0u : (0xffffffffu << hi);
        const uint32_t dmask = (1u << (hi - shift)) - 1u;
        for (int64_t u = s0 + tid; u < e0; u += kSelThreads) {
          const uint32_t key = keys[u];
          if ((key & himask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1);
        }
        __syncthreads();
        if (tid < 64) select_bin(hist, sel_state, prefix, shift, tid);
        __syncthreads();
      }
      const uint32_t T = sel_state[0];
      const int need = (int)sel_state[1];  // ties at T to take, lowest candidate positions first
      // stable compaction in candidate order: wave w owns the candidates [c0, c1) and walks
      // them 64 at a time; ranks come from ballots, and the waves before it give its offsets
      const int64_t per = ((e0 - s0 + kSelWaves - 1) / kSelWaves + 63) / 64 * 64;
      const int64_t c0 = s0 + per * wv < e0 ? s0 + per * wv : e0;
      const int64_t c1 = c0 + per < e0 ? c0 + per : e0;
      // counting pass: each key of the wave's range is replaced by its candidate id with the
      // class in the top bits (bit 31: above T, bit 30: equal to T). Ids of levels >= 1 are
      // below N / p < 2^30, as the host keeps the pyramid below 2^31 rows. The writing pass
      // then makes no global reads. Ids are loaded kB chunks at a time, all in flight together.
      int gt_w = 0, eq_w = 0;
      for (int64_t b0 = c0; b0 < c1; b0 += 64 * kB) {
        int32_t ids[kB];
#pragma unroll
        for (int j = 0; j < kB; ++j) {
          const int64_t u = b0 + 64 * j + lane;
          ids[j] = u < c1 ? Cl[u] : 0;
        }
#pragma unroll
        for (int j = 0; j < kB; ++j) {
          const int64_t u = b0 + 64 * j + lane;
          const uint32_t key = u < c1 ? keys[u] : 0u;
          const bool gt = u < c1 && key > T, eq = u < c1 && key == T;
          gt_w += __popcll(__ballot(gt));
          eq_w += __popcll(__ballot(eq));
          if (u < c1) keys[u] = (uint32_t)ids[j] | (gt ? 0x80000000u : 0u) | (eq ? 0x40000000u : 0u);
        }
      }
      if (lane == 0) {
        wave_gt[wv] = gt_w;
        wave_eq[wv] = eq_w;
      }
      if (GK) __threadfence_block();  // the keys rewritten above are read by the same wave below
      __syncthreads();
      int gt_rank = 0, eq_rank = 0;  // candidates of the earlier waves
      for (int i = 0; i < wv; ++i) {
        gt_rank += wave_gt[i];
        eq_rank += wave_eq[i];
      }
      const uint64_t below = (1ull << lane) - 1ull;
      for (int64_t base = c0; base < c1; base += 64) {
        const int64_t u = base + lane;
        const uint32_t e = u < c1 ? keys[u] : 0u;
        const bool gt = e >> 31, eq = (e >> 30) & 1u;
        const uint64_t bg = __ballot(gt);
        const uint64_t be = __ballot(eq);
        const int gr = gt_rank + __popcll(bg & below);
        const int er = eq_rank + __popcll(be & below);
        if (gt || (eq && er < need)) {
          const int64_t pos = first + gr + (er < need ? er : need);
          const int32_t i = (int32_t)(e & 0x3fffffffu);
          // one chunk: every id of the level was read before this pass, so the list can be
          // overwritten in place (several chunks reload it after the level)
          if (p == 4 && vec4) {
            const u32x4 v = {(uint32_t)(i * 4), (uint32_t)(i * 4 + 1), (uint32_t)(i * 4 + 2), (uint32_t)(i * 4 + 3)};
            *reinterpret_cast<u32x4*>(Cn + pos * 4) = v;
            if (ln && !a.stratified) *reinterpret_cast<u32x4*>(list + pos * 4) = v;
          } else {
            for (int r = 0; r < p; ++r) {
              Cn[pos * p + r] = i * p + r;
              if (ln && !a.stratified) list[pos * p + r] = i * p + r;
            }
          }
        }
        gt_rank += __popcll(bg);
        eq_rank += __popcll(be);
      }
      __syncthreads();  // sel_state and hist are reused by the next chunk
    }
    if (!LL || (ln && a.stratified)) __threadfence_block();
    __syncthreads();
    if (ln && a.stratified) {  // the next level's list, from the workspace just written
      for (int64_t u = tid; u < a.cand[l - 1]; u += kSelThreads) list[u] = Cn[u];
      __syncthreads();
    }
  }
}

struct OrdArgs {
  const int32_t* ws;
  int32_t* idx;   // [B, Hs, S]
  int32_t* slot;  // [B, Hs, Ptot]
  int64_t Scand;
  int32_t Ptot, S, N, L, p, replace;
  int32_t lsh[16];   // l log2(p) when p is a power of two, else -1
  int32_t pw[16];    // p^l
  int32_t off[17];   // flattened id of entry (l, 0)
  int32_t cand[16];  // candidates of level l
  int32_t coff[17];  // offset of level l's list in a selection's workspace row
};

// floor(x / p^l) for 0 <= x < 2^31
__device__ __forceinline__ int32_t div_pw(int32_t x, int l, const OrdArgs& a) {
  return a.lsh[l] >= 0 ? x >> a.lsh[l] : (int32_t)((uint32_t)x / (uint32_t)a.pw[l]);
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

// Window ends and threads per workgroup of order_kernel.
constexpr int kOrdE = 8192;
constexpr int kOrdThreads = 512;
constexpr int kOrdWaves = kOrdThreads / 64;

// order_kernel: workgroup x of a selection owns the window ends e in [e0, e1), e0 = x kOrdE:
// the level-l entries i in [floor(e0 / p^l), floor(e1 / p^l)), a contiguous part of each level's
// sorted candidate list. Ranks follow key = e L + (L - 1 - l), so an entry's rank is
//   (emitted entries whose window ends before e0) + (its position among the range's entries),
// the first term the sum of the lists' lower bounds at floor(e0 / p^l) (less the parents below
// them in replace mode), the second an exclusive scan over a flag per (e - e0, L - 1 - l). The
// workgroup then writes slot for every pyramid entry of its range (its rank, or -1) and idx for
// the emitted ones. No workgroup depends on another.
template <int NL>  // NL = L
__global__ void __launch_bounds__(kOrdThreads) order_kernel(OrdArgs a) {
  constexpr int NF = kOrdE * NL;  // flags of the range, one bit each
  constexpr int NW = NF / 32;     // flag words
  constexpr int NS = 3 * NL;      // lower bounds to find: lo, hi, parents below (replace)
  constexpr int NSW = (NS + kOrdWaves - 1) / kOrdWaves;
  __shared__ uint32_t fl[NW];
  __shared__ uint16_t wpre[NW];  // emitted entries of the range before flag word w
  __shared__ int32_t bnd[NS];
  __shared__ int32_t wsum[kOrdWaves];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int32_t* C = a.ws + bh * a.Scand;
  const int32_t e0 = (int32_t)blockIdx.x * kOrdE;
  const int32_t e1 = a.N - e0 < kOrdE ? a.N : e0 + kOrdE;
  for (int x = tid; x < NW; x += blockDim.x) fl[x] = 0u;
  // Lower bounds, 64-ary per wave: search j = wv + kOrdWaves r. j < NL: list j at floor(e0 / p^j);
  // j < 2 NL: list j - NL at floor(e1 / p^(j - NL)); else (replace, l = j - 2 NL >= 1): list
  // l - 1 at p floor(e0 / p^l), whose children count gives the parents of level l below e0.
  {
    int32_t slo[NSW], shi[NSW], sl[NSW], sx[NSW];
#pragma unroll
    for (int r = 0; r < NSW; ++r) {
      const int j = wv + kOrdWaves * r;
      const int l = j < NL ? j : j < 2 * NL ? j - NL : j - 2 * NL;
      bool live = j < NS;
      if (j >= 2 * NL) live = live && a.replace && l >= 1;
      sx[r] = j < NL ? div_pw(e0, l, a) : j < 2 * NL ? div_pw(e1, l, a) : div_pw(e0, l, a) * a.p;
      sl[r] = j >= 2 * NL ? (l >= 1 ? l - 1 : 0) : l;
      slo[r] = 0;
      shi[r] = live ? a.cand[sl[r]] : 0;
    }
    for (;;) {
      bool open = false;
      int32_t v[NSW];
#pragma unroll
      for (int r = 0; r < NSW; ++r) {
        v[r] = 0;
        if (slo[r] < shi[r]) {  // uniform over the wave
          const int32_t st = (shi[r] - slo[r] + 63) >> 6;
          const int32_t pos = slo[r] + lane * st;
          if (pos < shi[r]) v[r] = C[a.coff[sl[r]] + pos];
          open = true;
        }
      }
      if (!open) break;
#pragma unroll
      for (int r = 0; r < NSW; ++r) {
        if (slo[r] < shi[r]) {
          const int32_t n = shi[r] - slo[r], st = (n + 63) >> 6, T = (n + st - 1) / st;
          const int32_t pos = slo[r] + lane * st;
          const bool below = pos < shi[r] && v[r] < sx[r];
          const int32_t c = (int32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(below));
          const int32_t nlo = c > 0 ? slo[r] + (c - 1) * st + 1 : slo[r];
          const int32_t nhi = c < T ? slo[r] + c * st : shi[r];
          slo[r] = nlo, shi[r] = nhi;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < NSW; ++r) {
      const int j = wv + kOrdWaves * r;
      if (lane == 0 && j < NS) bnd[j] = slo[r];
    }
  }
  __syncthreads();
  // flag every emitted entry of the range (a parent is not emitted in replace mode); a thread
  // loads MB list entries before marking any, so their loads are in flight together
  int total = 0;
#pragma unroll
  for (int l = 0; l < NL; ++l) total += bnd[NL + l] - bnd[l];
  constexpr int MB = 4;
  for (int t0 = 0; t0 < total; t0 += MB * (int)blockDim.x) {
    int32_t iv[MB], lv[MB];
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      const int t = t0 + m * (int)blockDim.x + tid;
      lv[m] = -1;
      iv[m] = 0;
      if (t < total) {
        int l = 0, u = t;
        while (u >= bnd[NL + l] - bnd[l]) u -= bnd[NL + l] - bnd[l], ++l;
        lv[m] = l;
        iv[m] = C[a.coff[l] + bnd[l] + u];
      }
    }
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      const int l = lv[m];
      if (l < 0) continue;
      const int32_t i = iv[m];
      if (a.replace && l >= 1) {
        // a parent's children are in the next finer candidate list
        const int64_t c = lower_bound_val(C + a.coff[l - 1], a.cand[l - 1], (int64_t)i * a.p);
        if (c < a.cand[l - 1] && C[a.coff[l - 1] + c] == i * a.p) continue;
      }
      const int x = ((i + 1) * a.pw[l] - 1 - e0) * NL + (NL - 1 - l);
      atomicOr(&fl[x >> 5], 1u << (x & 31));
    }
  }
  __syncthreads();
  // exclusive scan of the flags by words: thread tid owns words [tid CW, tid CW + CW) of the NW
  constexpr int CW = (NW + kOrdThreads - 1) / kOrdThreads;
  static_assert(NF <= 65536, "ranks within a range fit 16 bits");
  int run = 0;
#pragma unroll
  for (int x = 0; x < CW; ++x)
    if (tid * CW + x < NW) run += (int)__builtin_popcount(fl[tid * CW + x]);
  int inc = run;  // inclusive scan over the wave
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(inc, d, 64);
    if (lane >= d) inc += y;
  }
  if (lane == 63) wsum[wv] = inc;
  __syncthreads();
  int base = inc - run;
  for (int w = 0; w < wv; ++w) base += wsum[w];
#pragma unroll
  for (int x = 0; x < CW; ++x) {
    if (tid * CW + x >= NW) break;
    wpre[tid * CW + x] = (uint16_t)base;
    base += (int)__builtin_popcount(fl[tid * CW + x]);
  }
  // emitted entries whose window ends before e0
  int32_t r0 = 0;
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    r0 += bnd[l];
    if (a.replace && l >= 1) r0 -= bnd[2 * NL + l] / a.p;
  }
  __syncthreads();
  // slot of every pyramid entry of the range; idx of the emitted ones
  int32_t* idxh = a.idx + bh * a.S;
  int32_t* sloth = a.slot + bh * a.Ptot;
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    const int32_t i0 = div_pw(e0, l, a), i1 = div_pw(e1, l, a);
    for (int32_t i = i0 + tid; i < i1; i += blockDim.x) {
      const int x = ((i + 1) * a.pw[l] - 1 - e0) * NL + (NL - 1 - l);
      const uint32_t word = fl[x >> 5], sh = (uint32_t)(x & 31);
      int32_t out = -1;
      if ((word >> sh) & 1u) {
        const int32_t rr = r0 + wpre[x >> 5] + (int32_t)__builtin_popcount(word & ((1u << sh) - 1u));
        if (rr < a.S) {  // cannot fail for lists written by select_kernel
          out = rr;
          idxh[rr] = a.off[l] + i;
        }
      }
      sloth[a.off[l] + i] = out;
    }
  }
}

}  // namespace lh

using namespace lh;

hipError_t lh_launch_select(const LhShape& s, const float* s_qk, const float* s_kq, int32_t* idx,
                            int32_t* slot, int32_t* ws, hipStream_t st) {
  const int64_t BH = s.B * s.Hs;  // one selection per (b, selection head)
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
  a.coff_aligned4 = 1;
  for (int l = 0; l <= s.L; ++l) a.coff_aligned4 &= (s.coff[l] % 4 == 0) ? 1 : 0;
  a.maxsel = s.maxsel;
  a.gkeys = s.maxsel > kSelLdsKeys ? reinterpret_cast<uint32_t*>(ws + BH * s.Scand) : nullptr;
  int64_t lmax = 0;  // the longest list select_kernel reads (levels >= 1)
  for (int l = 1; l < s.L; ++l) lmax = s.cand[l] > lmax ? s.cand[l] : lmax;
  if (a.gkeys) {
    hipLaunchKernelGGL((select_kernel<true, false>), dim3((unsigned)BH), dim3(kSelThreads), 0, st, a);
  } else if (lmax <= kSelLdsList && s.maxsel <= kSelLdsList) {
    const size_t shm = 2 * (size_t)kSelLdsList * sizeof(uint32_t);
    hipLaunchKernelGGL((select_kernel<false, true>), dim3((unsigned)BH), dim3(kSelThreads), shm, st, a);
  } else {
    const size_t shm = (size_t)(s.maxsel > 0 ? s.maxsel : 1) * sizeof(uint32_t);
    hipLaunchKernelGGL((select_kernel<false, false>), dim3((unsigned)BH), dim3(kSelThreads), shm, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  OrdArgs o;
  o.ws = ws;
  o.idx = idx;
  o.slot = slot;
  o.Scand = s.Scand;
  o.Ptot = (int32_t)s.Ptot;
  o.S = (int32_t)s.S;
  o.N = (int32_t)s.N;
  o.L = s.L;
  o.p = s.p;
  o.replace = (s.flags & LH_FLAG_REPLACE_PARENTS) ? 1 : 0;
  int pl = 0;
  while ((1 << pl) < s.p) ++pl;
  const bool pow2 = (1 << pl) == s.p;
  for (int l = 0; l < 17; ++l) o.off[l] = (int32_t)s.off[l], o.coff[l] = (int32_t)s.coff[l];
  for (int l = 0; l < 16; ++l) {
    o.pw[l] = l < s.L ? (int32_t)s.pw[l] : 1;
    o.cand[l] = (int32_t)s.cand[l];
    o.lsh[l] = pow2 ? l * pl : -1;
  }
  dim3 grid((unsigned)((s.N + kOrdE - 1) / kOrdE), (unsigned)BH);
  switch (s.L) {
    case 1: hipLaunchKernelGGL(order_kernel<1>, grid, dim3(kOrdThreads), 0, st, o); break;
    case 2: hipLaunchKernelGGL(order_kernel<2>, grid, dim3(kOrdThreads), 0, st, o); break;
    case 3: hipLaunchKernelGGL(order_kernel<3>, grid, dim3(kOrdThreads), 0, st, o); break;
    case 4: hipLaunchKernelGGL(order_kernel<4>, grid, dim3(kOrdThreads), 0, st, o); break;
    case 5: hipLaunchKernelGGL(order_kernel<5>, grid, dim3(kOrdThreads), 0, st, o); break;
    case 6: hipLaunchKernelGGL(order_kernel<6>, grid, dim3(kOrdThreads), 0, st, o); break;
    case 7: hipLaunchKernelGGL(order_kernel<7>, grid, dim3(kOrdThreads), 0, st, o); break;
    case 8: hipLaunchKernelGGL(order_kernel<8>, grid, dim3(kOrdThreads), 0, st, o); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
