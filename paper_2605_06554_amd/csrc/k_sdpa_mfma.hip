// k_sdpa_mfma.hip -- bf16 causal SDPA on the gathered sub-sequence with gfx950 MFMA
// (Sec. 3.5, Eq. attn-sub with Eq. sdpa): forward, and the deterministic backward
// (a dK/dV kernel and a dQ kernel), per (b, hq) over [S, D] rows.
//
// Numerics: v_mfma_f32_32x32x16_bf16 with fp32 accumulation; the softmax runs in the exp2
// domain with the scale folded into one FMA; P and dS are rounded to bf16 for their products.
// The forward rescales its accumulator only when the running row maximum grows by more than
// 2^8 (the final O / l uses the same maximum throughout, so the result is unchanged).
//
// Layout facts used throughout (lane l of a wave, h = l / 32):
//   MFMA 32x32x16: A[m = l % 32][k = 8h + 0..7], B[k = 8h + 0..7][n = l % 32],
//                  C[m = 8(i/4) + 4h + i%4][n = l % 32], i = 0..15.
//   Forward and dQ compute S^T = K Q^T, so each lane owns one query row; dK/dV computes
//   S = Q K^T, so each lane owns one key. The k-order inside every 16-row MFMA step follows
//   the C layout (slots 0-3 = rows 4h + 0..3, slots 4-7 = rows 8 + 4h + 0..3), so an
//   accumulator converted to bf16 is directly the next product's operand; the matching
//   transposed operand is read from the row-major LDS tile with ds_read_b64_tr_b16.
//
// LDS tiles: rows of D bf16 (2D bytes, no padding) with an XOR swizzle of 16-byte chunks
// (chunk c of row r sits at position c ^ swz(r)), filled straight from global memory with
// global_load_lds_dwordx4 (no staging registers), double-buffered so the next tile streams in
// while the current one is used. All three kernels use a swizzle under which both read
// patterns are bank-conflict free (measured with SQ_LDS_BANK_CONFLICT): 16 consecutive rows
// reading one logical chunk (b128 operand reads) land on 16 different chunk positions, and the
// 4 consecutive rows of a transposed read, each reading an aligned group of 4 chunks, land in 4
// different groups. Every lane's LDS offsets are computed once; tile bases are compile-time
// constants (the tile loop is unrolled over the ring of slots).
//
// Occupancy: the forward runs 12 waves per workgroup, 3 per SIMD (at most 168 registers), so
// that two waves can be in their softmax while a third feeds the MFMA unit. The two backward
// kernels hold 128 (dK/dV) or 160 (dQ) accumulator and operand registers per lane and run 2
// waves per SIMD.
//
// Pipeline: each kernel keeps an NS-slot ring of tiles in LDS. Before using tile t, a wave
// waits until at most (NS - 2) tiles' worth of its own LDS-DMA loads are outstanding (vmcnt
// counts this wave's loads in issue order), then the block barrier publishes tile t from every
// wave; right after the barrier the loads of tile t + NS - 1 go into the slot tile t - 1 used.
// Every wave issues the same number of loads per tile (loads past the end read clamped rows
// into the free slot), so the wait count is a compile-time constant.
#include <type_traits>

#include "lh_common.h"

#ifndef LH_FW
#define LH_FW 12  // forward: waves per workgroup (32 query rows each)
#endif
#ifndef LH_FEU
#define LH_FEU 3  // forward: waves per SIMD the register budget targets
#endif
#ifndef LH_FK
#define LH_FK 64  // forward: keys per tile
#endif
#ifndef LH_QW
#define LH_QW 8  // dQ: waves per workgroup (32 query rows each)
#endif
#ifndef LH_BK
#define LH_BK 64  // dQ: keys per tile
#endif
#ifndef LH_KWV
#define LH_KWV 8  // dK/dV: waves per workgroup (32 keys each)
#endif
#ifndef LH_KWV_EU
#define LH_KWV_EU 2  // dK/dV: waves per SIMD the register budget targets
#endif
#ifndef LH_CQ
#define LH_CQ 64  // dK/dV: query rows per tile
#endif
#ifndef LH_ORDER
#define LH_ORDER 1  // 1: blocks ordered by work across all heads (longest first); 0: head by head
#endif
#ifndef LH_FNS
#define LH_FNS 2  // forward: tile slots in the LDS ring
#endif
#ifndef LH_QNS
#define LH_QNS 2  // dQ: tile slots in the LDS ring
#endif

namespace lh {

typedef s16x4 __attribute__((address_space(3))) lds_s16x4;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescale = 8.0f;  // lazy rescaling threshold (log2 units)

template <int N>
using IC = std::integral_constant<int, N>;

// D = 128 (16 chunks per row): swap the two 2-bit halves of r % 16.
// D = 64 (8 chunks per row, two rows per 256-byte bank line): a bijection of (r / 2) % 8 whose
// top bit follows bit 1 of r.
// Two swizzles of the 16-byte chunks of a row (SW below):
//   SW = 2: a bijection of r % 16, so the 16 lanes that read one logical chunk of 16 consecutive
//           rows hit 16 different chunk positions: row and transposed reads are conflict free;
//   SW = 3: depends on r % 8 only, so rows r and r + 8 share it and a transposed read of rows
//           r0 + 8 is the read of rows r0 shifted by a constant (one lane offset fewer per
//           column block), at the price of a 2-way bank conflict on the row reads.
// D = 64 (8 chunks per row, two rows per 256-byte bank line): a bijection of (r / 2) % 8 whose
// top bit follows bit 1 of r (SW = 2), or of (r / 2) % 4 (SW = 3).
#ifndef LH_SWZ_F
#define LH_SWZ_F 2  // forward
#endif
#ifndef LH_SWZ_Q
#define LH_SWZ_Q 2  // dQ
#endif
#ifndef LH_SWZ_K
#define LH_SWZ_K 2  // dK/dV
#endif
template <int D, int SW>
__device__ __forceinline__ int swz(int r) {
  if constexpr (SW == 2) {
    if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
    else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
  } else {
    if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 1);
    else return (((r >> 1) & 1) << 2) | ((r >> 2) & 1);
  }
}

// Byte offsets of one lane inside any swizzled tile (row blocks start at multiples of 16).
template <int D>
struct LaneOff {
  int row[D / 16];  // row operand (A or B) of k-step kk: row l % 32, columns 16 kk + 8h .. +7
  int trl[D / 32];  // transposed operand, column block d, rows 4h + (l % 16) / 4 (slots 0-3)
  int trh[D / 32];  // the same 8 rows further (slots 4-7)
};

template <int D, int SW>
__device__ __forceinline__ LaneOff<D> lane_offsets(int lane) {
  constexpr int RB = 2 * D;
  LaneOff<D> o;
  const int h = lane >> 5, r = lane & 31;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) o.row[kk] = r * RB + (((2 * kk + h) ^ swz<D, SW>(r)) << 4);
  const int r0 = 4 * h + ((lane & 15) >> 2);
#pragma unroll
  for (int d = 0; d < D / 32; ++d) {
    const int chunk = 4 * d + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
    o.trl[d] = r0 * RB + ((chunk ^ swz<D, SW>(r0)) << 4) + 8 * (lane & 1);
    o.trh[d] = (r0 + 8) * RB + ((chunk ^ swz<D, SW>(r0 + 8)) << 4) + 8 * (lane & 1);
  }
  return o;
}

// Row operand at byte offset `off` (lane offset plus a constant) of an LDS tile.
__device__ __forceinline__ bf16x8 row8(const bf16_t* tile, int off) {
  return *reinterpret_cast<const bf16x8*>(reinterpret_cast<const char*>(tile) + off);
}

// Transposed operand: within each 16-lane group, lane i receives Mat[r0 + j][c0 + i] (j = 0..3)
// from the lanes' addresses (lane s points at Mat[r0 + s / 4][c0 + 4 (s % 4)]); two reads give
// slots 0-3 (rows +0..3) and 4-7 (rows +8..11).
__device__ __forceinline__ bf16x8 tr8(const bf16_t* tile, int off_lo, int off_hi) {
  typedef __attribute__((__vector_size__(8 * sizeof(short)))) short s16x8;
  const char* p = reinterpret_cast<const char*>(tile);
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + off_lo));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + off_hi));
  s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x8 cvt8(const float* f) {
  typedef __attribute__((__vector_size__(8 * sizeof(float)))) float f32x8;
  f32x8 v = {f[0], f[1], f[2], f[3], f[4], f[5], f[6], f[7]};
  return __builtin_convertvector(v, bf16x8);
}

__device__ __forceinline__ bf16x8 gld8(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

// Direct global -> LDS copy of TR rows starting at row r0 of a [S, D] bf16 matrix into a
// swizzled tile by the NW waves of the block. A wave instruction writes 1 KB of LDS
// contiguously (lane i -> byte 16 i), so every lane fetches the logical chunk that belongs at
// its physical position. Rows past S are clamped to row S - 1 (callers mask them out). Every
// wave issues loads_per_wave<D, TR, NW>() instructions; when the 1 KB blocks do not divide
// evenly, the extra instructions repeat a block another wave also writes (same bytes).
template <int D, int TR, int NW>
__device__ __forceinline__ constexpr int loads_per_wave() { return (TR * D / 512 + NW - 1) / NW; }

template <int D, int TR, int NW, int SW, bool CLAMP>
__device__ __forceinline__ void load_tile_rows(bf16_t* tile, const bf16_t* src, int r0, int S, int w, int lane) {
  constexpr int CPR = D / 8;
  constexpr int BLOCKS = TR * CPR / 64;  // 1 KB blocks of the tile
  static_assert(BLOCKS * 64 == TR * CPR, "a tile is a whole number of 1 KB blocks");
  const char* base = reinterpret_cast<const char*>(src + (int64_t)r0 * D);
#pragma unroll
  for (int j = 0; j < loads_per_wave<D, TR, NW>(); ++j) {
    int blk = j * NW + w;
    if (BLOCKS % NW != 0 && blk >= BLOCKS) blk -= BLOCKS;
    const int pos = blk * 64 + lane;
    const int r = pos / CPR;
    const int c = (pos % CPR) ^ swz<D, SW>(r);
    // rows past S read row S - 1; the clamp stays a 32-bit lane offset from the tile's uniform
    // base, so no lane holds a 64-bit address (fewer live registers in every kernel)
    const int rr = CLAMP ? (r < S - 1 - r0 ? r : S - 1 - r0) : r;
    const char* g = base + (int32_t)((rr * D + c * 8) * 2);
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                     (__attribute__((address_space(3))) void*)(tile + blk * 512), 16, 0, 0);
  }
}

// r0 and w are uniform: a tile that lies inside the matrix is one scalar base address plus a
// fixed 32-bit offset per lane; only a tile that crosses row S clamps row by row.
template <int D, int TR, int NW, int SW>
__device__ __forceinline__ void load_tile(bf16_t* tile, const bf16_t* src, int r0, int S, int w, int lane) {
  if (r0 + TR <= S) load_tile_rows<D, TR, NW, SW, false>(tile, src, r0, S, w, lane);
  else load_tile_rows<D, TR, NW, SW, true>(tile, src, r0, S, w, lane);
}

// Index-driven rows (the gather fused into the loads). Row m of a gathered head is pyramid id
// idx[m]: ids below N are rows of the input [B, N, H, D], the rest rows of the pyramid
// [B, R, H, D]. Ids outside [0, N + R) are clamped into it (never an out-of-range read).
struct SdpaIdx {
  const bf16_t *q, *k, *v, *qp, *kp, *vp;
  const int32_t* idx;  // [B, Hq, S]
  int64_t N, R;
  int32_t Hq, Hkv, G;
};

// Query heads and selection heads: query head hq reads the gathered K~, V~ (and idx) of
// selection head hq / Gq; there are Hs selection heads per batch (Hs = Hq, Gq = 1 when every
// query head selects on its own).
struct HeadMap {
  int32_t Hq, Hs, Gq;
};

// Block order. Blocks are dispatched in linear-id order and go round-robin to the 8 XCDs. With
// LH_ORDER = 1 linear id = rank * heads + head, where rank 0 is the longest block of a head
// (most causal tiles): the longest blocks of every head start first, so no long block is left
// to run alone at the end, and (heads being a multiple of 8) every block of a head lands on the
// same XCD, whose L2 then holds that head's streamed tiles.
struct BlockPos {
  int rank;      // 0 = the head's longest block
  int64_t head;  // blockIdx.y of the head-by-head order
};
__device__ __forceinline__ BlockPos block_pos() {
  if (LH_ORDER) {
    const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    return BlockPos{(int)(lin / gridDim.y), lin % gridDim.y};
  }
  return BlockPos{(int)blockIdx.x, (int64_t)blockIdx.y};
}

struct RowSrc {
  const char* l0;  // row 0 of the head in the input
  const char* py;  // row 0 of the head in the pyramid, less N rows: pyramid id i is at py + i rb
  uint32_t rb;     // bytes between consecutive rows: H * D * 2
  int32_t N, last;  // last = N + R - 1
};

__device__ __forceinline__ RowSrc row_src(const bf16_t* x, const bf16_t* pyr, int64_t b, int h, int H,
                                          const SdpaIdx& ix, int D) {
  RowSrc r;
  r.rb = (uint32_t)(H * D * 2);
  r.l0 = reinterpret_cast<const char*>(x + (b * ix.N * H + h) * D);
  r.py = reinterpret_cast<const char*>(pyr + (b * ix.R * H + h) * D) - (int64_t)ix.N * r.rb;
  r.N = (int32_t)ix.N;
  r.last = (int32_t)(ix.N + ix.R - 1);
  return r;
}

// One clamp (a median of three), one compare with two selects for the base, one 32 x 32 -> 64-bit
// multiply-add.
__device__ __forceinline__ const bf16_t* rs_row(const RowSrc& s, int32_t id) {
  id = id < 0 ? 0 : id > s.last ? s.last : id;
  const char* base = id < s.N ? s.l0 : s.py;
  return reinterpret_cast<const bf16_t*>(base + (uint64_t)(uint32_t)id * s.rb);
}

// Pyramid ids of the rows this lane copies in load_tile (rows past S take row S - 1's id).
template <int D, int TR, int NW>
__device__ __forceinline__ void tile_ids(const int32_t* idxh, int r0, int S, int w, int lane, int32_t* ids) {
  constexpr int CPR = D / 8;
  constexpr int BLOCKS = TR * CPR / 64;
#pragma unroll
  for (int j = 0; j < loads_per_wave<D, TR, NW>(); ++j) {
    int blk = j * NW + w;
    if (BLOCKS % NW != 0 && blk >= BLOCKS) blk -= BLOCKS;
    const int gr = r0 + (blk * 64 + lane) / CPR;
    ids[j] = idxh[gr < S ? gr : S - 1];
  }
}

// load_tile with every row read from its pyramid id.
template <int D, int TR, int NW, int SW>
__device__ __forceinline__ void load_tile_idx(bf16_t* tile, const RowSrc& src, const int32_t* ids, int w, int lane) {
  constexpr int CPR = D / 8;
  constexpr int BLOCKS = TR * CPR / 64;
#pragma unroll
  for (int j = 0; j < loads_per_wave<D, TR, NW>(); ++j) {
    int blk = j * NW + w;
    if (BLOCKS % NW != 0 && blk >= BLOCKS) blk -= BLOCKS;
    const int pos = blk * 64 + lane;
    const int c = (pos % CPR) ^ swz<D, SW>(pos / CPR);
    const bf16_t* g = rs_row(src, ids[j]) + c * 8;
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                     (__attribute__((address_space(3))) void*)(tile + blk * 512), 16, 0, 0);
  }
}

// Waits until at most N of this wave's vector-memory loads are outstanding and every LDS
// access of the wave has completed (s_waitcnt vmcnt(N) lgkmcnt(0)), then joins the block
// barrier. The empty asm statements keep the compiler from moving memory accesses across.
template <int N>
__device__ __forceinline__ void sync_tiles() {
  static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Ring slots are separate __shared__ arrays (not one indexed array), so the compiler can tell
// that a load streaming into one slot does not alias reads of another and does not wait for it.
#define LH_RING(T, name, n)                                                   \
  __shared__ __align__(16) T name##0[n], name##1[n], name##2[n], name##3[n]; \
  T* const name[4] = {name##0, name##1, name##2, name##3}

// Calls f(IC<slot>{}, t) for t = t0 .. min(t0 + NS, n) - 1 with slot = t - t0 (compile-time).
template <int I, int NS>
struct SlotLoop {
  template <typename F>
  static __device__ __forceinline__ void run(int t0, int n, F& f) {
    if (t0 + I < n) {
      f(IC<I>{}, t0 + I);
      SlotLoop<I + 1, NS>::run(t0, n, f);
    }
  }
};
template <int NS>
struct SlotLoop<NS, NS> {
  template <typename F>
  static __device__ __forceinline__ void run(int, int, F&) {}
};

// Calls f(IC<t % 2>{}, t) for t = begin .. end - 1: a loop over a two-slot ring that may start
// on either slot.
template <typename F>
__device__ __forceinline__ void ring2_loop(int begin, int end, F& f) {
  int t = begin;
  if (t < end && (t & 1)) {
    f(IC<1>{}, t);
    ++t;
  }
  for (; t + 1 < end; t += 2) {
    f(IC<0>{}, t);
    f(IC<1>{}, t + 1);
  }
  if (t < end) f(IC<0>{}, t);
}

// Stores a lane's O^T-layout accumulator row (query row q, columns 32 d + 8 g + 4h + 0..3).
template <int D>
__device__ __forceinline__ void store_qrow(bf16_t* row, const f32x16* acc, float mul, int h) {
#pragma unroll
  for (int d = 0; d < D / 32; ++d)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col = 32 * d + 8 * g + 4 * h;
      const uint32_t w0 = (uint32_t)f2bf(acc[d][4 * g + 0] * mul) | ((uint32_t)f2bf(acc[d][4 * g + 1] * mul) << 16);
      const uint32_t w1 = (uint32_t)f2bf(acc[d][4 * g + 2] * mul) | ((uint32_t)f2bf(acc[d][4 * g + 3] * mul) << 16);
      *reinterpret_cast<uint2*>(row + col) = make_uint2(w0, w1);
    }
}

// ------------------------------------------------------------------ forward
constexpr int FW = LH_FW, FQ = 32 * LH_FW, FK = LH_FK, FNS = LH_FNS;

// IDX: Q, K, V are unused; rows come from the input / pyramid through ix.idx.
template <int D, bool IDX>
__global__ void __launch_bounds__(64 * FW) __attribute__((amdgpu_waves_per_eu(LH_FEU, LH_FEU)))
sdpa_fwd_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
              bf16_t* __restrict__ O, float* __restrict__ LSE, int S, float sl2, SdpaIdx ix, HeadMap hm) {
  constexpr int RB = 2 * D;
  constexpr int NB = FK / 32;  // 32-key blocks per tile
  constexpr int LPT = 2 * loads_per_wave<D, FK, FW>();
  static_assert(FNS >= 2 && FNS <= 4, "ring of 2 to 4 slots");
  LH_RING(bf16_t, Ks, FK * D);
  LH_RING(bf16_t, Vs, FK * D);
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, r32 = lane & 31;
  const BlockPos bp = block_pos();
  const int64_t bh = bp.head;
  const int nqt = (S + FQ - 1) / FQ;
  const int q0 = (nqt - 1 - bp.rank) * FQ;  // longest rows first
  const int qw = q0 + 32 * w;
  const int myq = qw + r32;
  const int64_t kvh = (bh / hm.Hq) * hm.Hs + (bh % hm.Hq) / hm.Gq;  // selection head
  const bf16_t* Qh = Q + bh * S * D;
  const bf16_t* Kh = K + kvh * S * D;
  const bf16_t* Vh = V + kvh * S * D;
  const LaneOff<D> lo = lane_offsets<D, LH_SWZ_F>(lane);
  constexpr int LPW = loads_per_wave<D, FK, FW>();
  RowSrc qsrc{}, ksrc{}, vsrc{};
  const int32_t* idxh = nullptr;
  int32_t kv_ids[LPW];  // ids of the next tile to be loaded
  if constexpr (IDX) {
    const int64_t b = bh / ix.Hq;
    const int hq = (int)(bh - b * ix.Hq), g = hq / ix.G;
    qsrc = row_src(ix.q, ix.qp, b, hq, ix.Hq, ix, D);
    ksrc = row_src(ix.k, ix.kp, b, g, ix.Hkv, ix, D);
    vsrc = row_src(ix.v, ix.vp, b, g, ix.Hkv, ix, D);
    idxh = ix.idx + kvh * S;
  }
  auto load_kv = [&](int slot_, int r0) __attribute__((always_inline)) {
    bf16_t* kt_ = slot_ == 0 ? Ks[0] : slot_ == 1 ? Ks[1] : slot_ == 2 ? Ks[2] : Ks[3];
    bf16_t* vt_ = slot_ == 0 ? Vs[0] : slot_ == 1 ? Vs[1] : slot_ == 2 ? Vs[2] : Vs[3];
    if constexpr (IDX) {
      load_tile_idx<D, FK, FW, LH_SWZ_F>(kt_, ksrc, kv_ids, w, lane);
      load_tile_idx<D, FK, FW, LH_SWZ_F>(vt_, vsrc, kv_ids, w, lane);
      tile_ids<D, FK, FW>(idxh, r0 + FK, S, w, lane, kv_ids);  // the tile after this one
    } else {
      load_tile<D, FK, FW, LH_SWZ_F>(kt_, Kh, r0, S, w, lane);
      load_tile<D, FK, FW, LH_SWZ_F>(vt_, Vh, r0, S, w, lane);
    }
  };
  if constexpr (IDX) tile_ids<D, FK, FW>(idxh, 0, S, w, lane, kv_ids);

  const int kend = q0 + FQ < S ? q0 + FQ : S;
  const int nkt = (kend + FK - 1) / FK;
  bf16x8 qreg[D / 16];
  const int qrow = myq < S ? myq : S - 1;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    const bf16_t* qr = IDX ? rs_row(qsrc, idxh[qrow]) : Qh + (int64_t)qrow * D;
    qreg[kk] = gld8(qr + 16 * kk + 8 * h);
  }
#pragma unroll
  for (int t = 0; t < FNS - 1; ++t) load_kv(t, t * FK);
  f32x16 oacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) oacc[d] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;

  auto step = [&](auto slotc, int kt) {
    constexpr int SL = decltype(slotc)::value;
    constexpr int NX = (SL + FNS - 1) % FNS;  // slot of tile kt + FNS - 1 (tile kt - 1's)
    sync_tiles<(FNS - 2) * LPT>();  // tile kt landed in every wave; tile kt - 1 is done
    load_kv(NX, (kt + FNS - 1) * FK);
    const int k0 = kt * FK;
    if (qw + 31 < k0) return;  // every key of the tile is in the future of this wave's rows
    const bf16_t* Kt = Ks[SL];
    const bf16_t* Vt = Vs[SL];
    f32x16 sacc[NB];
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) sacc[kb] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int kb = 0; kb < NB; ++kb) sacc[kb] = mfma32(row8(Kt, kb * 32 * RB + lo.row[kk]), qreg[kk], sacc[kb]);
    if (k0 + FK - 1 > qw) {  // diagonal tile: mask keys after the row
#pragma unroll
      for (int kb = 0; kb < NB; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (k0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3) > myq) sacc[kb][i] = -INFINITY;
    }
    float mloc = sacc[0][0];
#pragma unroll
    for (int kb = 0; kb < NB; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mloc = fmaxf(mloc, sacc[kb][i]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * sl2;
    if (mloc > m_run + kRescale) {  // new running maximum: rescale what was accumulated
      const float alpha = __builtin_amdgcn_exp2f(m_run - mloc);
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[d][i] *= alpha;
      m_run = mloc;
    }
    // P of 16 keys at a time. Step st + 1's softmax (independent of step st's MFMAs) is
    // scheduled between step st's four P V MFMAs, each MFMA's V operand read one MFMA ahead.
    float la = 0.0f, lb = 0.0f;
    auto soft = [&](int st) __attribute__((always_inline)) {
      float f[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) f[t] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[st >> 1][8 * (st & 1) + t], sl2, -m_run));
      la += (f[0] + f[1]) + (f[2] + f[3]);
      lb += (f[4] + f[5]) + (f[6] + f[7]);
      return cvt8(f);
    };
    bf16x8 pcur = soft(0);
    asm volatile("" ::"v"(la), "v"(lb));  // the first step's sums stay ahead of the interleaving
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int st = 0; st < FK / 16; ++st) {
      bf16x8 pnext = pcur;
      if (st + 1 < FK / 16) pnext = soft(st + 1);
#pragma unroll
      for (int d = 0; d < D / 32; ++d)
        oacc[d] = mfma32(tr8(Vt, 16 * st * RB + lo.trl[d], 16 * st * RB + lo.trh[d]), pcur, oacc[d]);
      if (st + 1 < FK / 16) {
        // groups: DS reads (mask 0x100), MFMA (0x008), VALU (0x002), transcendental (0x400)
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
        for (int d = 0; d < D / 32; ++d) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if (d + 1 < D / 32) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
          __builtin_amdgcn_sched_group_barrier(0x400, 2, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      pcur = pnext;
    }
    l_run += la + lb;
  };
  for (int t0 = 0; t0 < nkt; t0 += FNS) SlotLoop<0, FNS>::run(t0, nkt, step);
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (myq < S) {
    store_qrow<D>(O + (bh * S + myq) * D, oacc, 1.0f / l_tot, h);
    if (h == 0) LSE[bh * S + myq] = (m_run + __log2f(l_tot)) * kLn2;
  }
}

// ------------------------------------------------------------------ backward: dQ
// Each wave owns 32 query rows (their Q and dO rows stay in registers) and streams the K/V
// tiles: S^T = K Q^T and dP^T = V dO^T give, per lane, one query row's
// P = exp2(S scale log2e - lse log2e) and dS = P (dP - Delta); dQ^T += K^T dS^T.
constexpr int QW = LH_QW, BQ = 32 * LH_QW, BK = LH_BK, QNS = LH_QNS;

template <int D, bool IDX>
__global__ void __launch_bounds__(64 * QW) __attribute__((amdgpu_waves_per_eu(2, 2)))
sdpa_bwd_dq_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
                 const bf16_t* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ DELTA,
                 bf16_t* __restrict__ dQ, int S, float sl2, float scale, SdpaIdx ix, HeadMap hm) {
  constexpr int RB = 2 * D;
  constexpr int LPT = 2 * loads_per_wave<D, BK, QW>();
  static_assert(QNS >= 2 && QNS <= 4, "ring of 2 to 4 slots");
  LH_RING(bf16_t, Ks, BK * D);
  LH_RING(bf16_t, Vs, BK * D);
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, r32 = lane & 31;
  const BlockPos bp = block_pos();
  const int64_t bh = bp.head;
  const int nqt = (S + BQ - 1) / BQ;
  const int q0 = (nqt - 1 - bp.rank) * BQ;
  const int qw = q0 + 32 * w;
  const int myq = qw + r32;
  const int64_t kvh = (bh / hm.Hq) * hm.Hs + (bh % hm.Hq) / hm.Gq;  // selection head
  const bf16_t* Qh = Q + bh * S * D;
  const bf16_t* Kh = K + kvh * S * D;
  const bf16_t* Vh = V + kvh * S * D;
  const bf16_t* dOh = dO + bh * S * D;
  const LaneOff<D> lo = lane_offsets<D, LH_SWZ_Q>(lane);
  constexpr int LPW = loads_per_wave<D, BK, QW>();
  RowSrc qsrc{}, ksrc{}, vsrc{};
  const int32_t* idxh = nullptr;
  int32_t kv_ids[LPW];  // ids of the next tile to be loaded
  if constexpr (IDX) {
    const int64_t b = bh / ix.Hq;
    const int hq = (int)(bh - b * ix.Hq), g = hq / ix.G;
    qsrc = row_src(ix.q, ix.qp, b, hq, ix.Hq, ix, D);
    ksrc = row_src(ix.k, ix.kp, b, g, ix.Hkv, ix, D);
    vsrc = row_src(ix.v, ix.vp, b, g, ix.Hkv, ix, D);
    idxh = ix.idx + kvh * S;
    tile_ids<D, BK, QW>(idxh, 0, S, w, lane, kv_ids);
  }
  auto load_kv = [&](int slot_, int r0) __attribute__((always_inline)) {
    bf16_t* kt_ = slot_ == 0 ? Ks[0] : slot_ == 1 ? Ks[1] : slot_ == 2 ? Ks[2] : Ks[3];
    bf16_t* vt_ = slot_ == 0 ? Vs[0] : slot_ == 1 ? Vs[1] : slot_ == 2 ? Vs[2] : Vs[3];
    if constexpr (IDX) {
      load_tile_idx<D, BK, QW, LH_SWZ_Q>(kt_, ksrc, kv_ids, w, lane);
      load_tile_idx<D, BK, QW, LH_SWZ_Q>(vt_, vsrc, kv_ids, w, lane);
      tile_ids<D, BK, QW>(idxh, r0 + BK, S, w, lane, kv_ids);
    } else {
      load_tile<D, BK, QW, LH_SWZ_Q>(kt_, Kh, r0, S, w, lane);
      load_tile<D, BK, QW, LH_SWZ_Q>(vt_, Vh, r0, S, w, lane);
    }
  };

  const int kend = q0 + BQ < S ? q0 + BQ : S;
  const int nkt = (kend + BK - 1) / BK;
  const int qrow = myq < S ? myq : S - 1;
  bf16x8 qreg[D / 16], doreg[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    const bf16_t* qr = IDX ? rs_row(qsrc, idxh[qrow]) : Qh + (int64_t)qrow * D;
    qreg[kk] = gld8(qr + 16 * kk + 8 * h);
    doreg[kk] = gld8(dOh + (int64_t)qrow * D + 16 * kk + 8 * h);
  }
  const float lse2 = myq < S ? LSE[bh * S + myq] * kLog2e : INFINITY;
  const float dlt = myq < S ? DELTA[bh * S + myq] : 0.0f;
  // every element of a lane's dP^T accumulator belongs to the lane's query row: the chain starts
  // from -Delta (a separate source operand of its first MFMA), so it ends as dP - Delta and no
  // subtraction is needed
  f32x16 ndlt;
#pragma unroll
  for (int i = 0; i < 16; ++i) ndlt[i] = -dlt;
#pragma unroll
  for (int t = 0; t < QNS - 1; ++t) load_kv(t, t * BK);
  f32x16 dqacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) dqacc[d] = f32x16{};

  // Key tiles before q0 hold no key after any row of the block: no mask. Only the last
  // BQ / BK tiles (the diagonal band) run the masked body.
  static_assert(QNS == 2, "the masked / unmasked split runs a two-slot ring");
  auto step = [&](auto slotc, auto maskc, int kt) __attribute__((always_inline)) {
    constexpr int SL = decltype(slotc)::value;
    constexpr bool MASK = decltype(maskc)::value != 0;
    constexpr int NX = (SL + QNS - 1) % QNS;
    sync_tiles<(QNS - 2) * LPT>();
    load_kv(NX, (kt + QNS - 1) * BK);
    const int k0 = kt * BK;
    if (qw + 31 < k0) return;
    const bf16_t* Kt = Ks[SL];
    const bf16_t* Vt = Vs[SL];
#pragma unroll
    for (int kb = 0; kb < BK / 32; ++kb) {
      f32x16 sacc = f32x16{};
      f32x16 pacc = mfma32(row8(Vt, kb * 32 * RB + lo.row[0]), doreg[0], ndlt);
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        sacc = mfma32(row8(Kt, kb * 32 * RB + lo.row[kk]), qreg[kk], sacc);
        if (kk > 0) pacc = mfma32(row8(Vt, kb * 32 * RB + lo.row[kk]), doreg[kk], pacc);
      }
      // causal mask: element i holds key k0 + 32 kb + 4h + c_i, c_i = 8 (i / 4) + i % 4, which is
      // in the future of the lane's query exactly when c_i > tm
      const int tm = myq - k0 - kb * 32 - 4 * h;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float f[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int i = 8 * u + t;
          float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[i], sl2, -lse2));
          if (MASK && 8 * (i >> 2) + (i & 3) > tm) pv = 0.0f;
          f[t] = pv * pacc[i];
        }
        const bf16x8 db = cvt8(f);
#pragma unroll
        for (int d = 0; d < D / 32; ++d)
          dqacc[d] = mfma32(tr8(Kt, (kb * 32 + 16 * u) * RB + lo.trl[d], (kb * 32 + 16 * u) * RB + lo.trh[d]), db,
                            dqacc[d]);
      }
    }
  };
  const int nfree = q0 / BK < nkt ? q0 / BK : nkt;  // tiles [0, nfree) need no mask
  auto plain = [&](auto slotc, int kt) __attribute__((always_inline)) { step(slotc, IC<0>{}, kt); };
  auto masked = [&](auto slotc, int kt) __attribute__((always_inline)) { step(slotc, IC<1>{}, kt); };
  ring2_loop(0, nfree, plain);
  ring2_loop(nfree, nkt, masked);
  if (myq < S) store_qrow<D>(dQ + (bh * S + myq) * D, dqacc, scale, h);
}

// ------------------------------------------------------------------ backward: dK, dV
// Each wave owns 32 keys: their V rows stay in registers and the workgroup's K rows stay in
// LDS for the whole kernel. Query tiles, with their lse and Delta, stream through two LDS slots:
// S = Q K^T and dP = dO V^T (per lane: one key, 16 queries), then dV += P^T dO and
// dK += dS^T Q with the transposed dO / Q operands read from the same tiles. Each query tile
// is processed in two 32-row halves to bound the live registers. The lse / Delta of a tile
// pass through registers, so each step waits for all of the wave's loads before the barrier.
constexpr int KWV = LH_KWV, CK = 32 * LH_KWV, CQ = LH_CQ;
static_assert(CQ % 32 == 0 && CQ <= 64, "query tile of 32 or 64 rows");

// GRP: the workgroup's keys belong to a selection shared by hm.Gq query heads; their dK, dV sum
// over those heads (one pass of the query-tile loop per head, the accumulators kept).
template <int D, bool IDX, bool GRP>
__global__ void __launch_bounds__(64 * KWV) __attribute__((amdgpu_waves_per_eu(LH_KWV_EU, LH_KWV_EU)))
sdpa_bwd_dkdv_bf16(const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
                   const bf16_t* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ DELTA,
                   bf16_t* __restrict__ dK, bf16_t* __restrict__ dV, int S, float sl2, float scale, SdpaIdx ix,
                   HeadMap hm) {
  constexpr int RB = 2 * D;
  // LDS is laid out by decreasing alignment: the lse / Delta rows (1 KB) first, then the query
  // tiles, so that both sit inside the first 64 KB, where a base address folds into the 16-bit
  // immediate offset of the LDS reads (the deepest tile read ends below 63 KB); K comes last.
  __shared__ __align__(128) float ls0[CQ], ls1[CQ], ds0[CQ], ds1[CQ];
  __shared__ __align__(64) bf16_t Qs0[CQ * D], Qs1[CQ * D], dOs0[CQ * D], dOs1[CQ * D];
  __shared__ __align__(16) bf16_t Kw[CK * D];
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, r32 = lane & 31;
  const BlockPos bp = block_pos();
  const int64_t bs = bp.head;  // b * Hs + hs: the selection head whose keys this block owns
  const int64_t bsb = bs / hm.Hs;
  const int hs0 = (int)(bs - bsb * hm.Hs);
  int64_t bh = bsb * hm.Hq + (int64_t)hs0 * hm.Gq;  // the query head being streamed
  const int k0 = bp.rank * CK;  // early keys see the most queries: launched first
  const int kw = k0 + 32 * w;
  const int mykey = kw + r32;
  const bf16_t* Qh = Q + bh * S * D;
  const bf16_t* Kh = K + bs * S * D;
  const bf16_t* Vh = V + bs * S * D;
  const bf16_t* dOh = dO + bh * S * D;
  const float* Lh = LSE + bh * S;
  const float* Dh = DELTA + bh * S;
  const LaneOff<D> lo = lane_offsets<D, LH_SWZ_K>(lane);
  RowSrc qsrc{}, ksrc{}, vsrc{};
  const int32_t* idxh = nullptr;
  int32_t q_ids[loads_per_wave<D, CQ, KWV>()];  // ids of the next query tile to be staged
  if constexpr (IDX) {
    const int hq = hs0 * hm.Gq, g = hq / ix.G;
    qsrc = row_src(ix.q, ix.qp, bsb, hq, ix.Hq, ix, D);
    ksrc = row_src(ix.k, ix.kp, bsb, g, ix.Hkv, ix, D);
    vsrc = row_src(ix.v, ix.vp, bsb, g, ix.Hkv, ix, D);
    idxh = ix.idx + bs * S;
  }

  const int qstart = (k0 / CQ) * CQ;
  const int nqt = (S - qstart + CQ - 1) / CQ;
  // lse and Delta of a query tile enter LDS through the first CQ threads. The tile staged
  // before the loop is written at once; a tile staged inside the loop has its two values loaded
  // into nl, nd when its Q / dO copies are issued and written to LDS just before the barrier that
  // publishes the tile, so no wave waits for those loads in the middle of a tile.
  float nl = 0.0f, nd = 0.0f;
  auto put_ld = [&](auto bufc, int qt0, float lv, float dv) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    const bool in = qt0 + tid < S;
    (BUF ? ls1 : ls0)[tid] = in ? lv * kLog2e : INFINITY;  // rows past S: P = 0
    (BUF ? ds1 : ds0)[tid] = in ? -dv : 0.0f;  // negated: it seeds the dP accumulator
  };
  auto stage = [&](auto bufc, auto deferc, int qt0) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    if constexpr (IDX) load_tile_idx<D, CQ, KWV, LH_SWZ_K>(BUF ? Qs1 : Qs0, qsrc, q_ids, w, lane);
    else load_tile<D, CQ, KWV, LH_SWZ_K>(BUF ? Qs1 : Qs0, Qh, qt0, S, w, lane);
    load_tile<D, CQ, KWV, LH_SWZ_K>(BUF ? dOs1 : dOs0, dOh, qt0, S, w, lane);
    if (tid < CQ) {
      const int q = qt0 + tid < S ? qt0 + tid : S - 1;  // clamped; rows past S are masked in put_ld
      if constexpr (decltype(deferc)::value) {
        nl = Lh[q];
        nd = Dh[q];
      } else {
        put_ld(bufc, qt0, Lh[q], Dh[q]);
      }
    }
    // tiles are staged from the last one down: the next one starts CQ rows earlier
    if constexpr (IDX) tile_ids<D, CQ, KWV>(idxh, qt0 - CQ > 0 ? qt0 - CQ : 0, S, w, lane, q_ids);
  };
  // Query tiles are visited from the last one down to the diagonal: every key block of a head
  // then starts on the same tile and streams the same tiles in step with the others, so the
  // blocks running together on an XCD share each Q / dO tile through its L2.
  const int qlast = qstart + (nqt - 1) * CQ;
  if constexpr (IDX) {
    int32_t k_ids[loads_per_wave<D, CK, KWV>()];
    tile_ids<D, CK, KWV>(idxh, k0, S, w, lane, k_ids);
    load_tile_idx<D, CK, KWV, LH_SWZ_K>(Kw, ksrc, k_ids, w, lane);
    tile_ids<D, CQ, KWV>(idxh, qlast, S, w, lane, q_ids);
  } else {
    load_tile<D, CK, KWV, LH_SWZ_K>(Kw, Kh, k0, S, w, lane);
  }
  stage(IC<0>{}, IC<0>{}, qlast);

  const int krow = mykey < S ? mykey : S - 1;
  const bf16_t* vrow = IDX ? rs_row(vsrc, idxh[krow]) : Vh + (int64_t)krow * D;
  bf16x8 vreg[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) vreg[kk] = gld8(vrow + 16 * kk + 8 * h);
  f32x16 dkacc[D / 32], dvacc[D / 32];
#pragma unroll
  for (int d = 0; d < D / 32; ++d) dkacc[d] = dvacc[d] = f32x16{};

  auto tile = [&](auto bufc, auto maskc, int it) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value;
    constexpr bool MASK = decltype(maskc)::value != 0;
    const bf16_t* Qt = BUF ? Qs1 : Qs0;
    const bf16_t* dOt = BUF ? dOs1 : dOs0;
    const float* lt = BUF ? ls1 : ls0;
    const float* dt = BUF ? ds1 : ds0;
    const int qt0 = qlast - it * CQ;
    if (it > 0 && tid < CQ) put_ld(bufc, qt0, nl, nd);  // staged with the previous tile
    sync_tiles<0>();  // this tile (and its lse / Delta) landed; the other slot is free
    if (it + 1 < nqt) stage(IC<BUF ^ 1>{}, IC<1>{}, qt0 - CQ);
    if (qt0 + CQ - 1 < kw || kw >= S) return;  // every query of the tile precedes this wave's keys
#pragma unroll
    for (int qb = 0; qb < CQ / 32; ++qb) {
      // causal mask: element i holds query row qt0 + 32 qb + 4h + c_i, c_i = 8 (i / 4) + i % 4, so
      // P = 0 exactly where c_i < t (t < 0 on every tile after this wave's diagonal one)
      const int tmask = mykey - qt0 - 32 * qb - 4 * h;
      // the dP accumulator starts at -Delta (stored negated), so it ends as dP - Delta
      f32x16 sacc = f32x16{}, pacc;
#pragma unroll
      for (int g = 0; g < 4; ++g) {  // rows qb * 32 + 8 g + 4 h + 0..3 of the C layout
        const float4 d4 = *reinterpret_cast<const float4*>(dt + qb * 32 + 8 * g + 4 * h);
        pacc[4 * g + 0] = d4.x, pacc[4 * g + 1] = d4.y, pacc[4 * g + 2] = d4.z, pacc[4 * g + 3] = d4.w;
      }
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        sacc = mfma32(row8(Qt, qb * 32 * RB + lo.row[kk]), row8(Kw, w * 32 * RB + lo.row[kk]), sacc);
        pacc = mfma32(row8(dOt, qb * 32 * RB + lo.row[kk]), vreg[kk], pacc);
        if (kk & 1) __builtin_amdgcn_sched_barrier(0);  // bound the operand loads in flight
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float pf[8], df[8];
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const int qg = qb * 32 + 16 * u + 8 * g + 4 * h;  // tile rows qg .. qg + 3
          const float4 l4 = *reinterpret_cast<const float4*>(lt + qg);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int i = 8 * u + 4 * g + j;
            float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[i], sl2, -lv[j]));
            if (MASK && 8 * (i >> 2) + (i & 3) < tmask) pv = 0.0f;
            pf[4 * g + j] = pv;
            df[4 * g + j] = pv * pacc[i];
          }
        }
        const bf16x8 pb = cvt8(pf), db = cvt8(df);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int d = 0; d < D / 32; ++d) {
          dvacc[d] = mfma32(pb, tr8(dOt, (qb * 32 + 16 * u) * RB + lo.trl[d], (qb * 32 + 16 * u) * RB + lo.trh[d]),
                            dvacc[d]);
          dkacc[d] = mfma32(db, tr8(Qt, (qb * 32 + 16 * u) * RB + lo.trl[d], (qb * 32 + 16 * u) * RB + lo.trh[d]),
                            dkacc[d]);
          if (d & 1) __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };
  // Query tiles at or after k0 + CK hold no query before any key of the block: no mask. Only the
  // last CK / CQ tiles visited (the diagonal band) run the masked body.
  const int nfree = nqt > CK / CQ ? nqt - CK / CQ : 0;
  auto plain = [&](auto bufc, int it) __attribute__((always_inline)) { tile(bufc, IC<0>{}, it); };
  auto masked = [&](auto bufc, int it) __attribute__((always_inline)) { tile(bufc, IC<1>{}, it); };
  for (int mq = 0;;) {
    ring2_loop(0, nfree, plain);
    ring2_loop(nfree, nqt, masked);
    if (!GRP || ++mq >= hm.Gq) break;
    // next query head of the selection: restart the tile stream once every wave is done with
    // the buffers of the last tile
    __syncthreads();
    ++bh;
    Qh += (int64_t)S * D;
    dOh += (int64_t)S * D;
    Lh += S;
    Dh += S;
    if constexpr (IDX) {
      qsrc = row_src(ix.q, ix.qp, bsb, hs0 * hm.Gq + mq, ix.Hq, ix, D);
      tile_ids<D, CQ, KWV>(idxh, qlast, S, w, lane, q_ids);
    }
    stage(IC<0>{}, IC<0>{}, qlast);
  }
  // C layout: row = key kw + 8(i/4) + 4h + i%4, column 32 d + lane % 32
#pragma unroll
  for (int d = 0; d < D / 32; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = kw + 8 * (i >> 2) + 4 * h + (i & 3);
      if (key < S) {
        dK[(bs * S + key) * D + 32 * d + r32] = f2bf(dkacc[d][i] * scale);
        dV[(bs * S + key) * D + 32 * d + r32] = f2bf(dvacc[d][i]);
      }
    }
}

template <bool IDX>
static void launch_fwd(const LhShape& s, const void* qs, const void* ks, const void* vs, void* os, float* lse,
                       const SdpaIdx& ix, hipStream_t st) {
  const int S = (int)s.S;
  const HeadMap hm{s.Hq, s.Hs, s.Gq};
  dim3 grid((unsigned)((S + FQ - 1) / FQ), (unsigned)(s.B * s.Hq));
  const float sl2 = s.scale * kLog2e;
  auto q = (const bf16_t*)qs;
  auto k = (const bf16_t*)ks;
  auto v = (const bf16_t*)vs;
  if (s.D == 128)
    hipLaunchKernelGGL((sdpa_fwd_bf16<128, IDX>), grid, dim3(64 * FW), 0, st, q, k, v, (bf16_t*)os, lse, S, sl2, ix,
                       hm);
  else
    hipLaunchKernelGGL((sdpa_fwd_bf16<64, IDX>), grid, dim3(64 * FW), 0, st, q, k, v, (bf16_t*)os, lse, S, sl2, ix, hm);
}

template <int D, bool IDX, bool GRP>
static void launch_bwd_D(const LhShape& s, const bf16_t* q, const bf16_t* k, const bf16_t* v, const bf16_t* g,
                         const float* lse, const float* delta, void* dqs, void* dks, void* dvs, const SdpaIdx& ix,
                         hipStream_t st) {
  const int S = (int)s.S;
  const float sl2 = s.scale * kLog2e;
  const HeadMap hm{s.Hq, s.Hs, s.Gq};
  dim3 gk((unsigned)((S + CK - 1) / CK), (unsigned)(s.B * s.Hs));  // per (key block, selection head)
  dim3 gq((unsigned)((S + BQ - 1) / BQ), (unsigned)(s.B * s.Hq));
  hipLaunchKernelGGL((sdpa_bwd_dkdv_bf16<D, IDX, GRP>), gk, dim3(64 * KWV), 0, st, q, k, v, g, lse, delta,
                     (bf16_t*)dks, (bf16_t*)dvs, S, sl2, s.scale, ix, hm);
  hipLaunchKernelGGL((sdpa_bwd_dq_bf16<D, IDX>), gq, dim3(64 * QW), 0, st, q, k, v, g, lse, delta, (bf16_t*)dqs, S,
                     sl2, s.scale, ix, hm);
}

template <bool IDX>
static void launch_bwd(const LhShape& s, const void* qs, const void* ks, const void* vs, const void* dos,
                       const float* lse, const float* delta, void* dqs, void* dks, void* dvs, const SdpaIdx& ix,
                       hipStream_t st) {
  auto q = (const bf16_t*)qs;
  auto k = (const bf16_t*)ks;
  auto v = (const bf16_t*)vs;
  auto g = (const bf16_t*)dos;
  const bool grp = s.Gq > 1;
  if (s.D == 128) {
    if (grp) launch_bwd_D<128, IDX, true>(s, q, k, v, g, lse, delta, dqs, dks, dvs, ix, st);
    else launch_bwd_D<128, IDX, false>(s, q, k, v, g, lse, delta, dqs, dks, dvs, ix, st);
  } else {
    if (grp) launch_bwd_D<64, IDX, true>(s, q, k, v, g, lse, delta, dqs, dks, dvs, ix, st);
    else launch_bwd_D<64, IDX, false>(s, q, k, v, g, lse, delta, dqs, dks, dvs, ix, st);
  }
}

static SdpaIdx make_idx(const LhShape& s, const void* q, const void* k, const void* v, const void* qp,
                        const void* kp, const void* vp, const int32_t* idx) {
  SdpaIdx ix{};
  ix.q = (const bf16_t*)q, ix.k = (const bf16_t*)k, ix.v = (const bf16_t*)v;
  // with L = 1 there is no pyramid: every id is below N, the pointers are never followed
  ix.qp = qp ? (const bf16_t*)qp : ix.q;
  ix.kp = kp ? (const bf16_t*)kp : ix.k;
  ix.vp = vp ? (const bf16_t*)vp : ix.v;
  ix.idx = idx;
  ix.N = s.N, ix.R = s.R > 0 ? s.R : 0;
  ix.Hq = s.Hq, ix.Hkv = s.Hkv, ix.G = s.G;
  return ix;
}

}  // namespace lh

using namespace lh;

hipError_t lh_launch_sdpa_fwd_bf16(const LhShape& s, const void* qs, const void* ks, const void* vs, void* os,
                                   float* lse, hipStream_t st) {
  launch_fwd<false>(s, qs, ks, vs, os, lse, SdpaIdx{}, st);
  return hipGetLastError();
}

hipError_t lh_launch_sdpa_bwd_bf16(const LhShape& s, const void* qs, const void* ks, const void* vs,
                                   const void* dos, const float* lse, const float* delta, void* dqs,
                                   void* dks, void* dvs, hipStream_t st) {
  launch_bwd<false>(s, qs, ks, vs, dos, lse, delta, dqs, dks, dvs, SdpaIdx{}, st);
  return hipGetLastError();
}

hipError_t lh_launch_sdpa_fwd_idx(const LhShape& s, const void* q, const void* k, const void* v, const void* qp,
                                  const void* kp, const void* vp, const int32_t* idx, void* os, float* lse,
                                  hipStream_t st) {
  launch_fwd<true>(s, nullptr, nullptr, nullptr, os, lse, make_idx(s, q, k, v, qp, kp, vp, idx), st);
  return hipGetLastError();
}

hipError_t lh_launch_sdpa_bwd_idx(const LhShape& s, const void* q, const void* k, const void* v, const void* qp,
                                  const void* kp, const void* vp, const int32_t* idx, const void* dos,
                                  const float* lse, const float* delta, void* dqs, void* dks, void* dvs,
                                  hipStream_t st) {
  launch_bwd<true>(s, nullptr, nullptr, nullptr, dos, lse, delta, dqs, dks, dvs,
                   make_idx(s, q, k, v, qp, kp, vp, idx), st);
  return hipGetLastError();
}
