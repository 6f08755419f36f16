/*
 * lighthouse.h -- C ABI of the Lighthouse attention hot path on AMD MI355X (gfx950).
 *
 * Lighthouse attention (Peng, Ghosh, Quesnelle, "Long Context Pre-Training with
 * Lighthouse Attention", arXiv 2605.06554) wraps ordinary causal scaled-dot-product
 * attention in four stages (Sec. 3.2):
 *   (i)   mean-pool Q, K, V into an L-level pyramid with pooling factor p  (Sec. 3.3, Eq. pool);
 *   (ii)  score every pyramid entry with parameter-free l2 norms, max-pooled from level 0
 *         (Sec. 3.4, Eqs. score-base and score-pool), and select entries by top-k (Eq. topk);
 *   (iii) gather the selected (Q, K, V) triples into a causally ordered sub-sequence of
 *         length S (Sec. 3.5, Eq. S-size) and run dense causal SDPA on it (Eq. attn-sub);
 *   (iv)  scatter each output row back to a shifted range of base positions and sum across
 *         levels (Sec. 3.6, Eqs. fanout and scatter).
 * Gradients flow back through (iv), (iii) and the pooling; nothing flows through the scores
 * or the selection (Sec. 3.2, App. C.4).
 *
 * Readings taken where the paper is silent or ambiguous (all shared by every entry point):
 *   - Selection is a per-level descent (Fig. 2 panel 3, Sec. 3.4, Eq. S-size): the coarsest
 *     level is kept whole; at each level l = L-1..1 the k best candidates (by
 *     c = max(s_QK, s_KQ), ties broken by the lower level-local index) are "parents", whose
 *     p children become the candidates of level l-1. Every candidate of every level is
 *     emitted, parents included. Hence S = N/p^(L-1) + sum over levels of p*min(k, #cand),
 *     which equals Eq. S-size whenever N/p^(L-1) >= k.
 *   - k counts parents per level per (batch, query head). Selection is per query head:
 *     s_QK comes from the query head hq, s_KQ from its KV head g = hq / (Hq/Hkv).
 *   - Scores are fp32: s = fp32_RNE(sqrt_RN_f64(sum_c x_c^2 accumulated in fp64, c ascending)).
 *   - Causal order of the gathered entries: by window end e(l,i) = (i+1) p^l - 1 ascending,
 *     coarser level first on equal e. The SDPA mask is lower-triangular on that order.
 *   - Softmax scale is 1/sqrt(D) for every entry (Eq. sdpa) unless lh_problem.scale != 0.
 *   - Scatter ranges past N-1 are clipped; base positions with no contributor get O = 0.
 *   - Pyramid entries are stored in the layer dtype, rounded once (to nearest, ties to even)
 *     from the mean of the p^l base rows.
 *
 * Conventions for every entry point below:
 *   - Pointers named q/k/v/o/... are DEVICE pointers unless noted; the caller owns all memory.
 *     The library never allocates, frees or keeps device memory, and never calls hipSetDevice:
 *     work runs on the current device.
 *   - Tensors are dense row-major in the stated layout, with 16-byte aligned base pointers.
 *     Inputs and outputs must not alias. Outputs are overwritten, never accumulated.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream). Work is enqueued
 *     asynchronously; no entry point synchronizes the host.
 *   - Every argument check runs on the host before anything is enqueued; a non-LH_OK status
 *     means nothing was enqueued, except LH_E_HIP (a launch error reported by the runtime).
 *     Nothing aborts or throws across this ABI. lh_last_error() holds a thread-local detail.
 *   - Identical problems and inputs give bitwise identical outputs (no floating-point atomics).
 *
 * Tensor layouts (B batch, N base length, Hq query heads, Hkv KV heads, D head dim,
 * Ptot = sum_{l<L} N/p^l pyramid entries, R = Ptot - N pooled rows, S gathered length):
 *   q, o, dq, dout            [B, N, Hq, D]      (dtype)
 *   k, v, dk, dv              [B, N, Hkv, D]     (dtype)
 *   qpyr                      [B, R, Hq, D]      (dtype)  rows of levels 1..L-1, level-major:
 *   kpyr, vpyr                [B, R, Hkv, D]     (dtype)  entry (l, i) is row off_l - N + i
 *   s_qk                      [B, Hq, Ptot]      float    flattened id of (l, i) is off_l + i
 *   s_kq                      [B, Hkv, Ptot]     float
 *   idx                       [B, Hq, S]         int32    flattened pyramid ids, causal order
 *   slot                      [B, Hq, Ptot]      int32    position of an entry in idx, or -1
 *   qs, ks, vs, os, dos, dqs, dks, dvs   [B, Hq, S, D]   (dtype)  gathered sub-sequence
 *   lse                       [B, Hq, S]         float    natural-log row log-sum-exp of SDPA
 */
#ifndef LIGHTHOUSE_H_
#define LIGHTHOUSE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LH_OK = 0,
  LH_E_NULL = -1,       /* a required pointer is NULL                                  */
  LH_E_SHAPE = -2,      /* p^(L-1) does not divide N, or a size is out of range       */
  LH_E_PARAM = -3,      /* invalid p, L, k, Hq/Hkv, D, flags, or level out of range   */
  LH_E_DTYPE = -4,      /* dtype not supported by this entry point                    */
  LH_E_ALIGN = -5,      /* a pointer is not 16-byte aligned                           */
  LH_E_WORKSPACE = -6,  /* workspace missing or smaller than lh_workspace_bytes()     */
  LH_E_HIP = -7,        /* the HIP runtime reported an error while enqueueing         */
  LH_E_NONFINITE = -8   /* a floating-point argument (the softmax scale) is NaN or inf */
} lh_status;

typedef enum { LH_F32 = 0, LH_BF16 = 1 } lh_dtype;

/* flags */
enum {
  /* Test-only selection variant: parents of levels >= 1 are NOT emitted (only their
     descendants are). With a budget that covers every entry it leaves exactly level 0,
     i.e. plain causal SDPA, which pins the gather/SDPA/scatter chain. */
  LH_FLAG_REPLACE_PARENTS = 1u << 0,
  /* Stratified selection (App. D.2, the chunked top-k the paper implements): a level that
     ranks its candidates (k < #cand) cuts them, in index order, into chunks of 2048; chunk
     [s, e) keeps its best floor(k e / #cand) - floor(k s / #cand) candidates by the same key
     and tie-break. Every chunk of the sequence contributes its share, the level still keeps
     k parents, and S and every shape are those of the exact mode. */
  LH_FLAG_STRATIFIED = 1u << 1,
  /* One selection per KV group (GQA-shared), a reading beyond the paper's MHA model: the
     group's query score of an entry is the max of its query heads' scores (Eq. score-pool), and
     it is combined with the KV head's score by the max of Eq. topk. idx [B,Hkv,S] and slot
     [B,Hkv,Ptot] are then per KV head, as are ks, vs (and dks, dvs); every query head of the
     group gathers its q rows with the group's idx and attends over the group's ks, vs, and the
     group's dks, dvs sum over its query heads. Without the flag (default) every query head
     selects on its own (the tensors above are per query head). */
  LH_FLAG_GQA_SHARED = 1u << 2
};

/* workspace owners for lh_workspace_bytes */
enum {
  LH_OP_SELECT = 0,         /* lh_select_topk          */
  LH_OP_SDPA_BWD = 1,       /* lh_sdpa_bwd             */
  LH_OP_ATTENTION_FWD = 2,  /* lh_attention_fwd        */
  LH_OP_ATTENTION_BWD = 3,  /* lh_attention_bwd and lh_attention_bwd_indexed */
  LH_OP_ATTENTION_FWD_INDEXED = 4  /* lh_attention_fwd_indexed */
};

typedef struct {
  int64_t B;        /* batch size, >= 1                                                  */
  int64_t N;        /* base sequence length, >= 1, divisible by p^(L-1)                  */
  int32_t Hq;       /* query heads, >= 1                                                 */
  int32_t Hkv;      /* key/value heads, >= 1, Hq % Hkv == 0 (query head hq uses hq/(Hq/Hkv)) */
  int32_t D;        /* head dimension: 64 or 128                                         */
  int32_t p;        /* pooling factor, >= 2 when L > 1                                   */
  int32_t L;        /* pyramid levels, >= 1 (L = 1 is plain causal SDPA)                 */
  int32_t k;        /* parents per level per (batch, query head), >= 0                   */
  int32_t dtype;    /* lh_dtype of every Q/K/V/O-like tensor and gradient                */
  float scale;      /* softmax scale, finite and >= 0; 0 selects 1/sqrt(D)               */
  uint32_t flags;   /* LH_FLAG_* bits                                                    */
} lh_problem;

/* ---------------- host-only helpers (no device access) ---------------- */

/* Validates a problem (the rules above and Sec. 3.3's divisibility requirement).
   Also rejects sizes whose flattened indices would not fit int32. */
lh_status lh_check(const lh_problem* pr);
/* N / p^level, or -1 if the problem is invalid or level is outside [0, L). */
int64_t lh_level_rows(const lh_problem* pr, int32_t level);
/* Flattened pyramid id of entry (level, 0): sum_{l < level} N / p^l; -1 on error. */
int64_t lh_level_offset(const lh_problem* pr, int32_t level);
/* Ptot = sum_{l < L} N / p^l (Sec. 3.3 bounds it by N p/(p-1)); -1 on error. */
int64_t lh_pyramid_rows(const lh_problem* pr);
/* Gathered length S (data independent): N/p^(L-1) + sum_{l=L-1..1} p*min(k, #cand_l),
   with #cand_{L-1} = N/p^(L-1) and #cand_{l-1} = p*min(k, #cand_l); Eq. S-size when
   N/p^(L-1) >= k. Without parents emitted (LH_FLAG_REPLACE_PARENTS) the parents are
   subtracted. -1 on error. */
int64_t lh_subseq_len(const lh_problem* pr);
/* Bytes of device workspace entry point `op` (LH_OP_*) needs for this problem; 0 is legal. */
lh_status lh_workspace_bytes(const lh_problem* pr, int32_t op, size_t* bytes);
const char* lh_status_str(lh_status s);
/* Thread-local detail of the last error raised on this thread ("" if none). */
const char* lh_last_error(void);

/* ---------------- stage entry points (asynchronous on `stream`) ---------------- */
/* Hs below is the number of selection heads: Hq, or Hkv with LH_FLAG_GQA_SHARED; query head hq
   uses selection head hq / (Hq / Hs). */

/* Sec. 3.3, Eq. pool: level-l entry i is the mean of base rows i p^l .. (i+1) p^l - 1, for
   l = 1..L-1 (level 0 is the input itself and is not copied). Writes qpyr, kpyr, vpyr. */
lh_status lh_pyramid_pool(const lh_problem* pr, const void* q, const void* k, const void* v,
                          void* qpyr, void* kpyr, void* vpyr, void* stream);

/* Sec. 3.4, Eqs. score-base and score-pool: level-0 scores are per-head l2 norms of Q rows
   (s_qk, per query head) and K rows (s_kq, per KV head); a level-l score is the max of the
   level-0 scores in its window. Writes s_qk [B,Hq,Ptot] and s_kq [B,Hkv,Ptot]. */
lh_status lh_score(const lh_problem* pr, const void* q, const void* k,
                   float* s_qk, float* s_kq, void* stream);

/* lh_pyramid_pool and lh_score in one streaming pass over Q, K, V (each input row is read
   once). Writes qpyr, kpyr, vpyr (when L > 1), s_qk and s_kq exactly as the two calls do. */
lh_status lh_pool_score(const lh_problem* pr, const void* q, const void* k, const void* v,
                        void* qpyr, void* kpyr, void* vpyr, float* s_qk, float* s_kq, void* stream);

/* Sec. 3.4 (Eq. topk, Fig. 2 panel 3) and Sec. 3.5 (causal order): per (b, selection head),
   the per-level descent described at the top of this file, then the causal ordering.
   Writes idx [B,Hs,S] and slot [B,Hs,Ptot] (-1 for entries not gathered).
   ws: device workspace of at least lh_workspace_bytes(LH_OP_SELECT) bytes. */
lh_status lh_select_topk(const lh_problem* pr, const float* s_qk, const float* s_kq,
                         int32_t* idx, int32_t* slot, void* ws, size_t ws_bytes, void* stream);

/* Sec. 3.5 (gather equation): qs[b,hq,m] = Q^(l_m)[b, i_m, hq], ks/vs likewise from KV head
   hq/(Hq/Hkv), where idx[b,hs,m] = off_{l_m} + i_m for the selection head hs of hq. Ids below N
   read q/k/v, the rest read the pyramid buffers. Bitwise copies. qs is [B,Hq,S,D]; ks and vs
   are [B,Hs,S,D] (per selection head). */
lh_status lh_gather(const lh_problem* pr, const void* q, const void* k, const void* v,
                    const void* qpyr, const void* kpyr, const void* vpyr, const int32_t* idx,
                    void* qs, void* ks, void* vs, void* stream);

/* Sec. 3.5, Eq. attn-sub with Eq. sdpa: os = softmax(scale qs ks^T + causal mask) vs per
   (b, hq) over the S gathered rows (ks, vs of the selection head of hq); lse = natural-log row
   log-sum-exp of the scaled, masked logits (fp32). Accumulation in fp32 (MFMA for bf16).
   os [B,Hq,S,D], lse [B,Hq,S]. */
lh_status lh_sdpa_fwd(const lh_problem* pr, const void* qs, const void* ks, const void* vs,
                      void* os, float* lse, void* stream);

/* Gradient of lh_sdpa_fwd (App. C.4: gradients flow through the gathered values):
   given dos = dL/dos, writes dqs [B,Hq,S,D] and dks, dvs [B,Hs,S,D] (the gradients of a
   selection head's rows summed over its query heads). Uses lse saved by the forward.
   ws: at least lh_workspace_bytes(LH_OP_SDPA_BWD) bytes. Deterministic. */
lh_status lh_sdpa_bwd(const lh_problem* pr, const void* qs, const void* ks, const void* vs,
                      const void* os, const float* lse, const void* dos,
                      void* dqs, void* dks, void* dvs, void* ws, size_t ws_bytes, void* stream);

/* lh_sdpa_bwd for callers that cannot allocate device memory (code under HIP graph capture,
   tight serving loops, harnesses that forbid allocation): the same computation and bits, with
   Delta kept in a static device array of the library instead of a caller workspace. No
   allocation or free happens in the call. Limit: B * Hq * S <= 4,194,304 (16 MiB of fp32);
   larger problems get LH_E_WORKSPACE before anything is enqueued. Each GPU the library runs on
   holds its own 16 MiB copy until the process ends. Every call on a GPU shares that GPU's
   array, so calls that overlap on one GPU (other streams, other threads) race; serialise them.
   The array needs no clearing: each call overwrites what it reads. */
lh_status lh_sdpa_bwd_noalloc(const lh_problem* pr, const void* qs, const void* ks, const void* vs,
                              const void* os, const float* lse, const void* dos,
                              void* dqs, void* dks, void* dvs, void* stream);

/* Sec. 3.6, Eqs. fanout and scatter: entry (l, i) at position m writes os[m] to base
   positions R(l,i) = [(i+1) p^l - 1, (i+2) p^l - 2] (clipped at N-1); contributions of
   different levels are summed in fp32 (level L-1 first) and rounded once. Base positions
   with no contributor get 0. Query head hq reads the slot row of its selection head.
   Writes o [B,N,Hq,D]. */
lh_status lh_scatter(const lh_problem* pr, const void* os, const int32_t* slot,
                     void* o, void* stream);

/* Adjoint of lh_scatter: dos[m] = sum of dout[j] over j in R(l_m, i_m), j < N
   (fp32 accumulation, one rounding). Writes dos [B,Hq,S,D]. */
lh_status lh_scatter_bwd(const lh_problem* pr, const void* dout, const int32_t* slot,
                         void* dos, void* stream);

/* Adjoint of lh_gather followed by the adjoint of lh_pyramid_pool:
   dq[b,j,hq] = sum_l dqs[slot(l, floor(j/p^l))] / p^l over gathered entries;
   dk[b,j,g], dv[b,j,g] are the same sums over the selection heads of group g (its query
   heads; the group itself with LH_FLAG_GQA_SHARED). fp32 accumulation, one rounding.
   Writes dq, dk, dv. */
lh_status lh_gather_bwd(const lh_problem* pr, const void* dqs, const void* dks, const void* dvs,
                        const int32_t* slot, void* dq, void* dk, void* dv, void* stream);

/* ---------------- fused layer (Algorithm 1 from the pyramid on) ---------------- */

/* One Lighthouse layer forward: pool, score, select, gather, SDPA, scatter.
   Outputs o; also writes the state the backward needs (idx, slot, qs, ks, vs, os, lse).
   ws: at least lh_workspace_bytes(LH_OP_ATTENTION_FWD) bytes (pyramid and scores live there). */
lh_status lh_attention_fwd(const lh_problem* pr, const void* q, const void* k, const void* v,
                           void* o, int32_t* idx, int32_t* slot, void* qs, void* ks, void* vs,
                           void* os, float* lse, void* ws, size_t ws_bytes, void* stream);

/* One Lighthouse layer backward from dout = dL/do to dq, dk, dv, using the forward state.
   ws: at least lh_workspace_bytes(LH_OP_ATTENTION_BWD) bytes. */
lh_status lh_attention_bwd(const lh_problem* pr, const int32_t* idx, const int32_t* slot,
                           const void* qs, const void* ks, const void* vs, const void* os,
                           const float* lse, const void* dout, void* dq, void* dk, void* dv,
                           void* ws, size_t ws_bytes, void* stream);

/* ---------------- gather fused into the SDPA loads ---------------- */
/* The same computation as the calls above with the gathered rows never materialised
   (Sec. 3.5, gather equation): the SDPA kernels read row m of Q~, K~, V~ of head (b, hq)
   straight from pyramid id idx[b,hq,m] of q / qpyr (query head hq) and k, v / kpyr, vpyr
   (KV head hq / (Hq / Hkv)). Given the same inputs, outputs are bitwise identical to those of
   lh_gather followed by lh_sdpa_fwd / lh_sdpa_bwd. bf16 only (LH_E_DTYPE otherwise). qpyr,
   kpyr, vpyr are the pyramid buffers of lh_pyramid_pool ([B,R,H,D], R = Ptot - N); they may be
   NULL when L = 1. idx must hold pyramid ids in [0, Ptot) as written by lh_select_topk; an id
   outside that range is clamped into it (no out-of-range read; the row it reads is
   unspecified). */
lh_status lh_sdpa_fwd_indexed(const lh_problem* pr, const void* q, const void* k, const void* v,
                              const void* qpyr, const void* kpyr, const void* vpyr,
                              const int32_t* idx, void* os, float* lse, void* stream);

/* Gradient of lh_sdpa_fwd_indexed: writes dqs, dks, dvs [B,Hq,S,D] (the gathered-row
   gradients, as lh_sdpa_bwd). ws: at least lh_workspace_bytes(LH_OP_SDPA_BWD) bytes. */
lh_status lh_sdpa_bwd_indexed(const lh_problem* pr, const void* q, const void* k, const void* v,
                              const void* qpyr, const void* kpyr, const void* vpyr,
                              const int32_t* idx, const void* os, const float* lse,
                              const void* dos, void* dqs, void* dks, void* dvs, void* ws,
                              size_t ws_bytes, void* stream);

/* lh_attention_fwd without qs, ks, vs: the caller keeps the pyramid instead (qpyr [B,R,Hq,D],
   kpyr and vpyr [B,R,Hkv,D]; unused and may be NULL when L = 1), which the backward reads.
   ws: at least lh_workspace_bytes(LH_OP_ATTENTION_FWD_INDEXED) bytes (scores and selection
   lists). bf16 only. Outputs are bitwise identical to those of lh_attention_fwd. */
lh_status lh_attention_fwd_indexed(const lh_problem* pr, const void* q, const void* k,
                                   const void* v, void* o, int32_t* idx, int32_t* slot,
                                   void* qpyr, void* kpyr, void* vpyr, void* os, float* lse,
                                   void* ws, size_t ws_bytes, void* stream);

/* lh_attention_bwd from the state of lh_attention_fwd_indexed (q, k, v and the pyramid in
   place of qs, ks, vs). ws: at least lh_workspace_bytes(LH_OP_ATTENTION_BWD) bytes. bf16 only.
   Outputs are bitwise identical to those of lh_attention_bwd. */
lh_status lh_attention_bwd_indexed(const lh_problem* pr, const void* q, const void* k,
                                   const void* v, const void* qpyr, const void* kpyr,
                                   const void* vpyr, const int32_t* idx, const int32_t* slot,
                                   const void* os, const float* lse, const void* dout, void* dq,
                                   void* dk, void* dv, void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LIGHTHOUSE_H_ */
