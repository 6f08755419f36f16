/*
 * lh_oracle.c -- plain, slow CPU reference of the Lighthouse attention hot path.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the oracle the GPU path is checked against. Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load it; the product
 * path never does. It shares no code, header or constant with the HIP library.
 *
 * Paper: Peng, Ghosh, Quesnelle, "Long Context Pre-Training with Lighthouse Attention",
 * arXiv 2605.06554. Every function cites the passage it follows. Arithmetic is fp64 except
 * (a) scores, which are fp32 by the reading stated at lho_scores, and (b) pooled pyramid
 * entries, which are rounded once to the layer dtype (the paper's pooling is a view+mean on
 * tensors of the model dtype, App. D.1), by the reading stated at lho_pool.
 *
 * The functions work on ONE (batch, query head) problem ("head problem"): X[n, c] arrays with
 * a row stride, so a caller can pass a strided head slice of a [B, N, H, D] tensor.
 * Flattened pyramid id of entry (l, i) is off_l + i with off_0 = 0 and
 * off_l = off_{l-1} + N / p^(l-1) (levels stored level-major).
 *
 * Parity pins (tests/): brute force on tiny inputs, the Fig. 2 toy values, closed forms of
 * the pooling, L = 1 and replace-mode full budget reducing to plain causal SDPA, the
 * all-pyramid brute force, causality, finite differences and adjoint identities.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define LHO_F32 0
#define LHO_BF16 1
#define LHO_F64 2 /* unrounded storage: used by finite-difference and adjoint pins */
#define LHO_REPLACE_PARENTS 1u
#define LHO_STRATIFIED 2u
/* Chunk of the stratified selection: the paper's chunked top-k cuts the score stream into
   chunks of 2048 scores (App. D.2). */
#define LHO_STRAT_CHUNK 2048

typedef struct {
  int64_t N;      /* base sequence length                 */
  int32_t D;      /* head dimension                       */
  int32_t p;      /* pooling factor                       */
  int32_t L;      /* pyramid levels                       */
  int32_t k;      /* parents kept per level               */
  int32_t dtype;  /* storage dtype of pooled entries      */
  uint32_t flags; /* LHO_REPLACE_PARENTS                  */
} lho_head;

/* ---------------------------------------------------------------- levels (Sec. 3.3) */

static int64_t ipow(int64_t b, int e) {
  int64_t r = 1;
  for (int i = 0; i < e; ++i) r *= b;
  return r;
}

/* Number of entries at level l: N / p^l (Sec. 3.3, window definition). */
int64_t lho_level_rows(const lho_head* h, int l) { return h->N / ipow(h->p, l); }

/* Flattened id of (l, 0). */
int64_t lho_level_offset(const lho_head* h, int l) {
  int64_t off = 0;
  for (int j = 0; j < l; ++j) off += lho_level_rows(h, j);
  return off;
}

int64_t lho_pyramid_rows(const lho_head* h) { return lho_level_offset(h, h->L); }

/* 0 if valid: p^(L-1) divides N (Sec. 3.3), L >= 1, p >= 2 when L > 1, k >= 0. */
int lho_check(const lho_head* h) {
  if (h->L < 1 || h->k < 0 || h->D < 1 || h->N < 1) return -3;
  if (h->L > 1 && h->p < 2) return -3;
  if (h->L > 1 && h->N % ipow(h->p, h->L - 1) != 0) return -2;
  return 0;
}

/* ---------------------------------------------------------------- storage rounding */

/* Round an fp64 value to the nearest bf16 value, ties to even, written out with frexp and
   nearbyint: x = m 2^e with 0.5 <= |m| < 1; a bf16 value has 8 significant bits, so the
   nearest one is nearbyint(m 2^8) 2^(e-8). Values below the smallest normal use the fixed
   subnormal spacing 2^-133. Overflow is not handled (inputs are finite and moderate). */
static double round_bf16(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  double m = frexp(x, &e);
  if (e - 1 < -126) return ldexp(nearbyint(ldexp(x, 133)), -133);
  return ldexp(nearbyint(ldexp(m, 8)), e - 8);
}

static double round_dtype(double x, int dtype) {
  if (dtype == LHO_BF16) return round_bf16(x);
  if (dtype == LHO_F64) return x;
  return (double)(float)x; /* C conversion to float rounds to nearest, ties to even */
}

double lho_round_bf16(double x) { return round_bf16(x); }

/* ---------------------------------------------------------------- pooling (Sec. 3.3) */

/* Eq. pool: Q^(l)_i = mean of Q_j over the window [i p^l, (i+1) p^l - 1], for every level;
   level 0 is the input itself. The sum runs over the base rows in index order, in fp64, and
   the mean is rounded once to the storage dtype (reading: pooled entries are tensors of the
   layer dtype). Output pyr[Ptot, D]; level 0 rows are copied unrounded. */
void lho_pool(const lho_head* h, const double* x, int64_t ldx, double* pyr) {
  const int D = h->D;
  for (int l = 0; l < h->L; ++l) {
    const int64_t w = ipow(h->p, l), n = lho_level_rows(h, l), off = lho_level_offset(h, l);
    for (int64_t i = 0; i < n; ++i) {
      for (int c = 0; c < D; ++c) {
        if (l == 0) {
          pyr[(off + i) * D + c] = x[i * ldx + c];
          continue;
        }
        double s = 0.0;
        for (int64_t t = 0; t < w; ++t) s += x[(i * w + t) * ldx + c];
        pyr[(off + i) * D + c] = round_dtype(s / (double)w, h->dtype);
      }
    }
  }
}

/* ---------------------------------------------------------------- scores (Sec. 3.4) */

/* Eq. score-base: level-0 score of row j is its l2 norm; Eq. score-pool: a level-l score is
   the max of the level-0 scores in its window (Alg. 1, scoring step). Reading for precision:
   the squares are summed in fp64 for c ascending, the square root is the correctly rounded
   fp64 sqrt, and the result is rounded to fp32; max-pooling is exact. Output s[Ptot]. */
void lho_scores(const lho_head* h, const double* x, int64_t ldx, float* s) {
  const int D = h->D;
  for (int64_t j = 0; j < h->N; ++j) {
    double acc = 0.0;
    for (int c = 0; c < D; ++c) acc += x[j * ldx + c] * x[j * ldx + c];
    s[j] = (float)sqrt(acc);
  }
  for (int l = 1; l < h->L; ++l) {
    const int64_t w = ipow(h->p, l), n = lho_level_rows(h, l), off = lho_level_offset(h, l);
    for (int64_t i = 0; i < n; ++i) {
      float m = s[i * w];
      for (int64_t t = 1; t < w; ++t)
        if (s[i * w + t] > m) m = s[i * w + t];
      s[off + i] = m;
    }
  }
}

/* ---------------------------------------------------------------- selection (Sec. 3.4) */

typedef struct {
  float c;   /* combined score max(s_QK, s_KQ) */
  int64_t i; /* level-local index              */
} cand_t;

/* (c desc, i asc): the total order used to rank candidates; lower index wins ties. */
static int cand_cmp(const void* a, const void* b) {
  const cand_t* x = (const cand_t*)a;
  const cand_t* y = (const cand_t*)b;
  if (x->c > y->c) return -1;
  if (x->c < y->c) return 1;
  return (x->i < y->i) ? -1 : (x->i > y->i) ? 1 : 0;
}

static int cmp_i64(const void* a, const void* b) {
  int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return x < y ? -1 : x > y ? 1 : 0;
}

typedef struct {
  int64_t key; /* e * L + (L - 1 - l) */
  int32_t id;  /* off_l + i           */
} ord_t;

static int ord_cmp(const void* a, const void* b) {
  int64_t x = ((const ord_t*)a)->key, y = ((const ord_t*)b)->key;
  return x < y ? -1 : x > y ? 1 : 0;
}

/* Selection (Eq. topk with Fig. 2 panel 3; Sec. 3.4 keeps the whole coarsest level) and
   causal ordering (Sec. 3.5, mask paragraph). Reading of the selection: per-level descent.
     E_{L-1} = all entries of the coarsest level.
     For l = L-1 down to 1: rank E_l by (c desc, i asc) with c = max(s_QK, s_KQ) (an entry
     picked through either stream enters as its own triple); the first min(k, |E_l|) are the
     parents; E_{l-1} = the p children {p i + r} of every parent.
     Emitted = union of all E_l (with LHO_REPLACE_PARENTS, parents of levels >= 1 are left out).
     With LHO_STRATIFIED, a level that ranks (k < |E_l|) takes its parents chunk by chunk: E_l in
     index order is cut into chunks of LHO_STRAT_CHUNK, and chunk [s, e) contributes its best
     floor(k e / |E_l|) - floor(k s / |E_l|) candidates (App. D.2 keeps a fixed-size top-m per
     chunk; sizing the shares from k keeps S and every shape of the exact mode).
   Causal order: entry (l, i) has window end e = (i+1) p^l - 1; entries are sorted by
   key = e L + (L - 1 - l), i.e. by e ascending with the coarser level first on equal e.
   Writes idx[0..S) (flattened ids in causal order), slot[Ptot] (position in idx or -1) and
   returns S, or -1 if idx_cap is too small or memory runs out. */
int64_t lho_select(const lho_head* h, const float* s_qk, const float* s_kq, int32_t* idx,
                   int64_t idx_cap, int32_t* slot) {
  const int L = h->L, p = h->p;
  const int64_t ptot = lho_pyramid_rows(h);
  for (int64_t t = 0; t < ptot; ++t) slot[t] = -1;

  /* emitted[l]: sorted level-local indices emitted at level l */
  int64_t** emitted = (int64_t**)calloc((size_t)L, sizeof(int64_t*));
  int64_t* n_emit = (int64_t*)calloc((size_t)L, sizeof(int64_t));
  int64_t n_cand = lho_level_rows(h, L - 1);
  int64_t* cand = (int64_t*)malloc((size_t)(n_cand > 0 ? n_cand : 1) * sizeof(int64_t));
  if (!emitted || !n_emit || !cand) return -1;
  for (int64_t i = 0; i < n_cand; ++i) cand[i] = i;

  for (int l = L - 1; l >= 0; --l) {
    const int64_t off = lho_level_offset(h, l);
    int64_t n_par = 0;
    int64_t* par = NULL;
    if (l >= 1) {
      cand_t* ranked = (cand_t*)malloc((size_t)(n_cand > 0 ? n_cand : 1) * sizeof(cand_t));
      if (!ranked) return -1;
      for (int64_t t = 0; t < n_cand; ++t) {
        float a = s_qk[off + cand[t]], b = s_kq[off + cand[t]];
        ranked[t].c = a > b ? a : b;
        ranked[t].i = cand[t];
      }
      n_par = n_cand < h->k ? n_cand : h->k;
      par = (int64_t*)malloc((size_t)(n_par > 0 ? n_par : 1) * sizeof(int64_t));
      if (!par) return -1;
      if ((h->flags & LHO_STRATIFIED) && n_par < n_cand) {
        /* stratified (App. D.2): the candidates, in index order, are cut into chunks of
           LHO_STRAT_CHUNK; chunk [s, e) keeps the best floor(k e / n) - floor(k s / n) of its
           own candidates, so every chunk contributes its share and the level still keeps k */
        int64_t np = 0;
        for (int64_t s0 = 0; s0 < n_cand; s0 += LHO_STRAT_CHUNK) {
          const int64_t e0 = s0 + LHO_STRAT_CHUNK < n_cand ? s0 + LHO_STRAT_CHUNK : n_cand;
          const int64_t quota = (h->k * e0) / n_cand - (h->k * s0) / n_cand;
          qsort(ranked + s0, (size_t)(e0 - s0), sizeof(cand_t), cand_cmp);
          for (int64_t t = 0; t < quota; ++t) par[np++] = ranked[s0 + t].i;
        }
        if (np != n_par) return -1;
      } else {
        qsort(ranked, (size_t)n_cand, sizeof(cand_t), cand_cmp);
        for (int64_t t = 0; t < n_par; ++t) par[t] = ranked[t].i;
      }
      qsort(par, (size_t)n_par, sizeof(int64_t), cmp_i64);
      free(ranked);
    }
    /* emitted set of this level */
    emitted[l] = (int64_t*)malloc((size_t)(n_cand > 0 ? n_cand : 1) * sizeof(int64_t));
    if (!emitted[l]) return -1;
    int64_t ne = 0;
    for (int64_t t = 0; t < n_cand; ++t) {
      int is_parent = 0;
      if (l >= 1 && (h->flags & LHO_REPLACE_PARENTS)) {
        for (int64_t u = 0; u < n_par; ++u)
          if (par[u] == cand[t]) is_parent = 1;
      }
      if (!is_parent) emitted[l][ne++] = cand[t];
    }
    n_emit[l] = ne;
    if (l == 0) break;
    /* children of the parents are the next level's candidates */
    int64_t* next = (int64_t*)malloc((size_t)(n_par * p > 0 ? n_par * p : 1) * sizeof(int64_t));
    if (!next) return -1;
    for (int64_t u = 0; u < n_par; ++u)
      for (int r = 0; r < p; ++r) next[u * p + r] = par[u] * p + r;
    free(par);
    free(cand);
    cand = next;
    n_cand = n_par * p;
  }
  free(cand);

  int64_t S = 0;
  for (int l = 0; l < L; ++l) S += n_emit[l];
  if (S > idx_cap) return -1;
  ord_t* ord = (ord_t*)malloc((size_t)(S > 0 ? S : 1) * sizeof(ord_t));
  if (!ord) return -1;
  int64_t m = 0;
  for (int l = 0; l < L; ++l) {
    const int64_t w = ipow(p, l), off = lho_level_offset(h, l);
    for (int64_t t = 0; t < n_emit[l]; ++t) {
      const int64_t i = emitted[l][t];
      const int64_t e = (i + 1) * w - 1;
      ord[m].key = e * L + (L - 1 - l);
      ord[m].id = (int32_t)(off + i);
      ++m;
    }
    free(emitted[l]);
  }
  qsort(ord, (size_t)S, sizeof(ord_t), ord_cmp);
  for (int64_t t = 0; t < S; ++t) {
    idx[t] = ord[t].id;
    slot[ord[t].id] = (int32_t)t;
  }
  free(ord);
  free(emitted);
  free(n_emit);
  return S;
}

/* Decodes a flattened id into (level, level-local index). */
static void decode_id(const lho_head* h, int64_t id, int* l_out, int64_t* i_out) {
  int l = 0;
  while (l + 1 < h->L && id >= lho_level_offset(h, l + 1)) ++l;
  *l_out = l;
  *i_out = id - lho_level_offset(h, l);
}

/* ---------------------------------------------------------------- gather (Sec. 3.5) */

/* Gather equation: xs[m] = pyr[idx[m]] (the selected entry's own pooled row). */
void lho_gather(const lho_head* h, const double* pyr, const int32_t* idx, int64_t S, double* xs) {
  for (int64_t m = 0; m < S; ++m) memcpy(xs + m * h->D, pyr + (int64_t)idx[m] * h->D, sizeof(double) * (size_t)h->D);
}

/* ---------------------------------------------------------------- SDPA (Eqs. sdpa, attn-sub) */

/* Causal softmax attention over the gathered order (the mask is lower-triangular on it), for
   one row m: a_t = scale <q_m, k_t> for t <= m, mu = max a, Z = sum exp(a - mu),
   os[m] = sum_t exp(a_t - mu) / Z v_t, lse[m] = mu + log Z. `a` has room for m + 1 values. */
static void sdpa_fwd_row(int D, double scale, const double* qs, const double* ks, const double* vs,
                         double* os, double* lse, int64_t m, double* a) {
  double mu = -INFINITY;
  for (int64_t t = 0; t <= m; ++t) {
    double d = 0.0;
    for (int c = 0; c < D; ++c) d += qs[m * D + c] * ks[t * D + c];
    a[t] = scale * d;
    if (a[t] > mu) mu = a[t];
  }
  double Z = 0.0;
  for (int64_t t = 0; t <= m; ++t) Z += exp(a[t] - mu);
  for (int c = 0; c < D; ++c) os[m * D + c] = 0.0;
  for (int64_t t = 0; t <= m; ++t) {
    const double w = exp(a[t] - mu) / Z;
    for (int c = 0; c < D; ++c) os[m * D + c] += w * vs[t * D + c];
  }
  lse[m] = mu + log(Z);
}

/* Rows m in [r0, r1) of the causal attention above. */
void lho_sdpa_fwd(int64_t S, int D, double scale, const double* qs, const double* ks,
                  const double* vs, double* os, double* lse, int64_t r0, int64_t r1) {
  if (r1 > S) r1 = S;
#pragma omp parallel
  {
    double* a = (double*)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
#pragma omp for schedule(dynamic, 4)
    for (int64_t m = r0; m < r1; ++m) sdpa_fwd_row(D, scale, qs, ks, vs, os, lse, m, a);
    free(a);
  }
}

/* The listed rows rows[0..n) (each in [0, S)) of the causal attention above; other rows of os
   and lse are not touched. Lets a test evaluate sampled rows of a long sequence. */
void lho_sdpa_fwd_rows(int64_t S, int D, double scale, const double* qs, const double* ks,
                       const double* vs, double* os, double* lse, const int64_t* rows, int64_t n) {
#pragma omp parallel
  {
    double* a = (double*)malloc(sizeof(double) * (size_t)(S > 0 ? S : 1));
#pragma omp for schedule(dynamic, 1)
    for (int64_t r = 0; r < n; ++r) sdpa_fwd_row(D, scale, qs, ks, vs, os, lse, rows[r], a);
    free(a);
  }
}

/* Adjoint of lho_sdpa_fwd, written from the definition with P recomputed from lse:
   P_mt = exp(scale <q_m, k_t> - lse_m) for t <= m; Delta_m = <dO_m, O_m>;
   dS_mt = P_mt (<dO_m, v_t> - Delta_m);
   dq_m = scale sum_{t<=m} dS_mt k_t
   dk_t = scale sum_{m>=t} dS_mt q_m, dv_t = sum_{m>=t} P_mt dO_m. */
static double sdpa_delta_row(int D, const double* os, const double* dos, int64_t m) {
  double d = 0.0;
  for (int c = 0; c < D; ++c) d += dos[m * D + c] * os[m * D + c];
  return d;
}

/* dq_m; needs os and lse of row m. */
static void sdpa_dq_row(int D, double scale, const double* qs, const double* ks, const double* vs,
                        const double* os, const double* lse, const double* dos, double* dqs, int64_t m) {
  const double delta = sdpa_delta_row(D, os, dos, m);
  for (int c = 0; c < D; ++c) dqs[m * D + c] = 0.0;
  for (int64_t t = 0; t <= m; ++t) {
    double a = 0.0, dp = 0.0;
    for (int c = 0; c < D; ++c) {
      a += qs[m * D + c] * ks[t * D + c];
      dp += dos[m * D + c] * vs[t * D + c];
    }
    const double P = exp(scale * a - lse[m]);
    const double dS = P * (dp - delta);
    for (int c = 0; c < D; ++c) dqs[m * D + c] += scale * dS * ks[t * D + c];
  }
}

/* dk_t and dv_t; needs os, lse and delta of every row m >= t. */
static void sdpa_dkv_row(int64_t S, int D, double scale, const double* qs, const double* ks,
                         const double* vs, const double* lse, const double* delta, const double* dos,
                         double* dks, double* dvs, int64_t t) {
  for (int c = 0; c < D; ++c) {
    dks[t * D + c] = 0.0;
    dvs[t * D + c] = 0.0;
  }
  for (int64_t m = t; m < S; ++m) {
    double a = 0.0, dp = 0.0;
    for (int c = 0; c < D; ++c) {
      a += qs[m * D + c] * ks[t * D + c];
      dp += dos[m * D + c] * vs[t * D + c];
    }
    const double P = exp(scale * a - lse[m]);
    const double dS = P * (dp - delta[m]);
    for (int c = 0; c < D; ++c) {
      dks[t * D + c] += scale * dS * qs[m * D + c];
      dvs[t * D + c] += P * dos[m * D + c];
    }
  }
}

/* dq for rows m in [q0, q1) and dk, dv for rows t in [k0, k1). The os and lse passed in must be
   the forward's for every row m >= k0 and every m in [q0, q1). */
void lho_sdpa_bwd(int64_t S, int D, double scale, const double* qs, const double* ks,
                  const double* vs, const double* os, const double* lse, const double* dos,
                  double* dqs, double* dks, double* dvs, int64_t q0, int64_t q1, int64_t k0,
                  int64_t k1) {
  if (q1 > S) q1 = S;
  if (k1 > S) k1 = S;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t m = q0; m < q1; ++m) sdpa_dq_row(D, scale, qs, ks, vs, os, lse, dos, dqs, m);
  if (k0 >= k1) return;
  double* delta = (double*)malloc(sizeof(double) * (size_t)S);
  for (int64_t m = k0; m < S; ++m) delta[m] = sdpa_delta_row(D, os, dos, m);
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t t = k0; t < k1; ++t) sdpa_dkv_row(S, D, scale, qs, ks, vs, lse, delta, dos, dks, dvs, t);
  free(delta);
}

/* dq for the listed rows rows[0..n) only (os and lse needed for those rows). */
void lho_sdpa_bwd_dq_rows(int64_t S, int D, double scale, const double* qs, const double* ks,
                          const double* vs, const double* os, const double* lse, const double* dos,
                          double* dqs, const int64_t* rows, int64_t n) {
  (void)S;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < n; ++r) sdpa_dq_row(D, scale, qs, ks, vs, os, lse, dos, dqs, rows[r]);
}

/* ---------------------------------------------------------------- scatter (Sec. 3.6) */

/* Eq. fanout: entry (l, i) owns the shifted range R = [(i+1) p^l - 1, (i+2) p^l - 2]; the
   part past N - 1 is dropped (reading). Eq. scatter: O_j = sum of os[m] over the entries whose
   range holds j; positions no range holds stay 0 (reading). Output o[N, D] (row stride ldo). */
void lho_scatter(const lho_head* h, const int32_t* idx, int64_t S, const double* os, double* o,
                 int64_t ldo) {
  const int D = h->D;
  for (int64_t j = 0; j < h->N; ++j)
    for (int c = 0; c < D; ++c) o[j * ldo + c] = 0.0;
  for (int64_t m = 0; m < S; ++m) {
    int l;
    int64_t i;
    decode_id(h, idx[m], &l, &i);
    const int64_t w = ipow(h->p, l);
    const int64_t lo = (i + 1) * w - 1, hi = (i + 2) * w - 2;
    for (int64_t j = lo; j <= hi && j < h->N; ++j)
      for (int c = 0; c < D; ++c) o[j * ldo + c] += os[m * D + c];
  }
}

/* Adjoint of lho_scatter: dos[m] = sum of dout[j] over j in R(l_m, i_m), j < N. */
void lho_scatter_bwd(const lho_head* h, const int32_t* idx, int64_t S, const double* dout,
                     int64_t ldd, double* dos) {
  const int D = h->D;
  for (int64_t m = 0; m < S; ++m) {
    int l;
    int64_t i;
    decode_id(h, idx[m], &l, &i);
    const int64_t w = ipow(h->p, l);
    const int64_t lo = (i + 1) * w - 1, hi = (i + 2) * w - 2;
    for (int c = 0; c < D; ++c) dos[m * D + c] = 0.0;
    for (int64_t j = lo; j <= hi && j < h->N; ++j)
      for (int c = 0; c < D; ++c) dos[m * D + c] += dout[j * ldd + c];
  }
}

/* ---------------------------------------------------------------- backward of gather + pool */

/* Gradient path (Sec. 3.2, App. C.4): gradients reach the pyramid only through the gathered
   rows. Adjoint of the gather: the gather is injective, so the pyramid gradient of entry
   idx[m] is dxs[m], and 0 for entries not gathered. Adjoint of Eq. pool: base row j receives
   (1/p^l) times the gradient of the level-l entry whose window holds it, summed over levels.
   ADDS into dx[N, D] (row stride ldx) so that a KV head can sum its query heads. */
void lho_gather_pool_bwd(const lho_head* h, const int32_t* idx, int64_t S, const double* dxs,
                         double* dx, int64_t ldx) {
  const int D = h->D;
  const int64_t ptot = lho_pyramid_rows(h);
  double* dpyr = (double*)calloc((size_t)ptot * (size_t)D, sizeof(double));
  for (int64_t m = 0; m < S; ++m)
    for (int c = 0; c < D; ++c) dpyr[(int64_t)idx[m] * D + c] = dxs[m * D + c];
  for (int l = 0; l < h->L; ++l) {
    const int64_t w = ipow(h->p, l), off = lho_level_offset(h, l);
    for (int64_t j = 0; j < h->N; ++j)
      for (int c = 0; c < D; ++c) dx[j * ldx + c] += dpyr[(off + j / w) * D + c] / (double)w;
  }
  free(dpyr);
}

/* ---------------------------------------------------------------- whole layer */

/* Alg. 1 from the pyramid on, for one (b, hq) head problem: pool, score, select, gather, SDPA,
   scatter. q is the query head's [N, D] slice, kk/vv its KV head's slices (row strides given).
   Outputs (caller-allocated): o[N, D] (stride ldo), idx[cap], slot[Ptot], s_qk/s_kq[Ptot],
   qs/ks/vs/os[cap, D], lse[cap]. Returns S or -1. The SDPA rows computed are [0, S). */
int64_t lho_head_forward(const lho_head* h, double scale, const double* q, int64_t ldq,
                         const double* kk, const double* vv, int64_t ldkv, double* o, int64_t ldo,
                         int32_t* idx, int64_t cap, int32_t* slot, float* s_qk, float* s_kq,
                         double* qs, double* ks, double* vs, double* os, double* lse) {
  const int64_t ptot = lho_pyramid_rows(h);
  const int D = h->D;
  double* pyr = (double*)malloc(sizeof(double) * (size_t)ptot * (size_t)D);
  if (!pyr) return -1;
  lho_scores(h, q, ldq, s_qk);
  lho_scores(h, kk, ldkv, s_kq);
  const int64_t S = lho_select(h, s_qk, s_kq, idx, cap, slot);
  if (S < 0) {
    free(pyr);
    return -1;
  }
  lho_pool(h, q, ldq, pyr);
  lho_gather(h, pyr, idx, S, qs);
  lho_pool(h, kk, ldkv, pyr);
  lho_gather(h, pyr, idx, S, ks);
  lho_pool(h, vv, ldkv, pyr);
  lho_gather(h, pyr, idx, S, vs);
  free(pyr);
  lho_sdpa_fwd(S, D, scale, qs, ks, vs, os, lse, 0, S);
  lho_scatter(h, idx, S, os, o, ldo);
  return S;
}

/* Backward of lho_head_forward from dout[N, D]: scatter adjoint, SDPA adjoint, gather and pool
   adjoints. dq is OVERWRITTEN; dk and dv are ADDED to (a KV head sums its query heads). */
int lho_head_backward(const lho_head* h, double scale, const int32_t* idx, int64_t S,
                      const double* qs, const double* ks, const double* vs, const double* os,
                      const double* lse, const double* dout, int64_t ldd, double* dq,
                      int64_t ldq, double* dk, double* dv, int64_t ldkv) {
  const int D = h->D;
  const size_t n = (size_t)(S > 0 ? S : 1) * (size_t)D;
  double* dos = (double*)malloc(sizeof(double) * n);
  double* dqs = (double*)malloc(sizeof(double) * n);
  double* dks = (double*)malloc(sizeof(double) * n);
  double* dvs = (double*)malloc(sizeof(double) * n);
  if (!dos || !dqs || !dks || !dvs) return -1;
  lho_scatter_bwd(h, idx, S, dout, ldd, dos);
  lho_sdpa_bwd(S, D, scale, qs, ks, vs, os, lse, dos, dqs, dks, dvs, 0, S, 0, S);
  for (int64_t j = 0; j < h->N; ++j)
    for (int c = 0; c < D; ++c) dq[j * ldq + c] = 0.0;
  lho_gather_pool_bwd(h, idx, S, dqs, dq, ldq);
  lho_gather_pool_bwd(h, idx, S, dks, dk, ldkv);
  lho_gather_pool_bwd(h, idx, S, dvs, dv, ldkv);
  free(dos);
  free(dqs);
  free(dks);
  free(dvs);
  return 0;
}
