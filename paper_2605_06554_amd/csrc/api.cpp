// api.cpp -- host side of the Lighthouse C ABI (include/lighthouse.h): argument validation,
// shape math (pyramid offsets, candidate counts, gathered length S), workspace sizing and
// carving, and kernel dispatch. No device memory is allocated here and nothing synchronizes.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "lh_common.h"

namespace {

thread_local char g_err[512] = "";

lh_status fail(lh_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

constexpr int kMaxLevels = 8;       // kernels are instantiated for L = 1..8
constexpr int64_t kSelLdsKeys = 32768;        // a level up to this many candidates ranks in LDS
constexpr int64_t kMaxSelect = (int64_t)1 << 26;  // beyond: keys in the workspace (ids < 2^30)

lh_status make_shape(const lh_problem* pr, LhShape* s) {
  if (!pr) return fail(LH_E_NULL, "problem is NULL");
  if (pr->B < 1 || pr->N < 1) return fail(LH_E_SHAPE, "B and N must be >= 1 (B=%lld, N=%lld)", (long long)pr->B, (long long)pr->N);
  if (pr->Hq < 1 || pr->Hkv < 1 || pr->Hq % pr->Hkv != 0)
    return fail(LH_E_PARAM, "need Hq >= 1, Hkv >= 1 and Hq %% Hkv == 0 (Hq=%d, Hkv=%d)", pr->Hq, pr->Hkv);
  if (pr->D != 64 && pr->D != 128) return fail(LH_E_PARAM, "head dim D must be 64 or 128 (D=%d)", pr->D);
  if (pr->L < 1 || pr->L > kMaxLevels) return fail(LH_E_PARAM, "levels L must be in [1, %d] (L=%d)", kMaxLevels, pr->L);
  if (pr->L > 1 && pr->p < 2) return fail(LH_E_PARAM, "pooling factor p must be >= 2 when L > 1 (p=%d)", pr->p);
  if (pr->k < 0) return fail(LH_E_PARAM, "budget k must be >= 0 (k=%d)", pr->k);
  if (pr->dtype != LH_F32 && pr->dtype != LH_BF16) return fail(LH_E_DTYPE, "dtype must be LH_F32 or LH_BF16 (%d)", pr->dtype);
  if (pr->flags & ~(uint32_t)(LH_FLAG_REPLACE_PARENTS | LH_FLAG_STRATIFIED | LH_FLAG_GQA_SHARED))
    return fail(LH_E_PARAM, "unknown flag bits 0x%x", pr->flags);
  if (isnan(pr->scale) || isinf(pr->scale))
    return fail(LH_E_NONFINITE, "scale must be finite (0 selects 1/sqrt(D))");
  if (pr->scale < 0.0f) return fail(LH_E_PARAM, "scale must be >= 0 (0 selects 1/sqrt(D))");
  memset(s, 0, sizeof(*s));
  s->B = pr->B;
  s->N = pr->N;
  s->Hq = pr->Hq;
  s->Hkv = pr->Hkv;
  s->G = pr->Hq / pr->Hkv;
  const bool shared = (pr->flags & LH_FLAG_GQA_SHARED) != 0;
  s->Hs = shared ? pr->Hkv : pr->Hq;
  s->Gq = shared ? s->G : 1;
  s->D = pr->D;
  s->p = pr->L > 1 ? pr->p : (pr->p >= 1 ? pr->p : 1);
  s->L = pr->L;
  s->k = pr->k;
  s->dtype = pr->dtype;
  s->flags = pr->flags;
  s->scale = pr->scale != 0.0f ? pr->scale : (float)(1.0 / sqrt((double)pr->D));
  s->pw[0] = 1;
  for (int l = 1; l < s->L; ++l) {
    if (s->pw[l - 1] > s->N / s->p) return fail(LH_E_SHAPE, "p^(L-1) exceeds N");
    s->pw[l] = s->pw[l - 1] * s->p;
  }
  s->P = s->pw[s->L - 1];
  if (s->N % s->P != 0)
    return fail(LH_E_SHAPE, "p^(L-1) = %lld must divide N = %lld", (long long)s->P, (long long)s->N);
  s->off[0] = 0;
  for (int l = 0; l < s->L; ++l) s->off[l + 1] = s->off[l] + s->N / s->pw[l];
  s->Ptot = s->off[s->L];
  s->R = s->Ptot - s->N;
  if (s->Ptot >= ((int64_t)1 << 31)) return fail(LH_E_SHAPE, "pyramid has %lld >= 2^31 entries", (long long)s->Ptot);
  s->cand[s->L - 1] = s->N / s->P;
  for (int l = s->L - 1; l >= 1; --l) {
    s->npar[l] = s->cand[l] < s->k ? s->cand[l] : s->k;
    s->cand[l - 1] = s->p * s->npar[l];
  }
  s->npar[0] = 0;
  s->coff[0] = 0;
  for (int l = 0; l < s->L; ++l) s->coff[l + 1] = s->coff[l] + s->cand[l];
  s->Scand = s->coff[s->L];
  s->S = s->Scand;
  if (s->flags & LH_FLAG_REPLACE_PARENTS)
    for (int l = 1; l < s->L; ++l) s->S -= s->npar[l];
  s->maxsel = 0;
  for (int l = 1; l < s->L; ++l)
    if (s->npar[l] > 0 && s->npar[l] < s->cand[l] && s->cand[l] > s->maxsel) s->maxsel = s->cand[l];
  if (s->maxsel > kMaxSelect)
    return fail(LH_E_PARAM, "a level ranks %lld candidates; at most %lld are supported", (long long)s->maxsel,
                (long long)kMaxSelect);
  if (s->S >= ((int64_t)1 << 31)) return fail(LH_E_SHAPE, "gathered length too large");
  return LH_OK;
}

size_t esize(const LhShape& s) { return s.dtype == LH_BF16 ? 2 : 4; }
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Selection workspace: the candidate lists [B, Hs, Scand] int32, then, when a level ranks more
// candidates than fit in LDS, one row of maxsel uint32 keys per selection.
size_t sel_bytes(const LhShape& s) {
  size_t b = (size_t)s.B * s.Hs * s.Scand * 4;
  if (s.maxsel > kSelLdsKeys) b += (size_t)s.B * s.Hs * s.maxsel * 4;
  return b;
}

// Workspace layouts (offsets in bytes, each segment 256-byte aligned).
struct FwdWs {
  size_t qpyr, kpyr, vpyr, s_qk, s_kq, sel, total;
};
FwdWs fwd_ws(const LhShape& s) {
  FwdWs w;
  size_t o = 0;
  const size_t es = esize(s);
  w.qpyr = o, o += align256((size_t)s.B * s.R * s.Hq * s.D * es);
  w.kpyr = o, o += align256((size_t)s.B * s.R * s.Hkv * s.D * es);
  w.vpyr = o, o += align256((size_t)s.B * s.R * s.Hkv * s.D * es);
  w.s_qk = o, o += align256((size_t)s.B * s.Hq * s.Ptot * 4);
  w.s_kq = o, o += align256((size_t)s.B * s.Hkv * s.Ptot * 4);
  w.sel = o, o += align256(sel_bytes(s));
  w.total = o;
  return w;
}
struct BwdWs {
  size_t dos, dqs, dks, dvs, delta, total;
};
BwdWs bwd_ws(const LhShape& s) {
  BwdWs w;
  size_t o = 0;
  const size_t t = align256((size_t)s.B * s.Hq * s.S * s.D * esize(s));
  const size_t tkv = align256((size_t)s.B * s.Hs * s.S * s.D * esize(s));  // per selection head
  w.dos = o, o += t;
  w.dqs = o, o += t;
  w.dks = o, o += tkv;
  w.dvs = o, o += tkv;
  w.delta = o, o += align256((size_t)s.B * s.Hq * s.S * 4);
  w.total = o;
  return w;
}

size_t ws_bytes(const LhShape& s, int op) {
  switch (op) {
    case LH_OP_SELECT: return align256(sel_bytes(s));
    case LH_OP_SDPA_BWD: return align256((size_t)s.B * s.Hq * s.S * 4);
    case LH_OP_ATTENTION_FWD: return fwd_ws(s).total;
    case LH_OP_ATTENTION_BWD: return bwd_ws(s).total;
    case LH_OP_ATTENTION_FWD_INDEXED: return fwd_ws(s).total - fwd_ws(s).s_qk;
    default: return (size_t)-1;
  }
}

lh_status need_ptr(const void* p, const char* name) {
  if (!p) return fail(LH_E_NULL, "%s is NULL", name);
  if (((uintptr_t)p & 15u) != 0) return fail(LH_E_ALIGN, "%s is not 16-byte aligned", name);
  return LH_OK;
}

lh_status need_ws(const LhShape& s, int op, const void* ws, size_t bytes) {
  const size_t need = ws_bytes(s, op);
  if (need == 0) return LH_OK;
  if (!ws) return fail(LH_E_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)ws & 255u) != 0) return fail(LH_E_ALIGN, "workspace is not 256-byte aligned");
  if (bytes < need) return fail(LH_E_WORKSPACE, "workspace has %zu bytes, %zu needed", bytes, need);
  return LH_OK;
}

lh_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return LH_OK;
  return fail(LH_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define LH_TRY(x)                   \
  do {                              \
    lh_status _st = (x);            \
    if (_st != LH_OK) return _st;   \
  } while (0)

template <typename T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(reinterpret_cast<unsigned char*>(base) + off);
}

lh_status need_bf16(const LhShape& s, const char* what) {
  if (s.dtype != LH_BF16) return fail(LH_E_DTYPE, "%s: the index-driven SDPA is built for bf16 only", what);
  return LH_OK;
}
lh_status need_inputs(const LhShape& s, const void* q, const void* k, const void* v, const void* qp,
                      const void* kp, const void* vp) {
  LH_TRY(need_ptr(q, "q"));
  LH_TRY(need_ptr(k, "k"));
  LH_TRY(need_ptr(v, "v"));
  if (s.L > 1) {
    LH_TRY(need_ptr(qp, "qpyr"));
    LH_TRY(need_ptr(kp, "kpyr"));
    LH_TRY(need_ptr(vp, "vpyr"));
  }
  return LH_OK;
}

}  // namespace

extern "C" {

lh_status lh_check(const lh_problem* pr) {
  LhShape s;
  return make_shape(pr, &s);
}

int64_t lh_level_rows(const lh_problem* pr, int32_t level) {
  LhShape s;
  if (make_shape(pr, &s) != LH_OK || level < 0 || level >= s.L) return -1;
  return s.N / s.pw[level];
}

int64_t lh_level_offset(const lh_problem* pr, int32_t level) {
  LhShape s;
  if (make_shape(pr, &s) != LH_OK || level < 0 || level >= s.L) return -1;
  return s.off[level];
}

int64_t lh_pyramid_rows(const lh_problem* pr) {
  LhShape s;
  if (make_shape(pr, &s) != LH_OK) return -1;
  return s.Ptot;
}

int64_t lh_subseq_len(const lh_problem* pr) {
  LhShape s;
  if (make_shape(pr, &s) != LH_OK) return -1;
  return s.S;
}

lh_status lh_workspace_bytes(const lh_problem* pr, int32_t op, size_t* bytes) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  if (!bytes) return fail(LH_E_NULL, "bytes is NULL");
  const size_t b = ws_bytes(s, op);
  if (b == (size_t)-1) return fail(LH_E_PARAM, "unknown workspace owner %d", op);
  *bytes = b;
  return LH_OK;
}

const char* lh_status_str(lh_status st) {
  switch (st) {
    case LH_OK: return "LH_OK";
    case LH_E_NULL: return "LH_E_NULL";
    case LH_E_SHAPE: return "LH_E_SHAPE";
    case LH_E_PARAM: return "LH_E_PARAM";
    case LH_E_DTYPE: return "LH_E_DTYPE";
    case LH_E_ALIGN: return "LH_E_ALIGN";
    case LH_E_WORKSPACE: return "LH_E_WORKSPACE";
    case LH_E_HIP: return "LH_E_HIP";
    case LH_E_NONFINITE: return "LH_E_NONFINITE";
    default: return "LH_E_UNKNOWN";
  }
}

const char* lh_last_error(void) { return g_err; }

lh_status lh_pyramid_pool(const lh_problem* pr, const void* q, const void* k, const void* v,
                          void* qpyr, void* kpyr, void* vpyr, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(q, "q"));
  LH_TRY(need_ptr(k, "k"));
  LH_TRY(need_ptr(v, "v"));
  if (s.L > 1) {
    LH_TRY(need_ptr(qpyr, "qpyr"));
    LH_TRY(need_ptr(kpyr, "kpyr"));
    LH_TRY(need_ptr(vpyr, "vpyr"));
  }
  g_err[0] = 0;
  return hip_status(lh_launch_pool_score(s, q, k, v, qpyr, kpyr, vpyr, nullptr, nullptr, (hipStream_t)stream),
                    "lh_pyramid_pool");
}

lh_status lh_score(const lh_problem* pr, const void* q, const void* k, float* s_qk, float* s_kq,
                   void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(q, "q"));
  LH_TRY(need_ptr(k, "k"));
  LH_TRY(need_ptr(s_qk, "s_qk"));
  LH_TRY(need_ptr(s_kq, "s_kq"));
  g_err[0] = 0;
  return hip_status(lh_launch_pool_score(s, q, k, nullptr, nullptr, nullptr, nullptr, s_qk, s_kq, (hipStream_t)stream),
                    "lh_score");
}

lh_status lh_pool_score(const lh_problem* pr, const void* q, const void* k, const void* v, void* qpyr,
                        void* kpyr, void* vpyr, float* s_qk, float* s_kq, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(q, "q"));
  LH_TRY(need_ptr(k, "k"));
  LH_TRY(need_ptr(v, "v"));
  if (s.L > 1) {
    LH_TRY(need_ptr(qpyr, "qpyr"));
    LH_TRY(need_ptr(kpyr, "kpyr"));
    LH_TRY(need_ptr(vpyr, "vpyr"));
  }
  LH_TRY(need_ptr(s_qk, "s_qk"));
  LH_TRY(need_ptr(s_kq, "s_kq"));
  g_err[0] = 0;
  return hip_status(lh_launch_pool_score(s, q, k, v, qpyr, kpyr, vpyr, s_qk, s_kq, (hipStream_t)stream),
                    "lh_pool_score");
}

lh_status lh_select_topk(const lh_problem* pr, const float* s_qk, const float* s_kq, int32_t* idx,
                         int32_t* slot, void* ws, size_t ws_bytes_, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(s_qk, "s_qk"));
  LH_TRY(need_ptr(s_kq, "s_kq"));
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ws(s, LH_OP_SELECT, ws, ws_bytes_));
  g_err[0] = 0;
  return hip_status(lh_launch_select(s, s_qk, s_kq, idx, slot, (int32_t*)ws, (hipStream_t)stream), "lh_select_topk");
}

lh_status lh_gather(const lh_problem* pr, const void* q, const void* k, const void* v,
                    const void* qpyr, const void* kpyr, const void* vpyr, const int32_t* idx,
                    void* qs, void* ks, void* vs, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(q, "q"));
  LH_TRY(need_ptr(k, "k"));
  LH_TRY(need_ptr(v, "v"));
  if (s.L > 1) {
    LH_TRY(need_ptr(qpyr, "qpyr"));
    LH_TRY(need_ptr(kpyr, "kpyr"));
    LH_TRY(need_ptr(vpyr, "vpyr"));
  }
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(qs, "qs"));
  LH_TRY(need_ptr(ks, "ks"));
  LH_TRY(need_ptr(vs, "vs"));
  g_err[0] = 0;
  return hip_status(lh_launch_gather(s, q, k, v, qpyr, kpyr, vpyr, idx, qs, ks, vs, (hipStream_t)stream), "lh_gather");
}

lh_status lh_sdpa_fwd(const lh_problem* pr, const void* qs, const void* ks, const void* vs, void* os,
                      float* lse, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(qs, "qs"));
  LH_TRY(need_ptr(ks, "ks"));
  LH_TRY(need_ptr(vs, "vs"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  g_err[0] = 0;
  return hip_status(lh_launch_sdpa_fwd(s, qs, ks, vs, os, lse, (hipStream_t)stream), "lh_sdpa_fwd");
}

lh_status lh_sdpa_bwd(const lh_problem* pr, const void* qs, const void* ks, const void* vs,
                      const void* os, const float* lse, const void* dos, void* dqs, void* dks,
                      void* dvs, void* ws, size_t ws_bytes_, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(qs, "qs"));
  LH_TRY(need_ptr(ks, "ks"));
  LH_TRY(need_ptr(vs, "vs"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  LH_TRY(need_ptr(dos, "dos"));
  LH_TRY(need_ptr(dqs, "dqs"));
  LH_TRY(need_ptr(dks, "dks"));
  LH_TRY(need_ptr(dvs, "dvs"));
  LH_TRY(need_ws(s, LH_OP_SDPA_BWD, ws, ws_bytes_));
  g_err[0] = 0;
  return hip_status(lh_launch_sdpa_bwd(s, qs, ks, vs, os, lse, dos, dqs, dks, dvs, (float*)ws, (hipStream_t)stream),
                    "lh_sdpa_bwd");
}

lh_status lh_sdpa_bwd_noalloc(const lh_problem* pr, const void* qs, const void* ks, const void* vs,
                              const void* os, const float* lse, const void* dos, void* dqs, void* dks,
                              void* dvs, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(qs, "qs"));
  LH_TRY(need_ptr(ks, "ks"));
  LH_TRY(need_ptr(vs, "vs"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  LH_TRY(need_ptr(dos, "dos"));
  LH_TRY(need_ptr(dqs, "dqs"));
  LH_TRY(need_ptr(dks, "dks"));
  LH_TRY(need_ptr(dvs, "dvs"));
  const size_t need = (size_t)s.B * s.Hq * s.S * sizeof(float);
  if (need > lh_sdpa_scratch_bytes())
    return fail(LH_E_WORKSPACE, "lh_sdpa_bwd_noalloc: Delta needs %zu bytes, the static scratch holds %zu (B*Hq*S <= %zu)",
                need, lh_sdpa_scratch_bytes(), lh_sdpa_scratch_bytes() / sizeof(float));
  float* delta = nullptr;
  LH_TRY(hip_status(lh_sdpa_scratch(&delta), "lh_sdpa_bwd_noalloc: scratch address"));
  g_err[0] = 0;
  return hip_status(lh_launch_sdpa_bwd(s, qs, ks, vs, os, lse, dos, dqs, dks, dvs, delta, (hipStream_t)stream),
                    "lh_sdpa_bwd_noalloc");
}

lh_status lh_scatter(const lh_problem* pr, const void* os, const int32_t* slot, void* o, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ptr(o, "o"));
  g_err[0] = 0;
  return hip_status(lh_launch_scatter(s, os, slot, o, (hipStream_t)stream), "lh_scatter");
}

lh_status lh_scatter_bwd(const lh_problem* pr, const void* dout, const int32_t* slot, void* dos,
                         void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(dout, "dout"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ptr(dos, "dos"));
  g_err[0] = 0;
  return hip_status(lh_launch_scatter_bwd(s, dout, slot, dos, (hipStream_t)stream), "lh_scatter_bwd");
}

lh_status lh_gather_bwd(const lh_problem* pr, const void* dqs, const void* dks, const void* dvs,
                        const int32_t* slot, void* dq, void* dk, void* dv, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(dqs, "dqs"));
  LH_TRY(need_ptr(dks, "dks"));
  LH_TRY(need_ptr(dvs, "dvs"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ptr(dq, "dq"));
  LH_TRY(need_ptr(dk, "dk"));
  LH_TRY(need_ptr(dv, "dv"));
  g_err[0] = 0;
  return hip_status(lh_launch_gather_bwd(s, dqs, dks, dvs, slot, dq, dk, dv, (hipStream_t)stream), "lh_gather_bwd");
}

lh_status lh_attention_fwd(const lh_problem* pr, const void* q, const void* k, const void* v, void* o,
                           int32_t* idx, int32_t* slot, void* qs, void* ks, void* vs, void* os,
                           float* lse, void* ws, size_t ws_bytes_, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(q, "q"));
  LH_TRY(need_ptr(k, "k"));
  LH_TRY(need_ptr(v, "v"));
  LH_TRY(need_ptr(o, "o"));
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ptr(qs, "qs"));
  LH_TRY(need_ptr(ks, "ks"));
  LH_TRY(need_ptr(vs, "vs"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  LH_TRY(need_ws(s, LH_OP_ATTENTION_FWD, ws, ws_bytes_));
  g_err[0] = 0;
  const FwdWs w = fwd_ws(s);
  hipStream_t st = (hipStream_t)stream;
  void* qp = s.L > 1 ? at<void>(ws, w.qpyr) : nullptr;
  void* kp = s.L > 1 ? at<void>(ws, w.kpyr) : nullptr;
  void* vp = s.L > 1 ? at<void>(ws, w.vpyr) : nullptr;
  float* sqk = at<float>(ws, w.s_qk);
  float* skq = at<float>(ws, w.s_kq);
  LH_TRY(hip_status(lh_launch_pool_score(s, q, k, v, qp, kp, vp, sqk, skq, st), "pool_score"));
  LH_TRY(hip_status(lh_launch_select(s, sqk, skq, idx, slot, at<int32_t>(ws, w.sel), st), "select"));
  LH_TRY(hip_status(lh_launch_gather(s, q, k, v, qp, kp, vp, idx, qs, ks, vs, st), "gather"));
  LH_TRY(hip_status(lh_launch_sdpa_fwd(s, qs, ks, vs, os, lse, st), "sdpa_fwd"));
  return hip_status(lh_launch_scatter(s, os, slot, o, st), "scatter");
}

lh_status lh_attention_bwd(const lh_problem* pr, const int32_t* idx, const int32_t* slot,
                           const void* qs, const void* ks, const void* vs, const void* os,
                           const float* lse, const void* dout, void* dq, void* dk, void* dv,
                           void* ws, size_t ws_bytes_, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ptr(qs, "qs"));
  LH_TRY(need_ptr(ks, "ks"));
  LH_TRY(need_ptr(vs, "vs"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  LH_TRY(need_ptr(dout, "dout"));
  LH_TRY(need_ptr(dq, "dq"));
  LH_TRY(need_ptr(dk, "dk"));
  LH_TRY(need_ptr(dv, "dv"));
  LH_TRY(need_ws(s, LH_OP_ATTENTION_BWD, ws, ws_bytes_));
  g_err[0] = 0;
  const BwdWs w = bwd_ws(s);
  hipStream_t st = (hipStream_t)stream;
  void* dos = at<void>(ws, w.dos);
  void* dqs = at<void>(ws, w.dqs);
  void* dks = at<void>(ws, w.dks);
  void* dvs = at<void>(ws, w.dvs);
  LH_TRY(hip_status(lh_launch_scatter_bwd(s, dout, slot, dos, st), "scatter_bwd"));
  LH_TRY(hip_status(lh_launch_sdpa_bwd(s, qs, ks, vs, os, lse, dos, dqs, dks, dvs, at<float>(ws, w.delta), st),
                    "sdpa_bwd"));
  return hip_status(lh_launch_gather_bwd(s, dqs, dks, dvs, slot, dq, dk, dv, st), "gather_bwd");
}


lh_status lh_sdpa_fwd_indexed(const lh_problem* pr, const void* q, const void* k, const void* v,
                              const void* qpyr, const void* kpyr, const void* vpyr,
                              const int32_t* idx, void* os, float* lse, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_bf16(s, "lh_sdpa_fwd_indexed"));
  LH_TRY(need_inputs(s, q, k, v, qpyr, kpyr, vpyr));
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  g_err[0] = 0;
  return hip_status(lh_launch_sdpa_fwd_indexed(s, q, k, v, qpyr, kpyr, vpyr, idx, os, lse, (hipStream_t)stream),
                    "lh_sdpa_fwd_indexed");
}

lh_status lh_sdpa_bwd_indexed(const lh_problem* pr, const void* q, const void* k, const void* v,
                              const void* qpyr, const void* kpyr, const void* vpyr,
                              const int32_t* idx, const void* os, const float* lse,
                              const void* dos, void* dqs, void* dks, void* dvs, void* ws,
                              size_t ws_bytes_, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_bf16(s, "lh_sdpa_bwd_indexed"));
  LH_TRY(need_inputs(s, q, k, v, qpyr, kpyr, vpyr));
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  LH_TRY(need_ptr(dos, "dos"));
  LH_TRY(need_ptr(dqs, "dqs"));
  LH_TRY(need_ptr(dks, "dks"));
  LH_TRY(need_ptr(dvs, "dvs"));
  LH_TRY(need_ws(s, LH_OP_SDPA_BWD, ws, ws_bytes_));
  g_err[0] = 0;
  return hip_status(lh_launch_sdpa_bwd_indexed(s, q, k, v, qpyr, kpyr, vpyr, idx, os, lse, dos, dqs, dks, dvs,
                                               (float*)ws, (hipStream_t)stream),
                    "lh_sdpa_bwd_indexed");
}

lh_status lh_attention_fwd_indexed(const lh_problem* pr, const void* q, const void* k, const void* v, void* o,
                                   int32_t* idx, int32_t* slot, void* qpyr, void* kpyr, void* vpyr, void* os,
                                   float* lse, void* ws, size_t ws_bytes_, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_bf16(s, "lh_attention_fwd_indexed"));
  LH_TRY(need_inputs(s, q, k, v, qpyr, kpyr, vpyr));
  LH_TRY(need_ptr(o, "o"));
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  LH_TRY(need_ws(s, LH_OP_ATTENTION_FWD_INDEXED, ws, ws_bytes_));
  g_err[0] = 0;
  // the workspace holds the scores and selection lists of lh_attention_fwd's, from offset 0
  const FwdWs w = fwd_ws(s);
  const size_t base = w.s_qk;
  hipStream_t st = (hipStream_t)stream;
  void* qp = s.L > 1 ? qpyr : nullptr;
  void* kp = s.L > 1 ? kpyr : nullptr;
  void* vp = s.L > 1 ? vpyr : nullptr;
  float* sqk = at<float>(ws, w.s_qk - base);
  float* skq = at<float>(ws, w.s_kq - base);
  LH_TRY(hip_status(lh_launch_pool_score(s, q, k, v, qp, kp, vp, sqk, skq, st), "pool_score"));
  LH_TRY(hip_status(lh_launch_select(s, sqk, skq, idx, slot, at<int32_t>(ws, w.sel - base), st), "select"));
  LH_TRY(hip_status(lh_launch_sdpa_fwd_indexed(s, q, k, v, qp, kp, vp, idx, os, lse, st), "sdpa_fwd_indexed"));
  return hip_status(lh_launch_scatter(s, os, slot, o, st), "scatter");
}

lh_status lh_attention_bwd_indexed(const lh_problem* pr, const void* q, const void* k, const void* v,
                                   const void* qpyr, const void* kpyr, const void* vpyr, const int32_t* idx,
                                   const int32_t* slot, const void* os, const float* lse, const void* dout,
                                   void* dq, void* dk, void* dv, void* ws, size_t ws_bytes_, void* stream) {
  LhShape s;
  LH_TRY(make_shape(pr, &s));
  LH_TRY(need_bf16(s, "lh_attention_bwd_indexed"));
  LH_TRY(need_inputs(s, q, k, v, qpyr, kpyr, vpyr));
  LH_TRY(need_ptr(idx, "idx"));
  LH_TRY(need_ptr(slot, "slot"));
  LH_TRY(need_ptr(os, "os"));
  LH_TRY(need_ptr(lse, "lse"));
  LH_TRY(need_ptr(dout, "dout"));
  LH_TRY(need_ptr(dq, "dq"));
  LH_TRY(need_ptr(dk, "dk"));
  LH_TRY(need_ptr(dv, "dv"));
  LH_TRY(need_ws(s, LH_OP_ATTENTION_BWD, ws, ws_bytes_));
  g_err[0] = 0;
  const BwdWs w = bwd_ws(s);
  hipStream_t st = (hipStream_t)stream;
  void* dos = at<void>(ws, w.dos);
  void* dqs = at<void>(ws, w.dqs);
  void* dks = at<void>(ws, w.dks);
  void* dvs = at<void>(ws, w.dvs);
  const void* qp = s.L > 1 ? qpyr : nullptr;
  const void* kp = s.L > 1 ? kpyr : nullptr;
  const void* vp = s.L > 1 ? vpyr : nullptr;
  LH_TRY(hip_status(lh_launch_scatter_bwd(s, dout, slot, dos, st), "scatter_bwd"));
  LH_TRY(hip_status(lh_launch_sdpa_bwd_indexed(s, q, k, v, qp, kp, vp, idx, os, lse, dos, dqs, dks, dvs,
                                               at<float>(ws, w.delta), st),
                    "sdpa_bwd_indexed"));
  return hip_status(lh_launch_gather_bwd(s, dqs, dks, dvs, slot, dq, dk, dv, st), "gather_bwd");
}

}  // extern "C"
