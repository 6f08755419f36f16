// Drives every entry point of the C ABI's host code (api.cpp, linked against host-only launcher
// stand-ins) under AddressSanitizer and UndefinedBehaviorSanitizer: valid calls, every pointer
// argument NULL and misaligned in turn, short workspaces, invalid problems, every query helper.
// Device pointers are fake aligned addresses: the host code only validates and offsets them.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "../../include/lighthouse.h"

extern int g_launches;

static int g_fail = 0;
#define EXPECT(cond, ...)              \
  do {                                 \
    if (!(cond)) {                     \
      fprintf(stderr, __VA_ARGS__);    \
      fprintf(stderr, "\n");           \
      ++g_fail;                        \
    }                                  \
  } while (0)

static void* fake(int i) { return (void*)(uintptr_t)(0x10000000ull + 0x100000ull * (uint64_t)i); }

// One entry point: argument i of n is a pointer; `call` runs it with the pointer array.
struct Entry {
  const char* name;
  int nptr;  // pointer arguments (device buffers), in order
  int op;    // workspace owner, or -1
  lh_status (*call)(const lh_problem*, void**, void*, size_t);
  bool bf16_only;
  int optional_from, optional_to;  // pointer args that may be NULL when L == 1 (pyramids), or -1
};

#define P(i) (v[i])
static const Entry kEntries[] = {
    {"lh_pyramid_pool", 6, -1,
     [](const lh_problem* pr, void** v, void*, size_t) { return lh_pyramid_pool(pr, P(0), P(1), P(2), P(3), P(4), P(5), nullptr); },
     false, 3, 6},
    {"lh_score", 4, -1,
     [](const lh_problem* pr, void** v, void*, size_t) {
       return lh_score(pr, P(0), P(1), (float*)P(2), (float*)P(3), nullptr);
     },
     false, -1, -1},
    {"lh_pool_score", 8, -1,
     [](const lh_problem* pr, void** v, void*, size_t) {
       return lh_pool_score(pr, P(0), P(1), P(2), P(3), P(4), P(5), (float*)P(6), (float*)P(7), nullptr);
     },
     false, 3, 6},
    {"lh_select_topk", 4, LH_OP_SELECT,
     [](const lh_problem* pr, void** v, void* ws, size_t n) {
       return lh_select_topk(pr, (float*)P(0), (float*)P(1), (int32_t*)P(2), (int32_t*)P(3), ws, n, nullptr);
     },
     false, -1, -1},
    {"lh_gather", 10, -1,
     [](const lh_problem* pr, void** v, void*, size_t) {
       return lh_gather(pr, P(0), P(1), P(2), P(3), P(4), P(5), (int32_t*)P(6), P(7), P(8), P(9), nullptr);
     },
     false, 3, 6},
    {"lh_sdpa_fwd", 5, -1,
     [](const lh_problem* pr, void** v, void*, size_t) { return lh_sdpa_fwd(pr, P(0), P(1), P(2), P(3), (float*)P(4), nullptr); },
     false, -1, -1},
    {"lh_sdpa_bwd", 9, LH_OP_SDPA_BWD,
     [](const lh_problem* pr, void** v, void* ws, size_t n) {
       return lh_sdpa_bwd(pr, P(0), P(1), P(2), P(3), (float*)P(4), P(5), P(6), P(7), P(8), ws, n, nullptr);
     },
     false, -1, -1},
    {"lh_sdpa_bwd_noalloc", 9, -1,
     [](const lh_problem* pr, void** v, void*, size_t) {
       return lh_sdpa_bwd_noalloc(pr, P(0), P(1), P(2), P(3), (float*)P(4), P(5), P(6), P(7), P(8), nullptr);
     },
     false, -1, -1},
    {"lh_scatter", 3, -1,
     [](const lh_problem* pr, void** v, void*, size_t) { return lh_scatter(pr, P(0), (int32_t*)P(1), P(2), nullptr); },
     false, -1, -1},
    {"lh_scatter_bwd", 3, -1,
     [](const lh_problem* pr, void** v, void*, size_t) { return lh_scatter_bwd(pr, P(0), (int32_t*)P(1), P(2), nullptr); },
     false, -1, -1},
    {"lh_gather_bwd", 7, -1,
     [](const lh_problem* pr, void** v, void*, size_t) {
       return lh_gather_bwd(pr, P(0), P(1), P(2), (int32_t*)P(3), P(4), P(5), P(6), nullptr);
     },
     false, -1, -1},
    {"lh_attention_fwd", 11, LH_OP_ATTENTION_FWD,
     [](const lh_problem* pr, void** v, void* ws, size_t n) {
       return lh_attention_fwd(pr, P(0), P(1), P(2), P(3), (int32_t*)P(4), (int32_t*)P(5), P(6), P(7), P(8), P(9),
                               (float*)P(10), ws, n, nullptr);
     },
     false, -1, -1},
    {"lh_attention_bwd", 11, LH_OP_ATTENTION_BWD,
     [](const lh_problem* pr, void** v, void* ws, size_t n) {
       return lh_attention_bwd(pr, (int32_t*)P(0), (int32_t*)P(1), P(2), P(3), P(4), P(5), (float*)P(6), P(7), P(8),
                               P(9), P(10), ws, n, nullptr);
     },
     false, -1, -1},
    {"lh_sdpa_fwd_indexed", 9, -1,
     [](const lh_problem* pr, void** v, void*, size_t) {
       return lh_sdpa_fwd_indexed(pr, P(0), P(1), P(2), P(3), P(4), P(5), (int32_t*)P(6), P(7), (float*)P(8), nullptr);
     },
     true, 3, 6},
    {"lh_sdpa_bwd_indexed", 13, LH_OP_SDPA_BWD,
     [](const lh_problem* pr, void** v, void* ws, size_t n) {
       return lh_sdpa_bwd_indexed(pr, P(0), P(1), P(2), P(3), P(4), P(5), (int32_t*)P(6), P(7), (float*)P(8), P(9),
                                  P(10), P(11), P(12), ws, n, nullptr);
     },
     true, 3, 6},
    {"lh_attention_fwd_indexed", 11, LH_OP_ATTENTION_FWD_INDEXED,
     [](const lh_problem* pr, void** v, void* ws, size_t n) {
       return lh_attention_fwd_indexed(pr, P(0), P(1), P(2), P(3), (int32_t*)P(4), (int32_t*)P(5), P(6), P(7), P(8),
                                       P(9), (float*)P(10), ws, n, nullptr);
     },
     true, 6, 9},
    {"lh_attention_bwd_indexed", 14, LH_OP_ATTENTION_BWD,
     [](const lh_problem* pr, void** v, void* ws, size_t n) {
       return lh_attention_bwd_indexed(pr, P(0), P(1), P(2), P(3), P(4), P(5), (int32_t*)P(6), (int32_t*)P(7), P(8),
                                       (float*)P(9), P(10), P(11), P(12), P(13), ws, n, nullptr);
     },
     true, 3, 6},
};
#undef P

static void check_entries(const lh_problem& pr) {
  for (const Entry& e : kEntries) {
    if (e.bf16_only && pr.dtype != LH_BF16) {
      std::vector<void*> v(e.nptr);
      for (int i = 0; i < e.nptr; ++i) v[i] = fake(i + 1);
      size_t n = 1ull << 40;
      EXPECT(e.call(&pr, v.data(), fake(0), n) == LH_E_DTYPE, "%s: fp32 must be LH_E_DTYPE", e.name);
      continue;
    }
    size_t need = 0;
    if (e.op >= 0) EXPECT(lh_workspace_bytes(&pr, e.op, &need) == LH_OK, "%s: workspace size", e.name);
    std::vector<void*> v(e.nptr);
    for (int i = 0; i < e.nptr; ++i) v[i] = fake(i + 1);
    const int before = g_launches;
    lh_status st = e.call(&pr, v.data(), fake(0), need);
    EXPECT(st == LH_OK, "%s: valid call returned %s (%s)", e.name, lh_status_str(st), lh_last_error());
    EXPECT(g_launches > before, "%s: nothing launched", e.name);
    for (int i = 0; i < e.nptr; ++i) {
      const bool optional = pr.L == 1 && i >= e.optional_from && i < e.optional_to;
      void* keep = v[i];
      v[i] = nullptr;
      const int b2 = g_launches;
      st = e.call(&pr, v.data(), fake(0), need);
      if (optional) {
        EXPECT(st == LH_OK, "%s: pointer %d may be NULL when L == 1", e.name, i);
      } else {
        EXPECT(st == LH_E_NULL, "%s: NULL pointer %d gave %s", e.name, i, lh_status_str(st));
        EXPECT(g_launches == b2, "%s: launched despite a NULL pointer", e.name);
      }
      v[i] = (void*)((char*)keep + 2);
      st = e.call(&pr, v.data(), fake(0), need);
      if (!optional) EXPECT(st == LH_E_ALIGN, "%s: misaligned pointer %d gave %s", e.name, i, lh_status_str(st));
      v[i] = keep;
    }
    if (need > 0) {
      EXPECT(e.call(&pr, v.data(), fake(0), need - 1) == LH_E_WORKSPACE, "%s: short workspace", e.name);
      EXPECT(e.call(&pr, v.data(), nullptr, need) == LH_E_WORKSPACE, "%s: NULL workspace", e.name);
      EXPECT(e.call(&pr, v.data(), (char*)fake(0) + 16, need) == LH_E_ALIGN, "%s: workspace alignment", e.name);
    }
  }
}

static lh_problem mk(int64_t B, int64_t N, int Hq, int Hkv, int D, int p, int L, int k, int dt, uint32_t flags) {
  lh_problem pr;
  pr.B = B, pr.N = N, pr.Hq = Hq, pr.Hkv = Hkv, pr.D = D, pr.p = p, pr.L = L, pr.k = k, pr.dtype = dt;
  pr.scale = 0.0f, pr.flags = flags;
  return pr;
}

int main() {
  const lh_problem valid[] = {
      mk(1, 1024, 2, 2, 64, 4, 3, 128, LH_F32, 0),       mk(1, 16384, 16, 16, 128, 4, 4, 2048, LH_BF16, 0),
      mk(2, 65536, 32, 32, 128, 4, 4, 4096, LH_BF16, 0), mk(1, 262144, 32, 8, 128, 4, 5, 4096, LH_BF16, 0),
      mk(1, 1048576, 16, 16, 128, 4, 6, 8192, LH_BF16, 0), mk(1, 262144, 32, 8, 128, 4, 5, 4096, LH_BF16, 4),
      mk(1, 777, 2, 2, 128, 4, 1, 0, LH_BF16, 0),         mk(1, 1024, 2, 2, 128, 4, 3, 0, LH_BF16, 0),
      mk(1, 2187, 2, 2, 64, 3, 3, 100, LH_BF16, 1),       mk(1, 16384, 2, 1, 64, 2, 3, 1500, LH_BF16, 2),
      mk(1, 2048, 2, 1, 64, 2, 8, 12, LH_BF16, 0),        mk(2, 1024, 4, 1, 64, 4, 3, 64, LH_F32, 4),
  };
  for (const lh_problem& pr : valid) {
    EXPECT(lh_check(&pr) == LH_OK, "valid problem rejected: %s", lh_last_error());
    const int64_t S = lh_subseq_len(&pr), Ptot = lh_pyramid_rows(&pr);
    EXPECT(S > 0 && Ptot >= pr.N, "shape queries");
    for (int l = -1; l <= pr.L; ++l) {
      const int64_t r = lh_level_rows(&pr, l), o = lh_level_offset(&pr, l);
      if (l < 0 || l >= pr.L) EXPECT(r == -1 && o == -1, "level %d out of range", l);
      else EXPECT(r > 0 && o >= 0 && o < Ptot, "level %d", l);
    }
    for (int op = 0; op <= 4; ++op) {
      size_t b = 0;
      EXPECT(lh_workspace_bytes(&pr, op, &b) == LH_OK, "workspace op %d", op);
    }
    size_t b = 0;
    EXPECT(lh_workspace_bytes(&pr, 99, &b) == LH_E_PARAM, "unknown workspace owner");
    EXPECT(lh_workspace_bytes(&pr, 0, nullptr) == LH_E_NULL, "NULL bytes");
    check_entries(pr);
  }
  const lh_problem invalid[] = {
      mk(1, 1000, 2, 2, 64, 4, 3, 128, LH_F32, 0),  mk(1, 1024, 2, 2, 64, 1, 3, 128, LH_F32, 0),
      mk(1, 1024, 2, 2, 64, 4, 0, 128, LH_F32, 0),  mk(1, 1024, 2, 2, 64, 4, 9, 128, LH_F32, 0),
      mk(1, 1024, 2, 2, 64, 4, 3, -1, LH_F32, 0),   mk(1, 1024, 3, 2, 64, 4, 3, 128, LH_F32, 0),
      mk(1, 1024, 2, 2, 96, 4, 3, 128, LH_F32, 0),  mk(1, 1024, 2, 2, 64, 4, 3, 128, 7, 0),
      mk(1, 1024, 2, 2, 64, 4, 3, 128, LH_F32, 8),  mk(0, 1024, 2, 2, 64, 4, 3, 128, LH_F32, 0),
      mk(1, (int64_t)1 << 28, 1, 1, 64, 2, 2, 1, LH_F32, 0), mk(1, (int64_t)1 << 31, 1, 1, 64, 2, 2, 1, LH_F32, 0),
      mk(1, 1024, 2, 2, 64, 4, 3, 128, LH_F32, 0) /* scale set below */,
  };
  const int n_invalid = (int)(sizeof(invalid) / sizeof(invalid[0]));
  ((lh_problem*)&invalid[n_invalid - 1])->scale = -0.125f;
  for (int i = 0; i < n_invalid; ++i) {
    const lh_problem& pr = invalid[i];
    const lh_status st = lh_check(&pr);
    EXPECT(st != LH_OK && lh_last_error()[0] != 0, "invalid problem %d accepted", i);
    EXPECT(lh_subseq_len(&pr) == -1 && lh_pyramid_rows(&pr) == -1, "queries on invalid problem %d", i);
    std::vector<void*> v(16, fake(1));
    const int before = g_launches;
    for (const Entry& e : kEntries) EXPECT(e.call(&pr, v.data(), fake(0), (size_t)1 << 40) == st, "%s on invalid %d", e.name, i);
    EXPECT(g_launches == before, "launch on an invalid problem");
  }
  {  // the static scratch of lh_sdpa_bwd_noalloc holds B * Hq * S <= 4,194,304 floats
    const lh_problem big = mk(4, 65536, 32, 32, 128, 4, 4, 4096, LH_BF16, 0);
    std::vector<void*> v(16);
    for (int i = 0; i < 16; ++i) v[i] = fake(i + 1);
    const int before = g_launches;
    EXPECT(lh_sdpa_bwd_noalloc(&big, v[0], v[1], v[2], v[3], (float*)v[4], v[5], v[6], v[7], v[8], nullptr) ==
               LH_E_WORKSPACE, "noalloc: oversize problem accepted");
    EXPECT(g_launches == before, "noalloc: launched an oversize problem");
  }
  EXPECT(lh_check(nullptr) == LH_E_NULL, "NULL problem");
  for (int c = 1; c >= -8; --c) EXPECT(lh_status_str((lh_status)c) != nullptr, "status string");
  if (g_fail) {
    fprintf(stderr, "%d failures\n", g_fail);
    return 1;
  }
  printf("abi host code: %d launches, all checks passed\n", g_launches);
  return 0;
}
