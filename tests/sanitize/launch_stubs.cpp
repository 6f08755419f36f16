// Host-only stand-ins for the kernel launchers, for the sanitizer build of the C ABI's host code
// (api.cpp): they check the shape facts every launcher relies on and count calls, and touch no
// memory and no device.
#include <stdio.h>
#include <stdlib.h>

#include "../../paper_2605_06554_amd/csrc/lh_common.h"

int g_launches = 0;

static hipError_t ok(const LhShape& s) {
  ++g_launches;
  if (s.L < 1 || s.L > 8 || s.Ptot != s.off[s.L] || s.R != s.Ptot - s.N || s.S < 1 || s.S > s.Scand ||
      s.Hq % s.Hkv != 0 || s.G != s.Hq / s.Hkv || s.Hq % s.Hs != 0 || s.Gq * s.Hs != s.Hq) {
    fprintf(stderr, "inconsistent shape passed to a launcher\n");
    abort();
  }
  return hipSuccess;
}

hipError_t lh_launch_pool_score(const LhShape& s, const void*, const void*, const void*, void*, void*, void*,
                                float*, float*, hipStream_t) { return ok(s); }
hipError_t lh_launch_select(const LhShape& s, const float*, const float*, int32_t*, int32_t*, int32_t*,
                            hipStream_t) { return ok(s); }
hipError_t lh_launch_gather(const LhShape& s, const void*, const void*, const void*, const void*, const void*,
                            const void*, const int32_t*, void*, void*, void*, hipStream_t) { return ok(s); }
hipError_t lh_launch_scatter(const LhShape& s, const void*, const int32_t*, void*, hipStream_t) { return ok(s); }
hipError_t lh_launch_scatter_bwd(const LhShape& s, const void*, const int32_t*, void*, hipStream_t) { return ok(s); }
hipError_t lh_launch_gather_bwd(const LhShape& s, const void*, const void*, const void*, const int32_t*, void*, void*,
                                void*, hipStream_t) { return ok(s); }
hipError_t lh_launch_sdpa_fwd(const LhShape& s, const void*, const void*, const void*, void*, float*, hipStream_t) {
  return ok(s);
}
hipError_t lh_launch_sdpa_bwd(const LhShape& s, const void*, const void*, const void*, const void*, const float*,
                              const void*, void*, void*, void*, float*, hipStream_t) { return ok(s); }
hipError_t lh_launch_sdpa_fwd_indexed(const LhShape& s, const void*, const void*, const void*, const void*,
                                      const void*, const void*, const int32_t*, void*, float*, hipStream_t) {
  return ok(s);
}
hipError_t lh_launch_sdpa_bwd_indexed(const LhShape& s, const void*, const void*, const void*, const void*,
                                      const void*, const void*, const int32_t*, const void*, const float*,
                                      const void*, void*, void*, void*, float*, hipStream_t) { return ok(s); }

// the static scratch of lh_sdpa_bwd_noalloc: a fake device address, never dereferenced here
size_t lh_sdpa_scratch_bytes() { return (size_t)16 << 20; }
hipError_t lh_sdpa_scratch(float** out) {
  *out = reinterpret_cast<float*>((uintptr_t)0x7f000000ull);
  return hipSuccess;
}
