/* Runs the oracle's whole head problem (pool, scores, select, gather, SDPA, scatter and every
   adjoint, plus the row-list variants) on small problems under AddressSanitizer and
   UndefinedBehaviorSanitizer. The oracle source is compiled into this program as is. */
#include <stdio.h>
#include <stdlib.h>

#include "../../oracle/lh_oracle.c"

static double urand(unsigned* s) {
  *s = *s * 1103515245u + 12345u;
  return ((*s >> 8) & 0xffff) / 32768.0 - 1.0;
}

static int run(int64_t N, int D, int p, int L, int k, int dtype, unsigned flags) {
  lho_head h = {N, D, p, L, k, dtype, flags};
  if (lho_check(&h) != 0) return 0;
  const int64_t ptot = lho_pyramid_rows(&h);
  unsigned seed = (unsigned)(N * 131 + D * 7 + p * 3 + L + k);
  double* q = malloc(sizeof(double) * N * D);
  double* kk = malloc(sizeof(double) * N * D);
  double* v = malloc(sizeof(double) * N * D);
  double* dout = malloc(sizeof(double) * N * D);
  for (int64_t i = 0; i < N * D; ++i) q[i] = urand(&seed), kk[i] = urand(&seed), v[i] = urand(&seed), dout[i] = urand(&seed);
  int32_t* idx = malloc(sizeof(int32_t) * ptot);
  int32_t* slot = malloc(sizeof(int32_t) * ptot);
  float* sqk = malloc(sizeof(float) * ptot);
  float* skq = malloc(sizeof(float) * ptot);
  double* buf[5];
  for (int i = 0; i < 5; ++i) buf[i] = malloc(sizeof(double) * ptot * D);
  double* lse = malloc(sizeof(double) * ptot);
  double* o = malloc(sizeof(double) * N * D);
  const int64_t S = lho_head_forward(&h, 0.125, q, D, kk, v, D, o, D, idx, ptot, slot, sqk, skq, buf[0], buf[1],
                                     buf[2], buf[3], lse);
  if (S <= 0) return 1;
  double* dq = calloc((size_t)(N * D), sizeof(double));
  double* dk = calloc((size_t)(N * D), sizeof(double));
  double* dv = calloc((size_t)(N * D), sizeof(double));
  if (lho_head_backward(&h, 0.125, idx, S, buf[0], buf[1], buf[2], buf[3], lse, dout, D, dq, D, dk, dv, D) != 0)
    return 1;
  /* row-list variants on every third row */
  int64_t nr = 0;
  int64_t* rows = malloc(sizeof(int64_t) * S);
  for (int64_t m = 0; m < S; m += 3) rows[nr++] = m;
  lho_sdpa_fwd_rows(S, D, 0.125, buf[0], buf[1], buf[2], buf[4], lse, rows, nr);
  lho_sdpa_bwd_dq_rows(S, D, 0.125, buf[0], buf[1], buf[2], buf[3], lse, buf[3], buf[4], rows, nr);
  lho_sdpa_bwd(S, D, 0.125, buf[0], buf[1], buf[2], buf[3], lse, buf[3], buf[4], buf[0], buf[1], S / 2, S, 0, S / 3);
  double acc = 0;
  for (int64_t i = 0; i < N * D; ++i) acc += o[i] + dq[i] + dk[i] + dv[i];
  printf("N=%lld D=%d p=%d L=%d k=%d dtype=%d flags=%u: S=%lld checksum %.6e\n", (long long)N, D, p, L, k, dtype,
         flags, (long long)S, acc);
  free(q), free(kk), free(v), free(dout), free(idx), free(slot), free(sqk), free(skq), free(lse), free(o);
  free(dq), free(dk), free(dv), free(rows);
  for (int i = 0; i < 5; ++i) free(buf[i]);
  return 0;
}

int main(void) {
  int bad = 0;
  bad |= run(1024, 64, 4, 3, 128, LHO_F32, 0);
  bad |= run(1024, 64, 4, 3, 256, LHO_BF16, 0);                 /* full budget */
  bad |= run(1024, 64, 4, 3, 256, LHO_BF16, LHO_REPLACE_PARENTS);
  bad |= run(777, 128, 4, 1, 0, LHO_BF16, 0);                   /* L = 1 */
  bad |= run(1024, 128, 4, 3, 0, LHO_BF16, 0);                  /* k = 0 */
  bad |= run(2187, 64, 3, 3, 100, LHO_BF16, 0);                 /* p = 3 */
  bad |= run(8192, 64, 2, 3, 1500, LHO_BF16, LHO_STRATIFIED);   /* several chunks */
  bad |= run(2048, 64, 2, 8, 12, LHO_F64, 0);                   /* L = 8 */
  bad |= run(112, 64, 2, 5, 5, LHO_BF16, 0);
  bad |= run(1000, 64, 5, 3, 30, LHO_BF16, 0);
  return bad;
}
