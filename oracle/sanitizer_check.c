/*
 * sanitizer_check.c -- drives every entry point of the CPU oracle on small
 * seeded cases (scalar and vector emission, n = k, L = 1, B = 0, one and
 * several threads) and prints one checksum line per call.  Built twice by
 * the tests, once with -fsanitize=address,undefined and once without: the
 * sanitized run must exit cleanly and print the same lines.
 * TEST INFRASTRUCTURE ONLY, like the oracle itself.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "bcjr_oracle.h"

static uint64_t rng_state = 0x243F6A8885A308D3ull;

/* uniform in [-2, 2) from a 64-bit linear congruential generator (Knuth's MMIX constants) */
static double draw(void) {
  rng_state = rng_state * 6364136223846793005ull + 1442695040888963407ull;
  return ((double)(rng_state >> 11) / 9007199254740992.0) * 4.0 - 2.0;
}

static double sum_abs(const double *x, int64_t n) {
  double s = 0.0;
  for (int64_t i = 0; i < n; ++i) s += fabs(x[i]) * (double)(1 + i % 7);
  return s;
}

static long isum(const int32_t *x, int64_t n) {
  long s = 0;
  for (int64_t i = 0; i < n; ++i) s += (long)x[i] * (long)(1 + i % 5);
  return s;
}

static int run_case(int n, int k, int V, int64_t B, int64_t L, double T, int threads) {
  const int64_t S = (int64_t)1 << n, N = L / V;
  double *c = malloc(sizeof(double) * (size_t)(S * V));
  double *w = malloc(sizeof(double) * (size_t)(B * L + 1));
  double *g = malloc(sizeof(double) * (size_t)(B * L + 1));
  double *ws = malloc(sizeof(double) * (size_t)(B * L + 1));
  double *lz = malloc(sizeof(double) * (size_t)(B + 1));
  double *dW = malloc(sizeof(double) * (size_t)(B * L + 1));
  double *dc = malloc(sizeof(double) * (size_t)(S * V));
  int32_t *st = malloc(sizeof(int32_t) * (size_t)(B * N + 1));
  double *cost = malloc(sizeof(double) * (size_t)(B + 1));
  double *gap = malloc(sizeof(double) * (size_t)(B * N + 1));
  double *al = malloc(sizeof(double) * (size_t)(N * S));
  double *be = malloc(sizeof(double) * (size_t)(N * S));
  double *A = malloc(sizeof(double) * (size_t)(N * S));
  double *Bt = malloc(sizeof(double) * (size_t)(N * S));
  int rc = 0;
  for (int64_t i = 0; i < S * V; ++i) c[i] = draw();
  for (int64_t i = 0; i < B * L; ++i) w[i] = draw();
  for (int64_t i = 0; i < B * L; ++i) g[i] = draw();
  rc |= oracle_soft_codeword_v(w, B, L, c, n, k, V, T, ws, lz, threads);
  printf("soft n=%d k=%d V=%d B=%ld L=%ld: %.17g %.17g\n", n, k, V, (long)B, (long)L,
         sum_abs(ws, B * L), sum_abs(lz, B));
  rc |= oracle_soft_codeword_vjp_v(w, B, L, c, n, k, V, T, g, ws, lz, dW, dc, threads);
  printf("vjp: %.17g %.17g\n", sum_abs(dW, B * L), sum_abs(dc, S * V));
  rc |= oracle_soft_codeword_vjp_v(w, B, L, c, n, k, V, T, g, NULL, NULL, dW, NULL, threads);
  printf("vjp dW only: %.17g\n", sum_abs(dW, B * L));
  rc |= oracle_viterbi_v(w, B, L, c, n, k, V, st, cost, threads);
  printf("viterbi: %ld %.17g\n", isum(st, B * N), sum_abs(cost, B));
  if (B > 0) {
    rc |= oracle_maxmarginal_gap_v(w, B, L, c, n, k, V, st, gap, threads);
    printf("gap: %.17g\n", sum_abs(gap, B * N));
    rc |= oracle_block_tables_v(w, L, c, n, k, V, T, g, al, be, A, Bt);
    printf("tables: %.17g %.17g %.17g %.17g\n", sum_abs(al, N * S), sum_abs(be, N * S),
           sum_abs(A, N * S), sum_abs(Bt, N * S));
    rc |= oracle_block_tables_v(w, L, c, n, k, V, T, NULL, al, be, NULL, NULL);
  }
  free(c); free(w); free(g); free(ws); free(lz); free(dW); free(dc); free(st); free(cost);
  free(gap); free(al); free(be); free(A); free(Bt);
  return rc;
}

int main(void) {
  int rc = 0;
  rc |= run_case(4, 2, 1, 5, 9, 0.7, 1);
  rc |= run_case(4, 2, 1, 7, 12, 0.05, 3);
  rc |= run_case(3, 1, 1, 4, 10, 1.5, 2);
  rc |= run_case(6, 3, 1, 3, 6, 0.3, 4);
  rc |= run_case(2, 2, 1, 3, 5, 0.4, 2);   /* n = k: fully connected */
  rc |= run_case(5, 2, 1, 6, 1, 0.2, 8);   /* L = 1 */
  rc |= run_case(4, 2, 1, 0, 8, 0.5, 2);   /* B = 0 */
  rc |= run_case(6, 4, 2, 3, 8, 0.6, 2);   /* vector emission, 16 predecessors */
  rc |= run_case(4, 2, 2, 2, 6, 0.9, 1);
  /* argument checks must reject, not read out of bounds */
  double x = 0.0;
  int32_t bad_state[2] = {-1, 99};
  double gap[2];
  if (oracle_soft_codeword(&x, 1, 0, &x, 4, 2, 1.0, &x, &x, 1) == 0) rc |= 1;
  if (oracle_viterbi(&x, 1, 1, &x, 3, 4, bad_state, NULL, 1) == 0) rc |= 1;
  if (oracle_maxmarginal_gap_v(&x, 2, 1, &x, 2, 1, 1, bad_state, gap, 1) == 0) rc |= 1;
  printf("status %d\n", rc);
  return rc == 0 ? 0 : 1;
}
