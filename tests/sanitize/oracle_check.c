/* Exercises the fp64 oracle (oracle/gdn_oracle.c) on small random problems
 * with exactly sized buffers, built with the address and undefined-behaviour
 * sanitizers by tests/test_sanitizers.py (without OpenMP).  The numbers it
 * produces are pinned elsewhere; here every call must stay in bounds, return
 * its documented code and leave finite outputs. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_gdn_prefill(int P, int HK, int HV, int dk, int dv, const double* k,
                       const double* v, const double* alpha, const double* beta,
                       double* S_out, int nthreads);
int oracle_ancestry(int T, const int* widths, const int* parents, int* h_out);
int oracle_gdn_decode(int T, const int* widths, int HK, int HV, int dk, int dv,
                      const double* S0, const double* q, const double* k, const double* v,
                      const double* alpha, const double* beta, const int* parents,
                      double* o, int nthreads);

static unsigned long long rs = 88172645463325252ull;
static double urand(void) {
  rs ^= rs << 13; rs ^= rs >> 7; rs ^= rs << 17;
  return (double)(rs >> 11) / 9007199254740992.0;
}
static double* vec(size_t n) {
  double* x = (double*)malloc(sizeof(double) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) x[i] = 2.0 * urand() - 1.0;
  return x;
}
static int finite_all(const double* x, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) return 0;
  return 1;
}

int main(void) {
  int bad = 0;
  for (int trial = 0; trial < 60; ++trial) {
    const int HK = 1 + trial % 3, G = 1 + (trial / 3) % 2, HV = HK * G;
    const int dk = 2 + trial % 5, dv = 1 + (trial * 7) % 6;
    const int P = trial % 9, T = 1 + trial % 4;
    int widths[4];
    size_t rows = 0, nparents = 0;
    for (int t = 0; t < T; ++t) {
      widths[t] = 1 + (trial * 5 + t * 3) % 6;
      rows += (size_t)widths[t];
      if (t > 0) nparents += (size_t)widths[t];
    }
    /* prefill */
    double *pk = vec((size_t)P * HK * dk), *pv = vec((size_t)P * HV * dv);
    double *pa = vec((size_t)P * HV), *pb = vec((size_t)P * HV);
    double* S = (double*)malloc(sizeof(double) * (size_t)HV * dv * dk);
    if (oracle_gdn_prefill(P, HK, HV, dk, dv, pk, pv, pa, pb, S, 1) != 0) ++bad;
    if (!finite_all(S, (size_t)HV * dv * dk)) ++bad;
    /* ancestry and decode */
    int* par = (int*)malloc(sizeof(int) * (nparents ? nparents : 1));
    size_t off = 0, hsize = 0;
    for (int t = 1; t < T; ++t)
      for (int b = 0; b < widths[t]; ++b) par[off++] = (int)(urand() * widths[t - 1]);
    for (int t = 0; t < T; ++t) hsize += (size_t)widths[t] * t;
    int* h = (int*)malloc(sizeof(int) * (hsize ? hsize : 1));
    if (oracle_ancestry(T, widths, par, h) != 0) ++bad;
    for (size_t i = 0; i < hsize; ++i)
      if (h[i] < 0 || h[i] >= 6) ++bad;
    double *q = vec(rows * HK * dk), *k = vec(rows * HK * dk), *v = vec(rows * HV * dv);
    double *al = vec(rows * HV), *be = vec(rows * HV);
    double* o = (double*)malloc(sizeof(double) * rows * HV * dv);
    if (oracle_gdn_decode(T, widths, HK, HV, dk, dv, S, q, k, v, al, be, par, o, 1) != 0) ++bad;
    if (!finite_all(o, rows * HV * dv)) ++bad;
    if (T > 1) { /* a parent out of range is reported, nothing is written out of bounds */
      par[0] = widths[0];
      if (oracle_gdn_decode(T, widths, HK, HV, dk, dv, S, q, k, v, al, be, par, o, 1) != -2) ++bad;
      if (oracle_ancestry(T, widths, par, h) != -1) ++bad;
    }
    /* value heads not a multiple of the key heads: rejected before any access */
    if ((HV + 1) % HK != 0 &&
        oracle_gdn_decode(T, widths, HK, HV + 1, dk, dv, S, q, k, v, al, be, par, o, 1) != -1)
      ++bad;
    free(pk); free(pv); free(pa); free(pb); free(S); free(par); free(h);
    free(q); free(k); free(v); free(al); free(be); free(o);
  }
  if (bad) {
    fprintf(stderr, "%d oracle check(s) failed\n", bad);
    return 1;
  }
  printf("oracle checks: ok\n");
  return 0;
}
