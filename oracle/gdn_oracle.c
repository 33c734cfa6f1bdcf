/*
 * gdn_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct fp64 CPU statement of what the large-beam
 * Gated DeltaNet (GDN) decode computes, written from the OneLA paper
 * ("OneLA: Scaling Linear-Attention Decoding to Large Beams in Generative
 * Recommendation", arXiv 2609.12399).  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load this code; the product
 * library never calls it and shares no code with it.
 *
 * What it computes (no blocking, no fusion, no reordering beyond the
 * definitions):
 *   - oracle_gdn_prefill: the GDN transition of Sec. 2.2, Eq. 1, applied
 *     token by token over a prompt, starting from the zero state.  Its
 *     result is the post-prefill context state S_ctx of Sec. 3.1.
 *   - oracle_ancestry: the ancestry index of Sec. 3.3, Eq. 5, on integers.
 *   - oracle_gdn_decode: the "FullState" meaning of a large-beam decode.
 *     Every live beam owns a materialised d_v x d_k state; at step t beam b
 *     copies the state of its parent pi_t(b) (Sec. 2.1 and 3.1; at t = 0 all
 *     beams start from S_ctx), applies Eq. 1 with its own (q, k, v, alpha,
 *     beta), and reads out o = S q after the update (Eq. 1, Eq. 4).
 *
 * Conventions (readings of the paper, stated once here):
 *   - S is d_v x d_k, row-major [d_v][d_k] (Sec. 2.2).
 *   - alpha and beta are given per (beam, value head) (Sec. 3.2, the sentence
 *     after Eq. 4 speaks of accumulators per beam and value head).
 *   - Grouped heads: value head hv reads query/key head hv / (HV / HK).
 *   - No 1/sqrt(d_k) query scaling: Eq. 1 has none.
 *   - All arithmetic is IEEE fp64; inputs arrive already rounded to the
 *     precision the device consumes and are upcast exactly by the caller.
 *
 * Parity pins for every function live in the test suite (closed forms,
 * exact-rational brute force, special cases); none of them re-types these
 * loops.
 */
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* One GDN transition step, Eq. 1, literally:
 *   u = S k                      (uses the old S)
 *   S <- alpha S + beta (v - alpha u) k^T
 * u is scratch of length dv. */
static void gdn_transition(double* S, int dv, int dk, const double* k,
                           const double* v, double alpha, double beta,
                           double* u) {
  for (int i = 0; i < dv; ++i) {
    double acc = 0.0;
    for (int j = 0; j < dk; ++j) acc += S[(size_t)i * dk + j] * k[j];
    u[i] = acc;
  }
  for (int i = 0; i < dv; ++i) {
    double w = beta * (v[i] - alpha * u[i]);
    for (int j = 0; j < dk; ++j)
      S[(size_t)i * dk + j] = alpha * S[(size_t)i * dk + j] + w * k[j];
  }
}

/* Read-out o = S q (Eq. 1, second line). */
static void gdn_readout(const double* S, int dv, int dk, const double* q,
                        double* o) {
  for (int i = 0; i < dv; ++i) {
    double acc = 0.0;
    for (int j = 0; j < dk; ++j) acc += S[(size_t)i * dk + j] * q[j];
    o[i] = acc;
  }
}

static int dims_ok(int HK, int HV, int dk, int dv) {
  return HK > 0 && HV > 0 && dk > 0 && dv > 0 && HV % HK == 0;
}

/* Post-prefill state (Sec. 3.1, S_ctx) of one request: Eq. 1 over P prompt
 * tokens from S = 0.
 *   k     [P][HK][dk]    v    [P][HV][dv]
 *   alpha [P][HV]        beta [P][HV]
 *   S_out [HV][dv][dk]
 * Returns 0, or -1 on bad dimensions. */
int oracle_gdn_prefill(int P, int HK, int HV, int dk, int dv, const double* k,
                       const double* v, const double* alpha,
                       const double* beta, double* S_out, int nthreads) {
  if (P < 0 || !dims_ok(HK, HV, dk, dv)) return -1;
  const int group = HV / HK;
  if (nthreads < 1) nthreads = 1;
#pragma omp parallel for num_threads(nthreads) schedule(dynamic, 1)
  for (int hv = 0; hv < HV; ++hv) {
    const int hk = hv / group;
    double* S = S_out + (size_t)hv * dv * dk;
    double* u = (double*)malloc(sizeof(double) * (size_t)dv);
    memset(S, 0, sizeof(double) * (size_t)dv * dk);
    for (int p = 0; p < P; ++p) {
      gdn_transition(S, dv, dk, k + ((size_t)p * HK + hk) * dk,
                     v + ((size_t)p * HV + hv) * dv,
                     alpha[(size_t)p * HV + hv], beta[(size_t)p * HV + hv], u);
    }
    free(u);
  }
  return 0;
}

/* Ancestry index of one request, Eq. 5:
 *   h_t(b, j) = h_{t-1}(pi_t(b), j)   for 0 <= j < t-1
 *   h_t(b, t-1) = pi_t(b)
 * widths  [T]             W_t, the live beams at step t
 * parents concat over t = 1..T-1 of [W_t], each in [0, W_{t-1})
 * h_out   concat over t = 0..T-1 of [W_t][t]   (step 0 contributes nothing)
 * Returns 0, or -1 if some parent is out of range (h_out then undefined). */
int oracle_ancestry(int T, const int* widths, const int* parents, int* h_out) {
  if (T < 0) return -1;
  for (int t = 0; t < T; ++t)
    if (widths[t] < 1) return -1;
  const int* h_prev = h_out; /* h_0 has zero columns */
  int* h_cur = h_out;
  const int* par = parents;
  for (int t = 1; t < T; ++t) {
    h_cur += (size_t)widths[t - 1] * (t - 1);
    for (int b = 0; b < widths[t]; ++b) {
      const int p = par[b];
      if (p < 0 || p >= widths[t - 1]) return -1;
      for (int j = 0; j < t - 1; ++j)
        h_cur[(size_t)b * t + j] = h_prev[(size_t)p * (t - 1) + j];
      h_cur[(size_t)b * t + (t - 1)] = p;
    }
    par += widths[t];
    h_prev = h_cur;
  }
  return 0;
}

/* Large-beam decode of one request with materialised per-beam states
 * ("FullState").
 *   widths  [T]
 *   S0      [HV][dv][dk]                 shared post-prefill state S_ctx
 *   q, k    concat_t [W_t][HK][dk]
 *   v       concat_t [W_t][HV][dv]
 *   alpha, beta concat_t [W_t][HV]
 *   parents concat_{t>=1} [W_t]          pi_t(b) in [0, W_{t-1})
 *   o       concat_t [W_t][HV][dv]       out
 * Returns 0, -1 on bad dimensions, -2 on a parent out of range, -3 on
 * allocation failure. */
int oracle_gdn_decode(int T, const int* widths, int HK, int HV, int dk, int dv,
                      const double* S0, const double* q, const double* k,
                      const double* v, const double* alpha, const double* beta,
                      const int* parents, double* o, int nthreads) {
  if (T < 0 || !dims_ok(HK, HV, dk, dv)) return -1;
  int wmax = 1;
  for (int t = 0; t < T; ++t) {
    if (widths[t] < 1) return -1;
    if (widths[t] > wmax) wmax = widths[t];
  }
  {
    const int* par = parents;
    for (int t = 1; t < T; ++t) {
      for (int b = 0; b < widths[t]; ++b)
        if (par[b] < 0 || par[b] >= widths[t - 1]) return -2;
      par += widths[t];
    }
  }
  const int group = HV / HK;
  const size_t ssz = (size_t)dv * dk;
  int failed = 0;
  if (nthreads < 1) nthreads = 1;
#pragma omp parallel for num_threads(nthreads) schedule(dynamic, 1)
  for (int hv = 0; hv < HV; ++hv) {
    const int hk = hv / group;
    double* prev = (double*)malloc(sizeof(double) * ssz * (size_t)wmax);
    double* cur = (double*)malloc(sizeof(double) * ssz * (size_t)wmax);
    double* u = (double*)malloc(sizeof(double) * (size_t)dv);
    if (!prev || !cur || !u) {
      free(prev); free(cur); free(u);
#pragma omp atomic write
      failed = 1;
      continue;
    }
    memcpy(prev, S0 + (size_t)hv * ssz, sizeof(double) * ssz);
    size_t row0 = 0;          /* first beam row of step t in the concat arrays */
    const int* par = parents; /* parents of step t (t >= 1) */
    for (int t = 0; t < T; ++t) {
      const int W = widths[t];
      for (int b = 0; b < W; ++b) {
        const size_t row = row0 + (size_t)b;
        const int src = (t == 0) ? 0 : par[b];
        double* S = cur + (size_t)b * ssz;
        memcpy(S, prev + (size_t)src * ssz, sizeof(double) * ssz);
        gdn_transition(S, dv, dk, k + (row * HK + hk) * dk,
                       v + (row * HV + hv) * dv, alpha[row * HV + hv],
                       beta[row * HV + hv], u);
        gdn_readout(S, dv, dk, q + (row * HK + hk) * dk,
                    o + (row * HV + hv) * dv);
      }
      if (t > 0) par += W;
      row0 += (size_t)W;
      double* tmp = prev; prev = cur; cur = tmp;
    }
    free(prev); free(cur); free(u);
  }
  return failed ? -3 : 0;
}

/* Number of OpenMP threads a parallel region would use (1 without OpenMP). */
int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
