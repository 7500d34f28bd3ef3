/*
 * jdob_brute.c — exhaustive search of problem (P1) for tiny instances.
 * TEST INFRASTRUCTURE ONLY (see jdob_oracle.h).
 *
 * Independent of jdob_oracle_body.h: it evaluates the model of Sec. II
 * layer by layer in long double -- Eq. (1) and (2) per layer summed over the
 * local part, Eq. (3)/(4) for the upload, Eq. (5) per offloaded layer summed
 * over the batch part -- and enumerates, for every partition point s < L and
 * GPU level j, every offloading set (all subsets, or only the tails of the
 * gamma-descending list of Alg. 1 when suffix_only) and every CPU level
 * vector of all users, without assuming that users decouple.  Constraints
 * (6), (7) and (8) are tested in their written form.  Users may be
 * heterogeneous (Sec. II): user m's latency uses zeta_m and its own CPU
 * levels, its energy kappa_m, its upload energy p_m.
 */
#include "jdob_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

typedef long double LD;

int jo_brute_f64(const jo_problem_f64 *p, int64_t inst, int suffix_only,
                 jo_brute_result *res) {
  if (!p || !res || inst < 0 || inst >= p->I) return -1;
  const int N = p->N, L = p->L, K = p->K, J = p->J;
  if (N < 1 || N > 10 || L < 1 || K < 1 || J < 1) return -1;
  long nvec = 1;
  for (int m = 0; m < N; ++m) {
    nvec *= K;
    if (nvec > (1L << 20)) return -1;
  }
  const double *cyc = p->cycles + (size_t)inst * L;
  const double *bits = p->bits + (size_t)inst * (L + 1);
  const double *al = p->alpha + (size_t)inst * L;
  const double *be = p->beta + (size_t)inst * L;
  const double *rate = p->rate + (size_t)inst * N;
  const double *T = p->deadline + (size_t)inst * N;
  const LD tfree = p->t_free ? (LD)p->t_free[inst] : 0.0L;

  /* per user m: local latency and energy of layers 1..s at level k */
  LD *lt = calloc((size_t)N * (L + 1) * K, sizeof(LD));
  LD *le = calloc((size_t)N * (L + 1) * K, sizeof(LD));
  LD *ptx = calloc(N, sizeof(LD));
  LD *ut = calloc((size_t)N * (L + 1), sizeof(LD)); /* upload latency      */
  int *kv = calloc(N, sizeof(int));
  int *list = calloc(N, sizeof(int));
  int *inS = calloc(N, sizeof(int));
  int *bestk = calloc(N, sizeof(int));
  int *bestS = calloc(N, sizeof(int));
  if (!lt || !le || !ptx || !ut || !kv || !list || !inS || !bestk || !bestS) {
    free(lt); free(le); free(ptx); free(ut); free(kv); free(list); free(inS);
    free(bestk); free(bestS);
    return -2;
  }
#define LT(m, s, k) lt[((size_t)(m) * (L + 1) + (s)) * K + (k)]
#define LE(m, s, k) le[((size_t)(m) * (L + 1) + (s)) * K + (k)]
  for (int m = 0; m < N; ++m) {
    const size_t o = (size_t)inst * N + m;
    const LD zeta = p->user_zeta ? (LD)p->user_zeta[o] : 1.0L;
    const LD kap = p->user_kappa ? (LD)p->user_kappa[o] : (LD)p->kappa;
    ptx[m] = p->user_p_tx ? (LD)p->user_p_tx[o] : (LD)p->p_tx;
    for (int k = 0; k < K; ++k) {
      LD fk = p->user_local_freq ? (LD)p->user_local_freq[o * K + k] : (LD)p->local_freq[k];
      LD tacc = 0, eacc = 0;
      for (int s = 0; s <= L; ++s) {
        if (s > 0) {
          tacc += zeta * (LD)cyc[s - 1] / fk;          /* Eq. (1) */
          eacc += kap * (LD)cyc[s - 1] * fk * fk;      /* Eq. (2) */
        }
        LT(m, s, k) = tacc;
        LE(m, s, k) = eacc;
      }
    }
  }
  for (int m = 0; m < N; ++m)
    for (int s = 0; s <= L; ++s) ut[m * (L + 1) + s] = (LD)bits[s] / (LD)rate[m]; /* Eq. (3) */

  int found = 0, bs = -1, bj = -1, bb = 0, nfeas = 0;
  LD best = INFINITY, second = INFINITY;

  /* local computing: every user meets (8) on its own; it competes last */
  LD lcE = INFINITY;
  int *lcK = calloc(N, sizeof(int));
  memset(kv, 0, sizeof(int) * N);
  for (long v = 0; v < nvec; ++v) {
    int ok = 1;
    LD E = 0;
    for (int m = 0; m < N && ok; ++m) {
      if (!(LT(m, L, kv[m]) <= (LD)T[m])) ok = 0;
      E += LE(m, L, kv[m]);
    }
    if (ok && E < lcE) {
      lcE = E;
      memcpy(lcK, kv, sizeof(int) * N);
    }
    for (int m = 0; m < N; ++m) { if (++kv[m] < K) break; kv[m] = 0; }
  }

  int *curk = calloc(N, sizeof(int)), *curS = calloc(N, sizeof(int));
  for (int s = 0; s < L; ++s) {
    /* list(M') of Alg. 1: gamma (Eq. (17)) descending; equal gamma puts the
     * higher index first so the lower index is offloaded first */
    for (int m = 0; m < N; ++m) list[m] = m;
    for (int a = 1; a < N; ++a) {
      int x = list[a], c = a - 1;
      LD gx = ut[x * (L + 1) + s] + LT(x, s, K - 1);
      while (c >= 0) {
        LD gc = ut[list[c] * (L + 1) + s] + LT(list[c], s, K - 1);
        if (gc < gx || (gc == gx && list[c] < x)) { list[c + 1] = list[c]; --c; }
        else break;
      }
      list[c + 1] = x;
    }
    for (int j = J - 1; j >= 0; --j) {
      LD stretch = (LD)p->gpu_freq[J - 1] / (LD)p->gpu_freq[j];
      LD gpow = (LD)p->gpu_c * (LD)p->gpu_freq[j] * (LD)p->gpu_freq[j] * (LD)p->gpu_freq[j]
                + (LD)p->gpu_p_static;
      for (long mask = (1L << N) - 1; mask >= 1; --mask) {
        int b = 0;
        for (int m = 0; m < N; ++m) { inS[m] = (int)((mask >> m) & 1); b += inS[m]; }
        if (suffix_only) { /* the set must be the last b entries of list */
          int ok = 1;
          for (int q = 0; q < N; ++q)
            if (inS[list[q]] != (q >= N - b)) { ok = 0; break; }
          if (!ok) continue;
        }
        LD lo = INFINITY;                                        /* Eq. (10) */
        for (int m = 0; m < N; ++m) if (inS[m] && (LD)T[m] < lo) lo = (LD)T[m];
        LD gl = 0;                                               /* Eq. (5)  */
        for (int l = s; l < L; ++l) gl += ((LD)al[l] + (LD)be[l] * (LD)b) * stretch;
        if (!(tfree + gl <= lo)) continue;                       /* (6)      */
        LD choice = INFINITY;
        memset(kv, 0, sizeof(int) * N);
        for (long v = 0; v < nvec; ++v) {
          int ok = 1;
          LD E = 0;
          for (int m = 0; m < N && ok; ++m) {
            if (inS[m]) {
              if (!(LT(m, s, kv[m]) + ut[m * (L + 1) + s] + gl <= lo)) ok = 0; /* (7) */
              E += LE(m, s, kv[m]) + ptx[m] * ut[m * (L + 1) + s];           /* (2),(4) */
            } else {
              if (!(LT(m, L, kv[m]) <= (LD)T[m])) ok = 0;                     /* (8) */
              E += LE(m, L, kv[m]);
            }
          }
          if (ok) {
            E += gpow * gl;                                      /* GPU energy */
            if (E < choice) {
              choice = E;
              for (int m = 0; m < N; ++m) { curk[m] = kv[m]; curS[m] = inS[m]; }
            }
          }
          for (int m = 0; m < N; ++m) { if (++kv[m] < K) break; kv[m] = 0; }
        }
        if (choice == INFINITY) continue;
        ++nfeas;
        if (!found || choice < best) {
          second = best;
          best = choice;
          bs = s; bj = j; bb = b;
          for (int m = 0; m < N; ++m) { bestk[m] = curk[m]; bestS[m] = curS[m]; }
          found = 1;
        } else if (choice < second) {
          second = choice;
        }
      }
    }
  }
  if (lcE < INFINITY) {
    ++nfeas;
    if (!found || lcE < best) {
      second = best;
      best = lcE;
      bs = L; bj = -1; bb = 0;
      for (int m = 0; m < N; ++m) { bestk[m] = lcK[m]; bestS[m] = 0; }
      found = 1;
    } else if (lcE < second) {
      second = lcE;
    }
  }
  res->found = found;
  res->energy = found ? (double)best : INFINITY;
  res->energy_second = (double)second;
  res->cut = found ? bs : -1;
  res->gpu_level = found ? bj : -1;
  res->batch = found ? bb : 0;
  res->num_feasible = nfeas;
  for (int m = 0; m < N; ++m) {
    if (res->user_level) res->user_level[m] = (int8_t)(found ? bestk[m] : -1);
    if (res->user_offload) res->user_offload[m] = (int8_t)(found ? bestS[m] : 0);
  }
  free(lt); free(le); free(ptx); free(ut); free(kv); free(list); free(inS);
  free(bestk); free(bestS); free(lcK); free(curk); free(curS);
#undef LT
#undef LE
  return 0;
}
