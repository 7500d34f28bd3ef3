/*
 * jdob_oracle_body.h — the oracle, written once and instantiated per
 * precision by jdob_oracle.c (REAL = float or double, SFX = f32 or f64).
 * TEST INFRASTRUCTURE ONLY (see jdob_oracle.h).
 *
 * Every function follows the paper's definitions in their plain form; the
 * comments name the equation or algorithm step each line implements.
 */

#define JO_CAT2(a, b) a##_##b
#define JO_CAT(a, b) JO_CAT2(a, b)
#define FN(name) JO_CAT(name, SFX)
#define PROB JO_CAT(jo_problem, SFX)
#define POLICY JO_CAT(jo_policy, SFX)
#define TABLES JO_CAT(jo_tables, SFX)
#define CAND JO_CAT(jo_candidate, SFX)
#define SCRATCH JO_CAT(jo_scratch, SFX)
#define GROUPED JO_CAT(jo_grouped, SFX)
#define GROUPING JO_CAT(jo_grouping, SFX)

/* Per-instance derived quantities. */
typedef struct {
  int N, L, K, J;
  REAL *C;   /* [L+1] cycles of layers 1..s (u, v of Sec. III with q = g = 1) */
  REAL *A;   /* [L+1] sum of alpha over layers s+1..L                        */
  REAL *B;   /* [L+1] sum of beta over layers s+1..L                         */
  REAL *t;   /* [(L+1)*K] local latency of layers 1..s at level k, Eq. (1)    */
  REAL *e;   /* [(L+1)*K] local energy of layers 1..s at level k, Eq. (2)     */
  REAL *r;   /* [J] latency stretch g_{J-1}/g_j of the GPU, Eq. (5)          */
  REAL *Pw;  /* [J] GPU power at level j                                      */
  REAL *up;  /* [N*(L+1)] upload latency of the i-th user of pi at s, Eq. (3) */
  REAL *lo;  /* [N+1] lo[b]: tightest deadline among pi[0..b-1], Eq. (10)     */
  REAL *eL;  /* [N] local-only energy of user m                              */
  int *pi;   /* [N] users by rate descending, ties by index                  */
  int *rank; /* [N] position of user m in pi                                 */
  int *kL;   /* [N] local-only level of user m, -1 if none                   */
  int *lv;   /* [N] levels of the offloaders of the current candidate        */
  REAL *fz;  /* [N] their frequencies (continuous CPU frequency)             */
  REAL *fL;  /* [N] local-only frequency of user m (continuous)              */
  int cont;  /* continuous CPU frequency (JO_MODE_CONTINUOUS)                */
  REAL fmin, fmax, kappa;
  int bmin;  /* smallest batch leaving only locally feasible users            */
  REAL tfree;
} SCRATCH;

static void FN(scratch_free)(SCRATCH *w) {
  free(w->C); free(w->A); free(w->B); free(w->t); free(w->e); free(w->r);
  free(w->Pw); free(w->up); free(w->lo); free(w->eL); free(w->pi);
  free(w->rank); free(w->kL); free(w->lv); free(w->fz); free(w->fL);
}

static int FN(scratch_alloc)(SCRATCH *w, int N, int L, int K, int J) {
  memset(w, 0, sizeof(*w));
  w->N = N; w->L = L; w->K = K; w->J = J;
  w->C = (REAL *)malloc(sizeof(REAL) * (L + 1));
  w->A = (REAL *)malloc(sizeof(REAL) * (L + 1));
  w->B = (REAL *)malloc(sizeof(REAL) * (L + 1));
  w->t = (REAL *)malloc(sizeof(REAL) * (L + 1) * K);
  w->e = (REAL *)malloc(sizeof(REAL) * (L + 1) * K);
  w->r = (REAL *)malloc(sizeof(REAL) * J);
  w->Pw = (REAL *)malloc(sizeof(REAL) * J);
  w->up = (REAL *)malloc(sizeof(REAL) * N * (L + 1));
  w->lo = (REAL *)malloc(sizeof(REAL) * (N + 1));
  w->eL = (REAL *)malloc(sizeof(REAL) * N);
  w->pi = (int *)malloc(sizeof(int) * N);
  w->rank = (int *)malloc(sizeof(int) * N);
  w->kL = (int *)malloc(sizeof(int) * N);
  w->lv = (int *)malloc(sizeof(int) * N);
  w->fz = (REAL *)malloc(sizeof(REAL) * N);
  w->fL = (REAL *)malloc(sizeof(REAL) * N);
  if (!w->C || !w->A || !w->B || !w->t || !w->e || !w->r || !w->Pw || !w->up ||
      !w->lo || !w->eL || !w->pi || !w->rank || !w->kL || !w->lv || !w->fz || !w->fL) {
    FN(scratch_free)(w);
    return -1;
  }
  return 0;
}

static int FN(check_problem)(const PROB *p) {
  if (!p || p->N < 1 || p->L < 1 || p->K < 1 || p->J < 1 || p->I < 0) return -1;
  if (!p->cycles || !p->bits || !p->alpha || !p->beta || !p->rate ||
      !p->deadline || !p->local_freq || !p->gpu_freq) return -1;
  return 0;
}

/* The lowest CPU level whose latency fits the budget: Eq. (20) on a discrete
 * level grid.  Latency decreases and energy increases with the level, so the
 * lowest feasible level is the minimum-energy one.  -1 if none fits. */
static int FN(lowest_level)(const REAL *t_row, int K, REAL budget) {
  for (int k = 0; k < K; ++k)
    if (t_row[k] <= budget) return k;
  return -1;
}

/* Eq. (20) with a continuous CPU frequency: the slowest frequency that
 * finishes cycles Cs within the budget, clamped to [f_min, f_max] (no local
 * layers: f_min).  Called only where the top frequency fits the budget. */
static REAL FN(cont_freq)(const SCRATCH *w, REAL Cs, REAL budget) {
  if (Cs == 0) return w->fmin;
  REAL g = Cs / budget;
  return g < w->fmin ? w->fmin : (g > w->fmax ? w->fmax : g);
}

/* Steps shared by every candidate of one instance. */
static void FN(prepare)(const PROB *p, int64_t inst, SCRATCH *w) {
  const int N = p->N, L = p->L, K = p->K, J = p->J;
  const REAL *cyc = p->cycles + (size_t)inst * L;
  const REAL *bits = p->bits + (size_t)inst * (L + 1);
  const REAL *al = p->alpha + (size_t)inst * L;
  const REAL *be = p->beta + (size_t)inst * L;
  const REAL *rate = p->rate + (size_t)inst * N;
  const REAL *T = p->deadline + (size_t)inst * N;
  const REAL *f = p->local_freq, *g = p->gpu_freq;
  const REAL kappa = (REAL)p->kappa;
  const REAL gc = (REAL)p->gpu_c, p0 = (REAL)p->gpu_p_static;

  w->N = N; w->L = L; w->K = K; w->J = J;  /* may be fewer users than allocated */
  w->tfree = p->t_free ? p->t_free[inst] : (REAL)0;
  w->cont = (p->mode & JO_MODE_CONTINUOUS) != 0;
  w->fmin = f[0];
  w->fmax = f[K - 1];
  w->kappa = kappa;

  /* Sec. III notation: cycles of the local part, and the per-layer GPU
   * latency coefficients summed over the offloaded part. */
  w->C[0] = 0;
  for (int s = 1; s <= L; ++s) w->C[s] = w->C[s - 1] + cyc[s - 1];
  w->A[L] = 0;
  w->B[L] = 0;
  for (int s = L - 1; s >= 0; --s) {
    w->A[s] = w->A[s + 1] + al[s];
    w->B[s] = w->B[s + 1] + be[s];
  }
  /* Eq. (1) latency and Eq. (2) energy of computing layers 1..s at f_k. */
  for (int s = 0; s <= L; ++s)
    for (int k = 0; k < K; ++k) {
      REAL eps = kappa * (f[k] * f[k]);
      w->t[s * K + k] = w->C[s] / f[k];
      w->e[s * K + k] = eps * w->C[s];
    }
  /* Eq. (5): latency scales with 1/f_e; power = dynamic + static. */
  for (int j = 0; j < J; ++j) {
    w->r[j] = g[J - 1] / g[j];
    w->Pw[j] = gc * ((g[j] * g[j]) * g[j]) + p0;
  }

  /* Alg. 1: order users by Eq. (17).  With cycles and CPU levels shared by
   * the users of an instance, gamma_m = O_s/R_m + const(s), so gamma
   * descending is rate ascending; the offload sets of Alg. 2 are the tails
   * of that list, i.e. the heads of pi (rate descending, ties by index). */
  for (int m = 0; m < N; ++m) w->pi[m] = m;
  for (int a = 1; a < N; ++a) { /* insertion sort */
    int x = w->pi[a], c = a - 1;
    while (c >= 0 && (rate[w->pi[c]] < rate[x] ||
                      (rate[w->pi[c]] == rate[x] && w->pi[c] > x))) {
      w->pi[c + 1] = w->pi[c];
      --c;
    }
    w->pi[c + 1] = x;
  }
  for (int i = 0; i < N; ++i) w->rank[w->pi[i]] = i;

  /* Eq. (3) upload latency of the i-th user of pi after layer s. */
  for (int i = 0; i < N; ++i)
    for (int s = 0; s <= L; ++s)
      w->up[i * (L + 1) + s] = bits[s] / rate[w->pi[i]];

  /* Eq. (10): the batch deadline is the tightest deadline in the batch. */
  w->lo[0] = (REAL)INFINITY;
  for (int b = 1; b <= N; ++b) {
    REAL d = T[w->pi[b - 1]];
    w->lo[b] = (d < w->lo[b - 1]) ? d : w->lo[b - 1];
  }

  /* Local computing of the whole chain, constraint (8) with Eq. (20). */
  w->bmin = 0;
  for (int m = 0; m < N; ++m) {
    w->kL[m] = FN(lowest_level)(w->t + L * K, K, T[m]);
    if (w->cont && w->kL[m] >= 0) {
      w->fL[m] = FN(cont_freq)(w, w->C[L], T[m]);
      w->eL[m] = (kappa * (w->fL[m] * w->fL[m])) * w->C[L];
    } else {
      w->fL[m] = (w->kL[m] >= 0) ? f[w->kL[m]] : (REAL)0;
      w->eL[m] = (w->kL[m] >= 0) ? w->e[L * K + w->kL[m]] : (REAL)INFINITY;
    }
  }
  for (int i = 0; i < N; ++i)
    if (w->kL[w->pi[i]] < 0) w->bmin = i + 1;
}

/* Candidate (s, j, b), s < L: users pi[0..b-1] offload after layer s, the
 * GPU runs layers s+1..L at level j for the batch of b.  Returns 1 if every
 * constraint holds, filling w->lv and the energy of Eq. (21). */
static int FN(candidate)(const PROB *p, SCRATCH *w, int s, int j, int b,
                         REAL *energy, REAL *gpu_latency) {
  const int N = w->N, L = w->L, K = w->K;
  const REAL ptx = (REAL)p->p_tx;
  /* Eq. (5) summed over layers s+1..L: sum (alpha_l + beta_l b) * g_max/g_j */
  REAL Phi = (w->A[s] + w->B[s] * (REAL)b) * w->r[j];
  /* time left between the end of the batch and the batch deadline (10) */
  REAL H = w->lo[b] - Phi;
  /* (8): every user that stays local meets its deadline */
  for (int i = b; i < N; ++i)
    if (w->kL[w->pi[i]] < 0) return 0;
  /* (6): the GPU is free early enough */
  if (!(H >= w->tfree)) return 0;
  /* (7) with Eq. (20): each offloader's lowest level finishing in time */
  for (int i = 0; i < b; ++i) {
    REAL budget = H - w->up[i * (L + 1) + s];
    int k = FN(lowest_level)(w->t + s * K, K, budget);
    if (k < 0) return 0;
    w->lv[i] = k;
    /* continuous frequency: Eq. (20) with the clamp */
    if (w->cont) w->fz[i] = FN(cont_freq)(w, w->C[s], budget);
  }
  /* Eq. (21), users in index order, then the GPU energy P_j * Phi */
  REAL acc = 0;
  for (int m = 0; m < N; ++m) {
    int i = w->rank[m];
    if (i < b) {
      REAL e = w->cont ? (w->kappa * (w->fz[i] * w->fz[i])) * w->C[s] : w->e[s * K + w->lv[i]];
      acc = acc + (e + ptx * w->up[i * (L + 1) + s]);
    } else {
      acc = acc + w->eL[m];
    }
  }
  acc = acc + w->Pw[j] * Phi;
  *energy = acc;
  *gpu_latency = Phi;
  return 1;
}

/* Eq. (18) for the head of the offloading list (the user with the largest
 * gamma of the suffix pi[0..b-1]): f_e = g_j is at or above that user's
 * threshold exactly when the user, computing at the top CPU level, meets
 * constraint (7) with the batch of b.  The test is written with the same
 * operations as the candidate's (7) so that the two agree on every input;
 * in exact arithmetic it is the comparison of g_j with the threshold. */
static int FN(meets_threshold)(SCRATCH *w, int s, int j, int b) {
  const int L = w->L, K = w->K;
  REAL gpu_time = (w->A[s] + w->B[s] * (REAL)b) * w->r[j];
  REAL slack = w->lo[b] - gpu_time;
  return w->t[s * K + K - 1] <= slack - w->up[(b - 1) * (L + 1) + s];
}

/* The CPU level (-1 with a continuous frequency) and the frequency user m
 * (pi position rk) runs at: as an offloader of the candidate just filled by
 * candidate(), or locally. */
static void FN(user_choice)(const PROB *p, const SCRATCH *w, int off, int rk, int m, int8_t *lv,
                            REAL *fq) {
  if (off) {
    *lv = (int8_t)(w->cont ? -1 : w->lv[rk]);
    *fq = w->cont ? w->fz[rk] : p->local_freq[w->lv[rk]];
  } else {
    *lv = (int8_t)(w->cont ? -1 : w->kL[m]);
    *fq = w->fL[m];
  }
}

/* Running minimum of Alg. 1/2: the first strict minimum wins. */
typedef struct {
  int found, s, j, b;
  REAL best, second;
  int32_t nfeas;
  int64_t nevals;
  REAL tfree_out; /* Eq. (22) of the winner, once solve_instance has filled it */
} JO_CAT(jo_best, SFX);

static void FN(consider)(JO_CAT(jo_best, SFX) *r, REAL E, int s, int j, int b) {
  ++r->nfeas;
  r->nevals += b;
  if (!r->found || E < r->best) {
    r->second = r->best;
    r->best = E;
    r->s = s; r->j = j; r->b = b;
    r->found = 1;
  } else if (E < r->second) {
    r->second = E;
  }
}

/* Local computing (the partition point s = L of Sec. III). */
static int FN(local_candidate)(SCRATCH *w, REAL *energy) {
  if (w->bmin != 0) return 0;
  REAL acc = 0;
  for (int m = 0; m < w->N; ++m) acc = acc + w->eL[m];
  *energy = acc;
  return 1;
}

/* Eq. (22): the GPU is released when the batch, started once the GPU is free
 * and every offloader has uploaded, ends. */
static REAL FN(release_time)(SCRATCH *w, int s, int b, REAL Phi) {
  const int L = w->L, K = w->K;
  REAL ready = w->tfree;
  for (int i = 0; i < b; ++i) {
    REAL tl = w->cont ? w->C[s] / w->fz[i] : w->t[s * K + w->lv[i]];
    REAL done = tl + w->up[i * (L + 1) + s];
    if (done > ready) ready = done;
  }
  return ready + Phi;
}

/* One instance: the first strict minimum over the mode's family of
 * candidates and local computing (Alg. 1 with Alg. 2 or the grid); for an
 * offloading winner w->lv holds its offloaders' levels afterwards and
 * tfree_out its Eq. (22). */
static JO_CAT(jo_best, SFX) FN(solve_instance)(const PROB *p, int64_t inst, SCRATCH *w) {
  const int N = p->N, L = p->L, J = p->J;
  /* the ablations of Sec. IV: binary offloading keeps the partition point 0
   * (besides local computing); without edge DVFS f_e stays at f_e,max */
  const int s_end = (p->mode & JO_MODE_BINARY) ? 1 : L;
  const int j_low = (p->mode & JO_MODE_FIXED_EDGE) ? J - 1 : 0;
  const int greedy = (p->mode & JO_MODE_GREEDY) != 0;
  FN(prepare)(p, inst, w);
  JO_CAT(jo_best, SFX) r = {0, -1, -1, 0, (REAL)INFINITY, (REAL)INFINITY, 0, 0, (REAL)INFINITY};
  /* Alg. 1 visits partition points upward, Alg. 2 GPU frequencies
   * downward with the batch shrinking; both keep the first strict minimum. */
  for (int s = 0; s < s_end; ++s) {
    if (greedy) {
      /* Alg. 2 with the GPU levels as its frequency sweep.  The set starts
       * as the whole list (a user whose threshold is negative, i.e. who
       * cannot make it at any f_e, fails the test at f_e,max and leaves
       * there); at each f_e the head of the list leaves while f_e is below
       * its threshold; a set that is kept is tried under (6) and (8) with
       * Eqs. (20)-(21); an empty set ends the sweep. */
      int b = N;
      for (int j = J - 1; j >= j_low; --j) {
        while (b >= 1 && !FN(meets_threshold)(w, s, j, b)) --b;
        if (b == 0) break;
        REAL E, Phi;
        if (FN(candidate)(p, w, s, j, b, &E, &Phi)) FN(consider)(&r, E, s, j, b);
      }
    } else {
      for (int j = J - 1; j >= j_low; --j)
        for (int b = N; b >= 1; --b) {
          REAL E, Phi;
          if (FN(candidate)(p, w, s, j, b, &E, &Phi)) FN(consider)(&r, E, s, j, b);
        }
    }
  }
  {
    REAL E;
    if (FN(local_candidate)(w, &E)) FN(consider)(&r, E, L, -1, 0);
  }
  if (r.found && r.s == L) {
    r.tfree_out = w->tfree;
  } else if (r.found) {
    REAL E, Phi;
    FN(candidate)(p, w, r.s, r.j, r.b, &E, &Phi); /* refill the levels */
    r.tfree_out = FN(release_time)(w, r.s, r.b, Phi);
  }
  return r;
}

#include "jdob_oracle_hetero.h"

int FN(jo_solve)(const PROB *p, int64_t start, int64_t count, POLICY *out) {
  if (FN(check_problem)(p) != 0 || !out || start < 0 || count < 0 ||
      start + count > p->I)
    return -1;
  if (FN(is_hetero)(p)) return FN(h_solve)(p, start, count, out);
  const int N = p->N, L = p->L;
  SCRATCH w;
  if (FN(scratch_alloc)(&w, N, L, p->K, p->J) != 0) return -2;

  for (int64_t inst = start; inst < start + count; ++inst) {
    JO_CAT(jo_best, SFX) r = FN(solve_instance)(p, inst, &w);
    const int found = r.found, bs = r.s, bj = r.j, bb = r.b;
    const REAL best = r.best, second = r.second;
    const int32_t nfeas = r.nfeas;
    const int64_t nevals = r.nevals;

    int8_t *ul = out->user_level + (size_t)inst * N;
    int8_t *uo = out->user_offload + (size_t)inst * N;
    if (out->num_feasible) out->num_feasible[inst] = nfeas;
    if (out->num_user_evals) out->num_user_evals[inst] = nevals;
    if (out->energy_second) out->energy_second[inst] = second;
    if (!found) {
      out->status[inst] = 1;
      out->cut[inst] = -1;
      out->gpu_level[inst] = -1;
      out->batch[inst] = 0;
      out->energy[inst] = (REAL)INFINITY;
      out->t_free_out[inst] = (REAL)INFINITY;
      for (int m = 0; m < N; ++m) { ul[m] = -1; uo[m] = 0; }
      if (out->user_freq)
        for (int m = 0; m < N; ++m) out->user_freq[(size_t)inst * N + m] = 0;
      continue;
    }
    out->status[inst] = 0;
    out->cut[inst] = bs;
    out->gpu_level[inst] = bj;
    out->batch[inst] = bb;
    out->energy[inst] = best;
    out->t_free_out[inst] = r.tfree_out;
    REAL *uf = out->user_freq ? out->user_freq + (size_t)inst * N : NULL;
    for (int m = 0; m < N; ++m) {
      const int i = w.rank[m], off = bs < L && i < bb;
      REAL fq;
      uo[m] = (int8_t)off;
      FN(user_choice)(p, &w, off, i, m, &ul[m], &fq);
      if (uf) uf[m] = fq;
    }
  }
  FN(scratch_free)(&w);
  return 0;
}

/* ------------------------------------------------------------------------
 * Outer grouping.  The paper's outer module groups users by deadline
 * similarity and calls the inner algorithm once per group (Sec. II); here
 * groups are runs of consecutive users in deadline order, served in that
 * order, and the GPU free time of a group is the release time (Eq. (22)) of
 * the group before it.
 * ---------------------------------------------------------------------- */

/* Users of one instance by deadline ascending, ties by lower index. */
static void FN(deadline_order)(const PROB *p, int64_t inst, int *ord) {
  const int N = p->N;
  const REAL *T = p->deadline + (size_t)inst * N;
  for (int m = 0; m < N; ++m) ord[m] = m;
  for (int a = 1; a < N; ++a) { /* insertion sort */
    int x = ord[a], c = a - 1;
    while (c >= 0 && (T[ord[c]] > T[x] || (T[ord[c]] == T[x] && ord[c] > x))) {
      ord[c + 1] = ord[c];
      --c;
    }
    ord[c + 1] = x;
  }
}

/* The one-instance problem of the group ord[a..b-1]: its users in user
 * index order (gid), the instance's layers and levels, the GPU free at *tf;
 * with heterogeneous users their parameters are copied to gu (3N + N*K
 * values). */
static void FN(group_problem)(const PROB *p, int64_t inst, const int *ord, int a, int b,
                              const REAL *tf, REAL *grate, REAL *gdl, int *gid, REAL *gu,
                              PROB *sub) {
  const int N = p->N, L = p->L, K = p->K, n = b - a;
  for (int q = 0; q < n; ++q) gid[q] = ord[a + q];
  for (int x = 1; x < n; ++x) { /* members by user index */
    int v = gid[x], c = x - 1;
    while (c >= 0 && gid[c] > v) { gid[c + 1] = gid[c]; --c; }
    gid[c + 1] = v;
  }
  for (int q = 0; q < n; ++q) {
    grate[q] = p->rate[(size_t)inst * N + gid[q]];
    gdl[q] = p->deadline[(size_t)inst * N + gid[q]];
  }
  *sub = *p;
  sub->I = 1;
  sub->N = n;
  sub->cycles = p->cycles + (size_t)inst * L;
  sub->bits = p->bits + (size_t)inst * (L + 1);
  sub->alpha = p->alpha + (size_t)inst * L;
  sub->beta = p->beta + (size_t)inst * L;
  sub->rate = grate;
  sub->deadline = gdl;
  sub->t_free = tf;
  if (FN(is_hetero)(p)) {
    REAL *gz = gu, *gk = gu + N, *gp = gu + 2 * N, *gl = gu + 3 * N;
    for (int q = 0; q < n; ++q) {
      const size_t o = (size_t)inst * N + gid[q];
      if (p->user_zeta) gz[q] = p->user_zeta[o];
      if (p->user_kappa) gk[q] = p->user_kappa[o];
      if (p->user_p_tx) gp[q] = p->user_p_tx[o];
      if (p->user_local_freq)
        for (int k = 0; k < K; ++k) gl[q * K + k] = p->user_local_freq[o * K + k];
    }
    sub->user_zeta = p->user_zeta ? gz : NULL;
    sub->user_kappa = p->user_kappa ? gk : NULL;
    sub->user_p_tx = p->user_p_tx ? gp : NULL;
    sub->user_local_freq = p->user_local_freq ? gl : NULL;
  }
}

/* One group's inner solve, for users sharing their parameters or not. */
static JO_CAT(jo_best, SFX) FN(group_solve)(const PROB *sub, SCRATCH *w,
                                            JO_CAT(jo_hscratch, SFX) *hw) {
  return FN(is_hetero)(sub) ? FN(h_solve_instance)(sub, 0, hw) : FN(solve_instance)(sub, 0, w);
}

/* Member q of a group whose candidate (s, b) was just evaluated (by
 * group_solve, or prepare/candidate): offload flag, level, frequency. */
static void FN(group_member)(const PROB *sub, const SCRATCH *w,
                             const JO_CAT(jo_hscratch, SFX) *hw, int s, int b, int q,
                             int8_t *off, int8_t *lv, REAL *fq) {
  if (FN(is_hetero)(sub)) {
    *off = (int8_t)(s < sub->L && hw->rank[q] < b);
    FN(h_user_choice)(hw, s, b, q, lv, fq);
  } else {
    const int rk = w->rank[q];
    *off = (int8_t)(s < sub->L && rk < b);
    FN(user_choice)(sub, w, *off, rk, q, lv, fq);
  }
}

/* Candidate (s, j, b) of the group sub-problem `sub` (s == L: local
 * computing): whether it meets (6)-(8), its energy (Eq. (21), user index
 * order) and the GPU release time after it (Eq. (22)).  Leaves the scratch
 * filled for group_member. */
static int FN(group_eval)(const PROB *sub, SCRATCH *w, JO_CAT(jo_hscratch, SFX) *hw, int s, int j,
                          int b, REAL *E, REAL *tf) {
  const REAL tin = sub->t_free ? sub->t_free[0] : (REAL)0;
  REAL Phi = 0;
  int ok;
  if (FN(is_hetero)(sub)) {
    FN(h_prepare)(sub, 0, hw);
    if (s == sub->L) {
      ok = FN(h_local)(hw, E);
      *tf = tin;
    } else {
      FN(h_order)(sub, 0, hw, s);
      ok = FN(h_candidate)(hw, s, j, b, E, &Phi);
      if (ok) *tf = FN(h_release)(hw, s, b, Phi);
    }
  } else {
    FN(prepare)(sub, 0, w);
    if (s == sub->L) {
      ok = FN(local_candidate)(w, E);
      *tf = tin;
    } else {
      ok = FN(candidate)(sub, w, s, j, b, E, &Phi);
      if (ok) *tf = FN(release_time)(w, s, b, Phi);
    }
  }
  return ok;
}

/* Adds the state (E, T, from) to the front fr[0..*n) of one prefix, kept
 * sorted by energy: nothing happens if a state of the front has no higher
 * energy and no later release (it was generated first); otherwise the
 * states the new one dominates leave, it enters at its energy's place, and
 * a front longer than JO_FRONT loses its highest energy. */
static void FN(front_add)(REAL *fE, REAL *fT, int *from, int *n, REAL E, REAL T, int src) {
  int m = 0;
  for (int q = 0; q < *n; ++q)
    if (fE[q] <= E && fT[q] <= T) return;
  for (int q = 0; q < *n; ++q) /* keep the states the new one does not dominate */
    if (!(E <= fE[q] && T <= fT[q])) {
      fE[m] = fE[q]; fT[m] = fT[q]; from[m] = from[q];
      ++m;
    }
  int at = m;
  while (at > 0 && fE[at - 1] > E) --at;
  if (at >= JO_FRONT) { /* a full front of lower energies: the new state leaves */
    *n = m;
    return;
  }
  for (int q = m < JO_FRONT ? m : JO_FRONT - 1; q > at; --q) { /* the last of a full front leaves */
    fE[q] = fE[q - 1]; fT[q] = fT[q - 1]; from[q] = from[q - 1];
  }
  fE[at] = E; fT[at] = T; from[at] = src;
  *n = m + 1 < JO_FRONT ? m + 1 : JO_FRONT;
}

int FN(jo_solve_grouped)(const PROB *p, int64_t start, int64_t count, GROUPED *out) {
  if (FN(check_problem)(p) != 0 || !out || start < 0 || count < 0 || start + count > p->I)
    return -1;
  const int N = p->N, L = p->L, F = JO_FRONT;
  SCRATCH w;
  JO_CAT(jo_hscratch, SFX) hw;
  if (FN(scratch_alloc)(&w, N, L, p->K, p->J) != 0) return -2;
  if (FN(h_alloc)(&hw, N, L, p->K, p->J) != 0) {
    FN(scratch_free)(&w);
    return -2;
  }
  REAL *gu = (REAL *)malloc(sizeof(REAL) * (size_t)N * (3 + p->K));
  int *ord = (int *)malloc(sizeof(int) * N), *gid = (int *)malloc(sizeof(int) * N);
  int *fn = (int *)malloc(sizeof(int) * (N + 1)), *from = (int *)malloc(sizeof(int) * (N + 1) * F);
  int *ends = (int *)malloc(sizeof(int) * (N + 1)), *ek = (int *)malloc(sizeof(int) * (N + 1));
  REAL *grate = (REAL *)malloc(sizeof(REAL) * N), *gdl = (REAL *)malloc(sizeof(REAL) * N);
  REAL *fE = (REAL *)malloc(sizeof(REAL) * (N + 1) * F), *fT = (REAL *)malloc(sizeof(REAL) * (N + 1) * F);
  if (!gu || !ord || !gid || !fn || !from || !ends || !ek || !grate || !gdl || !fE || !fT) {
    free(gu); free(ord); free(gid); free(fn); free(from); free(ends); free(ek); free(grate);
    free(gdl); free(fE); free(fT);
    FN(scratch_free)(&w);
    FN(h_free)(&hw);
    return -2;
  }
  for (int64_t inst = start; inst < start + count; ++inst) {
    FN(deadline_order)(p, inst, ord);
    int64_t ninner = 0, nfeas = 0, nevals = 0;
    /* the empty prefix: no energy yet, the GPU free at t_free */
    fn[0] = 1;
    fE[0] = 0;
    fT[0] = p->t_free ? p->t_free[inst] : (REAL)0;
    from[0] = -1;
    for (int i = 1; i <= N; ++i) {
      fn[i] = 0;
      for (int j = 0; j < i; ++j) { /* last group: ord[j..i-1] */
        /* The states of prefix j in the order of their release times, the
         * earliest (the front's last) first.  A later GPU free time only
         * removes candidates (constraint (6)), so the winner of the inner
         * solve at one state is also the winner at every later state whose
         * free time it meets: one inner solve serves that run of states. */
        int k = fn[j] - 1;
        while (k >= 0) {
          PROB sub;
          FN(group_problem)(p, inst, ord, j, i, &fT[j * F + k], grate, gdl, gid, gu, &sub);
          JO_CAT(jo_best, SFX) r = FN(group_solve)(&sub, &w, &hw);
          ++ninner;
          nfeas += r.nfeas;
          nevals += r.nevals;
          if (!r.found) break; /* the states left free the GPU later still */
          FN(front_add)(fE + i * F, fT + i * F, from + i * F, &fn[i], fE[j * F + k] + r.best,
                        r.tfree_out, j * F + k);
          for (--k; k >= 0; --k) {
            REAL E, tf;
            FN(group_problem)(p, inst, ord, j, i, &fT[j * F + k], grate, gdl, gid, gu, &sub);
            if (!FN(group_eval)(&sub, &w, &hw, r.s, r.j, r.b, &E, &tf)) break;
            FN(front_add)(fE + i * F, fT + i * F, from + i * F, &fn[i], fE[j * F + k] + E, tf,
                          j * F + k);
          }
        }
      }
    }
    const size_t o = (size_t)inst * N;
    for (int q = 0; q < N; ++q) {
      out->order[o + q] = (int16_t)ord[q];
      out->group_end[o + q] = 0;
      out->group_cut[o + q] = -1;
      out->group_gpu_level[o + q] = -1;
      out->group_batch[o + q] = 0;
      out->group_energy[o + q] = (REAL)INFINITY;
      out->group_t_free[o + q] = (REAL)INFINITY;
      out->user_level[o + q] = -1;
      out->user_offload[o + q] = 0;
      out->user_group[o + q] = -1;
      if (out->user_freq) out->user_freq[o + q] = 0;
    }
    if (out->num_inner) out->num_inner[inst] = ninner;
    if (out->num_feasible) out->num_feasible[inst] = nfeas;
    if (out->num_user_evals) out->num_user_evals[inst] = nevals;
    if (fn[N] == 0) {
      out->status[inst] = 1;
      out->num_groups[inst] = 0;
      out->energy[inst] = (REAL)INFINITY;
      out->t_free_out[inst] = (REAL)INFINITY;
      continue;
    }
    /* the lowest-energy state of the full order, back to the empty prefix,
     * then its groups replayed in order */
    int G = 0;
    for (int st = N * F; st > 0; st = from[st]) {
      ends[G] = st / F;
      ek[G] = st;
      ++G;
    }
    out->status[inst] = 0;
    out->num_groups[inst] = G;
    out->energy[inst] = fE[N * F];
    out->t_free_out[inst] = fT[N * F];
    int a = 0;
    for (int g = 0; g < G; ++g) {
      const int b = ends[G - 1 - g], prv = from[ek[G - 1 - g]];
      PROB sub;
      FN(group_problem)(p, inst, ord, a, b, &fT[prv], grate, gdl, gid, gu, &sub);
      JO_CAT(jo_best, SFX) r = FN(group_solve)(&sub, &w, &hw);
      out->group_end[o + g] = (int16_t)b;
      out->group_cut[o + g] = r.s;
      out->group_gpu_level[o + g] = r.j;
      out->group_batch[o + g] = r.b;
      out->group_energy[o + g] = r.best;
      out->group_t_free[o + g] = r.tfree_out;
      for (int q = 0; q < b - a; ++q) {
        const int m = gid[q];
        REAL fq;
        FN(group_member)(&sub, &w, &hw, r.s, r.b, q, &out->user_offload[o + m],
                         &out->user_level[o + m], &fq);
        if (out->user_freq) out->user_freq[o + m] = fq;
        out->user_group[o + m] = (int8_t)g;
      }
      a = b;
    }
  }
  free(gu); free(ord); free(gid); free(fn); free(from); free(ends); free(ek); free(grate);
  free(gdl); free(fE); free(fT);
  FN(scratch_free)(&w);
  FN(h_free)(&hw);
  return 0;
}

int FN(jo_eval_grouping)(const PROB *p, int64_t inst, GROUPING *g) {
  if (FN(check_problem)(p) != 0 || !g || inst < 0 || inst >= p->I) return -1;
  const int N = p->N, L = p->L, J = p->J, G = g->num_groups, hetero = FN(is_hetero)(p);
  if (G < 1 || G > N) return -1;
  SCRATCH w;
  JO_CAT(jo_hscratch, SFX) hw;
  if (FN(scratch_alloc)(&w, N, L, p->K, J) != 0) return -2;
  if (FN(h_alloc)(&hw, N, L, p->K, J) != 0) {
    FN(scratch_free)(&w);
    return -2;
  }
  REAL *gu = (REAL *)malloc(sizeof(REAL) * (size_t)N * (3 + p->K));
  int *ord = (int *)malloc(sizeof(int) * N), *gid = (int *)malloc(sizeof(int) * N);
  REAL *grate = (REAL *)malloc(sizeof(REAL) * N), *gdl = (REAL *)malloc(sizeof(REAL) * N);
  if (!gu || !ord || !gid || !grate || !gdl) {
    free(gu); free(ord); free(gid); free(grate); free(gdl);
    FN(scratch_free)(&w);
    FN(h_free)(&hw);
    return -2;
  }
  FN(deadline_order)(p, inst, ord);
  REAL tf = p->t_free ? p->t_free[inst] : (REAL)0, total = 0;
  int feasible = 1, a = 0;
  for (int m = 0; m < N; ++m) {
    g->user_level[m] = -1;
    g->user_offload[m] = 0;
    if (g->user_freq) g->user_freq[m] = 0;
  }
  for (int k = 0; k < G && feasible; ++k) {
    const int b = g->group_end[k], s = g->group_cut[k], j = g->group_gpu_level[k];
    const int bb = g->group_batch[k];
    if (b <= a || b > N || s < 0 || s > L || (s < L && (j < 0 || j >= J || bb < 1 || bb > b - a))) {
      feasible = 0;
      break;
    }
    PROB sub;
    const REAL tin = tf;
    FN(group_problem)(p, inst, ord, a, b, &tin, grate, gdl, gid, gu, &sub);
    REAL E = (REAL)INFINITY, Phi = 0;
    if (hetero) {
      FN(h_prepare)(&sub, 0, &hw);
      if (s == L) {
        feasible = FN(h_local)(&hw, &E);
      } else {
        FN(h_order)(&sub, 0, &hw, s);
        feasible = FN(h_candidate)(&hw, s, j, bb, &E, &Phi);
        if (feasible) tf = FN(h_release)(&hw, s, bb, Phi);
      }
    } else {
      FN(prepare)(&sub, 0, &w);
      if (s == L) {
        feasible = FN(local_candidate)(&w, &E);
      } else {
        feasible = FN(candidate)(&sub, &w, s, j, bb, &E, &Phi);
        if (feasible) tf = FN(release_time)(&w, s, bb, Phi);
      }
    }
    if (!feasible) break;
    total = total + E;
    for (int q = 0; q < b - a; ++q) {
      const int m = gid[q];
      REAL fq;
      FN(group_member)(&sub, &w, &hw, s, bb, q, &g->user_offload[m], &g->user_level[m], &fq);
      if (g->user_freq) g->user_freq[m] = fq;
    }
    a = b;
  }
  if (a != N) feasible = 0;
  g->feasible = feasible;
  g->energy = feasible ? total : (REAL)INFINITY;
  g->t_free_out = feasible ? tf : (REAL)INFINITY;
  free(gu); free(ord); free(gid); free(grate); free(gdl);
  FN(scratch_free)(&w);
  FN(h_free)(&hw);
  return 0;
}

int FN(jo_eval_candidate)(const PROB *p, int64_t inst, int s, int j, int b, CAND *res) {
  if (FN(check_problem)(p) != 0 || !res || inst < 0 || inst >= p->I) return -1;
  const int N = p->N, L = p->L;
  if (s < 0 || s > L) return -1;
  if (s < L && (j < 0 || j >= p->J || b < 1 || b > N)) return -1;
  if (FN(is_hetero)(p)) return FN(h_eval_candidate)(p, inst, s, j, b, res);
  SCRATCH w;
  if (FN(scratch_alloc)(&w, N, L, p->K, p->J) != 0) return -2;
  FN(prepare)(p, inst, &w);
  REAL E = (REAL)INFINITY, Phi = 0;
  if (s == L) {
    res->feasible = FN(local_candidate)(&w, &E);
    res->energy = res->feasible ? E : (REAL)INFINITY;
    res->t_free_out = res->feasible ? w.tfree : (REAL)INFINITY;
    res->gpu_latency = 0;
    for (int m = 0; m < N; ++m) {
      int8_t lv = -1;
      REAL fq = 0;
      if (res->feasible) FN(user_choice)(p, &w, 0, 0, m, &lv, &fq);
      if (res->user_level) res->user_level[m] = lv;
      if (res->user_offload) res->user_offload[m] = 0;
      if (res->user_freq) res->user_freq[m] = fq;
    }
  } else {
    res->feasible = FN(candidate)(p, &w, s, j, b, &E, &Phi);
    res->energy = res->feasible ? E : (REAL)INFINITY;
    res->t_free_out = res->feasible ? FN(release_time)(&w, s, b, Phi) : (REAL)INFINITY;
    res->gpu_latency = (w.A[s] + w.B[s] * (REAL)b) * w.r[j];
    for (int m = 0; m < N; ++m) {
      const int i = w.rank[m];
      int8_t lv = -1;
      REAL fq = 0;
      if (res->feasible) FN(user_choice)(p, &w, i < b, i, m, &lv, &fq); /* levels filled */
      if (res->user_level) res->user_level[m] = lv;
      if (res->user_offload) res->user_offload[m] = (int8_t)(i < b);
      if (res->user_freq) res->user_freq[m] = fq;
    }
  }
  FN(scratch_free)(&w);
  return 0;
}

/* Per-user options of every partition point s = 0..L (row L: local
 * computing, nothing uploaded): Eqs. (1)-(4), the deadline slack and the
 * user's own minimum-energy feasible level (Eq. (20) against T_m alone). */
int FN(jo_user_tables)(const PROB *p, int64_t start, int64_t count, TABLES *out) {
  if (FN(check_problem)(p) != 0 || !out || start < 0 || count < 0 ||
      start + count > p->I)
    return -1;
  if (FN(is_hetero)(p)) return -3; /* one rate order per instance: homogeneous users only */
  const int N = p->N, L = p->L, K = p->K;
  const REAL ptx = (REAL)p->p_tx;
  SCRATCH w;
  if (FN(scratch_alloc)(&w, N, L, K, p->J) != 0) return -2;
  for (int64_t inst = start; inst < start + count; ++inst) {
    FN(prepare)(p, inst, &w);
    const REAL *bits = p->bits + (size_t)inst * (L + 1);
    const REAL *rate = p->rate + (size_t)inst * N;
    const REAL *T = p->deadline + (size_t)inst * N;
    for (int i = 0; i < N; ++i) {
      out->order[inst * N + i] = (int16_t)w.pi[i];
      out->batch_deadline[inst * N + i] = w.lo[i + 1];
    }
    out->min_batch[inst] = w.bmin;
    for (int s = 0; s <= L; ++s)
      for (int m = 0; m < N; ++m) {
        size_t o = ((size_t)inst * (L + 1) + s) * N + m;
        REAL up = (s < L) ? bits[s] / rate[m] : (REAL)0;
        REAL budget = T[m] - up;
        int k = FN(lowest_level)(w.t + s * K, K, budget);
        out->uplink_time[o] = up;
        out->gamma[o] = up + w.t[s * K + K - 1];
        out->self_level[o] = (int8_t)k;
        out->self_energy[o] = (k >= 0) ? w.e[s * K + k] + ptx * up : (REAL)INFINITY;
        out->self_slack[o] = budget - w.t[s * K + (k >= 0 ? k : K - 1)];
      }
  }
  FN(scratch_free)(&w);
  return 0;
}

#undef FN
#undef PROB
#undef POLICY
#undef TABLES
#undef CAND
#undef SCRATCH
#undef GROUPED
#undef GROUPING
