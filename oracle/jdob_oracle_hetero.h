/*
 * jdob_oracle_hetero.h — the oracle for heterogeneous users, included by
 * jdob_oracle_body.h once per precision (REAL, SFX and FN defined there).
 * TEST INFRASTRUCTURE ONLY (see jdob_oracle.h).
 *
 * Sec. II gives every user m its own cycles-per-work ratio zeta_m (Eq. (1)),
 * switched capacitance kappa_m (Eq. (2)), transmit power p_m (Eq. (4)) and
 * CPU frequency range; the layer work is shared (the same DNN).  Here
 * C[s] = sum of the layer work of layers 1..s (v_s = u_s, g = q = 1):
 *   t_m[s][k] = (zeta_m * C[s]) / f_m[k]            Eq. (1)
 *   e_m[s][k] = (kappa_m * (f_m[k] * f_m[k])) * C[s]  Eq. (2)
 *   up_m[s]   = bits[s] / rate[m]                  Eq. (3), energy p_m * up
 *   gamma_m(s) = up_m[s] + t_m[s][K-1]              Eq. (17)
 * Alg. 1 sorts the users by gamma at every partition point, so the order,
 * the batch deadlines (Eq. (10)) and bmin depend on s.  The offloading sets
 * are the tails of the gamma-descending list, i.e. the first b users of the
 * gamma-ascending order pi_s (ties: lower index first).  Everything else is
 * the homogeneous oracle's: constraints (6)-(8), each offloader's lowest
 * level meeting its budget (Eq. (20)), the energy of Eq. (21) summed over
 * users in index order, the first strict minimum in the order s ascending,
 * j descending, b descending, local computing last, and Eq. (22).
 * With JO_MODE_GREEDY the batch of (s, j) is the largest b whose users all
 * meet (7) at their top CPU frequency (Alg. 2's greedy set: in exact
 * arithmetic that is the test of its head, the largest gamma); with
 * JO_MODE_CONTINUOUS user m's frequency is continuous in
 * [f_m[0], f_m[K-1]].
 */

typedef struct {
  int N, L, K, J;
  REAL *C, *A, *B, *r, *Pw; /* shared, as in prepare()                      */
  REAL *f;                  /* [N*K] CPU levels of user m                    */
  REAL *kap, *zet, *ptx;    /* [N] kappa_m, zeta_m, p_m                       */
  REAL *t, *e;              /* [(N*(L+1))*K] Eqs. (1), (2) of user m at s, k  */
  REAL *up;                 /* [N*(L+1)] Eq. (3) of user m at s               */
  int *kL;                  /* [N] local-only level of user m, -1 if none     */
  REAL *eL, *fL;            /* [N] its energy and frequency                   */
  /* the current partition point (h_order) */
  int *pi, *rank;           /* [N] users by gamma ascending; position of m    */
  REAL *lo;                 /* [N+1] tightest deadline among pi[0..b-1]       */
  int bmin;
  /* the current candidate (h_candidate), by position in pi */
  int *lv;
  REAL *fz;
  int cont;
  REAL tfree;
} JO_CAT(jo_hscratch, SFX);
#define HSCRATCH JO_CAT(jo_hscratch, SFX)

static int FN(is_hetero)(const PROB *p) {
  return p->user_zeta || p->user_kappa || p->user_p_tx || p->user_local_freq;
}

static void FN(h_free)(HSCRATCH *w) {
  free(w->C); free(w->A); free(w->B); free(w->r); free(w->Pw); free(w->f); free(w->kap);
  free(w->zet); free(w->ptx); free(w->t); free(w->e); free(w->up); free(w->kL); free(w->eL);
  free(w->fL); free(w->pi); free(w->rank); free(w->lo); free(w->lv); free(w->fz);
}

static int FN(h_alloc)(HSCRATCH *w, int N, int L, int K, int J) {
  memset(w, 0, sizeof(*w));
  w->N = N; w->L = L; w->K = K; w->J = J;
  const size_t nt = (size_t)N * (L + 1) * K;
  w->C = (REAL *)malloc(sizeof(REAL) * (L + 1));
  w->A = (REAL *)malloc(sizeof(REAL) * (L + 1));
  w->B = (REAL *)malloc(sizeof(REAL) * (L + 1));
  w->r = (REAL *)malloc(sizeof(REAL) * J);
  w->Pw = (REAL *)malloc(sizeof(REAL) * J);
  w->f = (REAL *)malloc(sizeof(REAL) * N * K);
  w->kap = (REAL *)malloc(sizeof(REAL) * N);
  w->zet = (REAL *)malloc(sizeof(REAL) * N);
  w->ptx = (REAL *)malloc(sizeof(REAL) * N);
  w->t = (REAL *)malloc(sizeof(REAL) * nt);
  w->e = (REAL *)malloc(sizeof(REAL) * nt);
  w->up = (REAL *)malloc(sizeof(REAL) * N * (L + 1));
  w->kL = (int *)malloc(sizeof(int) * N);
  w->eL = (REAL *)malloc(sizeof(REAL) * N);
  w->fL = (REAL *)malloc(sizeof(REAL) * N);
  w->pi = (int *)malloc(sizeof(int) * N);
  w->rank = (int *)malloc(sizeof(int) * N);
  w->lo = (REAL *)malloc(sizeof(REAL) * (N + 1));
  w->lv = (int *)malloc(sizeof(int) * N);
  w->fz = (REAL *)malloc(sizeof(REAL) * N);
  if (!w->C || !w->A || !w->B || !w->r || !w->Pw || !w->f || !w->kap || !w->zet || !w->ptx ||
      !w->t || !w->e || !w->up || !w->kL || !w->eL || !w->fL || !w->pi || !w->rank || !w->lo ||
      !w->lv || !w->fz) {
    FN(h_free)(w);
    return -1;
  }
  return 0;
}

#define HT(w, m, s, k) ((w)->t[((size_t)(m) * ((w)->L + 1) + (s)) * (w)->K + (k)])
#define HE(w, m, s, k) ((w)->e[((size_t)(m) * ((w)->L + 1) + (s)) * (w)->K + (k)])
#define HU(w, m, s) ((w)->up[(size_t)(m) * ((w)->L + 1) + (s)])

/* Eq. (20) with a continuous frequency for user m: the slowest frequency
 * finishing work W within the budget, clamped to the user's range (its
 * lowest frequency if W = 0). */
static REAL FN(h_cont_freq)(const HSCRATCH *w, int m, REAL W, REAL budget) {
  const REAL lo = w->f[m * w->K], hi = w->f[m * w->K + w->K - 1];
  if (W == 0) return lo;
  REAL g = W / budget;
  return g < lo ? lo : (g > hi ? hi : g);
}

/* Per-instance quantities: the shared sums (as prepare()), each user's
 * parameters and option tables, its local-only choice (8) with Eq. (20). */
static void FN(h_prepare)(const PROB *p, int64_t inst, HSCRATCH *w) {
  const int N = p->N, L = p->L, K = p->K, J = p->J;
  const REAL *cyc = p->cycles + (size_t)inst * L;
  const REAL *bits = p->bits + (size_t)inst * (L + 1);
  const REAL *al = p->alpha + (size_t)inst * L;
  const REAL *be = p->beta + (size_t)inst * L;
  const REAL *rate = p->rate + (size_t)inst * N;
  const REAL *T = p->deadline + (size_t)inst * N;
  const REAL *g = p->gpu_freq;
  const REAL gc = (REAL)p->gpu_c, p0 = (REAL)p->gpu_p_static;

  w->N = N; w->L = L; w->K = K; w->J = J;
  w->tfree = p->t_free ? p->t_free[inst] : (REAL)0;
  w->cont = (p->mode & JO_MODE_CONTINUOUS) != 0;
  /* layer work of layers 1..s and the GPU sums of layers s+1..L */
  w->C[0] = 0;
  for (int s = 0; s < L; ++s) w->C[s + 1] = w->C[s] + cyc[s];
  w->A[L] = 0;
  w->B[L] = 0;
  for (int s = L - 1; s >= 0; --s) {
    w->A[s] = w->A[s + 1] + al[s];
    w->B[s] = w->B[s + 1] + be[s];
  }
  for (int j = 0; j < J; ++j) {  /* Eq. (5): stretch and power at level j */
    w->r[j] = g[J - 1] / g[j];
    w->Pw[j] = gc * ((g[j] * g[j]) * g[j]) + p0;
  }
  for (int m = 0; m < N; ++m) {
    const size_t o = (size_t)inst * N + m;
    w->kap[m] = p->user_kappa ? p->user_kappa[o] : (REAL)p->kappa;
    w->zet[m] = p->user_zeta ? p->user_zeta[o] : (REAL)1;
    w->ptx[m] = p->user_p_tx ? p->user_p_tx[o] : (REAL)p->p_tx;
    for (int k = 0; k < K; ++k)
      w->f[m * K + k] = p->user_local_freq ? p->user_local_freq[o * K + k] : p->local_freq[k];
    for (int s = 0; s <= L; ++s) {
      const REAL W = w->zet[m] * w->C[s];
      for (int k = 0; k < K; ++k) {
        const REAL fk = w->f[m * K + k];
        HT(w, m, s, k) = W / fk;                              /* Eq. (1) */
        HE(w, m, s, k) = (w->kap[m] * (fk * fk)) * w->C[s];   /* Eq. (2) */
      }
      HU(w, m, s) = (s < L) ? bits[s] / rate[m] : (REAL)0;    /* Eq. (3) */
    }
    /* (8): the lowest level finishing every layer by the deadline */
    int kL = -1;
    for (int k = 0; k < K; ++k)
      if (HT(w, m, L, k) <= T[m]) { kL = k; break; }
    w->kL[m] = kL;
    if (kL < 0) {
      w->fL[m] = 0;
      w->eL[m] = (REAL)INFINITY;
    } else if (w->cont) {
      w->fL[m] = FN(h_cont_freq)(w, m, w->zet[m] * w->C[L], T[m]);
      w->eL[m] = (w->kap[m] * (w->fL[m] * w->fL[m])) * w->C[L];
    } else {
      w->fL[m] = w->f[m * K + kL];
      w->eL[m] = HE(w, m, L, kL);
    }
  }
}

/* Alg. 1 at partition point s: the users by gamma (Eq. (17)) ascending,
 * ties by lower index; the batch deadlines of Eq. (10) along that order;
 * bmin = one past the last position holding a user without a local level. */
static void FN(h_order)(const PROB *p, int64_t inst, HSCRATCH *w, int s) {
  const int N = w->N, K = w->K;
  const REAL *T = p->deadline + (size_t)inst * N;
  for (int m = 0; m < N; ++m) w->pi[m] = m;
  for (int a = 1; a < N; ++a) { /* insertion sort */
    const int x = w->pi[a];
    const REAL gx = HU(w, x, s) + HT(w, x, s, K - 1);
    int c = a - 1;
    while (c >= 0) {
      const int y = w->pi[c];
      const REAL gy = HU(w, y, s) + HT(w, y, s, K - 1);
      if (gy > gx || (gy == gx && y > x)) {
        w->pi[c + 1] = y;
        --c;
      } else {
        break;
      }
    }
    w->pi[c + 1] = x;
  }
  for (int i = 0; i < N; ++i) w->rank[w->pi[i]] = i;
  w->lo[0] = (REAL)INFINITY;
  for (int b = 1; b <= N; ++b) {
    const REAL d = T[w->pi[b - 1]];
    w->lo[b] = (d < w->lo[b - 1]) ? d : w->lo[b - 1];
  }
  w->bmin = 0;
  for (int i = 0; i < N; ++i)
    if (w->kL[w->pi[i]] < 0) w->bmin = i + 1;
}

/* Candidate (s, j, b) at the order of h_order(s): constraints (6)-(8), each
 * offloader's lowest level (or continuous frequency) meeting its budget,
 * the energy of Eq. (21) over users in index order plus the GPU's. */
static int FN(h_candidate)(HSCRATCH *w, int s, int j, int b, REAL *energy, REAL *gpu_latency) {
  const int N = w->N, K = w->K;
  const REAL Phi = (w->A[s] + w->B[s] * (REAL)b) * w->r[j];
  const REAL H = w->lo[b] - Phi;
  for (int i = b; i < N; ++i)
    if (w->kL[w->pi[i]] < 0) return 0; /* (8) */
  if (!(H >= w->tfree)) return 0;       /* (6) */
  for (int i = 0; i < b; ++i) {          /* (7) with Eq. (20) */
    const int m = w->pi[i];
    const REAL budget = H - HU(w, m, s);
    int k = -1;
    for (int q = 0; q < K; ++q)
      if (HT(w, m, s, q) <= budget) { k = q; break; }
    if (k < 0) return 0;
    w->lv[i] = k;
    if (w->cont) w->fz[i] = FN(h_cont_freq)(w, m, w->zet[m] * w->C[s], budget);
  }
  REAL acc = 0;
  for (int m = 0; m < N; ++m) {
    const int i = w->rank[m];
    if (i < b) {
      const REAL e = w->cont ? (w->kap[m] * (w->fz[i] * w->fz[i])) * w->C[s]
                             : HE(w, m, s, w->lv[i]);
      acc = acc + (e + w->ptx[m] * HU(w, m, s));
    } else {
      acc = acc + w->eL[m];
    }
  }
  acc = acc + w->Pw[j] * Phi;
  *energy = acc;
  *gpu_latency = Phi;
  return 1;
}

/* Alg. 2's test for the set pi[0..b-1] at level j: every member meets (7)
 * at its top CPU frequency. */
static int FN(h_all_meet_top)(const HSCRATCH *w, int s, int j, int b) {
  const int K = w->K;
  const REAL H = w->lo[b] - (w->A[s] + w->B[s] * (REAL)b) * w->r[j];
  for (int i = 0; i < b; ++i) {
    const int m = w->pi[i];
    if (!(HT(w, m, s, K - 1) <= H - HU(w, m, s))) return 0;
  }
  return 1;
}

static int FN(h_local)(const HSCRATCH *w, REAL *energy) {
  for (int m = 0; m < w->N; ++m)
    if (w->kL[m] < 0) return 0;
  REAL acc = 0;
  for (int m = 0; m < w->N; ++m) acc = acc + w->eL[m];
  *energy = acc;
  return 1;
}

/* Eq. (22) of the candidate just filled by h_candidate. */
static REAL FN(h_release)(const HSCRATCH *w, int s, int b, REAL Phi) {
  REAL ready = w->tfree;
  for (int i = 0; i < b; ++i) {
    const int m = w->pi[i];
    const REAL tl = w->cont ? (w->zet[m] * w->C[s]) / w->fz[i] : HT(w, m, s, w->lv[i]);
    const REAL done = tl + HU(w, m, s);
    if (done > ready) ready = done;
  }
  return ready + Phi;
}

/* Level (-1 with a continuous frequency) and frequency of user m for the
 * candidate (s, b) just filled by h_candidate (s == L: local computing). */
static void FN(h_user_choice)(const HSCRATCH *w, int s, int b, int m, int8_t *lv, REAL *fq) {
  const int i = w->rank[m];
  if (s < w->L && i < b) {
    *lv = (int8_t)(w->cont ? -1 : w->lv[i]);
    *fq = w->cont ? w->fz[i] : w->f[m * w->K + w->lv[i]];
  } else {
    *lv = (int8_t)(w->cont ? -1 : w->kL[m]);
    *fq = w->fL[m];
  }
}

static JO_CAT(jo_best, SFX) FN(h_solve_instance)(const PROB *p, int64_t inst, HSCRATCH *w) {
  const int N = p->N, L = p->L, J = p->J;
  const int s_end = (p->mode & JO_MODE_BINARY) ? 1 : L;
  const int j_low = (p->mode & JO_MODE_FIXED_EDGE) ? J - 1 : 0;
  const int greedy = (p->mode & JO_MODE_GREEDY) != 0;
  FN(h_prepare)(p, inst, w);
  JO_CAT(jo_best, SFX) r = {0, -1, -1, 0, (REAL)INFINITY, (REAL)INFINITY, 0, 0, (REAL)INFINITY};
  for (int s = 0; s < s_end; ++s) {
    FN(h_order)(p, inst, w, s);
    if (greedy) { /* Alg. 2: the set shrinks as f_e is swept downward */
      int b = N;
      for (int j = J - 1; j >= j_low; --j) {
        while (b >= 1 && !FN(h_all_meet_top)(w, s, j, b)) --b;
        if (b == 0) break;
        REAL E, Phi;
        if (FN(h_candidate)(w, s, j, b, &E, &Phi)) FN(consider)(&r, E, s, j, b);
      }
    } else {
      for (int j = J - 1; j >= j_low; --j)
        for (int b = N; b >= 1; --b) {
          REAL E, Phi;
          if (FN(h_candidate)(w, s, j, b, &E, &Phi)) FN(consider)(&r, E, s, j, b);
        }
    }
  }
  {
    REAL E;
    if (FN(h_local)(w, &E)) FN(consider)(&r, E, L, -1, 0);
  }
  if (r.found && r.s == L) {
    r.tfree_out = w->tfree;
  } else if (r.found) {
    REAL E, Phi;
    FN(h_order)(p, inst, w, r.s);
    FN(h_candidate)(w, r.s, r.j, r.b, &E, &Phi); /* refill the winner's levels */
    r.tfree_out = FN(h_release)(w, r.s, r.b, Phi);
  }
  return r;
}

/* jo_solve for heterogeneous users (same outputs). */
static int FN(h_solve)(const PROB *p, int64_t start, int64_t count, POLICY *out) {
  const int N = p->N;
  HSCRATCH w;
  if (FN(h_alloc)(&w, N, p->L, p->K, p->J) != 0) return -2;
  for (int64_t inst = start; inst < start + count; ++inst) {
    JO_CAT(jo_best, SFX) r = FN(h_solve_instance)(p, inst, &w);
    int8_t *ul = out->user_level + (size_t)inst * N;
    int8_t *uo = out->user_offload + (size_t)inst * N;
    REAL *uf = out->user_freq ? out->user_freq + (size_t)inst * N : NULL;
    if (out->num_feasible) out->num_feasible[inst] = r.nfeas;
    if (out->num_user_evals) out->num_user_evals[inst] = r.nevals;
    if (out->energy_second) out->energy_second[inst] = r.second;
    if (!r.found) {
      out->status[inst] = 1;
      out->cut[inst] = -1;
      out->gpu_level[inst] = -1;
      out->batch[inst] = 0;
      out->energy[inst] = (REAL)INFINITY;
      out->t_free_out[inst] = (REAL)INFINITY;
      for (int m = 0; m < N; ++m) {
        ul[m] = -1;
        uo[m] = 0;
        if (uf) uf[m] = 0;
      }
      continue;
    }
    out->status[inst] = 0;
    out->cut[inst] = r.s;
    out->gpu_level[inst] = r.j;
    out->batch[inst] = r.b;
    out->energy[inst] = r.best;
    out->t_free_out[inst] = r.tfree_out;
    for (int m = 0; m < N; ++m) {
      REAL fq;
      uo[m] = (int8_t)(r.s < p->L && w.rank[m] < r.b);
      FN(h_user_choice)(&w, r.s, r.b, m, &ul[m], &fq);
      if (uf) uf[m] = fq;
    }
  }
  FN(h_free)(&w);
  return 0;
}

/* jo_eval_candidate for heterogeneous users. */
static int FN(h_eval_candidate)(const PROB *p, int64_t inst, int s, int j, int b, CAND *res) {
  const int N = p->N, L = p->L;
  HSCRATCH w;
  if (FN(h_alloc)(&w, N, L, p->K, p->J) != 0) return -2;
  FN(h_prepare)(p, inst, &w);
  REAL E = (REAL)INFINITY, Phi = 0;
  if (s == L) {
    FN(h_order)(p, inst, &w, 0);  /* ranks are not used for local computing */
    res->feasible = FN(h_local)(&w, &E);
    res->t_free_out = res->feasible ? w.tfree : (REAL)INFINITY;
    res->gpu_latency = 0;
  } else {
    FN(h_order)(p, inst, &w, s);
    res->feasible = FN(h_candidate)(&w, s, j, b, &E, &Phi);
    res->t_free_out = res->feasible ? FN(h_release)(&w, s, b, Phi) : (REAL)INFINITY;
    res->gpu_latency = (w.A[s] + w.B[s] * (REAL)b) * w.r[j];
  }
  res->energy = res->feasible ? E : (REAL)INFINITY;
  for (int m = 0; m < N; ++m) {
    const int off = s < L && w.rank[m] < b;
    int8_t lv = -1;
    REAL fq = 0;
    if (res->feasible) FN(h_user_choice)(&w, s, b, m, &lv, &fq);
    if (res->user_level) res->user_level[m] = lv;
    if (res->user_offload) res->user_offload[m] = (int8_t)off;
    if (res->user_freq) res->user_freq[m] = fq;
  }
  FN(h_free)(&w);
  return 0;
}

#undef HT
#undef HE
#undef HU
#undef HSCRATCH
