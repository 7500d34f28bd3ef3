/*
 * jdob_oracle.h — plain single-threaded CPU oracle for batched J-DOB.
 *
 * TEST INFRASTRUCTURE ONLY.  This oracle exists to check the GPU library; it
 * is used by the tests, by the smoke check and by the benchmark's CPU
 * baseline, never by the product path.  It shares no code, header or
 * constant with the GPU library.
 *
 * What it computes (Sec. III, problem (P1) restricted to identical offloading
 * and one greedy batch, with the offload sets Alg. 1/2 use):  for every
 * instance, every candidate (s, j, b) -- partition point s in [0, L), GPU
 * frequency level j, the b users with the highest uplink rate offloading --
 * plus local computing, is tested against the deadline constraints
 * (6) GPU free in time, (7) co-inference latency of every offloader,
 * (8) local latency of every local user; each user's CPU level is the lowest
 * level meeting its budget, Eq. (20) on a discrete grid; the energy is
 * Eq. (21); the first strict minimum in the order s ascending, j descending,
 * b descending, local computing last, is returned with Eq. (22).
 * With JO_MODE_GREEDY the batch of each (s, j) is the one Alg. 2 keeps at
 * that frequency instead (the largest suffix meeting its threshold of
 * Eq. (18), found by sweeping f_e downward); JO_MODE_FIXED_EDGE keeps only the
 * top GPU level and JO_MODE_BINARY only s = 0.  With JO_MODE_CONTINUOUS a
 * user's CPU frequency is continuous in [local_freq[0], local_freq[K-1]]:
 * Eq. (20), f = min(max(C / budget, f_min), f_max), energy (kappa f^2) C;
 * feasibility is the same test as with levels (the top frequency fits the
 * budget); user_level is then -1 and user_freq holds the frequency.
 * Arithmetic: working precision REAL, operations in the written order, no
 * contraction (build with -ffp-contract=off).
 *
 * With per-user parameters (zeta_m, kappa_m, p_m, CPU levels: the
 * heterogeneous users of Sec. II) the users are ordered by gamma at every
 * partition point; jdob_oracle_hetero.h has the details.  The grouping
 * solves each group with its members' own parameters; the option tables
 * take homogeneous users only.
 *
 * Brute force (jdob_brute.c): every subset of offloaders x every CPU level
 * vector x every (s, j), in long double, straight from the model
 * definitions of Sec. II, for tiny instances.
 */
#ifndef JDOB_ORACLE_H
#define JDOB_ORACLE_H

#include <stdint.h>

#define JO_PROBLEM_FIELDS(REAL)                                              \
  int32_t I, N, L, K, J;                                                     \
  const REAL *cycles;     /* [I][L]   layer cycles                       */  \
  const REAL *bits;       /* [I][L+1] O_0..O_L                            */  \
  const REAL *alpha;      /* [I][L]   GPU latency at top freq, batch part 0 */ \
  const REAL *beta;       /* [I][L]   GPU latency per sample at top freq  */  \
  const REAL *rate;       /* [I][N]                                       */  \
  const REAL *deadline;   /* [I][N]                                       */  \
  const REAL *t_free;     /* [I] or NULL                                  */  \
  const REAL *local_freq; /* [K]                                          */  \
  const REAL *gpu_freq;   /* [J]                                          */  \
  double kappa, p_tx, gpu_c, gpu_p_static;                                   \
  int32_t mode;           /* JO_MODE_* bits, 0 = every suffix length     */  \
  /* heterogeneous users (jdob_oracle_hetero.h); NULL = the shared value */  \
  const REAL *user_zeta;  /* [I][N] cycles per unit of layer work (1)    */  \
  const REAL *user_kappa; /* [I][N] switched capacitance (kappa)         */  \
  const REAL *user_p_tx;  /* [I][N] transmit power (p_tx)                */  \
  const REAL *user_local_freq; /* [I][N][K] CPU levels (local_freq)      */

/* Search variants (Sec. III, and the ablations J-DOB w/o edge DVFS and
 * J-DOB binary of Sec. IV); any combination of the bits is valid. */
#define JO_MODE_GREEDY 1     /* Alg. 2: at each f_e only the greedy batching set */
#define JO_MODE_FIXED_EDGE 2 /* f_e fixed at f_e,max (the top GPU level)         */
#define JO_MODE_BINARY 4     /* partition point 0 (whole task) or local only     */
#define JO_MODE_CONTINUOUS 8 /* CPU frequency continuous in [f_0, f_{K-1}]: Eq.  \
                                (20) with its clamp instead of the lowest level */

#define JO_POLICY_FIELDS(REAL)                                               \
  int32_t *status, *cut, *gpu_level, *batch;                                 \
  REAL *energy, *t_free_out;                                                 \
  int8_t *user_level, *user_offload;                                         \
  REAL *energy_second;     /* [I] second-lowest feasible energy, or NULL  */ \
  int32_t *num_feasible;   /* [I] or NULL                                 */ \
  int64_t *num_user_evals; /* [I] or NULL                                 */ \
  REAL *user_freq;         /* [I][N] chosen CPU frequency, or NULL        */

#define JO_TABLE_FIELDS(REAL)                                                \
  int16_t *order;                                                            \
  REAL *batch_deadline;                                                      \
  int32_t *min_batch;                                                        \
  REAL *uplink_time, *gamma;                                                 \
  int8_t *self_level;                                                        \
  REAL *self_energy, *self_slack;

/* Outer grouping: users by deadline, consecutive groups served one after
 * another by the GPU, each group one inner solve (see jo_solve_grouped). */
#define JO_GROUPED_FIELDS(REAL)                                              \
  int32_t *status;         /* [I] 0 = every group feasible, 1 = none found */ \
  int32_t *num_groups;     /* [I] G                                        */ \
  REAL *energy;            /* [I] sum of the group energies, in order      */ \
  REAL *t_free_out;        /* [I] GPU release time after the last group    */ \
  int16_t *order;          /* [I][N] users by deadline ascending, ties by   \
                              lower index: the order groups are cut from  */ \
  int16_t *group_end;      /* [I][N] group g is order[end(g-1) .. end(g)-1] */ \
  int32_t *group_cut, *group_gpu_level, *group_batch; /* [I][N] per group  */ \
  REAL *group_energy, *group_t_free;                  /* [I][N] per group  */ \
  int8_t *user_level, *user_offload, *user_group;     /* [I][N] per user   */ \
  int64_t *num_inner;      /* [I] inner solves the DP ran, or NULL         */ \
  int64_t *num_feasible;   /* [I] their feasible candidates, or NULL       */ \
  int64_t *num_user_evals; /* [I] their sums of b, or NULL                 */ \
  REAL *user_freq;         /* [I][N] chosen CPU frequency, or NULL         */

/* A grouped policy to evaluate: G groups in deadline order with the
 * candidate each group uses (cut = L for local computing). */
#define JO_GROUPING_FIELDS(REAL)                                             \
  int32_t num_groups;                                                        \
  const int16_t *group_end;                                                  \
  const int32_t *group_cut, *group_gpu_level, *group_batch;                  \
  int32_t feasible;        /* out */                                          \
  REAL energy, t_free_out; /* out */                                          \
  int8_t *user_level, *user_offload; /* out, [N] */                           \
  REAL *user_freq;         /* out, [N], or NULL */

#define JO_CANDIDATE_FIELDS(REAL)                                            \
  int32_t feasible;                                                          \
  REAL energy, t_free_out, gpu_latency;                                      \
  int8_t *user_level;   /* [N] */                                            \
  int8_t *user_offload; /* [N] */                                            \
  REAL *user_freq;      /* [N] or NULL */

typedef struct { JO_PROBLEM_FIELDS(float) } jo_problem_f32;
typedef struct { JO_PROBLEM_FIELDS(double) } jo_problem_f64;
typedef struct { JO_POLICY_FIELDS(float) } jo_policy_f32;
typedef struct { JO_POLICY_FIELDS(double) } jo_policy_f64;
typedef struct { JO_TABLE_FIELDS(float) } jo_tables_f32;
typedef struct { JO_TABLE_FIELDS(double) } jo_tables_f64;
typedef struct { JO_GROUPED_FIELDS(float) } jo_grouped_f32;
typedef struct { JO_GROUPED_FIELDS(double) } jo_grouped_f64;
typedef struct { JO_GROUPING_FIELDS(float) } jo_grouping_f32;
typedef struct { JO_GROUPING_FIELDS(double) } jo_grouping_f64;
typedef struct { JO_CANDIDATE_FIELDS(float) } jo_candidate_f32;
typedef struct { JO_CANDIDATE_FIELDS(double) } jo_candidate_f64;

typedef struct {
  int32_t found;           /* 1 if any policy is feasible                 */
  double energy;           /* minimum energy                              */
  double energy_second;    /* min energy over the other (s, j, set) choices */
  int32_t cut, gpu_level, batch;
  int32_t num_feasible;    /* (s, j, set) choices with a feasible level
                              vector, plus local computing if feasible    */
  int8_t *user_level;      /* [N] one optimal level vector               */
  int8_t *user_offload;    /* [N]                                         */
} jo_brute_result;

#ifdef __cplusplus
extern "C" {
#endif

/* Solve instances [start, start+count); outputs are indexed by instance. */
int jo_solve_f32(const jo_problem_f32 *p, int64_t start, int64_t count, jo_policy_f32 *out);
int jo_solve_f64(const jo_problem_f64 *p, int64_t start, int64_t count, jo_policy_f64 *out);

/* Per-user option tables of instances [start, start+count). */
int jo_user_tables_f32(const jo_problem_f32 *p, int64_t start, int64_t count, jo_tables_f32 *out);
int jo_user_tables_f64(const jo_problem_f64 *p, int64_t start, int64_t count, jo_tables_f64 *out);

/* One candidate of one instance: s in [0, L) with j, b; s == L is local computing. */
int jo_eval_candidate_f32(const jo_problem_f32 *p, int64_t inst, int s, int j, int b, jo_candidate_f32 *res);
int jo_eval_candidate_f64(const jo_problem_f64 *p, int64_t inst, int s, int j, int b, jo_candidate_f64 *res);

/* Outer grouping of instances [start, start+count): users sorted by deadline
 * (ties by index) are cut into consecutive groups; the groups are served in
 * that order, each by one inner solve of the problem's mode whose GPU free
 * time is the previous group's release time (Eq. (22)).  The grouping is a
 * dynamic program over prefixes of the deadline order that keeps, for each
 * prefix i, a front of states (total energy, release time) none of which is
 * dominated by another (a state dominates one with no lower energy and no
 * earlier release; of two equal states the first generated stays): the
 * front of i collects, in the order j = 0..i-1 and then the states of the
 * front of j from the earliest release to the latest, the state of j
 * extended by one inner solve of order[j..i-1] with the GPU free at that
 * state's release time.  A later free time only removes candidates
 * (constraint (6)), so a winner that meets a later state's free time is
 * that state's winner too: num_inner counts only the inner solves this
 * leaves (one per run of states sharing a winner).  Fronts are kept sorted
 * by energy and hold at most JO_FRONT states (the highest energy leaves).
 * The answer is the lowest-energy state of the front of N. */
#ifndef JO_FRONT
#define JO_FRONT 16
#endif
int jo_solve_grouped_f32(const jo_problem_f32 *p, int64_t start, int64_t count, jo_grouped_f32 *out);
int jo_solve_grouped_f64(const jo_problem_f64 *p, int64_t start, int64_t count, jo_grouped_f64 *out);

/* Evaluate a given grouped policy of one instance: each group's candidate
 * on its sub-problem with the release time chained from group to group. */
int jo_eval_grouping_f32(const jo_problem_f32 *p, int64_t inst, jo_grouping_f32 *g);
int jo_eval_grouping_f64(const jo_problem_f64 *p, int64_t inst, jo_grouping_f64 *g);

/* Brute force over all offload subsets (suffix_only = 0) or over the
 * gamma-ordered suffixes only (suffix_only = 1), all CPU level vectors and
 * all (s, j).  Tiny instances only: cost grows as 2^N * K^N * L * J. */
int jo_brute_f64(const jo_problem_f64 *p, int64_t inst, int suffix_only, jo_brute_result *res);

#ifdef __cplusplus
}
#endif

#endif /* JDOB_ORACLE_H */
