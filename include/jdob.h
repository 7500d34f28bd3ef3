/*
 * jdob.h — C ABI of the batched J-DOB policy evaluator for MI355X (gfx950).
 *
 * J-DOB (joint DVFS, offloading and batching for multiuser edge-device
 * co-inference) picks, for one group of users sharing a DNN that is a chain
 * of L sub-tasks, an identical partition point s, the set of users that
 * offload after sub-task s, every user's CPU frequency and the edge GPU
 * frequency, so that the total device + edge energy is minimal while every
 * hard deadline holds (Sec. III, problem (P1) with constraints (6)-(15)).
 * This library evaluates that problem for many independent instances at
 * once on one GPU.
 *
 * Notation.  The library names users m = 0..N-1 and sub-tasks ("layers")
 * l = 1..L; the paper calls them M users and N sub-tasks.  Partition point
 * s in {0..L}: the user computes layers 1..s locally, uploads O_s bits and
 * the GPU runs layers s+1..L for the whole batch; s = L is local computing.
 *
 * The candidate family ("J-DOB grid").  Sec. III restricts (P1) to one
 * common partition point and one greedy batch, and Alg. 1/2 only ever offload
 * the users with the smallest minimum latency cost gamma (Eq. (17)), i.e. a
 * suffix of the gamma-descending list.  With per-instance shared cycles the
 * gamma order is the order of decreasing uplink rate, for every s.  Let pi be
 * the users sorted by rate descending (ties: lower user index first).  A
 * candidate is (s, j, b) with s in [0, L), GPU level j in [0, J) and batch
 * b in [1, N]: users pi[0..b-1] offload at s, the rest compute locally; plus
 * the local-computing candidate (LC).  The CPU and GPU frequencies are the
 * discrete level grids local_freq[K] and gpu_freq[J] (the paper sweeps the GPU
 * frequency with step rho, Alg. 2, which is such a grid).  The solver returns
 * the exact minimum-energy feasible candidate of this family; Alg. 2 keeps
 * only the largest feasible batch at each GPU frequency, the grid keeps all.
 *
 * Arithmetic contract.  Every quantity that decides feasibility or a level is
 * computed in the working precision P (binary32 for JDOB_F32, binary64 for
 * JDOB_F64) with IEEE round-to-nearest-even, no fused multiply-add
 * contraction and no reassociation, in exactly this order:
 *   C[0] = 0,  C[s] = C[s-1] + cyc[s-1]                (s = 1..L, sequential)
 *   A[L] = B[L] = 0, A[s] = A[s+1] + alpha[s], B[s] = B[s+1] + beta[s]
 *                                                      (s = L-1..0, sequential)
 *   t[s][k] = C[s] / f_k                  local latency, Eq. (1) with zeta*g = 1
 *   e[s][k] = (kappa * (f_k * f_k)) * C[s]  local energy, Eq. (2) with q = 1
 *   up[i][s] = bits[s] / rate[pi_i]       upload latency, Eq. (3)
 *   r_j = g_{J-1} / g_j,  P_j = (gpu_c * ((g_j * g_j) * g_j)) + P0
 *   Phi(s,j,b) = (A[s] + B[s] * b) * r_j  batch latency of layers s+1..L, Eq. (5)
 *   lo[b] = min(T[pi_0], .., T[pi_{b-1}])  batch deadline, Eq. (10)
 *   H = lo[b] - Phi
 *   kL[m] = min{k : t[L][k] <= T_m}        local-only level, (8) and (20)
 *   bmin = 1 + max{i : user pi_i has no local level}, or 0
 *   feasible(s,j,b) <=> b >= bmin  and  H >= t_free                 (6), (8)
 *                      and  t[s][K-1] <= H - up[b-1][s]             (7)
 *   k_i = min{k : t[s][k] <= H - up[i][s]}   (i < b)       Eq. (20), discrete
 *   E   = sum_{i<b} (e[s][k_i] + p_tx*up[i][s]) + sum_{i>=b} e[L][kL[pi_i]]
 *         + P_j * Phi                                      Eq. (21)
 *   E_LC = sum_m e[L][kL[m]], feasible <=> bmin == 0
 * Search modes (jdob_problem.mode, any OR of the bits; 0 = the grid):
 *   JDOB_MODE_GREEDY      Alg. 2 literally: at each (s, j) only the greedy
 *       batching set is a candidate, b = bg(s, j) = the largest b in [1, N]
 *       with  t[s][K-1] <= H - up[b-1][s]  ((7) for the head of the
 *       gamma-descending list, i.e. g_j at or above its threshold, Eq.
 *       (18)); it is feasible if also b >= bmin and H >= t_free.  bg does
 *       not increase as j decreases, which is the sweep of Alg. 2 from
 *       f_e,max downward; an (s, j) with no such b has no candidate (the
 *       empty set of Alg. 2 is local computing, which always competes).
 *   JDOB_MODE_FIXED_EDGE_FREQ  the ablation without edge DVFS (Sec. IV):
 *       only j = J-1 (f_e = f_e,max).
 *   JDOB_MODE_BINARY      the ablation with binary offloading (Sec. IV):
 *       only s = 0 (whole task offloaded) besides local computing.
 *   JDOB_MODE_CONTINUOUS_CPU  the CPU frequency of every user is continuous
 *       in [local_freq[0], local_freq[K-1]] (the levels in between are not
 *       used): Eq. (20) with its clamp, f = C[s] / budget raised to f_0 and
 *       capped at f_{K-1} (f_0 if C[s] = 0), energy (kappa * (f * f)) * C[s],
 *       local latency C[s] / f in Eq. (22).  Feasibility is decided by the
 *       same tests as with levels; user_level is then -1 and user_freq holds
 *       the frequency.
 * Heterogeneous users (Sec. II: each device m has its own zeta_m, kappa_m,
 * p_m and CPU levels f_m[k]; jdob_problem.user_*): layer_cycles is then the
 * layer work (v = u of Sec. III with g = q = 1) and
 *   t_m[s][k] = (zeta_m * C[s]) / f_m[k],  e_m[s][k] = (kappa_m * (f_m[k] *
 *   f_m[k])) * C[s],  upload energy p_m * up,  gamma_m(s) = up_m[s] +
 *   t_m[s][K-1]  (Eq. (17)).
 * Alg. 1 sorts users by gamma at every s: pi_s = users by gamma ascending
 * (ties: lower index), and lo[b], bmin and the candidates (s, j, b) use
 * pi_s.  Feasibility as above with each offloader's own test
 * t_m[s][K-1] <= H - up_m[s] (7).  The greedy batch bg(s, j) is the largest
 * b whose users all meet (7) at their top level (in exact arithmetic the test
 * of the head of Alg. 2's list).  With JDOB_MODE_CONTINUOUS_CPU user m's
 * frequency is continuous in [f_m[0], f_m[K-1]].  Energies are summed in
 * user index order as above.  jdob_solve_batch and jdob_solve_grouped (each
 * group with its members' own parameters) take heterogeneous users for
 * N <= JDOB_MAX_HETERO_USERS; the two-stage calls return
 * JDOB_ERR_UNSUPPORTED.
 * The winner is the lowest-energy feasible candidate; equal energies go to
 * the lowest flat index ((s*J + (J-1-j))*N + (N-b)), LC last, which is the
 * order in which Alg. 1 and Alg. 2 visit candidates with a strict "<".
 * The returned energy is re-summed in a fixed order: users m = 0..N-1, each
 * adding (e + p_tx*up) if it offloads or its local energy otherwise, then
 * P_j*Phi.  Energies used only to rank candidates may be summed in another
 * order, so candidates whose energies agree to within rounding may be ranked
 * either way.
 *
 * Memory and streams.  Every array pointer is a DEVICE pointer owned by the
 * caller; scalars are host values.  Floating arrays have the element type
 * given by `dtype`.  Arrays are instance-major: x[i*len + k].  Calls enqueue
 * work on `hip_stream` (a hipStream_t passed as void*, NULL = the null
 * stream) and return without synchronizing; outputs are valid once the
 * stream has reached the call.  The library allocates no device memory, keeps
 * no mutable global state and is thread-safe.  To process a batch in chunks,
 * offset every per-instance pointer by the chunk start.
 *
 * Errors.  The return value is a jdob_status.  Only host-detectable errors
 * are reported: a NULL required pointer, a dimension below its minimum (1,
 * or 0 for I) or above the limits below, a non-finite or negative scalar,
 * an unknown dtype (JDOB_ERR_INVALID_ARG / JDOB_ERR_UNSUPPORTED), checked
 * before any HIP call so nothing is launched; a failed launch or device
 * query (JDOB_ERR_HIP).
 * Device-array preconditions (rates, deadlines and frequencies > 0,
 * frequencies strictly ascending, cycles/bits/alpha/beta >= 0, finite) are
 * documented, not checked: violating them yields unspecified values but
 * never an out-of-bounds access or a non-terminating kernel.  An instance
 * with no feasible candidate is data, not an error (status = 1).  An empty
 * batch (num_instances = 0) is not an error either: its other arguments are
 * checked as usual, except that every array pointer may be NULL, nothing
 * is launched and the call returns JDOB_OK.
 */
#ifndef JDOB_H
#define JDOB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Limits: N users, L layers, K local levels, J GPU levels, I instances.
 * Besides these, the rows one instance keeps on chip (arrays of N, L, K and
 * J entries) must fit 64 KB of LDS; a larger shape returns
 * JDOB_ERR_UNSUPPORTED before anything is launched.  With binary32 every N
 * up to JDOB_MAX_USERS fits at short chains (N <= 1021 at L = 255, K = 64,
 * J = 256; 948 with a continuous CPU frequency); with binary64 about
 * N <= 640 fits at short chains (435 at the largest L, K and J).  The outer
 * grouping and heterogeneous users are limited to 64 users. */
#define JDOB_MAX_USERS 1024
#define JDOB_MAX_LAYERS 255
#define JDOB_MAX_LOCAL_LEVELS 64
#define JDOB_MAX_GPU_LEVELS 256
#define JDOB_MAX_INSTANCES 2147483647
#define JDOB_MAX_GROUPED_USERS 64
#define JDOB_MAX_HETERO_USERS 64

typedef enum { JDOB_F32 = 0, JDOB_F64 = 1 } jdob_dtype;

/* Search mode bits (jdob_problem.mode); see "Search modes" above. */
typedef enum {
  JDOB_MODE_GRID = 0,            /* every batch size b at every (s, j)      */
  JDOB_MODE_GREEDY = 1,          /* Alg. 2: the greedy batching set only    */
  JDOB_MODE_FIXED_EDGE_FREQ = 2, /* f_e = f_e,max only (w/o edge DVFS)      */
  JDOB_MODE_BINARY = 4,          /* s = 0 or local computing only           */
  JDOB_MODE_CONTINUOUS_CPU = 8   /* continuous CPU frequency, Eq. (20)      */
} jdob_mode;

typedef enum {
  JDOB_OK = 0,
  JDOB_ERR_INVALID_ARG = 1, /* NULL pointer, dimension < 1, bad scalar       */
  JDOB_ERR_UNSUPPORTED = 2, /* dimension above a limit, unknown dtype        */
  JDOB_ERR_HIP = 3          /* device query or kernel launch failed          */
} jdob_status;

/* One batch of independent instances (Sec. II system model).
 * Per-instance arrays (device, instance-major, element type `dtype`):        */
typedef struct {
  int32_t num_instances;    /* I >= 0 (0: an empty batch, nothing to do)      */
  int32_t num_users;        /* N, 1..JDOB_MAX_USERS                           */
  int32_t num_layers;       /* L, 1..JDOB_MAX_LAYERS                          */
  int32_t num_local_levels; /* K, 1..JDOB_MAX_LOCAL_LEVELS                    */
  int32_t num_gpu_levels;   /* J, 1..JDOB_MAX_GPU_LEVELS                      */
  int32_t dtype;            /* jdob_dtype                                     */
  const void *layer_cycles; /* [I][L]   CPU cycles of layer l = 1..L (zeta g A_n
                               of Eq. (1)); >= 0                              */
  const void *out_bits;     /* [I][L+1] O_0 (DNN input) .. O_L, bits (Sec.
                               II-A); >= 0                                    */
  const void *gpu_alpha;    /* [I][L]   batch latency of layer l at the top GPU
                               frequency is alpha_l + beta_l * b seconds      */
  const void *gpu_beta;     /* [I][L]   (Eq. (5) with d_n(b) A_n affine in b) */
  const void *uplink_rate;  /* [I][N]   R_m, bit/s, > 0 (Eq. (3))             */
  const void *deadline;     /* [I][N]   T_m, seconds, > 0                     */
  const void *t_free;       /* [I]      time the GPU becomes free, s; NULL = 0 */
  const void *local_freq;   /* [K]      CPU levels f_k, Hz, ascending, > 0    */
  const void *gpu_freq;     /* [J]      GPU levels g_j, Hz, ascending, > 0;
                               g_{J-1} is the frequency alpha/beta refer to   */
  double kappa;             /* effective switched capacitance, Eq. (2)       */
  double p_tx;              /* transmit power p^u, W, Eq. (4)                 */
  double gpu_c;             /* GPU dynamic power gpu_c * g^3, W               */
  double gpu_p_static;      /* GPU static power P0, W                        */
  int32_t mode;             /* OR of jdob_mode bits; other bits are
                               JDOB_ERR_INVALID_ARG                           */
  /* Heterogeneous users (see "Heterogeneous users" above).  Each pointer is
     optional: NULL means the shared value; any non-NULL one selects the
     heterogeneous path (jdob_solve_batch and jdob_solve_grouped).           */
  const void *user_zeta;       /* [I][N] cycles per unit of layer work (1)   */
  const void *user_kappa;      /* [I][N] switched capacitance (kappa)        */
  const void *user_p_tx;       /* [I][N] transmit power, W (p_tx)            */
  const void *user_local_freq; /* [I][N][K] CPU levels, ascending
                                  (local_freq)                               */
} jdob_problem;

/* The chosen policy per instance (Alg. 1 output (E*, t_free*, X*)).
 * Outputs are caller-allocated device arrays.                               */
typedef struct {
  int32_t *status;      /* [I] 0 = feasible, 1 = no feasible candidate       */
  int32_t *cut;         /* [I] s* in [0, L]; L = local computing; -1 if none */
  int32_t *gpu_level;   /* [I] j*; -1 for local computing or if infeasible   */
  int32_t *batch;       /* [I] b* = |M_o| (Eq. (12)); 0 for LC / infeasible  */
  void *energy;         /* [I] E*, joules (Eq. (21)); +inf if infeasible     */
  void *t_free_out;     /* [I] GPU release time, Eq. (22); t_free for LC;
                           +inf if infeasible                                */
  int8_t *user_level;   /* [I][N] CPU level of user m (Eq. (20)), -1 if
                           infeasible or with a continuous CPU frequency     */
  int8_t *user_offload; /* [I][N] 1 if user m offloads at cut*, else 0       */
  int32_t *num_feasible;   /* [I] optional (NULL = skip): number of feasible
                              candidates among the L*J*N + 1 (those of the
                              mode's family)                                 */
  int64_t *num_user_evals; /* [I] optional (NULL = skip): sum of b over the
                              feasible (s, j, b) candidates                   */
  void *user_freq;         /* [I][N] optional (NULL = skip): CPU frequency of
                              user m, Hz (0 if infeasible)                     */
} jdob_policy;

/* Per-user option tables (stage 1).  Columns are users m in input order;
 * row s = 0..L is the partition point, row L is local computing.            */
typedef struct {
  int16_t *order;          /* [I][N] pi: users by rate descending, ties by
                              lower index (Alg. 1, sorting by Eq. (17))      */
  void *batch_deadline;    /* [I][N] lo[b] for b = 1..N (Eq. (10))           */
  int32_t *min_batch;      /* [I] bmin; 0 => local computing is feasible     */
  void *uplink_time;       /* [I][L+1][N] O_s / R_m (Eq. (3)); row L = 0     */
  void *gamma;             /* [I][L+1][N] uplink_time + t[s][K-1] (Eq. (17)) */
  int8_t *self_level;      /* [I][L+1][N] min k with t[s][k] <= T_m - up:
                              the user's min-energy level against its own
                              deadline; -1 if none                           */
  void *self_energy;       /* [I][L+1][N] e[s][k] + p_tx*up at self_level
                              (Eqs. (2), (4)); +inf if none                  */
  void *self_slack;        /* [I][L+1][N] (T_m - up) - t[s][k] at self_level,
                              at k = K-1 if none (then negative)             */
} jdob_user_tables;

/* Stage 1: per-user tables of every (partition point x CPU level) option:
 * local latency and energy (Eqs. (1), (2)), upload latency and energy
 * (Eqs. (3), (4)), deadline slack and each user's min-energy feasible level,
 * plus the rate order, batch deadlines and bmin used by stage 2.
 * Output size: I*(L+1)*N*(4*sizeof(P)+1) + I*N*(2+sizeof(P)) + 4*I bytes
 * (four P-typed tables and one int8 table per (instance, s, user); order,
 * batch_deadline per (instance, user); min_batch per instance).            */
int jdob_eval_user_tables(const jdob_problem *p, jdob_user_tables *out,
                          void *hip_stream);

/* Stage 2: given the stage-1 tables of the same problem, evaluate every
 * (partition point s x GPU level j x batch b) candidate of the mode's
 * family (every b, or the greedy b of Alg. 2) with the GPU batch
 * latency and energy of Eq. (5) at the batch size b, mask the deadline
 * constraints (6)-(8), and return the per-instance argmin (Alg. 1, Alg. 2,
 * Eqs. (20)-(22)).  Reads order, batch_deadline, min_batch, uplink_time and
 * rows L of self_level and self_energy (with JDOB_MODE_CONTINUOUS_CPU the
 * local energy is recomputed from the deadline, row L of self_energy is not
 * read).  Results are bitwise identical to
 * jdob_solve_batch on the same problem.                                     */
int jdob_eval_joint(const jdob_problem *p, const jdob_user_tables *tab,
                    jdob_policy *out, void *hip_stream);

/* Stages 1 and 2 fused in one kernel: the per-instance tables live in LDS
 * and never reach HBM.  Same outputs as jdob_eval_joint.                    */
int jdob_solve_batch(const jdob_problem *p, jdob_policy *out, void *hip_stream);

/* Outer grouping (the outer module of Sec. II, with the inner solve of this
 * library in the problem's mode).  Users are sorted by deadline ascending
 * (ties: lower index) and cut into consecutive groups, served one after
 * another: group g is one inner solve over its users (in user index order,
 * as an instance of its own) with the GPU free at the release time, Eq.
 * (22), of group g-1 (t_free for the first).  The grouping is a dynamic
 * program over prefixes of that order: for each prefix i it keeps a front
 * of states (total energy, GPU release time) none of which another state
 * dominates (no higher energy and no later release; of two equal states the
 * first generated stays), at most 16, sorted by energy.  The front of i
 * collects, for j = 0..i-1 and the states of the front of j from the
 * earliest release on, the state extended by the inner solve of users
 * ord[j..i-1] with the GPU free at its release time.  The answer is the
 * lowest-energy state of the full order; totals are summed group by group
 * in order.  (The paper takes its grouping from reference [9] without giving
 * it; this program is this library's reading.)  num_inner counts inner
 * solves with one per run of states that share a winner: a later free time
 * only removes candidates (constraint (6)), so the winner at one state is
 * the winner at every later state whose free time it meets.  All per-instance arrays are
 * caller-allocated device arrays; entries g >= num_groups of the per-group
 * arrays hold end 0, cut -1, level -1, batch 0, energy and release +inf.   */
typedef struct {
  int32_t *status;          /* [I] 0 = feasible, 1 = no feasible grouping     */
  int32_t *num_groups;      /* [I] G (0 if infeasible)                        */
  void *energy;             /* [I] total energy; +inf if infeasible          */
  void *t_free_out;         /* [I] release time after the last group         */
  int16_t *order;           /* [I][N] users by deadline ascending            */
  int16_t *group_end;       /* [I][N] group g = order[end(g-1) .. end(g)-1]  */
  int32_t *group_cut;       /* [I][N] partition point of group g (L = local) */
  int32_t *group_gpu_level; /* [I][N] GPU level of group g (-1 if local)     */
  int32_t *group_batch;     /* [I][N] offloaders of group g                   */
  void *group_energy;       /* [I][N] energy of group g (Eq. (21))           */
  void *group_t_free;       /* [I][N] release time after group g             */
  int8_t *user_level;       /* [I][N] CPU level of user m (-1 if infeasible
                               or with a continuous CPU frequency)          */
  int8_t *user_offload;     /* [I][N] 1 if user m offloads                   */
  int8_t *user_group;       /* [I][N] group of user m (-1 if infeasible)     */
  int64_t *num_inner;       /* [I] optional: inner solves the program ran   */
  int64_t *num_feasible;    /* [I] optional: their feasible candidates      */
  int64_t *num_user_evals;  /* [I] optional: their sums of b                */
  void *user_freq;          /* [I][N] optional: CPU frequency of user m, Hz */
} jdob_grouped_policy;

/* Outer grouping of every instance; N <= 64 (JDOB_ERR_UNSUPPORTED beyond).
 * Inner solves follow the problem's mode.                                  */
int jdob_solve_grouped(const jdob_problem *p, jdob_grouped_policy *out, void *hip_stream);

/* Static string for a jdob_status value; "unknown status" otherwise. */
const char *jdob_status_string(int code);

#ifdef __cplusplus
}
#endif

#endif /* JDOB_H */
