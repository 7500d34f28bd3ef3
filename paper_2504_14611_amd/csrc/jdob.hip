// jdob.hip — batched J-DOB policy evaluation for MI355X (gfx950).
//
// One wave64 (one workgroup) evaluates one problem instance:
//   1. coalesced row loads of the instance into LDS, the sums of Sec. III
//      (cycles of the local part, GPU coefficients of the offloaded part) in
//      the sequential order fixed by the ABI, the GPU stretch and power per
//      level (Eq. (5));
//   2. the rate order pi (Alg. 1 sorts users by Eq. (17); with shared cycles
//      that is rate descending), batch deadlines lo[b] (Eq. (10)), each
//      user's local-only level and energy (constraint (8), Eq. (20)) and bmin;
//   3. for every partition point s: the row of local latencies/energies
//      (Eqs. (1), (2)) and upload latencies (Eq. (3)) in LDS, then passes over
//      (GPU level j x batch b) candidates with lanes = (j, b): the deadline
//      mask (6)-(8), each offloader's lowest feasible CPU level (Eq. (20)),
//      the energy (Eq. (21)) and a per-lane running argmin;
//   4. a wavefront argmin with lowest-index ties, the winner's per-user
//      levels, the canonical energy sum and the release time (Eq. (22)).
//
// Two facts let the kernel skip work without changing the result (both
// follow from the rounding of each operation being monotone):
//   * for fixed (s, j) the feasible batches are an interval [max(bmin,1),
//     bmax], and bmax grows with the GPU frequency (the monotone thresholds
//     of Eq. (18)): a pass over b with no feasible lane ends the partition
//     point, and the test at (top GPU level, smallest batch) decides whether
//     the partition point has any feasible candidate at all;
//   * inside a candidate the budget H - up[i] shrinks along pi, so the
//     offloaders' levels never decrease: each lane advances its level
//     instead of searching it per user.
// The kernel is a VALU/LDS-bound loop of compares, selects and adds: it is
// not a dense contraction and uses no matrix cores.

#include "jdob_common.h"

namespace {

using namespace jdob_dev;


template <typename T> struct Problem {
  const T *cyc, *bits, *alpha, *beta, *rate, *deadline, *tfree, *lf, *gf;
  T kappa, ptx, gc, p0;
  int N, L, K, J;
  int s_end;  // partition points searched: s in [0, s_end) (1 with binary offloading)
  int j_low;  // GPU levels searched: j in [j_low, J) (J-1 without edge DVFS)
  int cont;   // continuous CPU frequency in [lf[0], lf[K-1]]
};

template <typename T> struct Policy {
  int32_t *status, *cut, *gpu_level, *batch;
  T *energy, *tfree_out;
  int8_t *ulevel, *uoffload;
  int32_t *nfeas;
  int64_t *nevals;
  T *ufreq;
};

template <typename T> struct Tables {
  int16_t *order;
  T *lo;
  int32_t *bmin;
  T *up, *gamma;
  int8_t *slevel;
  T *senergy, *sslack;
};

// Everything one solve launch needs, passed as its single kernel argument so
// that parts of it can be read where they are used (see solve_args).
template <typename T> struct SolveArgs {
  Problem<T> p;
  Tables<T> tab;
  Policy<T> out;
  int64_t first;  // instance of block 0
};

template <typename T> struct Grouped {
  int32_t *status, *num_groups;
  T *energy, *tfree_out;
  int16_t *order, *group_end;
  int32_t *group_cut, *group_gpu_level, *group_batch;
  T *group_energy, *group_tfree;
  int8_t *ulevel, *uoffload, *ugroup;
  int64_t *ninner, *nfeas, *nevals;
  T *ufreq;
};

template <typename T> struct GroupedArgs {
  Problem<T> p;
  Grouped<T> out;
  int64_t first;
};

// Byte offsets of the per-instance LDS arrays.
struct Layout {
  int cyc, al, be, bits, C, A, B, f, eps, r, P, pi, rate, dl, lo, kL, eL, fL, SL, te, up, bt, term,
      sflag, q, total;
};

// Room of the queue of candidates whose offloaders span several CPU levels
// (entries of a pass join it; 64 of them are evaluated together).
constexpr int QCAP = 2 * WAVE;

// Whether the grid search with CPU levels queues those candidates: from 17
// users up (measured: c2 with 16 users 0.86 ms walking, 0.95 ms queued; c3
// with 32 users 11.1 ms walking, 10.8 ms queued, before other changes).
__host__ __device__ inline bool queued_search(int N, bool cont, bool greedy) {
  return N > 16 && !cont && !greedy;
}


// Entries of a row of CPU levels: K levels, then sentinels (latency -inf,
// which fits every budget) up to at least K + 2 and the next power of two,
// so that the level searches need no bounds tests.
__host__ __device__ inline int level_row_len(int K) {
  int k2 = 1;
  while (k2 < K) k2 <<= 1;
  return k2 > K + 2 ? k2 : K + 2;
}

// Batch records past N that the search reads: a pass of the grid holds
// WAVE / min(Jn, WAVE) batch sizes (Jn GPU levels searched), and its lanes
// read records up to b0 + that count with b0 <= N; the greedy search keeps
// WAVE + 1 (a second set of rows may share their room).
__host__ __device__ inline int batch_sentinels(int Jn, bool greedy) {
  return greedy ? WAVE + 1 : WAVE / (Jn < WAVE ? Jn : WAVE) + 1;
}

// cont: room for the local-only frequencies (continuous CPU frequency only;
// with levels they are the level table read at kL).
// queue: room for the queue of the grid search (queued_search).
// nsent: batch records past N (batch_sentinels).
__host__ __device__ inline Layout make_layout(int N, int L, int K, int J, int szT, bool cont,
                                              bool queue, int nsent) {
  const int room = N + 1 + nsent;  // batch records 0..N and the sentinels
  Layout y;
  int o = 0;
  auto take = [&](int bytes) { int r = o; o = align8(o + bytes); return r; };
  auto take32 = [&](int bytes) { o = (o + 31) & ~31; int r = o; o = align8(o + bytes); return r; };
  // raw layer rows of the instance: read only while the sums C, A, B are
  // formed, before anything else uses the batch-record room, so they sit in
  // that room when they fit
  const bool raw_in_bt = 3 * L <= 4 * room;
  if (!raw_in_bt) {
    y.cyc = take(L * szT);
    y.al = take(L * szT);
    y.be = take(L * szT);
  }
  y.bits = take((L + 1) * szT);   // output bits O_0..O_L (Eq. (3))
  y.C = take((L + 1) * szT);      // cycles of layers 1..s
  y.A = take((L + 1) * szT);      // alpha summed over layers s+1..L
  y.B = take((L + 1) * szT);      // beta summed over layers s+1..L
  y.f = take(K * szT);            // CPU levels
  y.eps = take(K * szT);          // kappa * f^2
  y.r = take(J * szT);            // g_{J-1} / g_j
  y.P = take(J * szT);            // GPU power at level j
  y.pi = take(N * 2);             // users by rate descending (N <= 1024)
  y.rate = take(N * szT);         // rate, by user (pi order after sorting)
  y.dl = take(N * szT);           // deadline by user
  y.lo = take((N + 1) * szT);     // lo[b], b = 1..N
  y.kL = take(N);                 // local-only level by user (-1: none; K <= 64)
  y.eL = take(N * szT);           // local-only energy by user
  y.fL = take(cont ? N * szT : 0);  // local-only CPU frequency by user
  y.SL = take((N + 1) * szT);     // SL[b] = sum_{i>=b} eL[pi_i]
  y.te = take(level_row_len(K) * 2 * szT); // row s: (latency, energy) per level, sentinels
  y.up = take32((((N + 3) & ~3) + 8) * szT);  // row s of upload latencies (+ read-ahead pad)
  y.bt = take32(room * 4 * szT);  // row s: per batch size b (+ sentinels)
  if (raw_in_bt) {
    y.cyc = y.bt;
    y.al = y.bt + L * szT;
    y.be = y.bt + 2 * L * szT;
  }
  y.sflag = take(L + 1);          // partition point has a feasible candidate
  y.q = take(queue ? QCAP * 4 : 0);  // queued candidates: b | j << 11 | first level << 19
  // per-user energy of the winner: written after the search has emptied the
  // queue, so it shares the queue's room where that holds it
  y.term = (queue && N * szT <= QCAP * 4) ? y.q : take(N * szT);
  y.total = o;
  return y;
}

// LDS of the grouped call beyond the single-instance layout: the instance's
// rate order and rates, each user's position in the deadline order and the
// deadline order itself, the dynamic program's fronts, the chosen groups.
struct GLayout {
  int pi_all, rate_all, drank, dord, fE, fT, from, fn, ends, eks, total;
};

__host__ __device__ inline GLayout make_glayout(const Layout &y, int N, int szT) {
  GLayout g;
  int o = y.total;
  auto take = [&](int bytes) { int r = o; o = align8(o + bytes); return r; };
  g.pi_all = take(N * 4);       // all users by rate descending
  g.rate_all = take(N * szT);   // their rates, in that order
  g.drank = take(N * 4);        // position of user m in the deadline order
  g.dord = take(N * 4);         // users by deadline ascending
  const int F = GROUP_FRONT;    // front of prefix i: slots i*F .. i*F + F-1
  g.fE = take((N + 1) * F * szT);  // total energy of the first i users
  g.fT = take((N + 1) * F * szT);  // GPU release time after them
  g.from = take((N + 1) * F * 2);  // the state it extends (prefix * F + slot)
  g.fn = take((N + 1) * 4);        // states in the front of prefix i
  g.ends = take((N + 1) * 4);      // ends of the chosen groups, in order
  g.eks = take((N + 1) * 4);       // the chosen state at each end
  g.total = o;
  return g;
}


// The launch's argument block in the kernel-argument segment.  The output
// pointers are read through it where the results are stored; read through
// the by-value parameter, they would be loaded at kernel entry and held (or
// spilled and restored) in scalar registers across the candidate loops.
template <typename T>
__device__ inline const __attribute__((address_space(4))) SolveArgs<T> *solve_args() {
  return (const __attribute__((address_space(4))) SolveArgs<T> *)
      __builtin_amdgcn_kernarg_segment_ptr();
}

template <typename T> __device__ inline Policy<T> output_pointers() {
  const auto *a = solve_args<T>();
  Policy<T> o;
  o.status = a->out.status;
  o.cut = a->out.cut;
  o.gpu_level = a->out.gpu_level;
  o.batch = a->out.batch;
  o.energy = a->out.energy;
  o.tfree_out = a->out.tfree_out;
  o.ulevel = a->out.ulevel;
  o.uoffload = a->out.uoffload;
  o.nfeas = a->out.nfeas;
  o.nevals = a->out.nevals;
  o.ufreq = nullptr;  // read where it is stored: freq_row
  return o;
}

// Row inst of the optional user_freq output, read from the kernel arguments
// only where the frequencies are stored (nullptr when not requested).
template <typename T> __device__ inline T *freq_row(int64_t inst, int N) {
  T *f = solve_args<T>()->out.ufreq;
  return f ? f + inst * N : nullptr;
}


template <typename T> __device__ inline Problem<T> own_problem(const Problem<T> &q) {
  Problem<T> p;
  p.cyc = own(q.cyc);
  p.bits = own(q.bits);
  p.alpha = own(q.alpha);
  p.beta = own(q.beta);
  p.rate = own(q.rate);
  p.deadline = own(q.deadline);
  p.tfree = own(q.tfree);
  p.lf = own(q.lf);
  p.gf = own(q.gf);
  p.kappa = own(q.kappa);
  p.ptx = own(q.ptx);
  p.gc = own(q.gc);
  p.p0 = own(q.p0);
  p.N = own(q.N);
  p.L = own(q.L);
  p.K = own(q.K);
  p.J = own(q.J);
  p.s_end = own(q.s_end);
  p.j_low = own(q.j_low);
  p.cont = q.cont;  // the kernels take it as a template argument
  return p;
}


// Position of each user in pi: the number of users before it (a higher rate,
// or an equal rate and a lower index).  For binary32 rates this is the order
// of the 64-bit keys (rate bits, ~index): non-negative IEEE values order like
// their bit patterns and the index makes every key distinct, so the ranks are
// always a permutation.  skey holds room for N + 1 keys.
template <bool WS = false, typename I>
__device__ inline void rank_users(const float *srate, uint64_t *skey, I *spi, int N, int lane) {
  for (int m = lane; m <= N; m += WAVE)  // key N: below every user's, pads an odd count
    skey[m] = m < N ? ((uint64_t)__float_as_uint(srate[m]) << 32) |
                          (uint64_t)(0xffffffffu - (unsigned)m)
                    : uint64_t(0);
  lds_sync<WS>();
  if (2 * N <= WAVE) {
    // two lanes per user: lane m counts the keys above its own among the
    // first half of the users, lane m + 32 among the others
    const int m = lane & (WAVE / 2 - 1), half = (N + 1) >> 1;
    const int q0 = (lane >> 5) * half;
    const uint64_t km = skey[m < N ? m : 0];
    int rank = 0;
    for (int i = 0; i < half; ++i) rank += (skey[q0 + i] > km) ? 1 : 0;
    rank += from_upper_half(rank);
    if (lane < N) spi[rank] = m;
    return;
  }
  for (int m0 = 0; m0 < N; m0 += WAVE) {
    const int m = m0 + lane;
    const uint64_t km = skey[m < N ? m : 0];
    int rank = 0;
    for (int q = 0; q < N; ++q) rank += (skey[q] > km) ? 1 : 0;
    if (m < N) spi[rank] = m;
  }
}
template <bool WS = false, typename I>
__device__ inline void rank_users(const double *srate, uint64_t *, I *spi, int N, int lane) {
  for (int m0 = 0; m0 < N; m0 += WAVE) {
    const int m = m0 + lane;
    const double rm = srate[m < N ? m : 0];
    int rank = 0;
    for (int q = 0; q < N; ++q) {
      const double rq = srate[q];
      rank += (rq > rm || (rq == rm && q < m)) ? 1 : 0;
    }
    if (m < N && rank < N) spi[rank] = m;
  }
}

// Everything an instance needs before its candidates are enumerated.

template <typename T, bool FROM_TABLES, bool CONT>
__device__ void prepare_instance(const Problem<T> &p, const Tables<T> &tab, int64_t inst,
                                 unsigned char *smem, const Layout &y, int lane, int &bmin_out) {
  const int N = p.N, L = p.L, K = p.K, J = p.J;
  T *sC = (T *)(smem + y.C), *sA = (T *)(smem + y.A), *sB = (T *)(smem + y.B);
  T *sf = (T *)(smem + y.f), *seps = (T *)(smem + y.eps);
  T *sr = (T *)(smem + y.r), *sP = (T *)(smem + y.P);
  int16_t *spi = (int16_t *)(smem + y.pi);
  T *srate = (T *)(smem + y.rate), *sdl = (T *)(smem + y.dl), *slo = (T *)(smem + y.lo);
  int8_t *skL = (int8_t *)(smem + y.kL);
  T *seL = (T *)(smem + y.eL), *sSL = (T *)(smem + y.SL), *sfL = (T *)(smem + y.fL);
  Level<T> *ste = (Level<T> *)(smem + y.te);
  T *scyc = (T *)(smem + y.cyc), *sal = (T *)(smem + y.al), *sbe = (T *)(smem + y.be);
  T *sbits = (T *)(smem + y.bits);
  T *sup = (T *)(smem + y.up);

  const T *cyc = p.cyc + inst * L;
  const T *al = p.alpha + inst * L;
  const T *be = p.beta + inst * L;
  const T *rate = p.rate + inst * N;
  const T *dl = p.deadline + inst * N;

  // shared level tables: CPU levels (Eq. (1), (2)), GPU levels (Eq. (5))
  for (int k = lane; k < K; k += WAVE) {
    T f = p.lf[k];
    sf[k] = f;
    seps[k] = p.kappa * (f * f);
  }
  for (int j = lane; j < J; j += WAVE) {
    T g = p.gf[j], gtop = p.gf[J - 1];
    sr[j] = gtop / g;
    sP[j] = p.gc * ((g * g) * g) + p.p0;
  }
  // instance rows (coalesced)
  for (int l = lane; l < L; l += WAVE) {
    scyc[l] = cyc[l];
    sal[L - 1 - l] = al[l];  // reversed: see chain_sums
    sbe[L - 1 - l] = be[l];
  }
  if (!FROM_TABLES)
    for (int l = lane; l <= L; l += WAVE) sbits[l] = p.bits[inst * (L + 1) + l];
  for (int m = lane; m < N; m += WAVE) {
    srate[m] = rate[m];
    sdl[m] = dl[m];
  }
  __syncthreads();
  // the sums C, A, B in the sequential order of the ABI contract
  chain_sums(scyc, sal, sbe, sC, sA, sB, L, lane);

  int bmin;
  if (!FROM_TABLES) {
    // rank of user m in pi: users with a higher rate, or an equal rate and a
    // lower index, come first
    for (int i = lane; i < N; i += WAVE) spi[i] = i;  // stays a permutation of valid users
    __syncthreads();
    rank_users(srate, (uint64_t *)(smem + y.bt), spi, N, lane);
    __syncthreads();
  } else {
    const int16_t *ord = tab.order + inst * N;
    for (int i = lane; i < N; i += WAVE) {
      int m = ord[i];
      spi[i] = (m >= 0 && m < N) ? m : 0;
    }
    __syncthreads();
  }

  // batch deadlines (Eq. (10)) and the rate of the i-th user of pi
  {
    T carry = inf_of<T>();
    for (int i0 = 0; i0 < N; i0 += WAVE) {
      const int i = i0 + lane;
      if (i < N) sup[i] = srate[spi[i]];
      if (!FROM_TABLES) {
        T d = (i < N) ? sdl[spi[i]] : inf_of<T>();
        T v = wave_scan<T, true>(d, lane);
        v = (carry < v) ? carry : v;
        if (i < N) slo[i + 1] = v;
        carry = lane_read(v, WAVE - 1);
      } else {
        if (i < N) slo[i + 1] = tab.lo[inst * N + i];
      }
    }
    if (lane == 0) slo[0] = inf_of<T>();
    __syncthreads();
    for (int i = lane; i < N; i += WAVE) srate[i] = sup[i];
    __syncthreads();
  }

  // local computing of the whole chain: constraint (8) with Eq. (20)
  for (int k = lane; k < K; k += WAVE) {
    ste[k].t = sC[L] / sf[k];
    ste[k].e = seps[k] * sC[L];
  }
  __syncthreads();
  for (int m = lane; m < N; m += WAVE) {
    int kL = -1;
    T eL = inf_of<T>();
    if (!FROM_TABLES) {
      const T Tm = sdl[m];
      for (int k = K - 1; k >= 0; --k)
        if (ste[k].t <= Tm) kL = k;
      if (kL >= 0) eL = ste[kL].e;
    } else {
      const int64_t o = (inst * (L + 1) + L) * N + m;
      kL = tab.slevel[o];
      if (kL < -1 || kL >= K) kL = -1;
      eL = (kL >= 0) ? tab.senergy[o] : inf_of<T>();
    }
    if (CONT) {  // Eq. (20) with its clamp against the user's deadline
      T fL = T(0);
      if (kL >= 0) {
        fL = cont_freq(sC[L], sdl[m], sf[0], sf[K - 1]);
        eL = (p.kappa * (fL * fL)) * sC[L];
      }
      sfL[m] = fL;
    }
    skL[m] = kL;
    seL[m] = eL;
  }
  __syncthreads();
  // bmin = 1 + last position in pi of a user with no local level
  {
    int bm = 0;
    for (int i0 = 0; i0 < N; i0 += WAVE) {  // the last such position, chunk by chunk
      const int i = i0 + lane;
      const uint64_t nl = __builtin_amdgcn_ballot_w64(i < N && skL[spi[i < N ? i : 0]] < 0);
      if (nl) bm = i0 + 64 - __clzll((long long)nl);
    }
    if (FROM_TABLES) {
      int tb = tab.bmin[inst];
      bm = (tb < 0) ? 0 : (tb > N ? N + 1 : tb);
    }
    bmin = bm;
  }
  // SL[b] = sum of the local energies of pi[b..N-1] (ranking only)
  {
    T carry = T(0);
    for (int i0 = ((N - 1) / WAVE) * WAVE; i0 >= 0; i0 -= WAVE) {
      // reversed inclusive scan inside the chunk: lane q holds pi index
      // i0 + WAVE - 1 - q
      const int i = i0 + WAVE - 1 - lane;
      T v = (i < N) ? seL[spi[i]] : T(0);
      v = wave_scan<T, false>(v, lane) + carry;
      if (i < N) sSL[i] = v;
      carry = lane_read(v, WAVE - 1);
    }
    if (lane == 0) sSL[N] = T(0);
  }
  __syncthreads();
  bmin_out = bmin;
}

// Wave-wide minimum and maximum (every lane gets the value).
template <typename T> __device__ inline T wave_min(T v) {
  v = wave_iscan(v, inf_of<T>(), [](T a, T b) { return b < a ? b : a; });
  return lane_read(v, WAVE - 1);
}
__device__ inline int wave_min_int(int v) {
  v = wave_iscan(v, 0x7fffffff, [](int a, int b) { return b < a ? b : a; });
  return lane_read(v, WAVE - 1);
}
__device__ inline int wave_sum_int(int v) {
  v = wave_iscan(v, 0, [](int a, int b) { return a + b; });
  return lane_read(v, WAVE - 1);
}

// Preparation of the fused solve.  Every step is exact (orders, minima and
// the tests of the contract), so the candidate search only runs where it can
// find something:
//   1. the rows, the level tables, the sums C, A, B, and each user's local
//      level and energy against its own deadline (constraint (8), Eq. (20));
//   2. without sorting the users: bmin, from the last user of pi that has no
//      local level (its position is the number of users before it in the
//      rate order), and the batch deadline lo[blo] and rate of the blo-th
//      user of pi that the partition-point test needs, blo = max(bmin, 1);
//   3. the test of every partition point at the top GPU level and batch blo
//      (feasibility is monotone in b and j, so a partition point failing it
//      has no feasible candidate);
//   4. only if some partition point passes: the rate order pi, the batch
//      deadlines lo[b], the rates in pi order and the local-energy suffix
//      sums SL that the search reads.
// Returns whether some partition point passed; bmin_out receives bmin.
template <typename T, bool CONT>
__device__ bool prepare_fused(const Problem<T> &p, int64_t inst, unsigned char *smem,
                              const Layout &y, int lane, T tfree, int &bmin_out) {
  const int N = p.N, L = p.L, K = p.K, J = p.J;
  T *sC = (T *)(smem + y.C), *sA = (T *)(smem + y.A), *sB = (T *)(smem + y.B);
  T *sf = (T *)(smem + y.f), *seps = (T *)(smem + y.eps);
  T *sr = (T *)(smem + y.r), *sP = (T *)(smem + y.P);
  int16_t *spi = (int16_t *)(smem + y.pi);
  T *srate = (T *)(smem + y.rate), *sdl = (T *)(smem + y.dl), *slo = (T *)(smem + y.lo);
  int8_t *skL = (int8_t *)(smem + y.kL);
  T *seL = (T *)(smem + y.eL), *sSL = (T *)(smem + y.SL), *sfL = (T *)(smem + y.fL);
  Level<T> *ste = (Level<T> *)(smem + y.te);
  T *scyc = (T *)(smem + y.cyc), *sal = (T *)(smem + y.al), *sbe = (T *)(smem + y.be);
  T *sbits = (T *)(smem + y.bits);
  T *sup = (T *)(smem + y.up);
  int8_t *sflag = (int8_t *)(smem + y.sflag);

  // 1. level tables (Eqs. (1), (2), (5)) and the instance rows (coalesced)
  for (int k = lane; k < K; k += WAVE) {
    const T f = p.lf[k];
    sf[k] = f;
    seps[k] = p.kappa * (f * f);
  }
  for (int j = lane; j < J; j += WAVE) {
    const T g = p.gf[j], gtop = p.gf[J - 1];
    sr[j] = gtop / g;
    sP[j] = p.gc * ((g * g) * g) + p.p0;
  }
  for (int l = lane; l < L; l += WAVE) {
    scyc[l] = p.cyc[inst * L + l];
    sal[L - 1 - l] = p.alpha[inst * L + l];  // reversed: see chain_sums
    sbe[L - 1 - l] = p.beta[inst * L + l];
  }
  for (int l = lane; l <= L; l += WAVE) sbits[l] = p.bits[inst * (L + 1) + l];
  for (int m = lane; m < N; m += WAVE) {
    srate[m] = p.rate[inst * N + m];
    sdl[m] = p.deadline[inst * N + m];
  }
  __syncthreads();
  // the sums C, A, B in the sequential order of the contract
  chain_sums(scyc, sal, sbe, sC, sA, sB, L, lane);
  // local computing of the whole chain: each user's lowest level meeting
  // its deadline (latency falls with the level: binary search for the
  // number of levels that are too slow)
  for (int k = lane; k < K; k += WAVE) {
    ste[k].t = sC[L] / sf[k];
    ste[k].e = seps[k] * sC[L];
  }
  __syncthreads();
  int K2 = 1;
  while (K2 < K) K2 <<= 1;
  for (int m = lane; m < N; m += WAVE) {
    const T Tm = sdl[m];
    int c = 0;
    for (int step = K2 >> 1; step > 0; step >>= 1) {
      const int nc = c + step;
      c = (nc <= K && ste[nc - 1].t > Tm) ? nc : c;
    }
    const int kL = (c < K && ste[c].t <= Tm) ? c : -1;
    T eL = kL >= 0 ? ste[kL].e : inf_of<T>();
    if (CONT) {  // Eq. (20) with its clamp against the user's deadline
      T fL = T(0);
      if (kL >= 0) {
        fL = cont_freq(sC[L], Tm, sf[0], sf[K - 1]);
        eL = (p.kappa * (fL * fL)) * sC[L];
      }
      sfL[m] = fL;
    }
    skL[m] = kL;
    seL[m] = eL;
  }

  // 2. bmin and the blo-th user of pi without sorting.  pi orders users by
  // rate descending, ties by lower index.  The last user of pi without a
  // local level has the lowest rate among them, then the highest index.
  T rbad = inf_of<T>();
  int nbad = 0;
  for (int m = lane; m < N; m += WAVE)
    if (skL[m] < 0) {
      rbad = srate[m] < rbad ? srate[m] : rbad;
      ++nbad;
    }
  rbad = wave_min(rbad);
  int bmin = 0, ub = -1;
  // (up to 64 users, lane m holds user m: the index maxima, minima and
  // counts are ballots)
  const bool one = N <= WAVE;
  const T rm = (one && lane < N) ? srate[lane] : T(0);
  if (__builtin_amdgcn_ballot_w64(nbad > 0)) {
    if (one) {
      const uint64_t bb = __builtin_amdgcn_ballot_w64(lane < N && skL[lane] < 0 && rm == rbad);
      ub = bb ? 63 - __clzll((long long)bb) : -1;
      bmin = __popcll(__builtin_amdgcn_ballot_w64(
          lane < N && (rm > rbad || (rm == rbad && lane <= ub))));
    } else {
      int ib = -1;
      for (int m = lane; m < N; m += WAVE)
        if (skL[m] < 0 && srate[m] == rbad) ib = m;
      ub = wave_max_int(ib);  // the last user of pi without a local level
      int cnt = 0;            // users at or before it in pi
      for (int m = lane; m < N; m += WAVE)
        cnt += (srate[m] > rbad || (srate[m] == rbad && m <= ub)) ? 1 : 0;
      bmin = wave_sum_int(cnt);
    }
  } else {                  // the first user of pi
    T rtop = -inf_of<T>();
    for (int m = lane; m < N; m += WAVE) rtop = srate[m] > rtop ? srate[m] : rtop;
    rtop = wave_max(rtop);
    if (one) {
      const uint64_t bt = __builtin_amdgcn_ballot_w64(lane < N && rm == rtop);
      ub = bt ? __builtin_ctzll(bt) : 0x7fffffff;
    } else {
      int it = 0x7fffffff;
      for (int m = lane; m < N; m += WAVE)
        if (srate[m] == rtop) it = m < it ? m : it;
      ub = wave_min_int(it);
    }
  }
  ub = ub < 0 ? 0 : (ub < N ? ub : N - 1);  // (only with rates outside the contract)
  // lo[blo]: the tightest deadline among the first blo users of pi
  const T rb = srate[ub];
  T dmin = inf_of<T>();
  for (int m = lane; m < N; m += WAVE)
    if (srate[m] > rb || (srate[m] == rb && m <= ub)) dmin = sdl[m] < dmin ? sdl[m] : dmin;
  const T lob = wave_min(dmin);
  const int blo = bmin > 1 ? bmin : 1;

  // 3. the test of every partition point at (top GPU level, blo); up to 32
  // partition points, one division sequence serves both quotients: lanes
  // [0, 32) divide C[s] by the top level, lanes [32, 64) O_s by the rate
  int any = 0;
  if (2 * p.s_end <= WAVE) {
    const bool hi = lane >= WAVE / 2;
    const int s = hi ? lane - WAVE / 2 : lane;
    const int sc = s < p.s_end ? s : 0;
    const T q = (hi ? sbits[sc] : sC[sc]) / (hi ? rb : sf[K - 1]);
    const T upl = from_upper_half(q);
    if (!hi && s < p.s_end) {
      const T Phi = (sA[s] + sB[s] * T(blo)) * sr[J - 1];
      const T H = lob - Phi;
      const int ok = (H >= tfree) && (q <= H - upl);  // q: the top level's latency
      sflag[s] = ok;
      any |= ok;
    }
  } else {
    for (int s = lane; s < p.s_end; s += WAVE) {
      const T tK1 = sC[s] / sf[K - 1];
      const T upl = sbits[s] / rb;
      const T Phi = (sA[s] + sB[s] * T(blo)) * sr[J - 1];
      const T H = lob - Phi;
      const int ok = (H >= tfree) && (tK1 <= H - upl);
      sflag[s] = ok;
      any |= ok;
    }
  }
  bmin_out = bmin;
  if (!__builtin_amdgcn_ballot_w64(any != 0)) {
    if (bmin == 0) {  // local computing is the only candidate: its ranking energy
      T e = T(0);
      for (int m = lane; m < N; m += WAVE) e = e + seL[m];
      e = wave_iscan(e, T(0), [](T a, T b) { return a + b; });
      if (lane == 0) sSL[0] = lane_read(e, WAVE - 1);
    }
    __syncthreads();
    return false;
  }

  // 4. the rate order, batch deadlines (Eq. (10)), rates in pi order and
  // the local-energy suffix sums (ranking only)
  for (int i = lane; i < N; i += WAVE) spi[i] = i;  // stays a permutation of valid users
  __syncthreads();
  rank_users(srate, (uint64_t *)(smem + y.bt), spi, N, lane);
  __syncthreads();
  {
    T carry = inf_of<T>();
    for (int i0 = 0; i0 < N; i0 += WAVE) {
      const int i = i0 + lane;
      if (i < N) sup[i] = srate[spi[i]];
      const T d = (i < N) ? sdl[spi[i]] : inf_of<T>();
      T v = wave_scan<T, true>(d, lane);
      v = (carry < v) ? carry : v;
      if (i < N) slo[i + 1] = v;
      carry = lane_read(v, WAVE - 1);
    }
    if (lane == 0) slo[0] = inf_of<T>();
    __syncthreads();
    for (int i = lane; i < N; i += WAVE) srate[i] = sup[i];
  }
  {
    T carry = T(0);
    for (int i0 = ((N - 1) / WAVE) * WAVE; i0 >= 0; i0 -= WAVE) {
      // reversed inclusive scan inside the chunk: lane q holds pi index
      // i0 + WAVE - 1 - q
      const int i = i0 + WAVE - 1 - lane;
      T v = (i < N) ? seL[spi[i]] : T(0);
      v = wave_scan<T, false>(v, lane) + carry;
      if (i < N) sSL[i] = v;
      carry = lane_read(v, WAVE - 1);
    }
    if (lane == 0) sSL[N] = T(0);
  }
  __syncthreads();
  return true;
}

// The CPU frequency of user m when it computes every layer locally: the
// continuous one stored by prepare_instance, or the frequency of its level.
template <typename T, bool CONT>
__device__ inline T local_freq(const unsigned char *smem, const Layout &y, int m) {
  if (CONT) return ((const T *)(smem + y.fL))[m];
  const int k = ((const int8_t *)(smem + y.kL))[m];
  return k >= 0 ? ((const T *)(smem + y.f))[k] : T(0);
}

// What an offloader with budget x runs at partition point s (row ste built
// for s): the lowest level meeting the budget (Eq. (20) on the levels), or
// the continuous frequency; its level (-1 if continuous), frequency, CPU
// energy (Eq. (2)) and local latency (Eq. (1)).
template <typename T, bool CONT>
__device__ inline void offloader_choice(const Problem<T> &p, const Level<T> *ste, const T *sf,
                                        T Cs, T x, int &lv, T &fq, T &e, T &tl) {
  const int K = p.K;
  int k = K - 1;
  for (int q = K - 1; q >= 0; --q)
    if (ste[q].t <= x) k = q;
  if (CONT) {
    fq = cont_freq(Cs, x, sf[0], sf[K - 1]);
    e = (p.kappa * (fq * fq)) * Cs;
    tl = Cs / fq;
    lv = -1;
  } else {
    fq = sf[k];
    e = ste[k].e;
    tl = ste[k].t;
    lv = k;
  }
}


// Continuous CPU frequency, for ranking only: the sum over a lane's
// offloaders 0..b-1 of f^2, f = Cs / (Hu - up) (hardware reciprocal) clamped
// to [fmin, fmax]; the CPU energy of the lane's candidate is kappa * Cs times
// it.  Users 0..b_all-1 belong to every feasible lane's batch and are summed
// unmasked (four per broadcast read; the padded row covers the read past
// b_all), users b_all..bw-1 only where the lane's batch holds them.  Lanes
// that are infeasible sum garbage that the caller drops.  Cs > 0.
template <typename T>
__device__ inline T cont_sum_f2(const T *sup, T Hu, int b, int b_all, int bw, T Cs, T fmin,
                                T fmax) {
  T acc = T(0);
  int g = 0;
  for (; g + 4 <= b_all; g += 4) {
    const Quad<T> q = *(const Quad<T> *)(sup + g);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const T fr = clamp_(Cs * fast_rcp(Hu - q.v[c]), fmin, fmax);
      acc = fma_(fr, fr, acc);
    }
  }
  for (; g < b_all; ++g) {
    const T fr = clamp_(Cs * fast_rcp(Hu - sup[g]), fmin, fmax);
    acc = fma_(fr, fr, acc);
  }
  for (; g < bw; ++g) {
    const T fr = clamp_(Cs * fast_rcp(Hu - sup[g]), fmin, fmax);
    acc = (g < b) ? fma_(fr, fr, acc) : acc;
  }
  return acc;
}

// Upload latencies of partition point s in pi order (Eq. (3)).
template <typename T, bool FROM_TABLES>
__device__ inline T upload_time(const Problem<T> &p, const Tables<T> &tab, int64_t inst,
                                const T *sbits, const T *srate, const int16_t *spi, int s,
                                int i) {
  if (FROM_TABLES) return tab.up[(inst * (p.L + 1) + s) * p.N + spi[i]];
  return sbits[s] / srate[i];
}

// The candidates of the mode's family for the user set held in LDS: N users
// in pi order (rate, lo, SL, pi arrays), smallest admissible batch blo, GPU
// free at tfree.  Leaves each lane's best (energy, flat index) in bestE,
// bestI (strict order over partition points, lowest index among equal
// energies) and adds the lane's work to nfeas and nevals when COUNT.
// Candidates whose offloaders span several CPU levels: with QUEUE they wait
// in a queue and are evaluated 64 at a time, each run of equal level found
// by binary search over the users; without it (few users) their runs are
// summed by a walk over the users during the pass.
template <typename T, bool FROM_TABLES, bool ONE_CHUNK, bool COUNT, bool GREEDY, bool CONT,
          bool QUEUE>
__device__ inline void search_candidates(const Problem<T> &p, const Tables<T> &tab, int64_t inst,
                                         unsigned char *smem, const Layout &y, int lane, int N,
                                         int blo, T tfree, T &bestE, int &bestI, int &nfeas,
                                         int &nevals, bool flags_ready = false) {
  const int L = p.L, K = p.K, J = p.J;
  const int s_end = p.s_end, j_low = p.j_low;
  T *sC = (T *)(smem + y.C), *sA = (T *)(smem + y.A), *sB = (T *)(smem + y.B);
  T *sf = (T *)(smem + y.f), *seps = (T *)(smem + y.eps);
  T *sr = (T *)(smem + y.r), *sP = (T *)(smem + y.P);
  int16_t *spi = (int16_t *)(smem + y.pi);
  T *srate = (T *)(smem + y.rate), *slo = (T *)(smem + y.lo);
  T *sSL = (T *)(smem + y.SL);
  Level<T> *ste = (Level<T> *)(smem + y.te);
  T *sup = (T *)(smem + y.up);
  Batch<T> *sbt = (Batch<T> *)(smem + y.bt);
  const T *sbits = (const T *)(smem + y.bits);
  int8_t *sflag = (int8_t *)(smem + y.sflag);
  const int KR = level_row_len(K);
  const bool fuse_div = !FROM_TABLES && N + KR <= WAVE;


  // Which partition points have any feasible candidate: the test at the top
  // GPU level and the smallest admissible batch (same operations as below;
  // the fused solve has run it during its preparation).
  if (!flags_ready) {
    for (int s = lane; s < s_end; s += WAVE) {
      int ok = 0;
      if (blo <= N) {
        const T tK1 = sC[s] / sf[K - 1];
        const T upl = upload_time<T, FROM_TABLES>(p, tab, inst, sbits, srate, spi, s, blo - 1);
        const T Phi = (sA[s] + sB[s] * T(blo)) * sr[J - 1];
        const T H = slo[blo] - Phi;
        ok = (H >= tfree) && (tK1 <= H - upl);
      }
      sflag[s] = ok;
    }
    __syncthreads();
  }

  // lane -> (j, b) inside a pass: j = j_low + jl fastest, nb batch sizes per
  // pass.  Lanes beyond nb*Jw (Jn not dividing 64) stay idle.
  const int Jn = J - j_low;  // GPU levels searched
  const int Jw = Jn < WAVE ? Jn : WAVE;
  const int nb = WAVE / Jw;
  const int jl = lane % Jw, bo = lane / Jw;
  // Lanes past the pass's (j, b) pairs (bo == nb) hold no candidate: their
  // GPU level counts as absent, so they are never feasible, whatever record
  // b0 + bo (at most N + nb, inside the sentinel-padded rows) they read.
  const bool idle = bo >= nb;
  // Within a partition point a lane meets its candidates in increasing b,
  // i.e. decreasing flat index, when one chunk of GPU levels covers J; then
  // "<=" keeps the lowest index among equal energies.
  const bool one_chunk = ONE_CHUNK;
  const int j1 = j_low + jl;           // this lane's GPU level when one_chunk
  const T rj1 = sr[j1], pj1 = sP[j1];
  const uint64_t jokm = __builtin_amdgcn_ballot_w64(!idle);  // lanes holding a candidate

  // batch records past N are infeasible sentinels (lo = -inf)
  for (int q = lane; q < batch_sentinels(Jn, GREEDY); q += WAVE) {
    Batch<T> z;
    z.lo = -inf_of<T>();
    z.upl = T(0);
    z.esl = T(0);
    z.ab = T(0);
    sbt[N + 1 + q] = z;
  }


  // Eq. (20) per offloader: the budget shrinks along pi, so a lane's level
  // only moves up.  The CPU part of Eq. (21) is summed by runs of equal
  // level: count * e[k] is added when a lane leaves level k.  A lane whose
  // budget is +inf (infeasible, or past its batch) never moves.
#define JDOB_USER(X, I)                                        \
  {                                                            \
    const T x = (X);                                           \
    bool mv = tk > x;                                          \
    if (__ballot(mv)) { /* rare: some lane moves up */         \
      const T ecur = lv->e;                                    \
      acc = mv ? fma_(T((I) - run), ecur, acc) : acc;          \
      run = mv ? (I) : run;                                    \
      do {                                                     \
        lv += mv ? 1 : 0;                                      \
        tk = lv->t;                                            \
        mv = tk > x;                                           \
      } while (__ballot(mv));                                  \
    }                                                          \
  }
// user 0 opens the first run: nothing to add when it moves up
#define JDOB_USER0(X)                                          \
  {                                                            \
    const T x = (X);                                           \
    bool mv = tk > x;                                          \
    while (__ballot(mv)) {                                     \
      lv += mv ? 1 : 0;                                        \
      tk = lv->t;                                              \
      mv = tk > x;                                             \
    }                                                          \
  }

  // Row s into (up_, bt_, te_): Eq. (1), (2) per level (-inf sentinels past
  // the last level stop the level searches), Eq. (3) per user, and per batch size b the
  // record {lo[b], up[b-1], EU[b] + SL[b], A[s] + B[s]*b} read by one
  // instruction.  When users and levels fit one wave together, one division
  // serves both rows: lanes [0, N) divide bits by rate, lanes [N, N+K)
  // cycles by f.
  auto build_row = [&](int s, T *up_, Batch<T> *bt_, Level<T> *te_) {
    const T Cs = uni(sC[s]), As = uni(sA[s]), Bs = uni(sB[s]);
    T u1 = T(0);
    if (fuse_div) {
      const int k = lane - N;
      const bool isk = k >= 0 && k < K;
      const T num = lane < N ? sbits[s] : Cs;
      const T den = lane < N ? srate[lane] : (isk ? sf[k] : T(1));
      const T q = num / den;
      u1 = q;
      if (isk) {
        te_[k].t = q;
        te_[k].e = seps[k] * Cs;
      } else if (k >= K && k < KR) {
        te_[k].t = -inf_of<T>();
        te_[k].e = T(0);
      }
    } else {
      for (int k = lane; k < KR; k += WAVE) {
        te_[k].t = (k < K) ? Cs / sf[k] : -inf_of<T>();
        te_[k].e = (k < K) ? seps[k] * Cs : T(0);
      }
    }
    T carry = T(0);
    for (int i0 = 0; i0 < N; i0 += WAVE) {
      const int i = i0 + lane;
      T u = (i < N) ? (fuse_div ? u1 : upload_time<T, FROM_TABLES>(p, tab, inst, sbits, srate, spi, s, i))
                    : T(0);
      const T v = scan_add((i < N) ? p.ptx * u : T(0)) + carry;  // EU[i+1]
      if (i < N) {
        up_[i] = u;
        Batch<T> r;
        r.lo = slo[i + 1];
        r.upl = u;
        r.esl = v + sSL[i + 1];
        r.ab = As + Bs * T(i + 1);
        bt_[i + 1] = r;
      }
      carry = lane_read(v, WAVE - 1);
    }
  };

  // Alg. 2 at GPU level j (one per lane) of partition point s, whose rows
  // are up_, bt_ and te_; the two halves of the wave may hold two partition
  // points.  The greedy set at level j is pi[0..bg-1], bg the largest b
  // whose last (largest-gamma) user meets (7) at the top CPU level, i.e.
  // g_j at or above that user's threshold (Eq. (18)).  The test only fails
  // more as b grows, so bg is found by binary search over b, and bg grows
  // with j.
  const int top = 1 << (31 - __clz(N));
  auto greedy_at = [&](int s, int j, bool jok, const T *up_, const Batch<T> *bt_,
                       const Level<T> *te_, T &bE, int &bI) {
    const T tK1 = te_[K - 1].t;
    const T rj = sr[jok ? j : J - 1];
    int bg = 0;
    for (int step = top; step > 0; step >>= 1) {
      const int c = bg + step;
      const Batch<T> rc = bt_[c <= N ? c : N + 1];  // past N: sentinel, fails
      const T Hc = rc.lo - rc.ab * rj;
      bg = (tK1 <= Hc - rc.upl) ? c : bg;
    }
    // the kept set is a candidate if (6) holds and nobody left behind
    // misses its deadline locally (8)
    const Batch<T> r = bt_[bg > 0 ? bg : N + 1];
    const T Phi = r.ab * rj;  // Eq. (5), layers s+1..L
    const T H = r.lo - Phi;
    const bool feas = jok & (bg >= blo) & (H >= tfree);
    const uint64_t mask = __builtin_amdgcn_ballot_w64(feas);
    if (mask == 0) return;
    const int b = bg;
    // per half of the wave the highest feasible lane has the largest batch
    // and the lowest the smallest
    const uint64_t mlo = mask & 0xffffffffull, mhi = mask & ~0xffffffffull;
    int bw = 0;
    if (mhi) bw = __builtin_amdgcn_readlane(b, 63 - __clzll((long long)mhi));
    if (mlo) {
      const int w = __builtin_amdgcn_readlane(b, 63 - __clzll((long long)mlo));
      bw = w > bw ? w : bw;
    }
    const T Hu = feas ? H : inf_of<T>();
    T E;
    if constexpr (CONT) {
      // continuous CPU frequency: kappa * C[s] and the frequency range
      int ball = N;
      if (mlo) ball = __builtin_amdgcn_readlane(b, __builtin_ctzll(mlo));
      if (mhi) {
        const int w = __builtin_amdgcn_readlane(b, __builtin_ctzll(mhi));
        ball = w < ball ? w : ball;
      }
      const T Cs = sC[s], kC = p.kappa * Cs;
      const T f2 = (Cs > T(0)) ? cont_sum_f2(up_, Hu, b, ball, bw, Cs, sf[0], sf[K - 1]) : T(0);
      E = fma_(sP[jok ? j : J - 1], Phi, fma_(kC, f2, r.esl));
    } else {
      const Level<T> *lv = te_;
      T tk = lv->t;
      T acc = T(0);
      int run = 0;
      // users in groups of four per broadcast read, the next group read
      // ahead (the padded row covers it); users at or past a lane's batch
      // get an infinite budget
      {
        const Quad<T> c = *(const Quad<T> *)(up_);
        JDOB_USER0(Hu - c.v[0]);
        JDOB_USER((1 < b) ? Hu - c.v[1] : inf_of<T>(), 1);
        JDOB_USER((2 < b) ? Hu - c.v[2] : inf_of<T>(), 2);
        JDOB_USER((3 < b) ? Hu - c.v[3] : inf_of<T>(), 3);
      }
      int g = 4;
      for (; g + 4 < bw; g += 8) {  // two quads per trip, both read up front
        const Quad<T> c0 = *(const Quad<T> *)(up_ + g);
        const Quad<T> c1 = *(const Quad<T> *)(up_ + g + 4);
        JDOB_USER((g < b) ? Hu - c0.v[0] : inf_of<T>(), g);
        JDOB_USER((g + 1 < b) ? Hu - c0.v[1] : inf_of<T>(), g + 1);
        JDOB_USER((g + 2 < b) ? Hu - c0.v[2] : inf_of<T>(), g + 2);
        JDOB_USER((g + 3 < b) ? Hu - c0.v[3] : inf_of<T>(), g + 3);
        JDOB_USER((g + 4 < b) ? Hu - c1.v[0] : inf_of<T>(), g + 4);
        JDOB_USER((g + 5 < b) ? Hu - c1.v[1] : inf_of<T>(), g + 5);
        JDOB_USER((g + 6 < b) ? Hu - c1.v[2] : inf_of<T>(), g + 6);
        JDOB_USER((g + 7 < b) ? Hu - c1.v[3] : inf_of<T>(), g + 7);
      }
      if (g < bw) {
        const Quad<T> c = *(const Quad<T> *)(up_ + g);
        JDOB_USER((g < b) ? Hu - c.v[0] : inf_of<T>(), g);
        JDOB_USER((g + 1 < b) ? Hu - c.v[1] : inf_of<T>(), g + 1);
        JDOB_USER((g + 2 < b) ? Hu - c.v[2] : inf_of<T>(), g + 2);
        JDOB_USER((g + 3 < b) ? Hu - c.v[3] : inf_of<T>(), g + 3);
      }
      acc = fma_(T(b - run), lv->e, acc);
      E = fma_(sP[jok ? j : J - 1], Phi, acc + r.esl);
    }
    const int idx = s * J * N + (J - 1 - j) * N + (N - b);
    const bool take = feas & better(E, idx, bE, bI);
    bE = take ? E : bE;
    bI = take ? idx : bI;
    if (COUNT) {
      nfeas += feas ? 1 : 0;
      nevals += feas ? b : 0;
    }
  };

  if constexpr (GREEDY && !CONT) {
    // Alg. 2 needs one lane per GPU level.  When the searched levels fit half
    // a wave, lanes [0, 32) take one flagged partition point and lanes
    // [32, 64) the next, the second set of rows in the room of the batch
    // sentinels (this family reads no record past N + 1, so the sentinel at
    // N + 1 of both sets is all it needs).
    const int half = WAVE / 2;
    if (Jn <= half && 8 * (N + 2) + ((N + 3) & ~3) + 8 + 2 * KR <= 4 * (N + 2 + WAVE)) {
      Batch<T> *bt2 = sbt + N + 2;  // its record N + 1 is sentinel N + 1 + (N + 2) <= N + 65
      T *up2 = (T *)(bt2 + N + 2);
      Level<T> *te2 = (Level<T> *)(up2 + ((N + 3) & ~3) + 8);
      const bool hi = lane >= half;
      const int j = j_low + lane - (hi ? half : 0);
      int s = 0;
      while (s < s_end && !uni(sflag[s])) ++s;
      while (s < s_end) {
        int s2 = s + 1;
        while (s2 < s_end && !uni(sflag[s2])) ++s2;
        build_row(s, sup, sbt, ste);
        if (s2 < s_end) build_row(s2, up2, bt2, te2);
        __syncthreads();
        T bE = inf_of<T>();
        int bI = 0x7fffffff;
        const bool jok = j < J && (!hi || s2 < s_end);
        greedy_at(hi ? s2 : s, j, jok, hi ? up2 : sup, hi ? bt2 : sbt, hi ? te2 : ste, bE, bI);
        // each lane meets its partition points in increasing order
        if (bE < bestE) { bestE = bE; bestI = bI; }
        __syncthreads();
        s = s2 + 1;
        while (s < s_end && !uni(sflag[s])) ++s;
      }
      return;
    }
  }

  for (int s = 0; s < s_end; ++s) {
    if (!uni(sflag[s])) continue;
    build_row(s, sup, sbt, ste);
    __syncthreads();
    const T Cs = uni(sC[s]);
    const T tK1 = uni(ste[K - 1].t);
    const int sJN = s * J * N;
    // continuous CPU frequency: kappa * C[s] and the frequency range
    const T kC = CONT ? p.kappa * Cs : T(0);
    const T fmin = CONT ? uni(sf[0]) : T(0), fmax = CONT ? uni(sf[K - 1]) : T(0);

    T bE = inf_of<T>();  // best of this lane within partition point s
    int bI = 0x7fffffff;
    if constexpr (GREEDY) {
      // Alg. 2 at every searched GPU level of partition point s, lane = j
      for (int jc = j_low; jc < J; jc += WAVE)
        greedy_at(s, jc + lane, jc + lane < J, sup, sbt, ste, bE, bI);
    } else {
    // Level of the first offloader of each lane's batch, carried across
    // passes: with one chunk a lane keeps its GPU level j and meets its
    // batches in increasing b, and the budget H - up[0] only shrinks as b
    // grows (H falls).
    const Level<T> *p0 = ste;
    Level<T> q0 = ste[0];  // (t, e) at p0
    const T up0 = uni(sup[0]);
    int K2 = 1;
    while (K2 < K) K2 <<= 1;
    // Candidates whose offloaders span several levels wait in the queue;
    // qE, qI is the best of those evaluated (flat indices).
    uint32_t *sq = (uint32_t *)(smem + (QUEUE ? y.q : 0));
    int qhead = 0, qtail = 0;
    T qE = inf_of<T>();
    int qI = 0x7fffffff;
    // Evaluates the first cnt (<= 64) queued candidates, one per lane: the
    // CPU part of Eq. (21) by runs of equal level from the first offloader's
    // level up; the end of the run at level k is the first user with
    // t[k] > H - up[i], found by binary search over the upload row (a level
    // that fits the last offloader ends the batch).  The same operations as
    // the pass give the same budgets.
    auto flush = [&](int cnt) {
      const bool act = lane < cnt;
      const uint32_t e = sq[(qhead + (act ? lane : 0)) & (QCAP - 1)];
      const int b = act ? (int)(e & 2047u) : 0;
      const int j = (int)((e >> 11) & 255u);
      const Level<T> *lv = ste + (e >> 19);
      const Batch<T> r = sbt[act ? b : N + 1];
      const T Phi = r.ab * sr[j];
      const T H = r.lo - Phi;
      const T hl = H - r.upl;
      T tk = lv->t;
      T acc = T(0);
      int run = 0;  // first user of the current run
      while (__builtin_amdgcn_ballot_w64(run < b)) {
        const bool a = run < b;
        int l = run, h = b;  // user l fits level tk; the run ends in (l, h]
        if (a && !(tk > hl)) l = h - 1;
        while (__builtin_amdgcn_ballot_w64(h - l > 1)) {
          const bool open = h - l > 1;
          const int mid = (l + h) >> 1;
          const bool miss = tk > H - sup[open ? mid : l];
          h = (open && miss) ? mid : h;
          l = (open && !miss) ? mid : l;
        }
        if (a) acc = fma_(T(h - run), lv->e, acc);
        run = a ? h : run;
        // the level of the next run's first user
        const T x = (run < b) ? H - sup[run < b ? run : 0] : inf_of<T>();
        bool mv = tk > x;
        while (__builtin_amdgcn_ballot_w64(mv)) {
          lv += mv ? 1 : 0;
          tk = lv->t;
          mv = tk > x;
        }
      }
      const T E = fma_(sP[j], Phi, acc + r.esl);
      const int idx = sJN + (J - 1 - j) * N + (N - b);
      const bool take = act && better(E, idx, qE, qI);
      qE = take ? E : qE;
      qI = take ? idx : qI;
      qhead += cnt;
    };
    for (int b0 = blo; b0 <= N; b0 += nb) {
      bool any = false;
      for (int jc = 0; jc < (ONE_CHUNK ? WAVE : Jn); jc += WAVE) {
        const int j = j_low + jc + jl;
        const bool jok = one_chunk ? !idle : j < J;
        const T rj = one_chunk ? rj1 : sr[jok ? j : 0];
        const Batch<T> r = sbt[b0 + bo];
        const T Phi = r.ab * rj;                              // Eq. (5), layers s+1..L
        const T H = r.lo - Phi;                               // slack to the batch deadline
        const T hl = H - r.upl;                               // budget of the last offloader
        const bool c6 = H >= tfree, c7 = tK1 <= hl;
        const bool feas = jok & c6 & c7;                      // (6), (7); (8): b >= bmin
        const uint64_t mask = __builtin_amdgcn_ballot_w64(c6) & __builtin_amdgcn_ballot_w64(c7) &
                              (one_chunk ? jokm : __builtin_amdgcn_ballot_w64(jok));
        if (mask == 0) continue;
        any = true;
        const int b = b0 + bo;
        T E;
        bool multi = false;  // queued: evaluated by flush
        if constexpr (CONT) {
          const int hi = 63 - __clzll((long long)mask);
          const int bpass = b0 + __builtin_amdgcn_readlane(bo, hi);  // largest feasible b
          const T Hu = feas ? H : inf_of<T>();
          const T f2 = (Cs > T(0)) ? cont_sum_f2(sup, Hu, b, b0, bpass, Cs, fmin, fmax) : T(0);
          E = fma_(one_chunk ? pj1 : sP[jok ? j : 0], Phi, fma_(kC, f2, r.esl));
        } else {
          // Eq. (20) for the first offloader: the number of levels too slow
          // for its budget (latency falls with the level), by steps up from
          // the level of the lane's previous pass with one chunk (a binary
          // search on the first pass measured slower), else by binary search
          // (an infeasible lane's budget is +inf: level 0, no steps)
          const T x0 = (feas ? H : inf_of<T>()) - up0;
          if (!one_chunk) {
            const Level<T> *c0 = ste - 1;  // one before the first level that fits
            for (int step = K2 >> 1; step > 0; step >>= 1)
              c0 += (c0[step].t > x0) ? step : 0;
            p0 = c0 + 1;
            q0 = *p0;
          } else {
            bool mv = q0.t > x0;
            if (__builtin_amdgcn_ballot_w64(mv)) {
              do {
                p0 += mv ? 1 : 0;
                q0 = *p0;
                mv = q0.t > x0;
              } while (__builtin_amdgcn_ballot_w64(mv));
            }
          }
          // When the last offloader fits the first one's level, every
          // offloader runs at it (the levels rise along pi): b of its energy.
          E = fma_(one_chunk ? pj1 : sP[jok ? j : 0], Phi, T(b) * q0.e + r.esl);
          const bool up_last = q0.t > hl;
          const uint64_t mm = mask & __builtin_amdgcn_ballot_w64(up_last);
          if (!QUEUE && mm) {
            // Otherwise, in short batches, the CPU part of Eq. (21) by runs
            // of equal level: a walk over the users, four per broadcast read
            // (user 0 is at level p0), until every such lane is at a level
            // that fits its last offloader.  Users below b0 belong to every
            // lane's batch; past a lane's batch the budget is +inf.  The
            // other lanes get an infinite budget and drop the result.
            const bool walk = feas & up_last;
            const T Hm = walk ? H : inf_of<T>();
            const T hm = walk ? hl : inf_of<T>();
            const int bw = b0 + __builtin_amdgcn_readlane(bo, 63 - __clzll((long long)mm));
            const Level<T> *lv = p0;
            T tk = q0.t;
            T acc = T(0);
            int run = 0;  // first user of the current level
            int g = 0;
            for (; g + 4 <= b0; g += 4) {
              if (!__builtin_amdgcn_ballot_w64(tk > hm)) break;
              const Quad<T> c = *(const Quad<T> *)(sup + g);
              JDOB_USER(Hm - c.v[0], g);
              JDOB_USER(Hm - c.v[1], g + 1);
              JDOB_USER(Hm - c.v[2], g + 2);
              JDOB_USER(Hm - c.v[3], g + 3);
            }
            for (; g < bw; ++g) {
              if (!__builtin_amdgcn_ballot_w64(tk > hm)) break;
              const T u = sup[g];
              const T Hg = (g < b) ? Hm : inf_of<T>();
              JDOB_USER(Hg - u, g);
            }
            acc = fma_(T(b - run), lv->e, acc);
            const T Ew = fma_(one_chunk ? pj1 : sP[jok ? j : 0], Phi, acc + r.esl);
            E = walk ? Ew : E;
          } else if (QUEUE && mm) {
            // the candidate joins the queue
            multi = feas & up_last;
            const int slot = qtail + (int)__builtin_amdgcn_mbcnt_hi(
                                         (uint32_t)(mm >> 32),
                                         __builtin_amdgcn_mbcnt_lo((uint32_t)mm, 0u));
            if (multi)
              sq[slot & (QCAP - 1)] =
                  (uint32_t)b | ((uint32_t)j << 11) | ((uint32_t)(p0 - ste) << 19);
            qtail += __builtin_popcountll(mm);
            if (qtail - qhead >= WAVE) flush(WAVE);  // (QUEUE only)
          }
        }
        if (one_chunk) {
          const bool take = feas & !(QUEUE && multi) & (E <= bE);
          bE = take ? E : bE;
          bI = take ? b : bI;
        } else {
          const int idx = sJN + (J - 1 - j) * N + (N - b);
          const bool take = feas & !(QUEUE && multi) & better(E, idx, bE, bI);
          bE = take ? E : bE;
          bI = take ? idx : bI;
        }
        if (COUNT) {
          nfeas += feas ? 1 : 0;
          nevals += feas ? b : 0;
        }
      }
      if (!any) break;
    }
    if (QUEUE && qtail > qhead) flush(qtail - qhead);
    if (one_chunk && bI != 0x7fffffff) bI = sJN + (J - 1 - j1) * N + (N - bI);
    if (QUEUE && better(qE, qI, bE, bI)) { bE = qE; bI = qI; }
    }
    // later partition points have higher flat indices: strict "<" merges
    if (bE < bestE) { bestE = bE; bestI = bI; }
    __syncthreads();
  }
#undef JDOB_USER
#undef JDOB_USER0
}

// ONE_CHUNK: the GPU levels searched fit one wave, so one pass covers them
// and each lane keeps one level j for the whole instance.  COUNT: fill the
// optional work counters.  GREEDY: Alg. 2's family, one batch per (s, j) with
// lane = j; otherwise every batch, lanes = (j, b).
// Eight waves per SIMD (the maximum): the level loop waits on LDS often and
// needs every resident wave to hide it; the register budget is sized to fit.
template <typename T, bool FROM_TABLES, bool ONE_CHUNK, bool COUNT, bool GREEDY, bool CONT,
          bool QUEUE>
__global__ __launch_bounds__(WAVE, 8) void jdob_solve_kernel(SolveArgs<T> args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x;
  const Problem<T> p = own_problem(args.p);
  const Tables<T> &tab = args.tab;
  const int64_t inst = instance_of_block(args.first);
  const int N = p.N, L = p.L, K = p.K, J = p.J;
  const Layout y = make_layout(N, L, K, J, (int)sizeof(T), CONT, QUEUE,
                               batch_sentinels(J - p.j_low, GREEDY));

  const T tfree = p.tfree ? p.tfree[inst] : T(0);
  int bmin;
  bool any = true;  // some partition point may have a feasible candidate
  if (FROM_TABLES)
    prepare_instance<T, FROM_TABLES, CONT>(p, tab, inst, smem, y, lane, bmin);
  else
    any = prepare_fused<T, CONT>(p, inst, smem, y, lane, tfree, bmin);

  T *sC = (T *)(smem + y.C), *sA = (T *)(smem + y.A), *sB = (T *)(smem + y.B);
  T *sf = (T *)(smem + y.f), *seps = (T *)(smem + y.eps);
  T *sr = (T *)(smem + y.r), *sP = (T *)(smem + y.P);
  int16_t *spi = (int16_t *)(smem + y.pi);
  T *srate = (T *)(smem + y.rate), *slo = (T *)(smem + y.lo);
  int8_t *skL = (int8_t *)(smem + y.kL);
  T *seL = (T *)(smem + y.eL), *sSL = (T *)(smem + y.SL);
  Level<T> *ste = (Level<T> *)(smem + y.te);
  T *sterm = (T *)(smem + y.term);

  const int blo = uni(bmin > 1 ? bmin : 1);  // smallest admissible batch
  T bestE = inf_of<T>();
  int bestI = 0x7fffffff;
  int nfeas = 0, nevals = 0;  // per lane
  if (any)
    search_candidates<T, FROM_TABLES, ONE_CHUNK, COUNT, GREEDY, CONT, QUEUE>(
        p, tab, inst, smem, y, lane, N, blo, tfree, bestE, bestI, nfeas, nevals, !FROM_TABLES);

  // local computing competes last
  const int idxLC = L * J * N;
  wave_argmin(bestE, bestI);
  if (bmin == 0) {
    nfeas += (lane == 0) ? 1 : 0;
    if (better(sSL[0], idxLC, bestE, bestI)) { bestE = sSL[0]; bestI = idxLC; }
  }
  const int64_t totfeas = wave_sum_i64((int64_t)nfeas);
  const int64_t totev = wave_sum_i64((int64_t)nevals);

  const Policy<T> out = output_pointers<T>();
  int8_t *ul = out.ulevel + inst * N;
  int8_t *uo = out.uoffload + inst * N;
  if (lane == 0) {
    if (out.nfeas) out.nfeas[inst] = (int32_t)totfeas;
    if (out.nevals) out.nevals[inst] = totev;
  }
  if (bestI == 0x7fffffff) {  // nothing feasible
    if (lane == 0) {
      out.status[inst] = 1;
      out.cut[inst] = -1;
      out.gpu_level[inst] = -1;
      out.batch[inst] = 0;
      out.energy[inst] = inf_of<T>();
      out.tfree_out[inst] = inf_of<T>();
    }
    for (int m = lane; m < N; m += WAVE) {
      ul[m] = -1;
      uo[m] = 0;
    }
    if (T *uf = freq_row<T>(inst, N))
      for (int m = lane; m < N; m += WAVE) uf[m] = T(0);
    return;
  }

  if (bestI == idxLC) {
    for (int m = lane; m < N; m += WAVE) {
      ul[m] = (int8_t)(CONT ? -1 : skL[m]);
      uo[m] = 0;
    }
    if (T *uf = freq_row<T>(inst, N))
      for (int m = lane; m < N; m += WAVE) uf[m] = local_freq<T, CONT>(smem, y, m);
    if (lane == 0) {
      T acc = T(0);
      for (int m = 0; m < N; ++m) acc = acc + seL[m];
      out.status[inst] = 0;
      out.cut[inst] = L;
      out.gpu_level[inst] = -1;
      out.batch[inst] = 0;
      out.energy[inst] = acc;
      out.tfree_out[inst] = tfree;
    }
    return;
  }

  // the winner (s*, j*, b*): per-user levels, canonical energy, Eq. (22)
  const T *sbits = (const T *)(smem + y.bits);
  const int s = bestI / (J * N);
  const int rem = bestI - s * (J * N);
  const int j = J - 1 - rem / N;
  const int b = N - (rem - (rem / N) * N);
  const T Cs = sC[s];
  for (int k = lane; k < K; k += WAVE) {
    ste[k].t = Cs / sf[k];
    ste[k].e = seps[k] * Cs;
  }
  __syncthreads();
  const T Phi = (sA[s] + sB[s] * T(b)) * sr[j];
  const T H = slo[b] - Phi;
  T ready = tfree;
  T *sfq = (T *)(smem + y.up);  // frequency by user (the upload row is free now)
  for (int i = lane; i < N; i += WAVE) {
    const int m = spi[i];
    if (i < b) {
      const T u = upload_time<T, FROM_TABLES>(p, tab, inst, sbits, srate, spi, s, i);
      int lv;
      T fq, e, tl;
      offloader_choice<T, CONT>(p, ste, sf, Cs, H - u, lv, fq, e, tl);
      ul[m] = (int8_t)lv;
      uo[m] = 1;
      sfq[m] = fq;
      sterm[m] = e + p.ptx * u;
      const T done = tl + u;
      ready = (done > ready) ? done : ready;
    } else {
      ul[m] = (int8_t)(CONT ? -1 : skL[m]);
      uo[m] = 0;
      sfq[m] = local_freq<T, CONT>(smem, y, m);
      sterm[m] = seL[m];
    }
  }
  ready = wave_max(ready);
  __syncthreads();
  if (T *uf = freq_row<T>(inst, N))
    for (int m = lane; m < N; m += WAVE) uf[m] = sfq[m];
  if (lane == 0) {
    T acc = T(0);
    for (int m = 0; m < N; ++m) acc = acc + sterm[m];
    acc = acc + sP[j] * Phi;
    out.status[inst] = 0;
    out.cut[inst] = s;
    out.gpu_level[inst] = j;
    out.batch[inst] = b;
    out.energy[inst] = acc;
    out.tfree_out[inst] = ready + Phi;
  }
}

// ------------------------------------------------------------ outer grouping

template <typename T> __device__ inline Grouped<T> grouped_pointers() {
  const auto *a = (const __attribute__((address_space(4))) GroupedArgs<T> *)
      __builtin_amdgcn_kernarg_segment_ptr();
  Grouped<T> o;
  o.status = a->out.status;
  o.num_groups = a->out.num_groups;
  o.energy = a->out.energy;
  o.tfree_out = a->out.tfree_out;
  o.order = a->out.order;
  o.group_end = a->out.group_end;
  o.group_cut = a->out.group_cut;
  o.group_gpu_level = a->out.group_gpu_level;
  o.group_batch = a->out.group_batch;
  o.group_energy = a->out.group_energy;
  o.group_tfree = a->out.group_tfree;
  o.ulevel = a->out.ulevel;
  o.uoffload = a->out.uoffload;
  o.ugroup = a->out.ugroup;
  o.ninner = a->out.ninner;
  o.nfeas = a->out.nfeas;
  o.nevals = a->out.nevals;
  o.ufreq = a->out.ufreq;
  return o;
}

// The group ord[j..i-1] as the user set of search_candidates: its members
// in the instance's rate order (pi, rate), its batch deadlines lo (Eq. (10))
// and its suffix sums SL of local energies.  Returns the group's bmin.
// One lane per user of the instance (N <= 64).
template <typename T>
__device__ inline int group_setup(unsigned char *smem, const Layout &y, const GLayout &gy, int N,
                                  int j, int i, int lane) {
  int16_t *spi = (int16_t *)(smem + y.pi);
  T *srate = (T *)(smem + y.rate), *slo = (T *)(smem + y.lo), *sdl = (T *)(smem + y.dl);
  const int8_t *skL = (const int8_t *)(smem + y.kL);
  const T *seL = (const T *)(smem + y.eL);
  T *sSL = (T *)(smem + y.SL);
  const int *pia = (const int *)(smem + gy.pi_all);
  const T *ra = (const T *)(smem + gy.rate_all);
  const int *dr = (const int *)(smem + gy.drank);
  __syncthreads();  // the previous group's rows are no longer read
  // (the lane's LDS addresses are formed here, not kept across the
  // grouping's loops, where the registers are short)
  int ln = lane;
  asm volatile("" : "+v"(ln));
  // keep the members of the instance's rate order, in that order
  const int m = ln < N ? pia[ln] : 0;
  const bool mem = ln < N && dr[m] >= j && dr[m] < i;
  const uint64_t mask = __builtin_amdgcn_ballot_w64(mem);
  const int pos = __builtin_amdgcn_mbcnt_hi((unsigned)(mask >> 32),
                                            __builtin_amdgcn_mbcnt_lo((unsigned)mask, 0u));
  if (mem) {
    spi[pos] = m;
    srate[pos] = ra[ln];
  }
  const int g = i - j;
  __syncthreads();
  const T d = ln < g ? sdl[spi[ln]] : inf_of<T>();
  const T v = wave_scan<T, true>(d, lane);
  if (ln < g) slo[ln + 1] = v;
  if (ln == 0) slo[0] = inf_of<T>();
  const uint64_t nl = __builtin_amdgcn_ballot_w64(ln < g && skL[spi[ln < g ? ln : 0]] < 0);
  const int bm = nl ? 64 - __clzll((long long)nl) : 0;
  // SL[r] = sum of eL over the group's pi positions r..g-1 (ranking only)
  const int r = g - 1 - ln;
  T e = r >= 0 ? seL[spi[r]] : T(0);
  e = wave_scan<T, false>(e, lane);
  if (r >= 0) sSL[r] = e;
  if (ln == 0) sSL[g] = T(0);
  __syncthreads();
  return bm;
}

// The winner (flat index idx over the group's candidates; local computing
// is L*J*g) of the group ord[j..i-1] set up in LDS: its energy summed as for
// an instance of its own (members in user index order, Eq. (21), then the
// GPU term) and its release time (Eq. (22)); with `out` set, each member's
// level (or frequency), offload flag and group number gno.  Optionally its
// slack H = lo[b] - Phi (+inf for local computing), the latest time an
// offloader is ready (-inf for local computing) and Phi (0), from which the
// release after any other GPU free time t follows: max(t, ready) + Phi.
template <typename T, bool CONT>
__device__ inline void group_winner(const Problem<T> &p, int64_t inst, unsigned char *smem,
                                    const Layout &y, const GLayout &gy, int N, int j, int i,
                                    int idx, T tfree, int lane, T &E, T &tf, const Grouped<T> *out,
                                    int gno, T *slack = nullptr, T *rdy = nullptr,
                                    T *phi = nullptr) {
  const int L = p.L, K = p.K, J = p.J, g = i - j;
  const T *sC = (const T *)(smem + y.C), *sA = (const T *)(smem + y.A);
  const T *sB = (const T *)(smem + y.B), *sf = (const T *)(smem + y.f);
  const T *seps = (const T *)(smem + y.eps), *sr = (const T *)(smem + y.r);
  const T *sP = (const T *)(smem + y.P);
  const int16_t *spi = (const int16_t *)(smem + y.pi);
  const T *srate = (const T *)(smem + y.rate), *slo = (const T *)(smem + y.lo);
  const int8_t *skL = (const int8_t *)(smem + y.kL);
  const T *seL = (const T *)(smem + y.eL);
  Level<T> *ste = (Level<T> *)(smem + y.te);
  T *sterm = (T *)(smem + y.term);
  const int *dr = (const int *)(smem + gy.drank);
  const size_t o = (size_t)inst * N;
  T acc = T(0), gpu = T(0), ready = tfree;
  if (idx == L * J * g) {  // local computing
    for (int m = lane; m < N; m += WAVE) {
      if (dr[m] < j || dr[m] >= i) continue;
      sterm[m] = seL[m];
      if (out) {
        out->ulevel[o + m] = (int8_t)(CONT ? -1 : skL[m]);
        out->uoffload[o + m] = 0;
        out->ugroup[o + m] = (int8_t)gno;
        if (out->ufreq) out->ufreq[o + m] = local_freq<T, CONT>(smem, y, m);
      }
    }
    __syncthreads();
    if (lane == 0)
      for (int m = 0; m < N; ++m)
        if (dr[m] >= j && dr[m] < i) acc = acc + sterm[m];
    E = lane_read(acc, 0);
    tf = tfree;
    if (slack) *slack = inf_of<T>();
    if (rdy) *rdy = -inf_of<T>();
    if (phi) *phi = T(0);
    __syncthreads();
    return;
  }
  const T *sbits = (const T *)(smem + y.bits);
  const int s = idx / (J * g);
  const int rem = idx - s * (J * g);
  const int jg = J - 1 - rem / g;
  const int b = g - (rem - (rem / g) * g);
  const T Cs = sC[s];
  for (int k = lane; k < K; k += WAVE) {
    ste[k].t = Cs / sf[k];
    ste[k].e = seps[k] * Cs;
  }
  __syncthreads();
  const T Phi = (sA[s] + sB[s] * T(b)) * sr[jg];
  const T H = slo[b] - Phi;
  ready = -inf_of<T>();  // the latest offloader, the GPU free time joins below
  for (int q = lane; q < g; q += WAVE) {
    const int m = spi[q];
    int lv;
    int8_t off;
    T fq;
    if (q < b) {
      const T u = sbits[s] / srate[q];
      T e, tl;
      offloader_choice<T, CONT>(p, ste, sf, Cs, H - u, lv, fq, e, tl);
      sterm[m] = e + p.ptx * u;
      const T done = tl + u;
      ready = (done > ready) ? done : ready;
      off = 1;
    } else {
      sterm[m] = seL[m];
      lv = CONT ? -1 : skL[m];
      fq = local_freq<T, CONT>(smem, y, m);
      off = 0;
    }
    if (out) {
      out->ulevel[o + m] = (int8_t)lv;
      out->uoffload[o + m] = off;
      out->ugroup[o + m] = (int8_t)gno;
      if (out->ufreq) out->ufreq[o + m] = fq;
    }
  }
  ready = wave_max(ready);
  __syncthreads();
  if (lane == 0) {
    for (int m = 0; m < N; ++m)
      if (dr[m] >= j && dr[m] < i) acc = acc + sterm[m];
    gpu = acc + sP[jg] * Phi;
  }
  E = lane_read(gpu, 0);
  tf = ((tfree > ready) ? tfree : ready) + Phi;
  if (slack) *slack = H;
  if (rdy) *rdy = ready;
  if (phi) *phi = Phi;
  __syncthreads();
}

// Outer grouping: one wave per instance runs the dynamic program over the
// deadline order (a front of non-dominated (energy, release) states per
// prefix; for each group j..i-1, one inner solve, search_candidates on the
// group's users, per run of prefix j's states that share a winner), then
// replays the chosen groups to write the policy.  Eight waves per SIMD: the
// program's state and the inner search want more than 64 registers, and
// fitting 64 spills a few values to scratch (outside the pass loops), but
// the short passes of small groups wait on LDS and barriers, and the extra
// resident waves hide that (measured: g10 22.5 ms at eight waves, 24.0 at
// seven, 25.9 at six; p5 16.0, 16.3, 17.1; only g20, with groups of up to
// 20 users, gains from fewer: 84.1, 82.9, 81.0).
template <typename T, bool ONE_CHUNK, bool COUNT, bool GREEDY, bool CONT>
__global__ __launch_bounds__(WAVE, 8) void jdob_grouped_kernel(GroupedArgs<T> args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x;
  const Problem<T> p = own_problem(args.p);
  const Tables<T> tab{};
  const int64_t inst = instance_of_block(args.first);
  const int N = p.N, L = p.L, K = p.K, J = p.J;
  const Layout y = make_layout(N, L, K, J, (int)sizeof(T), CONT, false,
                               batch_sentinels(J - p.j_low, GREEDY));
  const GLayout gy = make_glayout(y, N, (int)sizeof(T));

  int bmin_all;
  prepare_instance<T, false, CONT>(p, tab, inst, smem, y, lane, bmin_all);
  const int16_t *spi = (const int16_t *)(smem + y.pi);
  const T *srate = (const T *)(smem + y.rate), *sdl = (const T *)(smem + y.dl);
  const T *sSL = (const T *)(smem + y.SL);
  int *pia = (int *)(smem + gy.pi_all), *dr = (int *)(smem + gy.drank);
  int *dord = (int *)(smem + gy.dord), *fn = (int *)(smem + gy.fn);
  int *ends = (int *)(smem + gy.ends), *eks = (int *)(smem + gy.eks);
  T *ra = (T *)(smem + gy.rate_all), *fE = (T *)(smem + gy.fE), *fT = (T *)(smem + gy.fT);
  int16_t *from = (int16_t *)(smem + gy.from);
  constexpr int F = GROUP_FRONT;

  // the instance's rate order (left in pi by the preparation, with the
  // rates in that order) and deadline order (ties by lower index)
  if (lane < N) {
    pia[lane] = spi[lane];
    ra[lane] = srate[lane];
    const T Tm = sdl[lane];
    int r = 0;
    for (int q = 0; q < N; ++q) r += (sdl[q] < Tm || (sdl[q] == Tm && q < lane)) ? 1 : 0;
    dr[lane] = r;
    dord[r] = lane;
  }
  for (int i = lane; i <= N; i += WAVE) fn[i] = i == 0 ? 1 : 0;
  if (lane == 0) {  // the empty prefix: no energy, the GPU free at t_free
    fE[0] = T(0);
    fT[0] = p.tfree ? p.tfree[inst] : T(0);
    from[0] = -1;
  }
  __syncthreads();

  // The group's winner among its candidates and local computing: the flat
  // index (0x7fffffff if none is feasible), with the GPU free at tf0.
  // Counts into nf, ne when COUNT.
  auto group_search = [&](int g, int bmin, T tf0, int &nf, int &ne) -> int {
    T bestE = inf_of<T>();
    int bestI = 0x7fffffff;
    search_candidates<T, false, ONE_CHUNK, COUNT, GREEDY, CONT, false>(
        p, tab, inst, smem, y, lane, g, bmin > 1 ? bmin : 1, tf0, bestE, bestI, nf, ne);
    wave_argmin(bestE, bestI);
    if (bmin == 0) {  // local computing of the whole group competes last
      if (COUNT) nf += (lane == 0) ? 1 : 0;
      if (better(sSL[0], L * J * g, bestE, bestI)) { bestE = sSL[0]; bestI = L * J * g; }
    }
    return uni(bestI);
  };

  int nfeas = 0, nevals = 0, ninner = 0;
  for (int i = 1; i <= N; ++i) {
    int ni = 0;  // states in the front of prefix i
    for (int j = 0; j < i; ++j) {  // last group: ord[j..i-1]
      const int nj = uni(fn[j]);
      if (nj == 0) continue;
      const int g = i - j;
      const int bmin = uni(group_setup<T>(smem, y, gy, N, j, i, lane));  // wave-uniform
      // The states of prefix j from the earliest release (the front's last)
      // on.  A later GPU free time only removes candidates (constraint (6)),
      // so a winner whose slack meets a later state's free time is that
      // state's winner too: one inner solve serves the run of such states.
      int k = nj - 1;
      while (k >= 0) {
        const T tf0 = uni(fT[j * F + k]);
        const int idx = group_search(g, bmin, tf0, nfeas, nevals);
        ++ninner;
        if (idx == 0x7fffffff) break;  // the states left free the GPU later still
        T Eg, Tg, H, rd, Ph;
        group_winner<T, CONT>(p, inst, smem, y, gy, N, j, i, idx, tf0, lane, Eg, Tg, nullptr, 0,
                              &H, &rd, &Ph);
        Eg = uni(Eg);
        H = uni(H);
        rd = uni(rd);
        Ph = uni(Ph);
        T tk = tf0;
        do {
          const T Tk = ((tk > rd) ? tk : rd) + Ph;  // Eq. (22) after free time tk
          ni = front_add(fE + i * F, fT + i * F, from + i * F, ni, uni(fE[j * F + k]) + Eg, Tk,
                         j * F + k, lane);
          --k;
          tk = k >= 0 ? uni(fT[j * F + k]) : tk;
        } while (k >= 0 && H >= tk);
      }
    }
    if (lane == 0) fn[i] = ni;
    __syncthreads();
  }

  const Grouped<T> out = grouped_pointers<T>();
  const size_t o = (size_t)inst * N;
  for (int q = lane; q < N; q += WAVE) {
    out.order[o + q] = (int16_t)dord[q];
    out.group_end[o + q] = 0;
    out.group_cut[o + q] = -1;
    out.group_gpu_level[o + q] = -1;
    out.group_batch[o + q] = 0;
    out.group_energy[o + q] = inf_of<T>();
    out.group_tfree[o + q] = inf_of<T>();
    out.ulevel[o + q] = -1;
    out.uoffload[o + q] = 0;
    out.ugroup[o + q] = -1;
    if (out.ufreq) out.ufreq[o + q] = T(0);
  }
  const int64_t totfeas = wave_sum_i64((int64_t)nfeas);
  const int64_t totev = wave_sum_i64((int64_t)nevals);
  if (lane == 0) {
    if (out.ninner) out.ninner[inst] = ninner;
    if (out.nfeas) out.nfeas[inst] = totfeas;
    if (out.nevals) out.nevals[inst] = totev;
  }
  if (uni(fn[N]) == 0) {
    if (lane == 0) {
      out.status[inst] = 1;
      out.num_groups[inst] = 0;
      out.energy[inst] = inf_of<T>();
      out.tfree_out[inst] = inf_of<T>();
    }
    return;
  }
  // the lowest-energy state of the full order, back to the empty prefix;
  // its groups are then solved again in order to write the policy
  int G = 0;
  for (int st = N * F; st > 0; st = uni((int)from[st])) ++G;
  if (lane == 0) {
    int c = G;
    for (int st = N * F; st > 0; st = from[st]) {
      --c;
      ends[c] = st / F;
      eks[c] = st;
    }
  }
  __syncthreads();
  int a = 0;
  for (int gno = 0; gno < G; ++gno) {
    const int b = uni(ends[gno]), g = b - a;
    const T tf0 = uni(fT[from[uni(eks[gno])]]);
    const int bmin = uni(group_setup<T>(smem, y, gy, N, a, b, lane));
    int nf = 0, ne = 0;
    const int idx = group_search(g, bmin, tf0, nf, ne);
    T Eg, Tg;
    group_winner<T, CONT>(p, inst, smem, y, gy, N, a, b, idx, tf0, lane, Eg, Tg, &out, gno);
    if (lane == 0) {
      int s = L, jg = -1, bb = 0;
      if (idx != L * J * g) {
        s = idx / (J * g);
        const int rem = idx - s * (J * g);
        jg = J - 1 - rem / g;
        bb = g - (rem - (rem / g) * g);
      }
      out.group_end[o + gno] = (int16_t)b;
      out.group_cut[o + gno] = s;
      out.group_gpu_level[o + gno] = jg;
      out.group_batch[o + gno] = bb;
      out.group_energy[o + gno] = Eg;
      out.group_tfree[o + gno] = Tg;
    }
    a = b;
  }
  if (lane == 0) {
    out.status[inst] = 0;
    out.num_groups[inst] = G;
    out.energy[inst] = fE[N * F];
    out.tfree_out[inst] = fT[N * F];
  }
}

// Stage 1: per-user option tables of every partition point.
//
// The kernel is bound by the HBM writes of its tables ((L+1)*N entries of
// four P-typed tables and one int8 table per instance), so it keeps the
// per-instance work to what the tables need and writes wide:
//   * preparation: the instance's layer cycles, output bits, rates and
//     deadlines; the sequential cycle sums C (Sec. III, in the pinned order);
//     the rate order pi, the batch deadlines lo[b] (Eq. (10)) and bmin
//     (constraint (8): a user has a local level exactly when the top level
//     finishes the whole chain by its deadline);
//   * the CPU level rows (latency and energy per level, Eqs. (1), (2)) of a
//     run of partition points, padded to a power of two with levels that
//     always fit (latency -inf) and are never chosen;
//   * the table pass: an instance's (s, user) entries are contiguous in every
//     table, and each lane takes four consecutive ones per pass (VEC: one
//     16-byte store per P-typed table and one 4-byte store of the four
//     levels, non-temporal: nothing reads the tables back in this launch;
//     otherwise four element stores).  A user's lowest level within
//     its budget is found by binary search over the row, since latency falls
//     as the frequency rises.
// One wave takes one instance; on long launches whose instance rows are all
// resident, a workgroup of two waves takes two consecutive instances and
// stores their entries as one span (jdob_tables_group_kernel).
struct TLayout {
  int cyc, bits, C, f, eps, rate, dl, key, pi, rows, total;
  int lg;   // rows hold 2^lg levels
  int run;  // partition points whose rows are resident at once
};

constexpr int TABLE_ROW_BYTES = 4096;  // LDS for the level rows of one run

__host__ __device__ inline TLayout make_tlayout(int N, int L, int K, int szT) {
  TLayout y;
  int o = 0;
  auto take = [&](int bytes) { int r = o; o = align8(o + bytes); return r; };
  y.cyc = take(L * szT);
  y.bits = take((L + 1) * szT);
  y.C = take((L + 1) * szT);
  y.f = take(K * szT);
  y.eps = take(K * szT);
  o = (o + 4 * szT - 1) & ~(4 * szT - 1);  // rates and deadlines: four per LDS read
  y.rate = take(N * szT);
  o = (o + 4 * szT - 1) & ~(4 * szT - 1);
  y.dl = take(N * szT);
  y.key = take((N + 1) * 8);
  y.pi = take(N * 4);
  int lg = 0;
  while ((1 << lg) < K) ++lg;
  y.lg = lg;
  const int rowb = (1 << lg) * 2 * szT;  // at most 64 levels x 16 B = 1 KB
  int run = TABLE_ROW_BYTES / rowb;     // >= 4
  // a run that is not the last covers a multiple of four partition points,
  // so that its entries start on a four-entry boundary
  run = (run >= L + 1) ? L + 1 : (run & ~3);
  y.run = run;
  o = (o + 15) & ~15;
  y.rows = o;
  o += run * rowb;
  y.total = o;
  return y;
}

// A level's latency and energy by one LDS read (both are used; read apart,
// the energy's read would be deferred into a branch on the latency).
template <typename T> __device__ inline Level<T> level_at(const Level<T> *p) {
  if constexpr (sizeof(T) == 4) {
    const unsigned long long u = *(const unsigned long long *)p;
    Level<T> v;
    v.t = __uint_as_float((unsigned)u);
    v.e = __uint_as_float((unsigned)(u >> 32));
    return v;
  } else {
    return *p;
  }
}

// Four table entries of one lane, stored together.
template <typename T> struct alignas(4 * sizeof(T)) Vec4 { T v[4]; };
typedef float f4v __attribute__((ext_vector_type(4)));
typedef double d2v __attribute__((ext_vector_type(2)));
// Entries o..o+3 of a row that starts at base (o < 2^28: the byte offset is
// a 32-bit register added to the row's base held in scalar registers).
__device__ inline void nt4(float *base, unsigned o, const Vec4<float> &v) {
  f4v x = {v.v[0], v.v[1], v.v[2], v.v[3]};
  __builtin_nontemporal_store(x, (f4v *)((char *)base + o * 4u));
}
__device__ inline void nt4(double *base, unsigned o, const Vec4<double> &v) {
  d2v a = {v.v[0], v.v[1]}, b = {v.v[2], v.v[3]};
  __builtin_nontemporal_store(a, (d2v *)((char *)base + o * 8u));
  __builtin_nontemporal_store(b, (d2v *)((char *)base + o * 8u + 16u));
}

// Levels of a row too slow for the budget: a prefix of the row (latencies
// fall with the level), found by binary search over the row padded to 2^LG
// entries with pads that are never too slow.  The row starts rowb bytes into
// the LDS block; with LG fixed, every probe is an LDS read at an immediate
// offset from the running position.
template <typename T, int LG>
__device__ inline int too_slow(const unsigned char *smem, unsigned rowb, T budget) {
  constexpr unsigned S = sizeof(Level<T>);
  unsigned a = rowb;
#pragma unroll
  for (int h = (1 << LG) >> 1; h > 0; h >>= 1)
    a = (*(const T *)(smem + a + (h - 1) * S) > budget) ? a + h * S : a;
  return (int)((a - rowb) / S);
}

// Stage-1 preparation of one instance in its LDS block: the instance's rows
// (coalesced) and the CPU levels, C in the pinned order, the rate order pi,
// the batch deadlines lo[b] (a running minimum along pi) and bmin (written
// out when `out`).  WS: the workgroup holds other waves, each preparing an
// instance of its own (barriers of this wave only).
template <typename T, bool WS = false>
__device__ inline void tables_prepare(const Problem<T> &p, const Tables<T> &tab, int64_t inst,
                                      unsigned char *smem, const TLayout &y, int lane, bool out) {
  const int N = p.N, L = p.L, K = p.K;
  T *scyc = (T *)(smem + y.cyc), *sbits = (T *)(smem + y.bits), *sC = (T *)(smem + y.C);
  T *sf = (T *)(smem + y.f), *seps = (T *)(smem + y.eps);
  T *srate = (T *)(smem + y.rate), *sdl = (T *)(smem + y.dl);
  int *spi = (int *)(smem + y.pi);

  for (int l = lane; l < L; l += WAVE) scyc[l] = p.cyc[inst * L + l];
  for (int l = lane; l <= L; l += WAVE) sbits[l] = p.bits[inst * (L + 1) + l];
  for (int m = lane; m < N; m += WAVE) {
    srate[m] = p.rate[inst * N + m];
    sdl[m] = p.deadline[inst * N + m];
    spi[m] = m;  // stays a permutation of valid users
  }
  for (int k = lane; k < K; k += WAVE) {
    const T f = p.lf[k];
    sf[k] = f;
    seps[k] = p.kappa * (f * f);
  }
  lds_sync<WS>();
  // C[0] = 0, C[q+1] = C[q] + cyc[q] in order
  chain_sums<T, WS>(scyc, nullptr, nullptr, sC, nullptr, nullptr, L, lane);
  rank_users<WS>(srate, (uint64_t *)(smem + y.key), spi, N, lane);
  lds_sync<WS>();

  // the users without a local level are those whose deadline the whole
  // chain at the top level misses (t[L][k] falls with k)
  const T tLtop = sC[L] / sf[K - 1];
  T carry = inf_of<T>();
  int bm = 0;
  for (int i0 = 0; i0 < N; i0 += WAVE) {
    const int i = i0 + lane;
    const int m = (i < N) ? spi[i] : 0;
    const T d = (i < N) ? sdl[m] : inf_of<T>();
    T v = wave_scan<T, true>(d, lane);
    v = (carry < v) ? carry : v;
    carry = lane_read(v, WAVE - 1);
    if (out && i < N) {
      tab.order[inst * N + i] = (int16_t)m;
      tab.lo[inst * N + i] = v;
    }
    const uint64_t nl = __builtin_amdgcn_ballot_w64(i < N && !(tLtop <= d));
    if (nl) bm = i0 + 64 - __clzll((long long)nl);  // 1 + the last such position
  }
  if (out && lane == 0) tab.bmin[inst] = bm;
}

// The CPU level rows (Eqs. (1), (2)) of partition points s0 .. s0+ns-1 of
// one instance, 2^lg levels each, padded with levels that always fit
// (latency -inf) and are never chosen; a lane builds level lane mod 2^lg of
// its rows (2^lg divides WAVE).
template <typename T>
__device__ inline void tables_rows(unsigned char *smem, const TLayout &y, int s0, int ns, int lg,
                                   int K, int lane) {
  const T *sC = (const T *)(smem + y.C), *sf = (const T *)(smem + y.f);
  const T *seps = (const T *)(smem + y.eps);
  Level<T> *rows = (Level<T> *)(smem + y.rows);
  const int kl = lane & ((1 << lg) - 1);
  const T fk = sf[kl < K ? kl : K - 1], ek = seps[kl < K ? kl : K - 1];
  for (int e = lane; e < (ns << lg); e += WAVE) {
    const T Cs = sC[s0 + (e >> lg)];
    Level<T> v;
    v.t = (kl < K) ? Cs / fk : -inf_of<T>();
    v.e = (kl < K) ? ek * Cs : T(0);
    rows[e] = v;
  }
}

// The entries of users m..m+3 of one partition point (N a multiple of four:
// the four share the row, its top level and O_s = bs): upload time (Eq.
// (3), zero without offloading), gamma, and the user's own lowest level
// within its budget with its energy (Eqs. (2), (4)) and slack.  The row
// starts rowb bytes into LDS; rate4 and dl4 point at the four users' rates
// and deadlines.
template <typename T, int LG>
__device__ inline void table_quad(const unsigned char *smem, unsigned rowb, T bs, bool offl,
                                  const T *rate4, const T *dl4, int K, T ptx, Vec4<T> &vu,
                                  Vec4<T> &vg, Vec4<T> &ve, Vec4<T> &vs, uint32_t &lv4) {
  const Level<T> *row = (const Level<T> *)(smem + rowb);
  const T tK1 = row[K - 1].t;
  const Quad<T> r4 = *(const Quad<T> *)rate4;
  const Quad<T> d4 = *(const Quad<T> *)dl4;
  lv4 = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const T up = offl ? bs / r4.v[c] : T(0);
    const T budget = d4.v[c] - up;
    const int cnt = too_slow<T, (LG < 0 ? 0 : LG)>(smem, rowb, budget);
    const int k = cnt < K ? cnt : K - 1;
    const Level<T> lvk = level_at(row + k);
    const bool fits = lvk.t <= budget;
    vu.v[c] = up;
    vg.v[c] = up + tK1;
    ve.v[c] = fits ? lvk.e + ptx * up : inf_of<T>();
    vs.v[c] = budget - lvk.t;
    lv4 |= (uint32_t)(fits ? k : 0xff) << (8 * c);
  }
}

// One wave per instance.  VEC: the tables start on 16-byte boundaries (four
// entries per store).  LG >= 0: N is a multiple of four and rows hold 2^LG
// levels.
template <typename T, bool VEC, int LG>
__global__ __launch_bounds__(WAVE, 8) void jdob_tables_kernel(Problem<T> p, Tables<T> tab,
                                                               int64_t first) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x;
  const int64_t inst = instance_of_block(first);
  const int N = p.N, L = p.L, K = p.K;
  const TLayout y = make_tlayout(N, L, K, (int)sizeof(T));
  const T *sbits = (const T *)(smem + y.bits);
  const T *srate = (const T *)(smem + y.rate), *sdl = (const T *)(smem + y.dl);
  const Level<T> *rows = (const Level<T> *)(smem + y.rows);
  tables_prepare<T>(p, tab, inst, smem, y, lane, true);

  const int lg = LG >= 0 ? LG : y.lg, K4 = 1 << lg;
  const int total = (L + 1) * N;
  const int64_t base = inst * (int64_t)total;
  const T ptx = p.ptx;
  T *const tup = tab.up + base, *const tgam = tab.gamma + base, *const ten = tab.senergy + base;
  T *const tsl = tab.sslack + base;
  int8_t *const tlev = tab.slevel + base;
  // a pass advances 256 entries: q256 rows and r256 users
  const int q256 = (4 * WAVE) / N, r256 = (4 * WAVE) % N;
  for (int s0 = 0; s0 <= L; s0 += y.run) {
    const int ns = min(y.run, L + 1 - s0);
    __syncthreads();
    tables_rows<T>(smem, y, s0, ns, lg, K, lane);
    __syncthreads();
    const int e_lo = s0 * N, e_hi = min((s0 + ns) * N, total);
    int so = (4 * lane) / N, m = (4 * lane) - so * N;  // of the lane's first entry in the run
    if constexpr (VEC && LG >= 0) {
      for (int e = e_lo + 4 * lane; e < e_hi; e += 4 * WAVE) {
        const int s = s0 + so;
        const unsigned rowb = (unsigned)y.rows + (unsigned)(so << lg) * (unsigned)sizeof(Level<T>);
        Vec4<T> vu, vg, ve, vs;
        uint32_t lv4;
        table_quad<T, LG>(smem, rowb, sbits[s], s < L, srate + m, sdl + m, K, ptx, vu, vg, ve, vs,
                          lv4);
        const unsigned o = (unsigned)e;
        nt4(tup, o, vu);
        nt4(tgam, o, vg);
        nt4(ten, o, ve);
        nt4(tsl, o, vs);
        __builtin_nontemporal_store(lv4, (uint32_t *)(tlev + o));
        m += r256;
        so += q256;
        if (m >= N) {
          m -= N;
          ++so;
        }
      }
      continue;
    }
    for (int e = e_lo + 4 * lane; e < e_hi; e += 4 * WAVE) {
      Vec4<T> vu, vg, ve, vs;
      uint32_t lv4 = 0;
      int sc = so, mc = m;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int s = s0 + sc;
        const Level<T> *row = rows + (min(sc, ns - 1) << lg);  // past the run: masked below
        const T up = (s < L) ? sbits[min(s, L)] / srate[mc] : T(0);
        const T budget = sdl[mc] - up;
        int cnt = 0;  // levels slower than the budget (a prefix of the row)
        for (int step = K4 >> 1; step > 0; step >>= 1)
          cnt = (row[cnt + step - 1].t > budget) ? cnt + step : cnt;
        const int k = cnt < K ? cnt : K - 1;
        const Level<T> lvk = row[k];
        const bool fits = lvk.t <= budget;
        vu.v[c] = up;
        vg.v[c] = up + row[K - 1].t;
        ve.v[c] = fits ? lvk.e + ptx * up : inf_of<T>();
        vs.v[c] = budget - lvk.t;
        lv4 |= (uint32_t)(uint8_t)(int8_t)(fits ? k : -1) << (8 * c);
        if (++mc == N) {
          mc = 0;
          ++sc;
        }
      }
      const unsigned o = (unsigned)e;  // entry offset within the instance (< 2^18)
      if constexpr (VEC) {
        nt4(tup, o, vu);
        nt4(tgam, o, vg);
        nt4(ten, o, ve);
        nt4(tsl, o, vs);
        __builtin_nontemporal_store(lv4, (uint32_t *)(tlev + o));
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (o + c < (unsigned)e_hi) {
            tup[o + c] = vu.v[c];
            tgam[o + c] = vg.v[c];
            ten[o + c] = ve.v[c];
            tsl[o + c] = vs.v[c];
            tlev[o + c] = (int8_t)(lv4 >> (8 * c));
          }
      }
      m += r256;
      so += q256;
      if (m >= N) {
        m -= N;
        ++so;
      }
    }
  }
}

// LDS block of one instance in the group kernel (16-byte aligned).
__host__ __device__ inline int tables_block_bytes(const TLayout &y) { return (y.total + 15) & ~15; }

// G consecutive instances per workgroup of G waves, for N a multiple of four
// with every level row of an instance resident at once.  Each wave prepares
// its instance in its own LDS block (barriers of its own), then the
// workgroup stores the G instances' entries, which are contiguous in every
// table, as one span: each pass covers 256*G consecutive entries, so the
// stores of a pass form runs G times longer than one wave's, across
// instance boundaries.  Instances [first, end) are this launch's.
template <typename T, int LG, int G>
__global__ __launch_bounds__(WAVE *G, 8) void jdob_tables_group_kernel(Problem<T> p,
                                                                       Tables<T> tab,
                                                                       int64_t first,
                                                                       int64_t end) {
  extern __shared__ __align__(16) unsigned char smem_all[];
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int N = p.N, L = p.L, K = p.K;
  const TLayout y = make_tlayout(N, L, K, (int)sizeof(T));
  const int SB = tables_block_bytes(y);
  const int64_t g0 = first + G * instance_of_block(0);
  const int cnt = (int)((end - g0) < G ? (end - g0) : G);
  // waves past the last instance prepare the group's first one again (every
  // wave takes the same barriers) and write nothing of it
  unsigned char *smem = smem_all + w * SB;
  tables_prepare<T, true>(p, tab, g0 + (w < cnt ? w : 0), smem, y, lane, w < cnt);
  tables_rows<T>(smem, y, 0, L + 1, LG, K, lane);
  __syncthreads();

  const int E = (L + 1) * N, span = cnt * E;  // span < 2^21
  const int64_t base = g0 * (int64_t)E;
  const T ptx = p.ptx;
  T *const tup = tab.up + base, *const tgam = tab.gamma + base, *const ten = tab.senergy + base;
  T *const tsl = tab.sslack + base;
  int8_t *const tlev = tab.slevel + base;
  // a pass advances D entries: dq rows and dr users
  constexpr int D = 4 * WAVE * G;
  const int dq = D / N, dr = D % N;
  const int x0 = 4 * (int)threadIdx.x;
  int g = x0 / E, s = (x0 - g * E) / N, m = x0 - g * E - s * N;  // of the lane's first entry
  for (int x = x0; x < span; x += D) {
    const unsigned blk = (unsigned)(g * SB);
    const unsigned char *sg = smem_all + blk;
    const unsigned rowb = blk + (unsigned)y.rows + (unsigned)(s << LG) * (unsigned)sizeof(Level<T>);
    Vec4<T> vu, vg, ve, vs;
    uint32_t lv4;
    table_quad<T, LG>(smem_all, rowb, ((const T *)(sg + y.bits))[s], s < L,
                      (const T *)(sg + y.rate) + m, (const T *)(sg + y.dl) + m, K, ptx, vu, vg,
                      ve, vs, lv4);
    const unsigned o = (unsigned)x;
    nt4(tup, o, vu);
    nt4(tgam, o, vg);
    nt4(ten, o, ve);
    nt4(tsl, o, vs);
    __builtin_nontemporal_store(lv4, (uint32_t *)(tlev + o));
    m += dr;
    if (m >= N) {
      m -= N;
      ++s;
    }
    s += dq;
    if (s > L) {
      const int q = s / (L + 1);
      g += q;
      s -= q * (L + 1);
    }
  }
}

// ----------------------------------------------------------------- host side

bool finite_nonneg(double x) { return isfinite(x) && x >= 0.0; }

// The batch sentinels of a problem's search (batch_sentinels): the GPU
// levels searched are all J, or the top one without edge DVFS.
int sentinels_of(const jdob_problem *p) {
  const int Jn = (p->mode & JDOB_MODE_FIXED_EDGE_FREQ) ? 1 : p->num_gpu_levels;
  return batch_sentinels(Jn, (p->mode & JDOB_MODE_GREEDY) != 0);
}

int validate(const jdob_problem *p) {
  if (!p) return JDOB_ERR_INVALID_ARG;
  if (p->num_instances < 0 || p->num_users < 1 || p->num_layers < 1 ||
      p->num_local_levels < 1 || p->num_gpu_levels < 1)
    return JDOB_ERR_INVALID_ARG;
  if (p->dtype != JDOB_F32 && p->dtype != JDOB_F64) return JDOB_ERR_UNSUPPORTED;
  if (p->num_users > JDOB_MAX_USERS || p->num_layers > JDOB_MAX_LAYERS ||
      p->num_local_levels > JDOB_MAX_LOCAL_LEVELS || p->num_gpu_levels > JDOB_MAX_GPU_LEVELS)
    return JDOB_ERR_UNSUPPORTED;
  // an empty batch reads and writes nothing: its array pointers may be NULL
  if (p->num_instances > 0 &&
      (!p->layer_cycles || !p->out_bits || !p->gpu_alpha || !p->gpu_beta || !p->uplink_rate ||
       !p->deadline || !p->local_freq || !p->gpu_freq))
    return JDOB_ERR_INVALID_ARG;
  if (!finite_nonneg(p->kappa) || !finite_nonneg(p->p_tx) || !finite_nonneg(p->gpu_c) ||
      !finite_nonneg(p->gpu_p_static))
    return JDOB_ERR_INVALID_ARG;
  if (p->mode & ~(JDOB_MODE_GREEDY | JDOB_MODE_FIXED_EDGE_FREQ | JDOB_MODE_BINARY |
                  JDOB_MODE_CONTINUOUS_CPU))
    return JDOB_ERR_INVALID_ARG;
  // flat candidate indices must fit in int32
  if ((int64_t)p->num_layers * p->num_gpu_levels * p->num_users >= 0x7fffffffLL)
    return JDOB_ERR_UNSUPPORTED;
  if (has_user_params(p)) return validate_hetero(p, false);
  const int sz = p->dtype == JDOB_F64 ? 8 : 4;
  const bool cont = (p->mode & JDOB_MODE_CONTINUOUS_CPU) != 0;
  const bool greedy = (p->mode & JDOB_MODE_GREEDY) != 0;
  if (make_layout(p->num_users, p->num_layers, p->num_local_levels, p->num_gpu_levels, sz, cont,
                  queued_search(p->num_users, cont, greedy), sentinels_of(p))
          .total > LDS_LIMIT)
    return JDOB_ERR_UNSUPPORTED;
  return JDOB_OK;
}

template <typename T> Problem<T> to_problem(const jdob_problem *q) {
  Problem<T> p;
  p.cyc = (const T *)q->layer_cycles;
  p.bits = (const T *)q->out_bits;
  p.alpha = (const T *)q->gpu_alpha;
  p.beta = (const T *)q->gpu_beta;
  p.rate = (const T *)q->uplink_rate;
  p.deadline = (const T *)q->deadline;
  p.tfree = (const T *)q->t_free;
  p.lf = (const T *)q->local_freq;
  p.gf = (const T *)q->gpu_freq;
  p.kappa = (T)q->kappa;
  p.ptx = (T)q->p_tx;
  p.gc = (T)q->gpu_c;
  p.p0 = (T)q->gpu_p_static;
  p.N = q->num_users;
  p.L = q->num_layers;
  p.K = q->num_local_levels;
  p.J = q->num_gpu_levels;
  p.s_end = (q->mode & JDOB_MODE_BINARY) ? 1 : p.L;
  p.j_low = (q->mode & JDOB_MODE_FIXED_EDGE_FREQ) ? p.J - 1 : 0;
  p.cont = (q->mode & JDOB_MODE_CONTINUOUS_CPU) ? 1 : 0;
  return p;
}

template <typename T> Policy<T> to_policy(const jdob_policy *o) {
  Policy<T> r;
  r.status = o->status;
  r.cut = o->cut;
  r.gpu_level = o->gpu_level;
  r.batch = o->batch;
  r.energy = (T *)o->energy;
  r.tfree_out = (T *)o->t_free_out;
  r.ulevel = o->user_level;
  r.uoffload = o->user_offload;
  r.nfeas = o->num_feasible;
  r.nevals = o->num_user_evals;
  r.ufreq = (T *)o->user_freq;
  return r;
}

template <typename T> Tables<T> to_tables(const jdob_user_tables *t) {
  Tables<T> r{};
  if (!t) return r;
  r.order = t->order;
  r.lo = (T *)t->batch_deadline;
  r.bmin = t->min_batch;
  r.up = (T *)t->uplink_time;
  r.gamma = (T *)t->gamma;
  r.slevel = t->self_level;
  r.senergy = (T *)t->self_energy;
  r.sslack = (T *)t->self_slack;
  return r;
}

bool policy_ok(const jdob_policy *o) {
  return o && o->status && o->cut && o->gpu_level && o->batch && o->energy && o->t_free_out &&
         o->user_level && o->user_offload;
}

bool tables_ok(const jdob_user_tables *t) {
  return t && t->order && t->batch_deadline && t->min_batch && t->uplink_time && t->gamma &&
         t->self_level && t->self_energy && t->self_slack;
}

template <typename T, bool FROM_TABLES>
void launch_solve(bool greedy, bool one_chunk, bool count, dim3 grid, size_t lds,
                  hipStream_t stream, const Problem<T> &p, const Tables<T> &tab,
                  const Policy<T> &pol, int64_t first) {
  const dim3 block(WAVE);
  const SolveArgs<T> a{p, tab, pol, first};
  const bool queue = queued_search(p.N, p.cont, greedy);
#define JDOB_LAUNCH(OC, CN, GR)                                                                \
  do {                                                                                         \
    if (p.cont)                                                                                \
      hipLaunchKernelGGL((jdob_solve_kernel<T, FROM_TABLES, OC, CN, GR, true, false>), grid,   \
                         block, lds, stream, a);                                               \
    else if (queue)                                                                            \
      hipLaunchKernelGGL((jdob_solve_kernel<T, FROM_TABLES, OC, CN, GR, false, !GR>), grid,    \
                         block, lds, stream, a);                                               \
    else                                                                                       \
      hipLaunchKernelGGL((jdob_solve_kernel<T, FROM_TABLES, OC, CN, GR, false, false>), grid,  \
                         block, lds, stream, a);                                               \
  } while (0)
  if (greedy) {  // one lane per GPU level: the chunking of levels is the kernel's
    if (count) JDOB_LAUNCH(false, true, true);
    else JDOB_LAUNCH(false, false, true);
  } else if (one_chunk) {
    if (count) JDOB_LAUNCH(true, true, false);
    else JDOB_LAUNCH(true, false, false);
  } else {
    if (count) JDOB_LAUNCH(false, true, false);
    else JDOB_LAUNCH(false, false, false);
  }
#undef JDOB_LAUNCH
}

// Stage 1 with N a multiple of four, at the row size of the CPU levels.
template <typename T>
void launch_tables_quad(int lg, dim3 grid, size_t lds, hipStream_t stream, const Problem<T> &p,
                        const Tables<T> &tab, int64_t first) {
  const dim3 block(WAVE);
#define JDOB_TQ(G)                                                                        \
  case G:                                                                                 \
    hipLaunchKernelGGL((jdob_tables_kernel<T, true, G>), grid, block, lds, stream, p, tab, \
                       first);                                                            \
    break;
  switch (lg) {
    JDOB_TQ(0) JDOB_TQ(1) JDOB_TQ(2) JDOB_TQ(3) JDOB_TQ(4) JDOB_TQ(5) JDOB_TQ(6)
    default: break;
  }
#undef JDOB_TQ
}
static_assert(JDOB_MAX_LOCAL_LEVELS <= 64, "stage-1 rows of at most 2^6 levels");

// Instances per workgroup of a stage-1 launch of n instances with N a
// multiple of four: 2 when every level row of an instance is resident at
// once, two LDS blocks fit a workgroup, the launch is long and an
// instance's int8 level-table span is not a whole number of 128-byte lines;
// else 1 (one wave per instance).  Measured on 2^20 instances (N 32, L 22):
// 2.69 ms one wave per instance, 2.52 in pairs or fours (the pairs' passes
// store 2 KB runs of each table where single waves store 1 KB); on a short
// launch (2^16 instances, N 16, L 22) the waves' wait for each other costs
// more (0.086 ms alone, 0.088 in pairs); with whole lines per instance
// (N 128, L 50) pairs gain nothing.
int tables_group(int64_t n, int N, int L, const TLayout &y) {
  const int64_t E = (int64_t)(L + 1) * N;
  if (n < (int64_t(1) << 18) || y.run < L + 1 || E % 128 == 0) return 1;
  return 2 * (int64_t)tables_block_bytes(y) <= LDS_LIMIT ? 2 : 1;
}

// The group kernel at (row size 2^lg, G instances per workgroup) for
// instances [first, first + n).
template <typename T>
void launch_tables_group(int lg, int G, int64_t n, const TLayout &y, hipStream_t stream,
                         const Problem<T> &p, const Tables<T> &tab, int64_t first) {
  const dim3 grid((unsigned)((n + G - 1) / G)), block(WAVE * G);
  const size_t lds = (size_t)G * tables_block_bytes(y);
#define JDOB_TG(LGV, GV)                                                                 \
  case LGV * 16 + GV:                                                                    \
    hipLaunchKernelGGL((jdob_tables_group_kernel<T, LGV, GV>), grid, block, lds, stream, \
                       p, tab, first, first + n);                                        \
    break;
  switch (lg * 16 + G) {
    JDOB_TG(0, 2) JDOB_TG(1, 2) JDOB_TG(2, 2) JDOB_TG(3, 2) JDOB_TG(4, 2) JDOB_TG(5, 2)
    JDOB_TG(6, 2)
    default: break;
  }
#undef JDOB_TG
}

// entry 0: fused solve, 1: joint from tables, 2: tables
template <typename T>
int launch(int entry, const jdob_problem *q, const jdob_user_tables *t, const jdob_policy *o,
           hipStream_t stream) {
  const Problem<T> p = to_problem<T>(q);
  const Tables<T> tab = to_tables<T>(t);
  Policy<T> pol{};
  if (o) pol = to_policy<T>(o);
  const int64_t I = q->num_instances;
  const bool greedy = (q->mode & JDOB_MODE_GREEDY) != 0;
  const size_t lds = (size_t)make_layout(p.N, p.L, p.K, p.J, (int)sizeof(T), p.cont,
                                         queued_search(p.N, p.cont, greedy), sentinels_of(q))
                         .total;
  const bool one = p.J - p.j_low <= WAVE;
  const bool count = pol.nfeas != nullptr || pol.nevals != nullptr;
  // stage 1: wide stores when every instance's tables start on a 16-byte
  // boundary (four entries per instance row, aligned table pointers)
  const size_t tlds = (size_t)make_tlayout(p.N, p.L, p.K, (int)sizeof(T)).total;
  auto al = [](const void *q, uintptr_t a) { return ((uintptr_t)q & (a - 1)) == 0; };
  const bool vec = entry == 2 && ((int64_t)(p.L + 1) * p.N) % 4 == 0 && al(tab.up, 16) &&
                   al(tab.gamma, 16) && al(tab.senergy, 16) && al(tab.sslack, 16) &&
                   al(tab.slevel, 4);
  for (int64_t first = 0; first < I; first += MAX_BLOCKS_PER_LAUNCH) {
    const int64_t n = (I - first < MAX_BLOCKS_PER_LAUNCH) ? I - first : MAX_BLOCKS_PER_LAUNCH;
    const dim3 grid((unsigned)n), block(WAVE);
    if (entry == 0)
      launch_solve<T, false>(greedy, one, count, grid, lds, stream, p, tab, pol, first);
    else if (entry == 1)
      launch_solve<T, true>(greedy, one, count, grid, lds, stream, p, tab, pol, first);
    else if (vec && p.N % 4 == 0) {
      const TLayout ty = make_tlayout(p.N, p.L, p.K, (int)sizeof(T));
      const int G = tables_group(n, p.N, p.L, ty);
      if (G > 1)
        launch_tables_group<T>(ty.lg, G, n, ty, stream, p, tab, first);
      else
        launch_tables_quad<T>(ty.lg, grid, tlds, stream, p, tab, first);
    }
    else if (vec)
      hipLaunchKernelGGL((jdob_tables_kernel<T, true, -1>), grid, block, tlds, stream, p, tab,
                         first);
    else
      hipLaunchKernelGGL((jdob_tables_kernel<T, false, -1>), grid, block, tlds, stream, p, tab,
                         first);
    if (hipGetLastError() != hipSuccess) return JDOB_ERR_HIP;
  }
  return JDOB_OK;
}

bool grouped_ok(const jdob_grouped_policy *o) {
  return o && o->status && o->num_groups && o->energy && o->t_free_out && o->order &&
         o->group_end && o->group_cut && o->group_gpu_level && o->group_batch &&
         o->group_energy && o->group_t_free && o->user_level && o->user_offload && o->user_group;
}

template <typename T> Grouped<T> to_grouped(const jdob_grouped_policy *o) {
  Grouped<T> g;
  g.status = o->status;
  g.num_groups = o->num_groups;
  g.energy = (T *)o->energy;
  g.tfree_out = (T *)o->t_free_out;
  g.order = o->order;
  g.group_end = o->group_end;
  g.group_cut = o->group_cut;
  g.group_gpu_level = o->group_gpu_level;
  g.group_batch = o->group_batch;
  g.group_energy = (T *)o->group_energy;
  g.group_tfree = (T *)o->group_t_free;
  g.ulevel = o->user_level;
  g.uoffload = o->user_offload;
  g.ugroup = o->user_group;
  g.ninner = o->num_inner;
  g.nfeas = o->num_feasible;
  g.nevals = o->num_user_evals;
  g.ufreq = (T *)o->user_freq;
  return g;
}

template <typename T>
int launch_grouped(const jdob_problem *q, const jdob_grouped_policy *o, hipStream_t stream) {
  const Problem<T> p = to_problem<T>(q);
  const Grouped<T> g = to_grouped<T>(o);
  const Layout y = make_layout(p.N, p.L, p.K, p.J, (int)sizeof(T), p.cont, false,
                               sentinels_of(q));
  const size_t lds = (size_t)make_glayout(y, p.N, (int)sizeof(T)).total;
  const bool greedy = (q->mode & JDOB_MODE_GREEDY) != 0;
  const bool one = p.J - p.j_low <= WAVE;
  const bool count = g.ninner != nullptr || g.nfeas != nullptr || g.nevals != nullptr;
  const dim3 block(WAVE);
  const int64_t I = q->num_instances;
  for (int64_t first = 0; first < I; first += MAX_BLOCKS_PER_LAUNCH) {
    const int64_t n = (I - first < MAX_BLOCKS_PER_LAUNCH) ? I - first : MAX_BLOCKS_PER_LAUNCH;
    const dim3 grid((unsigned)n);
    const GroupedArgs<T> a{p, g, first};
#define JDOB_LAUNCH(OC, CN, GR)                                                               \
  do {                                                                                        \
    if (p.cont)                                                                               \
      hipLaunchKernelGGL((jdob_grouped_kernel<T, OC, CN, GR, true>), grid, block, lds, stream, \
                         a);                                                                  \
    else                                                                                      \
      hipLaunchKernelGGL((jdob_grouped_kernel<T, OC, CN, GR, false>), grid, block, lds,        \
                         stream, a);                                                          \
  } while (0)
    if (greedy) {
      if (count) JDOB_LAUNCH(false, true, true);
      else JDOB_LAUNCH(false, false, true);
    } else if (one) {
      if (count) JDOB_LAUNCH(true, true, false);
      else JDOB_LAUNCH(true, false, false);
    } else {
      if (count) JDOB_LAUNCH(false, true, false);
      else JDOB_LAUNCH(false, false, false);
    }
#undef JDOB_LAUNCH
    if (hipGetLastError() != hipSuccess) return JDOB_ERR_HIP;
  }
  return JDOB_OK;
}

int dispatch(int entry, const jdob_problem *q, const jdob_user_tables *t, const jdob_policy *o,
             void *stream) {
  hipStream_t s = (hipStream_t)stream;
  return q->dtype == JDOB_F64 ? launch<double>(entry, q, t, o, s)
                              : launch<float>(entry, q, t, o, s);
}

}  // namespace

extern "C" {

int jdob_solve_batch(const jdob_problem *p, jdob_policy *out, void *hip_stream) {
  int rc = validate(p);
  if (rc != JDOB_OK) return rc;
  if (p->num_instances == 0) return JDOB_OK;  // nothing to launch
  if (!policy_ok(out)) return JDOB_ERR_INVALID_ARG;
  if (has_user_params(p)) return launch_hetero(p, out, (hipStream_t)hip_stream);
  return dispatch(0, p, nullptr, out, hip_stream);
}

int jdob_eval_user_tables(const jdob_problem *p, jdob_user_tables *out, void *hip_stream) {
  int rc = validate(p);
  if (rc != JDOB_OK) return rc;
  if (has_user_params(p)) return JDOB_ERR_UNSUPPORTED;  // one rate order per instance
  if (p->num_instances == 0) return JDOB_OK;
  if (!tables_ok(out)) return JDOB_ERR_INVALID_ARG;
  return dispatch(2, p, out, nullptr, hip_stream);
}

int jdob_eval_joint(const jdob_problem *p, const jdob_user_tables *tab, jdob_policy *out,
                    void *hip_stream) {
  int rc = validate(p);
  if (rc != JDOB_OK) return rc;
  if (has_user_params(p)) return JDOB_ERR_UNSUPPORTED;
  if (p->num_instances == 0) return JDOB_OK;
  if (!tables_ok(tab) || !policy_ok(out)) return JDOB_ERR_INVALID_ARG;
  return dispatch(1, p, tab, out, hip_stream);
}

int jdob_solve_grouped(const jdob_problem *p, jdob_grouped_policy *out, void *hip_stream) {
  int rc = validate(p);
  if (rc != JDOB_OK) return rc;
  if (has_user_params(p)) {  // heterogeneous users: N <= 64 as well
    rc = validate_hetero(p, true);
    if (rc != JDOB_OK) return rc;
    if (p->num_instances == 0) return JDOB_OK;
    if (!grouped_ok(out)) return JDOB_ERR_INVALID_ARG;
    return launch_hetero_grouped(p, out, (hipStream_t)hip_stream);
  }
  if (p->num_users > JDOB_MAX_GROUPED_USERS) return JDOB_ERR_UNSUPPORTED;
  const int sz = p->dtype == JDOB_F64 ? 8 : 4;
  const Layout y = make_layout(p->num_users, p->num_layers, p->num_local_levels,
                               p->num_gpu_levels, sz, (p->mode & JDOB_MODE_CONTINUOUS_CPU) != 0,
                               false, sentinels_of(p));
  if (make_glayout(y, p->num_users, sz).total > LDS_LIMIT) return JDOB_ERR_UNSUPPORTED;
  if (p->num_instances == 0) return JDOB_OK;
  if (!grouped_ok(out)) return JDOB_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)hip_stream;
  return p->dtype == JDOB_F64 ? launch_grouped<double>(p, out, s) : launch_grouped<float>(p, out, s);
}

const char *jdob_status_string(int code) {
  switch (code) {
    case JDOB_OK: return "ok";
    case JDOB_ERR_INVALID_ARG: return "invalid argument";
    case JDOB_ERR_UNSUPPORTED: return "unsupported size or dtype";
    case JDOB_ERR_HIP: return "HIP launch or device error";
    default: return "unknown status";
  }
}

}  // extern "C"
