// jdob_hetero.hip — batched J-DOB for heterogeneous users on MI355X (gfx950).
//
// Sec. II gives each device m its own cycles-per-work ratio zeta_m (Eq. (1)),
// switched capacitance kappa_m (Eq. (2)), transmit power p_m (Eq. (4)) and
// CPU frequency range.  Alg. 1 then sorts the users by gamma (Eq. (17)) at
// every partition point, so the order pi_s, the batch deadlines lo[b]
// (Eq. (10)), bmin and the suffix sums all depend on s, and each offloader
// has its own level table.  One wave64 evaluates one instance (N <= 64, one
// lane per user wherever per-user work is done):
//   1. coalesced loads; the sums C, A, B in the pinned order; each user's
//      local-only level and energy (constraint (8), Eq. (20));
//   2. per partition point s: each user's gamma, its rank by comparison
//      counting (ties: lower index), its level row (Eqs. (1), (2)) and the
//      smallest slack at which it meets (7) at its top frequency; then min-,
//      max- and sum-scans along pi_s give the batch records;
//   3. passes over (GPU level j x batch b) or, in the greedy mode, one batch
//      per level found by binary search; each lane walks its offloaders:
//      the level is the number of the user's levels too slow for the budget
//      (its latencies fall with the level), counted with broadcast reads, or
//      the continuous frequency clamped to the user's range;
//   4. the argmin (lowest flat index among equal energies, local computing
//      last), the winner's levels from exact comparisons, the energy summed
//      in user index order and the release time (Eq. (22)).
// Constraint (7) for every offloader of batch b is one comparison: user i
// meets it at its top frequency exactly when the slack H = lo[b] - Phi is
// at least need_i, the smallest binary value with t_i <= H - up_i (the
// rounded difference grows with H), so the batch needs H >= max_{i<b} need_i.
// The search takes any subset of the instance's users (a bit mask): all of
// them for one solve, a group of consecutive users in deadline order for
// the outer grouping (jdob_hetero_grouped_kernel), which solves every group
// of the dynamic program as an instance of its own.

#include "jdob_common.h"

namespace jdob_dev {
namespace {

template <typename T> struct HProblem {
  const T *cyc, *bits, *alpha, *beta, *rate, *deadline, *tfree, *lf, *gf;
  const T *uzeta, *ukappa, *uptx, *ulf;  // per user, or nullptr: the shared value
  T kappa, ptx, gc, p0;
  int N, L, K, J;
  int s_end, j_low;
};

template <typename T> struct HPolicy {
  int32_t *status, *cut, *gpu_level, *batch;
  T *energy, *tfree_out;
  int8_t *ulevel, *uoffload;
  int32_t *nfeas;
  int64_t *nevals;
  T *ufreq;
};

template <typename T> struct HArgs {
  HProblem<T> p;
  HPolicy<T> out;
  int64_t first;
};

template <typename T> struct HGrouped {
  int32_t *status, *num_groups;
  T *energy, *tfree_out;
  int16_t *order, *group_end;
  int32_t *group_cut, *group_gpu_level, *group_batch;
  T *group_energy, *group_tfree;
  int8_t *ulevel, *uoffload, *ugroup;
  int64_t *ninner, *nfeas, *nevals;
  T *ufreq;
};

template <typename T> struct HGArgs {
  HProblem<T> p;
  HGrouped<T> out;
  int64_t first;
};

// Per-user outputs of a winner (rows of one instance; nullptr: not written).
template <typename T> struct UserOut {
  int8_t *level, *offload, *group;
  T *freq;
  int gno;
};

// Per offloader at the current partition point, read together: its upload
// latency, its work zeta*C[s], its frequency range (continuous mode).
template <typename T> struct alignas(4 * sizeof(T)) HUser { T up, z, fmin, fmax; };

// Byte offsets of the per-instance LDS arrays.
struct HLayout {
  int cyc, al, be, bits, C, A, B, r, P;           // layers and GPU levels
  int rate, dl, zet, kap, ptx, lf, kL, eL, fL;    // per user (index m)
  int gam, key, need;                             // per user, current s
  int pi, usr, kc, lv, bt, term;                  // per position in pi_s
  int drank, dord, fE, fT, from, fn, ends, eks;  // the grouping program
  int pre;                                        // per (s, user) table of the grouping, -1: none
  int K4, total;
};

__host__ __device__ inline HLayout make_hlayout(int N, int L, int K, int J, int szT,
                                               bool grouped) {
  HLayout y;
  int o = 0;
  auto take = [&](int bytes) { int r = o; o = align8(o + bytes); return r; };
  auto take32 = [&](int bytes) { o = (o + 31) & ~31; int r = o; o = align8(o + bytes); return r; };
  y.K4 = 4;
  while (y.K4 < K) y.K4 <<= 1;  // level row stride: a power of two, pads never too slow
  y.cyc = take(L * szT);
  y.al = take(L * szT);
  y.be = take(L * szT);
  y.bits = take((L + 1) * szT);
  y.C = take((L + 1) * szT);
  y.A = take((L + 1) * szT);
  y.B = take((L + 1) * szT);
  y.r = take(J * szT);
  y.P = take(J * szT);
  y.rate = take(N * szT);
  y.dl = take(N * szT);
  y.zet = take(N * szT);
  y.kap = take(N * szT);
  y.ptx = take(N * szT);
  y.lf = take(N * K * szT);                    // user m's levels, ascending
  y.kL = take(N * 4);
  y.eL = take(N * szT);
  y.fL = take(N * szT);
  y.gam = take(N * szT);
  y.key = take32(((N + 1) & ~1) * 8);          // rank keys (binary32), even count
  y.need = take(N * szT);
  y.pi = take(N * 4);
  y.usr = take32((N + 1) * 4 * szT);           // HUser by position (+1: read-ahead)
  y.kc = take(N * szT);                        // kappa * C[s] by position
  y.lv = take32(N * y.K4 * 2 * szT);           // Level rows by position, K4 apart
  y.bt = take32((N + 2 + WAVE) * 4 * szT);     // Batch records, b = 1..N (+ sentinels)
  y.term = take(N * szT);
  y.drank = y.dord = y.fE = y.fT = y.from = y.fn = y.ends = y.eks = 0;
  if (grouped) {
    y.drank = take(N * 4);        // position of user m in the deadline order
    y.dord = take(N * 4);         // users by deadline ascending
    const int F = GROUP_FRONT;    // front of prefix i: slots i*F .. i*F + F-1
    y.fE = take((N + 1) * F * szT);  // total energy of the first i users
    y.fT = take((N + 1) * F * szT);  // GPU release time after them
    y.from = take((N + 1) * F * 2);  // the state it extends (prefix * F + slot)
    y.fn = take((N + 1) * 4);        // states in the front of prefix i
    y.ends = take((N + 1) * 4);      // ends of the chosen groups, in order
    y.eks = take((N + 1) * 4);       // the chosen state at each end
  }
  // The grouping meets every partition point once per group: each user's
  // upload latency, top-level latency and need at s (none depends on the
  // group) are kept per (s, user) where the table costs no occupancy (the
  // workgroups that fit a CU's LDS, at most 32 of one wave each) and stays
  // within the limit of one workgroup.
  y.pre = -1;
  const int pre_bytes = L * N * 3 * szT;
  auto per_cu = [](int bytes) { const int w = LDS_PER_CU / (bytes > 0 ? bytes : 1); return w < 32 ? w : 32; };
  if (grouped && align8(o) + pre_bytes <= LDS_LIMIT && per_cu(align8(o) + pre_bytes) == per_cu(o))
    y.pre = take(pre_bytes);
  y.total = o;
  return y;
}

template <typename T> __device__ inline const __attribute__((address_space(4))) HArgs<T> *hargs() {
  return (const __attribute__((address_space(4))) HArgs<T> *)__builtin_amdgcn_kernarg_segment_ptr();
}
template <typename T>
__device__ inline const __attribute__((address_space(4))) HGArgs<T> *hgargs() {
  return (const __attribute__((address_space(4))) HGArgs<T> *)__builtin_amdgcn_kernarg_segment_ptr();
}

// The neighbouring binary values of a finite x (IEEE values of one sign are
// ordered like their bit patterns).
__device__ inline float next_down(float x) {
  if (x == 0.0f) return -__int_as_float(1);
  const int b = __float_as_int(x);
  return __int_as_float(x > 0.0f ? b - 1 : b + 1);
}
__device__ inline float next_up(float x) {
  if (x == 0.0f) return __int_as_float(1);
  const int b = __float_as_int(x);
  return __int_as_float(x > 0.0f ? b + 1 : b - 1);
}
__device__ inline double next_down(double x) {
  if (x == 0.0) return -__longlong_as_double(1);
  const long long b = __double_as_longlong(x);
  return __longlong_as_double(x > 0.0 ? b - 1 : b + 1);
}
__device__ inline double next_up(double x) {
  if (x == 0.0) return __longlong_as_double(1);
  const long long b = __double_as_longlong(x);
  return __longlong_as_double(x > 0.0 ? b + 1 : b - 1);
}

// The smallest binary value H with t <= H - u (rounded subtraction).  The
// predicate only turns true as H grows, and it does so within an ulp or two
// of t + u; the walk is capped so that it always ends.
template <typename T> __device__ inline T slack_needed(T t, T u) {
  T h = t + u;
  if (t <= h - u) {
    for (int it = 0; it < 64; ++it) {
      const T d = next_down(h);
      if (!(t <= d - u)) break;
      h = d;
    }
  } else {
    for (int it = 0; it < 64; ++it) {
      h = next_up(h);
      if (t <= h - u) break;
    }
  }
  return h;
}

// Instance rows, the pinned sums, per-user parameters and levels, and each
// user's local-only choice.
template <typename T, bool CONT>
__device__ void hprepare(const HProblem<T> &p, int64_t inst, unsigned char *smem, const HLayout &y,
                         int lane) {
  const int N = p.N, L = p.L, K = p.K, J = p.J;
  T *scyc = (T *)(smem + y.cyc), *sal = (T *)(smem + y.al), *sbe = (T *)(smem + y.be);
  T *sbits = (T *)(smem + y.bits);
  T *sC = (T *)(smem + y.C), *sA = (T *)(smem + y.A), *sB = (T *)(smem + y.B);
  T *sr = (T *)(smem + y.r), *sP = (T *)(smem + y.P);
  T *srate = (T *)(smem + y.rate), *sdl = (T *)(smem + y.dl), *szet = (T *)(smem + y.zet);
  T *skap = (T *)(smem + y.kap), *sptx = (T *)(smem + y.ptx), *slf = (T *)(smem + y.lf);
  int *skL = (int *)(smem + y.kL);
  T *seL = (T *)(smem + y.eL), *sfL = (T *)(smem + y.fL);

  for (int l = lane; l < L; l += WAVE) {
    scyc[l] = p.cyc[inst * L + l];
    sal[L - 1 - l] = p.alpha[inst * L + l];  // reversed: see chain_sums
    sbe[L - 1 - l] = p.beta[inst * L + l];
  }
  for (int l = lane; l <= L; l += WAVE) sbits[l] = p.bits[inst * (L + 1) + l];
  for (int j = lane; j < J; j += WAVE) {  // Eq. (5): stretch and power of level j
    const T g = p.gf[j], gtop = p.gf[J - 1];
    sr[j] = gtop / g;
    sP[j] = p.gc * ((g * g) * g) + p.p0;
  }
  if (lane < N) {
    const int64_t o = inst * N + lane;
    srate[lane] = p.rate[o];
    sdl[lane] = p.deadline[o];
    szet[lane] = p.uzeta ? p.uzeta[o] : T(1);
    skap[lane] = p.ukappa ? p.ukappa[o] : p.kappa;
    sptx[lane] = p.uptx ? p.uptx[o] : p.ptx;
  }
  for (int q = lane; q < N * K; q += WAVE)
    slf[q] = p.ulf ? p.ulf[inst * N * K + q] : p.lf[q % K];
  __syncthreads();
  // the sums C, A, B in the pinned order
  chain_sums(scyc, sal, sbe, sC, sA, sB, L, lane);
  // (8) with Eq. (20): the lowest level finishing every layer by the deadline
  if (lane < N) {
    const T W = szet[lane] * sC[L];
    const T *f = slf + lane * K;
    int kL = -1;
    for (int k = K - 1; k >= 0; --k)
      if (W / f[k] <= sdl[lane]) kL = k;
    T fL = T(0), eL = inf_of<T>();
    if (kL >= 0) {
      fL = CONT ? cont_freq(W, sdl[lane], f[0], f[K - 1]) : f[kL];
      eL = (skap[lane] * (fL * fL)) * sC[L];
    }
    skL[lane] = kL;
    seL[lane] = eL;
    sfL[lane] = fL;
  }
  __syncthreads();
}

// Each user's top-level latency, upload latency and need (Eqs. (1), (3),
// reading 31) at a run of partition points, computed together: lane
// r*W + m holds user m's at partition point s0 + r, W = 16, 32 or 64 lanes
// per point (the solve meets its partition points in order).
template <typename T> struct HRowCache {
  int s0 = -1;
  T tk = T(0), up = T(0), nd = T(0);
};

// Partition point s for the users in mask (n of them): the gamma order
// pi_s of those users, each one's record and, if the partition point has a
// feasible candidate (the test at the top GPU level and the smallest
// admissible batch, from the scans before any record is stored;
// feasibility only falls with b and rises with j) or `records` asks for
// them, the batch records b = 1..n, and then the level rows.  Returns bmin
// and sets *any (both wave-uniform).
template <typename T, bool CONT>
__device__ int hrow(const HProblem<T> &p, int64_t inst, unsigned char *smem, const HLayout &y,
                    int lane, int s, T tfree, uint64_t mask, int n, bool *any,
                    bool records = false, HRowCache<T> *hc = nullptr) {
  const int L = p.L, K = p.K, K4 = y.K4;
  const T *sC = (const T *)(smem + y.C), *sA = (const T *)(smem + y.A);
  const T *sB = (const T *)(smem + y.B);
  const T *srate = (const T *)(smem + y.rate), *sdl = (const T *)(smem + y.dl);
  const T *szet = (const T *)(smem + y.zet), *skap = (const T *)(smem + y.kap);
  const T *sptx = (const T *)(smem + y.ptx), *slf = (const T *)(smem + y.lf);
  const int *skL = (const int *)(smem + y.kL);
  const T *seL = (const T *)(smem + y.eL);
  T *sgam = (T *)(smem + y.gam), *sneed = (T *)(smem + y.need);
  uint64_t *skey = (uint64_t *)(smem + y.key);
  int *spi = (int *)(smem + y.pi);
  HUser<T> *susr = (HUser<T> *)(smem + y.usr);
  T *skc = (T *)(smem + y.kc);
  Level<T> *slv = (Level<T> *)(smem + y.lv);
  Batch<T> *sbt = (Batch<T> *)(smem + y.bt);

  const bool mem = (mask >> lane) & 1;  // lane = user m of the instance
  const T Cs = sC[s];
  T up = T(0), W = T(0), tK1 = T(0);
  const T *pre = y.pre >= 0 ? (const T *)(smem + y.pre) + (s * p.N + lane) * 3 : nullptr;
  T ndc = T(0);
  if (hc && !pre) {
    const int lps = p.N <= 16 ? 16 : (p.N <= 32 ? 32 : WAVE), R = WAVE / lps;
    if (hc->s0 < 0 || s < hc->s0 || s >= hc->s0 + R) {
      hc->s0 = s;
      const int r = lane / lps, mu = lane - r * lps, sb = s + r;
      T tk = T(0), u = T(0), nd = T(0);
      if (mu < p.N && sb < p.s_end) {
        const T Wb = szet[mu] * sC[sb];
        tk = Wb / slf[mu * K + K - 1];
        u = ((const T *)(smem + y.bits))[sb] / srate[mu];
        nd = slack_needed(tk, u);
      }
      hc->tk = tk;
      hc->up = u;
      hc->nd = nd;
    }
    const int src = (s - hc->s0) * lps + (lane < lps ? lane : 0);
    tK1 = __shfl(hc->tk, src, WAVE);
    up = __shfl(hc->up, src, WAVE);
    ndc = __shfl(hc->nd, src, WAVE);
  }
  if (mem) {
    W = szet[lane] * Cs;                               // cycles of layers 1..s
    if (pre) {                                         // the grouping's table
      up = pre[0];
      tK1 = pre[1];
    } else if (!hc) {
      tK1 = W / slf[lane * K + K - 1];                 // Eq. (1) at the top level
      up = ((const T *)(smem + y.bits))[s] / srate[lane];  // Eq. (3)
    }
    sgam[lane] = up + tK1;                             // Eq. (17)
  }
  // Rank of each member among the members: those with a lower gamma, or an
  // equal one and a lower index.  In binary32 the 64-bit key (gamma bits,
  // index) orders the members the same way (gamma >= +0: a sum of a
  // non-negative quotient and +0 or more, and non-negative IEEE values order
  // like their bit patterns); the other users, and the pad to an even
  // count, get the largest key.  Two keys per read, one compare each.
  const int N2 = (p.N + 1) & ~1;
  if (sizeof(T) == 4 && lane < N2)
    skey[lane] = mem ? ((uint64_t)__float_as_uint((float)(up + tK1)) << 32) | (uint32_t)lane
                     : ~(uint64_t)0;
  __syncthreads();
  if (mem) {
    int pos = 0;
    if (sizeof(T) == 4) {
      const uint64_t me = skey[lane];
      for (int q = 0; q < N2; q += 2) {
        const ulonglong2 kk = *(const ulonglong2 *)(skey + q);
        pos += (kk.x < me ? 1 : 0) + (kk.y < me ? 1 : 0);
      }
    } else {
      const T g = sgam[lane];
      for (uint64_t mm = mask; mm; mm &= mm - 1) {   // the other members
        const int q = __builtin_ctzll(mm);
        const T gq = sgam[q];
        pos += (gq < g || (gq == g && q < lane)) ? 1 : 0;
      }
    }
    spi[pos] = lane;
    HUser<T> u;
    u.up = up;
    u.z = W;
    u.fmin = slf[lane * K];
    u.fmax = slf[lane * K + K - 1];
    susr[pos] = u;
    skc[pos] = skap[lane] * Cs;
    sneed[pos] = pre ? pre[2] : (hc ? ndc : slack_needed(tK1, up));
  }
  __syncthreads();
  // along pi_s (lane = position): lo = prefix min of deadlines (Eq. (10)),
  // the prefix max of need, bmin, the upload energy EU and the local
  // energies SL of the others (ranking only); scans over n positions
  const bool in = lane < n;
  const int m = in ? spi[lane] : 0;
  T lo = in ? sdl[m] : inf_of<T>(), nd = in ? sneed[lane] : -inf_of<T>();
  T sl = in ? seL[m] : T(0);
  // the minimum and the maximum are exact in any order: DPP scans
  lo = wave_iscan(lo, inf_of<T>(), [](T a, T b) { return b < a ? b : a; });
  nd = wave_iscan(nd, -inf_of<T>(), [](T a, T b) { return b > a ? b : a; });
  const uint64_t nolocal = __builtin_amdgcn_ballot_w64(in && skL[m] < 0);
  const int bmin = nolocal ? 64 - __clzll((long long)nolocal) : 0;
  // the test, with the operations of batch record blo: lo and the largest
  // need at position blo - 1, A[s] + B[s]*blo
  const int blo = bmin > 1 ? bmin : 1;
  bool ok = false;
  if (blo <= n) {
    const T ab = sA[s] + sB[s] * T(blo);
    const T H = lane_read(lo, blo - 1) - ab * ((const T *)(smem + y.r))[p.J - 1];
    ok = (H >= tfree) && (H >= lane_read(nd, blo - 1));
  }
  *any = ok;
  if (!ok && !records) return bmin;
  for (int d = 1; d < n; d <<= 1) {
    const T nsl = __shfl_down(sl, d, WAVE);
    sl = sl + ((lane + d < n) ? nsl : T(0));
  }
  const T eu = scan_add(in ? sptx[m] * susr[lane].up : T(0));
  const T slnext = __shfl_down(sl, 1, WAVE);  // sum over positions > lane
  if (in) {
    Batch<T> r;
    r.lo = lo;
    r.upl = nd;
    r.esl = eu + ((lane + 1 < n) ? slnext : T(0));
    r.ab = sA[s] + sB[s] * T(lane + 1);
    sbt[lane + 1] = r;
  }
  for (int q = lane; q < WAVE + 1; q += WAVE) {  // past n: infeasible sentinels
    Batch<T> z;
    z.lo = -inf_of<T>();
    z.upl = T(0);
    z.esl = T(0);
    z.ab = T(0);
    sbt[n + 1 + q] = z;
  }
  __syncthreads();
  if (!CONT && ok) {
    // Eqs. (1), (2) per (position, level): K4 lanes per user, padding never
    // too slow
    const int upw = WAVE / K4, pk = lane / K4, kk = lane - pk * K4;
    for (int p0 = 0; p0 < n; p0 += upw) {
      const int q = p0 + pk;
      if (pk < upw && q < n) {
        const int mq = spi[q];
        const T f = slf[mq * K + (kk < K ? kk : 0)];
        const T Wq = susr[q].z;
        Level<T> v;
        v.t = kk < K ? Wq / f : -inf_of<T>();
        v.e = kk < K ? (skap[mq] * (f * f)) * Cs : T(0);
        slv[q * K4 + kk] = v;
      }
    }
    __syncthreads();
  }
  return bmin;
}

// The CPU energy of a lane's offloaders 0..b-1 for ranking, given its slack
// Hu (+inf on infeasible lanes, whose sum is dropped): the wave walks users
// 0..bw-1; users 0..ball-1 belong to every feasible lane's batch (no test),
// later ones past the lane's batch add nothing.  The sum runs in user order,
// over several users per trip, whose level searches are independent.  LG > 0: the
// level rows hold 2^LG entries (the halving steps unrolled, each probe an
// LDS read at an immediate offset); LG = 0: their size is read from the
// layout.
template <typename T, bool CONT, int LG = 0>
__device__ inline T offload_cpu_energy(const unsigned char *smem, const HLayout &y, int K, T Hu,
                                       int b, int ball, int bw) {
  const HUser<T> *susr = (const HUser<T> *)(smem + y.usr);
  const T *skc = (const T *)(smem + y.kc);
  const Level<T> *slv = (const Level<T> *)(smem + y.lv);
  const int K4 = y.K4;
  auto user_e = [&](int g) -> T {
    const HUser<T> u = susr[g];
    const T x = Hu - u.up;
    if (CONT) {  // Eq. (20) with its clamp, in the user's own range
      const T f = clamp_(u.z * fast_rcp(x), u.fmin, u.fmax);
      return (skc[g] * f) * f;
    }
    // Eq. (20): the levels too slow for the budget are a prefix of the row
    // (latencies fall with the level), found by binary search over the row
    // padded to a power of two with never-too-slow entries; its reads depend
    // on each other, which eight waves per SIMD hide (counting every level
    // from broadcast reads was 12 % slower on h1 there, and faster at six
    // waves)
    if constexpr (LG > 0) {
      // The search ends at the level itself: an offloader of a feasible
      // lane fits its top level (the batch's slack covers its need), so
      // fewer than K levels are too slow; elsewhere the level read (at
      // most one entry past the row, inside the block's LDS) is dropped.
      constexpr unsigned S = sizeof(Level<T>);
      unsigned a = (unsigned)y.lv + (unsigned)(g << LG) * S;
#pragma unroll
      for (int h = (1 << LG) >> 1; h > 0; h >>= 1)
        a = (*(const T *)(smem + a + (h - 1) * S) > x) ? a + h * S : a;
      return *(const T *)(smem + a + sizeof(T));
    } else {
      const Level<T> *row = slv + g * K4;
      int k = 0;
      for (int step = K4 >> 1; step > 0; step >>= 1)
        k = (row[k + step - 1].t > x) ? k + step : k;
      k = k < K ? k : K - 1;
      return row[k].e;
    }
  };
  T acc = T(0);
  int g = 0;
  if constexpr (!CONT && LG > 0) {
    // the searches of four (then two) users step together: each probe of
    // one user beside the same probe of the others
    constexpr unsigned S = sizeof(Level<T>), R = (1u << LG) * S;
    for (; g + 3 < ball; g += 4) {
      T x[4];
      unsigned a[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        x[q] = Hu - susr[g + q].up;
        a[q] = (unsigned)y.lv + (unsigned)(g + q) * R;
      }
#pragma unroll
      for (int h = (1 << LG) >> 1; h > 0; h >>= 1) {
        T t[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) t[q] = *(const T *)(smem + a[q] + (h - 1) * S);
#pragma unroll
        for (int q = 0; q < 4; ++q) a[q] = (t[q] > x[q]) ? a[q] + h * S : a[q];
      }
      T e[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) e[q] = *(const T *)(smem + a[q] + sizeof(T));
#pragma unroll
      for (int q = 0; q < 4; ++q) acc = acc + e[q];
    }
    for (; g + 1 < ball; g += 2) {
      const T x0 = Hu - susr[g].up, x1 = Hu - susr[g + 1].up;
      unsigned a0 = (unsigned)y.lv + (unsigned)g * R, a1 = a0 + R;
#pragma unroll
      for (int h = (1 << LG) >> 1; h > 0; h >>= 1) {
        const T t0 = *(const T *)(smem + a0 + (h - 1) * S);
        const T t1 = *(const T *)(smem + a1 + (h - 1) * S);
        a0 = (t0 > x0) ? a0 + h * S : a0;
        a1 = (t1 > x1) ? a1 + h * S : a1;
      }
      const T e0 = *(const T *)(smem + a0 + sizeof(T)), e1 = *(const T *)(smem + a1 + sizeof(T));
      acc = acc + e0;
      acc = acc + e1;
    }
  } else if constexpr (CONT) {
    for (; g + 1 < ball; g += 2) {
      const T e0 = user_e(g), e1 = user_e(g + 1);
      acc = acc + e0;
      acc = acc + e1;
    }
  }
  for (; g < ball; ++g) acc = acc + user_e(g);
  for (; g < bw; ++g) {
    const T e = user_e(g);
    acc = (g < b) ? acc + e : acc;
  }
  return acc;
}

// Every candidate (s, j, b) of the mode's family for the users in mask (n of
// them) with the GPU free at tfree: each lane's best (energy, flat index over
// the n users' family, lowest index among equal energies) in bestE, bestI,
// and its work in nfeas, nevals when COUNT.  RUN: the users' per-point
// values come from runs of partition points (HRowCache; the grouping has a
// table of its own instead).
template <typename T, bool COUNT, bool GREEDY, bool CONT, int LG = 0, bool RUN = false>
__device__ void hsearch(const HProblem<T> &p, int64_t inst, unsigned char *smem, const HLayout &y,
                        int lane, uint64_t mask, int n, T tfree, T &bestE, int &bestI, int &nfeas,
                        int64_t &nevals) {
  const int K = p.K, J = p.J, s_end = p.s_end, j_low = p.j_low;
  const T *sr = (const T *)(smem + y.r), *sP = (const T *)(smem + y.P);
  const Batch<T> *sbt = (const Batch<T> *)(smem + y.bt);
  const int Jn = J - j_low;
  const int Jw = Jn < WAVE ? Jn : WAVE;
  const int nb = WAVE / Jw;
  const int jl = lane % Jw, bo = lane / Jw;
  const bool idle = bo >= nb;  // past the pass's (j, b) pairs: never feasible

  HRowCache<T> hc;
  for (int s = 0; s < s_end; ++s) {
    bool any;
    const int bmin =
        hrow<T, CONT>(p, inst, smem, y, lane, s, tfree, mask, n, &any, false, RUN ? &hc : nullptr);
    const int blo = bmin > 1 ? bmin : 1;
    if (!any) continue;
    const int sJN = s * J * n;
    if (GREEDY) {
      // Alg. 2 at each GPU level (lane = j): the largest set whose users all
      // meet (7) at their top frequency; the test fails more as b grows
      const int top = 1 << (31 - __clz(n));
      for (int jc = j_low; jc < J; jc += WAVE) {
        const int j = jc + lane;
        const bool jok = j < J;
        const T rj = sr[jok ? j : J - 1];
        int bg = 0;
        for (int step = top; step > 0; step >>= 1) {
          const int c = bg + step;
          const Batch<T> rc = sbt[c <= n ? c : n + 1];
          const T Hc = rc.lo - rc.ab * rj;
          bg = (Hc >= rc.upl) ? c : bg;
        }
        const Batch<T> r = sbt[bg > 0 ? bg : n + 1];
        const T Phi = r.ab * rj;
        const T H = r.lo - Phi;
        const bool feas = jok & (bg >= blo) & (H >= tfree);
        const uint64_t fm = __builtin_amdgcn_ballot_w64(feas);
        if (fm == 0) continue;
        const int bw = __builtin_amdgcn_readlane(bg, 63 - __clzll((long long)fm));
        const T cpu =
            offload_cpu_energy<T, CONT, LG>(smem, y, K, feas ? H : inf_of<T>(), bg, 0, bw);
        const T E = fma_(sP[jok ? j : J - 1], Phi, cpu + r.esl);
        const int idx = sJN + (J - 1 - j) * n + (n - bg);
        const bool take = feas & better(E, idx, bestE, bestI);
        bestE = take ? E : bestE;
        bestI = take ? idx : bestI;
        if (COUNT) {
          nfeas += feas ? 1 : 0;
          nevals += feas ? bg : 0;
        }
      }
    } else {
      for (int b0 = blo; b0 <= n; b0 += nb) {
        bool anyp = false;
        for (int jc = 0; jc < Jn; jc += WAVE) {
          const int j = j_low + jc + jl;
          const bool jok = !idle && j < J;
          const int b = b0 + bo;
          const Batch<T> r = sbt[b0 + bo];
          const T Phi = r.ab * sr[jok ? j : J - 1];            // Eq. (5), layers s+1..L
          const T H = r.lo - Phi;                               // slack to the batch deadline
          const bool feas = jok & (H >= tfree) & (H >= r.upl);  // (6), (7); (8): b >= bmin
          const uint64_t fm = __builtin_amdgcn_ballot_w64(feas);
          if (fm == 0) continue;
          anyp = true;
          const int bw = b0 + __builtin_amdgcn_readlane(bo, 63 - __clzll((long long)fm));
          // every feasible lane of the pass has a batch of at least b0
          const T cpu =
              offload_cpu_energy<T, CONT, LG>(smem, y, K, feas ? H : inf_of<T>(), b, b0, bw);
          const T E = fma_(sP[jok ? j : J - 1], Phi, cpu + r.esl);
          const int idx = sJN + (J - 1 - j) * n + (n - b);
          const bool take = feas & better(E, idx, bestE, bestI);
          bestE = take ? E : bestE;
          bestI = take ? idx : bestI;
          if (COUNT) {
            nfeas += feas ? 1 : 0;
            nevals += feas ? b : 0;
          }
        }
        if (!anyp) break;
      }
    }
  }
}

// Local computing of the users in mask: whether every one of them meets
// its deadline locally (8), and their local energies summed for ranking
// (any order).  Both wave-uniform.
template <typename T>
__device__ inline bool hlocal(const unsigned char *smem, const HLayout &y, int lane, uint64_t mask,
                              T *e) {
  const int *skL = (const int *)(smem + y.kL);
  const T *seL = (const T *)(smem + y.eL);
  const bool mem = (mask >> lane) & 1;
  const bool ok = __builtin_amdgcn_ballot_w64(mem && skL[lane] < 0) == 0;
  T v = mem ? seL[lane] : T(0);
  for (int d = 1; d < WAVE; d <<= 1) v = v + __shfl_xor(v, d, WAVE);
  *e = uni(v);
  return ok;
}

// The winner idx of the users in mask (n of them; idx = L*J*n is local
// computing) with the GPU free at tfree: each member's choice from
// correctly rounded operations in the oracle's order, the energy summed
// over the members in user index order (Eq. (21)), the release time (Eq.
// (22)); each member's level, offload flag, group and frequency are stored
// through uo where its pointers are set.
template <typename T, bool CONT>
__device__ void hwinner(const HProblem<T> &p, int64_t inst, unsigned char *smem, const HLayout &y,
                        int lane, uint64_t mask, int n, int idx, T tfree, T &E, T &tf,
                        const UserOut<T> &uo, T *slack = nullptr, T *rdy = nullptr,
                        T *phi = nullptr) {
  const int L = p.L, K = p.K, J = p.J;
  const int *skL = (const int *)(smem + y.kL);
  const T *seL = (const T *)(smem + y.eL), *sfL = (const T *)(smem + y.fL);
  T *sterm = (T *)(smem + y.term);
  const bool mem = (mask >> lane) & 1;
  if (idx == L * J * n) {  // local computing
    if (mem) {
      sterm[lane] = seL[lane];
      if (uo.level) {
        uo.level[lane] = (int8_t)(CONT ? -1 : skL[lane]);
        uo.offload[lane] = 0;
        if (uo.group) uo.group[lane] = (int8_t)uo.gno;
        if (uo.freq) uo.freq[lane] = sfL[lane];
      }
    }
    __syncthreads();
    T acc = T(0);
    for (uint64_t mm = mask; mm; mm &= mm - 1) acc = acc + sterm[__builtin_ctzll(mm)];
    E = acc;
    tf = tfree;
    if (slack) *slack = inf_of<T>();
    if (rdy) *rdy = -inf_of<T>();
    if (phi) *phi = T(0);
    __syncthreads();
    return;
  }
  const int s = idx / (J * n);
  const int rem = idx - s * (J * n);
  const int j = J - 1 - rem / n;
  const int b = n - (rem - (rem / n) * n);
  bool any;
  hrow<T, CONT>(p, inst, smem, y, lane, s, tfree, mask, n, &any, true);
  const T *sC = (const T *)(smem + y.C), *sA = (const T *)(smem + y.A);
  const T *sB = (const T *)(smem + y.B), *slf = (const T *)(smem + y.lf);
  const T *szet = (const T *)(smem + y.zet), *skap = (const T *)(smem + y.kap);
  const T *sptx = (const T *)(smem + y.ptx), *srate = (const T *)(smem + y.rate);
  const T *sr = (const T *)(smem + y.r), *sP = (const T *)(smem + y.P);
  const int *spi = (const int *)(smem + y.pi);
  const Batch<T> *sbt = (const Batch<T> *)(smem + y.bt);
  const T Cs = sC[s];
  const T Phi = (sA[s] + sB[s] * T(b)) * sr[j];
  const T H = sbt[b].lo - Phi;
  T ready = -inf_of<T>();  // the latest offloader, the GPU free time joins below
  if (mem) {
    const int m = lane;
    int pos = 0;
    for (int q = 0; q < n; ++q) pos += (spi[q] == m) ? q : 0;
    int lv;
    int8_t off;
    T fq;
    if (pos < b) {
      const T up = ((const T *)(smem + y.bits))[s] / srate[m];
      const T x = H - up;
      const T W = szet[m] * Cs;
      const T *f = slf + m * K;
      int k = K - 1;
      for (int q = K - 1; q >= 0; --q)
        if (W / f[q] <= x) k = q;
      fq = CONT ? cont_freq(W, x, f[0], f[K - 1]) : f[k];
      const T e = (skap[m] * (fq * fq)) * Cs;
      sterm[m] = e + sptx[m] * up;
      const T done = W / fq + up;
      ready = (done > ready) ? done : ready;
      lv = CONT ? -1 : k;
      off = 1;
    } else {
      sterm[m] = seL[m];
      lv = CONT ? -1 : skL[m];
      fq = sfL[m];
      off = 0;
    }
    if (uo.level) {
      uo.level[m] = (int8_t)lv;
      uo.offload[m] = off;
      if (uo.group) uo.group[m] = (int8_t)uo.gno;
      if (uo.freq) uo.freq[m] = fq;
    }
  }
  ready = wave_max(ready);
  __syncthreads();
  T acc = T(0);
  for (uint64_t mm = mask; mm; mm &= mm - 1) acc = acc + sterm[__builtin_ctzll(mm)];
  E = acc + sP[j] * Phi;
  tf = ((tfree > ready) ? tfree : ready) + Phi;
  if (slack) *slack = H;
  if (rdy) *rdy = ready;
  if (phi) *phi = Phi;
  __syncthreads();
}

// Eight waves per SIMD: the rows and the level counts wait on LDS and
// barriers; 64 registers fit without spills.  LG > 0: level rows of 2^LG
// entries (launches without the work counters).
template <typename T, bool COUNT, bool GREEDY, bool CONT, int LG = 0>
__global__ __launch_bounds__(WAVE, 8) void jdob_hetero_kernel(HArgs<T> args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x;
  const HProblem<T> &p = args.p;
  const int64_t inst = instance_of_block(args.first);
  const int N = p.N, L = p.L, J = p.J;
  const HLayout y = make_hlayout(N, L, p.K, J, (int)sizeof(T), false);
  const T tfree = p.tfree ? p.tfree[inst] : T(0);
  const uint64_t all = (N == WAVE) ? ~uint64_t(0) : ((uint64_t(1) << N) - 1);

  hprepare<T, CONT>(p, inst, smem, y, lane);
  T bestE = inf_of<T>();
  int bestI = 0x7fffffff, nfeas = 0;
  int64_t nevals = 0;
  // (binary32 with rows of at most 16 levels: otherwise the run's registers
  // would spill)
  hsearch<T, COUNT, GREEDY, CONT, LG, (LG <= 4 && sizeof(T) == 4)>(
      p, inst, smem, y, lane, all, N, tfree, bestE, bestI, nfeas, nevals);
  // local computing competes last
  const int idxLC = L * J * N;
  wave_argmin(bestE, bestI);
  T eLC;
  if (hlocal<T>(smem, y, lane, all, &eLC)) {
    nfeas += (lane == 0) ? 1 : 0;
    if (better(eLC, idxLC, bestE, bestI)) { bestE = eLC; bestI = idxLC; }
  }
  const int64_t totfeas = wave_sum_i64((int64_t)nfeas);
  const int64_t totev = wave_sum_i64(nevals);

  const auto *a = hargs<T>();
  if (lane == 0) {
    if (a->out.nfeas) a->out.nfeas[inst] = (int32_t)totfeas;
    if (a->out.nevals) a->out.nevals[inst] = totev;
  }
  UserOut<T> uo;
  uo.level = a->out.ulevel + inst * N;
  uo.offload = a->out.uoffload + inst * N;
  uo.group = nullptr;
  uo.freq = a->out.ufreq ? a->out.ufreq + inst * N : nullptr;
  uo.gno = 0;
  if (bestI == 0x7fffffff) {  // nothing feasible
    if (lane == 0) {
      a->out.status[inst] = 1;
      a->out.cut[inst] = -1;
      a->out.gpu_level[inst] = -1;
      a->out.batch[inst] = 0;
      a->out.energy[inst] = inf_of<T>();
      a->out.tfree_out[inst] = inf_of<T>();
    }
    if (lane < N) {
      uo.level[lane] = -1;
      uo.offload[lane] = 0;
      if (uo.freq) uo.freq[lane] = T(0);
    }
    return;
  }
  T E, tf;
  hwinner<T, CONT>(p, inst, smem, y, lane, all, N, bestI, tfree, E, tf, uo);
  if (lane == 0) {
    int s = L, j = -1, b = 0;
    if (bestI != idxLC) {
      s = bestI / (J * N);
      const int rem = bestI - s * (J * N);
      j = J - 1 - rem / N;
      b = N - (rem - (rem / N) * N);
    }
    a->out.status[inst] = 0;
    a->out.cut[inst] = s;
    a->out.gpu_level[inst] = j;
    a->out.batch[inst] = b;
    a->out.energy[inst] = E;
    a->out.tfree_out[inst] = tf;
  }
}

// Outer grouping with heterogeneous users: users by deadline (ties: lower
// index), consecutive groups served in order, each group one search over
// its members with the GPU free at the previous group's release time.  The
// dynamic program keeps, per prefix of the deadline order, the front of
// non-dominated (total energy, GPU release time) states, as the other
// grouping kernel does.  Six waves per SIMD: with the 76-80 vector and 106
// scalar registers that allows, nothing spills (at eight waves 20-60 bytes
// per lane went to scratch and scalar values were kept in vector lanes;
// measured on h5: 30.9 ms at six waves, 31.2 at seven, 32.3 at eight).
template <typename T, bool COUNT, bool GREEDY, bool CONT>
__global__ __launch_bounds__(WAVE, 6) void jdob_hetero_grouped_kernel(HGArgs<T> args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x;
  const HProblem<T> &p = args.p;
  const int64_t inst = instance_of_block(args.first);
  const int N = p.N, L = p.L, J = p.J;
  const HLayout y = make_hlayout(N, L, p.K, J, (int)sizeof(T), true);
  const T *sdl = (const T *)(smem + y.dl);
  int *dr = (int *)(smem + y.drank), *dord = (int *)(smem + y.dord);
  int *fn = (int *)(smem + y.fn), *ends = (int *)(smem + y.ends), *eks = (int *)(smem + y.eks);
  T *fE = (T *)(smem + y.fE), *fT = (T *)(smem + y.fT);
  int16_t *from = (int16_t *)(smem + y.from);
  constexpr int F = GROUP_FRONT;

  hprepare<T, CONT>(p, inst, smem, y, lane);
  if (y.pre >= 0 && lane < N) {  // per (s, user), as hrow computes them
    const T *sC = (const T *)(smem + y.C), *szet = (const T *)(smem + y.zet);
    const T *slf = (const T *)(smem + y.lf), *srate = (const T *)(smem + y.rate);
    const T *sbits = (const T *)(smem + y.bits);
    T *pre = (T *)(smem + y.pre);
    for (int s = 0; s < p.s_end; ++s) {
      const T W = szet[lane] * sC[s];
      const T tK1 = W / slf[lane * p.K + p.K - 1];
      const T up = sbits[s] / srate[lane];
      T *q = pre + (s * N + lane) * 3;
      q[0] = up;
      q[1] = tK1;
      q[2] = slack_needed(tK1, up);
    }
  }
  if (lane < N) {  // the deadline order
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

  // users at deadline ranks [lo, hi) as a lane mask
  auto members = [&](int lo, int hi) -> uint64_t {
    const int r = dr[lane < N ? lane : 0];
    return __builtin_amdgcn_ballot_w64(lane < N && r >= lo && r < hi);
  };
  // the group's winner among its candidates and local computing, with the
  // GPU free at tf0 (0x7fffffff if none is feasible); counts into nf, ne
  auto group_search = [&](uint64_t mask, int n, T tf0, int &nf, int64_t &ne) -> int {
    T bestE = inf_of<T>();
    int bestI = 0x7fffffff;
    hsearch<T, COUNT, GREEDY, CONT>(p, inst, smem, y, lane, mask, n, tf0, bestE, bestI, nf, ne);
    wave_argmin(bestE, bestI);
    T eLC;
    if (hlocal<T>(smem, y, lane, mask, &eLC)) {
      if (COUNT) nf += (lane == 0) ? 1 : 0;
      if (better(eLC, L * J * n, bestE, bestI)) { bestE = eLC; bestI = L * J * n; }
    }
    return uni(bestI);
  };

  int nfeas = 0;
  int64_t nevals = 0, ninner = 0;
  const UserOut<T> none{nullptr, nullptr, nullptr, nullptr, 0};
  for (int i = 1; i <= N; ++i) {
    int ni = 0;  // states in the front of prefix i
    for (int j = 0; j < i; ++j) {  // last group: users at deadline ranks j..i-1
      const int nj = uni(fn[j]);
      if (nj == 0) continue;
      const int n = i - j;
      const uint64_t mask = members(j, i);
      // the states of prefix j from the earliest release on; a winner whose
      // slack meets a later state's free time is that state's winner too
      // (constraint (6) is its only test that depends on the free time)
      int k = nj - 1;
      while (k >= 0) {
        const T tf0 = uni(fT[j * F + k]);
        const int idx = group_search(mask, n, tf0, nfeas, nevals);
        ++ninner;
        if (idx == 0x7fffffff) break;  // the states left free the GPU later still
        T Eg, Tg, H, rd, Ph;
        hwinner<T, CONT>(p, inst, smem, y, lane, mask, n, idx, tf0, Eg, Tg, none, &H, &rd, &Ph);
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

  const auto *a = hgargs<T>();
  const int64_t o = inst * N;
  for (int q = lane; q < N; q += WAVE) {
    a->out.order[o + q] = (int16_t)dord[q];
    a->out.group_end[o + q] = 0;
    a->out.group_cut[o + q] = -1;
    a->out.group_gpu_level[o + q] = -1;
    a->out.group_batch[o + q] = 0;
    a->out.group_energy[o + q] = inf_of<T>();
    a->out.group_tfree[o + q] = inf_of<T>();
    a->out.ulevel[o + q] = -1;
    a->out.uoffload[o + q] = 0;
    a->out.ugroup[o + q] = -1;
    if (a->out.ufreq) a->out.ufreq[o + q] = T(0);
  }
  const int64_t totfeas = wave_sum_i64((int64_t)nfeas);
  const int64_t totev = wave_sum_i64(nevals);
  if (lane == 0) {
    if (a->out.ninner) a->out.ninner[inst] = ninner;
    if (a->out.nfeas) a->out.nfeas[inst] = totfeas;
    if (a->out.nevals) a->out.nevals[inst] = totev;
  }
  if (uni(fn[N]) == 0) {
    if (lane == 0) {
      a->out.status[inst] = 1;
      a->out.num_groups[inst] = 0;
      a->out.energy[inst] = inf_of<T>();
      a->out.tfree_out[inst] = inf_of<T>();
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
  UserOut<T> uo;
  uo.level = a->out.ulevel + o;
  uo.offload = a->out.uoffload + o;
  uo.group = a->out.ugroup + o;
  uo.freq = a->out.ufreq ? a->out.ufreq + o : nullptr;
  int start = 0;
  for (int gno = 0; gno < G; ++gno) {
    const int b = uni(ends[gno]), n = b - start;
    const uint64_t mask = members(start, b);
    const T tf0 = uni(fT[from[uni(eks[gno])]]);
    int nf = 0;
    int64_t ne = 0;
    const int idx = group_search(mask, n, tf0, nf, ne);
    uo.gno = gno;
    T Eg, Tg;
    hwinner<T, CONT>(p, inst, smem, y, lane, mask, n, idx, tf0, Eg, Tg, uo);
    if (lane == 0) {
      int s = L, jg = -1, bb = 0;
      if (idx != L * J * n) {
        s = idx / (J * n);
        const int rem = idx - s * (J * n);
        jg = J - 1 - rem / n;
        bb = n - (rem - (rem / n) * n);
      }
      a->out.group_end[o + gno] = (int16_t)b;
      a->out.group_cut[o + gno] = s;
      a->out.group_gpu_level[o + gno] = jg;
      a->out.group_batch[o + gno] = bb;
      a->out.group_energy[o + gno] = Eg;
      a->out.group_tfree[o + gno] = Tg;
    }
    start = b;
  }
  if (lane == 0) {
    a->out.status[inst] = 0;
    a->out.num_groups[inst] = G;
    a->out.energy[inst] = fE[N * F];
    a->out.tfree_out[inst] = fT[N * F];
  }
}

template <typename T> HProblem<T> to_hproblem(const jdob_problem *q) {
  HProblem<T> p;
  p.cyc = (const T *)q->layer_cycles;
  p.bits = (const T *)q->out_bits;
  p.alpha = (const T *)q->gpu_alpha;
  p.beta = (const T *)q->gpu_beta;
  p.rate = (const T *)q->uplink_rate;
  p.deadline = (const T *)q->deadline;
  p.tfree = (const T *)q->t_free;
  p.lf = (const T *)q->local_freq;
  p.gf = (const T *)q->gpu_freq;
  p.uzeta = (const T *)q->user_zeta;
  p.ukappa = (const T *)q->user_kappa;
  p.uptx = (const T *)q->user_p_tx;
  p.ulf = (const T *)q->user_local_freq;
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
  return p;
}

template <typename T> int launch_typed(const jdob_problem *q, const jdob_policy *o, hipStream_t stream) {
  HArgs<T> a;
  a.p = to_hproblem<T>(q);
  HPolicy<T> &r = a.out;
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
  const bool greedy = (q->mode & JDOB_MODE_GREEDY) != 0;
  const bool cont = (q->mode & JDOB_MODE_CONTINUOUS_CPU) != 0;
  const bool count = r.nfeas != nullptr || r.nevals != nullptr;
  const size_t lds = (size_t)make_hlayout(a.p.N, a.p.L, a.p.K, a.p.J, (int)sizeof(T), false).total;
  const int64_t I = q->num_instances;
  const dim3 block(WAVE);
  for (int64_t first = 0; first < I; first += MAX_BLOCKS_PER_LAUNCH) {
    const int64_t n = (I - first < MAX_BLOCKS_PER_LAUNCH) ? I - first : MAX_BLOCKS_PER_LAUNCH;
    const dim3 grid((unsigned)n);
    a.first = first;
#define JDOB_HLAUNCH(CN, GR, CT) \
  hipLaunchKernelGGL((jdob_hetero_kernel<T, CN, GR, CT>), grid, block, lds, stream, a)
    if (count) {
      if (greedy) { if (cont) JDOB_HLAUNCH(true, true, true); else JDOB_HLAUNCH(true, true, false); }
      else { if (cont) JDOB_HLAUNCH(true, false, true); else JDOB_HLAUNCH(true, false, false); }
    } else if (cont) {
      if (greedy) JDOB_HLAUNCH(false, true, true);
      else JDOB_HLAUNCH(false, false, true);
    } else {
      // level rows of K4 = 2^lg entries, 4 <= K4 <= 64 (K <= JDOB_MAX_LOCAL_LEVELS)
      static_assert(JDOB_MAX_LOCAL_LEVELS <= 64, "hetero level rows of at most 2^6 entries");
#define JDOB_HLG(G)                                                                         \
  case G:                                                                                   \
    if (greedy)                                                                             \
      hipLaunchKernelGGL((jdob_hetero_kernel<T, false, true, false, G>), grid, block, lds,  \
                         stream, a);                                                        \
    else                                                                                    \
      hipLaunchKernelGGL((jdob_hetero_kernel<T, false, false, false, G>), grid, block, lds, \
                         stream, a);                                                        \
    break;
      switch (__builtin_ctz((unsigned)make_hlayout(a.p.N, a.p.L, a.p.K, a.p.J, (int)sizeof(T),
                                                   false).K4)) {
        JDOB_HLG(2) JDOB_HLG(3) JDOB_HLG(4) JDOB_HLG(5) JDOB_HLG(6)
        default: return JDOB_ERR_UNSUPPORTED;
      }
#undef JDOB_HLG
    }
#undef JDOB_HLAUNCH
    if (hipGetLastError() != hipSuccess) return JDOB_ERR_HIP;
  }
  return JDOB_OK;
}

template <typename T>
int launch_grouped_typed(const jdob_problem *q, const jdob_grouped_policy *o, hipStream_t stream) {
  HGArgs<T> a;
  a.p = to_hproblem<T>(q);
  HGrouped<T> &g = a.out;
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
  const bool greedy = (q->mode & JDOB_MODE_GREEDY) != 0;
  const bool cont = (q->mode & JDOB_MODE_CONTINUOUS_CPU) != 0;
  const bool count = g.ninner != nullptr || g.nfeas != nullptr || g.nevals != nullptr;
  const size_t lds = (size_t)make_hlayout(a.p.N, a.p.L, a.p.K, a.p.J, (int)sizeof(T), true).total;
  const int64_t I = q->num_instances;
  const dim3 block(WAVE);
  for (int64_t first = 0; first < I; first += MAX_BLOCKS_PER_LAUNCH) {
    const int64_t n = (I - first < MAX_BLOCKS_PER_LAUNCH) ? I - first : MAX_BLOCKS_PER_LAUNCH;
    const dim3 grid((unsigned)n);
    a.first = first;
#define JDOB_HLAUNCH(CN, GR, CT) \
  hipLaunchKernelGGL((jdob_hetero_grouped_kernel<T, CN, GR, CT>), grid, block, lds, stream, a)
    if (count) {
      if (greedy) { if (cont) JDOB_HLAUNCH(true, true, true); else JDOB_HLAUNCH(true, true, false); }
      else { if (cont) JDOB_HLAUNCH(true, false, true); else JDOB_HLAUNCH(true, false, false); }
    } else {
      if (greedy) { if (cont) JDOB_HLAUNCH(false, true, true); else JDOB_HLAUNCH(false, true, false); }
      else { if (cont) JDOB_HLAUNCH(false, false, true); else JDOB_HLAUNCH(false, false, false); }
    }
#undef JDOB_HLAUNCH
    if (hipGetLastError() != hipSuccess) return JDOB_ERR_HIP;
  }
  return JDOB_OK;
}

}  // namespace

bool has_user_params(const jdob_problem *p) {
  return p->user_zeta || p->user_kappa || p->user_p_tx || p->user_local_freq;
}

// Checks beyond the shared ones (done before): the user count and the LDS
// the instance needs.
int validate_hetero(const jdob_problem *p, bool grouped) {
  if (p->num_users > JDOB_MAX_HETERO_USERS) return JDOB_ERR_UNSUPPORTED;
  const int sz = p->dtype == JDOB_F64 ? 8 : 4;
  if (make_hlayout(p->num_users, p->num_layers, p->num_local_levels, p->num_gpu_levels, sz,
                   grouped)
          .total > LDS_LIMIT)
    return JDOB_ERR_UNSUPPORTED;
  return JDOB_OK;
}

int launch_hetero(const jdob_problem *p, const jdob_policy *o, hipStream_t stream) {
  return p->dtype == JDOB_F64 ? launch_typed<double>(p, o, stream) : launch_typed<float>(p, o, stream);
}

int launch_hetero_grouped(const jdob_problem *p, const jdob_grouped_policy *o, hipStream_t stream) {
  return p->dtype == JDOB_F64 ? launch_grouped_typed<double>(p, o, stream)
                              : launch_grouped_typed<float>(p, o, stream);
}

}  // namespace jdob_dev
