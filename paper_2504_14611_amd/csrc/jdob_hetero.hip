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

// Per offloader at the current partition point, read together: its upload
// latency, its work zeta*C[s], its frequency range (continuous mode).
template <typename T> struct alignas(4 * sizeof(T)) HUser { T up, z, fmin, fmax; };

// Byte offsets of the per-instance LDS arrays.
struct HLayout {
  int cyc, al, be, C, A, B, r, P;                 // layers and GPU levels
  int rate, dl, zet, kap, ptx, lf, kL, eL, fL;    // per user (index m)
  int gam, need;                                  // per user, current s
  int pi, usr, kc, lv, bt, term;                  // per position in pi_s
  int K4, total;
};

__host__ __device__ inline HLayout make_hlayout(int N, int L, int K, int J, int szT) {
  HLayout y;
  int o = 0;
  auto take = [&](int bytes) { int r = o; o = align8(o + bytes); return r; };
  auto take32 = [&](int bytes) { o = (o + 31) & ~31; int r = o; o = align8(o + bytes); return r; };
  y.K4 = (K + 3) & ~3;
  y.cyc = take(L * szT);
  y.al = take(L * szT);
  y.be = take(L * szT);
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
  y.need = take(N * szT);
  y.pi = take(N * 4);
  y.usr = take32((N + 1) * 4 * szT);           // HUser by position (+1: read-ahead)
  y.kc = take(N * szT);                        // kappa * C[s] by position
  y.lv = take32(N * y.K4 * 2 * szT);           // Level rows by position, K4 apart
  y.bt = take32((N + 2 + WAVE) * 4 * szT);     // Batch records, b = 1..N (+ sentinels)
  y.term = take(N * szT);
  y.total = o;
  return y;
}

template <typename T> __device__ inline const __attribute__((address_space(4))) HArgs<T> *hargs() {
  return (const __attribute__((address_space(4))) HArgs<T> *)__builtin_amdgcn_kernarg_segment_ptr();
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
// user's local-only choice.  Returns (wave-uniform) whether every user can
// compute locally, and the local energies summed (ranking only) in *eLC.
template <typename T, bool CONT>
__device__ bool hprepare(const HProblem<T> &p, int64_t inst, unsigned char *smem, const HLayout &y,
                         int lane, T *eLC) {
  const int N = p.N, L = p.L, K = p.K, J = p.J;
  T *scyc = (T *)(smem + y.cyc), *sal = (T *)(smem + y.al), *sbe = (T *)(smem + y.be);
  T *sC = (T *)(smem + y.C), *sA = (T *)(smem + y.A), *sB = (T *)(smem + y.B);
  T *sr = (T *)(smem + y.r), *sP = (T *)(smem + y.P);
  T *srate = (T *)(smem + y.rate), *sdl = (T *)(smem + y.dl), *szet = (T *)(smem + y.zet);
  T *skap = (T *)(smem + y.kap), *sptx = (T *)(smem + y.ptx), *slf = (T *)(smem + y.lf);
  int *skL = (int *)(smem + y.kL);
  T *seL = (T *)(smem + y.eL), *sfL = (T *)(smem + y.fL);

  for (int l = lane; l < L; l += WAVE) {
    scyc[l] = p.cyc[inst * L + l];
    sal[l] = p.alpha[inst * L + l];
    sbe[l] = p.beta[inst * L + l];
  }
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
  // C[q+1] = C[q] + cyc[q]; A[q] = A[q+1] + alpha[q]; B likewise (one lane each)
  if (lane < 3) {
    const bool fwd = lane == 0;
    const T *src = fwd ? scyc : (lane == 1 ? sal : sbe);
    T *dst = fwd ? sC : (lane == 1 ? sA : sB);
    const int step = fwd ? 1 : -1;
    int rd = fwd ? 0 : L - 1, wr = fwd ? 1 : L - 1;
    T run = T(0);
    dst[fwd ? 0 : L] = run;
    for (int q = 0; q < L; ++q) {
      run = run + src[rd];
      dst[wr] = run;
      rd += step;
      wr += step;
    }
  }
  __syncthreads();
  // (8) with Eq. (20): the lowest level finishing every layer by the deadline
  int bad = 0;
  T e = T(0);
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
    bad = kL < 0;
    e = eL;
  }
  const bool lc = __builtin_amdgcn_ballot_w64(bad != 0) == 0;
  // ranking only: the order of the sum does not matter
  for (int d = 1; d < WAVE; d <<= 1) e = e + __shfl_xor(e, d, WAVE);
  *eLC = uni(e);
  __syncthreads();
  return lc;
}

// Partition point s: the gamma order pi_s, each offloader's record, the
// batch records b = 1..N and, if the partition point has a feasible
// candidate (the test at the top GPU level and the smallest admissible
// batch; feasibility only falls with b and rises with j), the level rows.
// Returns bmin and sets *any (both wave-uniform).
template <typename T, bool CONT>
__device__ int hrow(const HProblem<T> &p, int64_t inst, unsigned char *smem, const HLayout &y,
                    int lane, int s, T tfree, bool *any) {
  const int N = p.N, L = p.L, K = p.K, K4 = y.K4;
  const T *sC = (const T *)(smem + y.C), *sA = (const T *)(smem + y.A);
  const T *sB = (const T *)(smem + y.B);
  const T *srate = (const T *)(smem + y.rate), *sdl = (const T *)(smem + y.dl);
  const T *szet = (const T *)(smem + y.zet), *skap = (const T *)(smem + y.kap);
  const T *sptx = (const T *)(smem + y.ptx), *slf = (const T *)(smem + y.lf);
  const int *skL = (const int *)(smem + y.kL);
  const T *seL = (const T *)(smem + y.eL);
  T *sgam = (T *)(smem + y.gam), *sneed = (T *)(smem + y.need);
  int *spi = (int *)(smem + y.pi);
  HUser<T> *susr = (HUser<T> *)(smem + y.usr);
  T *skc = (T *)(smem + y.kc);
  Level<T> *slv = (Level<T> *)(smem + y.lv);
  Batch<T> *sbt = (Batch<T> *)(smem + y.bt);

  const T Cs = sC[s];
  T up = T(0), W = T(0), tK1 = T(0);
  if (lane < N) {
    W = szet[lane] * Cs;                               // cycles of layers 1..s
    tK1 = W / slf[lane * K + K - 1];                   // Eq. (1) at the top level
    up = p.bits[inst * (L + 1) + s] / srate[lane];     // Eq. (3)
    sgam[lane] = up + tK1;                             // Eq. (17)
  }
  __syncthreads();
  int pos = 0;
  if (lane < N) {
    const T g = sgam[lane];
    for (int q = 0; q < N; ++q) {
      const T gq = sgam[q];
      pos += (gq < g || (gq == g && q < lane)) ? 1 : 0;
    }
    spi[pos] = lane;
    HUser<T> u;
    u.up = up;
    u.z = W;
    u.fmin = slf[lane * K];
    u.fmax = slf[lane * K + K - 1];
    susr[pos] = u;
    skc[pos] = skap[lane] * Cs;
    sneed[pos] = slack_needed(tK1, up);
  }
  if (lane == 0) {  // read-ahead entry past the last user
    HUser<T> z;
    z.up = T(0);
    z.z = T(0);
    z.fmin = T(0);
    z.fmax = T(0);
    susr[N] = z;
  }
  __syncthreads();
  // along pi_s (lane = position): lo = prefix min of deadlines (Eq. (10)),
  // the prefix max of need, bmin, the upload energy EU and the local
  // energies SL of the others (ranking only)
  // (scans over the N positions only)
  const bool in = lane < N;
  const int m = in ? spi[lane] : 0;
  T lo = in ? sdl[m] : inf_of<T>(), nd = in ? sneed[lane] : -inf_of<T>();
  T sl = in ? seL[m] : T(0);
  for (int d = 1; d < N; d <<= 1) {
    const T plo = __shfl_up(lo, d, WAVE), pnd = __shfl_up(nd, d, WAVE);
    const T nsl = __shfl_down(sl, d, WAVE);
    if (lane >= d) {                   // prefix min of deadlines, prefix max of need
      lo = (plo < lo) ? plo : lo;
      nd = (pnd > nd) ? pnd : nd;
    }
    sl = sl + ((lane + d < N) ? nsl : T(0));  // suffix sum: positions above
  }
  const uint64_t nolocal = __builtin_amdgcn_ballot_w64(in && skL[m] < 0);
  const int bmin = nolocal ? 64 - __clzll((long long)nolocal) : 0;
  const T eu = scan_add(in ? sptx[m] * susr[lane].up : T(0));
  const T slnext = __shfl_down(sl, 1, WAVE);  // sum over positions > lane
  if (in) {
    Batch<T> r;
    r.lo = lo;
    r.upl = nd;
    r.esl = eu + ((lane + 1 < N) ? slnext : T(0));
    r.ab = sA[s] + sB[s] * T(lane + 1);
    sbt[lane + 1] = r;
  }
  for (int q = lane; q < WAVE + 1; q += WAVE) {  // past N: infeasible sentinels
    Batch<T> z;
    z.lo = -inf_of<T>();
    z.upl = T(0);
    z.esl = T(0);
    z.ab = T(0);
    sbt[N + 1 + q] = z;
  }
  __syncthreads();
  const int bm = bmin;
  const int blo = bm > 1 ? bm : 1;
  bool ok = false;
  if (blo <= N) {
    const Batch<T> r = sbt[blo];
    const T H = r.lo - r.ab * ((const T *)(smem + y.r))[p.J - 1];
    ok = (H >= tfree) && (H >= r.upl);
  }
  *any = ok;
  if (!CONT && ok) {
    // Eqs. (1), (2) per (position, level): K4 lanes per user, padding never
    // too slow
    const int upw = WAVE / K4, pk = lane / K4, kk = lane - pk * K4;
    for (int p0 = 0; p0 < N; p0 += upw) {
      const int q = p0 + pk;
      if (pk < upw && q < N) {
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
  return bm;
}

// The CPU energy of a lane's offloaders 0..b-1 for ranking, given its slack
// Hu (+inf on infeasible lanes, whose sum is dropped): the wave walks users
// 0..bw-1, users past the lane's batch add nothing.
template <typename T, bool CONT>
__device__ inline T offload_cpu_energy(const unsigned char *smem, const HLayout &y, int K, T Hu,
                                       int b, int bw) {
  const HUser<T> *susr = (const HUser<T> *)(smem + y.usr);
  const T *skc = (const T *)(smem + y.kc);
  const Level<T> *slv = (const Level<T> *)(smem + y.lv);
  const int K4 = y.K4;
  T acc = T(0);
  for (int g = 0; g < bw; ++g) {
    const HUser<T> u = susr[g];
    const T x = Hu - u.up;
    T e;
    if (CONT) {  // Eq. (20) with its clamp, in the user's own range
      const T f = clamp_(u.z * fast_rcp(x), u.fmin, u.fmax);
      e = (skc[g] * f) * f;
    } else {     // Eq. (20): levels too slow for the budget are a prefix,
      // counted two levels per broadcast read (a binary search with
      // per-lane reads was slower: its reads depend on each other)
      const Quad<T> *row = (const Quad<T> *)(slv + g * K4);
      int k = 0;
      for (int q = 0; q < K4 / 2; ++q) {
        const Quad<T> v = row[q];  // (t, e) of two levels
        k += (v.v[0] > x) ? 1 : 0;
        k += (v.v[2] > x) ? 1 : 0;
      }
      k = k < K ? k : K - 1;
      e = slv[g * K4 + k].e;
    }
    acc = (g < b) ? acc + e : acc;
  }
  return acc;
}

template <typename T, bool COUNT, bool GREEDY, bool CONT>
__global__ __launch_bounds__(WAVE, 4) void jdob_hetero_kernel(HArgs<T> args) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x;
  const HProblem<T> &p = args.p;
  const int64_t inst = instance_of_block(args.first);
  const int N = p.N, L = p.L, K = p.K, J = p.J;
  const int s_end = p.s_end, j_low = p.j_low;
  const HLayout y = make_hlayout(N, L, K, J, (int)sizeof(T));
  const T *sr = (const T *)(smem + y.r), *sP = (const T *)(smem + y.P);
  const Batch<T> *sbt = (const Batch<T> *)(smem + y.bt);
  const T tfree = p.tfree ? p.tfree[inst] : T(0);

  T eLC;
  const bool lc = hprepare<T, CONT>(p, inst, smem, y, lane, &eLC);
  T bestE = inf_of<T>();
  int bestI = 0x7fffffff, nfeas = 0;
  int64_t nevals = 0;
  const int Jn = J - j_low;
  const int Jw = Jn < WAVE ? Jn : WAVE;
  const int nb = WAVE / Jw;
  const int jl = lane % Jw, bo = lane / Jw;
  const int bo_rec = (bo < nb) ? bo : WAVE;  // idle lanes read a sentinel

  for (int s = 0; s < s_end; ++s) {
    bool any;
    const int bmin = hrow<T, CONT>(p, inst, smem, y, lane, s, tfree, &any);
    const int blo = bmin > 1 ? bmin : 1;
    if (!any) continue;
    const int sJN = s * J * N;
    if (GREEDY) {
      // Alg. 2 at each GPU level (lane = j): the largest set whose users all
      // meet (7) at their top frequency; the test fails more as b grows
      const int top = 1 << (31 - __clz(N));
      for (int jc = j_low; jc < J; jc += WAVE) {
        const int j = jc + lane;
        const bool jok = j < J;
        const T rj = sr[jok ? j : J - 1];
        int bg = 0;
        for (int step = top; step > 0; step >>= 1) {
          const int c = bg + step;
          const Batch<T> rc = sbt[c <= N ? c : N + 1];
          const T Hc = rc.lo - rc.ab * rj;
          bg = (Hc >= rc.upl) ? c : bg;
        }
        const Batch<T> r = sbt[bg > 0 ? bg : N + 1];
        const T Phi = r.ab * rj;
        const T H = r.lo - Phi;
        const bool feas = jok & (bg >= blo) & (H >= tfree);
        const uint64_t mask = __builtin_amdgcn_ballot_w64(feas);
        if (mask == 0) continue;
        const int bw = __builtin_amdgcn_readlane(bg, 63 - __clzll((long long)mask));
        const T cpu = offload_cpu_energy<T, CONT>(smem, y, K, feas ? H : inf_of<T>(), bg, bw);
        const T E = fma_(sP[jok ? j : J - 1], Phi, cpu + r.esl);
        const int idx = sJN + (J - 1 - j) * N + (N - bg);
        const bool take = feas & better(E, idx, bestE, bestI);
        bestE = take ? E : bestE;
        bestI = take ? idx : bestI;
        if (COUNT) {
          nfeas += feas ? 1 : 0;
          nevals += feas ? bg : 0;
        }
      }
    } else {
      for (int b0 = blo; b0 <= N; b0 += nb) {
        bool any = false;
        for (int jc = 0; jc < Jn; jc += WAVE) {
          const int j = j_low + jc + jl;
          const bool jok = j < J;
          const int b = b0 + bo;
          const Batch<T> r = sbt[b0 + bo_rec];
          const T Phi = r.ab * sr[jok ? j : J - 1];          // Eq. (5), layers s+1..L
          const T H = r.lo - Phi;                             // slack to the batch deadline
          const bool feas = jok & (H >= tfree) & (H >= r.upl);  // (6), (7); (8): b >= bmin
          const uint64_t mask = __builtin_amdgcn_ballot_w64(feas);
          if (mask == 0) continue;
          any = true;
          const int bw = b0 + __builtin_amdgcn_readlane(bo, 63 - __clzll((long long)mask));
          const T cpu = offload_cpu_energy<T, CONT>(smem, y, K, feas ? H : inf_of<T>(), b, bw);
          const T E = fma_(sP[jok ? j : J - 1], Phi, cpu + r.esl);
          const int idx = sJN + (J - 1 - j) * N + (N - b);
          const bool take = feas & better(E, idx, bestE, bestI);
          bestE = take ? E : bestE;
          bestI = take ? idx : bestI;
          if (COUNT) {
            nfeas += feas ? 1 : 0;
            nevals += feas ? b : 0;
          }
        }
        if (!any) break;
      }
    }
  }

  // local computing competes last
  const int idxLC = L * J * N;
  wave_argmin(bestE, bestI);
  if (lc) {
    nfeas += (lane == 0) ? 1 : 0;
    if (better(eLC, idxLC, bestE, bestI)) { bestE = eLC; bestI = idxLC; }
  }
  const int64_t totfeas = wave_sum_i64((int64_t)nfeas);
  const int64_t totev = wave_sum_i64(nevals);

  const auto *a = hargs<T>();
  int8_t *ul = a->out.ulevel + inst * N;
  int8_t *uo = a->out.uoffload + inst * N;
  T *uf = a->out.ufreq ? a->out.ufreq + inst * N : nullptr;
  if (lane == 0) {
    if (a->out.nfeas) a->out.nfeas[inst] = (int32_t)totfeas;
    if (a->out.nevals) a->out.nevals[inst] = totev;
  }
  const int *skL = (const int *)(smem + y.kL);
  const T *seL = (const T *)(smem + y.eL), *sfL = (const T *)(smem + y.fL);
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
      ul[lane] = -1;
      uo[lane] = 0;
      if (uf) uf[lane] = T(0);
    }
    return;
  }
  if (bestI == idxLC) {
    if (lane < N) {
      ul[lane] = (int8_t)(CONT ? -1 : skL[lane]);
      uo[lane] = 0;
      if (uf) uf[lane] = sfL[lane];
    }
    if (lane == 0) {
      T acc = T(0);
      for (int m = 0; m < N; ++m) acc = acc + seL[m];
      a->out.status[inst] = 0;
      a->out.cut[inst] = L;
      a->out.gpu_level[inst] = -1;
      a->out.batch[inst] = 0;
      a->out.energy[inst] = acc;
      a->out.tfree_out[inst] = tfree;
    }
    return;
  }

  // the winner (s*, j*, b*): the rows of s*, then each user's choice from
  // correctly rounded operations in the oracle's order
  const int s = bestI / (J * N);
  const int rem = bestI - s * (J * N);
  const int j = J - 1 - rem / N;
  const int b = N - (rem - (rem / N) * N);
  bool any;
  hrow<T, CONT>(p, inst, smem, y, lane, s, tfree, &any);
  const T *sC = (const T *)(smem + y.C), *sA = (const T *)(smem + y.A);
  const T *sB = (const T *)(smem + y.B), *slf = (const T *)(smem + y.lf);
  const T *szet = (const T *)(smem + y.zet), *skap = (const T *)(smem + y.kap);
  const T *sptx = (const T *)(smem + y.ptx), *srate = (const T *)(smem + y.rate);
  const int *spi = (const int *)(smem + y.pi);
  T *sterm = (T *)(smem + y.term);
  const T Cs = sC[s];
  const T Phi = (sA[s] + sB[s] * T(b)) * sr[j];
  const T H = sbt[b].lo - Phi;
  T ready = tfree;
  if (lane < N) {
    const int m = lane;
    int pos = 0;
    for (int q = 0; q < N; ++q) pos += (spi[q] == m) ? q : 0;
    if (pos < b) {
      const T up = p.bits[inst * (L + 1) + s] / srate[m];
      const T x = H - up;
      const T W = szet[m] * Cs;
      const T *f = slf + m * K;
      int k = K - 1;
      for (int q = K - 1; q >= 0; --q)
        if (W / f[q] <= x) k = q;
      T fq, e, tl;
      if (CONT) {
        fq = cont_freq(W, x, f[0], f[K - 1]);
        e = (skap[m] * (fq * fq)) * Cs;
        tl = W / fq;
      } else {
        fq = f[k];
        e = (skap[m] * (fq * fq)) * Cs;
        tl = W / fq;
      }
      ul[m] = (int8_t)(CONT ? -1 : k);
      uo[m] = 1;
      if (uf) uf[m] = fq;
      sterm[m] = e + sptx[m] * up;
      const T done = tl + up;
      ready = (done > ready) ? done : ready;
    } else {
      ul[m] = (int8_t)(CONT ? -1 : skL[m]);
      uo[m] = 0;
      if (uf) uf[m] = sfL[m];
      sterm[m] = seL[m];
    }
  }
  ready = wave_max(ready);
  __syncthreads();
  if (lane == 0) {
    T acc = T(0);
    for (int m = 0; m < N; ++m) acc = acc + sterm[m];
    acc = acc + sP[j] * Phi;
    a->out.status[inst] = 0;
    a->out.cut[inst] = s;
    a->out.gpu_level[inst] = j;
    a->out.batch[inst] = b;
    a->out.energy[inst] = acc;
    a->out.tfree_out[inst] = ready + Phi;
  }
}

template <typename T> int launch_typed(const jdob_problem *q, const jdob_policy *o, hipStream_t stream) {
  HArgs<T> a;
  HProblem<T> &p = a.p;
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
  const size_t lds = (size_t)make_hlayout(p.N, p.L, p.K, p.J, (int)sizeof(T)).total;
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
int validate_hetero(const jdob_problem *p) {
  if (p->num_users > JDOB_MAX_HETERO_USERS) return JDOB_ERR_UNSUPPORTED;
  const int sz = p->dtype == JDOB_F64 ? 8 : 4;
  if (make_hlayout(p->num_users, p->num_layers, p->num_local_levels, p->num_gpu_levels, sz).total >
      LDS_LIMIT)
    return JDOB_ERR_UNSUPPORTED;
  return JDOB_OK;
}

int launch_hetero(const jdob_problem *p, const jdob_policy *o, hipStream_t stream) {
  return p->dtype == JDOB_F64 ? launch_typed<double>(p, o, stream) : launch_typed<float>(p, o, stream);
}

}  // namespace jdob_dev
