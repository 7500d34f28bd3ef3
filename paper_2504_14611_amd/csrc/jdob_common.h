// jdob_common.h — constants and device helpers shared by the kernels of
// libjdob.so (jdob.hip: users sharing their parameters; jdob_hetero.hip:
// heterogeneous users), and the entry of the heterogeneous path.
#ifndef JDOB_COMMON_H
#define JDOB_COMMON_H

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "jdob.h"

namespace jdob_dev {

constexpr int WAVE = 64;
constexpr int64_t MAX_BLOCKS_PER_LAUNCH = int64_t(1) << 24;
constexpr int LDS_LIMIT = 64 * 1024;
constexpr int LDS_PER_CU = 160 * 1024;  // gfx950

__host__ __device__ inline int align8(int x) { return (x + 7) & ~7; }

template <typename T> __device__ inline T inf_of() { return T(INFINITY); }

// Four consecutive row entries, read by one LDS instruction (all lanes read
// the same address: a broadcast).
template <typename T> struct alignas(4 * sizeof(T)) Quad { T v[4]; };

// Local latency and energy of one CPU level (Eqs. (1), (2)), read together.
template <typename T> struct alignas(2 * sizeof(T)) Level { T t, e; };

// What a candidate of batch size b needs from row s, read together: the
// batch deadline lo[b] (Eq. (10)), the largest upload latency of the batch
// up[b-1] (Eq. (3)), EU[b] + SL[b] (upload energy of the batch, Eq. (4), plus
// local energy of the others) and A[s] + B[s]*b (batch latency at the top
// GPU level, Eq. (5)).
template <typename T> struct alignas(4 * sizeof(T)) Batch { T lo, upl, esl, ab; };

// A barrier for LDS that one wave shares among its lanes.  WS: the
// workgroup holds other waves, each with LDS of its own, which need not wait
// (LDS instructions of a wave take effect in program order, so ordering the
// compiler's code is enough); otherwise the workgroup's barrier.
template <bool WS> __device__ inline void lds_sync() {
  if constexpr (WS) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();
  }
}

// The sums of a layer chain in the sequential order of the ABI contract:
// C[0] = 0, C[q+1] = C[q] + cyc[q] (q = 0..L-1) and, when A is given,
// A[L] = 0, A[q] = A[q+1] + alpha[q] and B likewise (q = L-1..0).  The alpha
// and beta rows arrive reversed (ra[i] = alpha[L-1-i], rb[i] = beta[L-1-i]),
// so that lane 0 (cycles), lane 1 (alpha) and lane 2 (beta) all run their
// chains forward, four terms per trip at immediate offsets; lanes 1 and 2
// keep their running sums in place (ra[i] = A[L-1-i]), which are then
// copied out in layer order.  Every lane returns after a barrier.
template <typename T, bool WS = false>
__device__ inline void chain_sums(const T *cyc, T *ra, T *rb, T *C, T *A, T *B, int L,
                                  int lane) {
  if (lane < (A ? 3 : 1)) {
    const T *src = lane == 0 ? cyc : (lane == 1 ? ra : rb);
    T *dst = lane == 0 ? C + 1 : (lane == 1 ? ra : rb);
    T run = T(0);
    int q = 0;
    for (; q + 4 <= L; q += 4) {
      const T x0 = src[q], x1 = src[q + 1], x2 = src[q + 2], x3 = src[q + 3];
      run = run + x0;
      dst[q] = run;
      run = run + x1;
      dst[q + 1] = run;
      run = run + x2;
      dst[q + 2] = run;
      run = run + x3;
      dst[q + 3] = run;
    }
    for (; q < L; ++q) {
      run = run + src[q];
      dst[q] = run;
    }
    if (lane == 0) C[0] = T(0);
  }
  lds_sync<WS>();
  if (A) {
    for (int q = lane; q <= L; q += WAVE) {
      A[q] = q < L ? ra[L - 1 - q] : T(0);
      B[q] = q < L ? rb[L - 1 - q] : T(0);
    }
    lds_sync<WS>();
  }
}

// Lexicographic (energy, flat index) order: the lower energy wins, equal
// energies go to the lower index.
template <typename T>
__device__ inline bool better(T e1, int i1, T e2, int i2) {
  return (e1 < e2) || (e1 == e2 && i1 < i2);
}

// The outer grouping ranks a group ending the deadline order at i by the
// total dpE + E with E the exact (canonically summed) energy of the group's
// winner, which takes a recomputation of that winner.  Its ranking energy Er
// sums the same non-negative terms in another order and grouping (scans,
// runs of equal level, a fused GPU term; with a continuous frequency a
// hardware reciprocal good to an ulp or two): at most about a hundred
// roundings of 2^-24 each in binary32, so Er and E differ by less than 1e-5
// of either.  Rounded addition is monotone, so a total that exceeds the best
// one so far with Er lowered by 1e-4 exceeds it exactly as well: the group
// can neither win nor tie, and its recomputation is skipped.
template <typename T> __device__ inline bool cannot_win(T dpE, T Er, T best) {
  return dpE + Er * T(0.9999) > best;
}

// Lane moves by DPP (data-parallel primitives of the VALU, no LDS round
// trip): row_shr:n inside each row of 16 lanes, row_bcast:15 and
// row_bcast:31 across rows.  Lanes without a source, and rows outside
// RMASK, receive `id`.
template <int CTRL, int RMASK> __device__ inline int dpp_mov(int id, int v) {
  return __builtin_amdgcn_update_dpp(id, v, CTRL, RMASK, 0xf, false);
}
template <int CTRL, int RMASK> __device__ inline float dpp_mov(float id, float v) {
  return __int_as_float(dpp_mov<CTRL, RMASK>(__float_as_int(id), __float_as_int(v)));
}
template <int CTRL, int RMASK> __device__ inline double dpp_mov(double id, double v) {
  const long long qi = __double_as_longlong(id), qv = __double_as_longlong(v);
  const int lo = dpp_mov<CTRL, RMASK>((int)(qi & 0xffffffff), (int)(qv & 0xffffffff));
  const int hi = dpp_mov<CTRL, RMASK>((int)(qi >> 32), (int)(qv >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Inclusive scan over the 64 lanes with an associative, commutative op
// (identity id): Hillis-Steele inside each row of 16, then the row totals.
template <typename V, typename OP> __device__ inline V wave_iscan(V v, V id, OP op) {
  v = op(v, dpp_mov<0x111, 0xf>(id, v));  // row_shr:1
  v = op(v, dpp_mov<0x112, 0xf>(id, v));  // row_shr:2
  v = op(v, dpp_mov<0x114, 0xf>(id, v));  // row_shr:4
  v = op(v, dpp_mov<0x118, 0xf>(id, v));  // row_shr:8
  v = op(v, dpp_mov<0x142, 0xa>(id, v));  // row_bcast:15 into rows 1, 3
  v = op(v, dpp_mov<0x143, 0xc>(id, v));  // row_bcast:31 into rows 2, 3
  return v;
}

__device__ inline int lane_read(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ inline float lane_read(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ inline double lane_read(double v, int l) {
  const long long q = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)(q & 0xffffffff), l);
  const int hi = __builtin_amdgcn_readlane((int)(q >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Lowest (energy, index) of the wave, lexicographically; every lane gets it.
template <typename T>
__device__ inline void wave_argmin(T &e, int &idx) {
#define JDOB_ARGMIN_STEP(CTRL, RMASK)                                  \
  {                                                                   \
    const T oe = dpp_mov<CTRL, RMASK>(inf_of<T>(), e);                \
    const int oi = dpp_mov<CTRL, RMASK>(0x7fffffff, idx);             \
    const bool tk = better(oe, oi, e, idx);                           \
    e = tk ? oe : e;                                                  \
    idx = tk ? oi : idx;                                              \
  }
  JDOB_ARGMIN_STEP(0x111, 0xf);
  JDOB_ARGMIN_STEP(0x112, 0xf);
  JDOB_ARGMIN_STEP(0x114, 0xf);
  JDOB_ARGMIN_STEP(0x118, 0xf);
  JDOB_ARGMIN_STEP(0x142, 0xa);
  JDOB_ARGMIN_STEP(0x143, 0xc);
#undef JDOB_ARGMIN_STEP
  e = lane_read(e, WAVE - 1);
  idx = lane_read(idx, WAVE - 1);
}

__device__ inline int wave_max_int(int v) {
  v = wave_iscan(v, (int)0x80000000, [](int a, int b) { return a > b ? a : b; });
  return lane_read(v, WAVE - 1);
}

__device__ inline int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int d = 1; d < WAVE; d <<= 1) v += __shfl_xor(v, d, WAVE);
  return v;
}

template <typename T>
__device__ inline T wave_max(T v) {
  v = wave_iscan(v, -inf_of<T>(), [](T a, T b) { return b > a ? b : a; });
  return lane_read(v, WAVE - 1);
}

// Inclusive scan over the wave; OP is min (exact in any order) or add (used
// for energies that only rank candidates).
template <typename T, bool IS_MIN>
__device__ inline T wave_scan(T v, int) {
  if (IS_MIN) return wave_iscan(v, inf_of<T>(), [](T a, T b) { return b < a ? b : a; });
  return wave_iscan(v, T(0), [](T a, T b) { return a + b; });
}

// A copy of a uniform value in scalar registers of its own.  Kernel arguments
// arrive in wide loads (eight or sixteen registers at a time); without the
// copy, a spill under register pressure saves and restores the whole group.
template <typename X> __device__ inline X own(X v) {
  asm volatile("" : "+s"(v));
  return v;
}

// Lanes 0..31 receive the value of lane l + 32 (one v_permlane32_swap);
// lanes 32..63 keep their own.
__device__ inline int from_upper_half(int v) {
  return (int)__builtin_amdgcn_permlane32_swap(v, v, false, false)[1];
}
__device__ inline float from_upper_half(float v) {
  return __int_as_float(from_upper_half(__float_as_int(v)));
}
__device__ inline double from_upper_half(double v) {
  const long long q = __double_as_longlong(v);
  const int lo = from_upper_half((int)(q & 0xffffffff)), hi = from_upper_half((int)(q >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Wave-uniform copies of values the compiler cannot prove uniform.
__device__ inline int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ inline float uni(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}
__device__ inline double uni(double v) {
  const long long q = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readfirstlane((int)(q & 0xffffffff));
  const int hi = __builtin_amdgcn_readfirstlane((int)(q >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}
// Inclusive wavefront prefix sum with DPP row shifts and row broadcasts (the
// summation order differs from a sequential sum: used for energies that only
// rank candidates).
__device__ inline float scan_add(float v) {
#define JDOB_DPP_ADD(CTRL, RMASK) \
  v = v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, RMASK, 0xf, false))
  JDOB_DPP_ADD(0x111, 0xf);  // row_shr:1
  JDOB_DPP_ADD(0x112, 0xf);  // row_shr:2
  JDOB_DPP_ADD(0x114, 0xf);  // row_shr:4
  JDOB_DPP_ADD(0x118, 0xf);  // row_shr:8
  JDOB_DPP_ADD(0x142, 0xa);  // row_bcast:15
  JDOB_DPP_ADD(0x143, 0xc);  // row_bcast:31
#undef JDOB_DPP_ADD
  return v;
}
__device__ inline double scan_add(double v) {
#define JDOB_DPP_ADD(CTRL, RMASK)                                                         \
  {                                                                                       \
    const long long q = __double_as_longlong(v);                                          \
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(q & 0xffffffff), CTRL, RMASK, 0xf, false); \
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(q >> 32), CTRL, RMASK, 0xf, false);        \
    v = v + __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);               \
  }
  JDOB_DPP_ADD(0x111, 0xf);
  JDOB_DPP_ADD(0x112, 0xf);
  JDOB_DPP_ADD(0x114, 0xf);
  JDOB_DPP_ADD(0x118, 0xf);
  JDOB_DPP_ADD(0x142, 0xa);
  JDOB_DPP_ADD(0x143, 0xc);
#undef JDOB_DPP_ADD
  return v;
}

// Fused multiply-add for energies that only rank candidates (every decision
// uses separately rounded operations).
__device__ inline float fma_(float a, float b, float c) { return __builtin_fmaf(a, b, c); }
__device__ inline double fma_(double a, double b, double c) { return __builtin_fma(a, b, c); }

__device__ inline int64_t instance_of_block(int64_t first) {
  // Consecutive workgroups are dealt round-robin to the 8 XCDs; give each XCD
  // a contiguous range of instances so that neighbouring rows and output
  // words are touched through one L2.
  const int64_t nb = gridDim.x, b = blockIdx.x;
  const int64_t xcd = b % 8, pos = b / 8;
  const int64_t q = nb / 8, r = nb % 8;
  const int64_t start = xcd * q + (xcd < r ? xcd : r);
  return first + start + pos;
}

// Eq. (20) with a continuous CPU frequency: the slowest frequency finishing
// cycles Cs within the budget, clamped to [fmin, fmax]; fmin without local
// layers.  Used only where the top frequency fits the budget.
template <typename T> __device__ inline T cont_freq(T Cs, T budget, T fmin, T fmax) {
  if (Cs == T(0)) return fmin;
  const T g = Cs / budget;
  return g < fmin ? fmin : (g > fmax ? fmax : g);
}

__device__ inline float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ inline double fast_rcp(double x) { return 1.0 / x; }

__device__ inline float clamp_(float v, float lo, float hi) {
  return __builtin_amdgcn_fmed3f(v, lo, hi);  // lo <= hi
}
__device__ inline double clamp_(double v, double lo, double hi) {
  return v < lo ? lo : (v > hi ? hi : v);
}

// The outer grouping keeps, per prefix of the deadline order, a front of
// states (total energy, GPU release time) that no other state dominates (no
// higher energy and no later release), sorted by energy, at most
// GROUP_FRONT of them.
constexpr int GROUP_FRONT = 16;

// Adds the state (E, Tr, src) to the front fE/fT/from[0..n) of one prefix
// and returns the new size: nothing changes if a state of the front has no
// higher energy and no later release (it came first); otherwise the states
// the new one dominates leave, it enters at its energy's place, and a front
// longer than GROUP_FRONT loses its highest energy.  Lane q holds slot q;
// E, Tr, src and n are wave-uniform; the whole wave calls it.
template <typename T>
__device__ inline int front_add(T *fE, T *fT, int16_t *from, int n, T E, T Tr, int src, int lane) {
  const bool in = lane < n;
  const T e = in ? fE[lane] : T(0), t = in ? fT[lane] : T(0);
  const int fr = in ? from[lane] : 0;
  if (__builtin_amdgcn_ballot_w64(in && e <= E && t <= Tr)) return n;
  const bool keep = in && !(E <= e && Tr <= t);
  const uint64_t km = __builtin_amdgcn_ballot_w64(keep);
  const int m = __popcll(km);
  // kept states stay in energy order; those below E come first
  const int below = __popcll(__builtin_amdgcn_ballot_w64(keep && e < E));
  const int rk = __builtin_amdgcn_mbcnt_hi((unsigned)(km >> 32),
                                           __builtin_amdgcn_mbcnt_lo((unsigned)km, 0u));
  const int pos = rk < below ? rk : rk + 1;
  __syncthreads();  // every slot read before any is written
  if (keep && pos < GROUP_FRONT) {
    fE[pos] = e;
    fT[pos] = t;
    from[pos] = (int16_t)fr;
  }
  if (lane == 0 && below < GROUP_FRONT) {
    fE[below] = E;
    fT[below] = Tr;
    from[below] = (int16_t)src;
  }
  __syncthreads();
  return m + 1 < GROUP_FRONT ? m + 1 : GROUP_FRONT;
}

// Heterogeneous users (per-user zeta, kappa, transmit power and CPU levels),
// in jdob_hetero.hip.
bool has_user_params(const jdob_problem *p);
int validate_hetero(const jdob_problem *p, bool grouped);
int launch_hetero(const jdob_problem *p, const jdob_policy *o, hipStream_t stream);
int launch_hetero_grouped(const jdob_problem *p, const jdob_grouped_policy *o, hipStream_t stream);

}  // namespace jdob_dev

#endif  // JDOB_COMMON_H
