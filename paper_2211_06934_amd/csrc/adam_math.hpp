// Arithmetic of one differentiable Adam step, shared by the flat-buffer
// kernels (adam.hip) and the leaf-direct kernels (treemap.hip).
#pragma once

#include "common.hpp"

#ifndef DIFFOPT_NT_LOADS
#define DIFFOPT_NT_LOADS 1  // streaming (non-temporal) loads of the inputs
#endif
#ifndef DIFFOPT_NT_STORES
#define DIFFOPT_NT_STORES 1  // streaming (non-temporal) stores of the outputs
#endif

namespace diffopt {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Coefficients derived on the host in fp64 and rounded once to fp32.
struct AdamCoef {
  float b1, omb1, b2, omb2;  // b1, 1-b1, b2, 1-b2
  float inv_c2, lr_c1;       // 1/c2, lr/c1
  float eps, eps_root;
  // backward only
  float lr, two_omb2;  // lr, 2(1-b2)
  float bb1_c1;        // b b1 / c1        (b = (1-b2)/c2)
  float ab2_c2;        // a b2 / c2        (a = (1-b1)/c1)
  float a;             // (1-b1)/c1
  float kv;            // b2 lr / (2 c1 c2)
  float lr_a;          // lr a
  float b1_lr_c1;      // b1 lr / c1
};

// Validate the hyper-parameters and derive the coefficients for step count
// `count` (fp64, rounded once to fp32).  Returns DIFFOPT_OK or EINVAL with a
// message naming `who`.
int make_coef(const char* who, int64_t count, double lr, double b1, double b2, double eps,
              double eps_root, AdamCoef* c);

// Longest run of unrolled steps whose moments a K-step VJP recomputes in
// registers from one stored state (the run's trajectory is 3 vectors a step).
constexpr int kRematSpan = DIFFOPT_REMAT_SPAN;

// Store policy of a K-step trajectory (mu_traj, nu_traj: K+1 entries, flat
// buffers or leaf-address arrays): entry k (0 < k < K) may be NULL (not
// stored), mu and nu together.  The initial state is required; the final
// one too for the forward (need_last).  The VJP (bound_runs) recomputes a
// NULL state from the latest stored one before it, so at most
// kRematSpan - 1 consecutive entries may be NULL there.
template <typename P>
int check_trajectory(const char* who, int64_t K, const P* mu_traj, const P* nu_traj, bool need_last,
                     bool bound_runs) {
  if (!mu_traj[0] || !nu_traj[0]) return fail(DIFFOPT_EINVAL, "%s: null initial state mu_traj[0] / nu_traj[0]", who);
  if (need_last && (!mu_traj[K] || !nu_traj[K]))
    return fail(DIFFOPT_EINVAL, "%s: null final state mu_traj[K] / nu_traj[K]", who);
  int64_t last = 0;  // latest stored state
  for (int64_t k = 1; k < K; ++k) {
    if ((mu_traj[k] == nullptr) != (nu_traj[k] == nullptr))
      return fail(DIFFOPT_EINVAL, "%s: trajectory entry %lld: mu and nu must both be stored or both be NULL", who,
                  (long long)k);
    if (mu_traj[k]) last = k;
    else if (bound_runs && k + 1 - last > kRematSpan)
      return fail(DIFFOPT_EINVAL,
                  "%s: trajectory entries %lld..%lld are all NULL; at least every %d-th state must be stored", who,
                  (long long)(last + 1), (long long)k, kRematSpan);
  }
  return DIFFOPT_OK;
}

// How a recomputing VJP gets each step's input moments: 0 keeps the run's
// trajectory in registers, 1 recomputes each step's moments from the stored
// state (C(C-1)/2 moment steps instead of C-1).  Measured on MI355X (K = 3,
// n = 1.2e8): the flat kernel is faster with 1 (5.86 against 5.60 TB/s), the
// leaf-direct one with 0 (5.37 against 5.08 TB/s).
#ifndef DIFFOPT_REMAT_QUAD_FLAT
#define DIFFOPT_REMAT_QUAD_FLAT 1
#endif
#ifndef DIFFOPT_REMAT_QUAD_TREE
#define DIFFOPT_REMAT_QUAD_TREE 0
#endif

template <typename T>
__device__ __forceinline__ T ld(const T* p) {
#if DIFFOPT_NT_LOADS
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void st(T* p, T v) {
#if DIFFOPT_NT_STORES
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

// The same for pointers into the global address space (addresses that come
// from LDS-staged leaf tables).
template <typename T>
__device__ __forceinline__ T ld(const __attribute__((address_space(1))) T* p) {
#if DIFFOPT_NT_LOADS
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void st(__attribute__((address_space(1))) T* p, T v) {
#if DIFFOPT_NT_STORES
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

// ---- per-element arithmetic ------------------------------------------------

struct FwdOut {
  float p, m, v, u;
};

// The two moment recurrences of one step, m' = b1 m + (1-b1) g and
// v' = b2 v + (1-b2) g^2.  Every kernel that forms m', v' (the step, its VJP,
// the trajectory recomputation) goes through this one expression, so they all
// agree bit for bit.
__device__ __forceinline__ float moment1(float g, float m, const AdamCoef& c) { return fmaf(c.b1, m, c.omb1 * g); }
__device__ __forceinline__ float moment2(float g, float v, const AdamCoef& c) {
  return fmaf(c.b2, v, c.omb2 * (g * g));
}

// An opaque copy: the compiler cannot tell the result equals the argument,
// so a computation started from it is not merged with one started from the
// original (recomputing instead of keeping every intermediate live).
__device__ __forceinline__ f32x4 opaque(f32x4 x) {
  asm volatile("" : "+v"(x));
  return x;
}
__device__ __forceinline__ float opaque(float x) {
  asm volatile("" : "+v"(x));
  return x;
}

// The moments step s of a run consumed, from the run's stored state (M0, V0)
// and its gradients G[0..s-1], with the forward's recurrences (bit-identical
// to the values the forward formed).  T is f32x4 or float.
template <int C, typename T>
__device__ __forceinline__ void run_moments(int s, const T& M0, const T& V0, const T (&G)[C], const AdamCoef* c,
                                            T& m, T& v) {
  m = opaque(M0);
  v = opaque(V0);
#pragma unroll
  for (int r = 0; r < C; ++r) {
    if (r < s) {
      if constexpr (sizeof(T) == sizeof(float)) {
        m = moment1(G[r], m, c[r]);
        v = moment2(G[r], v, c[r]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          m[e] = moment1(G[r][e], m[e], c[r]);
          v[e] = moment2(G[r][e], v[e], c[r]);
        }
      }
    }
  }
}

// Quotients: 1 takes the hardware reciprocal v_rcp_f32 (at most 1 ulp) and
// multiplies, 0 the IEEE-exact divide sequence (about ten instructions
// each).  The VJP step needs 1/d and 1/(s d^2): two reciprocals in place of
// three divides.  The leaf-direct K-step kernels issue enough VALU work per
// byte that this shows (VJP 5.52 -> 5.92 TB/s, forward 5.79 -> 5.96 on
// MI355X); the flat ones are unchanged.  Every kernel shares these helpers,
// so all of them still agree with one another bit for bit; against the fp64
// oracle the reciprocal adds about 3 ulp, far inside the 1e-5 / 1e-4 bars.
#ifndef DIFFOPT_FAST_RECIP
#define DIFFOPT_FAST_RECIP 1
#endif
// Square root: 1 takes v_sqrt_f32 (1 ulp); 0 (kept) the correctly rounded
// sequence.  It measured no faster.
#ifndef DIFFOPT_FAST_SQRT
#define DIFFOPT_FAST_SQRT 0
#endif

__device__ __forceinline__ float root(float x) {
#if DIFFOPT_FAST_SQRT
  return __builtin_amdgcn_sqrtf(x);
#else
  return sqrtf(x);
#endif
}

__device__ __forceinline__ FwdOut fwd_elem(float p, float g, float m, float v, const AdamCoef& c) {
  FwdOut o;
  o.m = moment1(g, m, c);
  o.v = moment2(g, v, c);
  const float s = root(fmaf(o.v, c.inv_c2, c.eps_root));
  const float d = s + c.eps;
#if DIFFOPT_FAST_RECIP
  o.u = -(c.lr_c1 * o.m) * __builtin_amdgcn_rcpf(d);
#else
  o.u = -(c.lr_c1 * o.m) / d;
#endif
  o.p = p + o.u;
  return o;
}

struct BwdOut {
  float g, m, v;
};

// Reduced-form VJP.  With a = (1-b1)/c1, b = (1-b2)/c2 the plain chain rule's
// dupdate terms of dg, (1-b1)(-lr/(c1 d)) + 2(1-b2) g lr m^/(2 c2 s d^2), share
// the factor lr/(s d^2) and their g^2 parts cancel exactly, leaving
// N = b b1 g m/c1 - a b2 v/c2 - a (eps_root + s eps).  This is what keeps the
// fp32 result accurate where the two plain terms nearly cancel (fresh state,
// eps_root = 0: the plain form loses up to all digits there).
template <bool HAS_MV>
__device__ __forceinline__ BwdOut bwd_elem(float dP, float dM, float dV, float g, float m, float v,
                                           const AdamCoef& c) {
  const float m1 = moment1(g, m, c);
  const float v1 = moment2(g, v, c);
  const float s = root(fmaf(v1, c.inv_c2, c.eps_root));
  const float d = s + c.eps;
  const float N = fmaf(c.bb1_c1 * g, m, -fmaf(c.ab2_c2, v, c.a * fmaf(s, c.eps, c.eps_root)));
  float kg, kvv, km;  // dupdate coefficients of dg, dv and dm
  // The quotients x / (s d^2) are taken as ((x / s) / d) / d.  N / s stays
  // in range (each term of N carries g, v, eps_root or s, and s^2 = b2 v/c2 +
  // b g^2 + eps_root), so when s d^2 itself underflows (tiny s with eps = 0)
  // the result is still the finite quotient, and an exactly zero N gives 0
  // rather than 0 * inf.
#if DIFFOPT_FAST_RECIP
  // two reciprocals, 1/d and 1/s, serve all three quotients; the s == 0
  // case (the explicit 0/0 one, below) is a select, not a branch
  const float rd = __builtin_amdgcn_rcpf(d);
  const float rs = __builtin_amdgcn_rcpf(s);
  kg = s > 0.0f ? c.lr * (((N * rs) * rd) * rd) : -c.lr_a * rd;
  kvv = s > 0.0f ? c.kv * (((m1 * rs) * rd) * rd) : 0.0f;
  km = c.b1_lr_c1 * rd;
#else
  if (s > 0.0f) {
    kg = c.lr * (((N / s) / d) / d);
    kvv = c.kv * (((m1 / s) / d) / d);
  } else {
    // s == 0 needs eps_root == 0, v == 0, g == 0: the explicit 0/0 case.
    kg = -c.lr_a / d;
    kvv = 0.0f;
  }
  km = c.b1_lr_c1 / d;
#endif
  BwdOut o;
  if (HAS_MV) {
    o.g = fmaf(dP, kg, fmaf(c.omb1, dM, c.two_omb2 * g * dV));
    o.m = fmaf(c.b1, dM, -dP * km);
    o.v = fmaf(c.b2, dV, dP * kvv);
  } else {
    o.g = dP * kg;
    o.m = -dP * km;
    o.v = dP * kvv;
  }
  return o;
}

}  // namespace diffopt
