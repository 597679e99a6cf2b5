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

__device__ __forceinline__ FwdOut fwd_elem(float p, float g, float m, float v, const AdamCoef& c) {
  FwdOut o;
  o.m = moment1(g, m, c);
  o.v = moment2(g, v, c);
  const float s = sqrtf(fmaf(o.v, c.inv_c2, c.eps_root));
  const float d = s + c.eps;
  o.u = -(c.lr_c1 * o.m) / d;
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
  const float s = sqrtf(fmaf(v1, c.inv_c2, c.eps_root));
  const float d = s + c.eps;
  float kg, kvv;  // dupdate coefficients of dg and dv
  if (s > 0.0f) {
    const float sd2 = s * d * d;
    const float N = fmaf(c.bb1_c1 * g, m, -fmaf(c.ab2_c2, v, c.a * fmaf(s, c.eps, c.eps_root)));
    kg = c.lr * N / sd2;
    kvv = c.kv * m1 / sd2;
  } else {
    // s == 0 needs eps_root == 0, v == 0, g == 0: the explicit 0/0 case.
    kg = -c.lr_a / d;
    kvv = 0.0f;
  }
  BwdOut o;
  const float km = c.b1_lr_c1 / d;
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
