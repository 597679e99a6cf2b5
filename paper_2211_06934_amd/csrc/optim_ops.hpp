// Arithmetic of the fused differentiable SGD-momentum and RMSProp steps and
// their VJPs (TorchOpt, Sec. 1 contribution (2)(i), Sec. 2.3), shared by the
// flat-buffer kernels (optim.hip) and the leaf-direct ones (treemap.hip).
// The paper prints neither formula; these are the textbook forms as
// torch.optim implements them:
//   SGD:      t' = mu t + g,  u = -lr t'  (Nesterov: u = -lr (g + mu t'))
//   RMSProp:  v' = alpha v + (1-alpha) g^2,  d = sqrt(v' + eps_root) + eps,
//             mu == 0: u = -lr g/d;  mu > 0: b' = mu b + g/d, u = -lr b'
//   p' = p + u in both.
// Each op is a struct with NIN inputs and NOUT outputs per element; which
// variant runs depends on which optional operands the caller gives, so a
// missing state or cotangent costs no bytes.  The *_variant functions pick it
// and hand the op and its operand lists (inputs, then outputs, in the op's
// order) to a runner: run.go(op, in, out).
#pragma once

#include <cmath>

#include "adam_math.hpp"

namespace diffopt {

// ---- SGD ----------------------------------------------------------------------
// Inputs p, g[, t]; outputs p'[, t'].  MOM: momentum > 0 (a trace is kept);
// TIN: a previous trace is given (else it is zero).
template <bool MOM, bool TIN, bool NEST>
struct SgdFwd {
  static constexpr int NIN = (MOM && TIN) ? 3 : 2;
  static constexpr int NOUT = MOM ? 2 : 1;
  float lr, mu;
  __device__ __forceinline__ void apply(const float* x, float* y) const {
    const float p = x[0], g = x[1];
    if (!MOM) {
      y[0] = fmaf(-lr, g, p);
      return;
    }
    const float t1 = (MOM && TIN) ? fmaf(mu, x[2], g) : g;
    y[0] = NEST ? fmaf(-lr, fmaf(mu, t1, g), p) : fmaf(-lr, t1, p);
    y[1] = t1;
  }
};

// Inputs dP[, dT]; outputs dg[, dt].  The map is linear: no saved inputs.
template <bool MOM, bool DTIN, bool NEST>
struct SgdBwd {
  static constexpr int NIN = (MOM && DTIN) ? 2 : 1;
  static constexpr int NOUT = MOM ? 2 : 1;
  float lr, mu, lr_mu;
  __device__ __forceinline__ void apply(const float* x, float* y) const {
    const float dP = x[0];
    if (!MOM) {
      y[0] = -lr * dP;
      return;
    }
    const float dT = DTIN ? x[1] : 0.0f;
    const float Tt = fmaf(-(NEST ? lr_mu : lr), dP, dT);  // cotangent of t'
    y[0] = NEST ? fmaf(-lr, dP, Tt) : Tt;
    y[1] = mu * Tt;
  }
};

// ---- RMSProp ------------------------------------------------------------------
struct RmsCoef {
  float lr, alpha, oma, two_oma, eps, eps_root, mu;
};

// Inputs p, g, v[, b]; outputs p', v'[, b'].
template <bool MOM, bool BIN>
struct RmsFwd {
  static constexpr int NIN = (MOM && BIN) ? 4 : 3;
  static constexpr int NOUT = MOM ? 3 : 2;
  RmsCoef c;
  __device__ __forceinline__ void apply(const float* x, float* y) const {
    const float p = x[0], g = x[1], v = x[2];
    const float v1 = fmaf(c.alpha, v, c.oma * (g * g));
    const float d = sqrtf(v1 + c.eps_root) + c.eps;
    const float q = g / d;
    if (MOM) {
      const float b1 = BIN ? fmaf(c.mu, x[3], q) : q;
      y[0] = fmaf(-c.lr, b1, p);
      y[2] = b1;
    } else {
      y[0] = fmaf(-c.lr, q, p);
    }
    y[1] = v1;
  }
};

// Inputs dP[, dV][, dB], g, v; outputs dg, dv[, db].  Reduced form: with
// Bt = dB - lr dP (mu == 0: -lr dP) the chain rule's g^2 terms cancel,
//   dg = 2 (1-alpha) g dV + Bt (alpha v + eps_root + s eps) / (s d^2)
//   dv = alpha (dV - Bt g / (2 s d^2)),  db = mu Bt;
// at s == 0 (eps_root = 0, v = 0, g = 0): dg = Bt / d, dv = alpha dV.
template <bool MOM, bool DVIN, bool DBIN>
struct RmsBwd {
  static constexpr int NIN = 3 + (DVIN ? 1 : 0) + ((MOM && DBIN) ? 1 : 0);
  static constexpr int NOUT = MOM ? 3 : 2;
  RmsCoef c;
  __device__ __forceinline__ void apply(const float* x, float* y) const {
    int a = 0;
    const float dP = x[a++];
    const float dV = DVIN ? x[a++] : 0.0f;
    const float dB = (MOM && DBIN) ? x[a++] : 0.0f;
    const float g = x[a++];
    const float v = x[a++];
    const float Bt = fmaf(-c.lr, dP, dB);
    const float s = sqrtf(fmaf(c.alpha, v, c.oma * (g * g)) + c.eps_root);
    const float d = s + c.eps;
    float kg, kv;  // Bt coefficients of dg and of dL/dv'
    if (s > 0.0f) {
      // x / (s d^2) as ((x / s) / d) / d: x / s stays in range (s^2 >= alpha v
      // + eps_root and s >= sqrt(1 - alpha) |g|), so an underflowing s d^2
      // (tiny s with eps = 0) still gives the finite quotient
      kg = ((fmaf(c.alpha, v, fmaf(s, c.eps, c.eps_root)) / s) / d) / d;
      kv = -0.5f * (((g / s) / d) / d);
    } else {
      kg = 1.0f / d;
      kv = 0.0f;
    }
    y[0] = fmaf(Bt, kg, c.two_oma * g * dV);
    y[1] = c.alpha * fmaf(Bt, kv, dV);
    if (MOM) y[2] = c.mu * Bt;
  }
};

inline int rms_coef(const char* who, double lr, double alpha, double eps, double eps_root, double mu, RmsCoef* c) {
  if (!std::isfinite(lr)) return fail(DIFFOPT_EINVAL, "%s: lr must be finite", who);
  if (!(alpha >= 0.0 && alpha < 1.0)) return fail(DIFFOPT_EINVAL, "%s: alpha must be in [0, 1) (got %g)", who, alpha);
  if (!(eps >= 0.0 && std::isfinite(eps))) return fail(DIFFOPT_EINVAL, "%s: eps must be finite and >= 0", who);
  if (!(eps_root >= 0.0 && std::isfinite(eps_root)))
    return fail(DIFFOPT_EINVAL, "%s: eps_root must be finite and >= 0", who);
  if (!(mu >= 0.0 && std::isfinite(mu))) return fail(DIFFOPT_EINVAL, "%s: momentum must be finite and >= 0", who);
  c->lr = (float)lr;
  c->alpha = (float)alpha;
  c->oma = (float)(1.0 - alpha);
  c->two_oma = (float)(2.0 * (1.0 - alpha));
  c->eps = (float)eps;
  c->eps_root = (float)eps_root;
  c->mu = (float)mu;
  return DIFFOPT_OK;
}

// ---- variant selection ----------------------------------------------------------
// Operands are addresses of any kind (flat buffers or leaf-address arrays);
// NULL marks an optional operand that is absent.  Whether momentum is on is
// decided by the caller from the fp64 hyper-parameter (momentum > 0).

template <class R>
int sgd_fwd_variant(R& run, const void* p, const void* g, const void* t, const void* po, const void* to,
                    double lr, double momentum, bool nesterov) {
  const float lr_f = (float)lr, mu = (float)momentum;
  if (!(momentum > 0.0)) {
    const void* in[] = {p, g};
    const void* out[] = {po};
    return run.go(SgdFwd<false, false, false>{lr_f, mu}, in, out);
  }
  if (t) {
    const void* in[] = {p, g, t};
    const void* out[] = {po, to};
    return nesterov ? run.go(SgdFwd<true, true, true>{lr_f, mu}, in, out)
                    : run.go(SgdFwd<true, true, false>{lr_f, mu}, in, out);
  }
  const void* in[] = {p, g};
  const void* out[] = {po, to};
  return nesterov ? run.go(SgdFwd<true, false, true>{lr_f, mu}, in, out)
                  : run.go(SgdFwd<true, false, false>{lr_f, mu}, in, out);
}

template <class R>
int sgd_bwd_variant(R& run, const void* dP, const void* dT, const void* dg, const void* dt, double lr,
                    double momentum, bool nesterov) {
  const float lr_f = (float)lr, mu = (float)momentum, lr_mu = (float)(lr * momentum);
  if (!(momentum > 0.0)) {
    const void* in[] = {dP};
    const void* out[] = {dg};
    return run.go(SgdBwd<false, false, false>{lr_f, mu, lr_mu}, in, out);
  }
  const void* out[] = {dg, dt};
  if (dT) {
    const void* in[] = {dP, dT};
    return nesterov ? run.go(SgdBwd<true, true, true>{lr_f, mu, lr_mu}, in, out)
                    : run.go(SgdBwd<true, true, false>{lr_f, mu, lr_mu}, in, out);
  }
  const void* in[] = {dP};
  return nesterov ? run.go(SgdBwd<true, false, true>{lr_f, mu, lr_mu}, in, out)
                  : run.go(SgdBwd<true, false, false>{lr_f, mu, lr_mu}, in, out);
}

template <class R>
int rms_fwd_variant(R& run, const void* p, const void* g, const void* v, const void* b, const void* po,
                    const void* vo, const void* bo, const RmsCoef& c, bool mom) {
  if (!mom) {
    const void* in[] = {p, g, v};
    const void* out[] = {po, vo};
    return run.go(RmsFwd<false, false>{c}, in, out);
  }
  const void* out[] = {po, vo, bo};
  if (b) {
    const void* in[] = {p, g, v, b};
    return run.go(RmsFwd<true, true>{c}, in, out);
  }
  const void* in[] = {p, g, v};
  return run.go(RmsFwd<true, false>{c}, in, out);
}

template <class R>
int rms_bwd_variant(R& run, const void* dP, const void* dV, const void* dB, const void* g, const void* v,
                    const void* dg, const void* dv, const void* db, const RmsCoef& c, bool mom) {
  if (!mom) {
    const void* out[] = {dg, dv};
    if (dV) {
      const void* in[] = {dP, dV, g, v};
      return run.go(RmsBwd<false, true, false>{c}, in, out);
    }
    const void* in[] = {dP, g, v};
    return run.go(RmsBwd<false, false, false>{c}, in, out);
  }
  const void* out[] = {dg, dv, db};
  if (dV && dB) {
    const void* in[] = {dP, dV, dB, g, v};
    return run.go(RmsBwd<true, true, true>{c}, in, out);
  }
  if (dV) {
    const void* in[] = {dP, dV, g, v};
    return run.go(RmsBwd<true, true, false>{c}, in, out);
  }
  if (dB) {
    const void* in[] = {dP, dB, g, v};
    return run.go(RmsBwd<true, false, true>{c}, in, out);
  }
  const void* in[] = {dP, g, v};
  return run.go(RmsBwd<true, false, false>{c}, in, out);
}

}  // namespace diffopt
