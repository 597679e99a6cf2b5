// The paper's other fused differentiable optimizers on gfx950: SGD with
// momentum (optionally Nesterov) and RMSProp (optionally with momentum), each
// a fused forward and a fused VJP (TorchOpt, Sec. 1 contribution (2)(i) and
// Sec. 2.3 "CPU/GPU-accelerated optimizers").  The paper prints neither
// formula; these are the textbook forms as torch.optim implements them:
//   SGD:      t' = mu t + g,  u = -lr t'  (Nesterov: u = -lr (g + mu t'))
//   RMSProp:  v' = alpha v + (1-alpha) g^2,  d = sqrt(v' + eps_root) + eps,
//             mu == 0: u = -lr g/d;  mu > 0: b' = mu b + g/d, u = -lr b'
//   p' = p + u in both.
// Like Adam they are HBM-bound elementwise streams; they share one generic
// kernel skeleton with the measured Adam launch shape (1024-thread workgroups,
// one 16-byte vector per lane per array, bounds checks only on the last tile,
// a scalar kernel for pointers that are not 16-byte aligned).
#include <cmath>
#include <initializer_list>

#include "adam_math.hpp"

namespace diffopt {
namespace {

constexpr int kOB = 1024;  // threads per workgroup

template <int NIN, int NOUT>
struct Streams {
  const float* in[NIN > 0 ? NIN : 1];
  float* out[NOUT];
};

template <class Op, bool GUARD>
__device__ __forceinline__ void ew_tile(const Streams<Op::NIN, Op::NOUT>& s, int64_t t, int64_t nv, const Op& op) {
  const int64_t i = t * kOB + threadIdx.x;
  if (GUARD && i >= nv) return;
  f32x4 x[Op::NIN];
#pragma unroll
  for (int a = 0; a < Op::NIN; ++a) x[a] = ld(reinterpret_cast<const f32x4*>(s.in[a]) + i);
  f32x4 y[Op::NOUT];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float xi[Op::NIN], yo[Op::NOUT];
#pragma unroll
    for (int a = 0; a < Op::NIN; ++a) xi[a] = x[a][e];
    op.apply(xi, yo);
#pragma unroll
    for (int b = 0; b < Op::NOUT; ++b) y[b][e] = yo[b];
  }
#pragma unroll
  for (int b = 0; b < Op::NOUT; ++b) st(reinterpret_cast<f32x4*>(s.out[b]) + i, y[b]);
}

template <class Op>
__global__ __launch_bounds__(kOB) void ew_vec(Streams<Op::NIN, Op::NOUT> s, int64_t n, Op op) {
  const int64_t nv = n >> 2;
  const int64_t nfull = nv / kOB;
  const int64_t ntiles = (nv + kOB - 1) / kOB;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    if (t < nfull) ew_tile<Op, false>(s, t, nv, op);
    else ew_tile<Op, true>(s, t, nv, op);
  }
  if (blockIdx.x == gridDim.x - 1) {
    const int64_t e = (nv << 2) + threadIdx.x;
    if (e < n) {
      float xi[Op::NIN], yo[Op::NOUT];
#pragma unroll
      for (int a = 0; a < Op::NIN; ++a) xi[a] = s.in[a][e];
      op.apply(xi, yo);
#pragma unroll
      for (int b = 0; b < Op::NOUT; ++b) s.out[b][e] = yo[b];
    }
  }
}

template <class Op>
__global__ __launch_bounds__(kOB) void ew_scalar(Streams<Op::NIN, Op::NOUT> s, int64_t n, Op op) {
  const int64_t e = (int64_t)blockIdx.x * kOB + threadIdx.x;
  if (e >= n) return;
  float xi[Op::NIN], yo[Op::NOUT];
#pragma unroll
  for (int a = 0; a < Op::NIN; ++a) xi[a] = s.in[a][e];
  op.apply(xi, yo);
#pragma unroll
  for (int b = 0; b < Op::NOUT; ++b) s.out[b][e] = yo[b];
}

template <class Op>
int launch(const char* who, const Streams<Op::NIN, Op::NOUT>& s, int64_t n, const Op& op, hipStream_t st) {
  if (n == 0) return DIFFOPT_OK;
  bool vec = true;
  for (int a = 0; a < Op::NIN; ++a) vec = vec && (reinterpret_cast<uintptr_t>(s.in[a]) & 15u) == 0;
  for (int b = 0; b < Op::NOUT; ++b) vec = vec && (reinterpret_cast<uintptr_t>(s.out[b]) & 15u) == 0;
  if (vec) {
    int64_t tiles = ((n >> 2) + kOB - 1) / kOB;
    if (tiles < 1) tiles = 1;
    if (tiles > 0x7fffffff) tiles = 0x7fffffff;
    hipLaunchKernelGGL(ew_vec<Op>, dim3((unsigned)tiles), dim3(kOB), 0, st, s, n, op);
  } else {
    const int64_t blocks = (n + kOB - 1) / kOB;
    if (blocks > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large for the unaligned path", who);
    hipLaunchKernelGGL(ew_scalar<Op>, dim3((unsigned)blocks), dim3(kOB), 0, st, s, n, op);
  }
  return launch_status(who);
}

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
      const float sd2 = s * d * d;
      kg = fmaf(c.alpha, v, fmaf(s, c.eps, c.eps_root)) / sd2;
      kv = -g / (2.0f * sd2);
    } else {
      kg = 1.0f / d;
      kv = 0.0f;
    }
    y[0] = fmaf(Bt, kg, c.two_oma * g * dV);
    y[1] = c.alpha * fmaf(Bt, kv, dV);
    if (MOM) y[2] = c.mu * Bt;
  }
};

int rms_coef(const char* who, double lr, double alpha, double eps, double eps_root, double mu, RmsCoef* c) {
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

bool aligned4(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int check_ptrs(const char* who, std::initializer_list<const void*> ps) {
  for (const void* q : ps)
    if (!aligned4(q)) return fail(DIFFOPT_EINVAL, "%s: pointer %p is not 4-byte aligned", who, q);
  return DIFFOPT_OK;
}

template <bool MOM, bool TIN, bool NEST>
int sgd_fwd_t(const float* p, const float* g, const float* t, float* po, float* to, int64_t n, float lr, float mu,
              hipStream_t st) {
  SgdFwd<MOM, TIN, NEST> op{lr, mu};
  Streams<SgdFwd<MOM, TIN, NEST>::NIN, SgdFwd<MOM, TIN, NEST>::NOUT> s{};
  s.in[0] = p;
  s.in[1] = g;
  if (MOM && TIN) s.in[SgdFwd<MOM, TIN, NEST>::NIN - 1] = t;
  s.out[0] = po;
  if (MOM) s.out[SgdFwd<MOM, TIN, NEST>::NOUT - 1] = to;
  return launch("diffopt_sgd_fwd", s, n, op, st);
}

template <bool MOM, bool DTIN, bool NEST>
int sgd_bwd_t(const float* dP, const float* dT, float* dg, float* dt, int64_t n, float lr, float mu, float lr_mu,
              hipStream_t st) {
  SgdBwd<MOM, DTIN, NEST> op{lr, mu, lr_mu};
  Streams<SgdBwd<MOM, DTIN, NEST>::NIN, SgdBwd<MOM, DTIN, NEST>::NOUT> s{};
  s.in[0] = dP;
  if (MOM && DTIN) s.in[SgdBwd<MOM, DTIN, NEST>::NIN - 1] = dT;
  s.out[0] = dg;
  if (MOM) s.out[SgdBwd<MOM, DTIN, NEST>::NOUT - 1] = dt;
  return launch("diffopt_sgd_bwd", s, n, op, st);
}

template <bool MOM, bool BIN>
int rms_fwd_t(const float* p, const float* g, const float* v, const float* b, float* po, float* vo, float* bo,
              int64_t n, const RmsCoef& c, hipStream_t st) {
  RmsFwd<MOM, BIN> op{c};
  Streams<RmsFwd<MOM, BIN>::NIN, RmsFwd<MOM, BIN>::NOUT> s{};
  s.in[0] = p;
  s.in[1] = g;
  s.in[2] = v;
  if (MOM && BIN) s.in[RmsFwd<MOM, BIN>::NIN - 1] = b;
  s.out[0] = po;
  s.out[1] = vo;
  if (MOM) s.out[RmsFwd<MOM, BIN>::NOUT - 1] = bo;
  return launch("diffopt_rmsprop_fwd", s, n, op, st);
}

template <bool MOM, bool DVIN, bool DBIN>
int rms_bwd_t(const float* dP, const float* dV, const float* dB, const float* g, const float* v, float* dg, float* dv,
              float* db, int64_t n, const RmsCoef& c, hipStream_t st) {
  typedef RmsBwd<MOM, DVIN, DBIN> Op;
  Op op{c};
  Streams<Op::NIN, Op::NOUT> s{};
  int a = 0;
  s.in[a++] = dP;
  if (DVIN) s.in[a++] = dV;
  if (MOM && DBIN) s.in[a++] = dB;
  s.in[a++] = g;
  s.in[a++] = v;
  s.out[0] = dg;
  s.out[1] = dv;
  if (MOM) s.out[Op::NOUT - 1] = db;
  return launch("diffopt_rmsprop_bwd", s, n, op, st);
}

}  // namespace
}  // namespace diffopt

using namespace diffopt;

extern "C" int diffopt_sgd_fwd(const float* params, const float* grad, const float* trace, int64_t n, double lr,
                               double momentum, int32_t nesterov, float* params_out, float* trace_out, void* stream) {
  clear_error();
  static const char* who = "diffopt_sgd_fwd";
  if (n < 0) return fail(DIFFOPT_EINVAL, "%s: n must be >= 0", who);
  if (!std::isfinite(lr)) return fail(DIFFOPT_EINVAL, "%s: lr must be finite", who);
  if (!(momentum >= 0.0 && std::isfinite(momentum)))
    return fail(DIFFOPT_EINVAL, "%s: momentum must be finite and >= 0", who);
  if (n == 0) return DIFFOPT_OK;
  const bool mom = momentum > 0.0;
  if (!params || !grad || !params_out || (mom && !trace_out))
    return fail(DIFFOPT_EINVAL, "%s: null required pointer", who);
  int rc = check_ptrs(who, {params, grad, trace, params_out, trace_out});
  if (rc) return rc;
  const float lr_f = (float)lr, mu = (float)momentum;
  hipStream_t st = as_stream(stream);
  if (!mom) return sgd_fwd_t<false, false, false>(params, grad, nullptr, params_out, nullptr, n, lr_f, mu, st);
  if (trace) {
    return nesterov ? sgd_fwd_t<true, true, true>(params, grad, trace, params_out, trace_out, n, lr_f, mu, st)
                    : sgd_fwd_t<true, true, false>(params, grad, trace, params_out, trace_out, n, lr_f, mu, st);
  }
  return nesterov ? sgd_fwd_t<true, false, true>(params, grad, nullptr, params_out, trace_out, n, lr_f, mu, st)
                  : sgd_fwd_t<true, false, false>(params, grad, nullptr, params_out, trace_out, n, lr_f, mu, st);
}

extern "C" int diffopt_sgd_bwd(const float* dparams_out, const float* dtrace_out, int64_t n, double lr,
                               double momentum, int32_t nesterov, float* dgrad, float* dtrace_in, void* stream) {
  clear_error();
  static const char* who = "diffopt_sgd_bwd";
  if (n < 0) return fail(DIFFOPT_EINVAL, "%s: n must be >= 0", who);
  if (!std::isfinite(lr)) return fail(DIFFOPT_EINVAL, "%s: lr must be finite", who);
  if (!(momentum >= 0.0 && std::isfinite(momentum)))
    return fail(DIFFOPT_EINVAL, "%s: momentum must be finite and >= 0", who);
  if (n == 0) return DIFFOPT_OK;
  const bool mom = momentum > 0.0;
  if (!dparams_out || !dgrad || (mom && !dtrace_in)) return fail(DIFFOPT_EINVAL, "%s: null required pointer", who);
  int rc = check_ptrs(who, {dparams_out, dtrace_out, dgrad, dtrace_in});
  if (rc) return rc;
  const float lr_f = (float)lr, mu = (float)momentum, lr_mu = (float)(lr * momentum);
  hipStream_t st = as_stream(stream);
  if (!mom) return sgd_bwd_t<false, false, false>(dparams_out, nullptr, dgrad, nullptr, n, lr_f, mu, lr_mu, st);
  if (dtrace_out) {
    return nesterov ? sgd_bwd_t<true, true, true>(dparams_out, dtrace_out, dgrad, dtrace_in, n, lr_f, mu, lr_mu, st)
                    : sgd_bwd_t<true, true, false>(dparams_out, dtrace_out, dgrad, dtrace_in, n, lr_f, mu, lr_mu, st);
  }
  return nesterov ? sgd_bwd_t<true, false, true>(dparams_out, nullptr, dgrad, dtrace_in, n, lr_f, mu, lr_mu, st)
                  : sgd_bwd_t<true, false, false>(dparams_out, nullptr, dgrad, dtrace_in, n, lr_f, mu, lr_mu, st);
}

extern "C" int diffopt_rmsprop_fwd(const float* params, const float* grad, const float* nu, const float* mom,
                                   int64_t n, double lr, double alpha, double eps, double eps_root, double momentum,
                                   float* params_out, float* nu_out, float* mom_out, void* stream) {
  clear_error();
  static const char* who = "diffopt_rmsprop_fwd";
  if (n < 0) return fail(DIFFOPT_EINVAL, "%s: n must be >= 0", who);
  RmsCoef c;
  int rc = rms_coef(who, lr, alpha, eps, eps_root, momentum, &c);
  if (rc) return rc;
  if (n == 0) return DIFFOPT_OK;
  const bool m = momentum > 0.0;
  if (!params || !grad || !nu || !params_out || !nu_out || (m && !mom_out))
    return fail(DIFFOPT_EINVAL, "%s: null required pointer", who);
  rc = check_ptrs(who, {params, grad, nu, mom, params_out, nu_out, mom_out});
  if (rc) return rc;
  hipStream_t st = as_stream(stream);
  if (!m) return rms_fwd_t<false, false>(params, grad, nu, nullptr, params_out, nu_out, nullptr, n, c, st);
  if (mom) return rms_fwd_t<true, true>(params, grad, nu, mom, params_out, nu_out, mom_out, n, c, st);
  return rms_fwd_t<true, false>(params, grad, nu, nullptr, params_out, nu_out, mom_out, n, c, st);
}

extern "C" int diffopt_rmsprop_bwd(const float* dparams_out, const float* dnu_out, const float* dmom_out,
                                   const float* grad, const float* nu, int64_t n, double lr, double alpha, double eps,
                                   double eps_root, double momentum, float* dgrad, float* dnu_in, float* dmom_in,
                                   void* stream) {
  clear_error();
  static const char* who = "diffopt_rmsprop_bwd";
  if (n < 0) return fail(DIFFOPT_EINVAL, "%s: n must be >= 0", who);
  RmsCoef c;
  int rc = rms_coef(who, lr, alpha, eps, eps_root, momentum, &c);
  if (rc) return rc;
  if (n == 0) return DIFFOPT_OK;
  const bool m = momentum > 0.0;
  if (!dparams_out || !grad || !nu || !dgrad || !dnu_in || (m && !dmom_in))
    return fail(DIFFOPT_EINVAL, "%s: null required pointer", who);
  rc = check_ptrs(who, {dparams_out, dnu_out, dmom_out, grad, nu, dgrad, dnu_in, dmom_in});
  if (rc) return rc;
  hipStream_t st = as_stream(stream);
  const float* dP = dparams_out;
  if (!m) {
    return dnu_out ? rms_bwd_t<false, true, false>(dP, dnu_out, nullptr, grad, nu, dgrad, dnu_in, nullptr, n, c, st)
                   : rms_bwd_t<false, false, false>(dP, nullptr, nullptr, grad, nu, dgrad, dnu_in, nullptr, n, c, st);
  }
  if (dnu_out) {
    return dmom_out ? rms_bwd_t<true, true, true>(dP, dnu_out, dmom_out, grad, nu, dgrad, dnu_in, dmom_in, n, c, st)
                    : rms_bwd_t<true, true, false>(dP, dnu_out, nullptr, grad, nu, dgrad, dnu_in, dmom_in, n, c, st);
  }
  return dmom_out ? rms_bwd_t<true, false, true>(dP, nullptr, dmom_out, grad, nu, dgrad, dnu_in, dmom_in, n, c, st)
                  : rms_bwd_t<true, false, false>(dP, nullptr, nullptr, grad, nu, dgrad, dnu_in, dmom_in, n, c, st);
}
