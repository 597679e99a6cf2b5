// The paper's other fused differentiable optimizers on gfx950, over flat
// buffers: SGD with momentum (optionally Nesterov) and RMSProp (optionally
// with momentum), each a fused forward and a fused VJP (TorchOpt, Sec. 1
// contribution (2)(i) and Sec. 2.3 "CPU/GPU-accelerated optimizers"); the
// arithmetic is in optim_ops.hpp.
// Like Adam they are HBM-bound elementwise streams; they share one generic
// kernel skeleton with the measured Adam launch shape (1024-thread workgroups,
// one 16-byte vector per lane per array, bounds checks only on the last tile,
// a scalar kernel for pointers that are not 16-byte aligned).
#include <cmath>
#include <initializer_list>

#include "optim_ops.hpp"

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

bool aligned4(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int check_ptrs(const char* who, std::initializer_list<const void*> ps) {
  for (const void* q : ps)
    if (!aligned4(q)) return fail(DIFFOPT_EINVAL, "%s: pointer %p is not 4-byte aligned", who, q);
  return DIFFOPT_OK;
}

// Runner of the flat-buffer kernels for the *_variant selectors.
struct FlatRun {
  const char* who;
  int64_t n;
  hipStream_t st;
  template <class Op>
  int go(const Op& op, const void* const* in, const void* const* out) {
    Streams<Op::NIN, Op::NOUT> s{};
    for (int a = 0; a < Op::NIN; ++a) s.in[a] = static_cast<const float*>(in[a]);
    for (int b = 0; b < Op::NOUT; ++b) s.out[b] = static_cast<float*>(const_cast<void*>(out[b]));
    return launch(who, s, n, op, st);
  }
};

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
  FlatRun run{who, n, as_stream(stream)};
  return sgd_fwd_variant(run, params, grad, trace, params_out, trace_out, lr, momentum, nesterov != 0);
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
  FlatRun run{who, n, as_stream(stream)};
  return sgd_bwd_variant(run, dparams_out, dtrace_out, dgrad, dtrace_in, lr, momentum, nesterov != 0);
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
  FlatRun run{who, n, as_stream(stream)};
  return rms_fwd_variant(run, params, grad, nu, mom, params_out, nu_out, mom_out, c, m);
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
  FlatRun run{who, n, as_stream(stream)};
  return rms_bwd_variant(run, dparams_out, dnu_out, m ? dmom_out : nullptr, grad, nu, dgrad, dnu_in, dmom_in, c, m);
}
