// Differentiable Adam step on gfx950: fused forward, fused reduced-form VJP,
// and the K-step unrolled driver (TorchOpt, Sec. 2.3 "CPU/GPU-accelerated
// optimizers"; Listing 1 for the unrolled loop).
//
// Both kernels are HBM-bound elementwise streams (about 0.5 and 0.8 flop per
// byte, far below the chip's ~20 flop/byte balance), so the design is about
// bytes in flight: each thread issues all of its 128-bit loads before any
// arithmetic, consecutive lanes touch consecutive 16-byte vectors (one wave
// instruction moves 1 KiB, fully coalesced), and each kernel reads and writes
// every array exactly once.  No intermediate is stored for the backward: it
// recomputes m', v', s, d from the saved (g, m, v), which costs no bytes.
#include <cmath>

#include "adam_math.hpp"

// Launch shape, chosen by measurement on MI355X (fp32, n ~ 1.2e8):
// 1024-thread workgroups, one 16-byte vector per thread per array.  Smaller
// workgroups with more vectors per thread, and persistent grid-stride grids of
// 8-32 waves per CU, measured 1-20% slower.
#ifndef DIFFOPT_FWD_U
#define DIFFOPT_FWD_U 1  // 16-byte vectors per thread per array, forward
#endif
#ifndef DIFFOPT_BWD_U
#define DIFFOPT_BWD_U 1  // 16-byte vectors per thread per array, backward
#endif
#ifndef DIFFOPT_ADAM_BLOCK
#define DIFFOPT_ADAM_BLOCK 1024  // threads per workgroup of the Adam kernels
#endif

namespace diffopt {

int make_coef(const char* who, int64_t count, double lr, double b1, double b2, double eps,
              double eps_root, AdamCoef* c) {
  if (count < 0) return fail(DIFFOPT_EINVAL, "%s: count must be >= 0 (got %lld)", who, (long long)count);
  if (!(b1 >= 0.0 && b1 < 1.0)) return fail(DIFFOPT_EINVAL, "%s: b1 must be in [0, 1) (got %g)", who, b1);
  if (!(b2 >= 0.0 && b2 < 1.0)) return fail(DIFFOPT_EINVAL, "%s: b2 must be in [0, 1) (got %g)", who, b2);
  if (!std::isfinite(lr)) return fail(DIFFOPT_EINVAL, "%s: lr must be finite", who);
  if (!(eps >= 0.0 && std::isfinite(eps))) return fail(DIFFOPT_EINVAL, "%s: eps must be finite and >= 0", who);
  if (!(eps_root >= 0.0 && std::isfinite(eps_root)))
    return fail(DIFFOPT_EINVAL, "%s: eps_root must be finite and >= 0", who);
  const double t = (double)count + 1.0;
  // 1 - b^t without cancellation for b near 1; b = 0 gives log = -inf, c = 1.
  const double c1 = -std::expm1(t * std::log(b1));
  const double c2 = -std::expm1(t * std::log(b2));
  const double a = (1.0 - b1) / c1;
  const double b = (1.0 - b2) / c2;
  c->b1 = (float)b1;
  c->omb1 = (float)(1.0 - b1);
  c->b2 = (float)b2;
  c->omb2 = (float)(1.0 - b2);
  c->inv_c2 = (float)(1.0 / c2);
  c->lr_c1 = (float)(lr / c1);
  c->eps = (float)eps;
  c->eps_root = (float)eps_root;
  c->lr = (float)lr;
  c->two_omb2 = (float)(2.0 * (1.0 - b2));
  c->bb1_c1 = (float)(b * b1 / c1);
  c->ab2_c2 = (float)(a * b2 / c2);
  c->a = (float)a;
  c->kv = (float)(b2 * lr / (2.0 * c1 * c2));
  c->lr_a = (float)(lr * a);
  c->b1_lr_c1 = (float)(b1 * lr / c1);
  return DIFFOPT_OK;
}

namespace {

// ---- kernels -----------------------------------------------------------------
// Vector kernels: tile t covers 16-byte vectors [t*B*U, (t+1)*B*U) for B
// threads per workgroup; lane j of the workgroup takes vectors j, j+B, ... so
// each load instruction of a wave is one contiguous 1 KiB.  Workgroups walk
// tiles with a grid stride (one tile each when the grid covers them all).
// Full tiles skip the per-vector bounds checks.  The last workgroup also
// finishes the n % 4 tail element by element.

constexpr int kAB = DIFFOPT_ADAM_BLOCK;

template <int U, bool WU, bool GUARD>
__device__ __forceinline__ void fwd_tile(int64_t t, int64_t nv, const float* p, const float* g, const float* m,
                                         const float* v, float* po, float* mo, float* vo, float* uo,
                                         const AdamCoef& c) {
  const int64_t base = t * (kAB * U) + threadIdx.x;
  f32x4 P[U], G[U], M[U], V[U];
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int64_t i = base + (int64_t)k * kAB;
    if (!GUARD || i < nv) {
      P[k] = ld(reinterpret_cast<const f32x4*>(p) + i);
      G[k] = ld(reinterpret_cast<const f32x4*>(g) + i);
      M[k] = ld(reinterpret_cast<const f32x4*>(m) + i);
      V[k] = ld(reinterpret_cast<const f32x4*>(v) + i);
    }
  }
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int64_t i = base + (int64_t)k * kAB;
    if (!GUARD || i < nv) {
      f32x4 rp, rm, rv, ru;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const FwdOut o = fwd_elem(P[k][e], G[k][e], M[k][e], V[k][e], c);
        rp[e] = o.p;
        rm[e] = o.m;
        rv[e] = o.v;
        ru[e] = o.u;
      }
      st(reinterpret_cast<f32x4*>(po) + i, rp);
      st(reinterpret_cast<f32x4*>(mo) + i, rm);
      st(reinterpret_cast<f32x4*>(vo) + i, rv);
      if (WU) st(reinterpret_cast<f32x4*>(uo) + i, ru);
    }
  }
}

template <int U, bool WU>
__global__ __launch_bounds__(kAB) void adam_fwd_vec(const float* p, const float* g, const float* m,
                                                    const float* v, float* po, float* mo, float* vo, float* uo,
                                                    int64_t n, AdamCoef c) {
  const int64_t nv = n >> 2;
  const int64_t nfull = nv / (kAB * U);
  const int64_t ntiles = (nv + kAB * U - 1) / (kAB * U);
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    if (t < nfull) fwd_tile<U, WU, false>(t, nv, p, g, m, v, po, mo, vo, uo, c);
    else fwd_tile<U, WU, true>(t, nv, p, g, m, v, po, mo, vo, uo, c);
  }
  if (blockIdx.x == gridDim.x - 1) {
    const int64_t e = (nv << 2) + threadIdx.x;
    if (e < n) {
      const FwdOut o = fwd_elem(p[e], g[e], m[e], v[e], c);
      po[e] = o.p;
      mo[e] = o.m;
      vo[e] = o.v;
      if (WU) uo[e] = o.u;
    }
  }
}

// Scalar kernel for pointers that are not 16-byte aligned.
template <bool WU>
__global__ __launch_bounds__(kAB) void adam_fwd_scalar(const float* p, const float* g, const float* m,
                                                       const float* v, float* po, float* mo, float* vo, float* uo,
                                                       int64_t n, AdamCoef c) {
  const int64_t base = (int64_t)blockIdx.x * (kAB * 4) + threadIdx.x;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t e = base + (int64_t)k * kAB;
    if (e < n) {
      const FwdOut o = fwd_elem(p[e], g[e], m[e], v[e], c);
      po[e] = o.p;
      mo[e] = o.m;
      vo[e] = o.v;
      if (WU) uo[e] = o.u;
    }
  }
}

template <int U, bool HAS_MV, bool WDP, bool GUARD>
__device__ __forceinline__ void bwd_tile(int64_t t, int64_t nv, const float* dP, const float* dM,
                                         const float* dV, const float* g, const float* m, const float* v,
                                         float* dpo, float* dgo, float* dmo, float* dvo, const AdamCoef& c) {
  const int64_t base = t * (kAB * U) + threadIdx.x;
  f32x4 P[U], Mb[U], Vb[U], G[U], M[U], V[U];
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int64_t i = base + (int64_t)k * kAB;
    if (!GUARD || i < nv) {
      P[k] = ld(reinterpret_cast<const f32x4*>(dP) + i);
      if (HAS_MV) {
        Mb[k] = ld(reinterpret_cast<const f32x4*>(dM) + i);
        Vb[k] = ld(reinterpret_cast<const f32x4*>(dV) + i);
      }
      G[k] = ld(reinterpret_cast<const f32x4*>(g) + i);
      M[k] = ld(reinterpret_cast<const f32x4*>(m) + i);
      V[k] = ld(reinterpret_cast<const f32x4*>(v) + i);
    }
  }
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int64_t i = base + (int64_t)k * kAB;
    if (!GUARD || i < nv) {
      f32x4 rg, rm, rv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const BwdOut o = bwd_elem<HAS_MV>(P[k][e], HAS_MV ? Mb[k][e] : 0.0f, HAS_MV ? Vb[k][e] : 0.0f, G[k][e],
                                          M[k][e], V[k][e], c);
        rg[e] = o.g;
        rm[e] = o.m;
        rv[e] = o.v;
      }
      st(reinterpret_cast<f32x4*>(dgo) + i, rg);
      st(reinterpret_cast<f32x4*>(dmo) + i, rm);
      st(reinterpret_cast<f32x4*>(dvo) + i, rv);
      if (WDP) st(reinterpret_cast<f32x4*>(dpo) + i, P[k]);
    }
  }
}

template <int U, bool HAS_MV, bool WDP>
__global__ __launch_bounds__(kAB) void adam_bwd_vec(const float* dP, const float* dM, const float* dV,
                                                    const float* g, const float* m, const float* v, float* dpo,
                                                    float* dgo, float* dmo, float* dvo, int64_t n, AdamCoef c) {
  const int64_t nv = n >> 2;
  const int64_t nfull = nv / (kAB * U);
  const int64_t ntiles = (nv + kAB * U - 1) / (kAB * U);
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    if (t < nfull) bwd_tile<U, HAS_MV, WDP, false>(t, nv, dP, dM, dV, g, m, v, dpo, dgo, dmo, dvo, c);
    else bwd_tile<U, HAS_MV, WDP, true>(t, nv, dP, dM, dV, g, m, v, dpo, dgo, dmo, dvo, c);
  }
  if (blockIdx.x == gridDim.x - 1) {
    const int64_t e = (nv << 2) + threadIdx.x;
    if (e < n) {
      const BwdOut o = bwd_elem<HAS_MV>(dP[e], HAS_MV ? dM[e] : 0.0f, HAS_MV ? dV[e] : 0.0f, g[e], m[e], v[e], c);
      dgo[e] = o.g;
      dmo[e] = o.m;
      dvo[e] = o.v;
      if (WDP) dpo[e] = dP[e];
    }
  }
}

template <bool HAS_MV, bool WDP>
__global__ __launch_bounds__(kAB) void adam_bwd_scalar(const float* dP, const float* dM, const float* dV,
                                                       const float* g, const float* m, const float* v, float* dpo,
                                                       float* dgo, float* dmo, float* dvo, int64_t n, AdamCoef c) {
  const int64_t base = (int64_t)blockIdx.x * (kAB * 4) + threadIdx.x;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t e = base + (int64_t)k * kAB;
    if (e < n) {
      const BwdOut o = bwd_elem<HAS_MV>(dP[e], HAS_MV ? dM[e] : 0.0f, HAS_MV ? dV[e] : 0.0f, g[e], m[e], v[e], c);
      dgo[e] = o.g;
      dmo[e] = o.m;
      dvo[e] = o.v;
      if (WDP) dpo[e] = dP[e];
    }
  }
}

// ---- host launchers ------------------------------------------------------------

inline bool aligned16(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool aligned4(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// One workgroup per tile; the kernels' grid-stride loop covers the (never
// reached in practice) case of more tiles than a grid dimension holds.
int64_t grid_for(int64_t tiles) {
  if (tiles < 1) return 1;
  return tiles < 0x7fffffff ? tiles : 0x7fffffff;
}

int launch_fwd(const float* p, const float* g, const float* m, const float* v, int64_t n, const AdamCoef& c,
               float* po, float* mo, float* vo, float* uo, hipStream_t st) {
  if (n == 0) return DIFFOPT_OK;
  const bool vec = aligned16(p) && aligned16(g) && aligned16(m) && aligned16(v) && aligned16(po) &&
                   aligned16(mo) && aligned16(vo) && aligned16(uo);
  if (vec) {
    constexpr int U = DIFFOPT_FWD_U;
    const int64_t blocks = grid_for(((n >> 2) + kAB * U - 1) / (kAB * U));
    if (uo)
      hipLaunchKernelGGL((adam_fwd_vec<U, true>), dim3((unsigned)blocks), dim3(kAB), 0, st, p, g, m, v, po, mo, vo,
                         uo, n, c);
    else
      hipLaunchKernelGGL((adam_fwd_vec<U, false>), dim3((unsigned)blocks), dim3(kAB), 0, st, p, g, m, v, po, mo,
                         vo, uo, n, c);
  } else {
    const int64_t blocks = (n + kAB * 4 - 1) / (kAB * 4);
    if (uo)
      hipLaunchKernelGGL((adam_fwd_scalar<true>), dim3((unsigned)blocks), dim3(kAB), 0, st, p, g, m, v, po, mo, vo,
                         uo, n, c);
    else
      hipLaunchKernelGGL((adam_fwd_scalar<false>), dim3((unsigned)blocks), dim3(kAB), 0, st, p, g, m, v, po, mo,
                         vo, uo, n, c);
  }
  return launch_status("diffopt_adam_fwd");
}

template <bool HAS_MV, bool WDP>
void launch_bwd_t(bool vec, const float* dP, const float* dM, const float* dV, const float* g, const float* m,
                  const float* v, float* dpo, float* dgo, float* dmo, float* dvo, int64_t n, const AdamCoef& c,
                  hipStream_t st) {
  if (vec) {
    constexpr int U = DIFFOPT_BWD_U;
    const int64_t blocks = grid_for(((n >> 2) + kAB * U - 1) / (kAB * U));
    hipLaunchKernelGGL((adam_bwd_vec<U, HAS_MV, WDP>), dim3((unsigned)blocks), dim3(kAB), 0, st, dP, dM, dV, g, m,
                       v, dpo, dgo, dmo, dvo, n, c);
  } else {
    const int64_t blocks = (n + kAB * 4 - 1) / (kAB * 4);
    hipLaunchKernelGGL((adam_bwd_scalar<HAS_MV, WDP>), dim3((unsigned)blocks), dim3(kAB), 0, st, dP, dM, dV, g, m,
                       v, dpo, dgo, dmo, dvo, n, c);
  }
}

int launch_bwd(const float* dP, const float* dM, const float* dV, const float* g, const float* m, const float* v,
               int64_t n, const AdamCoef& c, float* dpo, float* dgo, float* dmo, float* dvo, hipStream_t st) {
  if (n == 0) return DIFFOPT_OK;
  const bool has_mv = dM != nullptr;  // the entry point makes dM, dV both null or both set
  const bool wdp = dpo != nullptr && dpo != dP;
  const bool vec = aligned16(dP) && aligned16(dM) && aligned16(dV) && aligned16(g) && aligned16(m) &&
                   aligned16(v) && aligned16(wdp ? dpo : nullptr) && aligned16(dgo) && aligned16(dmo) &&
                   aligned16(dvo);
  if (has_mv) {
    if (wdp) launch_bwd_t<true, true>(vec, dP, dM, dV, g, m, v, dpo, dgo, dmo, dvo, n, c, st);
    else launch_bwd_t<true, false>(vec, dP, dM, dV, g, m, v, dpo, dgo, dmo, dvo, n, c, st);
  } else {
    if (wdp) launch_bwd_t<false, true>(vec, dP, dM, dV, g, m, v, dpo, dgo, dmo, dvo, n, c, st);
    else launch_bwd_t<false, false>(vec, dP, dM, dV, g, m, v, dpo, dgo, dmo, dvo, n, c, st);
  }
  return launch_status("diffopt_adam_bwd");
}

}  // namespace
}  // namespace diffopt

using namespace diffopt;

extern "C" int diffopt_adam_fwd(const float* params, const float* grad, const float* mu, const float* nu, int64_t n,
                                int64_t count, double lr, double b1, double b2, double eps, double eps_root,
                                float* params_out, float* mu_out, float* nu_out, float* update_out, void* stream) {
  clear_error();
  if (n < 0) return fail(DIFFOPT_EINVAL, "diffopt_adam_fwd: n must be >= 0 (got %lld)", (long long)n);
  AdamCoef c;
  int rc = make_coef("diffopt_adam_fwd", count, lr, b1, b2, eps, eps_root, &c);
  if (rc) return rc;
  if (n == 0) return DIFFOPT_OK;
  if (!params || !grad || !mu || !nu || !params_out || !mu_out || !nu_out)
    return fail(DIFFOPT_EINVAL, "diffopt_adam_fwd: null required pointer");
  const void* all[] = {params, grad, mu, nu, params_out, mu_out, nu_out, update_out};
  for (const void* q : all)
    if (!aligned4(q)) return fail(DIFFOPT_EINVAL, "diffopt_adam_fwd: pointer %p is not 4-byte aligned", q);
  return launch_fwd(params, grad, mu, nu, n, c, params_out, mu_out, nu_out, update_out, as_stream(stream));
}

extern "C" int diffopt_adam_bwd(const float* dupdate, const float* dmu, const float* dnu, const float* grad,
                                const float* mu, const float* nu, int64_t n, int64_t count, double lr, double b1,
                                double b2, double eps, double eps_root, float* dparams, float* dgrad, float* dmu_in,
                                float* dnu_in, void* stream) {
  clear_error();
  if (n < 0) return fail(DIFFOPT_EINVAL, "diffopt_adam_bwd: n must be >= 0 (got %lld)", (long long)n);
  AdamCoef c;
  int rc = make_coef("diffopt_adam_bwd", count, lr, b1, b2, eps, eps_root, &c);
  if (rc) return rc;
  if (n == 0) return DIFFOPT_OK;
  if (!dupdate || !grad || !mu || !nu || !dgrad || !dmu_in || !dnu_in)
    return fail(DIFFOPT_EINVAL, "diffopt_adam_bwd: null required pointer");
  if ((dmu == nullptr) != (dnu == nullptr))
    return fail(DIFFOPT_EINVAL, "diffopt_adam_bwd: dmu and dnu must both be given or both be NULL");
  const void* all[] = {dupdate, dmu, dnu, grad, mu, nu, dparams, dgrad, dmu_in, dnu_in};
  for (const void* q : all)
    if (!aligned4(q)) return fail(DIFFOPT_EINVAL, "diffopt_adam_bwd: pointer %p is not 4-byte aligned", q);
  return launch_bwd(dupdate, dmu, dnu, grad, mu, nu, n, c, dparams, dgrad, dmu_in, dnu_in, as_stream(stream));
}

extern "C" int diffopt_adam_unrolled_fwd(int64_t K, int64_t n, const float* p0, const float* const* grads,
                                         float* const* mu_traj, float* const* nu_traj, float* pK, int64_t count0,
                                         double lr, double b1, double b2, double eps, double eps_root,
                                         void* stream) {
  clear_error();
  static const char* who = "diffopt_adam_unrolled_fwd";
  if (K < 1) return fail(DIFFOPT_EINVAL, "%s: K must be >= 1 (got %lld)", who, (long long)K);
  if (n < 0) return fail(DIFFOPT_EINVAL, "%s: n must be >= 0", who);
  if (!grads || !mu_traj || !nu_traj) return fail(DIFFOPT_EINVAL, "%s: null pointer array", who);
  AdamCoef c;
  for (int64_t k = 1; k <= K; ++k) {  // validate every step's scalars before enqueuing anything
    int rc = make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &c);
    if (rc) return rc;
  }
  if (n == 0) return DIFFOPT_OK;
  if (!p0 || !pK) return fail(DIFFOPT_EINVAL, "%s: null p0 or pK", who);
  for (int64_t k = 0; k <= K; ++k) {
    if (!mu_traj[k] || !nu_traj[k]) return fail(DIFFOPT_EINVAL, "%s: null trajectory entry %lld", who, (long long)k);
    if (k < K && !grads[k]) return fail(DIFFOPT_EINVAL, "%s: null grads entry %lld", who, (long long)k);
  }
  hipStream_t st = as_stream(stream);
  for (int64_t k = 1; k <= K; ++k) {
    make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &c);
    const float* src = (k == 1) ? p0 : pK;
    int rc = launch_fwd(src, grads[k - 1], mu_traj[k - 1], nu_traj[k - 1], n, c, pK, mu_traj[k], nu_traj[k],
                        nullptr, st);
    if (rc) return rc;
  }
  return DIFFOPT_OK;
}

extern "C" int diffopt_adam_unrolled_bwd(int64_t K, int64_t n, const float* dpK, const float* const* grads,
                                         const float* const* mu_traj, const float* const* nu_traj,
                                         float* const* dgrads, float* dmu0, float* dnu0, int64_t count0, double lr,
                                         double b1, double b2, double eps, double eps_root, void* stream) {
  clear_error();
  static const char* who = "diffopt_adam_unrolled_bwd";
  if (K < 1) return fail(DIFFOPT_EINVAL, "%s: K must be >= 1 (got %lld)", who, (long long)K);
  if (n < 0) return fail(DIFFOPT_EINVAL, "%s: n must be >= 0", who);
  if (!grads || !mu_traj || !nu_traj || !dgrads) return fail(DIFFOPT_EINVAL, "%s: null pointer array", who);
  AdamCoef c;
  for (int64_t k = 1; k <= K; ++k) {
    int rc = make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &c);
    if (rc) return rc;
  }
  if (n == 0) return DIFFOPT_OK;
  if (!dpK || !dmu0 || !dnu0) return fail(DIFFOPT_EINVAL, "%s: null dpK, dmu0 or dnu0", who);
  if (dmu0 == dnu0) return fail(DIFFOPT_EINVAL, "%s: dmu0 and dnu0 must be distinct", who);
  for (int64_t k = 0; k < K; ++k) {
    if (!grads[k] || !mu_traj[k] || !nu_traj[k] || !dgrads[k])
      return fail(DIFFOPT_EINVAL, "%s: null entry %lld in a pointer array", who, (long long)k);
  }
  hipStream_t st = as_stream(stream);
  for (int64_t k = K; k >= 1; --k) {
    make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &c);
    const bool first = (k == K);  // zero cotangents of mu_K, nu_K
    int rc = launch_bwd(dpK, first ? nullptr : dmu0, first ? nullptr : dnu0, grads[k - 1], mu_traj[k - 1],
                        nu_traj[k - 1], n, c, nullptr, dgrads[k - 1], dmu0, dnu0, st);
    if (rc) return rc;
  }
  return DIFFOPT_OK;
}
