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
// Fused K-step kernels, measured in the many-small step (K = 3).  Forward
// storing only the final state: 1024 threads 0.695 ms, 512 0.710, 256 0.731
// (with the whole trajectory stored the three were within 1%).  VJP reading
// the whole trajectory: 1024 threads 1.20 ms against 1.25 at 512 and 1.26 at
// 256.  VJP recomputing the moments: 512 threads 0.859 ms, 256 0.880, 1024
// 0.901.
#ifndef DIFFOPT_UFWD_BLOCK
#define DIFFOPT_UFWD_BLOCK 1024  // threads per workgroup, fused K-step forward
#endif
#ifndef DIFFOPT_UBWD_BLOCK
#define DIFFOPT_UBWD_BLOCK 1024  // threads per workgroup, fused K-step VJP
#endif
#ifndef DIFFOPT_URBWD_BLOCK
#define DIFFOPT_URBWD_BLOCK 512  // threads per workgroup, fused VJP recomputing the moments
#endif
// Runs of at least DIFFOPT_URBWD_LONG_RUN steps use DIFFOPT_URBWD_BLOCK_LONG
// threads.  Measured (n = 1.17e8): 512 threads are fastest for runs of 3 to 6
// steps (256: 1-5% slower); an 8-step run (151 VGPRs) took 2.02 ms at 512 and
// 1.91 ms at 256.
#ifndef DIFFOPT_URBWD_LONG_RUN
#define DIFFOPT_URBWD_LONG_RUN 7
#endif
#ifndef DIFFOPT_URBWD_BLOCK_LONG
#define DIFFOPT_URBWD_BLOCK_LONG 256
#endif
// Arrays of fewer than DIFFOPT_SMALL_VECS 16-byte vectors take workgroups of
// at most DIFFOPT_SMALL_BLOCK threads in the fused K-step kernels: with few
// large workgroups per CU, the last round of workgroups leaves CUs idle.
// Measured (graph replay, pack -> K steps -> unpack): ResNet-18 tree
// (1.17e7 params) K = 1 183 -> 178-179 us; K = 10 and the 3.6e6-param
// conv-net within 1% (128 threads: the same within noise, 512: no better).
#ifndef DIFFOPT_SMALL_VECS
#define DIFFOPT_SMALL_VECS (1 << 22)
#endif
#ifndef DIFFOPT_SMALL_BLOCK
#define DIFFOPT_SMALL_BLOCK 256
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

inline bool aligned16(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool aligned4(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// Order in which the single-step kernels' workgroups take the tiles.  The
// dispatcher deals workgroup b to XCD b mod 8: with 0, tile b, so the eight
// XCDs interleave through every array; with 1, XCD x takes a contiguous
// eighth of the tiles, so each XCD streams its own ranges of the arrays.
// Measured on the 1e9-element step, both orders on each of eight fresh
// allocations of the 13 arrays: 1 was slower on every allocation (forward
// 0.701 against 0.725 of 8 TB/s on average, VJP 0.705 against 0.728), while
// the allocation itself moved both orders together between 0.69 and 0.79.
#ifndef DIFFOPT_FLAT_ORDER
#define DIFFOPT_FLAT_ORDER 0
#endif

__device__ __forceinline__ int64_t flat_tile(int64_t b, int64_t ntiles) {
#if DIFFOPT_FLAT_ORDER == 1
  if ((int64_t)gridDim.x != ntiles) return b;  // grid-stride fallback: plain order
  const int64_t x = b & 7, l = b >> 3, per = ntiles >> 3, rem = ntiles & 7;
  return x * per + (x < rem ? x : rem) + l;   // a bijection of [0, ntiles)
#else
  (void)ntiles;
  return b;
#endif
}

// One workgroup per tile; the kernels' grid-stride loop covers the (never
// reached in practice) case of more tiles than a grid dimension holds.
int64_t grid_for(int64_t tiles) {
  if (tiles < 1) return 1;
  return tiles < 0x7fffffff ? tiles : 0x7fffffff;
}

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
  for (int64_t b = blockIdx.x; b < ntiles; b += gridDim.x) {
    const int64_t t = flat_tile(b, ntiles);
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
  for (int64_t b = blockIdx.x; b < ntiles; b += gridDim.x) {
    const int64_t t = flat_tile(b, ntiles);
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

// ---- fused K-step unrolled kernels -----------------------------------------------
// One launch runs up to kUK consecutive steps of the unrolled loop for every
// element it owns.  The running params (forward) and the running cotangents
// dP, dM, dV (backward) stay in registers between steps instead of making a
// round trip through HBM, so K steps move 16 + 12K bytes per element forward
// (p0, mu0, nu0 and K gradients in; K mu/nu pairs and p_K out) and 12 + 16K
// backward (dP and K (g, mu, nu) triples in; K dg and dmu0, dnu0 out), against
// 28K and 36K - 8 for K separate step kernels.  Each step's arithmetic is the
// same fwd_elem / bwd_elem as the single-step kernels, in the same order.
// The next step's loads are issued before the current step's arithmetic.

constexpr int kUK = 16;  // steps per fused launch (kernel-argument space bounds it)
constexpr int kUFB = DIFFOPT_UFWD_BLOCK;
constexpr int kUBB = DIFFOPT_UBWD_BLOCK;
constexpr int kSmallB = DIFFOPT_SMALL_BLOCK;
constexpr int64_t kSmallVecs = DIFFOPT_SMALL_VECS;
static_assert(kSmallB >= 64 && kSmallB % 64 == 0, "whole wavefronts; the tail needs 4 lanes");

// Step s of a launch is the launch's s-th step in execution order.
struct UFwdArgs {
  const float* p;   // params before the launch's first step
  const float* m0;  // mu, nu before the first step
  const float* v0;
  float* pK;  // params after the last step
  const float* g[kUK];
  float* m[kUK];  // mu, nu after step s; NULL: not stored (never for the last step)
  float* v[kUK];
  AdamCoef c[kUK];
  int64_t n;
  int32_t K;  // steps in this launch, 1..kUK
};

// Execution order of the backward is reverse step order: step s of a launch
// is unrolled step k_hi - s, with the state (g, mu, nu) that step consumed.
struct UBwdArgs {
  const float* dP;  // cotangent of the final params (constant through Adam steps)
  float* dm;        // running dM, dV: read first if init_mv, written at the end
  float* dv;
  const float* g[kUK];
  const float* m[kUK];
  const float* v[kUK];
  float* dg[kUK];
  AdamCoef c[kUK];
  int64_t n;
  int32_t K;
  int32_t init_mv;  // 0: dM = dV = 0 before the first step (the last unrolled step)
};

__device__ __forceinline__ const f32x4* cv4(const float* q) { return reinterpret_cast<const f32x4*>(q); }
__device__ __forceinline__ f32x4* v4(float* q) { return reinterpret_cast<f32x4*>(q); }

__device__ __forceinline__ void ufwd_vector(int64_t i, const UFwdArgs& a) {
  f32x4 P = ld(cv4(a.p) + i), M = ld(cv4(a.m0) + i), V = ld(cv4(a.v0) + i);
  f32x4 G = ld(cv4(a.g[0]) + i);
  for (int s = 0; s < a.K; ++s) {  // a runtime loop keeps the code small
    f32x4 Gn = G;
    if (s + 1 < a.K) Gn = ld(cv4(a.g[s + 1]) + i);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const FwdOut o = fwd_elem(P[e], G[e], M[e], V[e], a.c[s]);
      P[e] = o.p;
      M[e] = o.m;
      V[e] = o.v;
    }
    if (a.m[s]) {  // uniform: the same for every lane
      st(v4(a.m[s]) + i, M);
      st(v4(a.v[s]) + i, V);
    }
    G = Gn;
  }
  st(v4(a.pK) + i, P);
}

__device__ __forceinline__ void ufwd_element(int64_t e, const UFwdArgs& a) {
  float P = a.p[e], M = a.m0[e], V = a.v0[e];
  for (int s = 0; s < a.K; ++s) {
    const FwdOut o = fwd_elem(P, a.g[s][e], M, V, a.c[s]);
    P = o.p;
    M = o.m;
    V = o.v;
    if (a.m[s]) {
      a.m[s][e] = M;
      a.v[s][e] = V;
    }
  }
  a.pK[e] = P;
}

// Tile t covers 16-byte vectors [t B, (t+1) B) for B threads per workgroup;
// only the last tile checks bounds, and the last workgroup also runs the
// n % 4 tail elements.
template <int B>
__global__ __launch_bounds__(B) void adam_unrolled_fwd_vec(UFwdArgs a) {
  const int64_t nv = a.n >> 2;
  const int64_t ntiles = (nv + B - 1) / B;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t i = t * B + threadIdx.x;
    if (i < nv) ufwd_vector(i, a);
  }
  if (blockIdx.x == gridDim.x - 1) {
    const int64_t e = (nv << 2) + threadIdx.x;
    if (e < a.n) ufwd_element(e, a);
  }
}

// Any alignment: one element per thread (pointers only 4-byte aligned).
__global__ __launch_bounds__(kUFB) void adam_unrolled_fwd_elem(UFwdArgs a) {
  for (int64_t e = (int64_t)blockIdx.x * kUFB + threadIdx.x; e < a.n; e += (int64_t)gridDim.x * kUFB)
    ufwd_element(e, a);
}

template <bool HAS_MV>
__device__ __forceinline__ void ubwd_step(const f32x4& dP, f32x4& dM, f32x4& dV, const f32x4& g, const f32x4& m,
                                          const f32x4& v, const AdamCoef& c, f32x4* dgo) {
  f32x4 rg;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const BwdOut o = bwd_elem<HAS_MV>(dP[e], dM[e], dV[e], g[e], m[e], v[e], c);
    rg[e] = o.g;
    dM[e] = o.m;
    dV[e] = o.v;
  }
  st(dgo, rg);
}

__device__ __forceinline__ void ubwd_vector(int64_t i, const UBwdArgs& a) {
  const f32x4 dP = ld(cv4(a.dP) + i);
  f32x4 dM = {0.0f, 0.0f, 0.0f, 0.0f}, dV = {0.0f, 0.0f, 0.0f, 0.0f};
  f32x4 G = ld(cv4(a.g[0]) + i), M = ld(cv4(a.m[0]) + i), V = ld(cv4(a.v[0]) + i);
  int s = 0;
  if (a.init_mv) {
    dM = ld(cv4(a.dm) + i);
    dV = ld(cv4(a.dv) + i);
  } else {  // the last unrolled step: zero cotangents of its mu, nu outputs
    f32x4 Gn = G, Mn = M, Vn = V;
    if (1 < a.K) {
      Gn = ld(cv4(a.g[1]) + i);
      Mn = ld(cv4(a.m[1]) + i);
      Vn = ld(cv4(a.v[1]) + i);
    }
    ubwd_step<false>(dP, dM, dV, G, M, V, a.c[0], v4(a.dg[0]) + i);
    G = Gn;
    M = Mn;
    V = Vn;
    s = 1;
  }
  for (; s < a.K; ++s) {  // a runtime loop keeps the code small
    f32x4 Gn = G, Mn = M, Vn = V;
    if (s + 1 < a.K) {
      Gn = ld(cv4(a.g[s + 1]) + i);
      Mn = ld(cv4(a.m[s + 1]) + i);
      Vn = ld(cv4(a.v[s + 1]) + i);
    }
    ubwd_step<true>(dP, dM, dV, G, M, V, a.c[s], v4(a.dg[s]) + i);
    G = Gn;
    M = Mn;
    V = Vn;
  }
  st(v4(a.dm) + i, dM);
  st(v4(a.dv) + i, dV);
}

__device__ __forceinline__ void ubwd_element(int64_t e, const UBwdArgs& a) {
  const float dP = a.dP[e];
  float dM = 0.0f, dV = 0.0f;
  int s = 0;
  if (a.init_mv) {
    dM = a.dm[e];
    dV = a.dv[e];
  } else {
    const BwdOut o = bwd_elem<false>(dP, 0.0f, 0.0f, a.g[0][e], a.m[0][e], a.v[0][e], a.c[0]);
    a.dg[0][e] = o.g;
    dM = o.m;
    dV = o.v;
    s = 1;
  }
  for (; s < a.K; ++s) {
    const BwdOut o = bwd_elem<true>(dP, dM, dV, a.g[s][e], a.m[s][e], a.v[s][e], a.c[s]);
    a.dg[s][e] = o.g;
    dM = o.m;
    dV = o.v;
  }
  a.dm[e] = dM;
  a.dv[e] = dV;
}

template <int B>
__global__ __launch_bounds__(B) void adam_unrolled_bwd_vec(UBwdArgs a) {
  const int64_t nv = a.n >> 2;
  const int64_t ntiles = (nv + B - 1) / B;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t i = t * B + threadIdx.x;
    if (i < nv) ubwd_vector(i, a);
  }
  if (blockIdx.x == gridDim.x - 1) {
    const int64_t e = (nv << 2) + threadIdx.x;
    if (e < a.n) ubwd_element(e, a);
  }
}

__global__ __launch_bounds__(kUBB) void adam_unrolled_bwd_elem(UBwdArgs a) {
  for (int64_t e = (int64_t)blockIdx.x * kUBB + threadIdx.x; e < a.n; e += (int64_t)gridDim.x * kUBB)
    ubwd_element(e, a);
}

// ---- small buffers ---------------------------------------------------------------
// Up to kSmallElems elements the fused launches are bound by latency, not
// bandwidth: one element per lane (the shortest arithmetic chain per lane),
// the step count a template argument so that every load of every step is
// issued before the first step's arithmetic, and the kernel arguments
// warmed at the start.  Same per-element arithmetic as the kernels above, so
// the results agree bit for bit.
constexpr int64_t kSmallElems = int64_t(1) << 16;
constexpr int kSEB = 256;  // threads per workgroup of the small-buffer kernels

template <int K>
__global__ __launch_bounds__(kSEB) void adam_unrolled_fwd_small(UFwdArgs a) {
  warm_args(fold_lines(a));
  const int64_t e = (int64_t)blockIdx.x * kSEB + threadIdx.x;
  if (e >= a.n) return;
  float P = a.p[e], M = a.m0[e], V = a.v0[e];
  float G[K];
#pragma unroll
  for (int s = 0; s < K; ++s) G[s] = a.g[s][e];
#pragma unroll
  for (int s = 0; s < K; ++s) {
    const FwdOut o = fwd_elem(P, G[s], M, V, a.c[s]);
    P = o.p;
    M = o.m;
    V = o.v;
    if (a.m[s]) {  // uniform: a stored state
      a.m[s][e] = M;
      a.v[s][e] = V;
    }
  }
  a.pK[e] = P;
}

// Stored states: launch step s is unrolled step khi - s (as in ubwd_element).
// Without incoming moment cotangents their load slots read dP (unused), so
// no load waits behind a branch.
template <int K>
__global__ __launch_bounds__(kSEB) void adam_unrolled_bwd_small(UBwdArgs a) {
  warm_args(fold_lines(a));
  const int64_t e = (int64_t)blockIdx.x * kSEB + threadIdx.x;
  if (e >= a.n) return;
  const float dP = a.dP[e];
  const float dMi = (a.init_mv ? a.dm : a.dP)[e], dVi = (a.init_mv ? a.dv : a.dP)[e];
  float G[K], M[K], V[K];
#pragma unroll
  for (int s = 0; s < K; ++s) {
    G[s] = a.g[s][e];
    M[s] = a.m[s][e];
    V[s] = a.v[s][e];
  }
  float dM = dMi, dV = dVi;
  BwdOut o = a.init_mv ? bwd_elem<true>(dP, dM, dV, G[0], M[0], V[0], a.c[0])
                       : bwd_elem<false>(dP, 0.0f, 0.0f, G[0], M[0], V[0], a.c[0]);
  a.dg[0][e] = o.g;
  dM = o.m;
  dV = o.v;
#pragma unroll
  for (int s = 1; s < K; ++s) {
    o = bwd_elem<true>(dP, dM, dV, G[s], M[s], V[s], a.c[s]);
    a.dg[s][e] = o.g;
    dM = o.m;
    dV = o.v;
  }
  a.dm[e] = dM;
  a.dv[e] = dV;
}

template <int K>
void launch_ufwd_small(const UFwdArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((adam_unrolled_fwd_small<K>), dim3((unsigned)((a.n + kSEB - 1) / kSEB)), dim3(kSEB), 0, st, a);
}

template <int K>
void launch_ubwd_small(const UBwdArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((adam_unrolled_bwd_small<K>), dim3((unsigned)((a.n + kSEB - 1) / kSEB)), dim3(kSEB), 0, st, a);
}

// k in 1..kUK (16).
template <class Args, template <int> class L>
void dispatch_k(int k, const Args& a, hipStream_t st) {
  switch (k) {
    case 1: L<1>::run(a, st); break;
    case 2: L<2>::run(a, st); break;
    case 3: L<3>::run(a, st); break;
    case 4: L<4>::run(a, st); break;
    case 5: L<5>::run(a, st); break;
    case 6: L<6>::run(a, st); break;
    case 7: L<7>::run(a, st); break;
    case 8: L<8>::run(a, st); break;
    case 9: L<9>::run(a, st); break;
    case 10: L<10>::run(a, st); break;
    case 11: L<11>::run(a, st); break;
    case 12: L<12>::run(a, st); break;
    case 13: L<13>::run(a, st); break;
    case 14: L<14>::run(a, st); break;
    case 15: L<15>::run(a, st); break;
    default: L<16>::run(a, st); break;
  }
}
static_assert(kUK == 16, "dispatch_k instantiates 1..16 steps");

template <int K>
struct FwdSmall {
  static void run(const UFwdArgs& a, hipStream_t st) { launch_ufwd_small<K>(a, st); }
};
template <int K>
struct BwdSmall {
  static void run(const UBwdArgs& a, hipStream_t st) { launch_ubwd_small<K>(a, st); }
};

// ---- fused K-step VJP over a run of steps whose moments were not stored -------------
// For a run of C steps j+1..j+C of which only the state (mu_j, nu_j) before
// the first was stored, the lane reads that state and the C gradients once,
// recomputes mu_j+1..mu_j+C-1 (and nu) with the forward's own recurrences
// into registers, then runs the C VJP steps last step first.  Bytes per
// element: 12 + 8C (dP, mu_j, nu_j, C g in; C dg out; plus the running dM,
// dV: 8 in unless this run holds the last unrolled step, 8 out), against
// 12 + 16C when every state is read back.  Registers hold 3C vectors, so a
// run is at most kRS steps: the caller stores at least every kRS-th state.
constexpr int kRS = kRematSpan;
constexpr int kURB = DIFFOPT_URBWD_BLOCK;

// Step s of a run is unrolled step j+1+s (ascending); the VJP walks s = C-1..0.
struct URBwdArgs {
  const float* dP;
  float* dm;  // running dM, dV: read first if init_mv, written at the end
  float* dv;
  const float* m0;  // the stored state (mu_j, nu_j) before the run's first step
  const float* v0;
  const float* g[kRS];
  float* dg[kRS];
  AdamCoef c[kRS];
  int64_t n;
  int32_t init_mv;  // 0: the run holds the last unrolled step (zero dM, dV before it)
};

template <int C>
__device__ __forceinline__ void urbwd_vector(int64_t i, const URBwdArgs& a) {
  const f32x4 dP = ld(cv4(a.dP) + i);
  const f32x4 M0 = ld(cv4(a.m0) + i), V0 = ld(cv4(a.v0) + i);
  f32x4 G[C];
#pragma unroll
  for (int s = 0; s < C; ++s) G[s] = ld(cv4(a.g[s]) + i);
  f32x4 dM = {0.0f, 0.0f, 0.0f, 0.0f}, dV = {0.0f, 0.0f, 0.0f, 0.0f};
  if (a.init_mv) {
    dM = ld(cv4(a.dm) + i);
    dV = ld(cv4(a.dv) + i);
  }
#if DIFFOPT_REMAT_QUAD_FLAT
  // each VJP step recomputes its input moments from (M0, V0): C(C-1)/2
  // moment steps instead of C - 1, and no trajectory held in registers
#pragma unroll
  for (int s = C - 1; s >= 0; --s) {
    f32x4 M, V;
    run_moments<C>(s, M0, V0, G, a.c, M, V);
    if (s == C - 1 && !a.init_mv) ubwd_step<false>(dP, dM, dV, G[s], M, V, a.c[s], v4(a.dg[s]) + i);
    else ubwd_step<true>(dP, dM, dV, G[s], M, V, a.c[s], v4(a.dg[s]) + i);
  }
#else
  f32x4 M[C], V[C];  // M[s], V[s]: the moments step s consumed
  M[0] = M0;
  V[0] = V0;
#pragma unroll
  for (int s = 0; s + 1 < C; ++s) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      M[s + 1][e] = moment1(G[s][e], M[s][e], a.c[s]);
      V[s + 1][e] = moment2(G[s][e], V[s][e], a.c[s]);
    }
  }
  if (a.init_mv) ubwd_step<true>(dP, dM, dV, G[C - 1], M[C - 1], V[C - 1], a.c[C - 1], v4(a.dg[C - 1]) + i);
  else ubwd_step<false>(dP, dM, dV, G[C - 1], M[C - 1], V[C - 1], a.c[C - 1], v4(a.dg[C - 1]) + i);
#pragma unroll
  for (int s = C - 2; s >= 0; --s) ubwd_step<true>(dP, dM, dV, G[s], M[s], V[s], a.c[s], v4(a.dg[s]) + i);
#endif
  st(v4(a.dm) + i, dM);
  st(v4(a.dv) + i, dV);
}

template <int C>
__device__ __forceinline__ void urbwd_element(int64_t e, const URBwdArgs& a) {
  const float dP = a.dP[e];
  float G[C], M[C], V[C];
  M[0] = a.m0[e];
  V[0] = a.v0[e];
#pragma unroll
  for (int s = 0; s < C; ++s) G[s] = a.g[s][e];
#pragma unroll
  for (int s = 0; s + 1 < C; ++s) {
    M[s + 1] = moment1(G[s], M[s], a.c[s]);
    V[s + 1] = moment2(G[s], V[s], a.c[s]);
  }
  float dM = 0.0f, dV = 0.0f;
  BwdOut o;
  if (a.init_mv) o = bwd_elem<true>(dP, a.dm[e], a.dv[e], G[C - 1], M[C - 1], V[C - 1], a.c[C - 1]);
  else o = bwd_elem<false>(dP, 0.0f, 0.0f, G[C - 1], M[C - 1], V[C - 1], a.c[C - 1]);
  a.dg[C - 1][e] = o.g;
  dM = o.m;
  dV = o.v;
#pragma unroll
  for (int s = C - 2; s >= 0; --s) {
    o = bwd_elem<true>(dP, dM, dV, G[s], M[s], V[s], a.c[s]);
    a.dg[s][e] = o.g;
    dM = o.m;
    dV = o.v;
  }
  a.dm[e] = dM;
  a.dv[e] = dV;
}

// Small buffers (see adam_unrolled_fwd_small): the arithmetic of urbwd_element.
template <int C>
__global__ __launch_bounds__(kSEB) void adam_unrolled_bwd_remat_small(URBwdArgs a) {
  warm_args(fold_lines(a));
  const int64_t e = (int64_t)blockIdx.x * kSEB + threadIdx.x;
  if (e >= a.n) return;
  const float dP = a.dP[e];
  const float dMi = (a.init_mv ? a.dm : a.dP)[e], dVi = (a.init_mv ? a.dv : a.dP)[e];
  float G[C], M[C], V[C];
  M[0] = a.m0[e];
  V[0] = a.v0[e];
#pragma unroll
  for (int s = 0; s < C; ++s) G[s] = a.g[s][e];
#pragma unroll
  for (int s = 0; s + 1 < C; ++s) {
    M[s + 1] = moment1(G[s], M[s], a.c[s]);
    V[s + 1] = moment2(G[s], V[s], a.c[s]);
  }
  BwdOut o = a.init_mv ? bwd_elem<true>(dP, dMi, dVi, G[C - 1], M[C - 1], V[C - 1], a.c[C - 1])
                       : bwd_elem<false>(dP, 0.0f, 0.0f, G[C - 1], M[C - 1], V[C - 1], a.c[C - 1]);
  a.dg[C - 1][e] = o.g;
  float dM = o.m, dV = o.v;
#pragma unroll
  for (int s = C - 2; s >= 0; --s) {
    o = bwd_elem<true>(dP, dM, dV, G[s], M[s], V[s], a.c[s]);
    a.dg[s][e] = o.g;
    dM = o.m;
    dV = o.v;
  }
  a.dm[e] = dM;
  a.dv[e] = dV;
}

template <int C, int B>
__global__ __launch_bounds__(B) void adam_unrolled_bwd_remat_vec(URBwdArgs a) {
  const int64_t nv = a.n >> 2;
  const int64_t ntiles = (nv + B - 1) / B;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t i = t * B + threadIdx.x;
    if (i < nv) urbwd_vector<C>(i, a);
  }
  if (blockIdx.x == gridDim.x - 1) {
    const int64_t e = (nv << 2) + threadIdx.x;
    if (e < a.n) urbwd_element<C>(e, a);
  }
}

template <int C, int B>
__global__ __launch_bounds__(B) void adam_unrolled_bwd_remat_elem(URBwdArgs a) {
  for (int64_t e = (int64_t)blockIdx.x * B + threadIdx.x; e < a.n; e += (int64_t)gridDim.x * B)
    urbwd_element<C>(e, a);
}

// Long runs hold more registers per lane, so fewer waves fit on a SIMD; they
// take smaller workgroups so that whole workgroups still fill the CU.
template <int C>
void launch_urbwd(bool vec, const URBwdArgs& a, hipStream_t st) {
  constexpr int B = C >= DIFFOPT_URBWD_LONG_RUN ? DIFFOPT_URBWD_BLOCK_LONG : kURB;
  constexpr int BS = B < kSmallB ? B : kSmallB;
  if (a.n <= kSmallElems)
    hipLaunchKernelGGL((adam_unrolled_bwd_remat_small<C>), dim3((unsigned)((a.n + kSEB - 1) / kSEB)), dim3(kSEB), 0,
                       st, a);
  else if (vec && (a.n >> 2) < kSmallVecs)
    hipLaunchKernelGGL((adam_unrolled_bwd_remat_vec<C, BS>), dim3((unsigned)grid_for(((a.n >> 2) + BS - 1) / BS)),
                       dim3(BS), 0, st, a);
  else if (vec)
    hipLaunchKernelGGL((adam_unrolled_bwd_remat_vec<C, B>), dim3((unsigned)grid_for(((a.n >> 2) + B - 1) / B)),
                       dim3(B), 0, st, a);
  else
    hipLaunchKernelGGL((adam_unrolled_bwd_remat_elem<C, B>), dim3((unsigned)grid_for((a.n + B - 1) / B)), dim3(B),
                       0, st, a);
}

// Run length C is a template argument so the trajectory stays in registers.
int launch_urbwd_c(const char* who, int C, bool vec, const URBwdArgs& a, hipStream_t st) {
  switch (C) {
    case 1: launch_urbwd<1>(vec, a, st); break;
    case 2: launch_urbwd<2>(vec, a, st); break;
    case 3: launch_urbwd<3>(vec, a, st); break;
    case 4: launch_urbwd<4>(vec, a, st); break;
    case 5: launch_urbwd<5>(vec, a, st); break;
    case 6: launch_urbwd<6>(vec, a, st); break;
    case 7: launch_urbwd<7>(vec, a, st); break;
    case 8: launch_urbwd<8>(vec, a, st); break;
    default: return fail(DIFFOPT_EINVAL, "%s: recompute run of %d steps (at most %d)", who, C, kRS);
  }
  return DIFFOPT_OK;
}
static_assert(kRS == 8, "launch_urbwd_c instantiates run lengths 1..8");

// ---- host launchers ------------------------------------------------------------

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
  for (int64_t k = 0; k < K; ++k)
    if (!grads[k]) return fail(DIFFOPT_EINVAL, "%s: null grads entry %lld", who, (long long)k);
  int rc = check_trajectory(who, K, mu_traj, nu_traj, true, false);
  if (rc) return rc;
  hipStream_t st = as_stream(stream);
  bool vec = aligned16(p0) && aligned16(pK);
  for (int64_t k = 0; k <= K; ++k) {
    vec = vec && aligned16(mu_traj[k]) && aligned16(nu_traj[k]);
    if (k < K) vec = vec && aligned16(grads[k]);
  }
  for (int64_t k0 = 0; k0 < K; k0 += kUK) {  // one fused launch per kUK steps
    UFwdArgs a;
    a.K = (int32_t)(K - k0 < kUK ? K - k0 : kUK);
    a.n = n;
    // Between launches the running params pass through pK.  The running
    // moments pass through the state stored at the boundary, or, when that
    // entry is NULL, through the final-state buffers mu_traj[K], nu_traj[K]
    // (each lane reads its elements there before writing them).
    a.p = (k0 == 0) ? p0 : pK;
    a.m0 = mu_traj[k0] ? mu_traj[k0] : mu_traj[K];
    a.v0 = nu_traj[k0] ? nu_traj[k0] : nu_traj[K];
    a.pK = pK;
    for (int s = 0; s < kUK; ++s) {
      const bool on = s < a.K;
      a.g[s] = on ? grads[k0 + s] : nullptr;
      a.m[s] = on ? mu_traj[k0 + s + 1] : nullptr;
      a.v[s] = on ? nu_traj[k0 + s + 1] : nullptr;
      if (on) make_coef(who, count0 + k0 + s, lr, b1, b2, eps, eps_root, &a.c[s]);
      else a.c[s] = AdamCoef{};
    }
    if (!a.m[a.K - 1]) {  // boundary state not stored: carry it in the final-state buffers
      a.m[a.K - 1] = mu_traj[K];
      a.v[a.K - 1] = nu_traj[K];
    }
    if (n <= kSmallElems)
      dispatch_k<UFwdArgs, FwdSmall>(a.K, a, st);
    else if (vec && (n >> 2) < kSmallVecs)
      hipLaunchKernelGGL((adam_unrolled_fwd_vec<kSmallB>), dim3((unsigned)grid_for(((n >> 2) + kSmallB - 1) / kSmallB)),
                         dim3(kSmallB), 0, st, a);
    else if (vec)
      hipLaunchKernelGGL((adam_unrolled_fwd_vec<kUFB>), dim3((unsigned)grid_for(((n >> 2) + kUFB - 1) / kUFB)),
                         dim3(kUFB), 0, st, a);
    else  // some pointer is not 16-byte aligned: one element per lane, same arithmetic
      hipLaunchKernelGGL(adam_unrolled_fwd_elem, dim3((unsigned)grid_for((n + kUFB - 1) / kUFB)), dim3(kUFB), 0, st,
                         a);
    rc = launch_status(who);
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
  for (int64_t k = 0; k < K; ++k)
    if (!grads[k] || !dgrads[k]) return fail(DIFFOPT_EINVAL, "%s: null entry %lld in grads or dgrads", who,
                                             (long long)k);
  int rc = check_trajectory(who, K, mu_traj, nu_traj, false, true);
  if (rc) return rc;
  hipStream_t st = as_stream(stream);
  bool vec = aligned16(dpK) && aligned16(dmu0) && aligned16(dnu0);
  for (int64_t k = 0; k < K; ++k)
    vec = vec && aligned16(grads[k]) && aligned16(mu_traj[k]) && aligned16(nu_traj[k]) && aligned16(dgrads[k]);
  // Last steps first.  Steps whose input state was stored run up to kUK per
  // launch, reading it back; a run of steps j+1..khi whose states were not
  // stored (only mu_j, nu_j) runs in one launch that recomputes them.
  for (int64_t khi = K; khi >= 1;) {
    const bool init_mv = khi != K;  // the first launch starts from zero cotangents of mu_K, nu_K
    if (mu_traj[khi - 1]) {
      UBwdArgs a;
      int32_t run = 0;
      while (run < kUK && khi - run >= 1 && mu_traj[khi - run - 1]) ++run;
      a.K = run;
      a.n = n;
      a.dP = dpK;
      a.dm = dmu0;
      a.dv = dnu0;
      a.init_mv = init_mv;
      for (int s = 0; s < kUK; ++s) {
        const bool on = s < a.K;
        const int64_t k = khi - s;  // unrolled step (1-based) run as the launch's step s
        a.g[s] = on ? grads[k - 1] : nullptr;
        a.m[s] = on ? mu_traj[k - 1] : nullptr;
        a.v[s] = on ? nu_traj[k - 1] : nullptr;
        a.dg[s] = on ? dgrads[k - 1] : nullptr;
        if (on) make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &a.c[s]);
        else a.c[s] = AdamCoef{};
      }
      if (n <= kSmallElems)
        dispatch_k<UBwdArgs, BwdSmall>(a.K, a, st);
      else if (vec && (n >> 2) < kSmallVecs)
        hipLaunchKernelGGL((adam_unrolled_bwd_vec<kSmallB>),
                           dim3((unsigned)grid_for(((n >> 2) + kSmallB - 1) / kSmallB)), dim3(kSmallB), 0, st, a);
      else if (vec)
        hipLaunchKernelGGL((adam_unrolled_bwd_vec<kUBB>), dim3((unsigned)grid_for(((n >> 2) + kUBB - 1) / kUBB)),
                           dim3(kUBB), 0, st, a);
      else
        hipLaunchKernelGGL(adam_unrolled_bwd_elem, dim3((unsigned)grid_for((n + kUBB - 1) / kUBB)), dim3(kUBB), 0,
                           st, a);
      khi -= run;
    } else {
      int64_t j = khi - 1;
      while (!mu_traj[j]) --j;  // mu_traj[0] is stored; check_trajectory bounds khi - j by kRS
      URBwdArgs a;
      const int C = (int)(khi - j);
      a.n = n;
      a.dP = dpK;
      a.dm = dmu0;
      a.dv = dnu0;
      a.m0 = mu_traj[j];
      a.v0 = nu_traj[j];
      a.init_mv = init_mv;
      for (int s = 0; s < kRS; ++s) {
        const bool on = s < C;
        a.g[s] = on ? grads[j + s] : nullptr;
        a.dg[s] = on ? dgrads[j + s] : nullptr;
        if (on) make_coef(who, count0 + j + s, lr, b1, b2, eps, eps_root, &a.c[s]);
        else a.c[s] = AdamCoef{};
      }
      rc = launch_urbwd_c(who, C, vec, a, st);
      if (rc) return rc;
      khi = j;
    }
    rc = launch_status(who);
    if (rc) return rc;
  }
  return DIFFOPT_OK;
}
