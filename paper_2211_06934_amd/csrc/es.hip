// Zero-order (evolution-strategies) gradient estimation on gfx950 (TorchOpt,
// Sec. 2.2 "Zero-order Differentiation"): the gradient of the Gaussian
// smoothing E_z[f(theta + s z)] is (1/s) E_z[f(theta + s z) z], estimated by
// Monte-Carlo over N noise vectors.  The noise is an input ([N][n], row-major,
// drawn by the caller), so both kernels are plain streams over it:
//   perturb:   row i = theta + s z_i (antithetic: row N + i = theta - s z_i)
//   estimate:  grad_j = scale * sum_i w_i z_ij   (weights from the caller's f)
// The estimate is a weighted reduction of N rows: a [1 x N] x [N x n] product
// with about 0.5 flop per byte, HBM-bound, so it is a stream (each lane owns one
// 16-byte slice of grad and walks the N rows), not a matrix-core contraction.
#include <cmath>

#include "adam_math.hpp"

#ifndef DIFFOPT_ES_PERTURB_ROWS
#define DIFFOPT_ES_PERTURB_ROWS 8
#endif


namespace diffopt {
namespace {

constexpr int kEB = 256;   // threads per workgroup
constexpr int kRows = DIFFOPT_ES_PERTURB_ROWS;  // noise rows per workgroup in perturb
constexpr int kUnroll = 8; // rows in flight per lane in estimate
constexpr int kMaxClasses = 8;  // phase classes of the noise rows
// Measured on MI355X (n = 11,689,512, N = 64): 4 slices per lane 0.50 ms,
// 2 slices 0.51, 1 slice 0.54.
#ifndef DIFFOPT_ES_EST_U
#define DIFFOPT_ES_EST_U 4
#endif
constexpr int kEstU = DIFFOPT_ES_EST_U;  // 16-byte grad slices per lane in estimate

// Rows of the [N][n] noise start at 16-byte phases p_i = (base/16 + i nv) mod 8
// within the 128-byte lines; a wave's 64 vectors of a row then span 9 lines
// instead of 8 unless the lanes are shifted by p_i.  Rows i and i + P, with
// P = 8 / gcd(nv mod 8, 8), share a phase, so the rows are split into P
// phase classes and every workgroup takes kRows rows of one class, its lanes
// shifted by that class's phase: each wave touches whole lines of every row it
// reads.  At n = 11,689,512 (rows 32 bytes out of phase in turn) the
// unshifted layout fetched 15% more lines than it used; shifted, the kernel
// went from 1.84 to 1.64-1.71 ms.  The row stride inside a group (P, or a
// larger power of two) measured the same.
struct PerturbPlan {
  int64_t gstart[kMaxClasses + 1];  // first grid-y index of each class (gstart[P] = total)
  int32_t shift[kMaxClasses];       // lane shift of each class (vectors)
  int32_t P;                        // classes: rows i and i + P share a phase
};

// Grid: x over 16-byte vectors of theta (shifted per class), y over groups of
// kRows same-phase samples.  The dispatcher walks x fastest, so the chip
// works through one group of rows at a time (few DRAM pages open at once);
// theta is re-read per group, mostly from the Infinity Cache.  A lane issues
// all of its group's row loads first.
__global__ __launch_bounds__(kEB) void es_perturb_vec(const float* theta, const float* noise, int64_t N,
                                                       int64_t nv, float sigma, int antithetic, float* out,
                                                       PerturbPlan plan) {
  int r = 0;  // phase class of this group
  while (r + 1 < plan.P && (int64_t)blockIdx.y >= plan.gstart[r + 1]) ++r;
  const int64_t v = (int64_t)blockIdx.x * kEB + threadIdx.x - plan.shift[r];
  if (v < 0 || v >= nv) return;
  const int64_t P = plan.P;
  const int64_t i0 = r + P * ((int64_t)kRows * ((int64_t)blockIdx.y - plan.gstart[r]));  // first row; rows step by P
  const f32x4 t = ld(reinterpret_cast<const f32x4*>(theta) + v);
  const f32x4* z = reinterpret_cast<const f32x4*>(noise) + v;
  f32x4* o = reinterpret_cast<f32x4*>(out) + v;
  if (i0 + P * (kRows - 1) < N) {
    f32x4 rw[kRows];
#pragma unroll
    for (int u = 0; u < kRows; ++u) rw[u] = ld(z + (i0 + P * u) * nv);
#pragma unroll
    for (int u = 0; u < kRows; ++u) {
      const int64_t i = i0 + P * u;
      f32x4 a, b;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = fmaf(sigma, rw[u][e], t[e]);
        b[e] = fmaf(-sigma, rw[u][e], t[e]);
      }
      st(o + i * nv, a);
      if (antithetic) st(o + (N + i) * nv, b);
    }
  } else {
    for (int64_t i = i0; i < N; i += P) {
      const f32x4 rw = ld(z + i * nv);
      f32x4 a, b;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = fmaf(sigma, rw[e], t[e]);
        b[e] = fmaf(-sigma, rw[e], t[e]);
      }
      st(o + i * nv, a);
      if (antithetic) st(o + (N + i) * nv, b);
    }
  }
}

__global__ __launch_bounds__(kEB) void es_perturb_scalar(const float* theta, const float* noise, int64_t N,
                                                          int64_t n, float sigma, int antithetic, float* out) {
  const int64_t j = (int64_t)blockIdx.x * kEB + threadIdx.x;
  if (j >= n) return;
  const float t = theta[j];
  const int64_t i0 = (int64_t)blockIdx.y * kRows;
  const int64_t i1 = i0 + kRows < N ? i0 + kRows : N;
  for (int64_t i = i0; i < i1; ++i) {
    const float z = noise[i * n + j];
    out[i * n + j] = fmaf(sigma, z, t);
    if (antithetic) out[(N + i) * n + j] = fmaf(-sigma, z, t);
  }
}

// Each lane owns kEstU 16-byte slices of grad, kEB vectors apart, and
// accumulates the N rows in sample order, kUnroll rows in flight.  A
// workgroup thus covers kEB * kEstU contiguous vectors of every row; rows
// start at varying 16-byte phases of the 128-byte lines, so the lines at the
// ends of a workgroup's range are also fetched by its neighbours, and a wider
// range makes that a smaller share.
__global__ __launch_bounds__(kEB) void es_estimate_vec(const float* noise, const float* __restrict__ w, int64_t N,
                                                        int64_t nv, float scale, float* grad) {
  const int64_t v0 = (int64_t)blockIdx.x * (kEB * kEstU) + threadIdx.x;
  const f32x4* z = reinterpret_cast<const f32x4*>(noise);
  f32x4 acc[kEstU];
  bool on[kEstU];
#pragma unroll
  for (int q = 0; q < kEstU; ++q) {
    acc[q] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    on[q] = v0 + (int64_t)q * kEB < nv;
  }
  if (!on[0]) return;
  int64_t i = 0;
  for (; i + kUnroll <= N; i += kUnroll) {
    f32x4 r[kUnroll][kEstU];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int q = 0; q < kEstU; ++q)
        if (on[q]) r[u][q] = ld(z + (i + u) * nv + v0 + (int64_t)q * kEB);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const float wi = w[i + u];
#pragma unroll
      for (int q = 0; q < kEstU; ++q)
        if (on[q])
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[q][e] = fmaf(wi, r[u][q][e], acc[q][e]);
    }
  }
  for (; i < N; ++i) {
    const float wi = w[i];
#pragma unroll
    for (int q = 0; q < kEstU; ++q)
      if (on[q]) {
        const f32x4 r = ld(z + i * nv + v0 + (int64_t)q * kEB);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[q][e] = fmaf(wi, r[e], acc[q][e]);
      }
  }
#pragma unroll
  for (int q = 0; q < kEstU; ++q)
    if (on[q]) {
      f32x4 out;
#pragma unroll
      for (int e = 0; e < 4; ++e) out[e] = scale * acc[q][e];
      st(reinterpret_cast<f32x4*>(grad) + v0 + (int64_t)q * kEB, out);
    }
}

__global__ __launch_bounds__(kEB) void es_estimate_scalar(const float* noise, const float* __restrict__ w, int64_t N,
                                                           int64_t n, float scale, float* grad) {
  const int64_t j = (int64_t)blockIdx.x * kEB + threadIdx.x;
  if (j >= n) return;
  float acc = 0.0f;
  for (int64_t i = 0; i < N; ++i) acc = fmaf(w[i], noise[i * n + j], acc);
  grad[j] = scale * acc;
}

bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool al4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

}  // namespace
}  // namespace diffopt

using namespace diffopt;

extern "C" int diffopt_es_perturb(const float* params, const float* noise, int64_t num_samples, int64_t n,
                                  double sigma, int32_t antithetic, float* out, void* stream) {
  clear_error();
  static const char* who = "diffopt_es_perturb";
  if (n < 0 || num_samples < 0) return fail(DIFFOPT_EINVAL, "%s: n and num_samples must be >= 0", who);
  if (!std::isfinite(sigma)) return fail(DIFFOPT_EINVAL, "%s: sigma must be finite", who);
  if (n == 0 || num_samples == 0) return DIFFOPT_OK;
  if (!params || !noise || !out) return fail(DIFFOPT_EINVAL, "%s: null required pointer", who);
  if (!al4(params) || !al4(noise) || !al4(out)) return fail(DIFFOPT_EINVAL, "%s: pointers must be 4-byte aligned", who);
  const int64_t groups = (num_samples + kRows - 1) / kRows;
  hipStream_t st = as_stream(stream);
  const bool vec = (n % 4 == 0) && al16(params) && al16(noise) && al16(out);
  if (vec) {
    const int64_t nv = n / 4;
    PerturbPlan plan{};
    const int64_t q = nv % 8;
    int64_t g = 8;  // gcd(q, 8)
    if (q != 0) {
      g = q;
      for (int64_t b = 8; b != 0;) {
        const int64_t t = g % b;
        g = b;
        b = t;
      }
    }
    const int64_t P = 8 / g;  // rows i and i + P share a phase
    plan.P = (int32_t)(P < num_samples ? P : num_samples);
    const int64_t base = (int64_t)((reinterpret_cast<uintptr_t>(noise) >> 4) & 7u);
    int64_t gy = 0;
    for (int r = 0; r < plan.P; ++r) {
      plan.gstart[r] = gy;
      plan.shift[r] = (int32_t)((base + (int64_t)r * q) & 7);  // row r's phase, in vectors
      const int64_t rows = (num_samples - r + plan.P - 1) / plan.P;
      gy += (rows + kRows - 1) / kRows;
    }
    plan.gstart[plan.P] = gy;
    if (gy > 65535) return fail(DIFFOPT_EINVAL, "%s: num_samples too large (max about %d)", who, 65535 * kRows);
    const int64_t bx = (nv + 7 + kEB - 1) / kEB;  // lanes shifted by up to 7 vectors
    if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large", who);
    hipLaunchKernelGGL(es_perturb_vec, dim3((unsigned)bx, (unsigned)gy), dim3(kEB), 0, st, params, noise,
                       num_samples, nv, (float)sigma, antithetic ? 1 : 0, out, plan);
  } else {
    if (groups > 65535) return fail(DIFFOPT_EINVAL, "%s: num_samples too large (max %d)", who, 65535 * kRows);
    const int64_t bx = (n + kEB - 1) / kEB;
    if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large", who);
    hipLaunchKernelGGL(es_perturb_scalar, dim3((unsigned)bx, (unsigned)groups), dim3(kEB), 0, st, params, noise,
                       num_samples, n, (float)sigma, antithetic ? 1 : 0, out);
  }
  return launch_status(who);
}

extern "C" int diffopt_es_estimate(const float* noise, const float* weights, int64_t num_samples, int64_t n,
                                   double scale, float* grad, void* stream) {
  clear_error();
  static const char* who = "diffopt_es_estimate";
  if (n < 0 || num_samples < 0) return fail(DIFFOPT_EINVAL, "%s: n and num_samples must be >= 0", who);
  if (!std::isfinite(scale)) return fail(DIFFOPT_EINVAL, "%s: scale must be finite", who);
  if (n == 0) return DIFFOPT_OK;
  if (!grad || (num_samples > 0 && (!noise || !weights)))
    return fail(DIFFOPT_EINVAL, "%s: null required pointer", who);
  if (!al4(noise) || !al4(weights) || !al4(grad)) return fail(DIFFOPT_EINVAL, "%s: pointers must be 4-byte aligned", who);
  hipStream_t st = as_stream(stream);
  const bool vec = (n % 4 == 0) && al16(grad) && (num_samples == 0 || al16(noise));
  if (vec) {
    const int64_t nv = n / 4;
    const int64_t bx = (nv + kEB * kEstU - 1) / (kEB * kEstU);
    if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large", who);
    hipLaunchKernelGGL(es_estimate_vec, dim3((unsigned)bx), dim3(kEB), 0, st, noise, weights, num_samples, nv,
                       (float)scale, grad);
  } else {
    const int64_t bx = (n + kEB - 1) / kEB;
    if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large", who);
    hipLaunchKernelGGL(es_estimate_scalar, dim3((unsigned)bx), dim3(kEB), 0, st, noise, weights, num_samples, n,
                       (float)scale, grad);
  }
  return launch_status(who);
}
