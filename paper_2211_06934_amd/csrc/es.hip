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

// Grid: x over 16-byte vectors of theta, y over groups of kRows samples.  The
// dispatcher walks x fastest, so the chip works through the rows a group at a
// time (few DRAM pages open at once); theta is re-read per group, mostly from
// the Infinity Cache.  A lane issues all of its group's row loads first.
__global__ __launch_bounds__(kEB) void es_perturb_vec(const float* theta, const float* noise, int64_t N,
                                                       int64_t nv, float sigma, int antithetic, float* out) {
  const int64_t v = (int64_t)blockIdx.x * kEB + threadIdx.x;
  if (v >= nv) return;
  const int64_t i0 = (int64_t)blockIdx.y * kRows;
  const f32x4 t = ld(reinterpret_cast<const f32x4*>(theta) + v);
  const f32x4* z = reinterpret_cast<const f32x4*>(noise) + v;
  f32x4* o = reinterpret_cast<f32x4*>(out) + v;
  if (i0 + kRows <= N) {
    f32x4 r[kRows];
#pragma unroll
    for (int u = 0; u < kRows; ++u) r[u] = ld(z + (i0 + u) * nv);
#pragma unroll
    for (int u = 0; u < kRows; ++u) {
      f32x4 a, b;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = fmaf(sigma, r[u][e], t[e]);
        b[e] = fmaf(-sigma, r[u][e], t[e]);
      }
      st(o + (i0 + u) * nv, a);
      if (antithetic) st(o + (N + i0 + u) * nv, b);
    }
  } else {
    for (int64_t i = i0; i < N; ++i) {
      const f32x4 r = ld(z + i * nv);
      f32x4 a, b;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = fmaf(sigma, r[e], t[e]);
        b[e] = fmaf(-sigma, r[e], t[e]);
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

// Each lane owns one 16-byte slice of grad and accumulates the N rows in
// sample order, kUnroll rows in flight.
__global__ __launch_bounds__(kEB) void es_estimate_vec(const float* noise, const float* __restrict__ w, int64_t N,
                                                        int64_t nv, float scale, float* grad) {
  const int64_t v = (int64_t)blockIdx.x * kEB + threadIdx.x;
  if (v >= nv) return;
  const f32x4* z = reinterpret_cast<const f32x4*>(noise) + v;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  int64_t i = 0;
  for (; i + kUnroll <= N; i += kUnroll) {
    f32x4 r[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) r[u] = ld(z + (i + u) * nv);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const float wi = w[i + u];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = fmaf(wi, r[u][e], acc[e]);
    }
  }
  for (; i < N; ++i) {
    const f32x4 r = ld(z + i * nv);
    const float wi = w[i];
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = fmaf(wi, r[e], acc[e]);
  }
  f32x4 out;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = scale * acc[e];
  st(reinterpret_cast<f32x4*>(grad) + v, out);
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
  if (groups > 65535) return fail(DIFFOPT_EINVAL, "%s: num_samples too large (max %d)", who, 65535 * kRows);
  hipStream_t st = as_stream(stream);
  const bool vec = (n % 4 == 0) && al16(params) && al16(noise) && al16(out);
  if (vec) {
    const int64_t nv = n / 4;
    const int64_t bx = (nv + kEB - 1) / kEB;
    if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large", who);
    hipLaunchKernelGGL(es_perturb_vec, dim3((unsigned)bx, (unsigned)groups), dim3(kEB), 0, st, params, noise,
                       num_samples, nv, (float)sigma, antithetic ? 1 : 0, out);
  } else {
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
    const int64_t bx = (nv + kEB - 1) / kEB;
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
