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

// ---- Gaussian noise generated in registers -----------------------------------
//
// z_ij (sample i, parameter j) is a pure function of (seed, i, j), so the
// perturb and estimate kernels each regenerate the noise instead of reading
// an N x n array: the pass moves 4n + 8Nn bytes (antithetic) instead of
// about 4n + 20Nn.  The normals come from Philox-4x64-10 (Salmon et al.,
// SC 2011) blocks at counter (block, i, 0, 0) under key (seed, 0), through
// the Box-Muller transform.  Block 64 s + l (segment s of 512 parameters,
// slot l < 64) covers parameters 512 s + 4 l + e (words 0 and 1) and
// 512 s + 256 + 4 l + e (words 2 and 3), e < 4; even e takes its word's cosine
// normal, odd e the sine one.  A lane owns one block, so the 64 lanes of a
// wave own one segment and each of the wave's two 128-bit store
// instructions writes one contiguous 1 KiB run.

constexpr uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhiloxM1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kPhiloxW1 = 0xBB67AE8584CAA73Bull;

// Full 128-bit product of a 64-bit constant and a 64-bit value from four
// 32 x 32 -> 64-bit partial products, each with its carry-in folded into the
// same multiply-add (none of the sums can overflow 64 bits).  Forming the low
// and high halves separately (a 64-bit multiply and __umul64hi) repeats
// three of the four partial products.
template <uint64_t M>
__device__ __forceinline__ void mul128(uint64_t c, uint64_t& lo, uint64_t& hi) {
  constexpr uint64_t ml = M & 0xffffffffull, mh = M >> 32;
  const uint64_t cl = c & 0xffffffffull, ch = c >> 32;
  const uint64_t t0 = cl * ml;
  const uint64_t t1 = cl * mh + (t0 >> 32);
  const uint64_t t2 = ch * ml + (t1 & 0xffffffffull);
  hi = ch * mh + (t1 >> 32) + (t2 >> 32);
  lo = (t2 << 32) | (t0 & 0xffffffffull);
}

// a ^ b ^ c on 64-bit words through the three-input bitwise instruction
// (truth table 0x96), one per 32-bit half instead of two two-input xors.
__device__ __forceinline__ uint64_t xor3(uint64_t a, uint64_t b, uint64_t c) {
  const uint32_t lo = __builtin_amdgcn_bitop3_b32((uint32_t)a, (uint32_t)b, (uint32_t)c, 0x96);
  const uint32_t hi = __builtin_amdgcn_bitop3_b32((uint32_t)(a >> 32), (uint32_t)(b >> 32), (uint32_t)(c >> 32), 0x96);
  return ((uint64_t)hi << 32) | lo;
}

// Ten rounds of Philox-4x64: per round the two 64 x 64 -> 128-bit products
// M0 c0 and M1 c2, then c <- (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the
// key advances by the Weyl increments between rounds.  The counter here is
// (block, sample, 0, 0) and the key (seed, 0).
__device__ __forceinline__ void philox_block(uint64_t block, uint64_t sample, uint64_t seed, uint64_t out[4]) {
  uint64_t c0 = block, c1 = sample, c2 = 0, c3 = 0;
  uint64_t k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    uint64_t lo0, hi0, lo1, hi1;
    mul128<kPhiloxM0>(c0, lo0, hi0);
    mul128<kPhiloxM1>(c2, lo1, hi1);
    // The first two rounds are left to the compiler, which keeps their
    // sample- and seed-only terms in scalar registers.
    const uint64_t n0 = r < 2 ? hi1 ^ c1 ^ k0 : xor3(hi1, c1, k0);
    const uint64_t n2 = r < 2 ? hi0 ^ c3 ^ k1 : xor3(hi0, c3, k1);
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

// Box-Muller on one 64-bit word: 24-bit uniforms u1 = (lo/2^8 + 1) 2^-24 in
// (0, 1] and u2 = (hi/2^8) 2^-24 in [0, 1), exact in fp32; r = sqrt(-2 ln u1),
// za = r cos(2 pi u2), zb = r sin(2 pi u2).  The transcendentals are the
// hardware instructions: v_log_f32 (log2, so ln u1 = ln 2 log2 u1),
// v_sqrt_f32, and v_sin_f32 / v_cos_f32, whose argument is in revolutions,
// so they take u2 itself.  Over all 2^24 values of each uniform, measured
// against fp64 on MI355X: sin and cos within 1.3e-7 absolute, r within
// 1.4e-7 relative, so each normal is within about 3.5e-7 r of its exact
// value.  The library's logf / sincospif are about three times as accurate
// and cost several times the instructions in a kernel whose time is set by
// this arithmetic.
__device__ __forceinline__ void box_muller(uint64_t w, float& za, float& zb) {
  const uint32_t lo = static_cast<uint32_t>(w), hi = static_cast<uint32_t>(w >> 32);
  const float u1 = static_cast<float>((lo >> 8) + 1u) * 0x1p-24f;
  const float u2 = static_cast<float>(hi >> 8) * 0x1p-24f;
  constexpr float kMinus2Ln2 = -1.38629436111989061f;
  const float r = __builtin_amdgcn_sqrtf(kMinus2Ln2 * __builtin_amdgcn_logf(u1));
  za = r * __builtin_amdgcn_cosf(u2);
  zb = r * __builtin_amdgcn_sinf(u2);
}

// The eight normals of block `block` of sample `sample`: z[0..3] belong to
// the block's first four parameters, z[4..7] to its second four.
__device__ __forceinline__ void noise8(uint64_t block, uint64_t sample, uint64_t seed, float z[8]) {
  uint64_t w[4];
  philox_block(block, sample, seed, w);
#pragma unroll
  for (int q = 0; q < 4; ++q) box_muller(w[q], z[2 * q], z[2 * q + 1]);
}

// First parameter of the two runs of four that block b covers.
__device__ __forceinline__ int64_t run_start(int64_t b, int h) { return 512 * (b >> 6) + 256 * h + 4 * (b & 63); }

// Weight of sample i from the caller's evaluations f (method 0 plain: f_i;
// 1 baseline: f_i - f0; 2 antithetic: f_i - f_{N+i}).
__device__ __forceinline__ float es_weight(const float* __restrict__ f, const float* __restrict__ f0, int64_t N,
                                           int method, int64_t i) {
  if (method == 0) return f[i];
  if (method == 1) return f[i] - *f0;
  return f[i] - f[N + i];
}

#ifndef DIFFOPT_ES_GROWS
#define DIFFOPT_ES_GROWS 8
#endif
constexpr int kGRows = DIFFOPT_ES_GROWS;  // samples per lane in the Gaussian perturb

// Grid: x over Philox blocks (one per lane), y over groups of kGRows samples.
// A lane reads its eight theta values once and writes its eight parameters
// of every sample of the group (and of the antithetic rows).  VEC: n % 4 == 0
// and 16-byte aligned theta and out, so each run of four moves as one
// 128-bit access.
template <bool VEC>
__global__ __launch_bounds__(kEB) void es_perturb_gauss(const float* theta, int64_t N, int64_t n, uint64_t seed,
                                                         float sigma, int antithetic, float* out) {
  const int64_t b = (int64_t)blockIdx.x * kEB + threadIdx.x;
  const int64_t j[2] = {run_start(b, 0), run_start(b, 1)};
  if (j[0] >= n) return;
  int cnt[2];
  float t[8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int64_t left = n - j[h];
    cnt[h] = left <= 0 ? 0 : (left < 4 ? (int)left : 4);
    if (VEC) {
      const f32x4 a = cnt[h] ? *reinterpret_cast<const f32x4*>(theta + j[h]) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int e = 0; e < 4; ++e) t[4 * h + e] = a[e];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) t[4 * h + e] = e < cnt[h] ? theta[j[h] + e] : 0.0f;
    }
  }
  const int64_t i0 = (int64_t)blockIdx.y * kGRows;
  const int64_t i1 = i0 + kGRows < N ? i0 + kGRows : N;
  for (int64_t i = i0; i < i1; ++i) {
    float z[8], a[8], m[8];
    noise8(b, i, seed, z);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[e] = fmaf(sigma, z[e], t[e]);
      m[e] = fmaf(-sigma, z[e], t[e]);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (!cnt[h]) continue;
      float* row = out + i * n + j[h];
      float* rowm = out + (N + i) * n + j[h];
      if (VEC) {
        st(reinterpret_cast<f32x4*>(row), f32x4{a[4 * h], a[4 * h + 1], a[4 * h + 2], a[4 * h + 3]});
        if (antithetic) st(reinterpret_cast<f32x4*>(rowm), f32x4{m[4 * h], m[4 * h + 1], m[4 * h + 2], m[4 * h + 3]});
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (e < cnt[h]) {
            row[e] = a[4 * h + e];
            if (antithetic) rowm[e] = m[4 * h + e];
          }
      }
    }
  }
}

// 128-bit path with line-aligned stores.  A workgroup's waves own as many
// consecutive segments (8 waves: 4096 parameters, 16 KiB of each output row);
// a row starts at a 16-byte phase d within its 128-byte lines
// (d = (address / 16) mod 8, n mod 32 = 8 at the ResNet-18 size).  Stored
// lane by lane, every wave's 1 KiB run would then begin and end inside a
// line, and each partially written line goes to memory in two parts from
// two waves: on MI355X the perturbation took 1.43 ms at n = 11,689,512
// against 1.09 ms at n = 11,689,984 (a multiple of 32).  Here the workgroup
// stages each sample's plus and minus rows in LDS, then stores every row
// in 64-chunk spans that start on a line, chunk c = 64 q + lane - d: only the
// two lines at the workgroup's ends are shared with a neighbour (1.18 ms).
// Measured on MI355X (n = 11,689,512, N = 64 antithetic, two rounds): 8 waves
// per workgroup 1.18 ms, 4 waves 1.20, 2 waves 1.24 (with the sample groups
// outermost in the grid; the order is now chunk-major, below).
#ifndef DIFFOPT_ES_LINE_WAVES
#define DIFFOPT_ES_LINE_WAVES 8
#endif
constexpr int kLW = DIFFOPT_ES_LINE_WAVES;  // waves (segments) per workgroup
// Samples per workgroup.  The grid is one-dimensional with the sample groups
// of one parameter chunk consecutive, so the dispatcher runs them side by side
// and they share the chunk's theta through the cache.  Measured (n =
// 11,689,512, N = 64, six paired rounds): chunk-major order with 8, 4 or 2
// samples per workgroup 1.138, 1.129, 1.137 ms, against 1.176 ms for the
// sample groups outermost (8 per workgroup; 16, 32, 64: 1.185, 1.203, 1.257).
#ifndef DIFFOPT_ES_LINE_ROWS
#define DIFFOPT_ES_LINE_ROWS 4
#endif
constexpr int kLRows = DIFFOPT_ES_LINE_ROWS;
constexpr int kLB = 64 * kLW;
constexpr int kRowChunks = kLW * 128;  // 16-byte chunks of one row per workgroup

__global__ __launch_bounds__(kLB) void es_perturb_gauss_lines(const float* theta, int64_t N, int64_t n,
                                                               uint64_t seed, float sigma, int antithetic,
                                                               uint32_t groups, float* out) {
  __shared__ f32x4 rows[2][kRowChunks];  // the plus and minus rows of one sample
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t chunk = blockIdx.x / groups, group = blockIdx.x - chunk * groups;
  const int64_t b = (int64_t)chunk * kLB + threadIdx.x;
  const int64_t first = (int64_t)chunk * (kRowChunks * 4);  // the workgroup's first parameter
  const int64_t left = (n - first) >> 2;                          // n % 4 == 0 here
  const int nchunks = left < kRowChunks ? (int)left : kRowChunks;
  bool on[2];
  float t[8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    on[h] = run_start(b, h) < n;
    const f32x4 a = on[h] ? *reinterpret_cast<const f32x4*>(theta + run_start(b, h)) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int e = 0; e < 4; ++e) t[4 * h + e] = a[e];
  }
  const int64_t i0 = (int64_t)group * kLRows;
  const int64_t i1 = i0 + kLRows < N ? i0 + kLRows : N;
  const int nrows = antithetic ? 2 : 1;
  for (int64_t i = i0; i < i1; ++i) {
    if (on[0]) {  // a lane past the end computes nothing but still meets both barriers
      float z[8];
      noise8(b, i, seed, z);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        f32x4 pa, pm;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pa[e] = fmaf(sigma, z[4 * h + e], t[4 * h + e]);
          pm[e] = fmaf(-sigma, z[4 * h + e], t[4 * h + e]);
        }
        rows[0][128 * wave + 64 * h + lane] = pa;  // chunk of parameter run_start(b, h)
        if (antithetic) rows[1][128 * wave + 64 * h + lane] = pm;
      }
    }
    __syncthreads();
    for (int r = 0; r < nrows; ++r) {
      float* row = out + (r ? N + i : i) * n + first;
      const int d = (int)((reinterpret_cast<uintptr_t>(row) >> 4) & 7u);
      for (int q = wave; q <= 2 * kLW; q += kLW) {
        const int c = 64 * q + lane - d;
        if (c >= 0 && c < nchunks) st(reinterpret_cast<f32x4*>(row) + c, rows[r][c]);
      }
    }
    __syncthreads();
  }
}

// Each lane owns the eight gradient entries of one Philox block and walks
// the N samples in order, regenerating the block's noise and accumulating
// w_i z_ij in fp32; the result is scaled once at the end.
template <bool VEC>
__global__ __launch_bounds__(kEB) void es_estimate_gauss(const float* __restrict__ f, const float* __restrict__ f0,
                                                          int64_t N, int method, int64_t n, uint64_t seed, float scale,
                                                          float* grad) {
  const int64_t b = (int64_t)blockIdx.x * kEB + threadIdx.x;
  const int64_t j[2] = {run_start(b, 0), run_start(b, 1)};
  if (j[0] >= n) return;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
  for (int64_t i = 0; i < N; ++i) {
    const float wi = es_weight(f, f0, N, method, i);
    float z[8];
    noise8(b, i, seed, z);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = fmaf(wi, z[e], acc[e]);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int64_t left = n - j[h];
    if (left <= 0) continue;
    float* g = grad + j[h];
    if (VEC) {
      st(reinterpret_cast<f32x4*>(g),
         f32x4{scale * acc[4 * h], scale * acc[4 * h + 1], scale * acc[4 * h + 2], scale * acc[4 * h + 3]});
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < left) g[e] = scale * acc[4 * h + e];
    }
  }
}

// weights_i = scale * (method difference of the evaluations), for the
// explicit-noise estimate.
__global__ __launch_bounds__(kEB) void es_weights_kernel(const float* __restrict__ f, const float* __restrict__ f0,
                                                          int64_t N, int method, float scale, float* w) {
  const int64_t i = (int64_t)blockIdx.x * kEB + threadIdx.x;
  if (i < N) w[i] = scale * es_weight(f, f0, N, method, i);
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

namespace {

bool es_method_ok(int32_t method) { return method >= 0 && method <= 2; }

// 1 / (N s), or 1 / (2 N s) for antithetic sampling, formed in fp64 and
// rounded once.
float es_scale(int32_t method, int64_t num_samples, double sigma) {
  return static_cast<float>(1.0 / ((method == 2 ? 2.0 : 1.0) * static_cast<double>(num_samples) * sigma));
}

}  // namespace

extern "C" int diffopt_es_perturb_gaussian(const float* params, int64_t n, int64_t num_samples, uint64_t seed,
                                           double sigma, int32_t antithetic, float* out, void* stream) {
  clear_error();
  static const char* who = "diffopt_es_perturb_gaussian";
  if (n < 0 || num_samples < 0) return fail(DIFFOPT_EINVAL, "%s: n and num_samples must be >= 0", who);
  if (!std::isfinite(sigma)) return fail(DIFFOPT_EINVAL, "%s: sigma must be finite", who);
  if (n == 0 || num_samples == 0) return DIFFOPT_OK;
  if (!params || !out) return fail(DIFFOPT_EINVAL, "%s: null required pointer", who);
  if (!al4(params) || !al4(out)) return fail(DIFFOPT_EINVAL, "%s: pointers must be 4-byte aligned", who);
  const int64_t gy = (num_samples + kGRows - 1) / kGRows;
  if (gy > 65535) return fail(DIFFOPT_EINVAL, "%s: num_samples too large (max %d)", who, 65535 * kGRows);
  const int64_t blocks = 64 * ((n + 511) / 512);  // Philox blocks: 64 per 512 parameters
  const int64_t bx = (blocks + kEB - 1) / kEB;
  if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large", who);
  hipStream_t st = as_stream(stream);
  const dim3 grid((unsigned)bx, (unsigned)gy);
  if (n % 4 == 0 && al16(params) && al16(out)) {
    const int64_t chunks = (blocks + kLB - 1) / kLB, lgroups = (num_samples + kLRows - 1) / kLRows;
    if (chunks * lgroups > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n x num_samples too large", who);
    hipLaunchKernelGGL(es_perturb_gauss_lines, dim3((unsigned)(chunks * lgroups)), dim3(kLB), 0, st, params,
                       num_samples, n, seed, (float)sigma, antithetic ? 1 : 0, (uint32_t)lgroups, out);
  } else
    hipLaunchKernelGGL(es_perturb_gauss<false>, grid, dim3(kEB), 0, st, params, num_samples, n, seed, (float)sigma,
                       antithetic ? 1 : 0, out);
  return launch_status(who);
}

extern "C" int diffopt_es_estimate_gaussian(const float* fvals, const float* f0, int64_t num_samples, int32_t method,
                                            int64_t n, uint64_t seed, double sigma, float* grad, void* stream) {
  clear_error();
  static const char* who = "diffopt_es_estimate_gaussian";
  if (n < 0 || num_samples < 0) return fail(DIFFOPT_EINVAL, "%s: n and num_samples must be >= 0", who);
  if (!es_method_ok(method)) return fail(DIFFOPT_EINVAL, "%s: method must be 0 (plain), 1 (baseline) or 2 "
                                         "(antithetic)", who);
  if (!std::isfinite(sigma) || sigma == 0.0) return fail(DIFFOPT_EINVAL, "%s: sigma must be finite and nonzero", who);
  if (n == 0) return DIFFOPT_OK;
  if (!grad || (num_samples > 0 && (!fvals || (method == 1 && !f0))))
    return fail(DIFFOPT_EINVAL, "%s: null required pointer (f0 is required by the baseline method)", who);
  if (!al4(grad) || (num_samples > 0 && !al4(fvals))) return fail(DIFFOPT_EINVAL, "%s: pointers must be 4-byte "
                                                                  "aligned", who);
  const int64_t blocks = 64 * ((n + 511) / 512);  // Philox blocks: 64 per 512 parameters
  const int64_t bx = (blocks + kEB - 1) / kEB;
  if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: n too large", who);
  const float scale = num_samples > 0 ? es_scale(method, num_samples, sigma) : 0.0f;
  hipStream_t st = as_stream(stream);
  if (n % 4 == 0 && al16(grad))
    hipLaunchKernelGGL(es_estimate_gauss<true>, dim3((unsigned)bx), dim3(kEB), 0, st, fvals, f0, num_samples,
                       (int)method, n, seed, scale, grad);
  else
    hipLaunchKernelGGL(es_estimate_gauss<false>, dim3((unsigned)bx), dim3(kEB), 0, st, fvals, f0, num_samples,
                       (int)method, n, seed, scale, grad);
  return launch_status(who);
}

extern "C" int diffopt_es_weights(const float* fvals, const float* f0, int64_t num_samples, int32_t method,
                                  double sigma, float* weights, void* stream) {
  clear_error();
  static const char* who = "diffopt_es_weights";
  if (num_samples < 0) return fail(DIFFOPT_EINVAL, "%s: num_samples must be >= 0", who);
  if (!es_method_ok(method)) return fail(DIFFOPT_EINVAL, "%s: method must be 0 (plain), 1 (baseline) or 2 "
                                         "(antithetic)", who);
  if (!std::isfinite(sigma) || sigma == 0.0) return fail(DIFFOPT_EINVAL, "%s: sigma must be finite and nonzero", who);
  if (num_samples == 0) return DIFFOPT_OK;
  if (!fvals || !weights || (method == 1 && !f0))
    return fail(DIFFOPT_EINVAL, "%s: null required pointer (f0 is required by the baseline method)", who);
  if (!al4(fvals) || !al4(weights)) return fail(DIFFOPT_EINVAL, "%s: pointers must be 4-byte aligned", who);
  const int64_t bx = (num_samples + kEB - 1) / kEB;
  if (bx > 0x7fffffff) return fail(DIFFOPT_EINVAL, "%s: num_samples too large", who);
  hipLaunchKernelGGL(es_weights_kernel, dim3((unsigned)bx), dim3(kEB), 0, as_stream(stream), fvals, f0, num_samples,
                     (int)method, es_scale(method, num_samples, sigma), weights);
  return launch_status(who);
}
