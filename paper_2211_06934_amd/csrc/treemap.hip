// Leaf-direct ("tree map") differentiable Adam on gfx950: the fused step and
// its VJP applied to every leaf of parameter trees, reading and writing the
// leaves in place of flatten -> flat step -> unflatten (TorchOpt, Appendix D,
// Table 2 "Tree Map"; Sec. 2.3 for the step).  It saves the 8 bytes per element
// that each flatten or unflatten of an operand tree would move.
//
// Work decomposition: the segment table of tree.hip.  Group k of nonempty
// leaf j covers the leaf's elements [4k, 4k + 4); the table gives each leaf
// ceil(numel / 4) + 1 groups rounded up to a multiple of 8, so the last ones
// are empty here.  Leaves start on 8-group boundaries, so for 128-byte aligned
// leaves no cache line is shared by two tiles (which run on different XCDs).  A
// workgroup stages its window of the table in LDS together with the leaf
// addresses of every operand tree, each lane binary-searches the window for
// its groups, issues every operand load of all of its groups, then computes
// and stores.  A group whose four elements exist and whose leaf is 16-byte
// aligned in every operand takes 128-bit loads and stores; any other group is
// processed element by element with the same arithmetic.
#include "adam_math.hpp"
#include "optim_ops.hpp"
#include "segtable.hpp"

// Each workgroup covers one table tile (512 groups).  Measured on MI355X
// (20,000 leaves): the forward is fastest as 512 threads x 1 group (5.8 TB/s
// against 5.3 for 256 x 2), the VJP as 256 threads x 2 groups (5.7 against
// 5.55 for 512 x 1); 128 x 4 is slower for both.
#ifndef DIFFOPT_TM_FWD_BLOCK
#define DIFFOPT_TM_FWD_BLOCK 512
#endif
#ifndef DIFFOPT_TM_BWD_BLOCK
#define DIFFOPT_TM_BWD_BLOCK 256
#endif

namespace diffopt {
namespace {

constexpr int kFB = DIFFOPT_TM_FWD_BLOCK;
constexpr int kBB = DIFFOPT_TM_BWD_BLOCK;
static_assert(kTileGroups % kFB == 0 && kTileGroups % kBB == 0,
              "a workgroup must cover one table tile exactly");

// Device arrays of leaf addresses, one per operand tree (table order).
template <int NA>
struct LeafArrays {
  const uint64_t* a[NA];
};

// Stage the window of tile b: group offsets, element counts, one leaf address
// per operand and an all-operands-aligned flag.  Operands with a null array
// are skipped.  Returns the window length W.
template <int NA, int NT>
__device__ __forceinline__ int stage_window(const SegEntry* __restrict__ seg, const int64_t* __restrict__ tile_first,
                                            const LeafArrays<NA>& arr, int dense_orig, int64_t b, int64_t* s_goff,
                                            int64_t* s_numel, uint64_t (*s_ptr)[kWindowMax], int* s_al) {
  const int64_t j0 = tile_first[b];
  const int W = (int)(tile_first[b + 1] - j0 + 1);
  for (int t = threadIdx.x; t <= W; t += NT) {
    const SegEntry e = seg[j0 + t];
    s_goff[t] = e.goff;
    if (t < W) {
      const int64_t leaf = dense_orig ? j0 + t : e.orig;
      // Every operand's address is loaded unconditionally (a null operand
      // reads the table instead and keeps 0), so all NA loads go out before
      // one wait; a load under the null test was followed by its own wait.
      uint64_t v[NA];
#pragma unroll
      for (int q = 0; q < NA; ++q) {
        const uint64_t* src = arr.a[q] ? arr.a[q] + leaf : reinterpret_cast<const uint64_t*>(seg);
        v[q] = *src;
      }
      uint64_t any = 0;
#pragma unroll
      for (int q = 0; q < NA; ++q) {
        const uint64_t ptr = arr.a[q] ? v[q] : 0;
        s_ptr[q][t] = ptr;
        any |= ptr;
      }
      s_numel[t] = e.numel;
      s_al[t] = (any & 15u) == 0;
    }
  }
  return W;
}

__device__ __forceinline__ int find_leaf(const int64_t* s_goff, int W, int64_t gidx) {
  int lo = 0, hi = W - 1;  // s_goff[0] <= gidx by construction
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_goff[mid] <= gidx) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

template <typename T>
__device__ __forceinline__ gptr<T> at(uint64_t base, int64_t i) {
  return gaddr<T>(base) + i;
}

// Operands: 0 p, 1 g, 2 m, 3 v (inputs); 4 p', 5 m', 6 v' (outputs).
__global__ __launch_bounds__(kFB) void adam_fwd_tree_kernel(const SegEntry* __restrict__ seg,
                                                            const int64_t* __restrict__ tile_first, int64_t ngroups,
                                                            LeafArrays<7> arr, int dense_orig, AdamCoef c) {
  __shared__ int64_t s_goff[kWindowMax + 1];
  __shared__ int64_t s_numel[kWindowMax];
  __shared__ uint64_t s_ptr[7][kWindowMax];
  __shared__ int s_al[kWindowMax];
  const int64_t b = blockIdx.x;
  const int W = stage_window<7, kFB>(seg, tile_first, arr, dense_orig, b, s_goff, s_numel, s_ptr, s_al);
  __syncthreads();

  constexpr int kFU = (int)(kTileGroups / kFB);  // groups per lane
  f32x4 P[kFU], G[kFU], M[kFU], V[kFU];
  int leaf[kFU], kind[kFU];
  int64_t e0[kFU];
#pragma unroll
  for (int u = 0; u < kFU; ++u) {
    const int64_t gidx = b * kTileGroups + (int64_t)u * kFB + threadIdx.x;
    kind[u] = 0;
    leaf[u] = 0;
    e0[u] = 0;
    if (gidx < ngroups) {
      const int t = find_leaf(s_goff, W, gidx);
      leaf[u] = t;
      e0[u] = 4 * (gidx - s_goff[t]);
      const int64_t nel = s_numel[t];
      if (e0[u] < nel) {
        kind[u] = (e0[u] + 4 <= nel && s_al[t]) ? 1 : 2;
        if (kind[u] == 1) {
          const int64_t i = e0[u] >> 2;
          P[u] = ld(at<const f32x4>(s_ptr[0][t], i));
          G[u] = ld(at<const f32x4>(s_ptr[1][t], i));
          M[u] = ld(at<const f32x4>(s_ptr[2][t], i));
          V[u] = ld(at<const f32x4>(s_ptr[3][t], i));
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kFU; ++u) {
    const int t = leaf[u];
    if (kind[u] == 1) {
      f32x4 rp, rm, rv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const FwdOut o = fwd_elem(P[u][e], G[u][e], M[u][e], V[u][e], c);
        rp[e] = o.p;
        rm[e] = o.m;
        rv[e] = o.v;
      }
      const int64_t i = e0[u] >> 2;
      st(at<f32x4>(s_ptr[4][t], i), rp);
      st(at<f32x4>(s_ptr[5][t], i), rm);
      st(at<f32x4>(s_ptr[6][t], i), rv);
    } else if (kind[u] == 2) {
      const int64_t end = e0[u] + 4 < s_numel[t] ? e0[u] + 4 : s_numel[t];
      for (int64_t i = e0[u]; i < end; ++i) {
        const FwdOut o = fwd_elem(*at<const float>(s_ptr[0][t], i), *at<const float>(s_ptr[1][t], i),
                                  *at<const float>(s_ptr[2][t], i), *at<const float>(s_ptr[3][t], i), c);
        *at<float>(s_ptr[4][t], i) = o.p;
        *at<float>(s_ptr[5][t], i) = o.m;
        *at<float>(s_ptr[6][t], i) = o.v;
      }
    }
  }
}

// Operands: 0 dP, 1 dM, 2 dV (null unless HAS_MV), 3 g, 4 m, 5 v (inputs);
// 6 dg, 7 dm, 8 dv (outputs).
template <bool HAS_MV>
__global__ __launch_bounds__(kBB) void adam_bwd_tree_kernel(const SegEntry* __restrict__ seg,
                                                            const int64_t* __restrict__ tile_first, int64_t ngroups,
                                                            LeafArrays<9> arr, int dense_orig, AdamCoef c) {
  __shared__ int64_t s_goff[kWindowMax + 1];
  __shared__ int64_t s_numel[kWindowMax];
  __shared__ uint64_t s_ptr[9][kWindowMax];
  __shared__ int s_al[kWindowMax];
  const int64_t b = blockIdx.x;
  const int W = stage_window<9, kBB>(seg, tile_first, arr, dense_orig, b, s_goff, s_numel, s_ptr, s_al);
  __syncthreads();

  constexpr int kBU = (int)(kTileGroups / kBB);  // groups per lane
  f32x4 P[kBU], Mb[kBU], Vb[kBU], G[kBU], M[kBU], V[kBU];
  int leaf[kBU], kind[kBU];
  int64_t e0[kBU];
#pragma unroll
  for (int u = 0; u < kBU; ++u) {
    const int64_t gidx = b * kTileGroups + (int64_t)u * kBB + threadIdx.x;
    kind[u] = 0;
    leaf[u] = 0;
    e0[u] = 0;
    if (gidx < ngroups) {
      const int t = find_leaf(s_goff, W, gidx);
      leaf[u] = t;
      e0[u] = 4 * (gidx - s_goff[t]);
      const int64_t nel = s_numel[t];
      if (e0[u] < nel) {
        kind[u] = (e0[u] + 4 <= nel && s_al[t]) ? 1 : 2;
        if (kind[u] == 1) {
          const int64_t i = e0[u] >> 2;
          P[u] = ld(at<const f32x4>(s_ptr[0][t], i));
          if (HAS_MV) {
            Mb[u] = ld(at<const f32x4>(s_ptr[1][t], i));
            Vb[u] = ld(at<const f32x4>(s_ptr[2][t], i));
          }
          G[u] = ld(at<const f32x4>(s_ptr[3][t], i));
          M[u] = ld(at<const f32x4>(s_ptr[4][t], i));
          V[u] = ld(at<const f32x4>(s_ptr[5][t], i));
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kBU; ++u) {
    const int t = leaf[u];
    if (kind[u] == 1) {
      f32x4 rg, rm, rv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const BwdOut o = bwd_elem<HAS_MV>(P[u][e], HAS_MV ? Mb[u][e] : 0.0f, HAS_MV ? Vb[u][e] : 0.0f, G[u][e],
                                          M[u][e], V[u][e], c);
        rg[e] = o.g;
        rm[e] = o.m;
        rv[e] = o.v;
      }
      const int64_t i = e0[u] >> 2;
      st(at<f32x4>(s_ptr[6][t], i), rg);
      st(at<f32x4>(s_ptr[7][t], i), rm);
      st(at<f32x4>(s_ptr[8][t], i), rv);
    } else if (kind[u] == 2) {
      const int64_t end = e0[u] + 4 < s_numel[t] ? e0[u] + 4 : s_numel[t];
      for (int64_t i = e0[u]; i < end; ++i) {
        const BwdOut o = bwd_elem<HAS_MV>(
            *at<const float>(s_ptr[0][t], i), HAS_MV ? *at<const float>(s_ptr[1][t], i) : 0.0f,
            HAS_MV ? *at<const float>(s_ptr[2][t], i) : 0.0f, *at<const float>(s_ptr[3][t], i),
            *at<const float>(s_ptr[4][t], i), *at<const float>(s_ptr[5][t], i), c);
        *at<float>(s_ptr[6][t], i) = o.g;
        *at<float>(s_ptr[7][t], i) = o.m;
        *at<float>(s_ptr[8][t], i) = o.v;
      }
    }
  }
}

// ---- fused K-step leaf-direct kernels ----------------------------------------------
// The K-step driver in one launch per kTK steps, as the flat driver does it:
// each lane finds its group once, then walks the steps with the running params
// (forward) or dM, dV (backward) in registers, loading the next step's inputs
// before the current step's arithmetic.  The window stages the leaf address
// of every operand tree of every step in dynamic LDS (NA x kWindowMax x 8
// bytes: 18.5 KiB for the backward at 8 steps).  One group per lane, one
// table tile (512 groups) per workgroup.
constexpr int kTK = 8;  // steps per fused launch
constexpr int kUTB = (int)kTileGroups;
constexpr int kTFwdNA = 4 + 3 * kTK;  // 0 p, 1 mu0, 2 nu0, 3 pK; per step s: 4+3s g, 5+3s mu_s+1, 6+3s nu_s+1
constexpr int kTBwdNA = 3 + 4 * kTK;  // 0 dP, 1 dmu, 2 dnu; per step s: 3+4s g, 4+4s mu, 5+4s nu, 6+4s dg

struct TFwdArgs {
  const uint64_t* a[kTFwdNA];
  AdamCoef c[kTK];
  int32_t K;
};

// Execution order is reverse step order, as in the flat fused backward.
struct TBwdArgs {
  const uint64_t* a[kTBwdNA];
  AdamCoef c[kTK];
  int32_t K;
  int32_t init_mv;  // 0: dM = dV = 0 before the first step
};

// Stage the window of tile b for `na` operand trees: (operand, leaf) pairs
// are spread over the workgroup, then each leaf's all-operands-aligned flag
// is formed from LDS.  A NULL operand (a trajectory state the caller does
// not store) stages address 0 and is never dereferenced.  Ends with the
// workgroup synchronised.
template <int NT = kUTB>
__device__ __forceinline__ int stage_window_n(const SegEntry* __restrict__ seg, const int64_t* __restrict__ tile_first,
                                              const uint64_t* const* arrs, int na, int dense_orig, int64_t b,
                                              int64_t* s_goff, int64_t* s_numel, uint64_t* s_ptr, int* s_al) {
  const int64_t j0 = tile_first[b];
  const int W = (int)(tile_first[b + 1] - j0 + 1);
  for (int t = threadIdx.x; t <= W; t += NT) {
    const SegEntry e = seg[j0 + t];
    s_goff[t] = e.goff;
    if (t < W) s_numel[t] = e.numel;
  }
  for (int x = threadIdx.x; x < W * na; x += NT) {
    const int q = x / W, t = x - q * W;
    const int64_t leaf = dense_orig ? j0 + t : seg[j0 + t].orig;
    s_ptr[q * kWindowMax + t] = arrs[q] ? arrs[q][leaf] : 0;  // NULL operand: an unstored state
  }
  __syncthreads();
  for (int t = threadIdx.x; t < W; t += NT) {
    uint64_t any = 0;
    for (int q = 0; q < na; ++q) any |= s_ptr[q * kWindowMax + t];
    s_al[t] = (any & 15u) == 0;
  }
  __syncthreads();
  return W;
}

__global__ __launch_bounds__(kUTB) void adam_unrolled_fwd_tree_kernel(const SegEntry* __restrict__ seg,
                                                                     const int64_t* __restrict__ tile_first,
                                                                     int64_t ngroups, int dense_orig, TFwdArgs a) {
  __shared__ int64_t s_goff[kWindowMax + 1];
  __shared__ int64_t s_numel[kWindowMax];
  __shared__ int s_al[kWindowMax];
  extern __shared__ uint64_t s_ptr[];  // [na][kWindowMax]
  const int na = 4 + 3 * a.K;
  const int64_t b = blockIdx.x;
  const int W = stage_window_n(seg, tile_first, a.a, na, dense_orig, b, s_goff, s_numel, s_ptr, s_al);
  const int64_t gidx = b * kTileGroups + threadIdx.x;
  if (gidx >= ngroups) return;
  const int t = find_leaf(s_goff, W, gidx);
  const int64_t e0 = 4 * (gidx - s_goff[t]);
  const int64_t nel = s_numel[t];
  if (e0 >= nel) return;
  const uint64_t* P = s_ptr + t;  // P[q * kWindowMax]: leaf address in operand q
#define OP(q) P[(q) * kWindowMax]
  if (e0 + 4 <= nel && s_al[t]) {
    const int64_t i = e0 >> 2;
    f32x4 p = ld(at<const f32x4>(OP(0), i)), m = ld(at<const f32x4>(OP(1), i)), v = ld(at<const f32x4>(OP(2), i));
    f32x4 g = ld(at<const f32x4>(OP(4), i));
    for (int s = 0; s < a.K; ++s) {
      f32x4 gn = g;
      if (s + 1 < a.K) gn = ld(at<const f32x4>(OP(4 + 3 * (s + 1)), i));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const FwdOut o = fwd_elem(p[e], g[e], m[e], v[e], a.c[s]);
        p[e] = o.p;
        m[e] = o.m;
        v[e] = o.v;
      }
      if (a.a[5 + 3 * s]) {  // uniform: a stored state
        st(at<f32x4>(OP(5 + 3 * s), i), m);
        st(at<f32x4>(OP(6 + 3 * s), i), v);
      }
      g = gn;
    }
    st(at<f32x4>(OP(3), i), p);
  } else {
    const int64_t end = e0 + 4 < nel ? e0 + 4 : nel;
    for (int64_t i = e0; i < end; ++i) {
      float p = *at<const float>(OP(0), i), m = *at<const float>(OP(1), i), v = *at<const float>(OP(2), i);
      for (int s = 0; s < a.K; ++s) {
        const FwdOut o = fwd_elem(p, *at<const float>(OP(4 + 3 * s), i), m, v, a.c[s]);
        p = o.p;
        m = o.m;
        v = o.v;
        if (a.a[5 + 3 * s]) {
          *at<float>(OP(5 + 3 * s), i) = m;
          *at<float>(OP(6 + 3 * s), i) = v;
        }
      }
      *at<float>(OP(3), i) = p;
    }
  }
#undef OP
}

__global__ __launch_bounds__(kUTB) void adam_unrolled_bwd_tree_kernel(const SegEntry* __restrict__ seg,
                                                                     const int64_t* __restrict__ tile_first,
                                                                     int64_t ngroups, int dense_orig, TBwdArgs a) {
  __shared__ int64_t s_goff[kWindowMax + 1];
  __shared__ int64_t s_numel[kWindowMax];
  __shared__ int s_al[kWindowMax];
  extern __shared__ uint64_t s_ptr[];  // [na][kWindowMax]
  const int na = 3 + 4 * a.K;
  const int64_t b = blockIdx.x;
  const int W = stage_window_n(seg, tile_first, a.a, na, dense_orig, b, s_goff, s_numel, s_ptr, s_al);
  const int64_t gidx = b * kTileGroups + threadIdx.x;
  if (gidx >= ngroups) return;
  const int t = find_leaf(s_goff, W, gidx);
  const int64_t e0 = 4 * (gidx - s_goff[t]);
  const int64_t nel = s_numel[t];
  if (e0 >= nel) return;
  const uint64_t* P = s_ptr + t;
#define OP(q) P[(q) * kWindowMax]
  if (e0 + 4 <= nel && s_al[t]) {
    const int64_t i = e0 >> 2;
    const f32x4 dP = ld(at<const f32x4>(OP(0), i));
    f32x4 dM = {0.0f, 0.0f, 0.0f, 0.0f}, dV = {0.0f, 0.0f, 0.0f, 0.0f};
    f32x4 g = ld(at<const f32x4>(OP(3), i)), m = ld(at<const f32x4>(OP(4), i)), v = ld(at<const f32x4>(OP(5), i));
    if (a.init_mv) {
      dM = ld(at<const f32x4>(OP(1), i));
      dV = ld(at<const f32x4>(OP(2), i));
    }
    for (int s = 0; s < a.K; ++s) {
      f32x4 gn = g, mn = m, vn = v;
      if (s + 1 < a.K) {
        gn = ld(at<const f32x4>(OP(3 + 4 * (s + 1)), i));
        mn = ld(at<const f32x4>(OP(4 + 4 * (s + 1)), i));
        vn = ld(at<const f32x4>(OP(5 + 4 * (s + 1)), i));
      }
      f32x4 rg;
      if (s == 0 && !a.init_mv) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const BwdOut o = bwd_elem<false>(dP[e], 0.0f, 0.0f, g[e], m[e], v[e], a.c[s]);
          rg[e] = o.g;
          dM[e] = o.m;
          dV[e] = o.v;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const BwdOut o = bwd_elem<true>(dP[e], dM[e], dV[e], g[e], m[e], v[e], a.c[s]);
          rg[e] = o.g;
          dM[e] = o.m;
          dV[e] = o.v;
        }
      }
      st(at<f32x4>(OP(6 + 4 * s), i), rg);
      g = gn;
      m = mn;
      v = vn;
    }
    st(at<f32x4>(OP(1), i), dM);
    st(at<f32x4>(OP(2), i), dV);
  } else {
    const int64_t end = e0 + 4 < nel ? e0 + 4 : nel;
    for (int64_t i = e0; i < end; ++i) {
      const float dP = *at<const float>(OP(0), i);
      float dM = 0.0f, dV = 0.0f;
      if (a.init_mv) {
        dM = *at<const float>(OP(1), i);
        dV = *at<const float>(OP(2), i);
      }
      for (int s = 0; s < a.K; ++s) {
        const float g = *at<const float>(OP(3 + 4 * s), i), m = *at<const float>(OP(4 + 4 * s), i),
                    v = *at<const float>(OP(5 + 4 * s), i);
        const BwdOut o = (s == 0 && !a.init_mv) ? bwd_elem<false>(dP, 0.0f, 0.0f, g, m, v, a.c[s])
                                                : bwd_elem<true>(dP, dM, dV, g, m, v, a.c[s]);
        *at<float>(OP(6 + 4 * s), i) = o.g;
        dM = o.m;
        dV = o.v;
      }
      *at<float>(OP(1), i) = dM;
      *at<float>(OP(2), i) = dV;
    }
  }
#undef OP
}

// ---- fused VJP over a run of steps whose moments were not stored ----------------
// Leaf-direct form of the flat driver's recomputing VJP: for a run of C steps
// j+1..j+C with only (mu_j, nu_j) stored, each lane reads that state and the
// C gradients of its group once, recomputes the run's moments in registers
// with the forward's recurrences, then walks the C VJP steps last first.
constexpr int kTRS = kRematSpan;
constexpr int kTRBwdNA = 5 + 2 * kTRS;  // 0 dP, 1 dmu, 2 dnu, 3 mu_j, 4 nu_j; per step s: 5+2s g, 6+2s dg

// Step s of a run is unrolled step j+1+s (ascending).
struct TRBwdArgs {
  const uint64_t* a[kTRBwdNA];
  AdamCoef c[kTRS];
  int32_t init_mv;  // 0: the run holds the last unrolled step (zero dM, dV before it)
};

// Workgroups per table tile: each stages the tile's whole window and takes
// its share of the tile's groups, one per lane.  With its register count
// (78 VGPRs at C = 3) a CU holds two 512-thread workgroups but five of 256
// threads; measured on MI355X (K = 3, 20,000 leaves) the split of 2 runs at
// 5.46 TB/s against 5.27 unsplit (4: 5.50, within noise).
#ifndef DIFFOPT_TRBWD_SPLIT
#define DIFFOPT_TRBWD_SPLIT 2
#endif
constexpr int kTRSplit = DIFFOPT_TRBWD_SPLIT;
constexpr int kTRB = kUTB / kTRSplit;
static_assert(kUTB % kTRSplit == 0, "the split must divide the tile");

template <int C>
__global__ __launch_bounds__(kTRB) void adam_unrolled_bwd_tree_remat_kernel(const SegEntry* __restrict__ seg,
                                                                           const int64_t* __restrict__ tile_first,
                                                                           int64_t ngroups, int dense_orig,
                                                                           TRBwdArgs a) {
  __shared__ int64_t s_goff[kWindowMax + 1];
  __shared__ int64_t s_numel[kWindowMax];
  __shared__ int s_al[kWindowMax];
  extern __shared__ uint64_t s_ptr[];  // [na][kWindowMax]
  constexpr int na = 5 + 2 * C;
  const int64_t b = blockIdx.x / kTRSplit;  // table tile
  const int W = stage_window_n<kTRB>(seg, tile_first, a.a, na, dense_orig, b, s_goff, s_numel, s_ptr, s_al);
  const int64_t gidx = b * kTileGroups + (int64_t)(blockIdx.x % kTRSplit) * kTRB + threadIdx.x;
  if (gidx >= ngroups) return;
  const int t = find_leaf(s_goff, W, gidx);
  const int64_t e0 = 4 * (gidx - s_goff[t]);
  const int64_t nel = s_numel[t];
  if (e0 >= nel) return;
  const uint64_t* P = s_ptr + t;
#define OP(q) P[(q) * kWindowMax]
  if (e0 + 4 <= nel && s_al[t]) {
    const int64_t i = e0 >> 2;
    const f32x4 dP = ld(at<const f32x4>(OP(0), i));
    const f32x4 M0 = ld(at<const f32x4>(OP(3), i)), V0 = ld(at<const f32x4>(OP(4), i));
    f32x4 G[C];
#pragma unroll
    for (int s = 0; s < C; ++s) G[s] = ld(at<const f32x4>(OP(5 + 2 * s), i));
    f32x4 dM = {0.0f, 0.0f, 0.0f, 0.0f}, dV = {0.0f, 0.0f, 0.0f, 0.0f};
    if (a.init_mv) {
      dM = ld(at<const f32x4>(OP(1), i));
      dV = ld(at<const f32x4>(OP(2), i));
    }
#if !DIFFOPT_REMAT_QUAD_TREE
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
#endif
#pragma unroll
    for (int s = C - 1; s >= 0; --s) {
#if DIFFOPT_REMAT_QUAD_TREE
      f32x4 Ms, Vs;  // this step's input moments, recomputed from (M0, V0)
      run_moments<C>(s, M0, V0, G, a.c, Ms, Vs);
#else
      const f32x4 Ms = M[s], Vs = V[s];
#endif
      f32x4 rg;
      if (s == C - 1 && !a.init_mv) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const BwdOut o = bwd_elem<false>(dP[e], 0.0f, 0.0f, G[s][e], Ms[e], Vs[e], a.c[s]);
          rg[e] = o.g;
          dM[e] = o.m;
          dV[e] = o.v;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const BwdOut o = bwd_elem<true>(dP[e], dM[e], dV[e], G[s][e], Ms[e], Vs[e], a.c[s]);
          rg[e] = o.g;
          dM[e] = o.m;
          dV[e] = o.v;
        }
      }
      st(at<f32x4>(OP(6 + 2 * s), i), rg);
    }
    st(at<f32x4>(OP(1), i), dM);
    st(at<f32x4>(OP(2), i), dV);
  } else {
    const int64_t end = e0 + 4 < nel ? e0 + 4 : nel;
    for (int64_t i = e0; i < end; ++i) {
      const float dP = *at<const float>(OP(0), i);
      float G[C], M[C], V[C];
      M[0] = *at<const float>(OP(3), i);
      V[0] = *at<const float>(OP(4), i);
#pragma unroll
      for (int s = 0; s < C; ++s) G[s] = *at<const float>(OP(5 + 2 * s), i);
#pragma unroll
      for (int s = 0; s + 1 < C; ++s) {
        M[s + 1] = moment1(G[s], M[s], a.c[s]);
        V[s + 1] = moment2(G[s], V[s], a.c[s]);
      }
      float dM = 0.0f, dV = 0.0f;
      if (a.init_mv) {
        dM = *at<const float>(OP(1), i);
        dV = *at<const float>(OP(2), i);
      }
#pragma unroll
      for (int s = C - 1; s >= 0; --s) {
        const BwdOut o = (s == C - 1 && !a.init_mv) ? bwd_elem<false>(dP, 0.0f, 0.0f, G[s], M[s], V[s], a.c[s])
                                                    : bwd_elem<true>(dP, dM, dV, G[s], M[s], V[s], a.c[s]);
        *at<float>(OP(6 + 2 * s), i) = o.g;
        dM = o.m;
        dV = o.v;
      }
      *at<float>(OP(1), i) = dM;
      *at<float>(OP(2), i) = dV;
    }
  }
#undef OP
}

template <int C>
void launch_trbwd(const diffopt_segtable* t, const TRBwdArgs& a, hipStream_t st) {
  const size_t lds = sizeof(uint64_t) * kWindowMax * (5 + 2 * C);
  hipLaunchKernelGGL((adam_unrolled_bwd_tree_remat_kernel<C>), dim3((unsigned)(t->ntiles * kTRSplit)), dim3(kTRB),
                     lds, st, t->d_seg, t->d_tile_first, t->ngroups, t->dense_orig, a);
}

// Run length C is a template argument so the trajectory stays in registers.
int launch_trbwd_c(const char* who, int C, const diffopt_segtable* t, const TRBwdArgs& a, hipStream_t st) {
  switch (C) {
    case 1: launch_trbwd<1>(t, a, st); break;
    case 2: launch_trbwd<2>(t, a, st); break;
    case 3: launch_trbwd<3>(t, a, st); break;
    case 4: launch_trbwd<4>(t, a, st); break;
    case 5: launch_trbwd<5>(t, a, st); break;
    case 6: launch_trbwd<6>(t, a, st); break;
    case 7: launch_trbwd<7>(t, a, st); break;
    case 8: launch_trbwd<8>(t, a, st); break;
    default: return fail(DIFFOPT_EINVAL, "%s: recompute run of %d steps (at most %d)", who, C, kTRS);
  }
  return DIFFOPT_OK;
}
static_assert(kTRS == 8, "launch_trbwd_c instantiates run lengths 1..8");

// ---- small trees ------------------------------------------------------------------
// When the leaves fit a TinyTable the fused steps run one element per lane
// with the table in kernel arguments (no staged window, no barrier): a lane
// finds its leaf by a scan over the table, loads its leaf's address in every
// operand, then every input of every step, and only then computes.  The
// arithmetic per element is that of the kernels above, so the results are
// the same bit for bit.  Measured on MI355X for the 1,761-parameter tree at
// K = 5: about 7.4 and 8.2 us per fused forward and VJP launch through the
// staged window (each step a serial load and a four-element arithmetic chain
// per lane), which this form shortens to the latency of two dependent loads
// and one element's chain.
constexpr int kTinyB = 256;

// Leaf addresses as global-space pointers (see gptr): every load below is then
// a global_* instruction, counted by the vector-memory counter alone.
__device__ __forceinline__ gptr<const float> leaf_in(const uint64_t* arr, int orig) {
  return gaddr<const float>(arr[orig]);
}
__device__ __forceinline__ gptr<float> leaf_out(const uint64_t* arr, int orig) {
  return gaddr<float>(arr[orig]);
}

// The fused forward over K <= kTK steps (operands as in TFwdArgs, a.K == K).
// Every address and every input is loaded before the first step; an unstored
// step state takes the address of pK for its (unused) load slot, so no load
// waits behind a branch.
template <int K>
__global__ __launch_bounds__(kTinyB) void adam_unrolled_fwd_tree_tiny(TinyTable tt, TFwdArgs a) {
  warm_args(fold_lines(tt) ^ fold_lines(a));
  int leaf;
  int64_t i;
  if (!tiny_slot(tt, (int64_t)blockIdx.x * kTinyB + threadIdx.x, leaf, i)) return;
  const auto P0 = leaf_in(a.a[0], leaf);
  const auto M0 = leaf_in(a.a[1], leaf);
  const auto V0 = leaf_in(a.a[2], leaf);
  const auto PK = leaf_out(a.a[3], leaf);
  gptr<const float> Gp[K];
  gptr<float> Mo[K], Vo[K];
#pragma unroll
  for (int s = 0; s < K; ++s) {
    Gp[s] = leaf_in(a.a[4 + 3 * s], leaf);
    const bool kept = a.a[5 + 3 * s] != nullptr;  // uniform: a stored state
    Mo[s] = leaf_out(kept ? a.a[5 + 3 * s] : a.a[3], leaf);
    Vo[s] = leaf_out(kept ? a.a[6 + 3 * s] : a.a[3], leaf);
  }
  float p = P0[i], m = M0[i], v = V0[i];
  float G[K];
#pragma unroll
  for (int s = 0; s < K; ++s) G[s] = Gp[s][i];
#pragma unroll
  for (int s = 0; s < K; ++s) {
    const FwdOut o = fwd_elem(p, G[s], m, v, a.c[s]);
    p = o.p;
    m = o.m;
    v = o.v;
    if (a.a[5 + 3 * s]) {
      Mo[s][i] = m;
      Vo[s][i] = v;
    }
  }
  PK[i] = p;
}

// The VJP over a run of C steps from one stored state (mu_j, nu_j), last step
// first, as adam_unrolled_bwd_tree_remat_kernel; the incoming and outgoing
// moment cotangents have their own operands so that the single-step VJP (C =
// 1, separate input and output trees) takes the same kernel.
constexpr int kTinyBwdNA = 7 + 2 * kTRS;  // 0 dP, 1 dM in, 2 dV in, 3 dM out, 4 dV out, 5 mu_j, 6 nu_j;
                                          // per step s: 7+2s g, 8+2s dg
struct TinyBwdArgs {
  const uint64_t* a[kTinyBwdNA];
  AdamCoef c[kTRS];
  int32_t init_mv;  // 0: zero dM, dV before the run's last step (operands 1, 2 unused)
};

template <int C>
__global__ __launch_bounds__(kTinyB) void adam_unrolled_bwd_tree_tiny(TinyTable tt, TinyBwdArgs a) {
  warm_args(fold_lines(tt) ^ fold_lines(a));
  int leaf;
  int64_t i;
  if (!tiny_slot(tt, (int64_t)blockIdx.x * kTinyB + threadIdx.x, leaf, i)) return;
  // without incoming moment cotangents their load slots read dP (unused)
  const auto DP = leaf_in(a.a[0], leaf);
  const auto DMi = leaf_in(a.init_mv ? a.a[1] : a.a[0], leaf);
  const auto DVi = leaf_in(a.init_mv ? a.a[2] : a.a[0], leaf);
  const auto DMo = leaf_out(a.a[3], leaf);
  const auto DVo = leaf_out(a.a[4], leaf);
  const auto Mj = leaf_in(a.a[5], leaf);
  const auto Vj = leaf_in(a.a[6], leaf);
  gptr<const float> Gp[C];
  gptr<float> DG[C];
#pragma unroll
  for (int s = 0; s < C; ++s) {
    Gp[s] = leaf_in(a.a[7 + 2 * s], leaf);
    DG[s] = leaf_out(a.a[8 + 2 * s], leaf);
  }
  const float dP = DP[i];
  const float dMi = DMi[i], dVi = DVi[i];
  float G[C], M[C], V[C];
  M[0] = Mj[i];
  V[0] = Vj[i];
#pragma unroll
  for (int s = 0; s < C; ++s) G[s] = Gp[s][i];
  float dM = a.init_mv ? dMi : 0.0f, dV = a.init_mv ? dVi : 0.0f;
#pragma unroll
  for (int s = 0; s + 1 < C; ++s) {
    M[s + 1] = moment1(G[s], M[s], a.c[s]);
    V[s + 1] = moment2(G[s], V[s], a.c[s]);
  }
#pragma unroll
  for (int s = C - 1; s >= 0; --s) {
    const BwdOut o = (s == C - 1 && !a.init_mv) ? bwd_elem<false>(dP, 0.0f, 0.0f, G[s], M[s], V[s], a.c[s])
                                                : bwd_elem<true>(dP, dM, dV, G[s], M[s], V[s], a.c[s]);
    DG[s][i] = o.g;
    dM = o.m;
    dV = o.v;
  }
  DMo[i] = dM;
  DVo[i] = dV;
}

unsigned tiny_blocks(const diffopt_segtable* t) { return (unsigned)((t->small.total + kTinyB - 1) / kTinyB); }

template <int K>
void launch_tiny_fwd(const diffopt_segtable* t, const TFwdArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((adam_unrolled_fwd_tree_tiny<K>), dim3(tiny_blocks(t)), dim3(kTinyB), 0, st, t->small, a);
}

void launch_tiny_fwd_k(const diffopt_segtable* t, const TFwdArgs& a, hipStream_t st) {
  switch (a.K) {  // 1 <= a.K <= kTK
    case 1: launch_tiny_fwd<1>(t, a, st); break;
    case 2: launch_tiny_fwd<2>(t, a, st); break;
    case 3: launch_tiny_fwd<3>(t, a, st); break;
    case 4: launch_tiny_fwd<4>(t, a, st); break;
    case 5: launch_tiny_fwd<5>(t, a, st); break;
    case 6: launch_tiny_fwd<6>(t, a, st); break;
    case 7: launch_tiny_fwd<7>(t, a, st); break;
    default: launch_tiny_fwd<8>(t, a, st); break;
  }
}
static_assert(kTK == 8, "launch_tiny_fwd_k instantiates 1..8 steps");

template <int C>
void launch_tiny_bwd(const diffopt_segtable* t, const TinyBwdArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((adam_unrolled_bwd_tree_tiny<C>), dim3(tiny_blocks(t)), dim3(kTinyB), 0, st, t->small, a);
}

int launch_tiny_bwd_c(const char* who, int C, const diffopt_segtable* t, const TinyBwdArgs& a, hipStream_t st) {
  switch (C) {
    case 1: launch_tiny_bwd<1>(t, a, st); break;
    case 2: launch_tiny_bwd<2>(t, a, st); break;
    case 3: launch_tiny_bwd<3>(t, a, st); break;
    case 4: launch_tiny_bwd<4>(t, a, st); break;
    case 5: launch_tiny_bwd<5>(t, a, st); break;
    case 6: launch_tiny_bwd<6>(t, a, st); break;
    case 7: launch_tiny_bwd<7>(t, a, st); break;
    case 8: launch_tiny_bwd<8>(t, a, st); break;
    default: return fail(DIFFOPT_EINVAL, "%s: recompute run of %d steps (at most %d)", who, C, kTRS);
  }
  return DIFFOPT_OK;
}

// ---- leaf-direct SGD-momentum and RMSProp ------------------------------------------
// The ops of optim_ops.hpp applied leaf by leaf, in the layout of the fused
// Adam kernels: one table tile per workgroup, one group per lane, the leaf
// address of every operand staged in the window.  Operands: the op's inputs,
// then its outputs.
template <class Op>
__global__ __launch_bounds__(kUTB) void ew_tree_kernel(const SegEntry* __restrict__ seg,
                                                      const int64_t* __restrict__ tile_first, int64_t ngroups,
                                                      int dense_orig, LeafArrays<Op::NIN + Op::NOUT> arr, Op op) {
  constexpr int NA = Op::NIN + Op::NOUT;
  __shared__ int64_t s_goff[kWindowMax + 1];
  __shared__ int64_t s_numel[kWindowMax];
  __shared__ int s_al[kWindowMax];
  __shared__ uint64_t s_ptr[NA * kWindowMax];
  const int64_t b = blockIdx.x;
  const int W = stage_window_n(seg, tile_first, arr.a, NA, dense_orig, b, s_goff, s_numel, s_ptr, s_al);
  const int64_t gidx = b * kTileGroups + threadIdx.x;
  if (gidx >= ngroups) return;
  const int t = find_leaf(s_goff, W, gidx);
  const int64_t e0 = 4 * (gidx - s_goff[t]);
  const int64_t nel = s_numel[t];
  if (e0 >= nel) return;
  const uint64_t* P = s_ptr + t;
  float xi[Op::NIN], yo[Op::NOUT];
  if (e0 + 4 <= nel && s_al[t]) {
    const int64_t i = e0 >> 2;
    f32x4 x[Op::NIN], y[Op::NOUT];
#pragma unroll
    for (int a = 0; a < Op::NIN; ++a) x[a] = ld(at<const f32x4>(P[a * kWindowMax], i));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
#pragma unroll
      for (int a = 0; a < Op::NIN; ++a) xi[a] = x[a][e];
      op.apply(xi, yo);
#pragma unroll
      for (int q = 0; q < Op::NOUT; ++q) y[q][e] = yo[q];
    }
#pragma unroll
    for (int q = 0; q < Op::NOUT; ++q) st(at<f32x4>(P[(Op::NIN + q) * kWindowMax], i), y[q]);
  } else {
    const int64_t end = e0 + 4 < nel ? e0 + 4 : nel;
    for (int64_t i = e0; i < end; ++i) {
#pragma unroll
      for (int a = 0; a < Op::NIN; ++a) xi[a] = *at<const float>(P[a * kWindowMax], i);
      op.apply(xi, yo);
#pragma unroll
      for (int q = 0; q < Op::NOUT; ++q) *at<float>(P[(Op::NIN + q) * kWindowMax], i) = yo[q];
    }
  }
}

// Small trees (a TinyTable): one element per lane, the table in the kernel
// arguments, every leaf address then every input loaded before the op, as in
// the small-tree Adam kernels; the same op.apply per element.
template <class Op>
__global__ __launch_bounds__(kTinyB) void ew_tree_tiny(TinyTable tt, LeafArrays<Op::NIN + Op::NOUT> arr, Op op) {
  warm_args(fold_lines(tt) ^ fold_lines(arr) ^ fold_lines(op));
  int leaf;
  int64_t i;
  if (!tiny_slot(tt, (int64_t)blockIdx.x * kTinyB + threadIdx.x, leaf, i)) return;
  gptr<const float> in[Op::NIN];
  gptr<float> out[Op::NOUT];
#pragma unroll
  for (int a = 0; a < Op::NIN; ++a) in[a] = leaf_in(arr.a[a], leaf);
#pragma unroll
  for (int q = 0; q < Op::NOUT; ++q) out[q] = leaf_out(arr.a[Op::NIN + q], leaf);
  float xi[Op::NIN], yo[Op::NOUT];
#pragma unroll
  for (int a = 0; a < Op::NIN; ++a) xi[a] = in[a][i];
  op.apply(xi, yo);
#pragma unroll
  for (int q = 0; q < Op::NOUT; ++q) out[q][i] = yo[q];
}

// Runner of the leaf-direct kernel for the *_variant selectors: every
// operand is a device array of leaf addresses.
struct TreeRun {
  const char* who;
  const diffopt_segtable* t;
  hipStream_t st;
  template <class Op>
  int go(const Op& op, const void* const* in, const void* const* out) {
    LeafArrays<Op::NIN + Op::NOUT> arr{};
    for (int a = 0; a < Op::NIN; ++a) arr.a[a] = static_cast<const uint64_t*>(in[a]);
    for (int q = 0; q < Op::NOUT; ++q) arr.a[Op::NIN + q] = static_cast<const uint64_t*>(out[q]);
    if (t->tiny)
      hipLaunchKernelGGL((ew_tree_tiny<Op>), dim3(tiny_blocks(t)), dim3(kTinyB), 0, st, t->small, arr, op);
    else
      hipLaunchKernelGGL((ew_tree_kernel<Op>), dim3((unsigned)t->ntiles), dim3(kUTB), 0, st, t->d_seg,
                         t->d_tile_first, t->ngroups, t->dense_orig, arr, op);
    return launch_status(who);
  }
};

int check_table(const char* who, const diffopt_segtable* t) {
  if (!t) return fail(DIFFOPT_EINVAL, "%s: table is NULL", who);
  if (t->elem_bytes != 4) return fail(DIFFOPT_EINVAL, "%s: the table must describe fp32 leaves (elem_bytes 4)", who);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != t->device)
    return fail(DIFFOPT_EINVAL, "%s: the table lives on device %d, the current device is %d", who, t->device, dev);
  return DIFFOPT_OK;
}

int launch_fwd_tree(const diffopt_segtable* t, const LeafArrays<7>& arr, const AdamCoef& c, hipStream_t st) {
  if (t->ntiles == 0) return DIFFOPT_OK;
  hipLaunchKernelGGL(adam_fwd_tree_kernel, dim3((unsigned)t->ntiles), dim3(kFB), 0, st, t->d_seg, t->d_tile_first,
                     t->ngroups, arr, t->dense_orig, c);
  return launch_status("diffopt_adam_fwd_tree");
}

// Workgroups of the leaf-direct VJP resident per CU.  Its registers allow
// seven; with six reads and three writes per element that many oversubscribe
// the memory system, and five ran the 20,000-leaf tree's VJP 4% faster (four:
// the same; six: no gain).  The launch reserves otherwise unused dynamic LDS
// so that no more than kBwdTreeResident workgroups fit in a CU's 160 KiB.
constexpr int kBwdTreeResident = 5;
constexpr size_t kLdsPerCU = 160 * 1024;
constexpr size_t kBwdTreeStaticLds = (kWindowMax + 1) * 8 + kWindowMax * (8 + 9 * 8 + 4);
constexpr size_t kBwdTreeLdsPad = kLdsPerCU / kBwdTreeResident - kBwdTreeStaticLds - 256;
static_assert(kLdsPerCU / (kBwdTreeStaticLds + kBwdTreeLdsPad) == kBwdTreeResident,
              "the reserved LDS must leave room for exactly kBwdTreeResident workgroups");

int launch_bwd_tree(const diffopt_segtable* t, const LeafArrays<9>& arr, const AdamCoef& c, hipStream_t st) {
  if (t->ntiles == 0) return DIFFOPT_OK;
  if (arr.a[1])
    hipLaunchKernelGGL((adam_bwd_tree_kernel<true>), dim3((unsigned)t->ntiles), dim3(kBB), kBwdTreeLdsPad, st,
                       t->d_seg, t->d_tile_first, t->ngroups, arr, t->dense_orig, c);
  else
    hipLaunchKernelGGL((adam_bwd_tree_kernel<false>), dim3((unsigned)t->ntiles), dim3(kBB), kBwdTreeLdsPad, st,
                       t->d_seg, t->d_tile_first, t->ngroups, arr, t->dense_orig, c);
  return launch_status("diffopt_adam_bwd_tree");
}

}  // namespace
}  // namespace diffopt

using namespace diffopt;

extern "C" int diffopt_adam_fwd_tree(const diffopt_segtable* table, const uint64_t* params, const uint64_t* grad,
                                     const uint64_t* mu, const uint64_t* nu, int64_t count, double lr, double b1,
                                     double b2, double eps, double eps_root, const uint64_t* params_out,
                                     const uint64_t* mu_out, const uint64_t* nu_out, void* stream) {
  clear_error();
  static const char* who = "diffopt_adam_fwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  AdamCoef c;
  rc = make_coef(who, count, lr, b1, b2, eps, eps_root, &c);
  if (rc) return rc;
  if (table->ntiles == 0) return DIFFOPT_OK;
  if (!params || !grad || !mu || !nu || !params_out || !mu_out || !nu_out)
    return fail(DIFFOPT_EINVAL, "%s: null leaf-address array", who);
  if (table->tiny) {  // the fused forward at K = 1, its step state stored in the outputs
    TFwdArgs a{};
    a.K = 1;
    a.a[0] = params;
    a.a[1] = mu;
    a.a[2] = nu;
    a.a[3] = params_out;
    a.a[4] = grad;
    a.a[5] = mu_out;
    a.a[6] = nu_out;
    a.c[0] = c;
    launch_tiny_fwd<1>(table, a, as_stream(stream));
    return launch_status(who);
  }
  const LeafArrays<7> arr{{params, grad, mu, nu, params_out, mu_out, nu_out}};
  return launch_fwd_tree(table, arr, c, as_stream(stream));
}

extern "C" int diffopt_adam_bwd_tree(const diffopt_segtable* table, const uint64_t* dupdate, const uint64_t* dmu,
                                     const uint64_t* dnu, const uint64_t* grad, const uint64_t* mu,
                                     const uint64_t* nu, int64_t count, double lr, double b1, double b2, double eps,
                                     double eps_root, const uint64_t* dgrad, const uint64_t* dmu_in,
                                     const uint64_t* dnu_in, void* stream) {
  clear_error();
  static const char* who = "diffopt_adam_bwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  AdamCoef c;
  rc = make_coef(who, count, lr, b1, b2, eps, eps_root, &c);
  if (rc) return rc;
  if ((dmu == nullptr) != (dnu == nullptr))
    return fail(DIFFOPT_EINVAL, "%s: dmu and dnu must both be given or both be NULL", who);
  if (table->ntiles == 0) return DIFFOPT_OK;
  if (!dupdate || !grad || !mu || !nu || !dgrad || !dmu_in || !dnu_in)
    return fail(DIFFOPT_EINVAL, "%s: null leaf-address array", who);
  if (table->tiny) {  // the recomputing VJP over one step from the stored (mu, nu)
    TinyBwdArgs a{};
    a.init_mv = dmu != nullptr;
    a.a[0] = dupdate;
    a.a[1] = dmu;
    a.a[2] = dnu;
    a.a[3] = dmu_in;
    a.a[4] = dnu_in;
    a.a[5] = mu;
    a.a[6] = nu;
    a.a[7] = grad;
    a.a[8] = dgrad;
    a.c[0] = c;
    launch_tiny_bwd<1>(table, a, as_stream(stream));
    return launch_status(who);
  }
  const LeafArrays<9> arr{{dupdate, dmu, dnu, grad, mu, nu, dgrad, dmu_in, dnu_in}};
  return launch_bwd_tree(table, arr, c, as_stream(stream));
}

extern "C" int diffopt_adam_unrolled_fwd_tree(const diffopt_segtable* table, int64_t K, const uint64_t* p0,
                                              const uint64_t* const* grads, const uint64_t* const* mu_traj,
                                              const uint64_t* const* nu_traj, const uint64_t* pK, int64_t count0,
                                              double lr, double b1, double b2, double eps, double eps_root,
                                              void* stream) {
  clear_error();
  static const char* who = "diffopt_adam_unrolled_fwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  if (K < 1) return fail(DIFFOPT_EINVAL, "%s: K must be >= 1 (got %lld)", who, (long long)K);
  if (!grads || !mu_traj || !nu_traj) return fail(DIFFOPT_EINVAL, "%s: null pointer array", who);
  AdamCoef c;
  for (int64_t k = 1; k <= K; ++k) {
    rc = make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &c);
    if (rc) return rc;
  }
  if (table->ntiles == 0) return DIFFOPT_OK;
  if (!p0 || !pK) return fail(DIFFOPT_EINVAL, "%s: null p0 or pK", who);
  for (int64_t k = 0; k < K; ++k)
    if (!grads[k]) return fail(DIFFOPT_EINVAL, "%s: null grads entry %lld", who, (long long)k);
  rc = check_trajectory(who, K, mu_traj, nu_traj, true, false);
  if (rc) return rc;
  hipStream_t st = as_stream(stream);
  for (int64_t k0 = 0; k0 < K; k0 += kTK) {  // one fused launch per kTK steps
    TFwdArgs a{};
    a.K = (int32_t)(K - k0 < kTK ? K - k0 : kTK);
    // between launches the running moments pass through the state stored at
    // the boundary, or through the final-state trees when it is not stored
    a.a[0] = (k0 == 0) ? p0 : pK;
    a.a[1] = mu_traj[k0] ? mu_traj[k0] : mu_traj[K];
    a.a[2] = nu_traj[k0] ? nu_traj[k0] : nu_traj[K];
    a.a[3] = pK;
    for (int s = 0; s < a.K; ++s) {
      a.a[4 + 3 * s] = grads[k0 + s];
      a.a[5 + 3 * s] = mu_traj[k0 + s + 1];
      a.a[6 + 3 * s] = nu_traj[k0 + s + 1];
      make_coef(who, count0 + k0 + s, lr, b1, b2, eps, eps_root, &a.c[s]);
    }
    if (!a.a[5 + 3 * (a.K - 1)]) {
      a.a[5 + 3 * (a.K - 1)] = mu_traj[K];
      a.a[6 + 3 * (a.K - 1)] = nu_traj[K];
    }
    if (table->tiny) {
      launch_tiny_fwd_k(table, a, st);
    } else {
      const size_t lds = sizeof(uint64_t) * kWindowMax * (4 + 3 * a.K);
      hipLaunchKernelGGL(adam_unrolled_fwd_tree_kernel, dim3((unsigned)table->ntiles), dim3(kUTB), lds, st,
                         table->d_seg, table->d_tile_first, table->ngroups, table->dense_orig, a);
    }
    rc = launch_status(who);
    if (rc) return rc;
  }
  return DIFFOPT_OK;
}

extern "C" int diffopt_adam_unrolled_bwd_tree(const diffopt_segtable* table, int64_t K, const uint64_t* dpK,
                                              const uint64_t* const* grads, const uint64_t* const* mu_traj,
                                              const uint64_t* const* nu_traj, const uint64_t* const* dgrads,
                                              const uint64_t* dmu0, const uint64_t* dnu0, int64_t count0, double lr,
                                              double b1, double b2, double eps, double eps_root, void* stream) {
  clear_error();
  static const char* who = "diffopt_adam_unrolled_bwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  if (K < 1) return fail(DIFFOPT_EINVAL, "%s: K must be >= 1 (got %lld)", who, (long long)K);
  if (!grads || !mu_traj || !nu_traj || !dgrads) return fail(DIFFOPT_EINVAL, "%s: null pointer array", who);
  AdamCoef c;
  for (int64_t k = 1; k <= K; ++k) {
    rc = make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &c);
    if (rc) return rc;
  }
  if (table->ntiles == 0) return DIFFOPT_OK;
  if (!dpK || !dmu0 || !dnu0) return fail(DIFFOPT_EINVAL, "%s: null dpK, dmu0 or dnu0", who);
  if (dmu0 == dnu0) return fail(DIFFOPT_EINVAL, "%s: dmu0 and dnu0 must be distinct", who);
  for (int64_t k = 0; k < K; ++k)
    if (!grads[k] || !dgrads[k])
      return fail(DIFFOPT_EINVAL, "%s: null entry %lld in grads or dgrads", who, (long long)k);
  rc = check_trajectory(who, K, mu_traj, nu_traj, false, true);
  if (rc) return rc;
  hipStream_t st = as_stream(stream);
  // Last steps first: runs of steps whose input states are stored take one
  // launch per kTK steps; a run j+1..khi after one stored state j takes one
  // launch that recomputes the states it needs.
  for (int64_t khi = K; khi >= 1;) {
    const int32_t init_mv = khi != K;  // the first launch starts from zero cotangents of mu_K, nu_K
    if (mu_traj[khi - 1]) {
      int32_t run = 0;
      while (run < kTK && khi - run >= 1 && mu_traj[khi - run - 1]) ++run;
      if (table->tiny && run == 1) {  // one step from its stored state: the small form at C = 1
        TinyBwdArgs a{};
        a.init_mv = init_mv;
        a.a[0] = dpK;
        a.a[1] = dmu0;
        a.a[2] = dnu0;
        a.a[3] = dmu0;
        a.a[4] = dnu0;
        a.a[5] = mu_traj[khi - 1];
        a.a[6] = nu_traj[khi - 1];
        a.a[7] = grads[khi - 1];
        a.a[8] = dgrads[khi - 1];
        make_coef(who, count0 + khi - 1, lr, b1, b2, eps, eps_root, &a.c[0]);
        launch_tiny_bwd<1>(table, a, st);
        khi -= 1;
        rc = launch_status(who);
        if (rc) return rc;
        continue;
      }
      TBwdArgs a{};
      a.K = run;
      a.init_mv = init_mv;
      a.a[0] = dpK;
      a.a[1] = dmu0;
      a.a[2] = dnu0;
      for (int s = 0; s < a.K; ++s) {
        const int64_t k = khi - s;  // unrolled step (1-based) run as the launch's step s
        a.a[3 + 4 * s] = grads[k - 1];
        a.a[4 + 4 * s] = mu_traj[k - 1];
        a.a[5 + 4 * s] = nu_traj[k - 1];
        a.a[6 + 4 * s] = dgrads[k - 1];
        make_coef(who, count0 + k - 1, lr, b1, b2, eps, eps_root, &a.c[s]);
      }
      const size_t lds = sizeof(uint64_t) * kWindowMax * (3 + 4 * a.K);
      hipLaunchKernelGGL(adam_unrolled_bwd_tree_kernel, dim3((unsigned)table->ntiles), dim3(kUTB), lds, st,
                         table->d_seg, table->d_tile_first, table->ngroups, table->dense_orig, a);
      khi -= run;
    } else {
      int64_t j = khi - 1;
      while (!mu_traj[j]) --j;  // mu_traj[0] is stored; check_trajectory bounds khi - j by kTRS
      const int C = (int)(khi - j);
      if (table->tiny) {
        TinyBwdArgs a{};
        a.init_mv = init_mv;
        a.a[0] = dpK;
        a.a[1] = dmu0;
        a.a[2] = dnu0;
        a.a[3] = dmu0;
        a.a[4] = dnu0;
        a.a[5] = mu_traj[j];
        a.a[6] = nu_traj[j];
        for (int s = 0; s < C; ++s) {
          a.a[7 + 2 * s] = grads[j + s];
          a.a[8 + 2 * s] = dgrads[j + s];
          make_coef(who, count0 + j + s, lr, b1, b2, eps, eps_root, &a.c[s]);
        }
        rc = launch_tiny_bwd_c(who, C, table, a, st);
        if (rc) return rc;
        khi = j;
        rc = launch_status(who);
        if (rc) return rc;
        continue;
      }
      TRBwdArgs a{};
      a.init_mv = init_mv;
      a.a[0] = dpK;
      a.a[1] = dmu0;
      a.a[2] = dnu0;
      a.a[3] = mu_traj[j];
      a.a[4] = nu_traj[j];
      for (int s = 0; s < C; ++s) {
        a.a[5 + 2 * s] = grads[j + s];
        a.a[6 + 2 * s] = dgrads[j + s];
        make_coef(who, count0 + j + s, lr, b1, b2, eps, eps_root, &a.c[s]);
      }
      rc = launch_trbwd_c(who, C, table, a, st);
      if (rc) return rc;
      khi = j;
    }
    rc = launch_status(who);
    if (rc) return rc;
  }
  return DIFFOPT_OK;
}

// ---- leaf-direct SGD-momentum and RMSProp entry points ---------------------------------

static int check_sgd_hyper(const char* who, double lr, double momentum) {
  if (!std::isfinite(lr)) return fail(DIFFOPT_EINVAL, "%s: lr must be finite", who);
  if (!(momentum >= 0.0 && std::isfinite(momentum)))
    return fail(DIFFOPT_EINVAL, "%s: momentum must be finite and >= 0", who);
  return DIFFOPT_OK;
}

extern "C" int diffopt_sgd_fwd_tree(const diffopt_segtable* table, const uint64_t* params, const uint64_t* grad,
                                    const uint64_t* trace, double lr, double momentum, int32_t nesterov,
                                    const uint64_t* params_out, const uint64_t* trace_out, void* stream) {
  clear_error();
  static const char* who = "diffopt_sgd_fwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  rc = check_sgd_hyper(who, lr, momentum);
  if (rc) return rc;
  if (table->ntiles == 0) return DIFFOPT_OK;
  const bool mom = momentum > 0.0;
  if (!params || !grad || !params_out || (mom && !trace_out))
    return fail(DIFFOPT_EINVAL, "%s: null leaf-address array", who);
  TreeRun run{who, table, as_stream(stream)};
  return sgd_fwd_variant(run, params, grad, mom ? trace : nullptr, params_out, mom ? trace_out : nullptr, lr,
                         momentum, nesterov != 0);
}

extern "C" int diffopt_sgd_bwd_tree(const diffopt_segtable* table, const uint64_t* dparams_out,
                                    const uint64_t* dtrace_out, double lr, double momentum, int32_t nesterov,
                                    const uint64_t* dgrad, const uint64_t* dtrace_in, void* stream) {
  clear_error();
  static const char* who = "diffopt_sgd_bwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  rc = check_sgd_hyper(who, lr, momentum);
  if (rc) return rc;
  if (table->ntiles == 0) return DIFFOPT_OK;
  const bool mom = momentum > 0.0;
  if (!dparams_out || !dgrad || (mom && !dtrace_in)) return fail(DIFFOPT_EINVAL, "%s: null leaf-address array", who);
  TreeRun run{who, table, as_stream(stream)};
  return sgd_bwd_variant(run, dparams_out, mom ? dtrace_out : nullptr, dgrad, mom ? dtrace_in : nullptr, lr,
                         momentum, nesterov != 0);
}

extern "C" int diffopt_rmsprop_fwd_tree(const diffopt_segtable* table, const uint64_t* params, const uint64_t* grad,
                                        const uint64_t* nu, const uint64_t* mom, double lr, double alpha, double eps,
                                        double eps_root, double momentum, const uint64_t* params_out,
                                        const uint64_t* nu_out, const uint64_t* mom_out, void* stream) {
  clear_error();
  static const char* who = "diffopt_rmsprop_fwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  RmsCoef c;
  rc = rms_coef(who, lr, alpha, eps, eps_root, momentum, &c);
  if (rc) return rc;
  if (table->ntiles == 0) return DIFFOPT_OK;
  const bool m = momentum > 0.0;
  if (!params || !grad || !nu || !params_out || !nu_out || (m && !mom_out))
    return fail(DIFFOPT_EINVAL, "%s: null leaf-address array", who);
  TreeRun run{who, table, as_stream(stream)};
  return rms_fwd_variant(run, params, grad, nu, m ? mom : nullptr, params_out, nu_out, m ? mom_out : nullptr, c, m);
}

extern "C" int diffopt_rmsprop_bwd_tree(const diffopt_segtable* table, const uint64_t* dparams_out,
                                        const uint64_t* dnu_out, const uint64_t* dmom_out, const uint64_t* grad,
                                        const uint64_t* nu, double lr, double alpha, double eps, double eps_root,
                                        double momentum, const uint64_t* dgrad, const uint64_t* dnu_in,
                                        const uint64_t* dmom_in, void* stream) {
  clear_error();
  static const char* who = "diffopt_rmsprop_bwd_tree";
  int rc = check_table(who, table);
  if (rc) return rc;
  RmsCoef c;
  rc = rms_coef(who, lr, alpha, eps, eps_root, momentum, &c);
  if (rc) return rc;
  if (table->ntiles == 0) return DIFFOPT_OK;
  const bool m = momentum > 0.0;
  if (!dparams_out || !grad || !nu || !dgrad || !dnu_in || (m && !dmom_in))
    return fail(DIFFOPT_EINVAL, "%s: null leaf-address array", who);
  TreeRun run{who, table, as_stream(stream)};
  return rms_bwd_variant(run, dparams_out, dnu_out, m ? dmom_out : nullptr, grad, nu, dgrad, dnu_in,
                         m ? dmom_in : nullptr, c, m);
}
