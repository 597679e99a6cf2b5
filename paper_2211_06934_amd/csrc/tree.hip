// Tree flatten / unflatten through a segment table on gfx950 (TorchOpt,
// Sec. 2.3 "Memory-efficient and cache-friendly PyTree"; Appendix D, Table 2).
//
// Work decomposition.  Every copy writes whole, naturally aligned 16-byte
// vectors of its DESTINATION (the flat buffer for flatten, the leaves for
// unflatten).  Nonempty leaf j owns G_j = ceil(bytes_j / 16) + 8 consecutive
// "groups" of a global group index space, rounded up to a multiple of 8; group
// k of leaf j is the aligned 16-byte destination vector number k counted from
// the 128-byte line that holds the leaf's first destination byte.  The +8
// covers any phase within that line, so the G_j groups always cover the leaf;
// a group may be partial (head, tail) or empty.  Leaves start on multiples of
// 8 groups and tiles hold multiples of 8 groups, so every tile boundary falls
// on a line boundary of the destination, for pack (the flat buffer, whatever
// the leaves' offsets) as for unpack: no line is written in parts by two
// tiles.
// Each lane owns one group per step: full groups take one aligned 128-bit
// store, fed by one or two aligned 128-bit source vectors and a funnel shift
// when source and destination phases differ (dense offsets put ~3/4 of leaves
// out of phase with their flat range); partial groups copy element by
// element.  Consecutive lanes own consecutive groups, so within a leaf the
// second source vector of one lane is the first of the next lane, which hands
// it over through a cross-lane read instead of a second load.  Every byte is
// copied through integer registers, so NaN payloads, signed zeros and
// subnormals survive.
//
// Segment lookup.  Block b handles groups [b*TG, (b+1)*TG).  The host
// precomputes tile_first[b], the leaf holding group b*TG; the leaves a tile
// touches are the window tile_first[b] .. tile_first[b+1].  A window of one
// leaf is read straight into scalar registers.  Otherwise the block stages
// the window (group offsets, flat offsets, byte sizes, leaf addresses) in LDS
// once, then every lane binary-searches the LDS window for its group.  Since
// every nonempty leaf owns >= 8 groups, a window never exceeds TG/8 + 1
// leaves, which bounds the LDS footprint.
//
// Page safety of the two source vectors: a full group's 16 source bytes are
// all valid leaf bytes, the first aligned source vector contains the first of
// them and the second contains the last, and an aligned 16-byte vector never
// spans two pages, so no load touches a page the copy does not already use
// (a lane that takes its second vector from the next lane loads nothing more).
#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "segtable.hpp"

namespace diffopt {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int E>
struct ElemT;
template <>
struct ElemT<1> {
  typedef uint8_t T;
};
template <>
struct ElemT<2> {
  typedef uint16_t T;
};
template <>
struct ElemT<4> {
  typedef uint32_t T;
};
template <>
struct ElemT<8> {
  typedef uint64_t T;
};

__device__ __forceinline__ uint32_t pick4(uint32_t a, uint32_t b, uint32_t c, uint32_t d, uint32_t q) {
  return q == 0 ? a : (q == 1 ? b : (q == 2 ? c : d));
}

// The 16 bytes starting s bytes into the 32-byte window (w0, w1), 0 <= s < 16
// (s = 0 gives w0, whatever w1 holds).
template <int E>
__device__ __forceinline__ u32x4 funnel(u32x4 w0, u32x4 w1, uint32_t s) {
  const uint32_t q = s >> 2;
  if (E >= 4) {  // s is a multiple of 4: whole-dword selection
    u32x4 o;
    o.x = pick4(w0.x, w0.y, w0.z, w0.w, q);
    o.y = pick4(w0.y, w0.z, w0.w, w1.x, q);
    o.z = pick4(w0.z, w0.w, w1.x, w1.y, q);
    o.w = pick4(w0.w, w1.x, w1.y, w1.z, q);
    return o;
  } else {
    const uint32_t r = s & 3u;
    const uint32_t y0 = pick4(w0.x, w0.y, w0.z, w0.w, q);
    const uint32_t y1 = pick4(w0.y, w0.z, w0.w, w1.x, q);
    const uint32_t y2 = pick4(w0.z, w0.w, w1.x, w1.y, q);
    const uint32_t y3 = pick4(w0.w, w1.x, w1.y, w1.z, q);
    const uint32_t y4 = pick4(w1.x, w1.y, w1.z, w1.w, q);
    u32x4 o;
    o.x = __builtin_amdgcn_alignbyte(y1, y0, r);
    o.y = __builtin_amdgcn_alignbyte(y2, y1, r);
    o.z = __builtin_amdgcn_alignbyte(y3, y2, r);
    o.w = __builtin_amdgcn_alignbyte(y4, y3, r);
    return o;
  }
}

// Trees of one structure copied by one launch: grid y selects the tree.
constexpr int kMaxBatch = 16;
struct CopyBatch {
  const uint64_t* leaf_ptrs[kMaxBatch];  // device arrays of leaf addresses
  uint64_t flat[kMaxBatch];              // flat buffers
};

// Tile order.  The dispatcher deals workgroups to the eight XCDs in turn, so
// neighbouring tiles -- which share the source line that straddles their
// boundary when source and destination are out of phase -- would run on
// different XCDs and both fetch that line from HBM.  With DIFFOPT_TREE_RUN =
// R > 1, each block of 8R workgroups takes 8R consecutive tiles so that the R
// workgroups an XCD receives get R consecutive tiles (the chip still works
// through one 8R-tile block at a time); a ragged last block keeps the plain
// order.  Measured on the 20,000-leaf tree, four trees per launch, fetched
// bytes over algorithmic (pack / unpack): plain order 1.042, R = 4 1.020 /
// 1.018, R = 8 1.014 / 1.012, R = 16 1.011 / 1.008, R = 32 1.009 / 1.006,
// R = 64 1.008 / 1.005 (the rest is the table and the partial head/tail
// groups).  The rate is the same within noise up to R = 32 (paired runs:
// R = 4 pack 6.12 against 6.10 TB/s for the plain order; R = 32 5.96 against
// 5.99 for R = 16 on a slower box) and 1% lower at R = 64.  A workgroup that
// copies a run of 2, 4 or 8 tiles in turn, with the next window prefetched,
// was slower (pack 5.1, 4.7, 4.6 TB/s against 6.1): the memory counter
// retires in order and counts stores too, so each tile's loads wait for the
// previous tile's stores, where one-tile workgroups end with their stores in
// flight.
#ifndef DIFFOPT_TREE_RUN
#define DIFFOPT_TREE_RUN 32
#endif

__device__ __forceinline__ int64_t tree_tile(int64_t b, int64_t ntiles) {
  constexpr int64_t R = DIFFOPT_TREE_RUN;
  if (R <= 1) return b;
  const int64_t base = b - b % (8 * R);
  if (base + 8 * R > ntiles) return b;
  const int64_t l = b - base;
  return base + (l % 8) * R + l / 8;
}

// The leaf holding a group, as the copy needs it: the leaf's first group and
// the next leaf's, the flat byte address of its range, its byte size and its
// address.
struct LeafRef {
  int64_t goff, goff_next;
  uint64_t fbase, bytes, leaf;
};

// Copies the groups of tile b.  find(gidx) returns the leaf holding group
// gidx; dummy is a valid, 16-byte aligned device address (see below).
template <int E, bool PACK, class Find>
__device__ __forceinline__ void copy_tile(const int64_t b, const int64_t ngroups, const uint64_t dummy, Find find) {
  // Phase 1 locates every group of this lane and issues all of its source
  // loads; phase 2 stores.  Sources never overlap destinations, so all loads
  // may go out before any store and each lane keeps kTreeU groups in flight.
  // The first load of a group is issued by every lane, outside any branch:
  // lanes without a full group read 16 bytes at dummy (the segment table:
  // valid, aligned, cached) and discard them.  A load under a branch leaves
  // its register undefined on the other path, and the join copied part of it
  // into another register, which waited for the load to return and so held
  // back the next group's search and loads.
  u32x4 w0[kTreeU], w1[kTreeU];
  uint64_t dst[kTreeU], lo_b[kTreeU], hi_b[kTreeU], delta[kTreeU], src_v[kTreeU];
  uint32_t shift[kTreeU];
  int kind[kTreeU];  // 0: nothing, 1: full aligned vector, 2: partial (element copy)
  bool own1[kTreeU];  // this lane loads its second source vector itself
#pragma unroll
  for (int u = 0; u < kTreeU; ++u) {
    const int64_t gidx = b * kTileGroups + (int64_t)u * kTB + threadIdx.x;
    kind[u] = 0;
    own1[u] = false;
    shift[u] = 0;
    src_v[u] = dummy;
    if (gidx < ngroups) {
      const LeafRef r = find(gidx);
      const uint64_t k = (uint64_t)(gidx - r.goff);
      const uint64_t fb = r.fbase;
      const uint64_t lb = r.leaf;
      const uint64_t nb = r.bytes;
      const uint64_t dst0 = PACK ? fb : lb;
      const uint64_t src0 = PACK ? lb : fb;
      const uint64_t A = (dst0 & ~uint64_t(127)) + 16u * k;  // groups count from dst0's line
      lo_b[u] = A > dst0 ? A : dst0;
      hi_b[u] = (A + 16u) < (dst0 + nb) ? (A + 16u) : (dst0 + nb);
      delta[u] = src0 - dst0;  // modular; the source byte of x is x + delta
      dst[u] = A;
      if (lo_b[u] < hi_b[u]) {
        if (lo_b[u] == A && hi_b[u] == A + 16u) {
          kind[u] = 1;
          const uint64_t S = A + delta[u];
          shift[u] = (uint32_t)(S & 15u);
          src_v[u] = S - shift[u];
#if DIFFOPT_TREE_SHARE
          // Lane l+1 of the wave holds group gidx+1.  When that group is a
          // full vector of the same leaf (same source-destination distance),
          // its first source vector is this lane's second one, so this lane
          // takes it from there instead of loading it again.
          const bool next_full = (threadIdx.x & 63) != 63 && gidx + 1 < r.goff_next && A + 32u <= dst0 + nb;
          own1[u] = shift[u] != 0 && !next_full;
#else
          own1[u] = shift[u] != 0;
#endif
        } else {
          kind[u] = 2;
        }
      }
    }
    const gptr<const u32x4> L = gaddr<const u32x4>(src_v[u]);
    w1[u] = u32x4{0u, 0u, 0u, 0u};
#if DIFFOPT_TREE_NT_LOADS
    w0[u] = __builtin_nontemporal_load(L);
#else
    w0[u] = L[0];
#endif
    if (own1[u]) {
      if (E >= 4) {
        // Whole-dword shifts read only the first three words of the second
        // vector.  Loading just those leaves the fourth register free, so it
        // can be reused without waiting for the load.
        const gptr<const uint32_t> L1 = gaddr<const uint32_t>(src_v[u] + 16u);
        w1[u].x = L1[0];
        w1[u].y = L1[1];
        w1[u].z = L1[2];
      } else {
#if DIFFOPT_TREE_NT_LOADS
        w1[u] = __builtin_nontemporal_load(L + 1);
#else
        w1[u] = L[1];
#endif
      }
    }
  }
  typedef typename ElemT<E>::T T;
#if DIFFOPT_TREE_SHARE
  // Every lane of the wave takes part in the cross-lane reads (ds_bpermute
  // from lane l+1; lane 63 wraps to lane 0 and never uses the value).
  const int next_lane = (int)((((threadIdx.x & 63) + 1) & 63) << 2);
#pragma unroll
  for (int u = 0; u < kTreeU; ++u) {
    u32x4 nv;
    nv.x = (uint32_t)__builtin_amdgcn_ds_bpermute(next_lane, (int)w0[u].x);
    nv.y = (uint32_t)__builtin_amdgcn_ds_bpermute(next_lane, (int)w0[u].y);
    nv.z = (uint32_t)__builtin_amdgcn_ds_bpermute(next_lane, (int)w0[u].z);
    nv.w = (uint32_t)__builtin_amdgcn_ds_bpermute(next_lane, (int)w0[u].w);
    if (!own1[u]) w1[u] = nv;
  }
#endif
  // Full groups first, partial groups after: the memory counter also counts
  // stores and retires in order, so a load issued between stores would make
  // the next full group's store wait for the earlier ones.
  u32x4 out[kTreeU];
#pragma unroll
  for (int u = 0; u < kTreeU; ++u) out[u] = funnel<E>(w0[u], w1[u], shift[u]);
#pragma unroll
  for (int u = 0; u < kTreeU; ++u) {
    if (kind[u] == 1) {
#if DIFFOPT_TREE_NT_STORES
      __builtin_nontemporal_store(out[u], gaddr<u32x4>(dst[u]));
#else
      *gaddr<u32x4>(dst[u]) = out[u];
#endif
    }
  }
#pragma unroll
  for (int u = 0; u < kTreeU; ++u) {
    if (kind[u] == 2) {
      for (uint64_t x = lo_b[u]; x < hi_b[u]; x += E) {
        *gaddr<T>(x) = *gaddr<const T>(x + delta[u]);
      }
    }
  }
}

// A tile that lies in one leaf reads that leaf's entry into scalar registers
// instead of staging a window in LDS: the entry, the next entry's first group
// and, with DENSE (no empty leaves, so the table index is the leaf index), the
// leaf's address are read together.  Extending this to windows of up to four
// leaves (a lane picking its leaf by comparing its group with the leaf starts)
// measured no faster on the 20,000-leaf tree, so wider windows keep the LDS
// path.
template <int E, bool PACK, bool DENSE>
__device__ __forceinline__ void copy_tile_one_leaf(const SegEntry* seg, const uint64_t* leaf_ptrs, uint64_t flat,
                                                   int64_t j0, int64_t b, int64_t ngroups) {
  const cptr<int64_t> e = caddr<int64_t>(seg + j0);  // goff, off, numel, orig; then the next entry
  int64_t goff = e[0], off = e[1], numel = e[2], goff_next = e[4];
  uint64_t leaf = *caddr<uint64_t>(leaf_ptrs + (DENSE ? j0 : e[3]));
  // The empty asm takes all five values at one point, so every read is issued
  // before the single wait for them (left alone, the compiler issued the
  // leaf-address read only after waiting for the entry).
  asm volatile("" : "+s"(goff), "+s"(off), "+s"(numel), "+s"(goff_next), "+s"(leaf));
  const LeafRef r{goff, goff_next, flat + (uint64_t)(off * E), (uint64_t)(numel * E), leaf};
  copy_tile<E, PACK>(b, ngroups, (uint64_t)seg, [&](int64_t) { return r; });
}

template <int E, bool PACK, bool DENSE>
__global__ __launch_bounds__(kTB) void tree_copy_kernel(const SegEntry* __restrict__ seg,
                                                        const int64_t* __restrict__ tile_first, int64_t ngroups,
                                                        CopyBatch batch) {
  const uint64_t* __restrict__ leaf_ptrs = batch.leaf_ptrs[blockIdx.y];
  const uint64_t flat = batch.flat[blockIdx.y];
  __shared__ int64_t s_goff[kWindowMax + 1];
  __shared__ int64_t s_fbase[kWindowMax];  // flat byte address of the leaf's range
  __shared__ int64_t s_bytes[kWindowMax];
  __shared__ uint64_t s_leaf[kWindowMax];

  const int64_t b = tree_tile(blockIdx.x, gridDim.x);
  const int64_t j0 = tile_first[b];
  const int W = (int)(tile_first[b + 1] - j0 + 1);  // the same for every lane of the block
  if (W == 1) {  // most tiles of large leaves
    copy_tile_one_leaf<E, PACK, DENSE>(seg, leaf_ptrs, flat, j0, b, ngroups);
    return;
  }
  for (int t = threadIdx.x; t <= W; t += kTB) {
    // With DENSE the leaf address is fetched alongside the table entry
    // instead of after it.
    const uint64_t lp = (DENSE && t < W) ? leaf_ptrs[j0 + t] : 0;
    const SegEntry e = seg[j0 + t];
    s_goff[t] = e.goff;
    if (t < W) {
      s_fbase[t] = (int64_t)(flat + (uint64_t)(e.off * E));
      s_bytes[t] = e.numel * E;
      s_leaf[t] = DENSE ? lp : leaf_ptrs[e.orig];
    }
  }
  __syncthreads();
  copy_tile<E, PACK>(b, ngroups, (uint64_t)seg, [&](int64_t gidx) {
    // largest t with s_goff[t] <= gidx; s_goff[0] <= gidx holds by construction
    int lo = 0, hi = W - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_goff[mid] <= gidx) lo = mid;
      else hi = mid - 1;
    }
    return LeafRef{s_goff[lo], s_goff[lo + 1], (uint64_t)s_fbase[lo], (uint64_t)s_bytes[lo], s_leaf[lo]};
  });
}

// Small trees whose flat layout is the plain concatenation of the leaves (a
// TinyTable and no gaps): one element per lane, element j of the flat buffer
// being element j of the concatenated leaves; the leaf comes from a scan of
// the table in the kernel arguments, so a lane's only dependent loads are its
// leaf's address and then the element.  The launch is bound by latency, not
// bandwidth (1,761 elements: seven waves).
constexpr int kTinyCB = 256;

template <int E, bool PACK>
__global__ __launch_bounds__(kTinyCB) void tree_copy_tiny(TinyTable tt, CopyBatch batch) {
  warm_args(fold_lines(tt) ^ fold_lines(batch));
  typedef typename ElemT<E>::T T;
  const uint64_t* __restrict__ leaf_ptrs = batch.leaf_ptrs[blockIdx.y];
  const uint64_t flat = batch.flat[blockIdx.y];
  const int64_t j = (int64_t)blockIdx.x * kTinyCB + threadIdx.x;
  int orig;
  int64_t i;
  if (!tiny_slot(tt, j, orig, i)) return;
  const gptr<T> f = gaddr<T>(flat) + j;
  const gptr<T> l = gaddr<T>(leaf_ptrs[orig]) + i;
  if (PACK) *f = *l;
  else *l = *f;
}

}  // namespace
}  // namespace diffopt

using namespace diffopt;

extern "C" int diffopt_segtable_create(int64_t nseg, const int64_t* numel, const int64_t* offsets,
                                       int32_t elem_bytes, diffopt_segtable** out) {
  clear_error();
  static const char* who = "diffopt_segtable_create";
  if (!out) return fail(DIFFOPT_EINVAL, "%s: out is NULL", who);
  *out = nullptr;
  if (nseg < 0) return fail(DIFFOPT_EINVAL, "%s: nseg must be >= 0", who);
  if (nseg > 0 && !numel) return fail(DIFFOPT_EINVAL, "%s: numel is NULL", who);
  if (elem_bytes != 1 && elem_bytes != 2 && elem_bytes != 4 && elem_bytes != 8)
    return fail(DIFFOPT_EINVAL, "%s: elem_bytes must be 1, 2, 4 or 8 (got %d)", who, elem_bytes);
  const int64_t kMaxElems = (int64_t(1) << 58) / elem_bytes;

  std::vector<SegEntry> host;
  std::vector<std::pair<int64_t, int64_t>> ranges;  // (off, end) of nonempty leaves
  try {
    host.reserve((size_t)nseg + 1);
    ranges.reserve((size_t)nseg);
  } catch (const std::bad_alloc&) {
    return fail(DIFFOPT_ENOMEM, "%s: host allocation failed", who);
  }
  int64_t run = 0, total = 0, goff = 0;
  for (int64_t j = 0; j < nseg; ++j) {
    const int64_t k = numel[j];
    if (k < 0) return fail(DIFFOPT_EINVAL, "%s: numel[%lld] < 0", who, (long long)j);
    if (k > kMaxElems) return fail(DIFFOPT_EINVAL, "%s: numel[%lld] too large", who, (long long)j);
    const int64_t off = offsets ? offsets[j] : run;
    if (off < 0 || off > kMaxElems - k)
      return fail(DIFFOPT_EINVAL, "%s: offset of leaf %lld out of range", who, (long long)j);
    run = off + k;
    if (k == 0) continue;
    total = std::max(total, off + k);
    const int64_t need = (k * elem_bytes + 15) / 16 + 8;  // +8 absorbs any phase within the first line
    const int64_t groups = (need + kLeafGroupAlign - 1) / kLeafGroupAlign * kLeafGroupAlign;
    host.push_back(SegEntry{goff, off, k, j});
    ranges.emplace_back(off, off + k);
    goff += groups;
  }
  if (offsets) {
    std::sort(ranges.begin(), ranges.end());
    for (size_t i = 1; i < ranges.size(); ++i)
      if (ranges[i].first < ranges[i - 1].second)
        return fail(DIFFOPT_EINVAL, "%s: flat ranges of two leaves overlap at element %lld", who,
                    (long long)ranges[i].first);
  }
  const int64_t nact = (int64_t)host.size();
  host.push_back(SegEntry{goff, 0, 0, 0});  // sentinel

  diffopt_segtable* t = new (std::nothrow) diffopt_segtable();
  if (!t) return fail(DIFFOPT_ENOMEM, "%s: host allocation failed", who);
  t->nseg = nseg;
  t->total = total;
  t->nact = nact;
  t->ngroups = goff;
  t->elem_bytes = elem_bytes;
  t->ntiles = (goff + kTileGroups - 1) / kTileGroups;
  t->dense_orig = (nact == nseg) ? 1 : 0;
  if (hipGetDevice(&t->device) != hipSuccess) t->device = -1;
  int64_t elems = 0;
  for (int64_t j = 0; j < nact; ++j) elems += host[(size_t)j].numel;
  t->contiguous = 1;
  for (int64_t j = 0, at = 0; j < nact; at += host[(size_t)j].numel, ++j)
    if (host[(size_t)j].off != at) t->contiguous = 0;
  if (nact >= 1 && nact <= kTinyLeaves && elems <= kTinyElems) {
    t->tiny = 1;
    t->small.n = (int32_t)nact;
    int32_t at = 0;
    for (int64_t j = 0; j < kTinyLeaves; ++j) {
      t->small.start[j] = j < nact ? at : INT32_MAX;
      t->small.orig[j] = j < nact ? (int32_t)host[(size_t)j].orig : 0;
      if (j < nact) at += (int32_t)host[(size_t)j].numel;
    }
    t->small.total = at;
  }

  std::vector<int64_t> tf;
  if (t->ntiles > 0) {
    tf.resize((size_t)t->ntiles + 1);
    // tile_first[b] = the leaf whose group range holds group b*TG
    int64_t j = 0;
    for (int64_t b = 0; b < t->ntiles; ++b) {
      const int64_t g = b * kTileGroups;
      while (j + 1 < nact && host[(size_t)j + 1].goff <= g) ++j;
      tf[(size_t)b] = j;
    }
    tf[(size_t)t->ntiles] = nact - 1;
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&t->d_seg), sizeof(SegEntry) * host.size());
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&t->d_tile_first), sizeof(int64_t) * tf.size());
    if (e == hipSuccess)
      e = hipMemcpy(t->d_seg, host.data(), sizeof(SegEntry) * host.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = hipMemcpy(t->d_tile_first, tf.data(), sizeof(int64_t) * tf.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      int code = (e == hipErrorOutOfMemory) ? DIFFOPT_ENOMEM : DIFFOPT_EHIP;
      diffopt_segtable_destroy(t);
      return fail(code, "%s: %s", who, hipGetErrorString(e));
    }
  }
  *out = t;
  return DIFFOPT_OK;
}

extern "C" void diffopt_segtable_destroy(diffopt_segtable* t) {
  if (!t) return;
  if (t->d_seg) (void)hipFree(t->d_seg);  // nothing to report to: destroy has no error return
  if (t->d_tile_first) (void)hipFree(t->d_tile_first);
  delete t;
}

extern "C" int64_t diffopt_segtable_total(const diffopt_segtable* t) { return t ? t->total : -1; }

extern "C" int64_t diffopt_segtable_nseg(const diffopt_segtable* t) { return t ? t->nseg : -1; }

namespace {

template <int E, bool PACK>
void launch_copy(dim3 grid, hipStream_t st, const diffopt_segtable* t, const CopyBatch& batch) {
  if (t->dense_orig)
    hipLaunchKernelGGL((tree_copy_kernel<E, PACK, true>), grid, dim3(kTB), 0, st, t->d_seg, t->d_tile_first,
                       t->ngroups, batch);
  else
    hipLaunchKernelGGL((tree_copy_kernel<E, PACK, false>), grid, dim3(kTB), 0, st, t->d_seg, t->d_tile_first,
                       t->ngroups, batch);
}

// ntrees copies of one structure: leaf_ptrs[t] is tree t's device array of
// leaf addresses, flat[t] its flat buffer; up to kMaxBatch trees per launch.
template <bool PACK>
int tree_copy(const char* who, const diffopt_segtable* t, int64_t ntrees, const uint64_t* const* leaf_ptrs,
              const uint64_t* flat, void* stream) {
  if (!t) return fail(DIFFOPT_EINVAL, "%s: table is NULL", who);
  if (ntrees < 0) return fail(DIFFOPT_EINVAL, "%s: ntrees must be >= 0", who);
  if (t->ntiles == 0 || ntrees == 0) return DIFFOPT_OK;
  for (int64_t k = 0; k < ntrees; ++k) {
    if (!leaf_ptrs[k] || !flat[k]) return fail(DIFFOPT_EINVAL, "%s: null leaf_ptrs or flat (tree %lld)", who,
                                               (long long)k);
    if (flat[k] % (uint64_t)t->elem_bytes != 0)
      return fail(DIFFOPT_EINVAL, "%s: flat buffer of tree %lld is not aligned to elem_bytes", who, (long long)k);
  }
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != t->device)
    return fail(DIFFOPT_EINVAL, "%s: the table lives on device %d, the current device is %d", who, t->device, dev);
  hipStream_t st = as_stream(stream);
  for (int64_t k0 = 0; k0 < ntrees; k0 += kMaxBatch) {
    const int nb = (int)(ntrees - k0 < kMaxBatch ? ntrees - k0 : kMaxBatch);
    CopyBatch batch{};
    for (int k = 0; k < nb; ++k) {
      batch.leaf_ptrs[k] = leaf_ptrs[k0 + k];
      batch.flat[k] = flat[k0 + k];
    }
    if (t->tiny && t->contiguous) {
      const dim3 tgrid((unsigned)((t->small.total + kTinyCB - 1) / kTinyCB), (unsigned)nb);
      switch (t->elem_bytes) {
        case 1:
          hipLaunchKernelGGL((tree_copy_tiny<1, PACK>), tgrid, dim3(kTinyCB), 0, st, t->small, batch);
          break;
        case 2:
          hipLaunchKernelGGL((tree_copy_tiny<2, PACK>), tgrid, dim3(kTinyCB), 0, st, t->small, batch);
          break;
        case 4:
          hipLaunchKernelGGL((tree_copy_tiny<4, PACK>), tgrid, dim3(kTinyCB), 0, st, t->small, batch);
          break;
        default:
          hipLaunchKernelGGL((tree_copy_tiny<8, PACK>), tgrid, dim3(kTinyCB), 0, st, t->small, batch);
          break;
      }
      int rc = launch_status(who);
      if (rc) return rc;
      continue;
    }
    const dim3 grid((unsigned)t->ntiles, (unsigned)nb);
    switch (t->elem_bytes) {
      case 1:
        launch_copy<1, PACK>(grid, st, t, batch);
        break;
      case 2:
        launch_copy<2, PACK>(grid, st, t, batch);
        break;
      case 4:
        launch_copy<4, PACK>(grid, st, t, batch);
        break;
      default:
        launch_copy<8, PACK>(grid, st, t, batch);
        break;
    }
    int rc = launch_status(who);
    if (rc) return rc;
  }
  return DIFFOPT_OK;
}

}  // namespace

extern "C" int diffopt_tree_flatten(const diffopt_segtable* t, const uint64_t* leaf_ptrs, void* flat, void* stream) {
  clear_error();
  const uint64_t f = reinterpret_cast<uint64_t>(flat);
  return tree_copy<true>("diffopt_tree_flatten", t, 1, &leaf_ptrs, &f, stream);
}

extern "C" int diffopt_tree_unflatten(const diffopt_segtable* t, const void* flat, const uint64_t* leaf_ptrs,
                                      void* stream) {
  clear_error();
  const uint64_t f = reinterpret_cast<uint64_t>(flat);
  return tree_copy<false>("diffopt_tree_unflatten", t, 1, &leaf_ptrs, &f, stream);
}

extern "C" int diffopt_tree_flatten_batch(const diffopt_segtable* t, int64_t ntrees, const uint64_t* const* leaf_ptrs,
                                          void* const* flats, void* stream) {
  clear_error();
  static const char* who = "diffopt_tree_flatten_batch";
  if (ntrees > 0 && (!leaf_ptrs || !flats)) return fail(DIFFOPT_EINVAL, "%s: null pointer array", who);
  return tree_copy<true>(who, t, ntrees, leaf_ptrs, reinterpret_cast<const uint64_t*>(flats), stream);
}

extern "C" int diffopt_tree_unflatten_batch(const diffopt_segtable* t, int64_t ntrees, const void* const* flats,
                                            const uint64_t* const* leaf_ptrs, void* stream) {
  clear_error();
  static const char* who = "diffopt_tree_unflatten_batch";
  if (ntrees > 0 && (!leaf_ptrs || !flats)) return fail(DIFFOPT_EINVAL, "%s: null pointer array", who);
  return tree_copy<false>(who, t, ntrees, leaf_ptrs, reinterpret_cast<const uint64_t*>(flats), stream);
}
