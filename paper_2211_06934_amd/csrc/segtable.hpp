// Device segment table shared by tree flatten / unflatten (tree.hip) and the
// leaf-direct Adam kernels (treemap.hip): the group index space, the tile plan
// and the window bound.
#pragma once

#include "common.hpp"

// Launch shape, chosen by measurement on MI355X (20,000 leaves, n ~ 1.2e8):
// 256 threads x 2 groups per tile with streaming stores.  One group per lane
// (any workgroup size) spends too long per staged window; 4 groups per lane
// (5-6% slower in a paired run on six allocations), 512-thread tiles (1-3%
// slower), and renumbering tiles so that each XCD walks a contiguous eighth
// of them, were slower.
#ifndef DIFFOPT_TREE_U
#define DIFFOPT_TREE_U 2  // groups (16-byte vectors) per lane per tile
#endif
#ifndef DIFFOPT_TREE_BLOCK
#define DIFFOPT_TREE_BLOCK 256  // threads per workgroup of the copy kernel
#endif
#ifndef DIFFOPT_TREE_NT_LOADS
#define DIFFOPT_TREE_NT_LOADS 0  // streaming loads of source vectors
#endif
#ifndef DIFFOPT_TREE_SHARE
#define DIFFOPT_TREE_SHARE 1  // second source vector taken from the next lane
#endif
#ifndef DIFFOPT_TREE_NT_STORES
#define DIFFOPT_TREE_NT_STORES 1  // streaming stores of full destination vectors
#endif

namespace diffopt {

constexpr int kTreeU = DIFFOPT_TREE_U;
constexpr int kTB = DIFFOPT_TREE_BLOCK;
constexpr int64_t kTileGroups = (int64_t)kTB * kTreeU;
// Every nonempty leaf owns a multiple of kLeafGroupAlign groups (at least 16),
// so leaves start on 8-group (128-byte) boundaries of the group space: tile
// boundaries then fall on line boundaries of the copy's destination and of
// 128-byte aligned leaves, and a tile touches at most kTileGroups / 8 + 1
// leaves.
constexpr int64_t kLeafGroupAlign = 8;
constexpr int kWindowMax = (int)(kTileGroups / kLeafGroupAlign + 2);

// Leaf and flat-buffer memory is device (global) memory, but its addresses
// come from the staged LDS window as integers, so a plain pointer would be
// generic and every access a flat_* instruction.  Flat instructions count
// against the LDS wait counter too: a lane's next window lookup would then
// wait for all of its outstanding HBM loads.  Address space 1 makes the
// compiler emit global_* instructions, which count only as vector memory.
template <typename T>
using gptr = __attribute__((address_space(1))) T*;

template <typename T>
__device__ __forceinline__ gptr<T> gaddr(uint64_t addr) {
  return (gptr<T>)addr;
}

// Read-only memory that no kernel writes while it runs (the segment table and
// the caller's leaf-address arrays), read at an address the same for the whole
// workgroup: address space 4 lets the compiler use scalar loads, which issue
// together and count on their own wait counter.
template <typename T>
using cptr = const __attribute__((address_space(4))) T*;

template <typename T>
__device__ __forceinline__ cptr<T> caddr(const void* addr) {
  return (cptr<T>)(uint64_t)addr;
}

// One nonempty leaf, in table order.  The entry after the last nonempty leaf
// is a sentinel whose goff is the total group count.
struct SegEntry {  // four int64 fields in this order (read as such)
  int64_t goff;   // first group index
  int64_t off;    // flat element offset
  int64_t numel;  // elements
  int64_t orig;   // index into the caller's leaf-address array
};

// Small trees: the table of nonempty leaves, passed to the leaf-direct Adam
// kernels by value so that a lane finds its leaf from kernel arguments alone.
// Lane j takes element j of the concatenated leaves (no group padding).  The
// launch is then bound by dependent memory latency and by each lane's chain
// of arithmetic rather than by bandwidth, so each lane takes one element and
// issues every load before any arithmetic.
constexpr int kTinyLeaves = 32;
constexpr int64_t kTinyElems = int64_t(1) << 16;

struct TinyTable {
  int32_t n = 0;                 // nonempty leaves
  int32_t total = 0;             // their element count
  int32_t start[kTinyLeaves]{};  // first element of each leaf; INT32_MAX past the last leaf
  int32_t orig[kTinyLeaves]{};   // the leaf's index in the caller's leaf-address arrays
};

// Element j of the concatenated leaves: its leaf's caller index and its index
// in the leaf.  The scan is unrolled over the whole table (entries past the
// last leaf start at INT32_MAX), so it reads the kernel arguments at fixed
// offsets and takes no branch.  Each entry passes through an empty asm
// statement so that it is selected as a value held in a scalar register:
// otherwise the compiler selects its address instead and reads the chosen
// entry with a per-lane load, one more memory round trip before the leaf
// addresses can be loaded.
__device__ __forceinline__ bool tiny_slot(const TinyTable& tt, int64_t j, int& orig, int64_t& i) {
  if (j >= tt.total) return false;
  const int32_t jj = (int32_t)j;
  int o = tt.orig[0];
  int32_t first = 0;
#pragma unroll
  for (int t = 1; t < kTinyLeaves; ++t) {
    int32_t st = tt.start[t], ot = tt.orig[t];
    asm volatile("" : "+s"(st), "+s"(ot));
    const bool in = jj >= st;
    o = in ? ot : o;
    first = in ? st : first;
  }
  orig = o;
  i = jj - first;
  return true;
}

}  // namespace diffopt

struct diffopt_segtable {
  int64_t nseg = 0;
  int64_t total = 0;
  int64_t nact = 0;
  int64_t ngroups = 0;
  int64_t ntiles = 0;
  int32_t elem_bytes = 4;
  int device = 0;
  int dense_orig = 1;               // no empty leaves: table index == leaf index
  int tiny = 0;                     // the leaves fit a TinyTable (held in `small`)
  int contiguous = 0;               // every nonempty leaf's flat offset is the element count before it
  diffopt::TinyTable small;
  diffopt::SegEntry* d_seg = nullptr;       // [nact + 1]
  int64_t* d_tile_first = nullptr;  // [ntiles + 1]
};

