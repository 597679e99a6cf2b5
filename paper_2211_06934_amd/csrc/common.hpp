// Shared internals of the diffopt HIP library: error state and launch checks.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "diffopt.h"

namespace diffopt {

// Threads per workgroup for every kernel: four 64-wide wavefronts.
constexpr int kBlock = 256;

// Record a message for diffopt_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clear the calling thread's message (start of every entry point).
void clear_error();

// Map the state left by a kernel launch to a return code.
int launch_status(const char* what);

// hipStream_t from the ABI's void*.
inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ---- kernel arguments of the small-problem kernels ---------------------------
// Kernel arguments are read through the scalar cache, one 64-byte line at a
// time, and the compiler loads each step's coefficients just before that
// step: in a kernel bound by latency every step then waits for a memory
// round trip of its own (about 0.4 us per step on MI355X).  Folding one word
// of every line of an argument into a single value that an empty asm
// statement consumes makes the kernel issue all of those loads at its start,
// with one wait; the later reads of the same lines hit the cache.
// The words are copied out with memcpy, the defined way to read an object's
// bytes as another type.
template <class T>
__device__ __forceinline__ int32_t fold_lines(const T& x) {
  constexpr int kWords = (int)(sizeof(T) / 4);
  const char* bytes = reinterpret_cast<const char*>(&x);
  int32_t acc, w;
  __builtin_memcpy(&acc, bytes + 4 * (kWords - 1), 4);
#pragma unroll
  for (int l = 0; l * 16 < kWords; ++l) {
    __builtin_memcpy(&w, bytes + 64 * l, 4);
    acc ^= w;
  }
  return acc;
}

__device__ __forceinline__ void warm_args(int32_t folded) { asm volatile("" : : "s"(folded)); }

}  // namespace diffopt
