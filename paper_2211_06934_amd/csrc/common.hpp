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

}  // namespace diffopt
