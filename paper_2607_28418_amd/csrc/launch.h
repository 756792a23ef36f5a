// Kernel launch wrapper with optional per-launch HIP-event timing.
#pragma once

#include <hip/hip_runtime.h>

namespace wide {

// Returns a timing slot (>= 0) when timing is enabled and the event pool has
// room, else -1.  Both record on `s`, the stream the kernel is launched on.
int timing_begin(const char* name, hipStream_t s);
void timing_end(int slot, hipStream_t s);

}  // namespace wide

// KERN may be a parenthesised template instance: (kern<A, B>).  NAME is the
// label timing queries match against.
#define WIDE_LAUNCH_NAMED(NAME, KERN, GRID, BLOCK, SHMEM, STREAM, ...)    \
  do {                                                                    \
    const int wide_slot_ = ::wide::timing_begin((NAME), (STREAM));        \
    hipLaunchKernelGGL(KERN, (GRID), (BLOCK), (SHMEM), (STREAM), __VA_ARGS__); \
    ::wide::timing_end(wide_slot_, (STREAM));                             \
  } while (0)

#define WIDE_LAUNCH(KERN, GRID, BLOCK, SHMEM, STREAM, ...) \
  WIDE_LAUNCH_NAMED(#KERN, KERN, GRID, BLOCK, SHMEM, STREAM, __VA_ARGS__)
