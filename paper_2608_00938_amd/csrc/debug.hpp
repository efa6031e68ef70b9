// Device-side checks of the debug build (sources compiled with -DGRACE_DEBUG,
// library libgrace_debug.so).
//
// The release kernels clamp every index that comes from the data (request
// offsets, parents, block ids) so that a bad input cannot reach outside its
// buffers.  The debug build also counts every such clamp, and checks the row
// index of every global access the attention kernels compute against the
// extent of its buffer, so a test can tell a clean run from one that a clamp
// (or an indexing error hidden by one) rescued.  grace_debug_counts() reads
// and clears the counters.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace grace {

enum DebugKind : int {
  kDbgOffsets = 0,   // a request's offsets out of order or outside [0, sum_L]
  kDbgParent = 1,    // a parent outside [0, M_prev)
  kDbgBlockId = 2,   // a block id outside the pool
  kDbgRow = 3,       // a computed row index outside its buffer, or a work item outside the grid's problem
  kDbgKinds = 8,
};

}  // namespace grace

#ifdef GRACE_DEBUG
// One counter array per source file (device variables are not shared across
// files without relocatable device code); each file's debug_take_* reads and
// clears its own.
#define GRACE_DEBUG_COUNTERS static __device__ unsigned int g_grace_debug[grace::kDbgKinds]
#define GRACE_DCHECK(cond, kind)                                   \
  do {                                                             \
    if (!(cond)) atomicAdd(&g_grace_debug[(kind)], 1u);            \
  } while (0)
#else
#define GRACE_DEBUG_COUNTERS static_assert(true, "")
#define GRACE_DCHECK(cond, kind) \
  do {                           \
  } while (0)
#endif
