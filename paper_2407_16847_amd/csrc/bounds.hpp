// bounds.hpp -- optional device-side index checks (-DSPLAT_DEBUG_BOUNDS).
//
// The kernels compute their global-memory indices from the plan and the ACSR
// runs: query rows from the grouped row list, key rows from tile descriptors
// and runs, value positions in S and P from row_ptr and running counts,
// column-major positions from column descriptors.  A library built with
// -DSPLAT_DEBUG_BOUNDS checks each such index against the size it indexes.
// An index outside [0, n) sets the flag of its kind in the kernel file's
// flag array and is replaced by 0, so the access stays inside the buffer
// (the result is then wrong, and the flag says so).  The host collects and
// clears the flags with splat_debug_bounds().  In the regular build every
// check is the index itself and the flag arrays do not exist.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace splat {
namespace dbg {

// kinds of checked index, one flag bit each in splat_debug_bounds()
enum Kind : int {
  kRow = 0,      // a query row, [0, L)
  kKey = 1,      // a key row of K or V, [0, L)
  kValue = 2,    // a position in S or P: [0, nnz) in a head, [0, B*H*nnz) overall
  kColPos = 3,   // a position in one head's column-major values, [0, nnz)
  kKinds = 4
};

#ifdef SPLAT_DEBUG_BOUNDS
// one word per kind, per kernel file (internal linkage: every file that
// includes this header has its own array, read by its own bounds_collect)
static __device__ uint32_t g_flags[kKinds];
#endif

template <typename I>
__device__ __forceinline__ I idx(I i, I n, Kind kind) {
#ifdef SPLAT_DEBUG_BOUNDS
  if (!(i >= 0 && i < n)) {
    g_flags[kind] = 1u;   // plain vector store: every violation writes the same value
    return 0;
  }
#else
  (void)n;
  (void)kind;
#endif
  return i;
}

// A condition on a whole range (a row's values): false, with its kind
// recorded, when it fails in a checked build; always true in the regular one.
__device__ __forceinline__ bool check(bool ok, Kind kind) {
#ifdef SPLAT_DEBUG_BOUNDS
  if (!ok) g_flags[kind] = 1u;
  return ok;
#else
  (void)ok;
  (void)kind;
  return true;
#endif
}

// An offset o from base position b, checked as position b + o in [0, n):
// o itself, or the offset of position 0 when b + o is outside (the regular
// build computes exactly the unchecked expression base + o).
template <typename I, typename J>
__device__ __forceinline__ I rel(I o, J b, J n, Kind kind) {
#ifdef SPLAT_DEBUG_BOUNDS
  const J p = b + (J)o;
  if (!(p >= 0 && p < n)) {
    g_flags[kind] = 1u;
    return (I)(-b);
  }
#else
  (void)b;
  (void)n;
  (void)kind;
#endif
  return o;
}

// Host side, current device: ORs this file's flags into *bits (bit k = kind
// k) and, when `clear`, zeroes them.  A no-op in the regular build.
static inline hipError_t collect(uint32_t* bits, bool clear) {
#ifdef SPLAT_DEBUG_BOUNDS
  uint32_t w[kKinds];
  hipError_t e = hipMemcpyFromSymbol(w, HIP_SYMBOL(g_flags), sizeof(w), 0, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return e;
  for (int k = 0; k < kKinds; ++k)
    if (w[k]) *bits |= 1u << k;
  if (clear) {
    const uint32_t z[kKinds] = {0, 0, 0, 0};
    e = hipMemcpyToSymbol(HIP_SYMBOL(g_flags), z, sizeof(z), 0, hipMemcpyHostToDevice);
  }
  return e;
#else
  (void)bits;
  (void)clear;
  return hipSuccess;
#endif
}

}  // namespace dbg
}  // namespace splat
