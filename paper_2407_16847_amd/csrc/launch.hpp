// launch.hpp -- internal interface between the C ABI and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "acsr_core.hpp"

namespace splat {

// Device view of an ACSR handle's metadata.
struct DevAcsr {
  int32_t L;
  int64_t nnz;
  int32_t max_row_nnz;
  int32_t n_groups;
  const int32_t* row_ptr;   // L + 1
  const RowRuns* runs;      // L
  const int32_t* rows;      // L (grouped)
  const Group* groups;      // n_groups
  const Tile* tiles;
  const uint64_t* masks;    // kBM row masks per tile that has a PARTIAL wavefront
  const ColRun* cols;       // L single-run column descriptors, or null (no column-major layout)
};

// Position of `row` in the column-major value array of one head, for a row
// that is in column c: c.ptr + (row - c.start) / c.stride.  The quotient is
// exact and below 2^16, so the float reciprocal (1 ulp) rounds back to it.
__device__ __forceinline__ int col_pos(const ColRun& c, int row) {
  const float t = (float)(row - c.start) * __builtin_amdgcn_rcpf((float)c.stride);
  return c.ptr + (int)__builtin_rintf(t);
}

// Every launcher enqueues on `st` and returns the launch status.
// dtype / out dtype: 0 = fp32, 1 = bf16.

// Row-per-wave kernels: any d in {64, 128}, both dtypes.
hipError_t launch_rsddmm_rows(const DevAcsr& a, int dtype, int BH, int d, const void* Q,
                              const void* K, float scale, float* S, hipStream_t st);
// colmajor: P holds the column-major values (requires a.cols).
hipError_t launch_rspmm_rows(const DevAcsr& a, int dtype, int BH, int d, const float* P,
                             const void* V, void* O, int out_dtype, bool colmajor, hipStream_t st);
hipError_t launch_fused_rows(const DevAcsr& a, int dtype, int BH, int d, const void* Q,
                             const void* K, const void* V, float scale, void* O, int out_dtype,
                             hipStream_t st);

// Matrix-core kernels over the tile plan: bf16 inputs, d in {64, 128}.
hipError_t launch_rsddmm_tiles(const DevAcsr& a, int BH, int d, const void* Q, const void* K,
                               float scale, float* S, hipStream_t st);
hipError_t launch_rspmm_tiles(const DevAcsr& a, int BH, int d, const float* P, const void* V,
                              void* O, int out_dtype, bool colmajor, hipStream_t st);

// Row-major (CSR order) values -> column-major values (requires a.cols).
hipError_t launch_transpose_colmajor(const DevAcsr& a, int BH, const float* P, float* Pt,
                                     hipStream_t st);

// Row softmax, any row length (rows of up to 2048 values in registers).
hipError_t launch_softmax(const DevAcsr& a, int BH, const float* S, float* P, hipStream_t st);

// Allows the fused kernels their dynamic LDS (above the default limit at
// d = 128) on the current device.  Called once per handle at build time, on
// the handle's device, so launches never change kernel attributes.
hipError_t prepare_fused_mfma();

// Index checks of a build with -DSPLAT_DEBUG_BOUNDS (no-ops otherwise): each
// kernel file's flags on the current device, OR-ed into *bits (bit k = kind
// k of bounds.hpp), cleared when `clear`.
hipError_t bounds_collect_rows(uint32_t* bits, bool clear);
hipError_t bounds_collect_mfma(uint32_t* bits, bool clear);
hipError_t bounds_collect_tiles(uint32_t* bits, bool clear);
// One check of `index` against [0, n) as kind `kind`, run on the device
// (allocates and frees one int); *result = the checked index.
hipError_t bounds_probe(int kind, int index, int n, int* result);

hipError_t launch_fused_mfma(const DevAcsr& a, int BH, int d, const void* Q, const void* K,
                             const void* V, float scale, void* O, int out_dtype, hipStream_t st);

}  // namespace splat
