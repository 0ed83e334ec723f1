// kernels_rows.hip -- one wavefront per (batch*head, row) kernels.
//
// These walk each row's affine runs directly (the ACSR index map of section
// 5.1: the k-th value of run r sits at column start + stride * k) and serve
// every dtype and pattern: they are the fp32 path (fp32 FMA throughout, the
// library's accurate path) and run any request the matrix-core kernels do
// not take.  Lanes own keys (SDDMM, fused) or output features (SpMM).
#include <hip/hip_runtime.h>
#include <math.h>

#include "bounds.hpp"
#include "launch.hpp"

namespace splat {
namespace {

constexpr int kWave = 64;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(__bf16 x) { return (float)x; }
__device__ __forceinline__ void store(float* p, float v) { *p = v; }
__device__ __forceinline__ void store(__bf16* p, float v) { *p = (__bf16)v; }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// column of the k-th value of a row (k < row nnz)
__device__ __forceinline__ int col_of(const RowRuns& rr, int k) {
  int j = 0;
#pragma unroll
  for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
    const Run q = rr.r[r];
    if (k >= q.prefix && k < q.prefix + q.count) j = q.start + q.stride * (k - q.prefix);
  }
  return j;
}

// dot(qs[0:d], row[0:d]) in fp32, sequential FMA over the features
template <typename T>
__device__ __forceinline__ float dot_row(const float* qs, const T* row, int d) {
  float s = 0.f;
  for (int c = 0; c < d; c += 4) {
    s = fmaf(qs[c + 0], to_f32(row[c + 0]), s);
    s = fmaf(qs[c + 1], to_f32(row[c + 1]), s);
    s = fmaf(qs[c + 2], to_f32(row[c + 2]), s);
    s = fmaf(qs[c + 3], to_f32(row[c + 3]), s);
  }
  return s;
}

template <typename T>
__global__ __launch_bounds__(kWave) void k_rsddmm_rows(DevAcsr a, int d, const T* __restrict__ Q,
                                                       const T* __restrict__ K, float scale,
                                                       float* __restrict__ S) {
  const int i = blockIdx.x, bh = blockIdx.y, lane = threadIdx.x;
  __shared__ float qs[128];
  const size_t head = (size_t)bh * a.L * d;
  for (int c = lane; c < d; c += kWave) qs[c] = to_f32(Q[head + (size_t)i * d + c]);
  __syncthreads();
  const RowRuns rr = a.runs[i];
  float* out = S + (size_t)bh * a.nnz + a.row_ptr[i];
  const int64_t r0 = a.row_ptr[i];   // out's position in the head
#pragma unroll
  for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
    const Run q = rr.r[r];
    for (int k = lane; k < q.count; k += kWave) {
      const int j = dbg::idx(q.start + q.stride * k, a.L, dbg::kKey);
      out[dbg::rel(q.prefix + k, r0, a.nnz, dbg::kValue)] =
          dot_row(qs, K + head + (size_t)j * d, d) * scale;
    }
  }
}

// COL: P holds the head's values in column-major order, value (i, j) at
// col_pos(cols[j], i).
template <typename T, typename OutT, bool COL>
__global__ __launch_bounds__(kWave) void k_rspmm_rows(DevAcsr a, int d, const float* __restrict__ P,
                                                      const T* __restrict__ V,
                                                      OutT* __restrict__ O) {
  const int i = blockIdx.x, bh = blockIdx.y, lane = threadIdx.x;
  const size_t head = (size_t)bh * a.L * d;
  const float* p = P + (size_t)bh * a.nnz + (COL ? 0 : a.row_ptr[i]);
  const int64_t r0 = COL ? 0 : a.row_ptr[i];   // p's position in the head
  const RowRuns rr = a.runs[i];
  const bool two = d > kWave;
  float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
  for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
    const Run q = rr.r[r];
#pragma unroll 4
    for (int k = 0; k < q.count; ++k) {
      const int j = dbg::idx(q.start + q.stride * k, a.L, dbg::kKey);
      const float pk = COL ? p[dbg::idx((int64_t)col_pos(a.cols[j], i), a.nnz, dbg::kColPos)]
                           : p[dbg::rel(q.prefix + k, r0, a.nnz, dbg::kValue)];
      const T* v = V + head + (size_t)j * d;
      acc0 = fmaf(pk, to_f32(v[lane]), acc0);
      if (two) acc1 = fmaf(pk, to_f32(v[lane + kWave]), acc1);
    }
  }
  OutT* o = O + head + (size_t)i * d;
  store(o + lane, acc0);
  if (two) store(o + lane + kWave, acc1);
}

// Online softmax (running max m, running sum l) over the row's keys, 64 keys
// per step; fp32 throughout.
template <typename T, typename OutT>
__global__ __launch_bounds__(kWave) void k_fused_rows(DevAcsr a, int d, const T* __restrict__ Q,
                                                      const T* __restrict__ K,
                                                      const T* __restrict__ V, float scale,
                                                      OutT* __restrict__ O) {
  const int i = blockIdx.x, bh = blockIdx.y, lane = threadIdx.x;
  __shared__ float qs[128];
  __shared__ float ps[kWave];
  __shared__ int js[kWave];
  const size_t head = (size_t)bh * a.L * d;
  for (int c = lane; c < d; c += kWave) qs[c] = to_f32(Q[head + (size_t)i * d + c]);
  __syncthreads();
  const RowRuns rr = a.runs[i];
  const int n = a.row_ptr[i + 1] - a.row_ptr[i];
  const bool two = d > kWave;
  float m = -INFINITY, l = 0.f, acc0 = 0.f, acc1 = 0.f;
  for (int k0 = 0; k0 < n; k0 += kWave) {
    const int k = k0 + lane;
    const bool valid = k < n;
    int j = 0;
    float s = -INFINITY;
    if (valid) {
      j = dbg::idx(col_of(rr, k), a.L, dbg::kKey);
      s = dot_row(qs, K + head + (size_t)j * d, d) * scale;
    }
    const float mn = fmaxf(m, wave_max(s));      // finite: lane 0 is valid
    const float alpha = expf(m - mn);            // 0 on the first step (m = -inf)
    const float p = valid ? expf(s - mn) : 0.f;
    l = l * alpha + wave_sum(p);
    acc0 *= alpha;
    acc1 *= alpha;
    ps[lane] = p;
    js[lane] = j;
    __syncthreads();
    const int cnt = min(kWave, n - k0);
    for (int t = 0; t < cnt; ++t) {
      const float pt = ps[t];
      const T* v = V + head + (size_t)js[t] * d;
      acc0 = fmaf(pt, to_f32(v[lane]), acc0);
      if (two) acc1 = fmaf(pt, to_f32(v[lane + kWave]), acc1);
    }
    __syncthreads();
    m = mn;
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  OutT* o = O + head + (size_t)i * d;
  store(o + lane, acc0 * inv);
  if (two) store(o + lane + kWave, acc1 * inv);
}

#ifdef SPLAT_DEBUG_BOUNDS
// One index check on the device (the checked build's own test): out = the
// checked index.
__global__ void k_bounds_probe(int kind, int index, int n, int* out) {
  *out = dbg::idx(index, n, (dbg::Kind)kind);
}
#endif

}  // namespace

hipError_t bounds_collect_rows(uint32_t* bits, bool clear) { return dbg::collect(bits, clear); }

hipError_t bounds_probe(int kind, int index, int n, int* result) {
#ifndef SPLAT_DEBUG_BOUNDS
  (void)kind;
  (void)index;
  (void)n;
  (void)result;
  return hipErrorNotSupported;
#else
  int* d = nullptr;
  hipError_t e = hipMalloc(&d, sizeof(int));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_bounds_probe, dim3(1), dim3(1), 0, 0, kind, index, n, d);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipMemcpy(result, d, sizeof(int), hipMemcpyDeviceToHost);
  const hipError_t f = hipFree(d);
  return e != hipSuccess ? e : f;
#endif
}

hipError_t launch_rsddmm_rows(const DevAcsr& a, int dtype, int BH, int d, const void* Q,
                              const void* K, float scale, float* S, hipStream_t st) {
  dim3 grid(a.L, BH);
  if (dtype == 0)
    hipLaunchKernelGGL(k_rsddmm_rows<float>, grid, dim3(kWave), 0, st, a, d, (const float*)Q,
                       (const float*)K, scale, S);
  else
    hipLaunchKernelGGL(k_rsddmm_rows<__bf16>, grid, dim3(kWave), 0, st, a, d, (const __bf16*)Q,
                       (const __bf16*)K, scale, S);
  return hipGetLastError();
}

template <typename T, bool COL>
static hipError_t rspmm_t(const DevAcsr& a, int BH, int d, const float* P, const void* V, void* O,
                          int out_dtype, hipStream_t st) {
  dim3 grid(a.L, BH);
  if (out_dtype == 0)
    hipLaunchKernelGGL((k_rspmm_rows<T, float, COL>), grid, dim3(kWave), 0, st, a, d, P,
                       (const T*)V, (float*)O);
  else
    hipLaunchKernelGGL((k_rspmm_rows<T, __bf16, COL>), grid, dim3(kWave), 0, st, a, d, P,
                       (const T*)V, (__bf16*)O);
  return hipGetLastError();
}

hipError_t launch_rspmm_rows(const DevAcsr& a, int dtype, int BH, int d, const float* P,
                             const void* V, void* O, int out_dtype, bool colmajor, hipStream_t st) {
  if (colmajor)
    return dtype == 0 ? rspmm_t<float, true>(a, BH, d, P, V, O, out_dtype, st)
                      : rspmm_t<__bf16, true>(a, BH, d, P, V, O, out_dtype, st);
  return dtype == 0 ? rspmm_t<float, false>(a, BH, d, P, V, O, out_dtype, st)
                    : rspmm_t<__bf16, false>(a, BH, d, P, V, O, out_dtype, st);
}

template <typename T>
static hipError_t fused_t(const DevAcsr& a, int BH, int d, const void* Q, const void* K,
                          const void* V, float scale, void* O, int out_dtype, hipStream_t st) {
  dim3 grid(a.L, BH);
  if (out_dtype == 0)
    hipLaunchKernelGGL((k_fused_rows<T, float>), grid, dim3(kWave), 0, st, a, d, (const T*)Q,
                       (const T*)K, (const T*)V, scale, (float*)O);
  else
    hipLaunchKernelGGL((k_fused_rows<T, __bf16>), grid, dim3(kWave), 0, st, a, d, (const T*)Q,
                       (const T*)K, (const T*)V, scale, (__bf16*)O);
  return hipGetLastError();
}

hipError_t launch_fused_rows(const DevAcsr& a, int dtype, int BH, int d, const void* Q,
                             const void* K, const void* V, float scale, void* O, int out_dtype,
                             hipStream_t st) {
  return dtype == 0 ? fused_t<float>(a, BH, d, Q, K, V, scale, O, out_dtype, st)
                    : fused_t<__bf16>(a, BH, d, Q, K, V, scale, O, out_dtype, st);
}

}  // namespace splat
