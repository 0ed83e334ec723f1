// mfma_util.hpp -- device helpers shared by the matrix-core kernels: operand
// vector types, the bf16 32x32x16 MFMA, LDS transpose reads, global->LDS
// loads, lane exchange and the ring barrier.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace splat {
namespace mfma {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

constexpr bf16x2_t kOnes2 = {(__bf16)1.f, (__bf16)1.f};

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// LDS transpose read (ds_read_b64_tr_b16): within each group of 16 lanes, lane
// i receives element i%4 of the 8-byte chunks addressed by lanes i/4, 4 + i/4,
// 8 + i/4 and 12 + i/4 -- a 4 x 16 block of 16-bit values read transposed.
__device__ __forceinline__ bf16x4_t tr16(const __bf16* lds) {
  const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4_t*)(__attribute__((address_space(3))) __bf16*)(lds));
  return __builtin_bit_cast(bf16x4_t, v);
}

// value of lane l ^ 32: one v_permlane32_swap of x with itself leaves the low
// half's values in the first result and the high half's in the second
__device__ __forceinline__ float lane_xor32(float x) {
  const int xi = __builtin_bit_cast(int, x);
  const auto sw = __builtin_amdgcn_permlane32_swap(xi, xi, false, false);
  const int lane = __lane_id();
  return __builtin_bit_cast(float, lane < 32 ? sw[1] : sw[0]);
}

// The same transpose read issued as inline assembly: the compiler then does
// not treat it as a possible reader of the in-flight global->LDS loads (it
// would otherwise wait for all of them).  Its results are only valid after
// lds_wait() below.
__device__ __forceinline__ bf16x4_t tr16_async(unsigned lds_addr) {
  i16x4_t v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(lds_addr));
  return __builtin_bit_cast(bf16x4_t, v);
}
// ... with a constant byte offset folded into the instruction (no address add)
template <int OFF>
__device__ __forceinline__ bf16x4_t tr16_async_at(unsigned lds_addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  i16x4_t v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(lds_addr), "i"(OFF));
  return __builtin_bit_cast(bf16x4_t, v);
}

// Wait for every outstanding LDS read of this wavefront; the operands make the
// values read by tr16_async depend on the wait.
template <int NDB>
__device__ __forceinline__ void lds_wait(bf16x8_t (*va)[4]);
template <>
__device__ __forceinline__ void lds_wait<2>(bf16x8_t (*va)[4]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(va[0][0]), "+v"(va[0][1]), "+v"(va[0][2]), "+v"(va[0][3]), "+v"(va[1][0]),
                 "+v"(va[1][1]), "+v"(va[1][2]), "+v"(va[1][3]));
}
template <>
__device__ __forceinline__ void lds_wait<4>(bf16x8_t (*va)[4]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(va[0][0]), "+v"(va[0][1]), "+v"(va[0][2]), "+v"(va[0][3]), "+v"(va[1][0]),
                 "+v"(va[1][1]), "+v"(va[1][2]), "+v"(va[1][3]), "+v"(va[2][0]), "+v"(va[2][1]),
                 "+v"(va[2][2]), "+v"(va[2][3]), "+v"(va[3][0]), "+v"(va[3][1]), "+v"(va[3][2]),
                 "+v"(va[3][3]));
}

// 32-bit LDS address of a pointer into dynamic shared memory.
__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
}

template <typename OutT>
__device__ __forceinline__ void store4(OutT* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  *(float4*)p = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<__bf16>(__bf16* p, float a, float b, float c, float d) {
  bf16x4_t v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
  *(bf16x4_t*)p = v;
}

constexpr int kDmaBytes = 16;                 // bytes per lane of one global->LDS load
constexpr int kDmaBlock = 64 * kDmaBytes;     // bytes one wavefront load writes to LDS

// Chunk swizzles.  K rows are read 32 rows x one 16-byte chunk per
// instruction; V rows 4 rows x two chunks per 16 lanes (transpose reads).
__device__ __forceinline__ int swz_k(int r) { return ((r >> 1) & 7) ^ ((r & 1) << 2); }
__device__ __forceinline__ int swz_v(int r) { return (r & 3) << 1; }

__device__ __forceinline__ void dma16(const void* g, char* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, kDmaBytes, 0, 0);
}

// Wait until at most `pending` vector-memory ops (the global->LDS loads) of
// this wavefront are outstanding, then barrier.  The LDS/scalar counter is
// left alone: every LDS read before a ring barrier has its result consumed
// by then (the compiler waits before the first use, lds_wait() covers the
// transpose reads), and waiting on it here would also wait for the scalar
// loads of upcoming tile descriptors.  The empty asm statements keep the
// compiler from moving LDS accesses across the barrier.
template <int PENDING>
__device__ __forceinline__ void ring_sync() {
  static_assert(PENDING < 64, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((PENDING & 15) | ((PENDING >> 4) << 14) | (7 << 4) | (15 << 8));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// V^T operand of O^T += V^T P^T from a V tile in LDS (rows of 2*D bytes, 16-byte
// chunks placed by swz_v).  Within each 16-lane group, lane i addresses key
// row 4*h + i/4 (+ 16*j, + 8), features 32*b + 16*(lane/16 % 2) + 4*(i%4)
// .. +3, and receives V[4 rows][feature 32*b + lane%32]; k-step j, element e
// of lane half h is then key 16*j + 8*(e/4) + 4*h + e%4 of the tile.
template <int D>
__device__ __forceinline__ void v_operand_offsets(int lane, int (&voff)[D / 32]) {
  constexpr int RB = 2 * D;
  const int h = lane >> 5, i = lane & 15;
  const int rv = 4 * h + (i >> 2);
  const int cl = 2 * ((lane >> 4) & 1) + ((i & 3) >> 1);
#pragma unroll
  for (int b = 0; b < D / 32; ++b) voff[b] = rv * RB + 16 * ((4 * b + cl) ^ swz_v(rv)) + 8 * (i & 1);
}

template <int D, int J = 0>
__device__ __forceinline__ void read_v_block(unsigned vp, bf16x8_t (&vb)[4]) {
  constexpr int RB = 2 * D;
  if constexpr (J < 4) {
    vb[J] = __builtin_shufflevector(tr16_async_at<16 * J * RB>(vp),
                                    tr16_async_at<16 * J * RB + 8 * RB>(vp), 0, 1, 2, 3, 4, 5, 6, 7);
    read_v_block<D, J + 1>(vp, vb);
  }
}

template <int D>
__device__ __forceinline__ void read_v_operands(unsigned vbase, const int (&voff)[D / 32],
                                                bf16x8_t (*va)[4]) {
#pragma unroll
  for (int b = 0; b < D / 32; ++b) read_v_block<D>(vbase + voff[b], va[b]);
  lds_wait<D / 32>(va);
}

// Two fp32 values to a bf16 pair, rounded to nearest even (one
// v_cvt_pk_bf16_f32).
__device__ __forceinline__ unsigned pack_bf16_rn(float lo, float hi) {
  const bf16x2_t p = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(unsigned, p);
}

// 16-byte non-temporal store (streamed past the caches)
__device__ __forceinline__ void store16_nt(void* p, u32x4_t v) {
  __builtin_nontemporal_store(v, (u32x4_t*)p);
}

// x where bit u of `word` is set, -inf elsewhere (v_bfe_i32 + v_bfi_b32)
__device__ __forceinline__ float keep_if_bit(float x, unsigned word, int u) {
  const unsigned m = (unsigned)__builtin_amdgcn_sbfe((int)word, u, 1);
  return __builtin_bit_cast(float, (__builtin_bit_cast(unsigned, x) & m) | (0xff800000u & ~m));
}

}  // namespace mfma
}  // namespace splat
