// kernels_mfma.hip -- matrix-core (MFMA) kernels over the tile plan, bf16.
//
// Fused forward: O = softmax_nz(scale * M (x) Q K^T) V (Equation 1 with the
// softmax over each row's non-zeros), one workgroup per (row group, batch*head),
// 4 wavefronts x 32 query rows.  For every planned key tile of its group:
//
//   1. K and V tiles [64 keys][d] -> LDS, double-buffered: the next tile's
//      global loads are issued before the current tile is computed
//   2. S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (Q^T stays in registers); in this
//      orientation each lane holds 32 scores of ONE query, so the row max and
//      row sum need one exchange with lane ^ 32 only
//   3. per wavefront (32 rows) the plan marks the tile EMPTY (skipped), FULL
//      or PARTIAL; on PARTIAL tiles the scores outside each row's affine
//      runs are set to -inf from the row's precomputed 64-bit tile mask
//   4. online softmax in the log2 domain: p = exp2(s * scale*log2(e) - m);
//      the running max m is only raised when a score exceeds it by more
//      than 2^8 (so p <= 256 and O is rescaled rarely)
//   5. O^T += V^T P^T on the same MFMA, P^T taken straight from the score
//      registers (rounded to bf16), V^T gathered by LDS transpose reads in
//      the key order the score registers imply
//
// At the end O = O^T / (row sum), written in the requested dtype.
#include <hip/hip_runtime.h>
#include <math.h>

#include "launch.hpp"

namespace splat {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

constexpr bf16x2_t kOnes2 = {(__bf16)1.f, (__bf16)1.f};

constexpr int kThreads = 256;           // 4 waves
constexpr float kRescaleThreshold = 8.f; // log2 units

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

template <int D, typename OutT>
__global__ __launch_bounds__(kThreads, D == 64 ? 4 : 1) void k_fused_mfma(DevAcsr a, int BH,
                                                            const __bf16* __restrict__ Q,
                                                            const __bf16* __restrict__ K,
                                                            const __bf16* __restrict__ V, float sl2,
                                                            OutT* __restrict__ O) {
  constexpr int BN = kBN;
  constexpr int P = D + 8;        // K and V tile row pitch (elements): 16-byte aligned rows
  constexpr int CPR = D / 8;      // 16-byte chunks per K/V row
  constexpr int CPT = BN * CPR / kThreads;  // chunks per thread per tile
  constexpr int NKS = D / 16;     // k-steps of the QK^T product
  constexpr int NDB = D / 32;     // 32-wide feature blocks of O
  static_assert(CPT * kThreads == BN * CPR, "tile chunks must divide evenly");
  __shared__ __attribute__((aligned(16))) __bf16 sK[2][BN * P];
  __shared__ __attribute__((aligned(16))) __bf16 sV[2][BN * P];

  const int g = blockIdx.x / BH;
  const int bh = blockIdx.x - g * BH;
  const Group grp = a.groups[g];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int qi = lane & 31, h = lane >> 5;
  const int m = wave * 32 + qi;
  const bool row_valid = m < grp.nrows;
  const int row = row_valid ? a.rows[grp.row_off + m] : 0;
  const size_t head = (size_t)bh * a.L * D;
  const __bf16* Kh = K + head;
  const __bf16* Vh = V + head;

  // Q^T operand: lane holds Q[row][16*ks + 8*h .. +7]
  bf16x8_t qf[NKS];
  {
    const __bf16* qrow = Q + head + (size_t)row * D;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      if (row_valid) {
        qf[ks] = *(const bf16x8_t*)(qrow + ks * 16 + h * 8);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[ks][e] = (__bf16)0.f;
      }
    }
  }
  // V^T operand by LDS transpose reads: within each 16-lane group, lane i
  // addresses row k0 + i/4, features d0 + 4*(i%4) .. +3 and receives
  // V[k0 + 0..3][d0 + i]; k0 = 4*h, d0 = 16 * (lane/16 % 2)
  const int voff = (4 * h + ((lane & 15) >> 2)) * P + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int koff = qi * P + h * 8;

  f32x16_t oacc[NDB];
#pragma unroll
  for (int b = 0; b < NDB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[b][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // K/V tile staging: global -> registers (issued one tile ahead) -> LDS
  uint4 pk[CPT], pv[CPT];
  auto gload = [&](const Tile& tl) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + i * kThreads;
      const int u = c / CPR, dc = (c % CPR) * 8;
      pk[i] = make_uint4(0u, 0u, 0u, 0u);
      pv[i] = pk[i];
      if (u < tl.nk) {
        const size_t off = (size_t)(tl.kb + tl.ks * u) * D + dc;
        pk[i] = *(const uint4*)(Kh + off);
        pv[i] = *(const uint4*)(Vh + off);
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + i * kThreads;
      const int u = c / CPR, dc = (c % CPR) * 8;
      *(uint4*)(&sK[buf][u * P + dc]) = pk[i];
      *(uint4*)(&sV[buf][u * P + dc]) = pv[i];
    }
  };

  if (grp.tile_begin < grp.tile_end) {
    gload(a.tiles[grp.tile_begin]);
    sstore(0);
  }
  __syncthreads();

  for (int t = grp.tile_begin; t < grp.tile_end; ++t) {
    const int buf = (t - grp.tile_begin) & 1;
    const Tile tl = a.tiles[t];
    // this wavefront's 32 rows: no key in the tile / some (precomputed
    // per-row masks) / every key
    const int wst = (tl.flags >> (kWaveShift + 2 * wave)) & 3;
    uint64_t bits = ~0ull;
    if (wst == kWavePartial) bits = a.masks[(size_t)tl.mask_block * kBM + m] >> (4 * h);
    const bool has_next = t + 1 < grp.tile_end;
    if (has_next) gload(a.tiles[t + 1]);
    if (wst != kWaveEmpty) {
      const __bf16* cK = sK[buf];
      const __bf16* cV = sV[buf];

      // S^T[key][query] for the tile's two 32-key blocks
      f32x16_t sacc[2];
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[kb2][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const bf16x8_t ka = *(const bf16x8_t*)(cK + kb2 * 32 * P + koff + ks * 16);
          sacc[kb2] = mfma32(ka, qf[ks], sacc[kb2]);
        }
      }
      // sacc[kb2][r] is the score of key u = 32*kb2 + 8*(r/4) + 4*h + r%4
      if (wst == kWavePartial) {
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int u = 32 * kb2 + 8 * (r >> 2) + (r & 3);
            if (!((bits >> u) & 1ull)) sacc[kb2][r] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb2][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx * sl2);
      if (__any(m_new > m_run + kRescaleThreshold)) {
        const float alpha = (m_new == -INFINITY) ? 1.f : exp2_hw(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int b = 0; b < NDB; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[b][r] *= alpha;
      }
      const float neg_m = (m_run == -INFINITY) ? 0.f : -m_run;
      bf16x8_t pf[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pf[j][e] = (__bf16)exp2_hw(fmaf(sacc[j >> 1][(j & 1) * 8 + e], sl2, neg_m));
        // row sum of the bf16-rounded p, two at a time
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const bf16x2_t pair = {pf[j][e], pf[j][e + 1]};
          l_run = __builtin_amdgcn_fdot2_f32_bf16(pair, kOnes2, l_run, false);
        }
      }
      // O^T[d][query] += V^T[d][key] P^T[key][query]; k-step j, element e of lane
      // half h is key 16*j + 8*(e/4) + 4*h + e%4
#pragma unroll
      for (int b = 0; b < NDB; ++b) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const __bf16* vp = cV + voff + 16 * j * P + 32 * b;
          const bf16x4_t lo = tr16(vp);
          const bf16x4_t hi = tr16(vp + 8 * P);
          const bf16x8_t va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          oacc[b] = mfma32(va, pf[j], oacc[b]);
        }
      }
    }
    if (has_next) sstore(buf ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (row_valid) {
    OutT* orow = O + head + (size_t)row * D;
#pragma unroll
    for (int b = 0; b < NDB; ++b)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int d0 = b * 32 + rg * 8 + 4 * h;
        store4<OutT>(orow + d0, oacc[b][4 * rg] * inv, oacc[b][4 * rg + 1] * inv,
                     oacc[b][4 * rg + 2] * inv, oacc[b][4 * rg + 3] * inv);
      }
  }
}

template <int D>
hipError_t fused_d(const DevAcsr& a, int BH, const void* Q, const void* K, const void* V,
                   float sl2, void* O, int out_dtype, hipStream_t st) {
  const dim3 grid(a.n_groups * BH), block(kThreads);
  if (out_dtype == 0)
    hipLaunchKernelGGL((k_fused_mfma<D, float>), grid, block, 0, st, a, BH, (const __bf16*)Q,
                       (const __bf16*)K, (const __bf16*)V, sl2, (float*)O);
  else
    hipLaunchKernelGGL((k_fused_mfma<D, __bf16>), grid, block, 0, st, a, BH, (const __bf16*)Q,
                       (const __bf16*)K, (const __bf16*)V, sl2, (__bf16*)O);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fused_mfma(const DevAcsr& a, int BH, int d, const void* Q, const void* K,
                             const void* V, float scale, void* O, int out_dtype, hipStream_t st) {
  const float sl2 = (float)((double)scale * 1.4426950408889634074);  // scale * log2(e)
  if (d == 64) return fused_d<64>(a, BH, Q, K, V, sl2, O, out_dtype, st);
  return fused_d<128>(a, BH, Q, K, V, sl2, O, out_dtype, st);
}

}  // namespace splat
