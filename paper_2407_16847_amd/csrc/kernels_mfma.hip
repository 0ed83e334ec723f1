// kernels_mfma.hip -- matrix-core (MFMA) kernels over the tile plan, bf16.
//
// Fused forward: O = softmax_nz(scale * M (x) Q K^T) V (Equation 1 with the
// softmax over each row's non-zeros), one workgroup per (row group, batch*head),
// 4 wavefronts x 32 query rows.  For every planned key tile of its group:
//
//   1. K and V tiles [64 keys][d] and the rows' tile masks travel from global
//      memory straight into a two-slot LDS ring (global_load_lds from a scalar
//      tile base plus per-lane offsets, no staging registers), the next tile
//      issued while this one is computed; rows are stored unpadded with their
//      16-byte chunks XOR-swizzled so the MFMA operand reads below are free of
//      bank conflicts.  With 34 KiB of LDS and at most 128 VGPRs (d = 64),
//      four workgroups share a CU: four wavefronts per SIMD to hide latency
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
//      registers (rounded toward zero to bf16 by one v_perm_b32 per pair; the
//      row sum adds the same rounded values), V^T gathered by LDS transpose
//      reads in the key order the score registers imply
//
// At the end O = O^T / (row sum), written in the requested dtype.
#include <hip/hip_runtime.h>
#include <math.h>

#include "launch.hpp"
#include "mfma_util.hpp"

namespace splat {
namespace {

using namespace mfma;

constexpr int kThreads = 256;           // 4 waves
constexpr float kRescaleThreshold = 8.f; // log2 units

template <int D>
struct Geo {
  static constexpr int RB = 2 * D;                      // bytes per K/V row in LDS
  static constexpr int CPR = RB / 16;                   // 16-byte chunks per row
  static constexpr int TB = kBN * RB;                   // bytes of a K (or V) tile
  static constexpr int NBW = TB / kDmaBlock / 4;        // loads per wavefront per tile
  static constexpr int RPB = kDmaBlock / RB;            // rows per load
  static constexpr int SLOT = 2 * TB + kBM * 8;         // K tile, V tile, row masks
  static constexpr int NSLOT = 2;                       // ring depth (the loop waits for
                                                        // all loads at each barrier)
  static constexpr int LDS = NSLOT * SLOT;
  static constexpr int NKS = D / 16, NDB = D / 32;
};


// Issue this wavefront's share of one tile's global->LDS loads into a slot.
// Keys past the tile's end re-read its last key (finite data the masks
// exclude).  The 16 lanes of the mask load bring the wavefront's 32 row masks.
template <int D>
__device__ __forceinline__ void issue_tile(char* slot, const Tile tl, const __bf16* Kh,
                                           const __bf16* Vh, const uint64_t* masks, int wave,
                                           int lane) {
  using G = Geo<D>;
  const int last = tl.nk - 1;
  // uniform tile bases (scalar registers) + 32-bit per-lane byte offsets
  const char* kbase = (const char*)(Kh + (size_t)tl.kb * D);
  const char* vbase = (const char*)(Vh + (size_t)tl.kb * D);
#pragma unroll
  for (int k = 0; k < G::NBW; ++k) {
    const int bk = wave + 4 * k;
    const int r = bk * G::RPB + lane / G::CPR;
    const int pos = lane % G::CPR;
    const unsigned row = (unsigned)(tl.ks * min(r, last)) * (2u * D);
    dma16(kbase + row + 16u * (pos ^ swz_k(r)), slot + bk * kDmaBlock);
    dma16(vbase + row + 16u * (pos ^ swz_v(r)), slot + G::TB + bk * kDmaBlock);
  }
  // row masks only for tiles with a PARTIAL wavefront (the others never read
  // them; the ring barrier waits for every outstanding load, so the count of
  // loads issued per tile may vary)
  if (tl.mask_block >= 0) {
    const uint64_t* mrow = masks + (size_t)tl.mask_block * kBM + wave * 32 + 2 * lane;
    if (lane < 16) dma16(mrow, slot + 2 * G::TB + wave * 256);
  }
}

// p = exp2(s * sl2 - m) for this lane's 32 scores, rounded toward zero to bf16
// into the P^T operand (key order of the score registers); returns the sum
// of the rounded values.
__device__ __forceinline__ float tile_exp(const f32x16_t* s, float sl2, float neg_m,
                                          bf16x8_t* pf) {
  float l0 = 0.f, l1 = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float e8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) e8[e] = exp2_hw(fmaf(s[j >> 1][(j & 1) * 8 + e], sl2, neg_m));
    bf16x2_t p2[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) p2[e] = pack_bf16_rz(e8[2 * e], e8[2 * e + 1]);
    pf[j] = __builtin_shufflevector(__builtin_shufflevector(p2[0], p2[1], 0, 1, 2, 3),
                                    __builtin_shufflevector(p2[2], p2[3], 0, 1, 2, 3), 0, 1, 2, 3,
                                    4, 5, 6, 7);
    l0 = __builtin_amdgcn_fdot2_f32_bf16(p2[0], kOnes2, l0, false);
    l1 = __builtin_amdgcn_fdot2_f32_bf16(p2[1], kOnes2, l1, false);
    l0 = __builtin_amdgcn_fdot2_f32_bf16(p2[2], kOnes2, l0, false);
    l1 = __builtin_amdgcn_fdot2_f32_bf16(p2[3], kOnes2, l1, false);
  }
  return l0 + l1;
}

// Online-softmax step of one tile for this lane's row: optional mask, tile
// max, lazy update of the running max (only when a score exceeds it by more
// than 2^kRescaleThreshold), p = exp2(s * scale*log2(e) - m) into the P^T
// operand and the running sum of the rounded p.  alpha is the factor the
// output accumulator must be scaled by before this tile's P V is added; the
// return value says whether any lane of the wavefront needs it.
template <bool MASKED>
__device__ __forceinline__ bool tile_softmax(f32x16_t* s, uint64_t mk, int h, float sl2,
                                             float& m_run, float& l_run, float& alpha,
                                             bf16x8_t* pf) {
  if (MASKED) {
    const uint64_t bits = mk >> (4 * h);
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
      const unsigned word = (unsigned)(bits >> (32 * kb2));
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb2][r] = keep_if_bit(s[kb2][r], word, 8 * (r >> 2) + (r & 3));
    }
  }
  float mx0 = -INFINITY, mx1 = -INFINITY;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    mx0 = fmaxf(mx0, s[0][r]);
    mx1 = fmaxf(mx1, s[1][r]);
  }
  float mx = fmaxf(mx0, mx1);
  mx = fmaxf(mx, lane_xor32(mx));
  const float m_new = fmaxf(m_run, mx * sl2);
  const bool need = m_new > m_run + kRescaleThreshold;
  alpha = need ? exp2_hw(m_run - m_new) : 1.f;   // exp2(-inf) = 0 on the first tile
  m_run = need ? m_new : m_run;
  l_run *= alpha;
  const float neg_m = (m_run == -INFINITY) ? 0.f : -m_run;
  l_run += tile_exp(s, sl2, neg_m, pf);
  return __any(need);
}

// The plan arrays are kernel arguments of their own, const and __restrict__,
// so their (wavefront-uniform) reads are scalar loads, independent of the
// vector-memory counter that tracks the global->LDS loads.
template <int D, typename OutT>
__global__ __launch_bounds__(kThreads, D == 64 ? 4 : 2) void k_fused_mfma(
    const Group* __restrict__ groups, const int32_t* __restrict__ rows,
    const Tile* __restrict__ tiles, const uint64_t* __restrict__ masks, int L, int BH,
    const __bf16* __restrict__ Q, const __bf16* K, const __bf16* V, float sl2,
    OutT* __restrict__ O) {
  using G = Geo<D>;
  constexpr int NKS = G::NKS, NDB = G::NDB, NSLOT = G::NSLOT, RB = G::RB;
  extern __shared__ __attribute__((aligned(16))) char smem[];

  const int g = blockIdx.x / BH;
  const int bh = blockIdx.x - g * BH;
  const Group grp = groups[g];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int qi = lane & 31, h = lane >> 5;
  const int m = wave * 32 + qi;
  const bool row_valid = m < grp.nrows;
  const int row = row_valid ? rows[grp.row_off + m] : 0;
  const size_t head = (size_t)bh * L * D;
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
  // K operand of key row r = 32*kb2 + qi, chunk 2*ks + h (swizzle depends on r % 16)
  int koff[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    koff[ks] = qi * RB + 16 * ((((2 * ks + h) & 7) ^ swz_k(qi)) | ((2 * ks + h) & ~7));
  // V^T operand by LDS transpose reads
  int voff[NDB];
  v_operand_offsets<D>(lane, voff);

  f32x16_t oacc[NDB];
#pragma unroll
  for (int b = 0; b < NDB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[b][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int tb = grp.tile_begin, nt = grp.tile_end - grp.tile_begin;
  if (nt > 0) {
    // prologue: the first NSLOT-1 tiles
#pragma unroll
    for (int sl = 0; sl < NSLOT - 1; ++sl)
      issue_tile<D>(smem + sl * G::SLOT, tiles[tb + min(sl, nt - 1)], Kh, Vh, masks, wave, lane);
    // descriptors are read one iteration before they are needed
    Tile next_issue = tiles[tb + min(NSLOT - 1, nt - 1)];
    int next_flags = tiles[tb].flags;
    ring_sync<0>();

    for (int i = 0; i < nt; ++i) {
      char* cur = smem + (i % NSLOT) * G::SLOT;
      const Tile to_issue = next_issue;
      const int flags = next_flags;
      next_issue = tiles[tb + min(i + NSLOT, nt - 1)];
      next_flags = tiles[tb + min(i + 1, nt - 1)].flags;
      issue_tile<D>(smem + ((i + NSLOT - 1) % NSLOT) * G::SLOT, to_issue, Kh, Vh, masks, wave,
                    lane);
      const int wst = (flags >> (kWaveShift + 2 * wave)) & 3;
      if (wst != kWaveEmpty) {
        const __bf16* cK = (const __bf16*)cur;
        const __bf16* cV = (const __bf16*)(cur + G::TB);
        // S^T[key][query]: all K operands read, then the products
        auto scores = [&](f32x16_t* sacc) {
          bf16x8_t ka[2][NKS];
#pragma unroll
          for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks)
              ka[kb2][ks] = *(const bf16x8_t*)((const char*)cK + kb2 * 32 * RB + koff[ks]);
#pragma unroll
          for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
            for (int r = 0; r < 16; ++r) sacc[kb2][r] = 0.f;
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) sacc[kb2] = mfma32(ka[kb2][ks], qf[ks], sacc[kb2]);
          }
        };
        f32x16_t sacc[2];
        scores(sacc);
        float alpha;
        bf16x8_t pf[4];
        bool need;
        if (wst == kWavePartial) {
          const uint64_t mk = *(const uint64_t*)(cur + 2 * G::TB + m * 8);
          need = tile_softmax<true>(sacc, mk, h, sl2, m_run, l_run, alpha, pf);
        } else {
          need = tile_softmax<false>(sacc, 0, h, sl2, m_run, l_run, alpha, pf);
        }
        if (need) {
#pragma unroll
          for (int b = 0; b < NDB; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[b][r] *= alpha;
        }
        // O^T[d][query] += V^T[d][key] P^T[key][query]; k-step j, element e of
        // lane half h is key 16*j + 8*(e/4) + 4*h + e%4
        bf16x8_t va[NDB][4];
        read_v_operands<D>(lds_addr(cV), voff, va);
#pragma unroll
        for (int b = 0; b < NDB; ++b)
#pragma unroll
          for (int j = 0; j < 4; ++j) oacc[b] = mfma32(va[b][j], pf[j], oacc[b]);
      }
      // the next tile's loads (issued at the top of this iteration) have
      // landed, and every wavefront is done with this slot
      ring_sync<0>();
    }
  }

  const float l_tot = l_run + lane_xor32(l_run);
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

template <int D, typename OutT>
hipError_t fused_launch(const DevAcsr& a, int BH, const void* Q, const void* K, const void* V,
                        float sl2, void* O, hipStream_t st) {
  constexpr int lds = Geo<D>::LDS;
  static bool attr_set = false;   // the LDS size attribute is per kernel, set once
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute((const void*)k_fused_mfma<D, OutT>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((k_fused_mfma<D, OutT>), dim3(a.n_groups * BH), dim3(kThreads), lds, st,
                     a.groups, a.rows, a.tiles, a.masks, a.L, BH, (const __bf16*)Q,
                     (const __bf16*)K, (const __bf16*)V, sl2, (OutT*)O);
  return hipGetLastError();
}

template <int D>
hipError_t fused_d(const DevAcsr& a, int BH, const void* Q, const void* K, const void* V,
                   float sl2, void* O, int out_dtype, hipStream_t st) {
  return out_dtype == 0 ? fused_launch<D, float>(a, BH, Q, K, V, sl2, O, st)
                        : fused_launch<D, __bf16>(a, BH, Q, K, V, sl2, O, st);
}

}  // namespace

hipError_t launch_fused_mfma(const DevAcsr& a, int BH, int d, const void* Q, const void* K,
                             const void* V, float scale, void* O, int out_dtype, hipStream_t st) {
  const float sl2 = (float)((double)scale * 1.4426950408889634074);  // scale * log2(e)
  if (d == 64) return fused_d<64>(a, BH, Q, K, V, sl2, O, out_dtype, st);
  return fused_d<128>(a, BH, Q, K, V, sl2, O, out_dtype, st);
}

}  // namespace splat
