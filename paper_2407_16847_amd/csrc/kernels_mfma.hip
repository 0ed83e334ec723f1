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
//   2. S^T = K Q^T on v_mfma_f32_32x32x16_bf16, with Q^T held in registers and
//      pre-scaled by scale*log2(e) (rounded to bf16), so the products are the
//      scores in the log2 domain, t = s * scale*log2(e); in this orientation
//      each lane holds 32 scores of ONE query, so row reductions need one
//      exchange with lane ^ 32 only
//   3. per wavefront (32 rows) the plan marks the tile EMPTY (skipped), FULL
//      or PARTIAL; on PARTIAL tiles the scores outside each row's affine
//      runs are set to -inf from the row's precomputed 64-bit tile mask
//   4. online softmax against a per-row integer reference m: p = exp2(t - m).
//      The fast pass computes exp2(t), rounds it to nearest even bf16 and,
//      only when some row has m > 0, applies 2^-m to each bf16 pair with one
//      saturating 16-bit subtract from the exponent fields -- no per-score
//      max, offset or multiply.  m stays 0 while a row's scores stay within
//      2^6 of it.  A slow pass redoes the tile from the exact row max when a
//      row's tile sum exceeds 2^12 (the reference then rises to the next
//      integer above the max and O is rescaled by a power of two), when a
//      row has nothing accumulated yet and its sum is tiny, or when the
//      reference lies outside [0, 100]
//   5. O^T += V^T P^T on the same MFMA, P^T taken straight from the score
//      registers, V^T gathered by LDS transpose reads in the key order the
//      score registers imply; the row sum adds the same rounded p, so a row
//      with one key returns that key's V row exactly
//
// At the end O = O^T / (row sum), written in the requested dtype through LDS
// as whole rows (16-byte non-temporal stores along each row).
#include <hip/hip_runtime.h>
#include <math.h>

#include "bounds.hpp"
#include "launch.hpp"
#include "mfma_util.hpp"

namespace splat {
namespace {

using namespace mfma;

constexpr int kThreads = 256;           // 4 waves
constexpr float kSumLimit = 4096.f;   // largest tile row sum the fast pass accepts
constexpr float kRefMax = 100.f;      // references the fast pass can apply, [0, kRefMax]
constexpr float kRefLow = -100.f;     // row maxima below this keep their own reference
constexpr float kRefSlack = 6.f;      // a row keeps its reference while its max stays within
                                      // this of it (p <= 2^6, a 64-key tile sum <= 2^12)
constexpr float kFirstMin = 0x1p-60f; // smallest first tile sum the fast pass accepts

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
                                           const __bf16* Vh, const uint64_t* masks, int L,
                                           int wave, int lane) {
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
    // one 32-bit lane offset from the scalar base: the load adds them itself
    // (no 64-bit vector address arithmetic)
    const int key = dbg::idx(tl.kb + tl.ks * min(r, last), L, dbg::kKey);
    const unsigned row = (unsigned)(key - tl.kb) * (2u * D);
    const unsigned ko = row + 16u * (pos ^ swz_k(r)), vo = row + 16u * (pos ^ swz_v(r));
    dma16(kbase + ko, slot + bk * kDmaBlock);
    dma16(vbase + vo, slot + G::TB + bk * kDmaBlock);
  }
  // row masks only for tiles with a PARTIAL wavefront (the others never read
  // them; the ring barrier waits for every outstanding load, so the count of
  // loads issued per tile may vary)
  if (tl.mask_block >= 0) {
    const uint64_t* mrow = masks + (size_t)tl.mask_block * kBM + wave * 32 + 2 * lane;
    if (lane < 16) dma16(mrow, slot + 2 * G::TB + wave * 256);
  }
}

// One tile's exponentials for this lane's 32 scores t (s * scale*log2(e),
// from the pre-scaled Q): p = exp2(t - m) with REF, else p = exp2(t) (the fast
// pass, whose factor 2^-m is applied afterwards by scale_pairs, only when some
// row of the wavefront has m > 0).  Each p goes to the P^T operand rounded to
// nearest even bf16 (one v_cvt_pk_bf16_f32 per pair); returns the sum of the
// rounded p (v_dot2c_f32_bf16 against ones, fp32 accumulation).
template <bool REF>
__device__ __forceinline__ float tile_exp(const f32x16_t* s, float m, bf16x8_t* pf) {
  float l0 = 0.f, l1 = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float e8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float t = s[j >> 1][(j & 1) * 8 + e];
      e8[e] = exp2_hw(REF ? t - m : t);
    }
    // the row sum adds exactly the rounded values the MFMA multiplies; the
    // dot products take the packed pairs as scalars (taken back out of a
    // vector, the compiler merged the two sums into one)
    const unsigned u0 = pack_bf16_rn(e8[0], e8[1]), u1 = pack_bf16_rn(e8[2], e8[3]);
    const unsigned u2 = pack_bf16_rn(e8[4], e8[5]), u3 = pack_bf16_rn(e8[6], e8[7]);
    l0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u0), kOnes2, l0, false);
    l1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u1), kOnes2, l1, false);
    l0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u2), kOnes2, l0, false);
    l1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u3), kOnes2, l1, false);
    pf[j] = __builtin_bit_cast(bf16x8_t, u32x4_t{u0, u1, u2, u3});
  }
  return l0 + l1;
}

// p * 2^-m on the bf16 P^T operand: m subtracted from both exponent fields of
// each pair with unsigned saturation (msub = m*128 in each half), exact for
// normal results, flushing results below 2^-126 to zero.
__device__ __forceinline__ void scale_pairs(bf16x8_t* pf, unsigned msub) {
  typedef unsigned short u16x8_t __attribute__((ext_vector_type(8)));
  u16x8_t sub;
#pragma unroll
  for (int e = 0; e < 8; ++e) sub[e] = (unsigned short)((e & 1) ? msub >> 16 : msub);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    pf[j] = __builtin_bit_cast(bf16x8_t, __builtin_elementwise_sub_sat(
                                             __builtin_bit_cast(u16x8_t, pf[j]), sub));
}

// scores outside the row's affine runs in this tile set to -inf
__device__ __forceinline__ void mask_scores(f32x16_t* s, uint64_t mk, int h) {
  const uint64_t bits = mk >> (4 * h);
#pragma unroll
  for (int kb2 = 0; kb2 < 2; ++kb2) {
    const unsigned word = (unsigned)(bits >> (32 * kb2));
#pragma unroll
    for (int r = 0; r < 16; ++r) s[kb2][r] = keep_if_bit(s[kb2][r], word, 8 * (r >> 2) + (r & 3));
  }
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
  const int row = row_valid ? dbg::idx(rows[grp.row_off + m], L, dbg::kRow) : 0;
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
        const bf16x8_t q = *(const bf16x8_t*)(qrow + ks * 16 + h * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[ks][e] = (__bf16)((float)q[e] * sl2);
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
  // the row's reference m (an integer; p = exp2(t - m)), the running sum of p
  // and the reference as the fast pass applies it
  // (l_run holds this lane's half of the row's keys; acc says whether the
  // whole row has accumulated any weight, identical in both halves)
  float m_run = 0.f, l_run = 0.f;
  unsigned msub = 0u;
  float mscale = 1.f;
  bool fast_ok = true, acc = false;

  const int tb = grp.tile_begin, nt = grp.tile_end - grp.tile_begin;
  if (nt > 0) {
    // prologue: the first NSLOT-1 tiles
#pragma unroll
    for (int sl = 0; sl < NSLOT - 1; ++sl)
      issue_tile<D>(smem + sl * G::SLOT, tiles[tb + min(sl, nt - 1)], Kh, Vh, masks, L, wave,
                    lane);
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
      issue_tile<D>(smem + ((i + NSLOT - 1) % NSLOT) * G::SLOT, to_issue, Kh, Vh, masks, L, wave,
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
        uint64_t mk = ~0ull;
        if (wst == kWavePartial) {
          mk = *(const uint64_t*)(cur + 2 * G::TB + m * 8);
          mask_scores(sacc, mk, h);
        }
        bf16x8_t pf[4];
        float lt = tile_exp<false>(sacc, 0.f, pf);
        if (__any(msub != 0u)) {
          scale_pairs(pf, msub);
          lt *= mscale;   // 2^-m: the sum of the scaled pairs, exactly
        }
        float lrow = lt + lane_xor32(lt);
        // the slow pass takes the tile when, for some row, the fast pass
        // cannot apply the reference, exceeds kSumLimit, or gives the row's
        // first keys a total weight below kFirstMin (values that small may
        // be fp32 subnormals, with too few bits left for bf16)
        const bool redo = !fast_ok || !(lrow <= kSumLimit) ||
                          (mk != 0 && lrow < kFirstMin && !acc);
        if (__any(redo)) {
          float mx0 = -INFINITY, mx1 = -INFINITY;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            mx0 = fmaxf(mx0, sacc[0][r]);
            mx1 = fmaxf(mx1, sacc[1][r]);
          }
          float mx = fmaxf(mx0, mx1);
          mx = fmaxf(mx, lane_xor32(mx));
          // a row with nothing accumulated takes its reference from this
          // tile; otherwise the reference only rises, to the next integer
          // at or above the tile's max
          float m_new = m_run;
          if (!acc) {
            if (mx > -INFINITY) m_new = (mx < kRefLow || mx > kRefSlack) ? ceilf(mx) : 0.f;
          } else if (mx > m_run + kRefSlack) {
            m_new = ceilf(mx);
          }
          // a power of two, 1 if unchanged; a row with nothing accumulated
          // has nothing to rescale (and its reference may fall)
          const float alpha = acc ? exp2_hw(m_run - m_new) : 0.f;
          lt = tile_exp<true>(sacc, m_new, pf);
          lrow = lt + lane_xor32(lt);
          l_run *= alpha;
          m_run = m_new;
          fast_ok = m_run >= 0.f && m_run <= kRefMax;
          msub = fast_ok ? 0x00800080u * (unsigned)m_run : 0u;
          mscale = exp2_hw(-m_run);
#pragma unroll
          for (int b = 0; b < NDB; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[b][r] *= alpha;
        }
        l_run += lt;
        acc = acc || lrow > 0.f;
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
  // O leaves through LDS: each wavefront stages its 32 rows (rows padded by
  // 16 bytes; after the loop's last barrier no wavefront reads the ring), then
  // writes whole rows, 16 bytes per lane with consecutive lanes along a row,
  // as non-temporal stores: no partial lines, and nothing left dirty in L2.
  constexpr int SZ = (int)sizeof(OutT);
  constexpr int RS = D * SZ + 16;      // staged row stride, bytes
  constexpr int CPRO = D * SZ / 16;    // 16-byte chunks per output row
  static_assert(4 * 32 * RS <= G::LDS, "output staging fits in the ring");
  char* stage = smem + wave * 32 * RS;
#pragma unroll
  for (int b = 0; b < NDB; ++b)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int d0 = b * 32 + rg * 8 + 4 * h;
      store4<OutT>((OutT*)(stage + qi * RS + d0 * SZ), oacc[b][4 * rg] * inv,
                   oacc[b][4 * rg + 1] * inv, oacc[b][4 * rg + 2] * inv,
                   oacc[b][4 * rg + 3] * inv);
    }
  const int nrows_w = grp.nrows - wave * 32;   // valid rows of this wavefront
  char* ohead = (char*)(O + head);
#pragma unroll
  for (int k = 0; k < 32 * CPRO / 64; ++k) {
    const int idx = k * 64 + lane;
    const int r = idx / CPRO, c = idx % CPRO;
    const int orow = __shfl(row, r);           // lane r holds query row r of the wavefront
    const u32x4_t v = *(const u32x4_t*)(stage + r * RS + c * 16);
    if (r < nrows_w) store16_nt(ohead + (size_t)orow * (D * SZ) + c * 16, v);
  }
}

template <int D, typename OutT>
hipError_t allow_lds() {
  return hipFuncSetAttribute((const void*)k_fused_mfma<D, OutT>,
                             hipFuncAttributeMaxDynamicSharedMemorySize, Geo<D>::LDS);
}

template <int D, typename OutT>
hipError_t fused_launch(const DevAcsr& a, int BH, const void* Q, const void* K, const void* V,
                        float sl2, void* O, hipStream_t st) {
  constexpr int lds = Geo<D>::LDS;
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

hipError_t bounds_collect_mfma(uint32_t* bits, bool clear) { return dbg::collect(bits, clear); }

hipError_t prepare_fused_mfma() {
  hipError_t e = allow_lds<64, float>();
  if (e == hipSuccess) e = allow_lds<64, __bf16>();
  if (e == hipSuccess) e = allow_lds<128, float>();
  if (e == hipSuccess) e = allow_lds<128, __bf16>();
  return e;
}

hipError_t launch_fused_mfma(const DevAcsr& a, int BH, int d, const void* Q, const void* K,
                             const void* V, float scale, void* O, int out_dtype, hipStream_t st) {
  const float sl2 = (float)((double)scale * 1.4426950408889634074);  // scale * log2(e)
  if (d == 64) return fused_d<64>(a, BH, Q, K, V, sl2, O, out_dtype, st);
  return fused_d<128>(a, BH, Q, K, V, sl2, O, out_dtype, st);
}

}  // namespace splat
