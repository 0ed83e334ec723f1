// kernels_tiles.hip -- the unfused chain of Equation 1 for bf16 inputs, over the
// tile plan: R-SDDMM on the matrix cores, the row softmax with each row held
// in registers, and R-SpMM on the matrix cores.  S and P are fp32 in the
// ACSR value order (row i's values at row_ptr[i] .. row_ptr[i+1], ascending
// column).
//
// Position of a tile element in its row.  The tiles of a row group cover
// disjoint, ascending column intervals and every column of the group's rows
// lies in exactly one of them, so a row's values for tile t start right after
// its values for tiles 0 .. t-1: each lane keeps a running count `cnt` of its
// row's columns in the tiles already passed, and key u of tile t sits at
//     row_ptr[i] + cnt + popcount(rowbits & ((1 << u) - 1)),
// rowbits being the row's membership mask in the tile (all ones for a
// wavefront the plan marks FULL, the stored 64-bit mask for PARTIAL).  No
// run arithmetic and no division is needed on the device.
#include <hip/hip_runtime.h>
#include <math.h>

#include "bounds.hpp"
#include "launch.hpp"
#include "mfma_util.hpp"

namespace splat {
namespace {

using namespace mfma;

constexpr int kTileThreads = 256;   // 4 wavefronts x 32 rows of a group
// A staged score row: up to 31 values carried from earlier tiles (before
// kCarry), then the tile's 64; 100 floats keep rows 16-byte aligned.
constexpr int kCarry = 32;
constexpr int kStageStride = 100;

// 4 floats at a 4-byte aligned address (values of a row start anywhere)
typedef float f32x4u_t __attribute__((ext_vector_type(4), aligned(4)));

__device__ __forceinline__ int popc64(uint64_t x) { return __builtin_popcountll(x); }

// The keys a lane of half h holds in both MFMA layouts used here come in
// eight groups of four: keys 8*g + 4*h + e (g < 8, e < 4).  For a row's
// membership mask `bits` in a tile, f(g, e, present, pos) is called for each
// of them with `pos` the key's position among the row's keys of the tile
// (meaningful when present).  Only constant shifts are used, so nothing
// lane-dependent is kept live across the tile loop.
template <typename F>
__device__ __forceinline__ void for_each_key(uint64_t bits, int h, F&& f) {
  const uint64_t b = bits >> (4 * h);
  int off = h ? __builtin_popcount((uint32_t)bits & 0xFu) : 0;
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    const uint32_t nib = (uint32_t)(b >> (8 * g)) & 0xFu;
    const uint32_t oth = (uint32_t)(b >> (8 * g + 4)) & 0xFu;   // the other half's next four
#pragma unroll
    for (int e = 0; e < 4; ++e) f(g, e, (nib >> e) & 1u, off + __builtin_popcount(nib & ((1u << e) - 1u)));
    off += __builtin_popcount(nib) + __builtin_popcount(oth);
  }
}

// --------------------------------------------------------------------------
// R-SDDMM: S[b,h,row_ptr[i] + k] = scale * <Q[b,h,i,:], K[b,h,col(i,k),:]>.
// One workgroup per (row group, batch*head).  Per key tile a wavefront forms
// S^T = K Q^T for its 32 rows on v_mfma_f32_32x32x16_bf16 with both operands
// read straight from global memory (16 bytes per lane; the 4 wavefronts of a
// group read the same K tile, which stays in cache), then stores the scores
// of the row's columns.  Lane (qi, h) holds keys 32*kb2 + 8*(r/4) + 4*h + r%4
// of query row qi.  On FULL tiles the 32 x 64 scores go through a per-
// wavefront LDS buffer and come back as row segments, so each store writes
// 4 rows x 256 contiguous bytes (16 lanes per row) instead of 32 rows x 32
// bytes; on PARTIAL tiles each present score is stored at its rank.  This is
// a store stream: occupancy (three wavefronts per SIMD for d = 64) is what
// keeps enough of it in flight.
template <int D>
__global__ __launch_bounds__(kTileThreads, D == 64 ? 3 : 2) void k_rsddmm_tiles(
    const Group* __restrict__ groups, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ row_ptr, const Tile* __restrict__ tiles,
    const uint64_t* __restrict__ masks, int L, int BH, int64_t nnz,
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, float scale,
    float* __restrict__ S) {
  constexpr int NKS = D / 16;
  const int g = blockIdx.x / BH;
  const int bh = blockIdx.x - g * BH;
  const Group grp = groups[g];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (wave * kWaveRows >= grp.nrows) return;   // no barriers below
  const int qi = lane & 31, h = lane >> 5;
  const int m = wave * kWaveRows + qi;
  const bool row_valid = m < grp.nrows;
  const int row = row_valid ? dbg::idx(rows[grp.row_off + m], L, dbg::kRow) : 0;
  const size_t head = (size_t)bh * L * D;
  const __bf16* Kh = K + head;

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
  // Positions within a row are 32-bit float indices counted from the start
  // of the 128-byte line that holds the row's first value, so that 16-byte
  // chunks and 128-byte lines of the index are those of the address space
  // (S is 16-byte aligned): the row's values sit at [lead, lead + row_len)
  // from its line base S + rline.
  const int64_t sidx = row_valid ? (int64_t)bh * nnz + row_ptr[row] : 0;
  const int64_t total = (int64_t)BH * nnz;   // values of S over all heads
  const int lead = (int)((((uintptr_t)S >> 2) + (uint64_t)sidx) & 31u);
  const int64_t rline = sidx - lead;
  const int row_len = row_valid ? row_ptr[row + 1] - row_ptr[row] : 0;
  int cnt = 0;                 // the row's values produced so far
  int wr = lead;               // the row's values written so far end here
  // the write-out below serves rows 4*it + lane/16; their line bases, once
  const int rr = lane >> 4, cc = lane & 15;
  int64_t rl[kWaveRows / 4];
#pragma unroll
  for (int it = 0; it < kWaveRows / 4; ++it) rl[it] = __shfl(rline, 4 * it + rr, 64);
  __shared__ __attribute__((aligned(16))) float stage[kTileThreads / 64][kWaveRows * kStageStride];
  float* const stw = stage[wave];

  // K operands of a tile (keys past its end re-read the last key)
  auto load_k = [&](const Tile& tl, bf16x8_t (&ka)[2][NKS]) {
    const int last = tl.nk - 1;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
      const int key = dbg::idx(tl.kb + tl.ks * min(32 * kb2 + qi, last), L, dbg::kKey);
      const __bf16* krow = Kh + (size_t)key * D + 8 * h;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) ka[kb2][ks] = *(const bf16x8_t*)(krow + 16 * ks);
    }
  };
  // One tile: this wavefront's scores of the tile go to their staging rows
  // (after the values a row still carries from earlier tiles), then every
  // row writes the whole 128-byte lines it has completed.
  auto tile = [&](const Tile& tl, const bf16x8_t (&ka)[2][NKS]) {
    const int wst = (tl.flags >> (kWaveShift + 2 * wave)) & 3;
    if (wst == kWaveEmpty) return;
    const uint64_t bits =
        wst == kWaveFull ? ~0ull : masks[(size_t)max(tl.mask_block, 0) * kBM + m];
    f32x16_t sacc[2];
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb2][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) sacc[kb2] = mfma32(ka[kb2][ks], qf[ks], sacc[kb2]);
    }
    // A row's present keys of the tile take consecutive places of S (their
    // ranks): staged at kCarry + rank.
    if (wst == kWaveFull) {
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const float4 v = make_float4(sacc[kb2][4 * rg] * scale, sacc[kb2][4 * rg + 1] * scale,
                                       sacc[kb2][4 * rg + 2] * scale, sacc[kb2][4 * rg + 3] * scale);
          *(float4*)(stw + qi * kStageStride + kCarry + 32 * kb2 + 8 * rg + 4 * h) = v;
        }
    } else if (row_valid) {
      // key 8*g + 4*h + e is element 4*(g%4) + e of sacc[g/4]
      for_each_key(bits, h, [&](int g, int e, unsigned present, int pos) {
        if (present)
          stw[qi * kStageStride + kCarry + pos] = sacc[g >> 2][4 * (g & 3) + e] * scale;
      });
    }
    // This row's staged values cover [wr, end): the carried part then the
    // tile's.  Written now: up to the last line boundary, or to the row's
    // end once the row is complete.
    const int n = row_valid ? popc64(bits) : 0;
    const int start = lead + cnt, end = start + n;
    const int new_wr = (cnt + n == row_len) ? end : max(end & ~31, wr);
#pragma unroll
    for (int it = 0; it < kWaveRows / 4; ++it) {
      const int r = 4 * it + rr;
      const int lo = __shfl(wr, r, 64), hi = __shfl(new_wr, r, 64);
      const int st = __shfl(start, r, 64), en = __shfl(end, r, 64);
      const float* srow = stw + r * kStageStride + kCarry - st;   // srow[g]: value at index g
      float* const grow = S + rl[it];                              // the row's line base
      // 16-byte chunks from the chunk holding lo; at most (31 + 64) / 4 + 1 of them
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int a = (lo & ~3) + 4 * (cc + 16 * k);
        if (a >= hi) continue;
        if (a >= lo && a + 4 <= hi) {
          const f32x4u_t v = *(const f32x4u_t*)(srow + a);
          __builtin_nontemporal_store(v, (f32x4u_t*)(grow + dbg::rel(a, rl[it], total - 3,
                                                                     dbg::kValue)));
        } else {
          // the row's first or last line: single values, cached so that the
          // rest of the line (the neighbouring row's) merges with them
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (a + e >= lo && a + e < hi)
              grow[dbg::rel(a + e, rl[it], total, dbg::kValue)] = srow[a + e];
        }
      }
      // what is left of the row, [hi, en), moves to just before kCarry
      const int left = en - hi;
      float keep[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) keep[k] = (cc + 16 * k < left) ? srow[hi + cc + 16 * k] : 0.f;
#pragma unroll
      for (int k = 0; k < 2; ++k)
        if (cc + 16 * k < left) stw[r * kStageStride + kCarry - left + cc + 16 * k] = keep[k];
    }
    wr = new_wr;
    cnt += n;
  };
  for (int t = grp.tile_begin; t < grp.tile_end; ++t) {
    const Tile tl = tiles[t];
    if (((tl.flags >> (kWaveShift + 2 * wave)) & 3) == kWaveEmpty) continue;
    bf16x8_t ka[2][NKS];
    load_k(tl, ka);
    tile(tl, ka);
  }
}

// --------------------------------------------------------------------------
// Row softmax over the non-zeros (section 6): one wavefront per (batch*head,
// row).  A row of at most 256 * NV values is held in registers (4 consecutive
// values per lane and load), so S is read once and P written once; a longer
// row is streamed twice, first for its maximum and sum (a running maximum per
// lane, the sum rescaled when it grows), then to write P.  P may alias S:
// every value is read before it is written, by the lane that writes it.
// NV is kept small (registers bound how many wavefronts keep loads in flight)
// since rows far longer than the typical one are rare.
__device__ __forceinline__ float ex2_from(float x, float m) {
  constexpr float kLog2e = 1.4426950408889634f;
  return x == -INFINITY ? 0.f : exp2_hw((x - m) * kLog2e);
}

__device__ __forceinline__ void load4_row(const float* s, int idx, int n, float (&x)[4]) {
  if (idx + 3 < n) {
    const f32x4u_t v = *(const f32x4u_t*)(s + idx);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = v[e];
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = idx + e < n ? s[idx + e] : -INFINITY;
  }
}

// P is streamed out in 16-byte non-temporal stores: it is far larger than
// the caches, and dirty P lines left there slow the R-SpMM that reads P next
__device__ __forceinline__ void store4_row(float* p, int idx, int n, const float (&y)[4]) {
  if (idx + 3 < n) {
    const f32x4u_t v = {y[0], y[1], y[2], y[3]};
    __builtin_nontemporal_store(v, (f32x4u_t*)(p + idx));
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (idx + e < n) p[idx + e] = y[e];   // single values: ordinary stores
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Grid: x over blocks of rows, y over batch*head, so that the work-item
// count of each dimension stays far below 2^32 at every allowed size.
//
// Short rows: LPR lanes per row (LPR a power of two below 64, 4*LPR values
// at most), 64 / LPR rows per wavefront, reductions within the lane segment.
template <int LPR>
__global__ __launch_bounds__(256) void k_softmax_seg(const int32_t* __restrict__ row_ptr, int L,
                                                     int64_t nnz, const float* S, float* P) {
  constexpr int RPW = 64 / LPR;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int sub = lane & (LPR - 1);
  const int i = (blockIdx.x * 4 + wave) * RPW + lane / LPR;
  const int bh = blockIdx.y;
  int n = 0;
  size_t base = 0;
  if (i < L) {
    const int32_t b0 = row_ptr[i];
    n = row_ptr[i + 1] - b0;
    base = (size_t)bh * nnz + b0;
    if (!dbg::check(n == 0 || (b0 >= 0 && b0 + (int64_t)n <= nnz), dbg::kValue)) n = 0;
  }
  // every lane takes part in the segment reductions; lanes without a row see n = 0
  float x[4];
  load4_row(S + base, 4 * sub, n, x);
  float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  float sum = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[e] = ex2_from(x[e], mx);
    sum += x[e];
  }
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
  if (n == 0) return;
  const float inv = 1.f / sum;
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] *= inv;
  store4_row(P + base, 4 * sub, n, x);
}

// One wavefront per row.
template <int NV>
__global__ __launch_bounds__(256) void k_softmax(const int32_t* __restrict__ row_ptr, int L,
                                                 int64_t nnz, const float* S, float* P) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + wave;
  if (i >= L) return;
  const int bh = blockIdx.y;
  const int32_t b0 = row_ptr[i];
  const int n = row_ptr[i + 1] - b0;
  if (n == 0) return;
  if (!dbg::check(b0 >= 0 && b0 + (int64_t)n <= nnz, dbg::kValue)) return;
  const size_t base = (size_t)bh * nnz + b0;
  const float* s = S + base;
  float* p = P + base;

  if (n <= 256 * NV) {
    float x[NV][4];
    float mx = -INFINITY;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      load4_row(s, 4 * (lane + 64 * k), n, x[k]);
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = fmaxf(mx, x[k][e]);
    }
    mx = wave_max(mx);
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[k][e] = ex2_from(x[k][e], mx);
        sum += x[k][e];
      }
    const float inv = 1.f / wave_sum(sum);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
#pragma unroll
      for (int e = 0; e < 4; ++e) x[k][e] *= inv;
      store4_row(p, 4 * (lane + 64 * k), n, x[k]);
    }
    return;
  }
  // long row: running maximum and rescaled sum per lane, then the write pass
  float mx = -INFINITY, sum = 0.f;
  for (int c0 = 0; c0 < n; c0 += 256) {
    float x[4];
    load4_row(s, c0 + 4 * lane, n, x);
    const float cm = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    if (cm > mx) {
      sum *= ex2_from(mx, cm);
      mx = cm;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) sum += ex2_from(x[e], mx);
  }
  const float gm = wave_max(mx);
  const float inv = 1.f / wave_sum(sum * ex2_from(mx, gm));
  for (int c0 = 0; c0 < n; c0 += 256) {
    float x[4];
    load4_row(s, c0 + 4 * lane, n, x);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = ex2_from(x[e], gm) * inv;
    store4_row(p, c0 + 4 * lane, n, x);
  }
}

// --------------------------------------------------------------------------
// R-SpMM: O[b,h,i,:] = sum_k P[b,h,row_ptr[i] + k] V[b,h,col(i,k),:].  One
// workgroup per (row group, batch*head).  The V tile goes through LDS (two
// slots: the next tile's rows are loaded into registers while the current
// one is multiplied, then written to the other slot; one barrier per tile)
// so that the V^T operand can be read transposed; the P^T operand comes
// straight from P in the key order of those reads, split into a bf16 high
// part and a bf16 remainder (p - hi), each multiplied on the matrix cores:
// P then enters with about 16 significant bits instead of 8, at the cost of
// MFMA work this HBM-bound kernel has to spare.
//
// COL: P holds the values in the column-compressed, column-major layout
// (section 9): the value of (row, key) is read at col_pos(cols[key], row),
// with the tile's column descriptors staged in LDS beside its V rows.  The
// same values enter the same MFMAs in the same order, so the result equals
// the row-major kernel's.  At d = 128 its 32 scattered P loads per tile need
// more than the 256 registers of two workgroups per CU, so it runs one.
template <int D, typename OutT, bool COL>
__global__ __launch_bounds__(kTileThreads, (COL && D == 128) ? 1 : 2) void k_rspmm_tiles(
    const Group* __restrict__ groups, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ row_ptr, const Tile* __restrict__ tiles,
    const uint64_t* __restrict__ masks, const ColRun* __restrict__ cols, int L, int BH,
    int64_t nnz, const float* __restrict__ P, const __bf16* __restrict__ V,
    OutT* __restrict__ O) {
  constexpr int RB = 2 * D, CPR = RB / 16, TB = kBN * RB, NDB = D / 32;
  constexpr int CPT = TB / 16 / kTileThreads;   // 16-byte chunks per thread and tile
  __shared__ __attribute__((aligned(16))) char vt[2][TB];
  __shared__ ColRun ct[COL ? 2 : 1][COL ? kBN : 1];

  const int g = blockIdx.x / BH;
  const int bh = blockIdx.x - g * BH;
  const Group grp = groups[g];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int qi = lane & 31, h = lane >> 5;
  const int m = wave * kWaveRows + qi;
  const bool row_valid = m < grp.nrows;
  const int row = row_valid ? dbg::idx(rows[grp.row_off + m], L, dbg::kRow) : 0;
  const size_t head = (size_t)bh * L * D;
  const __bf16* Vh = V + head;
  const float* prow = P + (size_t)bh * nnz + (COL ? 0 : row_ptr[row]);

  int voff[NDB];
  v_operand_offsets<D>(lane, voff);
  f32x16_t oacc[NDB];
#pragma unroll
  for (int b = 0; b < NDB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[b][r] = 0.f;

  // chunk c of tile row r is stored at chunk c ^ swz_v(r) of the row
  auto load_v = [&](const Tile& tl, u32x4_t (&reg)[CPT]) {
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int idx = tid + kTileThreads * k;
      const int r = idx / CPR, c = idx % CPR;
      const int key = dbg::idx(tl.kb + tl.ks * min(r, tl.nk - 1), L, dbg::kKey);
      reg[k] = *(const u32x4_t*)(Vh + (size_t)key * D + 8 * c);
    }
  };
  auto store_v = [&](char* slot, const u32x4_t (&reg)[CPT]) {
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int idx = tid + kTileThreads * k;
      const int r = idx / CPR, c = idx % CPR;
      *(u32x4_t*)(slot + r * RB + 16 * (c ^ swz_v(r))) = reg[k];
    }
  };

  // column descriptors of a tile's keys (COL only): one per thread below nk
  auto load_c = [&](const Tile& tl, ColRun& c) {
    if (COL && tid < tl.nk) c = cols[tl.kb + tl.ks * tid];
  };
  auto store_c = [&](int slot, const Tile& tl, const ColRun& c) {
    if (COL && tid < tl.nk) ct[slot][tid] = c;
  };

  const int tb = grp.tile_begin, nt = grp.tile_end - grp.tile_begin;
  int cnt = 0;
  if (nt > 0) {
    u32x4_t vreg[CPT];
    ColRun creg{0, 1, 0, 0};
    load_v(tiles[tb], vreg);
    load_c(tiles[tb], creg);
    store_v(vt[0], vreg);
    store_c(0, tiles[tb], creg);
    __syncthreads();
    for (int i = 0; i < nt; ++i) {
      const Tile tl = tiles[tb + i];
      if (i + 1 < nt) {
        load_v(tiles[tb + i + 1], vreg);
        load_c(tiles[tb + i + 1], creg);
      }
      const int wst = (tl.flags >> (kWaveShift + 2 * wave)) & 3;
      if (wst != kWaveEmpty) {
        const uint64_t bits =
            wst == kWaveFull ? ~0ull : masks[(size_t)max(tl.mask_block, 0) * kBM + m];
        // P^T operand: k-step j, element e of lane half h is key
        // u = 16*j + 8*(e/4) + 4*h + e%4
        float pv[4][8];
        if (COL && row_valid) {
          const ColRun* cc = ct[COL ? (i & 1) : 0];
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int u = 16 * j + 8 * (e >> 2) + 4 * h + (e & 3);
              pv[j][e] = ((bits >> u) & 1ull)
                             ? prow[dbg::idx((int64_t)col_pos(cc[u], row), nnz, dbg::kColPos)]
                             : 0.f;
            }
        } else if (row_valid) {
          const float* src = prow + cnt;
          const int64_t rpos = (int64_t)row_ptr[row] + cnt;   // src's position in the head
          if (wst == kWaveFull) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const f32x4u_t a =
                  *(const f32x4u_t*)(src + dbg::rel(16 * j + 4 * h, rpos, nnz - 3, dbg::kValue));
              const f32x4u_t b = *(const f32x4u_t*)(src + dbg::rel(16 * j + 8 + 4 * h, rpos,
                                                                     nnz - 3, dbg::kValue));
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                pv[j][e] = a[e];
                pv[j][4 + e] = b[e];
              }
            }
          } else {
            // key 8*g + 4*h + e is element 4*(g%2) + e of k-step g/2
            for_each_key(bits, h, [&](int g, int e, unsigned present, int pos) {
              pv[g >> 1][4 * (g & 1) + e] =
                  present ? src[dbg::rel(pos, rpos, nnz, dbg::kValue)] : 0.f;
            });
          }
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 8; ++e) pv[j][e] = 0.f;
        }
        cnt += popc64(bits);
        bf16x8_t phi[4], plo[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            phi[j][e] = (__bf16)pv[j][e];
            plo[j][e] = (__bf16)(pv[j][e] - (float)phi[j][e]);
          }
        bf16x8_t va[NDB][4];
        read_v_operands<D>(lds_addr(vt[i & 1]), voff, va);
#pragma unroll
        for (int b = 0; b < NDB; ++b)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            oacc[b] = mfma32(va[b][j], phi[j], oacc[b]);
            oacc[b] = mfma32(va[b][j], plo[j], oacc[b]);
          }
      }
      if (i + 1 < nt) {
        store_v(vt[(i + 1) & 1], vreg);
        store_c((i + 1) & 1, tiles[tb + i + 1], creg);
      }
      __syncthreads();
    }
  }

  if (row_valid) {
    OutT* orow = O + head + (size_t)row * D;
#pragma unroll
    for (int b = 0; b < NDB; ++b)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg)
        store4<OutT>(orow + b * 32 + rg * 8 + 4 * h, oacc[b][4 * rg], oacc[b][4 * rg + 1],
                     oacc[b][4 * rg + 2], oacc[b][4 * rg + 3]);
  }
}

// Column-major copy of P (data-layout reordering, section 9).  One workgroup
// per (row group, batch*head) walks the group's tiles as R-SpMM does; lane
// (row m, half h) moves its row's values for keys 32h .. 32h+31 of each tile.
// All lanes step through the keys together, so at each step the 32 lanes of
// a half store one column at their rows' positions: consecutive rows of a
// column land at consecutive addresses.
__global__ __launch_bounds__(kTileThreads) void k_colmajor_tiles(
    const Group* __restrict__ groups, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ row_ptr, const Tile* __restrict__ tiles,
    const uint64_t* __restrict__ masks, const ColRun* __restrict__ cols, int BH, int64_t nnz,
    const float* __restrict__ P, float* __restrict__ Pt) {
  __shared__ ColRun ct[kBN];
  const int g = blockIdx.x / BH;
  const int bh = blockIdx.x - g * BH;
  const Group grp = groups[g];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int qi = lane & 31, h = lane >> 5;
  const int m = wave * kWaveRows + qi;
  const bool row_valid = m < grp.nrows;
  const int row = row_valid ? rows[grp.row_off + m] : 0;
  const float* prow = P + (size_t)bh * nnz + row_ptr[row];
  float* dst = Pt + (size_t)bh * nnz;
  int cnt = 0;
  for (int t = grp.tile_begin; t < grp.tile_end; ++t) {
    const Tile tl = tiles[t];
    __syncthreads();   // every wavefront is done with the previous tile's descriptors
    if (tid < tl.nk) ct[tid] = cols[tl.kb + tl.ks * tid];
    __syncthreads();
    const int wst = (tl.flags >> (kWaveShift + 2 * wave)) & 3;
    if (wst == kWaveEmpty) continue;
    const uint64_t bits =
        wst == kWaveFull ? ~0ull : masks[(size_t)max(tl.mask_block, 0) * kBM + m];
    if (row_valid && wst == kWaveFull) {
      // the row's 32 values for this half are contiguous: 16-byte loads
      const float* src = prow + cnt + 32 * h;
      const int64_t rpos = (int64_t)row_ptr[row] + cnt + 32 * h;   // src's position in the head
      float v[32];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const f32x4u_t x = *(const f32x4u_t*)(src + dbg::rel(4 * q, rpos, nnz - 3, dbg::kValue));
#pragma unroll
        for (int e = 0; e < 4; ++e) v[4 * q + e] = x[e];
      }
#pragma unroll
      for (int u = 0; u < 32; ++u)
        dst[dbg::idx((int64_t)col_pos(ct[32 * h + u], row), nnz, dbg::kColPos)] = v[u];
    } else if (row_valid) {
      const unsigned hb = (unsigned)(bits >> (32 * h));
      const float* src = prow + cnt + (h ? __builtin_popcount((unsigned)bits) : 0);
      const int64_t rpos =   // src's position in the head
          (int64_t)row_ptr[row] + cnt + (h ? __builtin_popcount((unsigned)bits) : 0);
      int k = 0;
      for (int u = 0; u < 32; ++u) {
        if ((hb >> u) & 1u) {
          dst[dbg::idx((int64_t)col_pos(ct[32 * h + u], row), nnz, dbg::kColPos)] =
              src[dbg::rel(k, rpos, nnz, dbg::kValue)];
          ++k;
        }
      }
    }
    cnt += popc64(bits);
  }
}

}  // namespace

hipError_t bounds_collect_tiles(uint32_t* bits, bool clear) { return dbg::collect(bits, clear); }

namespace {

template <int NV>
hipError_t softmax_launch(const DevAcsr& a, int BH, const float* S, float* P, hipStream_t st) {
  hipLaunchKernelGGL(k_softmax<NV>, dim3((unsigned)((a.L + 3) / 4), (unsigned)BH), dim3(256), 0,
                     st, a.row_ptr, a.L, a.nnz, S, P);
  return hipGetLastError();
}

template <int LPR>
hipError_t softmax_seg_launch(const DevAcsr& a, int BH, const float* S, float* P, hipStream_t st) {
  constexpr int rows_per_block = 4 * (64 / LPR);
  hipLaunchKernelGGL(k_softmax_seg<LPR>, dim3((unsigned)((a.L + rows_per_block - 1) / rows_per_block),
                                              (unsigned)BH),
                     dim3(256), 0, st, a.row_ptr, a.L, a.nnz, S, P);
  return hipGetLastError();
}

template <int D, typename OutT, bool COL>
hipError_t rspmm_launch(const DevAcsr& a, int BH, const float* P, const void* V, void* O,
                        hipStream_t st) {
  hipLaunchKernelGGL((k_rspmm_tiles<D, OutT, COL>), dim3(a.n_groups * BH), dim3(kTileThreads), 0,
                     st, a.groups, a.rows, a.row_ptr, a.tiles, a.masks, a.cols, a.L, BH, a.nnz, P,
                     (const __bf16*)V, (OutT*)O);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rsddmm_tiles(const DevAcsr& a, int BH, int d, const void* Q, const void* K,
                               float scale, float* S, hipStream_t st) {
  if (d == 64)
    hipLaunchKernelGGL(k_rsddmm_tiles<64>, dim3(a.n_groups * BH), dim3(kTileThreads), 0, st,
                       a.groups, a.rows, a.row_ptr, a.tiles, a.masks, a.L, BH, a.nnz,
                       (const __bf16*)Q, (const __bf16*)K, scale, S);
  else
    hipLaunchKernelGGL(k_rsddmm_tiles<128>, dim3(a.n_groups * BH), dim3(kTileThreads), 0, st,
                       a.groups, a.rows, a.row_ptr, a.tiles, a.masks, a.L, BH, a.nnz,
                       (const __bf16*)Q, (const __bf16*)K, scale, S);
  return hipGetLastError();
}

hipError_t launch_softmax(const DevAcsr& a, int BH, const float* S, float* P, hipStream_t st) {
  const int n = a.max_row_nnz;
  if (n <= 4) return softmax_seg_launch<1>(a, BH, S, P, st);
  if (n <= 8) return softmax_seg_launch<2>(a, BH, S, P, st);
  if (n <= 16) return softmax_seg_launch<4>(a, BH, S, P, st);
  if (n <= 32) return softmax_seg_launch<8>(a, BH, S, P, st);
  if (n <= 64) return softmax_seg_launch<16>(a, BH, S, P, st);
  if (n <= 128) return softmax_seg_launch<32>(a, BH, S, P, st);
  if (n <= 256) return softmax_launch<1>(a, BH, S, P, st);
  if (n <= 512) return softmax_launch<2>(a, BH, S, P, st);
  if (n <= 1024) return softmax_launch<4>(a, BH, S, P, st);
  return softmax_launch<8>(a, BH, S, P, st);   // longer rows take the two-pass path
}

template <bool COL>
static hipError_t rspmm_tiles_t(const DevAcsr& a, int BH, int d, const float* P, const void* V,
                                void* O, int out_dtype, hipStream_t st) {
  if (d == 64)
    return out_dtype == 0 ? rspmm_launch<64, float, COL>(a, BH, P, V, O, st)
                          : rspmm_launch<64, __bf16, COL>(a, BH, P, V, O, st);
  return out_dtype == 0 ? rspmm_launch<128, float, COL>(a, BH, P, V, O, st)
                        : rspmm_launch<128, __bf16, COL>(a, BH, P, V, O, st);
}

hipError_t launch_rspmm_tiles(const DevAcsr& a, int BH, int d, const float* P, const void* V,
                              void* O, int out_dtype, bool colmajor, hipStream_t st) {
  return colmajor ? rspmm_tiles_t<true>(a, BH, d, P, V, O, out_dtype, st)
                  : rspmm_tiles_t<false>(a, BH, d, P, V, O, out_dtype, st);
}

hipError_t launch_transpose_colmajor(const DevAcsr& a, int BH, const float* P, float* Pt,
                                     hipStream_t st) {
  hipLaunchKernelGGL(k_colmajor_tiles, dim3(a.n_groups * BH), dim3(kTileThreads), 0, st, a.groups,
                     a.rows, a.row_ptr, a.tiles, a.masks, a.cols, BH, a.nnz, P, Pt);
  return hipGetLastError();
}

}  // namespace splat
