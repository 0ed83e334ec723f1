// acsr_core.hpp -- ACSR metadata, work plan and the membership arithmetic
// shared by the host planner and the device kernels.
//
// Per row, the column set is held as at most SPLAT_MAX_RUNS disjoint ascending
// runs {start + stride * k : 0 <= k < count}; `prefix` is the number of
// columns in the row's earlier runs, so the value of run r, element k sits at
// row_ptr[i] + prefix + k (section 5.1: sparse index = a * j + b inside a run
// with a = 1/stride, b = -start/stride).
//
// The plan cuts every row group's column span into key tiles of at most BN
// keys; tile keys are kb + ks * u (u < nk).  Tiles of one group cover
// disjoint, ascending column intervals [kb, kb + ks*(nk-1)], and every column
// of the group's rows that falls inside a tile's interval is one of its keys.
// This makes the position of a key inside its row
//     rank = count_lt(row, kb) + popcount(rowbits & ((1 << u) - 1))
// where rowbits = tile_row_bits(...) is the row's membership mask in the tile.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define SPLAT_HD __host__ __device__ __forceinline__
#else
#define SPLAT_HD inline
#endif

#ifndef SPLAT_MAX_RUNS
#define SPLAT_MAX_RUNS 4
#endif

namespace splat {

constexpr int kBM = 128;   // rows per group (4 waves x 32 rows)
constexpr int kBN = 64;    // keys per tile
constexpr int kWaveRows = 32;  // rows of a group handled by one wavefront
constexpr int kWavesPerGroup = kBM / kWaveRows;

// Tile::flags: bit 0 = every key of the tile is in every row of the group;
// bits 8 + 2w, 9 + 2w = state of the tile for rows [32w, 32w + 32) of the
// group: kWaveEmpty (no row has a key here), kWavePartial (per-row masks in
// the plan's mask block), kWaveFull (every key in every row).
constexpr int kTileFull = 1;
constexpr int kWaveEmpty = 0;
constexpr int kWavePartial = 1;
constexpr int kWaveFull = 3;
constexpr int kWaveShift = 8;

struct Run {
  int32_t start, stride, count, prefix;
};

struct RowRuns {
  Run r[SPLAT_MAX_RUNS];   // unused runs have count == 0
};

// A column held as one affine run of rows (column-wise affine
// compressibility, section 5.2): rows start + stride * t for t < count, whose
// values sit at ptr + t of the head's column-compressed, column-major value
// array (ptr = the column's offset in that array).
struct ColRun {
  int32_t start, stride, count, ptr;
};

struct Group {
  int32_t row_off, nrows, tile_begin, tile_end;
};

struct Tile {
  int32_t kb, ks, nk, flags;
  int32_t mask_block;   // -1, or index of the tile's kBM per-row masks in the mask array
  int32_t pad[3];
};

SPLAT_HD int32_t floor_div(int32_t a, int32_t b) {  // b > 0
  int32_t q = a / b;
  return (a % b != 0 && a < 0) ? q - 1 : q;
}

SPLAT_HD int32_t ceil_div(int32_t a, int32_t b) {   // b > 0
  int32_t q = a / b;
  return (a % b != 0 && a > 0) ? q + 1 : q;
}

SPLAT_HD int32_t imin(int32_t a, int32_t b) { return a < b ? a : b; }
SPLAT_HD int32_t imax(int32_t a, int32_t b) { return a > b ? a : b; }

// bits lo..hi set (0 <= lo <= hi <= 63)
SPLAT_HD uint64_t range_bits(int32_t lo, int32_t hi) {
  return (~0ull >> (63 - hi)) & (~0ull << lo);
}

// bits at 0, p, 2p, ... below 64 (p >= 1)
SPLAT_HD uint64_t periodic_bits(int32_t p) {
  if (p >= 64) return 1ull;
  uint64_t pat = 1ull;
  for (int32_t w = p; w < 64; w <<= 1) pat |= pat << w;
  return pat;
}

// Membership bits of one run inside a tile: bit u set iff kb + ks*u is in the
// run, for u < nk (nk <= 64).  O(1) for the combinations the planner emits
// (ks == 1, or run stride 1, or run stride == ks); any other combination is
// answered key by key.
SPLAT_HD uint64_t run_tile_bits(const Run& run, int32_t kb, int32_t ks, int32_t nk) {
  if (run.count <= 0 || nk <= 0) return 0;
  const int32_t last = run.start + run.stride * (run.count - 1);
  const int32_t tlast = kb + ks * (nk - 1);
  if (last < kb || run.start > tlast) return 0;
  if (ks == 1) {
    const int32_t lo = imax(run.start, kb) - kb;
    const int32_t hi = imin(last, tlast) - kb;
    if (run.stride == 1) return range_bits(lo, hi);
    // u = (run.start - kb) mod stride, first such u >= lo
    int32_t r = (run.start - kb) % run.stride;
    if (r < 0) r += run.stride;
    int32_t d = (r - lo) % run.stride;
    if (d < 0) d += run.stride;
    const int32_t u0 = lo + d;
    if (u0 > hi) return 0;
    return (periodic_bits(run.stride) << u0) & range_bits(u0, hi);
  }
  if (run.stride == 1 || run.stride == ks) {
    if (run.stride == ks && (run.start - kb) % ks != 0) return 0;
    const int32_t ulo = imax(0, ceil_div(run.start - kb, ks));
    const int32_t uhi = imin(nk - 1, floor_div(last - kb, ks));
    if (ulo > uhi) return 0;
    return range_bits(ulo, uhi);
  }
  uint64_t bits = 0;
  for (int32_t u = 0; u < nk; ++u) {
    const int32_t j = kb + ks * u;
    const int32_t off = j - run.start;
    if (off >= 0 && off % run.stride == 0 && off / run.stride < run.count) bits |= 1ull << u;
  }
  return bits;
}

SPLAT_HD uint64_t tile_row_bits(const RowRuns& rr, int32_t kb, int32_t ks, int32_t nk) {
  uint64_t bits = 0;
#pragma unroll
  for (int r = 0; r < SPLAT_MAX_RUNS; ++r) bits |= run_tile_bits(rr.r[r], kb, ks, nk);
  return bits;
}

// number of the row's columns strictly below x
SPLAT_HD int32_t count_lt(const RowRuns& rr, int32_t x) {
  int32_t n = 0;
#pragma unroll
  for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
    const Run& q = rr.r[r];
    if (q.count > 0 && x > q.start) n += imin(q.count, ceil_div(x - q.start, q.stride));
  }
  return n;
}

}  // namespace splat
