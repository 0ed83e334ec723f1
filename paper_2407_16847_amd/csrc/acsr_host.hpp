// acsr_host.hpp -- host-side ACSR construction and work planning (no HIP).
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/splat.h"
#include "acsr_core.hpp"

namespace splat {

struct HostAcsr {
  int32_t L = 0;
  int64_t nnz = 0;
  int32_t max_row_nnz = 0;
  int32_t max_runs = 0;
  std::vector<int32_t> row_ptr;   // L + 1
  std::vector<RowRuns> runs;      // L
  std::vector<int32_t> nruns;     // L
  // work plan (launch order)
  std::vector<int32_t> rows;      // L, grouped
  std::vector<Group> groups;
  std::vector<Tile> tiles;
  std::vector<uint64_t> masks;    // kBM row masks per tile with a PARTIAL wavefront
  int64_t computed = 0;           // kWaveRows * kBN per non-empty wavefront tile
  int32_t n_full = 0;
  uint32_t plan_flags = 0;        // SPLAT_PLAN_* bits the plan was built with
  // column-wise analysis (SPLAT_PLAN_COLUMNS): -1 not done, 0 some column is
  // not one affine run, 1 every column is; cols[j] describes column j
  int32_t col_regular = -1;
  std::vector<ColRun> cols;       // L when col_regular == 1
};

// Union of the descriptor's terms per row -> canonical runs, row_ptr, plan.
splat_status build_from_desc(const splat_pattern_desc& desc, HostAcsr& out, std::string& err,
                            uint32_t plan_flags = 0);

// Paper's analysis pass on an explicit 0/1 mask: one affine run per row or
// SPLAT_ERR_NOT_REGULAR.
splat_status build_from_mask(int32_t L, const uint8_t* mask, HostAcsr& out, std::string& err);

// Row grouping and key tiling (called by both builders).
void plan_work(HostAcsr& a);

splat_status pattern_window(int32_t L, int32_t w, splat_pattern_desc* out);
splat_status pattern_blocked(int32_t L, int32_t block, splat_pattern_desc* out);
splat_status pattern_strided_local(int32_t L, int32_t local, int32_t stride, splat_pattern_desc* out);
splat_status pattern_dilated(int32_t L, int32_t w, int32_t dilation, splat_pattern_desc* out);
splat_status pattern_window_global(int32_t L, int32_t w, int32_t n_global, splat_pattern_desc* out);
splat_status pattern_full(int32_t L, splat_pattern_desc* out);

}  // namespace splat
