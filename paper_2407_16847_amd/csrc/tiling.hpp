// tiling.hpp -- thread-block arrangements and the cost model of section 7
// (host-side diagnostic).
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "acsr_host.hpp"

namespace splat {

struct TilingStats {
  int64_t blocks = 0, points = 0, divergent = 0, redundant = 0;
  double reuse = 0, coalesced = 0, cost = 0;
  int32_t stretch = 1, iterations = 0;
};

// method: SPLAT_TILING_POSET, SPLAT_TILING_GRID or SPLAT_TILING_NAIVE; stretch 0 selects it
// (poset only).  anchors (optional) receives (row, col) pairs in placement
// order.
splat_status tile_mask(const HostAcsr& a, int32_t method, int32_t m, int32_t n, int32_t stretch,
                       std::vector<int32_t>* anchors, TilingStats& st, std::string& err);

}  // namespace splat
