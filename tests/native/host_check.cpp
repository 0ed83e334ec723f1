// host_check.cpp -- a driver for the host planner (ACSR construction, work
// plan, tiling arrangements) built on its own with the address and
// undefined-behaviour sanitizers by the CPU tests.  It reads one request per
// line on stdin and prints one JSON line per request:
//
//   desc <L> <flags> <n_terms> <10 ints per term>   build from a descriptor
//   mask <L> <L*L characters 0/1>                   build from a dense mask
//   tile <method> <m> <n> <stretch>                 tile the last build
//
// A build prints its status, row_ptr, the expanded column indices, the plan
// (groups, rows, tiles, row masks) and its counters; a tiling prints its
// statistics and anchors.  The tests compare the output with the regular
// library's, so any sanitizer report (which ends the process) or any
// difference fails them.
#include <cstdio>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "../../paper_2407_16847_amd/csrc/acsr_host.hpp"
#include "../../paper_2407_16847_amd/csrc/tiling.hpp"

using namespace splat;

namespace {

template <typename T>
void put_list(std::ostream& o, const char* name, const std::vector<T>& v) {
  o << "\"" << name << "\":[";
  for (size_t k = 0; k < v.size(); ++k) o << (k ? "," : "") << v[k];
  o << "]";
}

void print_build(splat_status s, const HostAcsr& a, const std::string& err) {
  std::ostringstream o;
  o << "{\"status\":" << (int)s;
  if (s != SPLAT_OK) {
    o << ",\"error\":\"" << (err.find('"') == std::string::npos ? err : "?") << "\"}";
    std::cout << o.str() << std::endl;
    return;
  }
  std::vector<int32_t> cols;
  for (int32_t i = 0; i < a.L; ++i)
    for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
      const Run& q = a.runs[i].r[r];
      for (int32_t k = 0; k < q.count; ++k) cols.push_back(q.start + q.stride * k);
    }
  std::vector<int32_t> groups, tiles;
  for (const Group& g : a.groups) {
    groups.push_back(g.row_off);
    groups.push_back(g.nrows);
    groups.push_back(g.tile_begin);
    groups.push_back(g.tile_end);
  }
  for (const Tile& t : a.tiles) {
    tiles.push_back(t.kb);
    tiles.push_back(t.ks);
    tiles.push_back(t.nk);
    tiles.push_back(t.flags);
    tiles.push_back(t.mask_block);
  }
  o << ",\"nnz\":" << a.nnz << ",\"computed\":" << a.computed << ",\"n_full\":" << a.n_full
    << ",\"max_runs\":" << a.max_runs << ",\"columns\":" << a.col_regular << ",";
  put_list(o, "row_ptr", a.row_ptr);
  o << ",";
  put_list(o, "col_idx", cols);
  o << ",";
  put_list(o, "groups", groups);
  o << ",";
  put_list(o, "rows", a.rows);
  o << ",";
  put_list(o, "tiles", tiles);
  o << ",";
  put_list(o, "masks", a.masks);
  o << "}";
  std::cout << o.str() << std::endl;
}

}  // namespace

int main() {
  std::string line;
  HostAcsr last;
  bool have = false;
  while (std::getline(std::cin, line)) {
    std::istringstream in(line);
    std::string cmd;
    in >> cmd;
    if (cmd == "desc") {
      splat_pattern_desc d{};
      uint32_t flags = 0;
      in >> d.L >> flags >> d.n_terms;
      for (int t = 0; t < d.n_terms && t < SPLAT_MAX_TERMS; ++t) {
        splat_affine_term& x = d.terms[t];
        in >> x.row_lo >> x.row_hi >> x.group >> x.lo_i >> x.lo_q >> x.lo_c >> x.hi_i >> x.hi_q >>
            x.hi_c >> x.stride;
      }
      HostAcsr a;
      std::string err;
      const splat_status s = build_from_desc(d, a, err, flags);
      print_build(s, a, err);
      if (s == SPLAT_OK) last = std::move(a), have = true;
    } else if (cmd == "mask") {
      int32_t L = 0;
      std::string bits;
      in >> L >> bits;
      if (L < 1 || (int64_t)bits.size() != (int64_t)L * L) {
        std::cout << "{\"status\":-1}" << std::endl;
        continue;
      }
      std::vector<uint8_t> m(bits.size());
      for (size_t k = 0; k < bits.size(); ++k) m[k] = bits[k] == '1';
      HostAcsr a;
      std::string err;
      const splat_status s = build_from_mask(L, m.data(), a, err);
      print_build(s, a, err);
      if (s == SPLAT_OK) last = std::move(a), have = true;
    } else if (cmd == "tile") {
      int32_t method = 0, m = 0, n = 0, stretch = 0;
      in >> method >> m >> n >> stretch;
      if (!have) {
        std::cout << "{\"status\":-1}" << std::endl;
        continue;
      }
      TilingStats st;
      std::vector<int32_t> anchors;
      std::string err;
      const splat_status s = tile_mask(last, method, m, n, stretch, &anchors, st, err);
      std::ostringstream o;
      o << "{\"status\":" << (int)s;
      if (s == SPLAT_OK) {
        o << ",\"blocks\":" << st.blocks << ",\"divergent\":" << st.divergent
          << ",\"redundant\":" << st.redundant << ",\"stretch\":" << st.stretch
          << ",\"iterations\":" << st.iterations << ",";
        put_list(o, "anchors", anchors);
      }
      o << "}";
      std::cout << o.str() << std::endl;
    } else if (!cmd.empty()) {
      std::cout << "{\"status\":-2}" << std::endl;
    }
  }
  return 0;
}
