// tiling.cpp -- thread-block arrangements of a mask for the SDDMM cost model
// of section 7 (host C++ only; a diagnostic, the kernels use the row-group
// plan of acsr_host.cpp).
//
// A thread-block of m x n threads with anchor t and stretch s computes the
// points t + (i*s, j*s), i < m, j < n (section 7.2).  Poset tiling
// (section 7.3) covers the mask's point set P in rounds: every round takes
// the uncovered points that no other uncovered point comes before (x' <= x
// and y' <= y) as new anchors and removes what their blocks compute.  Naive
// Tiling (Appendix C) cuts the mask into patches of m consecutive rows and
// tiles each from its leftmost to its rightmost point with ceil(width / n)
// unstretched blocks, n columns apart.  The grid arrangement places
// unstretched blocks at every multiple of (m, n) whose block meets P.  For
// every arrangement the cost-model quantities of section 7.2 are reported:
// divergent threads (computed points outside P), redundant threads, reuse,
// coalescing (mean 1/stretch) and cost.
#include "tiling.hpp"

#include <algorithm>
#include <vector>

namespace splat {
namespace {

// A bitmap of rows x cols bits, row-major, 64-bit words.
struct Bitmap {
  int32_t rows, cols, words;
  std::vector<uint64_t> w;
  Bitmap(int32_t r, int32_t c) : rows(r), cols(c), words((c + 63) / 64), w((size_t)r * words, 0ull) {}
  uint64_t* row(int32_t x) { return w.data() + (size_t)x * words; }
  const uint64_t* row(int32_t x) const { return w.data() + (size_t)x * words; }
  bool get(int32_t x, int32_t y) const { return (row(x)[y >> 6] >> (y & 63)) & 1ull; }
  void set(int32_t x, int32_t y) { row(x)[y >> 6] |= 1ull << (y & 63); }
  void clear(int32_t x, int32_t y) { row(x)[y >> 6] &= ~(1ull << (y & 63)); }
  int64_t count() const {
    int64_t c = 0;
    for (uint64_t v : w) c += __builtin_popcountll(v);
    return c;
  }
};

Bitmap point_set(const HostAcsr& a) {
  Bitmap p(a.L, a.L);
  for (int32_t i = 0; i < a.L; ++i)
    for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
      const Run& q = a.runs[i].r[r];
      for (int32_t k = 0; k < q.count; ++k) p.set(i, q.start + q.stride * k);
    }
  return p;
}

// Marks the block's computed points in `comp` (which has room for blocks
// reaching past the mask) and removes them from `rem` (mask-sized).
void place(int32_t x, int32_t y, int32_t m, int32_t n, int32_t s, Bitmap& comp, Bitmap* rem) {
  for (int32_t i = 0; i < m; ++i) {
    const int32_t r = x + i * s;
    for (int32_t j = 0; j < n; ++j) {
      const int32_t c = y + j * s;
      comp.set(r, c);
      if (rem && r < rem->rows && c < rem->cols) rem->clear(r, c);
    }
  }
}

void finish(const Bitmap& comp, int64_t points, int32_t m, int32_t n, int32_t s, int64_t blocks,
            TilingStats& st) {
  st.blocks = blocks;
  st.points = points;
  st.stretch = s;
  st.divergent = comp.count() - points;   // every point of P is computed
  st.redundant = blocks * m * n - points - st.divergent;
  st.reuse = blocks ? (double)points / ((double)blocks * m * n) : 1.0;
  st.coalesced = 1.0 / s;
  st.cost = (double)blocks / st.coalesced;
}

// One poset tiling with a fixed stretch.
void poset(const HostAcsr& a, const Bitmap& P, int64_t points, int32_t m, int32_t n, int32_t s,
           std::vector<int32_t>* anchors, TilingStats& st) {
  const int32_t L = a.L;
  Bitmap rem = P;
  Bitmap comp(L + (m - 1) * s, L + (n - 1) * s);
  std::vector<int32_t> first(L, 0);   // first word of a row that may hold an uncovered point
  std::vector<int32_t> top;
  int64_t blocks = 0, left = points;
  int32_t rounds = 0;
  if (anchors) anchors->clear();
  while (left > 0) {
    // the round's minimal set: a row's leftmost uncovered point, when every
    // earlier row's uncovered points all lie strictly to its right
    top.clear();
    int32_t run_min = L;
    for (int32_t x = 0; x < L; ++x) {
      const uint64_t* w = rem.row(x);
      int32_t& f = first[x];
      while (f < rem.words && w[f] == 0) ++f;
      if (f == rem.words) continue;
      const int32_t y = 64 * f + __builtin_ctzll(w[f]);
      if (y < run_min) {
        top.push_back(x);
        top.push_back(y);
        run_min = y;
      }
    }
    for (size_t k = 0; k < top.size(); k += 2) {
      place(top[k], top[k + 1], m, n, s, comp, &rem);
      ++blocks;
      if (anchors) {
        anchors->push_back(top[k]);
        anchors->push_back(top[k + 1]);
      }
    }
    left = rem.count();
    ++rounds;
  }
  finish(comp, points, m, n, s, blocks, st);
  st.iterations = rounds;
}

// The stride shared by every non-empty row when each is a single run of
// stride > 1 (a strided mask in the paper's sense), else 1.
int32_t common_stride(const HostAcsr& a) {
  int32_t X = 0;
  for (int32_t i = 0; i < a.L; ++i) {
    int32_t runs = 0, stride = 1;
    for (int r = 0; r < SPLAT_MAX_RUNS; ++r)
      if (a.runs[i].r[r].count > 0) {
        ++runs;
        stride = a.runs[i].r[r].count > 1 ? a.runs[i].r[r].stride : 0;
      }
    if (runs == 0) continue;
    if (runs > 1) return 1;
    if (stride == 0) continue;   // a single point fits any stride
    if (stride == 1) return 1;
    if (X == 0) X = stride;
    if (stride != X) return 1;
  }
  return X > 1 ? X : 1;
}

// Bounds the bitmap of computed points, which reaches (m-1)*s rows and
// (n-1)*s columns past the mask.
bool fits(int32_t L, int32_t m, int32_t n, int32_t s) {
  return (int64_t)(m - 1) * s <= (int64_t)L + 1024 && (int64_t)(n - 1) * s <= (int64_t)L + 1024;
}

}  // namespace

splat_status tile_mask(const HostAcsr& a, int32_t method, int32_t m, int32_t n, int32_t stretch,
                       std::vector<int32_t>* anchors, TilingStats& st, std::string& err) {
  if (m < 1 || n < 1 || m > 1024 || n > 1024) {
    err = "thread-block dimensions must be in [1, 1024]";
    return SPLAT_ERR_INVALID_ARG;
  }
  if (stretch < 0 || stretch > a.L) {
    err = "stretch must be 0 (select) or in [1, L]";
    return SPLAT_ERR_INVALID_ARG;
  }
  if (stretch >= 1 && !fits(a.L, m, n, stretch)) {
    err = "a block may reach at most L + 1024 past its anchor ((m-1)*s, (n-1)*s <= L + 1024)";
    return SPLAT_ERR_INVALID_ARG;
  }
  if (a.L > SPLAT_TILING_MAX_L) {
    err = "tiling diagnostics are limited to L <= " + std::to_string(SPLAT_TILING_MAX_L);
    return SPLAT_ERR_UNSUPPORTED;
  }
  st = TilingStats();
  const Bitmap P = point_set(a);
  const int64_t points = a.nnz;
  if (method == SPLAT_TILING_GRID) {
    if (stretch > 1) {
      err = "the grid arrangement is unstretched";
      return SPLAT_ERR_INVALID_ARG;
    }
    Bitmap comp(a.L + m - 1, a.L + n - 1);
    int64_t blocks = 0;
    if (anchors) anchors->clear();
    for (int32_t x = 0; x < a.L; x += m)
      for (int32_t y = 0; y < a.L; y += n) {
        bool meets = false;
        for (int32_t i = x; i < std::min(a.L, x + m) && !meets; ++i)
          for (int32_t j = y; j < std::min(a.L, y + n); ++j)
            if (P.get(i, j)) {
              meets = true;
              break;
            }
        if (!meets) continue;
        place(x, y, m, n, 1, comp, nullptr);
        ++blocks;
        if (anchors) {
          anchors->push_back(x);
          anchors->push_back(y);
        }
      }
    finish(comp, points, m, n, 1, blocks, st);
    st.iterations = 1;
    return SPLAT_OK;
  }
  if (method == SPLAT_TILING_NAIVE) {
    if (stretch > 1) {
      err = "naive tiling is unstretched";
      return SPLAT_ERR_INVALID_ARG;
    }
    Bitmap comp(a.L + m - 1, a.L + n - 1);
    int64_t blocks = 0;
    if (anchors) anchors->clear();
    for (int32_t x = 0; x < a.L; x += m) {
      // the patch's leftmost and rightmost points, from the rows' runs
      int32_t left = a.L, right = -1;
      for (int32_t i = x; i < std::min(a.L, x + m); ++i)
        for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
          const Run& q = a.runs[i].r[r];
          if (q.count <= 0) continue;
          left = std::min(left, q.start);
          right = std::max(right, q.start + q.stride * (q.count - 1));
        }
      if (right < 0) continue;   // a patch without points takes no block
      const int32_t nb = (right - left + n) / n;
      for (int32_t k = 0; k < nb; ++k) {
        place(x, left + k * n, m, n, 1, comp, nullptr);
        ++blocks;
        if (anchors) {
          anchors->push_back(x);
          anchors->push_back(left + k * n);
        }
      }
    }
    finish(comp, points, m, n, 1, blocks, st);
    st.iterations = 1;
    return SPLAT_OK;
  }
  if (method != SPLAT_TILING_POSET) {
    err = "method must be SPLAT_TILING_POSET, SPLAT_TILING_GRID or SPLAT_TILING_NAIVE";
    return SPLAT_ERR_INVALID_ARG;
  }
  if (stretch >= 1) {
    poset(a, P, points, m, n, stretch, anchors, st);
    return SPLAT_OK;
  }
  // stretch selection: 1 for polygonal masks; for a strided mask of stride
  // X the divisors of X, keeping the lowest cost (ties: fewer blocks)
  const int32_t X = common_stride(a);
  bool have = false;
  for (int32_t s = 1; s <= X; ++s) {
    if (X % s || !fits(a.L, m, n, s)) continue;
    TilingStats cand;
    std::vector<int32_t> anc;
    poset(a, P, points, m, n, s, anchors ? &anc : nullptr, cand);
    if (!have || cand.cost < st.cost || (cand.cost == st.cost && cand.blocks < st.blocks)) {
      st = cand;
      if (anchors) *anchors = std::move(anc);
      have = true;
    }
  }
  return SPLAT_OK;
}

}  // namespace splat
