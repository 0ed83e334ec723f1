// acsr_host.cpp -- just-in-time analysis of a regular mask into ACSR runs and
// the kernels' work plan.  Host C++ only; no HIP calls.
//
// Construction (section 5.1): every row's column set is compressed to affine
// runs.  The paper gives each row one pair of affine indices (a, b), found
// from the row's first two columns and verified on the rest; here a row may
// hold up to SPLAT_MAX_RUNS runs so that unions such as window + global
// tokens stay in O(rows) metadata.  Integers only: a run's stride is 1/a and
// its start is -b/a, so no real-valued index is ever rounded.
//
// Planning: rows whose single run has the same stride and residue are grouped
// (section 5.2: rows with identical affine structure share a warp; section
// 8.2, linear-transformation alignment), and each group's column span
// (section 8.2, span specialisation: only the columns its rows reach) is cut
// into key tiles -- contiguous, or gathered along the group's common stride
// when that covers more of its columns.  Groups are launched heaviest first.
#include "acsr_host.hpp"

#include <algorithm>
#include <cstring>
#include <map>
#include <utility>

namespace splat {
namespace {

// ---- a bitmap over [0, L) -------------------------------------------------
struct Bits {
  std::vector<uint64_t> w;
  int32_t n = 0;
  explicit Bits(int32_t n_) : w((n_ + 63) / 64, 0ull), n(n_) {}
  void clear() { std::fill(w.begin(), w.end(), 0ull); }
  void set(int32_t j) { w[j >> 6] |= 1ull << (j & 63); }
  void set_range(int32_t lo, int32_t hi) {  // inclusive, lo <= hi
    int32_t wl = lo >> 6, wh = hi >> 6;
    if (wl == wh) {
      w[wl] |= range_bits(lo & 63, hi & 63);
      return;
    }
    w[wl] |= range_bits(lo & 63, 63);
    for (int32_t k = wl + 1; k < wh; ++k) w[k] = ~0ull;
    w[wh] |= range_bits(0, hi & 63);
  }
  void set_progression(int32_t start, int32_t stride, int32_t count) {
    if (count <= 0) return;
    if (stride == 1) {
      set_range(start, start + count - 1);
      return;
    }
    for (int32_t k = 0; k < count; ++k) set(start + stride * k);
  }
  // first set bit >= pos, or -1
  int32_t next(int32_t pos) const {
    if (pos >= n) return -1;
    int32_t wi = pos >> 6;
    uint64_t cur = w[wi] & (~0ull << (pos & 63));
    while (true) {
      if (cur) {
        int32_t j = (wi << 6) + __builtin_ctzll(cur);
        return j < n ? j : -1;
      }
      if (++wi >= (int32_t)w.size()) return -1;
      cur = w[wi];
    }
  }
  int32_t count_range(int32_t lo, int32_t hi) const {  // inclusive
    int32_t c = 0;
    for (int32_t wi = lo >> 6; wi <= (hi >> 6); ++wi) {
      uint64_t m = w[wi];
      int32_t a = (wi == (lo >> 6)) ? (lo & 63) : 0;
      int32_t b = (wi == (hi >> 6)) ? (hi & 63) : 63;
      c += __builtin_popcountll(m & range_bits(a, b));
    }
    return c;
  }
};

// Canonical decomposition of an ascending column list into runs: maximal
// contiguous runs first; otherwise a run keeps the gap of its first two
// columns and stops before a column that starts a contiguous pair.  A lone
// column is a run of stride 1 and count 1.  Returns the number of runs, or
// -1 if more than SPLAT_MAX_RUNS would be needed.
int32_t decompose(const std::vector<int32_t>& c, RowRuns& rr) {
  std::memset(&rr, 0, sizeof(rr));
  for (int r = 0; r < SPLAT_MAX_RUNS; ++r) rr.r[r].stride = 1;
  const int32_t n = (int32_t)c.size();
  int32_t p = 0, nr = 0, prefix = 0;
  auto starts_pair = [&](int32_t q) { return q + 1 < n && c[q + 1] == c[q] + 1; };
  while (p < n) {
    int32_t stride = 1, q = p;
    if (starts_pair(p)) {
      while (starts_pair(q)) ++q;
    } else if (p + 1 < n && !starts_pair(p + 1)) {
      stride = c[p + 1] - c[p];
      q = p + 1;
      while (q + 1 < n && c[q + 1] - c[q] == stride && !starts_pair(q + 1)) ++q;
    }
    if (nr == SPLAT_MAX_RUNS) return -1;
    rr.r[nr] = Run{c[p], stride, q - p + 1, prefix};
    prefix += q - p + 1;
    ++nr;
    p = q + 1;
  }
  return nr;
}

splat_status finish_rows(HostAcsr& a, std::string& err) {
  a.row_ptr.assign(a.L + 1, 0);
  int64_t acc = 0;
  for (int32_t i = 0; i < a.L; ++i) {
    int32_t n = 0;
    for (int r = 0; r < SPLAT_MAX_RUNS; ++r) n += a.runs[i].r[r].count;
    acc += n;
    if (acc >= (int64_t(1) << 31)) {
      err = "mask has 2^31 or more non-zeros per head";
      return SPLAT_ERR_UNSUPPORTED;
    }
    a.row_ptr[i + 1] = (int32_t)acc;
    a.max_row_nnz = std::max(a.max_row_nnz, n);
    a.max_runs = std::max(a.max_runs, a.nruns[i]);
  }
  a.nnz = acc;
  plan_work(a);
  return SPLAT_OK;
}

// Column-wise analysis (section 5.2): the mask's transpose is affine-
// compressible when every column's rows form one affine run.  Rows are
// visited in ascending order, so each column's rows arrive sorted; a column
// is one run iff every gap equals its first gap.
splat_status analyse_columns(HostAcsr& a, std::string& err) {
  const int32_t L = a.L;
  if (a.nnz > (int64_t(1) << 28)) {
    err = "the column-wise analysis is limited to 2^28 non-zeros per head";
    return SPLAT_ERR_UNSUPPORTED;
  }
  std::vector<ColRun> c(L, ColRun{0, 1, 0, 0});
  std::vector<int32_t> last(L, -1);
  bool regular = true;
  for (int32_t i = 0; i < L && regular; ++i) {
    for (int r = 0; r < SPLAT_MAX_RUNS && regular; ++r) {
      const Run& q = a.runs[i].r[r];
      for (int32_t k = 0; k < q.count; ++k) {
        const int32_t j = q.start + q.stride * k;
        ColRun& cj = c[j];
        if (cj.count == 0) {
          cj.start = i;
        } else if (cj.count == 1) {
          cj.stride = i - cj.start;
        } else if (i - last[j] != cj.stride) {
          regular = false;
          break;
        }
        last[j] = i;
        ++cj.count;
      }
    }
  }
  a.cols.clear();
  a.col_regular = regular ? 1 : 0;
  if (!regular) return SPLAT_OK;
  int64_t ptr = 0;
  for (int32_t j = 0; j < L; ++j) {
    c[j].ptr = (int32_t)ptr;
    ptr += c[j].count;
  }
  a.cols = std::move(c);
  return SPLAT_OK;
}

bool term_ok(const splat_affine_term& t, int32_t L) {
  const int32_t lim = 1 << 20;
  auto small = [&](int32_t v) { return v >= -lim && v <= lim; };
  return t.row_lo >= 0 && t.row_lo <= t.row_hi && t.row_hi <= L && t.group >= 1 && t.stride >= 1 &&
         small(t.lo_i) && small(t.lo_q) && small(t.lo_c) && small(t.hi_i) && small(t.hi_q) &&
         small(t.hi_c) && t.stride <= lim;
}

}  // namespace

// ---------------------------------------------------------------------------
splat_status build_from_desc(const splat_pattern_desc& d, HostAcsr& a, std::string& err,
                            uint32_t plan_flags) {
  if (d.L < 1 || d.L > SPLAT_MAX_L) {
    err = "L must be in [1, " + std::to_string(SPLAT_MAX_L) + "], got " + std::to_string(d.L);
    return SPLAT_ERR_INVALID_ARG;
  }
  if (d.n_terms < 0 || d.n_terms > SPLAT_MAX_TERMS) {
    err = "n_terms must be in [0, " + std::to_string(SPLAT_MAX_TERMS) + "]";
    return SPLAT_ERR_INVALID_ARG;
  }
  for (int t = 0; t < d.n_terms; ++t) {
    if (!term_ok(d.terms[t], d.L)) {
      err = "term " + std::to_string(t) + " is malformed (row range, group >= 1, stride >= 1, |coefficients| <= 2^20)";
      return SPLAT_ERR_INVALID_ARG;
    }
  }
  const int32_t L = d.L;
  a = HostAcsr();
  a.L = L;
  a.plan_flags = plan_flags;
  a.runs.resize(L);
  a.nruns.assign(L, 0);
  Bits row(L);
  std::vector<int32_t> cols;
  cols.reserve(L);
  for (int32_t i = 0; i < L; ++i) {
    row.clear();
    for (int t = 0; t < d.n_terms; ++t) {
      const splat_affine_term& T = d.terms[t];
      if (i < T.row_lo || i >= T.row_hi) continue;
      const int64_t qg = int64_t(i / T.group) * T.group;
      int64_t lo = int64_t(T.lo_i) * i + int64_t(T.lo_q) * qg + T.lo_c;
      int64_t hi = int64_t(T.hi_i) * i + int64_t(T.hi_q) * qg + T.hi_c;
      const int64_t s = T.stride;
      if (lo < 0) lo += ((-lo + s - 1) / s) * s;  // keep lo mod s
      if (hi > L - 1) hi = L - 1;
      if (lo > hi) continue;
      row.set_progression((int32_t)lo, (int32_t)s, (int32_t)((hi - lo) / s + 1));
    }
    cols.clear();
    for (int32_t j = row.next(0); j >= 0; j = row.next(j + 1)) cols.push_back(j);
    const int32_t nr = decompose(cols, a.runs[i]);
    if (nr < 0) {
      err = "row " + std::to_string(i) + " needs more than " + std::to_string(SPLAT_MAX_RUNS) +
            " affine runs";
      return SPLAT_ERR_UNSUPPORTED;
    }
    a.nruns[i] = nr;
  }
  splat_status s = finish_rows(a, err);
  if (s == SPLAT_OK && (plan_flags & SPLAT_PLAN_COLUMNS)) s = analyse_columns(a, err);
  return s;
}

splat_status build_from_mask(int32_t L, const uint8_t* mask, HostAcsr& a, std::string& err) {
  if (L < 1 || L > SPLAT_MAX_L) {
    err = "L must be in [1, " + std::to_string(SPLAT_MAX_L) + "]";
    return SPLAT_ERR_INVALID_ARG;
  }
  if (!mask) {
    err = "mask is NULL";
    return SPLAT_ERR_INVALID_ARG;
  }
  a = HostAcsr();
  a.L = L;
  a.runs.resize(L);
  a.nruns.assign(L, 0);
  std::vector<int32_t> cols;
  for (int32_t i = 0; i < L; ++i) {
    cols.clear();
    const uint8_t* m = mask + int64_t(i) * L;
    for (int32_t j = 0; j < L; ++j)
      if (m[j]) cols.push_back(j);
    RowRuns& rr = a.runs[i];
    std::memset(&rr, 0, sizeof(rr));
    for (int r = 0; r < SPLAT_MAX_RUNS; ++r) rr.r[r].stride = 1;
    const int32_t n = (int32_t)cols.size();
    if (n == 0) continue;
    // Two-point solve: a = 1 / (i1 - i0), b = -a * i0, held as stride = i1 - i0
    // and start = i0; then every later column must sit one step further.
    int32_t stride = n >= 2 ? cols[1] - cols[0] : 1;
    for (int32_t t = 1; t < n; ++t) {
      if (cols[t] - cols[t - 1] != stride) {
        err = "row " + std::to_string(i) + " is not affine-compressible: columns " +
              std::to_string(cols[t - 1]) + ", " + std::to_string(cols[t]) + " break stride " +
              std::to_string(stride);
        return SPLAT_ERR_NOT_REGULAR;
      }
    }
    rr.r[0] = Run{cols[0], stride, n, 0};
    a.nruns[i] = 1;
  }
  return finish_rows(a, err);
}

// ---------------------------------------------------------------------------
void plan_work(HostAcsr& a) {
  const int32_t L = a.L;
  // 1. group rows by affine signature: (stride, start mod stride) of a row
  //    held in one strided run, (1, 0) for every other row
  std::map<std::pair<int32_t, int32_t>, std::vector<int32_t>> classes;
  for (int32_t i = 0; i < L; ++i) {
    std::pair<int32_t, int32_t> sig(1, 0);
    const Run& r0 = a.runs[i].r[0];
    if (a.nruns[i] == 1 && r0.stride > 1) sig = {r0.stride, r0.start % r0.stride};
    classes[sig].push_back(i);
  }
  a.rows.clear();
  a.groups.clear();
  a.tiles.clear();
  a.computed = 0;
  a.n_full = 0;
  a.masks.clear();
  struct Pending {
    Group g;
    std::vector<Tile> t;
  };
  std::vector<Pending> pend;
  Bits U(L);
  for (auto& kv : classes) {
    const std::vector<int32_t>& rows = kv.second;
    for (size_t off = 0; off < rows.size(); off += kBM) {
      const int32_t nrows = (int32_t)std::min<size_t>(kBM, rows.size() - off);
      Pending p;
      p.g.row_off = (int32_t)a.rows.size();
      p.g.nrows = nrows;
      for (int32_t m = 0; m < nrows; ++m) a.rows.push_back(rows[off + m]);
      // union of the group's columns; strides present in the group
      U.clear();
      std::vector<int32_t> strides;
      for (int32_t m = 0; m < nrows; ++m) {
        const RowRuns& rr = a.runs[rows[off + m]];
        for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
          const Run& q = rr.r[r];
          if (q.count <= 0) continue;
          U.set_progression(q.start, q.stride, q.count);
          if (q.stride > 1 && q.count > 1 &&
              std::find(strides.begin(), strides.end(), q.stride) == strides.end())
            strides.push_back(q.stride);
        }
      }
      // the kernels evaluate a gathered tile of step s in O(1) per run only
      // when every run has stride 1 or s
      auto gather_ok = [&](int32_t s) {
        for (int32_t x : strides)
          if (x != s) return false;
        return true;
      };
      // Without span specialisation every group walks the whole key range
      // [0, L) in contiguous tiles and evaluates the predicate on each.
      const bool no_span = (a.plan_flags & SPLAT_PLAN_NO_SPAN) != 0;
      int32_t pos = 0;
      for (int32_t c = no_span ? 0 : U.next(pos); c >= 0 && c < L; c = no_span ? pos : U.next(pos)) {
        Tile t{};
        if (no_span) {
          t.kb = c, t.ks = 1, t.nk = std::min(kBN, L - c);
          pos = c + t.nk;
        } else {
          const int32_t dense_end = std::min(L - 1, c + kBN - 1);
          const int32_t k1 = U.count_range(c, dense_end);
          int32_t k2 = 0, last = c, step = 1;
          const int32_t nx = U.next(c + 1);
          if (nx > 0 && nx - c > 1 && gather_ok(nx - c)) {
            step = nx - c;
            k2 = 1;
            while (k2 < kBN) {
              const int32_t y = U.next(last + 1);
              if (y < 0 || y - last != step) break;
              last = y;
              ++k2;
            }
          }
          if (k2 > k1) {
            t.kb = c, t.ks = step, t.nk = k2;
            pos = last + 1;
          } else {
            t.kb = c, t.ks = 1, t.nk = dense_end - c + 1;
            pos = dense_end + 1;
          }
        }
        t.mask_block = -1;
        // per-row membership, per-wavefront state
        uint64_t rb[kBM];
        const uint64_t all = t.nk == 64 ? ~0ull : ((1ull << t.nk) - 1);
        bool group_full = t.nk == kBN;
        bool any_partial = false;
        for (int32_t m = 0; m < kBM; ++m)
          rb[m] = m < nrows ? tile_row_bits(a.runs[rows[off + m]], t.kb, t.ks, t.nk) : 0ull;
        for (int32_t w = 0; w < kWavesPerGroup; ++w) {
          bool full = t.nk == kBN, empty = true;
          for (int32_t m = w * kWaveRows; m < (w + 1) * kWaveRows && m < nrows; ++m) {
            full = full && rb[m] == all;
            empty = empty && rb[m] == 0;
          }
          if (w * kWaveRows >= nrows) full = false;   // no real row: nothing to do
          // without span specialisation a wavefront with real rows computes every tile
          if (no_span && w * kWaveRows < nrows) empty = false;
          const int32_t st = empty ? kWaveEmpty : (full ? kWaveFull : kWavePartial);
          t.flags |= st << (kWaveShift + 2 * w);
          group_full = group_full && (st == kWaveFull || w * kWaveRows >= nrows);
          any_partial = any_partial || st == kWavePartial;
          if (st != kWaveEmpty) a.computed += int64_t(kWaveRows) * kBN;
        }
        if (group_full) t.flags |= kTileFull;
        if (any_partial) {
          t.mask_block = (int32_t)(a.masks.size() / kBM);
          a.masks.insert(a.masks.end(), rb, rb + kBM);
        }
        p.t.push_back(t);
        if (pos >= L) break;
      }
      pend.push_back(std::move(p));
    }
  }
  // 2. heaviest groups first (longest-processing-time order), stable
  std::stable_sort(pend.begin(), pend.end(),
                   [](const Pending& x, const Pending& y) { return x.t.size() > y.t.size(); });
  for (Pending& p : pend) {
    p.g.tile_begin = (int32_t)a.tiles.size();
    for (const Tile& t : p.t) {
      a.tiles.push_back(t);
      if (t.flags & kTileFull) ++a.n_full;
    }
    p.g.tile_end = (int32_t)a.tiles.size();
    a.groups.push_back(p.g);
  }
}

// ---------------------------------------------------------------------------
// descriptor helpers
namespace {
splat_affine_term term(int32_t L) {
  splat_affine_term t;
  std::memset(&t, 0, sizeof(t));
  t.row_lo = 0;
  t.row_hi = L;
  t.group = 1;
  t.stride = 1;
  return t;
}
bool begin(int32_t L, splat_pattern_desc* out) {
  if (!out || L < 1 || L > SPLAT_MAX_L) return false;
  std::memset(out, 0, sizeof(*out));
  out->L = L;
  return true;
}
}  // namespace

splat_status pattern_window(int32_t L, int32_t w, splat_pattern_desc* out) {
  if (!begin(L, out) || w < 0) return SPLAT_ERR_INVALID_ARG;
  splat_affine_term t = term(L);
  t.lo_i = 1, t.lo_c = -w;   // j >= i - w
  t.hi_i = 1, t.hi_c = w;    // j <= i + w
  out->terms[out->n_terms++] = t;
  return SPLAT_OK;
}

splat_status pattern_blocked(int32_t L, int32_t block, splat_pattern_desc* out) {
  if (!begin(L, out) || block < 1) return SPLAT_ERR_INVALID_ARG;
  splat_affine_term t = term(L);
  t.group = block;
  t.lo_q = 1, t.lo_c = -block;     // start of the previous block
  t.hi_q = 1, t.hi_c = block - 1;  // end of the own block
  out->terms[out->n_terms++] = t;
  return SPLAT_OK;
}

splat_status pattern_strided_local(int32_t L, int32_t local, int32_t stride, splat_pattern_desc* out) {
  if (!begin(L, out) || local < 1 || stride < 1) return SPLAT_ERR_INVALID_ARG;
  splat_affine_term t = term(L);
  t.lo_i = 1, t.lo_c = -(local - 1);  // causal local window [i - local + 1, i]
  t.hi_i = 1;
  out->terms[out->n_terms++] = t;
  splat_affine_term s = term(L);
  s.lo_c = stride - 1;                // columns stride-1, 2*stride-1, ... up to i
  s.hi_i = 1;
  s.stride = stride;
  out->terms[out->n_terms++] = s;
  return SPLAT_OK;
}

splat_status pattern_dilated(int32_t L, int32_t w, int32_t dilation, splat_pattern_desc* out) {
  if (!begin(L, out) || w < 0 || dilation < 1 || int64_t(w) * dilation > (1 << 20))
    return SPLAT_ERR_INVALID_ARG;
  splat_affine_term t = term(L);
  t.lo_i = 1, t.lo_c = -w * dilation;
  t.hi_i = 1, t.hi_c = w * dilation;
  t.stride = dilation;
  out->terms[out->n_terms++] = t;
  return SPLAT_OK;
}

splat_status pattern_window_global(int32_t L, int32_t w, int32_t n_global, splat_pattern_desc* out) {
  if (!begin(L, out) || w < 0 || n_global < 0) return SPLAT_ERR_INVALID_ARG;
  splat_affine_term t = term(L);
  t.lo_i = 1, t.lo_c = -w;
  t.hi_i = 1, t.hi_c = w;
  out->terms[out->n_terms++] = t;
  if (n_global > 0) {
    splat_affine_term gr = term(L);   // global rows see every column
    gr.row_hi = std::min(L, n_global);
    gr.hi_c = L - 1;
    out->terms[out->n_terms++] = gr;
    splat_affine_term gc = term(L);   // every row sees the global columns
    gc.hi_c = std::min(L, n_global) - 1;
    out->terms[out->n_terms++] = gc;
  }
  return SPLAT_OK;
}

splat_status pattern_full(int32_t L, splat_pattern_desc* out) {
  if (!begin(L, out)) return SPLAT_ERR_INVALID_ARG;
  splat_affine_term t = term(L);
  t.hi_c = L - 1;
  out->terms[out->n_terms++] = t;
  return SPLAT_OK;
}

}  // namespace splat
