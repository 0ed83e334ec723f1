// api.hip -- the C ABI declared in include/splat.h: argument validation,
// ACSR handle lifetime (host analysis + one device upload) and kernel dispatch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <mutex>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>

#include "../../include/splat.h"
#include "acsr_host.hpp"
#include "launch.hpp"
#include "tiling.hpp"

using splat::DevAcsr;
using splat::HostAcsr;

struct splat_acsr {
  HostAcsr host;
  int device = -1;
  void* dmem = nullptr;
  DevAcsr dev{};
};

namespace {

thread_local std::string g_err;

splat_status fail(splat_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

splat_status ok() { return SPLAT_OK; }

// One allocation holds every metadata array, each 256-byte aligned.
splat_status upload(splat_acsr* h) {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n == 0) {
    (void)hipGetLastError();  // a missing GPU is not an error for a host-only handle
    h->device = -1;
    return SPLAT_OK;
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPLAT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  e = splat::prepare_fused_mfma();
  if (e != hipSuccess)
    return fail(SPLAT_ERR_HIP, "hipFuncSetAttribute (fused kernel LDS): %s", hipGetErrorString(e));
  const HostAcsr& a = h->host;
  auto al = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t s_rowptr = al(sizeof(int32_t) * (a.L + 1));
  const size_t s_runs = al(sizeof(splat::RowRuns) * a.L);
  const size_t s_rows = al(sizeof(int32_t) * a.L);
  const size_t s_groups = al(sizeof(splat::Group) * a.groups.size());
  const size_t s_tiles = al(sizeof(splat::Tile) * (a.tiles.size() + 1));
  // one extra zero block: tiles without masks still issue (unused) mask loads
  const size_t s_masks = al(sizeof(uint64_t) * (a.masks.size() + splat::kBM));
  const size_t s_cols = al(sizeof(splat::ColRun) * a.cols.size());
  const size_t total = s_rowptr + s_runs + s_rows + s_groups + s_tiles + s_masks + s_cols;
  void* mem = nullptr;
  e = hipMalloc(&mem, total);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(SPLAT_ERR_OOM, "hipMalloc(%zu) for ACSR metadata: %s", total, hipGetErrorString(e));
  }
  e = hipMemset(mem, 0, total);
  if (e != hipSuccess) {
    (void)hipFree(mem);
    return fail(SPLAT_ERR_HIP, "hipMemset of ACSR metadata: %s", hipGetErrorString(e));
  }
  char* p = (char*)mem;
  struct Part {
    const void* src;
    size_t n, sz;
  } parts[] = {{a.row_ptr.data(), sizeof(int32_t) * (a.L + 1), s_rowptr},
               {a.runs.data(), sizeof(splat::RowRuns) * a.L, s_runs},
               {a.rows.data(), sizeof(int32_t) * a.L, s_rows},
               {a.groups.data(), sizeof(splat::Group) * a.groups.size(), s_groups},
               {a.tiles.data(), sizeof(splat::Tile) * a.tiles.size(), s_tiles},
               {a.masks.data(), sizeof(uint64_t) * a.masks.size(), s_masks},
               {a.cols.data(), sizeof(splat::ColRun) * a.cols.size(), s_cols}};
  char* dst[7];
  for (int k = 0; k < 7; ++k) {
    dst[k] = p;
    if (parts[k].n) {
      e = hipMemcpy(p, parts[k].src, parts[k].n, hipMemcpyHostToDevice);
      if (e != hipSuccess) {
        (void)hipFree(mem);
        return fail(SPLAT_ERR_HIP, "hipMemcpy of ACSR metadata: %s", hipGetErrorString(e));
      }
    }
    p += parts[k].sz;
  }
  h->dmem = mem;
  h->device = dev;
  h->dev.L = a.L;
  h->dev.nnz = a.nnz;
  h->dev.max_row_nnz = a.max_row_nnz;
  h->dev.n_groups = (int32_t)a.groups.size();
  h->dev.row_ptr = (const int32_t*)dst[0];
  h->dev.runs = (const splat::RowRuns*)dst[1];
  h->dev.rows = (const int32_t*)dst[2];
  h->dev.groups = (const splat::Group*)dst[3];
  h->dev.tiles = (const splat::Tile*)dst[4];
  h->dev.masks = (const uint64_t*)dst[5];
  h->dev.cols = a.cols.empty() ? nullptr : (const splat::ColRun*)dst[6];
  return SPLAT_OK;
}

splat_status finish_build(splat_acsr* h, splat_status s, const std::string& err, splat_acsr_t* out) {
  if (s != SPLAT_OK) {
    delete h;
    return fail(s, "%s", err.c_str());
  }
  s = upload(h);
  if (s != SPLAT_OK) {
    delete h;
    return s;
  }
  *out = h;
  return ok();
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Validation shared by the compute calls.  Returns SPLAT_OK or the failure.
splat_status check_handle(splat_acsr_t h, int32_t B, int32_t H) {
  if (!h) return fail(SPLAT_ERR_INVALID_ARG, "ACSR handle is NULL");
  if (B < 1 || H < 1 || (int64_t)B * H > 65535)
    return fail(SPLAT_ERR_INVALID_ARG, "B and H must be >= 1 with B*H <= 65535 (got B=%d, H=%d)", B, H);
  if (h->device < 0)
    return fail(SPLAT_ERR_NO_DEVICE, "the ACSR handle was built without a GPU");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPLAT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev != h->device)
    return fail(SPLAT_ERR_INVALID_ARG, "current device %d differs from the handle's device %d", dev,
                h->device);
  return SPLAT_OK;
}

// The bf16 kernels run one 256-thread workgroup per (row group, batch*head)
// in a one-dimensional grid, whose work-item count must stay below 2^32.
splat_status check_tile_grid(splat_acsr_t h, int32_t B, int32_t H) {
  const int64_t wgs = (int64_t)h->dev.n_groups * B * H;
  if (wgs * 256 > (int64_t)UINT32_MAX)
    return fail(SPLAT_ERR_UNSUPPORTED,
                "the plan's %d row groups x B*H = %lld workgroups exceed one launch (2^24)",
                h->dev.n_groups, (long long)wgs);
  return SPLAT_OK;
}

// The column-major layout needs the column-wise analysis and single-run columns.
splat_status check_columns(splat_acsr_t h) {
  if (h->host.col_regular < 0)
    return fail(SPLAT_ERR_INVALID_ARG, "the handle was built without SPLAT_PLAN_COLUMNS");
  if (h->host.col_regular == 0)
    return fail(SPLAT_ERR_NOT_REGULAR, "some column of the mask is not one affine run of rows");
  return SPLAT_OK;
}

splat_status check_d(int32_t d) {
  if (d != 64 && d != 128) return fail(SPLAT_ERR_UNSUPPORTED, "d must be 64 or 128, got %d", d);
  return SPLAT_OK;
}

splat_status check_dtype(splat_dtype t, const char* what) {
  if (t != SPLAT_F32 && t != SPLAT_BF16)
    return fail(SPLAT_ERR_INVALID_ARG, "%s must be SPLAT_F32 or SPLAT_BF16", what);
  return SPLAT_OK;
}

splat_status check_ptr(const void* p, const char* what) {
  if (!p) return fail(SPLAT_ERR_INVALID_ARG, "%s is NULL", what);
  if (!aligned16(p)) return fail(SPLAT_ERR_INVALID_ARG, "%s is not 16-byte aligned", what);
  return SPLAT_OK;
}

splat_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(SPLAT_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
  return ok();
}

#define CHECK(x)                     \
  do {                               \
    splat_status _s = (x);           \
    if (_s != SPLAT_OK) return _s;   \
  } while (0)

// Validation of an R-SpMM call (row-major or column-major values).
splat_status check_rspmm(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                         const float* P, const void* V, const void* O, splat_dtype out_dtype,
                         bool colmajor) {
  CHECK(check_handle(h, B, H));
  CHECK(check_dtype(dtype, "dtype"));
  CHECK(check_dtype(out_dtype, "out_dtype"));
  CHECK(check_d(d));
  if (colmajor) CHECK(check_columns(h));
  if (h->host.nnz > 0) CHECK(check_ptr(P, "P"));
  CHECK(check_ptr(V, "V"));
  CHECK(check_ptr(O, "O"));
  if (dtype == SPLAT_BF16) CHECK(check_tile_grid(h, B, H));
  return SPLAT_OK;
}

splat_status launch_rspmm(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                          const float* P, const void* V, void* O, splat_dtype out_dtype,
                          bool colmajor, hipStream_t st) {
  if (dtype == SPLAT_BF16)
    return launched(splat::launch_rspmm_tiles(h->dev, B * H, d, P, V, O, out_dtype, colmajor, st),
                    "rspmm");
  return launched(
      splat::launch_rspmm_rows(h->dev, dtype, B * H, d, P, V, O, out_dtype, colmajor, st), "rspmm");
}

splat_status launch_rsddmm(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                           const void* Q, const void* K, float scale, float* S, hipStream_t st) {
  if (dtype == SPLAT_BF16)
    return launched(splat::launch_rsddmm_tiles(h->dev, B * H, d, Q, K, scale, S, st), "rsddmm");
  return launched(splat::launch_rsddmm_rows(h->dev, dtype, B * H, d, Q, K, scale, S, st), "rsddmm");
}

bool overlap(const float* a, const float* b, size_t n) {
  const char *x = (const char*)a, *y = (const char*)b;
  const size_t bytes = n * sizeof(float);
  return x < y + bytes && y < x + bytes;
}

splat_status check_transpose(splat_acsr_t h, int32_t B, int32_t H, const float* P, const float* Pt) {
  CHECK(check_handle(h, B, H));
  CHECK(check_columns(h));
  if (h->host.nnz == 0) return SPLAT_OK;
  CHECK(check_ptr(P, "P"));
  CHECK(check_ptr(Pt, "Pt"));
  if (overlap(P, Pt, (size_t)B * H * h->host.nnz))
    return fail(SPLAT_ERR_INVALID_ARG, "P and Pt must not overlap");
  CHECK(check_tile_grid(h, B, H));
  return SPLAT_OK;
}

// The paper's density analysis (section 9): masks at or above the density
// alpha whose columns are single affine runs take the column-major layout.
bool use_colmajor(const HostAcsr& a, float alpha) {
  const double density = (double)a.nnz / ((double)a.L * (double)a.L);
  return a.col_regular == 1 && a.nnz > 0 && density >= (double)alpha;
}

// Scratch of splat_sparse_mhsa_unfused_noalloc: the S values and, on the
// column-major branch, their transposed copy.  Every GPU the library runs on
// holds its own copy for the life of the process.  In host code `scratch`
// names a host-side stand-in, never the device array: its device address is
// looked up once per device (scratch_on) and only that address is used.
constexpr size_t kScratchBytes = size_t(SPLAT_NOALLOC_SCRATCH_BYTES);
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
char* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// The scratch array's address on device `dev`, which is the current device.
splat_status scratch_on(int dev, char** out) {
  if (dev < 0 || dev >= kMaxDevices)
    return fail(SPLAT_ERR_UNSUPPORTED, "the allocation-free call supports device ordinals below %d",
                kMaxDevices);
  std::call_once(g_scratch_once[dev], [dev] {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? (char*)p : nullptr;
  });
  if (g_scratch_err[dev] != hipSuccess || !g_scratch_ptr[dev])
    return fail(SPLAT_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                hipGetErrorString(g_scratch_err[dev]));
  *out = g_scratch_ptr[dev];
  return ok();
}

}  // namespace

extern "C" {

const char* splat_last_error(void) { return g_err.c_str(); }

const char* splat_version(void) { return "splat-mi355x 0.1 (gfx950)"; }

splat_status splat_pattern_window(int32_t L, int32_t w, splat_pattern_desc* out) {
  return splat::pattern_window(L, w, out) == SPLAT_OK ? ok() : fail(SPLAT_ERR_INVALID_ARG, "bad window pattern arguments");
}
splat_status splat_pattern_blocked(int32_t L, int32_t block, splat_pattern_desc* out) {
  return splat::pattern_blocked(L, block, out) == SPLAT_OK ? ok() : fail(SPLAT_ERR_INVALID_ARG, "bad blocked pattern arguments");
}
splat_status splat_pattern_strided_local(int32_t L, int32_t local, int32_t stride, splat_pattern_desc* out) {
  return splat::pattern_strided_local(L, local, stride, out) == SPLAT_OK ? ok() : fail(SPLAT_ERR_INVALID_ARG, "bad strided_local pattern arguments");
}
splat_status splat_pattern_dilated(int32_t L, int32_t w, int32_t dilation, splat_pattern_desc* out) {
  return splat::pattern_dilated(L, w, dilation, out) == SPLAT_OK ? ok() : fail(SPLAT_ERR_INVALID_ARG, "bad dilated pattern arguments");
}
splat_status splat_pattern_window_global(int32_t L, int32_t w, int32_t n_global, splat_pattern_desc* out) {
  return splat::pattern_window_global(L, w, n_global, out) == SPLAT_OK ? ok() : fail(SPLAT_ERR_INVALID_ARG, "bad window_global pattern arguments");
}
splat_status splat_pattern_full(int32_t L, splat_pattern_desc* out) {
  return splat::pattern_full(L, out) == SPLAT_OK ? ok() : fail(SPLAT_ERR_INVALID_ARG, "bad full pattern arguments");
}

splat_status splat_acsr_build_ex(const splat_pattern_desc* desc, uint32_t flags, splat_acsr_t* out) {
  if (!desc || !out) return fail(SPLAT_ERR_INVALID_ARG, "desc and out must be non-NULL");
  if (flags & ~(SPLAT_PLAN_NO_SPAN | SPLAT_PLAN_COLUMNS))
    return fail(SPLAT_ERR_INVALID_ARG, "unknown plan flags 0x%x", flags);
  if ((flags & SPLAT_PLAN_NO_SPAN) && desc->L > SPLAT_NO_SPAN_MAX_L)
    return fail(SPLAT_ERR_UNSUPPORTED, "SPLAT_PLAN_NO_SPAN needs L <= %d, got %d", SPLAT_NO_SPAN_MAX_L,
                desc->L);
  splat_acsr* h = new (std::nothrow) splat_acsr();
  if (!h) return fail(SPLAT_ERR_OOM, "host allocation failed");
  std::string err;
  splat_status s;
  try {
    s = splat::build_from_desc(*desc, h->host, err, flags);
  } catch (const std::bad_alloc&) {
    s = SPLAT_ERR_OOM;
    err = "host allocation failed during the analysis";
  }
  return finish_build(h, s, err, out);
}

splat_status splat_acsr_build(const splat_pattern_desc* desc, splat_acsr_t* out) {
  return splat_acsr_build_ex(desc, 0u, out);
}

splat_status splat_acsr_from_mask(int32_t L, const uint8_t* mask, splat_acsr_t* out) {
  if (!out) return fail(SPLAT_ERR_INVALID_ARG, "out must be non-NULL");
  splat_acsr* h = new (std::nothrow) splat_acsr();
  if (!h) return fail(SPLAT_ERR_OOM, "host allocation failed");
  std::string err;
  splat_status s;
  try {
    s = splat::build_from_mask(L, mask, h->host, err);
  } catch (const std::bad_alloc&) {
    s = SPLAT_ERR_OOM;
    err = "host allocation failed during the analysis";
  }
  return finish_build(h, s, err, out);
}

void splat_acsr_destroy(splat_acsr_t h) {
  if (!h) return;
  if (h->dmem) (void)hipFree(h->dmem);
  delete h;
}

splat_status splat_acsr_info(splat_acsr_t h, splat_acsr_info_t* out) {
  if (!h || !out) return fail(SPLAT_ERR_INVALID_ARG, "handle and out must be non-NULL");
  const HostAcsr& a = h->host;
  std::memset(out, 0, sizeof(*out));
  out->L = a.L;
  out->max_row_nnz = a.max_row_nnz;
  out->max_runs = a.max_runs;
  out->on_device = h->device >= 0;
  out->device = h->device;
  out->bm = splat::kBM;
  out->bn = splat::kBN;
  out->n_groups = (int32_t)a.groups.size();
  out->n_tiles = (int32_t)a.tiles.size();
  out->n_full_tiles = a.n_full;
  out->nnz = a.nnz;
  out->computed = a.computed;
  out->columns = a.col_regular;
  return ok();
}

splat_status splat_acsr_tiling(splat_acsr_t h, int32_t method, int32_t m, int32_t n, int32_t stretch,
                               splat_tiling_stats_t* out, int32_t* anchors, int64_t anchor_capacity) {
  if (!h || !out) return fail(SPLAT_ERR_INVALID_ARG, "handle and out must be non-NULL");
  if (anchor_capacity < 0) return fail(SPLAT_ERR_INVALID_ARG, "anchor_capacity must be >= 0");
  splat::TilingStats st;
  std::vector<int32_t> anc;
  std::string err;
  splat_status s;
  try {
    s = splat::tile_mask(h->host, method, m, n, stretch, anchors ? &anc : nullptr, st, err);
  } catch (const std::bad_alloc&) {
    s = SPLAT_ERR_OOM;
    err = "host allocation failed during tiling";
  }
  if (s != SPLAT_OK) return fail(s, "%s", err.c_str());
  out->blocks = st.blocks;
  out->points = st.points;
  out->divergent = st.divergent;
  out->redundant = st.redundant;
  out->reuse = st.reuse;
  out->coalesced = st.coalesced;
  out->cost = st.cost;
  out->stretch = st.stretch;
  out->iterations = st.iterations;
  if (anchors) {
    const int64_t k = std::min<int64_t>(anchor_capacity, st.blocks);
    std::memcpy(anchors, anc.data(), sizeof(int32_t) * 2 * (size_t)k);
  }
  return ok();
}

splat_status splat_acsr_export_csc(splat_acsr_t h, int32_t* col_ptr, int32_t* row_idx) {
  if (!h || !col_ptr || (!row_idx && h->host.nnz > 0))
    return fail(SPLAT_ERR_INVALID_ARG, "handle, col_ptr and row_idx must be non-NULL");
  CHECK(check_columns(h));
  const HostAcsr& a = h->host;
  for (int32_t j = 0; j < a.L; ++j) {
    const splat::ColRun& c = a.cols[j];
    col_ptr[j] = c.ptr;
    for (int32_t t = 0; t < c.count; ++t) row_idx[c.ptr + t] = c.start + c.stride * t;
  }
  col_ptr[a.L] = (int32_t)a.nnz;
  return ok();
}

splat_status splat_acsr_export(splat_acsr_t h, int32_t* row_ptr, int32_t* col_idx) {
  if (!h || !row_ptr || (!col_idx && h->host.nnz > 0))
    return fail(SPLAT_ERR_INVALID_ARG, "handle, row_ptr and col_idx must be non-NULL");
  const HostAcsr& a = h->host;
  std::memcpy(row_ptr, a.row_ptr.data(), sizeof(int32_t) * (a.L + 1));
  for (int32_t i = 0; i < a.L; ++i) {
    int32_t* o = col_idx + a.row_ptr[i];
    for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
      const splat::Run& q = a.runs[i].r[r];
      for (int32_t k = 0; k < q.count; ++k) o[q.prefix + k] = q.start + q.stride * k;
    }
  }
  return ok();
}

splat_status splat_acsr_row_runs(splat_acsr_t h, int32_t row, int32_t* runs, int32_t* nruns) {
  if (!h || !runs || !nruns) return fail(SPLAT_ERR_INVALID_ARG, "NULL argument");
  if (row < 0 || row >= h->host.L) return fail(SPLAT_ERR_INVALID_ARG, "row %d out of range", row);
  *nruns = h->host.nruns[row];
  for (int r = 0; r < SPLAT_MAX_RUNS; ++r) {
    const splat::Run& q = h->host.runs[row].r[r];
    runs[3 * r] = q.start;
    runs[3 * r + 1] = q.stride;
    runs[3 * r + 2] = q.count;
  }
  return ok();
}

splat_status splat_acsr_export_plan(splat_acsr_t h, int32_t* groups, int32_t* rows, int32_t* tiles) {
  if (!h || !groups || !rows || !tiles) return fail(SPLAT_ERR_INVALID_ARG, "NULL argument");
  const HostAcsr& a = h->host;
  for (size_t g = 0; g < a.groups.size(); ++g) {
    groups[4 * g] = a.groups[g].row_off;
    groups[4 * g + 1] = a.groups[g].nrows;
    groups[4 * g + 2] = a.groups[g].tile_begin;
    groups[4 * g + 3] = a.groups[g].tile_end;
  }
  std::memcpy(rows, a.rows.data(), sizeof(int32_t) * a.L);
  for (size_t t = 0; t < a.tiles.size(); ++t) {
    tiles[5 * t] = a.tiles[t].kb;
    tiles[5 * t + 1] = a.tiles[t].ks;
    tiles[5 * t + 2] = a.tiles[t].nk;
    tiles[5 * t + 3] = a.tiles[t].flags;
    tiles[5 * t + 4] = a.tiles[t].mask_block;
  }
  return ok();
}

splat_status splat_acsr_tile_row_mask(splat_acsr_t h, int32_t tile, int32_t row, uint64_t* bits) {
  if (!h || !bits) return fail(SPLAT_ERR_INVALID_ARG, "NULL argument");
  if (tile < 0 || tile >= (int32_t)h->host.tiles.size())
    return fail(SPLAT_ERR_INVALID_ARG, "tile %d out of range", tile);
  if (row < 0 || row >= h->host.L) return fail(SPLAT_ERR_INVALID_ARG, "row %d out of range", row);
  const splat::Tile& t = h->host.tiles[tile];
  *bits = splat::tile_row_bits(h->host.runs[row], t.kb, t.ks, t.nk);
  return ok();
}

splat_status splat_rsddmm(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                          const void* Q, const void* K, float scale, float* S, void* stream) {
  CHECK(check_handle(h, B, H));
  CHECK(check_dtype(dtype, "dtype"));
  CHECK(check_d(d));
  CHECK(check_ptr(Q, "Q"));
  CHECK(check_ptr(K, "K"));
  if (h->host.nnz == 0) return ok();
  CHECK(check_ptr(S, "S"));
  if (dtype == SPLAT_BF16) CHECK(check_tile_grid(h, B, H));
  return launch_rsddmm(h, dtype, B, H, d, Q, K, scale, S, (hipStream_t)stream);
}

splat_status splat_row_softmax(splat_acsr_t h, int32_t B, int32_t H, const float* S, float* P,
                               void* stream) {
  CHECK(check_handle(h, B, H));
  if (h->host.nnz == 0) return ok();
  CHECK(check_ptr(S, "S"));
  CHECK(check_ptr(P, "P"));
  const size_t bytes = sizeof(float) * (size_t)B * H * h->host.nnz;
  const char *s0 = (const char*)S, *p0 = (const char*)P;
  if (s0 != p0 && s0 < p0 + bytes && p0 < s0 + bytes)
    return fail(SPLAT_ERR_INVALID_ARG, "S and P overlap without being equal");
  hipStream_t st = (hipStream_t)stream;
  return launched(splat::launch_softmax(h->dev, B * H, S, P, st), "row_softmax");
}

splat_status splat_rspmm(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                         const float* P, const void* V, void* O, splat_dtype out_dtype, void* stream) {
  CHECK(check_rspmm(h, dtype, B, H, d, P, V, O, out_dtype, false));
  return launch_rspmm(h, dtype, B, H, d, P, V, O, out_dtype, false, (hipStream_t)stream);
}

splat_status splat_rspmm_colmajor(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                                  const float* Pt, const void* V, void* O, splat_dtype out_dtype,
                                  void* stream) {
  CHECK(check_rspmm(h, dtype, B, H, d, Pt, V, O, out_dtype, true));
  return launch_rspmm(h, dtype, B, H, d, Pt, V, O, out_dtype, true, (hipStream_t)stream);
}

splat_status splat_transpose_colmajor(splat_acsr_t h, int32_t B, int32_t H, const float* P, float* Pt,
                                      void* stream) {
  CHECK(check_transpose(h, B, H, P, Pt));
  if (h->host.nnz == 0) return ok();
  return launched(splat::launch_transpose_colmajor(h->dev, B * H, P, Pt, (hipStream_t)stream),
                  "transpose_colmajor");
}

splat_status splat_sparse_mhsa_fwd(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                                   const void* Q, const void* K, const void* V, float scale,
                                   void* O, splat_dtype out_dtype, void* stream) {
  CHECK(check_handle(h, B, H));
  CHECK(check_dtype(dtype, "dtype"));
  CHECK(check_dtype(out_dtype, "out_dtype"));
  CHECK(check_d(d));
  CHECK(check_ptr(Q, "Q"));
  CHECK(check_ptr(K, "K"));
  CHECK(check_ptr(V, "V"));
  CHECK(check_ptr(O, "O"));
  hipStream_t st = (hipStream_t)stream;
  if (dtype == SPLAT_BF16) CHECK(check_tile_grid(h, B, H));
  if (dtype == SPLAT_BF16)
    return launched(splat::launch_fused_mfma(h->dev, B * H, d, Q, K, V, scale, O, out_dtype, st),
                    "sparse_mhsa_fwd");
  return launched(splat::launch_fused_rows(h->dev, dtype, B * H, d, Q, K, V, scale, O, out_dtype, st),
                  "sparse_mhsa_fwd");
}

splat_status splat_sparse_mhsa_unfused(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H,
                                       int32_t d, const void* Q, const void* K, const void* V,
                                       float scale, float* S, float* Pt, void* O,
                                       splat_dtype out_dtype, float alpha, int32_t* used_colmajor,
                                       void* stream) {
  CHECK(check_handle(h, B, H));
  const HostAcsr& a = h->host;
  // the paper's density analysis: dense masks take the column-major layout
  const bool col = use_colmajor(a, alpha);
  // every step is validated before anything is enqueued
  CHECK(check_dtype(dtype, "dtype"));
  CHECK(check_d(d));
  CHECK(check_ptr(Q, "Q"));
  CHECK(check_ptr(K, "K"));
  CHECK(check_rspmm(h, dtype, B, H, d, S, V, O, out_dtype, false));
  if (col) CHECK(check_transpose(h, B, H, S, Pt));
  hipStream_t st = (hipStream_t)stream;
  if (a.nnz > 0) {
    CHECK(launch_rsddmm(h, dtype, B, H, d, Q, K, scale, S, st));
    CHECK(launched(splat::launch_softmax(h->dev, B * H, S, S, st), "row_softmax"));
    if (col)
      CHECK(launched(splat::launch_transpose_colmajor(h->dev, B * H, S, Pt, st),
                     "transpose_colmajor"));
  }
  if (used_colmajor) *used_colmajor = col ? 1 : 0;
  return launch_rspmm(h, dtype, B, H, d, col ? Pt : S, V, O, out_dtype, col, st);
}

splat_status splat_sparse_mhsa_unfused_noalloc(splat_acsr_t h, splat_dtype dtype, int32_t B,
                                               int32_t H, int32_t d, const void* Q, const void* K,
                                               const void* V, float scale, void* O,
                                               splat_dtype out_dtype, float alpha,
                                               int32_t* used_colmajor, void* stream) {
  CHECK(check_handle(h, B, H));
  const HostAcsr& a = h->host;
  const bool col = use_colmajor(a, alpha);
  const size_t vals = (size_t)B * H * (size_t)a.nnz * sizeof(float);
  const size_t s_bytes = (vals + 255) & ~size_t(255);
  const size_t need = s_bytes + (col ? vals : 0);
  if (need > kScratchBytes)
    return fail(SPLAT_ERR_UNSUPPORTED,
                "the allocation-free call needs %zu bytes of scratch (B*H*nnz*4%s), more than its "
                "maximum of %zu bytes",
                need, col ? ", twice for the column-major layout" : "", kScratchBytes);
  char* base = nullptr;
  CHECK(scratch_on(h->device, &base));
  return splat_sparse_mhsa_unfused(h, dtype, B, H, d, Q, K, V, scale, (float*)base,
                                   col ? (float*)(base + s_bytes) : nullptr, O, out_dtype, alpha,
                                   used_colmajor, stream);
}

splat_status splat_debug_bounds(uint32_t* flags, int32_t clear) {
  CHECK(check_ptr(flags, "flags"));
#ifndef SPLAT_DEBUG_BOUNDS
  return fail(SPLAT_ERR_UNSUPPORTED,
              "this library was built without SPLAT_DEBUG_BOUNDS (libsplat_checked.so has it)");
#else
  uint32_t bits = 0;
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = splat::bounds_collect_rows(&bits, clear != 0);
  if (e == hipSuccess) e = splat::bounds_collect_mfma(&bits, clear != 0);
  if (e == hipSuccess) e = splat::bounds_collect_tiles(&bits, clear != 0);
  if (e != hipSuccess) return fail(SPLAT_ERR_HIP, "splat_debug_bounds: %s", hipGetErrorString(e));
  *flags = bits;
  return SPLAT_OK;
#endif
}

splat_status splat_debug_bounds_probe(int32_t kind, int32_t index, int32_t n, int32_t* result) {
  CHECK(check_ptr(result, "result"));
  if (kind < 0 || kind > 3) return fail(SPLAT_ERR_INVALID_ARG, "kind %d is not 0..3", kind);
#ifndef SPLAT_DEBUG_BOUNDS
  (void)index;
  (void)n;
  return fail(SPLAT_ERR_UNSUPPORTED,
              "this library was built without SPLAT_DEBUG_BOUNDS (libsplat_checked.so has it)");
#else
  int r = 0;
  const hipError_t e = splat::bounds_probe(kind, index, n, &r);
  if (e != hipSuccess) return fail(SPLAT_ERR_HIP, "splat_debug_bounds_probe: %s", hipGetErrorString(e));
  *result = r;
  return SPLAT_OK;
#endif
}

}  // extern "C"
