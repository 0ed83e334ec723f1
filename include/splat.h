/*
 * splat.h -- C ABI of the MI355X (gfx950) sparse multi-head self-attention
 * library over affine-compressed-sparse-row (ACSR) masks.
 *
 * The method is SPLAT (arXiv 2407.16847).  Sparse attention (section 2,
 * Equation 1) is the chain
 *
 *     S = scale * (M (x) Q K^T)      regular SDDMM, sampled at the mask's non-zeros
 *     P = row softmax of S           over each row's non-zeros (section 6)
 *     O = P V                        regular SpMM
 *
 * where the 0/1 mask M is "regular": every row's column set is described by
 * a few affine indices instead of a column list (sections 4.1 and 5.1).
 *
 * Conventions shared by every call
 * --------------------------------
 * Shapes.  Q, K, V, O are dense, contiguous, row-major [B, H, L, d] arrays
 *   (batch, head, token, feature).  d is 64 or 128.  One mask is shared by
 *   every batch and head (the paper's masks are fixed ahead of time).
 * ACSR values.  S and P are fp32 [B, H, nnz] arrays: the values of head
 *   (b, h) start at element (b*H + h) * nnz and, inside it, row i occupies
 *   [row_ptr[i], row_ptr[i+1]) with its columns in ascending order -- the
 *   paper's row-compressed, row-major ACSR layout (section 5.1, Figure 5b).
 * Memory.  Every tensor argument is DEVICE memory owned by the caller, on the
 *   device the ACSR handle was built on, 16-byte aligned.  No compute call
 *   allocates memory.  The handle owns only the mask metadata (host copy plus
 *   one small device allocation).
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = the default
 *   stream).  Compute calls validate their arguments on the host, enqueue
 *   the kernels and return; kernel faults surface at the caller's next
 *   synchronisation.
 * Errors.  Every call returns a splat_status; on anything but SPLAT_OK the
 *   thread-local message behind splat_last_error() says what was wrong.  A
 *   failed call has enqueued nothing and written no output.
 * Threads.  Handles are immutable after splat_acsr_build and may be used by
 *   several host threads at once.
 */
#ifndef SPLAT_H
#define SPLAT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPLAT_OK = 0,
  SPLAT_ERR_INVALID_ARG = 1,  /* null / misaligned pointer, bad size, bad descriptor */
  SPLAT_ERR_UNSUPPORTED = 2,  /* valid request outside what is implemented: d, runs per row, or a
                                 bf16 call whose plan needs more than 2^24 (row group, batch*head)
                                 workgroups (n_groups * B * H, see splat_acsr_info) */
  SPLAT_ERR_NOT_REGULAR = 3,  /* mask input whose rows are not affine-compressible */
  SPLAT_ERR_OOM = 4,          /* host or device allocation failed (build only) */
  SPLAT_ERR_HIP = 5,          /* a HIP runtime call failed; message holds hipGetErrorString */
  SPLAT_ERR_NO_DEVICE = 6     /* compute call on a handle built without a GPU */
} splat_status;

typedef enum { SPLAT_F32 = 0, SPLAT_BF16 = 1 } splat_dtype;

typedef struct splat_acsr* splat_acsr_t; /* opaque, owned by the caller, freed by splat_acsr_destroy */

#define SPLAT_MAX_TERMS 8
#define SPLAT_MAX_RUNS 4

/*
 * Pattern descriptor.  A mask is the union of up to SPLAT_MAX_TERMS affine
 * terms.  Term t applies to rows i in [row_lo, row_hi); with
 * q = floor(i / group) its columns are
 *
 *     j = j_lo(i) + stride * k,   k = 0, 1, ...,   j <= j_hi(i)
 *     j_lo(i) = lo_i * i + lo_q * q * group + lo_c
 *     j_hi(i) = hi_i * i + hi_q * q * group + hi_c      (inclusive)
 *
 * clamped to [0, L) without changing the residue j_lo mod stride.  A column
 * produced by several terms counts once.  Every term keeps, per row, the
 * affine form of section 4.1 (equal gaps of `stride`); the union of a row's
 * terms is stored as at most SPLAT_MAX_RUNS such runs.
 */
typedef struct {
  int32_t row_lo, row_hi; /* rows the term applies to, 0 <= row_lo <= row_hi <= L */
  int32_t group;          /* >= 1 */
  int32_t lo_i, lo_q, lo_c;
  int32_t hi_i, hi_q, hi_c;
  int32_t stride;         /* >= 1 */
} splat_affine_term;

typedef struct {
  int32_t L;        /* sequence length, 1 <= L <= SPLAT_MAX_L */
  int32_t n_terms;  /* 0 <= n_terms <= SPLAT_MAX_TERMS (0 = empty mask) */
  splat_affine_term terms[SPLAT_MAX_TERMS];
} splat_pattern_desc;

#define SPLAT_MAX_L 65536

/*
 * Descriptor helpers for the sparse-MHSA patterns the paper evaluates
 * (section 2 "Sparse-MHSA Patterns", section 10.2) and their variants.  Each
 * fills *out and returns SPLAT_ERR_INVALID_ARG on out == NULL or a bad size.
 *   window        |i - j| <= w
 *   blocked       j in the block of i (blocks of `block` tokens) or the block before it
 *   strided_local causal: j in [i - local + 1, i], or j = stride - 1 (mod stride) with j <= i
 *   dilated       j = i + dilation * k, |k| <= w
 *   window_global |i - j| <= w, or i < n_global, or j < n_global
 *   full          every (i, j)
 */
splat_status splat_pattern_window(int32_t L, int32_t w, splat_pattern_desc* out);
splat_status splat_pattern_blocked(int32_t L, int32_t block, splat_pattern_desc* out);
splat_status splat_pattern_strided_local(int32_t L, int32_t local, int32_t stride, splat_pattern_desc* out);
splat_status splat_pattern_dilated(int32_t L, int32_t w, int32_t dilation, splat_pattern_desc* out);
splat_status splat_pattern_window_global(int32_t L, int32_t w, int32_t n_global, splat_pattern_desc* out);
splat_status splat_pattern_full(int32_t L, splat_pattern_desc* out);

/*
 * splat_acsr_build -- the just-in-time analysis (section 4, section 9
 * "Analysis pass"; section 5.1 construction).
 *
 * For every row it forms the sorted union of the descriptor's columns and
 * stores it as at most SPLAT_MAX_RUNS disjoint ascending affine runs
 * (start, stride, count): the paper's per-row affine indices with
 * a = 1/stride, b = -start/stride, nnzs = count, generalised from one run to
 * a few (so window+global and strided+local masks, which are not regular in
 * the paper's sense, are still held in O(rows) metadata).  It then plans the
 * kernels' work: rows with identical affine geometry are grouped
 * (section 5.2, rows with identical affine indices mapped together), and each
 * row group's column span (section 8.2, span specialisation) is cut into key
 * tiles, each marked FULL (every element in the mask) or PARTIAL.  When a GPU
 * is present the metadata is copied to the current HIP device, which every
 * later compute call on this handle must use.  Without a GPU the handle is
 * host-only: the query calls below work, compute calls return
 * SPLAT_ERR_NO_DEVICE.
 *
 * Returns INVALID_ARG for a malformed descriptor, UNSUPPORTED when a row
 * needs more than SPLAT_MAX_RUNS runs or nnz >= 2^31, OOM / HIP on failed
 * allocations.  *out is written only on SPLAT_OK.
 */
splat_status splat_acsr_build(const splat_pattern_desc* desc, splat_acsr_t* out);

/*
 * splat_acsr_build_ex -- splat_acsr_build with planning options.  `flags` is
 * 0 (the same handle as splat_acsr_build) or a combination of:
 *
 * SPLAT_PLAN_NO_SPAN -- for the ablation study of section 10 (the R-SpMM
 *   kernel with and without span specialisation, section 8.2): every row
 *   group walks the whole key range [0, L) in contiguous 64-key tiles and
 *   every wavefront that holds rows evaluates the membership predicate on
 *   every tile, including tiles where none of its rows has a key.  The index
 *   set, every compute call's result and its tolerance are unchanged; only
 *   the work differs (splat_acsr_info's `computed` becomes rows x L, rounded
 *   up to tiles).  UNSUPPORTED with L > SPLAT_NO_SPAN_MAX_L (its per-row
 *   masks take L*L/8 bytes of device memory).
 * SPLAT_PLAN_COLUMNS -- the column-wise analysis of section 5.2 (a regular
 *   mask is also column-wise affine-compressible): when every column's rows
 *   form one affine run, the handle also describes the column-compressed,
 *   column-major value layout (splat_acsr_export_csc,
 *   splat_transpose_colmajor, splat_rspmm_colmajor); splat_acsr_info's
 *   `columns` reports the outcome.  A mask whose columns are not single runs
 *   still builds (columns = 0).  O(nnz) host time; UNSUPPORTED above 2^28
 *   non-zeros per head.
 *
 * Returns INVALID_ARG for unknown flag bits; otherwise as splat_acsr_build.
 */
#define SPLAT_PLAN_NO_SPAN 1u
#define SPLAT_PLAN_COLUMNS 2u
#define SPLAT_NO_SPAN_MAX_L 16384
splat_status splat_acsr_build_ex(const splat_pattern_desc* desc, uint32_t flags, splat_acsr_t* out);

/*
 * splat_acsr_from_mask -- build from an explicit row-major 0/1 byte mask
 * (L*L bytes, host memory) with the paper's analysis pass: per row, the affine
 * indices come from the first two columns (section 5.1, the 2x2 solve) and
 * every further column is verified against them; a row that fails makes the
 * whole mask non-regular and the call returns SPLAT_ERR_NOT_REGULAR (the paper
 * terminates on such masks, section 9).  On success the handle is the same as
 * one built from an equivalent descriptor.
 */
splat_status splat_acsr_from_mask(int32_t L, const uint8_t* mask, splat_acsr_t* out);

void splat_acsr_destroy(splat_acsr_t h); /* NULL is a no-op */

typedef struct {
  int32_t L;
  int32_t max_row_nnz;
  int32_t max_runs;        /* largest number of runs any row needed */
  int32_t on_device;       /* 1 if the metadata lives on a HIP device */
  int32_t device;          /* that device's ordinal, -1 if none */
  int32_t bm, bn;          /* rows per group, keys per tile of the plan */
  int32_t n_groups;
  int32_t n_tiles;
  int32_t n_full_tiles;
  int64_t nnz;             /* non-zeros per (batch, head) */
  int64_t computed;        /* rows x keys of the 32-row x 64-key tiles the kernels compute (>= nnz) */
  int32_t columns;         /* column-wise analysis: -1 not requested, 0 some column is not one
                              affine run, 1 every column is (column-major layout available) */
  int32_t reserved;
} splat_acsr_info_t;

splat_status splat_acsr_info(splat_acsr_t h, splat_acsr_info_t* out);

/* Host copies of the index set: row_ptr[L+1] and col_idx[nnz] (CSR order). */
splat_status splat_acsr_export(splat_acsr_t h, int32_t* row_ptr, int32_t* col_idx);

/*
 * Host copies of the transposed index set: col_ptr[L+1] and row_idx[nnz] in
 * column-compressed order (column by column, ascending row), which is also
 * the value order of the column-major layout.  Needs a handle built with
 * SPLAT_PLAN_COLUMNS whose columns are single runs: INVALID_ARG without the
 * analysis, NOT_REGULAR when some column is not one affine run.
 */
splat_status splat_acsr_export_csc(splat_acsr_t h, int32_t* col_ptr, int32_t* row_idx);

/* Runs of one row: runs[3*r + {0,1,2}] = (start, stride, count), r < *nruns. */
splat_status splat_acsr_row_runs(splat_acsr_t h, int32_t row, int32_t* runs, int32_t* nruns);

/*
 * Host copy of the work plan.  groups[4*g + {0,1,2,3}] = (first index into
 * rows, number of rows, first tile, one past the last tile), in launch order;
 * rows[L] lists every row once (grouped); tiles[5*t + {0,1,2,3,4}] =
 * (first key, key step, number of keys, flags, mask block).  The keys of a
 * tile are first + step * u for u < number of keys.  flags bit 0 = every key
 * is in every row of the group; bits 8+2w..9+2w = the tile's state for the
 * group's rows [32w, 32w+32): 0 none of them has a key here, 1 some do (the
 * per-row masks are precomputed, mask block >= 0), 3 all keys in all rows.
 * Sizes come from splat_acsr_info (n_groups, n_tiles).
 */
splat_status splat_acsr_export_plan(splat_acsr_t h, int32_t* groups, int32_t* rows, int32_t* tiles);

/*
 * Mask bits of one row inside one planned tile: bit u is set iff key
 * first + step * u of tile `tile` is in row `row`'s column set.  This is the
 * O(1)-per-run membership test of section 5.2 ("fast indexing") that the
 * kernels evaluate on PARTIAL tiles; exported for host-side verification.
 */
splat_status splat_acsr_tile_row_mask(splat_acsr_t h, int32_t tile, int32_t row, uint64_t* bits);

/*
 * splat_acsr_tiling -- thread-block arrangements of the mask under the SDDMM
 * cost model of section 7 (a host-side diagnostic for the tiling ablation of
 * section 10; the kernels run the row-group plan above).
 *
 * A thread-block of m x n threads with anchor t and stretch s computes the
 * points t + (i*s, j*s), i < m, j < n (section 7.2).
 * method SPLAT_TILING_POSET -- poset tiling (section 7.3, Algorithm 1): in
 *   rounds, every uncovered point that no other uncovered point comes before
 *   (row and column both <=) becomes an anchor, and the points its block
 *   computes are removed, until the mask is covered.  stretch 0 selects the
 *   stretch (section 7.3.1): 1 unless every non-empty row is one run of a
 *   common stride X > 1, then the divisor of X of lowest cost (ties: fewer
 *   blocks); stretch >= 1 fixes it.
 * method SPLAT_TILING_NAIVE -- Naive Tiling (Appendix C, the comparison
 *   point of the SDDMM tiling ablation in section 10): the mask is cut into
 *   patches of m consecutive rows (starting at row 0) and each patch is tiled
 *   from left to right by unstretched blocks, the first at the patch's
 *   leftmost point and the others n columns apart, ceil(w / n) of them for a
 *   patch of width w (leftmost to rightmost point, inclusive); patches
 *   without points take none (stretch must be 0 or 1).
 * method SPLAT_TILING_GRID -- unstretched blocks at every multiple of
 *   (m, n) whose block meets the mask (stretch must be 0 or 1).
 * *out receives the arrangement's block count lambda, |P| = nnz, and the
 * quantities of section 7.2: divergent threads (computed points outside the
 * mask, blocks reaching past the matrix included), redundant threads
 * (lambda*m*n - |P| - divergent), reuse |P| / (lambda*m*n), coalescing
 * (mean 1/stretch) and cost lambda / coalescing, plus the stretch used and
 * the number of rounds.  anchors (optional) receives the first
 * min(anchor_capacity, lambda) anchors as (row, column) pairs in placement
 * order.  INVALID_ARG for bad sizes (m, n in [1, 1024]; (m-1)*s and
 * (n-1)*s at most L + 1024), UNSUPPORTED above L = SPLAT_TILING_MAX_L.
 * Host only.
 */
#define SPLAT_TILING_POSET 0
#define SPLAT_TILING_GRID 1
#define SPLAT_TILING_NAIVE 2
#define SPLAT_TILING_MAX_L 8192
typedef struct {
  int64_t blocks;
  int64_t points;
  int64_t divergent;
  int64_t redundant;
  double reuse;
  double coalesced;
  double cost;
  int32_t stretch;
  int32_t iterations;
} splat_tiling_stats_t;

splat_status splat_acsr_tiling(splat_acsr_t h, int32_t method, int32_t m, int32_t n, int32_t stretch,
                               splat_tiling_stats_t* out, int32_t* anchors, int64_t anchor_capacity);

/*
 * splat_rsddmm -- regular SDDMM (Equation 1, section 7.4):
 *   S[b,h, row_ptr[i] + k] = scale * sum_c Q[b,h,i,c] * K[b,h,col(i,k),c]
 * for every row i and its k-th column col(i, k) in ascending order.
 * Q, K: [B,H,L,d] of `dtype` (SPLAT_F32 or SPLAT_BF16).  S: fp32 [B,H,nnz].
 * Products are accumulated in fp32.
 */
splat_status splat_rsddmm(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                          const void* Q, const void* K, float scale, float* S, void* stream);

/*
 * splat_row_softmax -- softmax over each row's non-zeros (section 6, section 9
 * "Code-generation"): P_ik = exp(S_ik - max_k S_ik) / sum_k exp(S_ik - max_k S_ik).
 * S, P: fp32 [B,H,nnz]; P may equal S (in place), otherwise they must not overlap.
 * Rows with no non-zero are left untouched (they own no values).
 */
splat_status splat_row_softmax(splat_acsr_t h, int32_t B, int32_t H, const float* S, float* P,
                               void* stream);

/*
 * splat_rspmm -- regular SpMM (Equation 1, section 8):
 *   O[b,h,i,:] = sum_k P[b,h,row_ptr[i]+k] * V[b,h,col(i,k),:]
 * P: fp32 [B,H,nnz].  V: [B,H,L,d] of `dtype`.  O: [B,H,L,d] of `out_dtype`
 * (a row without non-zeros gets O = 0).  Accumulation is fp32; with bf16 V the
 * products are formed on the matrix cores from P split into a bf16 high part
 * and a bf16 low part, so P keeps about 16 significant bits.
 */
splat_status splat_rspmm(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                         const float* P, const void* V, void* O, splat_dtype out_dtype, void* stream);

/*
 * splat_transpose_colmajor -- the data-layout reordering of section 9: the
 * values of every (batch, head) moved from the row-compressed, row-major
 * order (CSR order, as splat_rsddmm and splat_row_softmax write them) to the
 * column-compressed, column-major order of section 5.2 (column by column,
 * ascending row; the order of splat_acsr_export_csc):
 *   Pt[b,h, col_ptr[j] + t] = P[b,h, row_ptr[i] + k]
 * where row i is the t-th row of column j and j the k-th column of row i.
 * P, Pt: fp32 [B,H,nnz], distinct, non-overlapping.  The handle must have
 * been built with SPLAT_PLAN_COLUMNS and have single-run columns
 * (INVALID_ARG / NOT_REGULAR otherwise).  A pure permutation: bit-exact.
 */
splat_status splat_transpose_colmajor(splat_acsr_t h, int32_t B, int32_t H, const float* P, float* Pt,
                                      void* stream);

/*
 * splat_rspmm_colmajor -- splat_rspmm reading P in the column-compressed,
 * column-major layout (section 9: the layout the paper selects for dense
 * masks so that consecutive rows of a column are read from consecutive
 * addresses).  Pt as written by splat_transpose_colmajor; every other
 * argument, the result and its rounding as splat_rspmm (with bf16 V the
 * result equals splat_rspmm's bit for bit).  Handle requirements as
 * splat_transpose_colmajor.
 */
splat_status splat_rspmm_colmajor(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                                  const float* Pt, const void* V, void* O, splat_dtype out_dtype,
                                  void* stream);

/*
 * splat_sparse_mhsa_unfused -- the paper's unfused chain with its density
 * switch (section 9: analysis pass, data-layout reordering): S = R-SDDMM,
 * P = softmax of S in place, then, when the mask's density nnz / L^2 is at
 * least `alpha` and the handle has the column-major layout
 * (SPLAT_PLAN_COLUMNS with single-run columns), Pt = the column-major copy
 * of P and O = splat_rspmm_colmajor(Pt); otherwise O = splat_rspmm(P).  The
 * paper's threshold is alpha = 0.10 (SPLAT_DENSE_ALPHA); alpha > 1 never
 * transposes.  S: fp32 [B,H,nnz] workspace (holds P afterwards); Pt: fp32
 * [B,H,nnz] workspace, used (and required non-NULL) only on the column-major
 * branch.  *used_colmajor (if non-NULL) is set to 1 on the column-major
 * branch, 0 otherwise.  Results as the individual calls.
 */
#define SPLAT_DENSE_ALPHA 0.10f
splat_status splat_sparse_mhsa_unfused(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H,
                                       int32_t d, const void* Q, const void* K, const void* V,
                                       float scale, float* S, float* Pt, void* O,
                                       splat_dtype out_dtype, float alpha, int32_t* used_colmajor,
                                       void* stream);

/*
 * splat_sparse_mhsa_unfused_noalloc -- splat_sparse_mhsa_unfused for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): the same chain, the same
 * kernels and the same results, with S (and, on the column-major branch,
 * Pt) held in a scratch array inside the library instead of caller
 * workspaces.  The caller passes Q, K, V and O as for
 * splat_sparse_mhsa_unfused; the call allocates nothing.
 *
 * The scratch is a fixed SPLAT_NOALLOC_SCRATCH_BYTES (64 MiB) per device,
 * held by every GPU the library runs on until the process ends.  A call needs
 * B*H*nnz*4 bytes (rounded up to 256), plus B*H*nnz*4 more on the
 * column-major branch; a larger request returns SPLAT_ERR_UNSUPPORTED before
 * anything is enqueued.  The scratch is shared by every call on one device
 * and keeps the last call's contents (every value it needs is rewritten
 * first): calls that overlap on one device -- on different streams, or from
 * several host threads without ordering -- race, so a caller serialises them
 * (one stream does).  Other errors as splat_sparse_mhsa_unfused.
 */
#define SPLAT_NOALLOC_SCRATCH_BYTES (64u << 20)
splat_status splat_sparse_mhsa_unfused_noalloc(splat_acsr_t h, splat_dtype dtype, int32_t B,
                                               int32_t H, int32_t d, const void* Q, const void* K,
                                               const void* V, float scale, void* O,
                                               splat_dtype out_dtype, float alpha,
                                               int32_t* used_colmajor, void* stream);

/*
 * splat_sparse_mhsa_fwd -- the three steps fused: O = softmax_nz(scale * M (x) Q K^T) V
 * with an online (running max / running sum) softmax over the planned key
 * tiles, so S and P never reach device memory.  Q, K, V: [B,H,L,d] of `dtype`;
 * O: [B,H,L,d] of `out_dtype`.  bf16 inputs: scores and softmax in fp32, P
 * rounded toward zero to bf16 for the P V product (the row sum adds the same
 * rounded values), fp32 accumulation.  fp32 inputs: fp32 throughout.  A row
 * without non-zeros gets O = 0.
 */
splat_status splat_sparse_mhsa_fwd(splat_acsr_t h, splat_dtype dtype, int32_t B, int32_t H, int32_t d,
                                   const void* Q, const void* K, const void* V, float scale,
                                   void* O, splat_dtype out_dtype, void* stream);

/*
 * splat_debug_bounds -- index checks of a checked build (built with
 * -DSPLAT_DEBUG_BOUNDS: libsplat_checked.so beside libsplat.so; a debugging
 * aid, not part of the method).  In a checked build every kernel checks the
 * global-memory indices it derives from the plan and the ACSR runs -- query
 * rows (bit 0), key rows of K and V (bit 1), positions in S and P (bit 2),
 * positions in the column-major values (bit 3) -- against the sizes they
 * index; an index outside is recorded and replaced by 0, so the access stays
 * inside its buffer (the result is then wrong).  This call waits for the
 * current device (hipDeviceSynchronize), sets *flags to the bits recorded on
 * it since the last clear and, when `clear` is non-zero, clears them.
 * Returns SPLAT_ERR_UNSUPPORTED in the regular build, SPLAT_ERR_INVALID_ARG
 * for a NULL flags, SPLAT_ERR_HIP when the device reports an error.
 */
splat_status splat_debug_bounds(uint32_t* flags, int32_t clear);

/*
 * splat_debug_bounds_probe -- the checked build's test of its own mechanism:
 * runs one index check on the current device, `index` against [0, n) as
 * kind `kind` (0..3, the bits above), and sets *result to the checked index
 * (index, or 0 when outside, with the kind's bit then recorded for
 * splat_debug_bounds).  Allocates and frees one int of device memory and
 * synchronises.  SPLAT_ERR_UNSUPPORTED in the regular build,
 * SPLAT_ERR_INVALID_ARG for a NULL result or a kind outside 0..3.
 */
splat_status splat_debug_bounds_probe(int32_t kind, int32_t index, int32_t n, int32_t* result);

/* Message of the calling thread's last non-OK status ("" if none). */
const char* splat_last_error(void);

/* Library version string. */
const char* splat_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPLAT_H */
