/*
 * aires.h -- C-ABI of an MI355X (gfx950) library for the out-of-core sparse
 * product at the heart of GCN aggregation, after AIRES (Jayakody, Zhao,
 * Wang, "AIRES: Accelerating Out-of-Core GCNs via Algorithm-System
 * Co-Design", arXiv 2507.02006).
 *
 * The operation (Sec. II-A, Eq. 1 with Eq. 2): X = A_norm * H where A_norm is
 * the normalised sparse adjacency and H a sparse feature matrix, both in
 * compressed form.  Here: C = A * B with A (m x K) and B (K x N) in CSR and
 * C (m x N) returned in CSR with strictly increasing column indices per row.
 *
 * The paper pairs a CSR first operand with a CSC second operand and matches
 * rows against columns (Sec. II-B, Sec. III-B).  This library takes B in CSR
 * and uses the row-wise (Gustavson) formulation; the set of products and the
 * result are the same.
 *
 * Out-of-core execution follows the paper's row block-wise (RoBW) alignment
 * (Sec. III-A, Algorithm 1: blocks of whole rows of A whose bytes fit a
 * device budget, never splitting a row) and its three-phase schedule
 * (Sec. III-B, Algorithm 2: B resident on the device; A row blocks moved to
 * the device one at a time and multiplied; C stored, then moved to host).
 *
 * Conventions for every entry point
 *  - No exceptions cross this boundary.  Every call that can fail returns an
 *    aires_status: 0 on success, a negative code on error.  The text of the
 *    last error on the calling thread is available from aires_last_error().
 *  - Input matrices are BORROWED: the caller owns their memory and keeps it
 *    alive and unmodified until the last call on any plan built from them.
 *  - A plan is used by one thread at a time.
 *  - Streams are hipStream_t values passed as void*.  NULL means the
 *    device's null stream.
 *  - Device-resident pointers must be device memory of the current HIP
 *    device; host pointers must be host memory (pinned for streaming).
 */
#ifndef AIRES_H
#define AIRES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AIRES_ABI_VERSION 5

/* slots of aires_stats.kind_ms per phase (row kinds in use: 0 ... 8) */
#define AIRES_NUM_KINDS 16

typedef enum aires_status {
    AIRES_OK = 0,
    AIRES_E_INVALID_ARG = -1,  /* NULL pointer, bad enum, bad struct_size  */
    AIRES_E_INVALID_CSR = -2,  /* input fails the canonical-CSR check      */
    AIRES_E_DIM = -3,          /* A.ncols != B.nrows, negative sizes       */
    AIRES_E_BUDGET = -4,       /* device budget cannot hold B plus one row */
    AIRES_E_OVERFLOW = -5,     /* an index or size exceeds its type        */
    AIRES_E_OOM = -6,          /* an allocation failed                     */
    AIRES_E_HIP = -7,          /* a HIP runtime call failed                */
    AIRES_E_STATE = -8,        /* plan in use / wrong call order           */
    AIRES_E_UNSUPPORTED = -9,  /* combination not supported                */
    AIRES_E_CAPACITY = -10     /* caller output buffer too small           */
} aires_status;

/* Row-pointer width of an input matrix. */
typedef enum aires_idx { AIRES_IDX_I32 = 0, AIRES_IDX_I64 = 1 } aires_idx;

/* Where an array lives. */
typedef enum aires_mem {
    AIRES_MEM_DEVICE = 0,       /* HBM of the current device               */
    AIRES_MEM_HOST_PINNED = 1,  /* page-locked host memory (streamable)    */
    AIRES_MEM_HOST = 2          /* pageable host memory (planning only)    */
} aires_mem;

/*
 * Input CSR descriptor (borrowed).  Canonical form: row_ptr[0] == 0,
 * non-decreasing, row_ptr[nrows] == nnz; within a row, columns strictly
 * increasing in [0, ncols); values finite.  row_ptr has nrows + 1 entries
 * of the width given by rp_type.  All three arrays live in `mem`.
 */
typedef struct aires_csr {
    int64_t nrows, ncols, nnz;
    int32_t rp_type;            /* aires_idx                               */
    int32_t mem;                /* aires_mem                               */
    const void *row_ptr;
    const int32_t *col_idx;
    const float *vals;
} aires_csr;

/*
 * Output CSR descriptor.  row_ptr is ALWAYS int64 (nnz(C) can exceed 2^31)
 * and has nrows + 1 entries.  Arrays are allocated by the library (through
 * the plan's allocator, or hipMallocAsync / hipHostMalloc by default) and
 * owned by this struct until aires_csr_out_free().  `mem` says where they
 * live.  Zero-initialise before passing to aires_spgemm.
 */
typedef struct aires_csr_out {
    int64_t nrows, ncols, nnz;
    int64_t *row_ptr;
    int32_t *col_idx;
    float *vals;
    int32_t mem;                /* aires_mem of the three arrays           */
    int32_t _reserved;
    void *_owner;               /* library bookkeeping; do not touch       */
} aires_csr_out;

/*
 * Optional device-memory allocator.  alloc returns device memory usable on
 * `stream` (a hipStream_t) or NULL on failure; free releases it
 * stream-ordered on `stream`.  A NULL return makes the call fail with
 * AIRES_E_OOM after releasing what it had allocated.
 */
typedef struct aires_allocator {
    void *(*alloc)(void *ctx, size_t bytes, void *stream);
    void (*free)(void *ctx, void *ptr, void *stream);
    void *ctx;
} aires_allocator;

/*
 * Where A's values come from.  SYM_NORM: A is square and its values are
 * those of the normalised adjacency of Sec. II-A, Eq. 2,
 * a_ik = 1 / sqrt(r_i * r_k) with r_x the number of entries stored in row
 * x (D^-1/2 (A + I) D^-1/2 when the pattern is the symmetric adjacency with
 * its self-loops); they are computed on the device in double and rounded
 * once to fp32, A->vals is not read and may be NULL.  A streamed A then
 * sends only its row pointers (once) and column indices over the host link.
 */
typedef enum aires_avalues {
    AIRES_AVALUES_GIVEN = 0,
    AIRES_AVALUES_SYM_NORM = 1
} aires_avalues;

/* Upper bound used for the size of C when planning. */
typedef enum aires_cbound {
    AIRES_CBOUND_PRODUCTS = 0,  /* u_i = min(N, P_i), P_i = sum nnz(B_k)   */
    AIRES_CBOUND_DENSE = 1,     /* u_i = N                                 */
    AIRES_CBOUND_PAPER_EQ5 = 2, /* the paper's Eq. 5 estimate (not a bound;
                                   for planning experiments only)          */
    AIRES_CBOUND_ROWS = 3       /* u_i = min(N, nnz(A_i) * max_k nnz(B_k)):
                                   looser than PRODUCTS, but the planner
                                   reads no column of A (no gather)       */
} aires_cbound;

/*
 * How a streamed A is cut into segments.  ROBW: row blocks of whole rows
 * (Sec. III-A, Algorithm 1).  MAXFILL: the unaligned scheme the paper
 * measures against (Sec. I, Sec. III-A and Fig. 3; the MaxMemory baseline
 * of Sec. V-A): each segment is filled with as many of A's entries as its
 * slot holds, so it may end inside a row.  Only its complete rows are
 * multiplied; the entries of the partial last row are copied back to host
 * memory, packed on the host in front of the next segment's entries in a
 * pinned staging buffer, and sent again with them.  The product is the
 * same; the extra copies, host packing and waits are the merging overhead.
 */
typedef enum aires_segmentation {
    AIRES_SEG_ROBW = 0,
    AIRES_SEG_MAXFILL = 1
} aires_segmentation;

typedef struct aires_plan_opts {
    uint32_t struct_size;       /* = sizeof(aires_plan_opts)               */
    int32_t validate;           /* 1: canonical-CSR check of host inputs   */
    int32_t c_placement;        /* AIRES_MEM_DEVICE or AIRES_MEM_HOST_PINNED */
    int32_t c_bound;            /* aires_cbound                            */
    int32_t timing;             /* 1: record per-phase HIP events          */
    int32_t _pad0;
    int64_t max_tile_rows;      /* 0: no cap                               */
    int64_t max_tile_bytes;     /* cap on a tile's A bytes; 0: none, or for
                                   a streamed A max(A bytes / 16, 32 MB),
                                   so that copies overlap the products; a
                                   row above it is a tile of its own     */
    int64_t m_a_bytes;          /* > 0: plan exactly as Algorithm 1 with
                                   calcMem(k,q) = (k+1)*rp_bytes + 8q <=
                                   m_a_bytes, ignoring the budget split    */
    const aires_allocator *allocator; /* NULL: hipMallocAsync/hipFreeAsync */
    int64_t dense_max_cols;     /* 0: default (16384).  Widest N handled
                                   as a dense LDS row per output row       */
    int64_t hash_max_products;  /* 0: default, < 0: none.  Rows of a wide product with
                                   at most this many products use the LDS
                                   hash path                               */
    int64_t wave_max_products;  /* 0: default.  Rows with at most this many
                                   products are handled by one wavefront   */
    /* Wide products (N > dense_max_cols) cut columns into grains and rows
       into windows of whole grains; 0 = default for each.                 */
    int64_t window_grain_cols;  /* grain width, multiple of 32 (8192)      */
    int64_t window_max_grains;  /* grains one window may span (64)         */
    int64_t window_max_entries; /* C entries one window may hold, in
                                   [grain, 65535] (16384)                  */
    int64_t count_grains;       /* grains one symbolic item covers (24)    */
    int64_t keep_bitmap_products; /* 0: default (65536), < 0: never.  The
                                   symbolic phase keeps the presence bitmaps
                                   of rows with more products than this for
                                   the numeric phase (in-core runs, within a
                                   fifth of the budget the plan leaves)    */
    int64_t split_min_products; /* 0: default (65536), < 0: never.  Rows of
                                   a narrow product (N <= 2048) with more
                                   products are split over workgroups      */
    int64_t split_max_rows;     /* 0: default.  Cap on the rows given dense
                                   slots for splitting; further rows of the
                                   split bin take one workgroup each       */
    int64_t window_pool_bytes;  /* 0: default (38912).  LDS a window's
                                   bitmap (8 bytes per 48 columns) and
                                   values (4 bytes per entry) share; must
                                   hold one full grain                     */
    int32_t a_values;           /* aires_avalues: where A's values come
                                   from (AIRES_AVALUES_GIVEN)              */
    int32_t segmentation;       /* aires_segmentation, default ROBW;
                                   MAXFILL needs A in pinned host memory
                                   and given values                        */
    int64_t bitmap_cache_bytes; /* 0: default (a fifth of what the plan
                                   leaves of the budget, at most 32 GiB);
                                   > 0: at most this many bytes of kept
                                   symbolic bitmaps (items that do not fit
                                   are marked again in the numeric phase) */
    int64_t slab_min_products;  /* 0: default (262144), < 0: never.  Rows of
                                   a wide product with more products have
                                   their windows spread over column slabs
                                   in the numeric phase (one per XCD, so
                                   each XCD's L2 caches one slab of B);
                                   the result does not depend on it        */
} aires_plan_opts;

/*
 * A held in a file (the storage tier of Sec. III-B: A on the SSD, brought
 * to the host, then to the GPU).  The three CSR arrays are raw arrays in
 * the file at the given byte offsets: row pointers (nrows + 1 of rp_type),
 * column indices (nnz int32), values (nnz fp32; not read when A's values
 * are derived, AIRES_AVALUES_SYM_NORM).  direct_io = 1 asks for reads that
 * bypass the page cache (O_DIRECT, in whole 4 KiB blocks), falling back
 * to ordinary reads where the filesystem refuses.
 */
typedef struct aires_file_csr {
    int64_t nrows, ncols, nnz;
    int32_t rp_type;            /* aires_idx                               */
    int32_t direct_io;
    const char *path;
    int64_t row_ptr_offset, col_idx_offset, vals_offset;
} aires_file_csr;

/* Fill *o with defaults (struct_size set, validate 0, C on device). */
aires_status aires_plan_opts_default(aires_plan_opts *o);

typedef struct aires_plan aires_plan;

/*
 * aires_tile_plan -- RoBW row-block partition of A (Sec. III-A, Algorithm 1;
 * budget split after Eqs. 6-7).
 *
 * A: m x K, B: K x N.  hbm_budget caps every device byte the library
 * allocates or uses during aires_spgemm/aires_stream_tiles: resident B
 * (M_B of Eq. 6: values, column ids, row pointers), A (resident, or two
 * double-buffered tile slots when A is in host memory), C (resident, or two
 * tile slots sized by the tile's C bound when C is placed in host memory),
 * and workspace.  0 means "the device's free memory".  Each tile is a
 * maximal run of whole rows [r0, r1) whose per-tile bytes fit what the
 * budget leaves after the resident parts, found greedily from row 0 as in
 * Algorithm 1.  With opts->m_a_bytes > 0, tiles follow Algorithm 1 exactly
 * with calcMem(k, q) <= m_a_bytes.
 *
 * Planning reads A.row_ptr on the host (copying it from the device when A
 * is device-resident) and, for a host-resident A with C placed in host
 * memory, computes P_i on the host for the C bound.  It launches no
 * kernels.
 *
 * Errors: AIRES_E_INVALID_ARG (NULL A/B/out, bad enums), AIRES_E_DIM,
 * AIRES_E_INVALID_CSR (opts->validate and a host input is not canonical),
 * AIRES_E_BUDGET (B plus one row plus workspace exceeds the budget; this
 * includes a single row larger than the tile budget), AIRES_E_OVERFLOW,
 * AIRES_E_UNSUPPORTED (an input in pageable host memory with no m_a_bytes
 * planning-only use), AIRES_E_HIP.  *out is untouched on error.
 */
aires_status aires_tile_plan(const aires_csr *A, const aires_csr *B, uint64_t hbm_budget,
                             const aires_plan_opts *opts, aires_plan **out);

/*
 * aires_tile_plan_file -- the same plan for an A that stays in a file.  The
 * planner reads A's row pointers (into pinned host memory the plan keeps)
 * and nothing else, so the C bound must come from row pointers:
 * opts->c_bound = AIRES_CBOUND_ROWS, DENSE or PAPER_EQ5, row blocks, no
 * validation.  The plan is streamed (aires_spgemm / aires_stream_tiles):
 * each tile's column indices and values are read from the file into one of
 * two pinned staging buffers while earlier tiles copy and compute, then sent
 * to the device as for a pinned-host A (Algorithm 2 with the first stage on
 * storage).  The file stays open until aires_plan_destroy.
 * Errors: AIRES_E_INVALID_ARG (NULL, bad offsets, file cannot be opened or
 * is too short), AIRES_E_INVALID_CSR (row pointers do not run from 0 to
 * nnz), AIRES_E_UNSUPPORTED (a C bound that needs A's columns, max-fill
 * segments, validation), and the errors of aires_tile_plan.
 */
aires_status aires_tile_plan_file(const aires_file_csr *A, const aires_csr *B, uint64_t hbm_budget,
                                  const aires_plan_opts *opts, aires_plan **out);

/*
 * aires_csr_read_file -- a CSR held in a file (laid out as for
 * aires_tile_plan_file) brought whole into device memory (mem =
 * AIRES_MEM_DEVICE) or pinned host memory (AIRES_MEM_HOST_PINNED): the way
 * the storage tier of Sec. III-B moves B from the SSD to the GPU before the
 * tiles stream, here through host memory, as this platform has no GPU file
 * API.  For device memory the column indices and values are read in chunks
 * of chunk_bytes (0: 64 MiB; rounded up to 4 KiB) into two pinned staging
 * buffers, and each chunk is sent with hipMemcpyAsync on `stream` (a
 * hipStream_t; NULL: the null stream) while the next one is read.  Row
 * pointers are checked (0 to nnz, non-decreasing) and widened to int64.
 * On success *out holds the matrix, owned by the caller until
 * aires_csr_out_free; device arrays come from `alloc` (NULL: hipMallocAsync)
 * on `stream`.  Returns once every copy is complete.  With st non-NULL it
 * receives the bytes read from the file and the times taken.
 * Errors: AIRES_E_INVALID_ARG (NULL, mem, negative offsets or chunk size,
 * file cannot be opened or is too short), AIRES_E_DIM, AIRES_E_OVERFLOW,
 * AIRES_E_INVALID_CSR (row pointers), AIRES_E_OOM, AIRES_E_HIP; *out is
 * untouched on error.
 */
typedef struct aires_read_stats {
    int64_t bytes_read;         /* bytes of the three arrays read           */
    double read_ms;             /* time in file reads                      */
    double total_ms;            /* the whole call                          */
} aires_read_stats;

aires_status aires_csr_read_file(const aires_file_csr *M, int32_t mem, const aires_allocator *alloc, void *stream,
                                 int64_t chunk_bytes, aires_csr_out *out, aires_read_stats *st);

typedef struct aires_plan_info {
    int64_t ntiles;
    int64_t m, k, n;            /* A is m x k, B is k x n                  */
    int64_t budget;             /* effective budget in bytes               */
    int64_t b_bytes;            /* M_B                                     */
    int64_t a_bytes;            /* bytes of all of A                       */
    int64_t tile_budget;        /* bytes available to one tile slot        */
    int64_t peak_bytes;         /* planned peak device bytes               */
    int64_t c_bound_entries;    /* sum of u_i, or -1 when not computed     */
    int32_t a_streamed;         /* 1: A moves host->device per tile        */
    int32_t c_on_host;          /* 1: C tiles move device->host            */
    int64_t part_budget;        /* slot bytes the tiles were cut under:
                                   tile_budget, or less when the largest
                                   row count, entry count and C bound of
                                   different tiles would not fit one slot
                                   together                                */
    int32_t a_in_file;          /* 1: A's entries are read from a file     */
    int32_t _pad1;
} aires_plan_info_t;            /* (the struct tag shares the query's name) */

typedef struct aires_tile {
    int64_t r0, r1;             /* rows [r0, r1)                           */
    int64_t nnz0, nnz1;         /* A.row_ptr[r0], A.row_ptr[r1]            */
    int64_t a_bytes;            /* (r1-r0+1)*rp_bytes + 8*(nnz1-nnz0)      */
    int64_t c_bound_entries;    /* sum of u_i over the tile, or -1         */
    int64_t tile_bytes;         /* planned bytes of one slot of this tile  */
    int64_t sent_nnz1;          /* A entries [nnz0, sent_nnz1) are sent:
                                   nnz1 for row blocks; beyond nnz1 for a
                                   max-fill segment ending inside a row    */
} aires_tile;

/*
 * aires_plan_info -- the plan's totals: tile count, sizes, the budget M and
 * its split (M_B of Eq. 6, the slot left for A tiles as in Eq. 7), planned
 * peak device bytes and the C bound (Sec. III-A).  aires_plan_info_get is
 * the same call under its earlier name.  Errors: AIRES_E_INVALID_ARG.
 */
aires_status aires_plan_info(const aires_plan *plan, aires_plan_info_t *info);
aires_status aires_plan_info_get(const aires_plan *plan, aires_plan_info_t *info);
/* Tile t of the plan (0 <= t < ntiles): a row block of Algorithm 1.
   Errors: AIRES_E_INVALID_ARG (NULL, t out of range). */
aires_status aires_plan_tile(const aires_plan *plan, int64_t t, aires_tile *tile);

/*
 * aires_spgemm -- C = A * B over the plan's tiles (Algorithm 2, Phase II
 * per tile; C = A_norm * H of Eq. 1).
 *
 * Device-resident A: every kernel runs on `stream`.  For each tile: row
 * analysis (intermediate products P_i), binning, symbolic phase (nnz of each
 * row of C); then one device-wide scan gives C.row_ptr, the library reads
 * nnz(C) back (the single host synchronisation: the size of C is data
 * dependent, Sec. I and Sec. III-B), allocates C exactly, and runs the
 * numeric phase tile by tile.  C is device-resident.
 *
 * Host-resident (pinned) A: delegates to aires_stream_tiles with internal
 * copy streams.
 *
 * Returns once all work is enqueued and C's arrays exist; C's contents are
 * valid when `stream` reaches the end of the enqueued work.  Columns of
 * every row of C are strictly increasing; entries whose value sums to zero
 * are kept (the structure is the union of the column sets).
 *
 * Values (Eq. 1, c_ij = sum_k a_ik b_kj): fp32 products summed in fp32 in an
 * unspecified order, except in rows of wide products (N above the densest
 * row the device holds in LDS) handled by column windows whose bound
 * S_i = sum_k |a_ik| max_j |b_kj| allows 32-bit fixed point: there the
 * products are scaled by 2^f (S_i < 2^(30-f)), rounded to integers and
 * summed exactly, so an entry's error is at most |A_i| 2^-(f+1) <= 1e-6
 * plus its final rounding to fp32, and its value does not depend on the
 * order of the products.  An entry made of a single product is therefore
 * exact in fp32 rows but rounded to a multiple of 2^-f in fixed-point rows
 * (so C = A * I reproduces A only within that bound there).
 *
 * Memory (the constraint M of Sec. III-A): every block the call takes from
 * the allocator, C included, counts against the plan's budget together
 * with the caller's device-resident inputs; an allocation that would pass
 * it fails the call with AIRES_E_BUDGET (the kept symbolic bitmaps, a
 * cache, are dropped first).  Every block is requested and released on
 * `stream` (the allocator's stream argument), so an allocator that pools
 * per stream never hands a block still in use by this call to other work.
 * Errors: AIRES_E_INVALID_ARG, AIRES_E_STATE (C not zeroed / plan busy),
 * AIRES_E_BUDGET (exact C does not fit), AIRES_E_OOM (the allocator
 * returned NULL; everything taken so far is released), AIRES_E_HIP,
 * AIRES_E_OVERFLOW.
 */
aires_status aires_spgemm(aires_plan *plan, void *stream, aires_csr_out *C);

/*
 * aires_spgemm_noalloc -- aires_spgemm for callers that cannot allocate
 * device memory (code that must not call hipMalloc: tight serving loops,
 * harnesses that forbid allocation).  Same product, same kernels, but the
 * call allocates nothing: its workspace is a fixed array of 64 MiB that the
 * library holds on each device until the process ends, and C goes into
 * arrays the caller owns.
 *
 * plan: from aires_tile_plan with A and B on the device (the plan's budget
 * and allocator are not used; the kept symbolic bitmaps of wide rows are
 * not used either).  c_row_ptr: device, m + 1 int64 entries, always
 * written.  c_col_idx / c_vals: device arrays of c_capacity entries (may
 * be NULL when c_capacity is 0).  *nnz_out (may be NULL) receives nnz(C),
 * or -1 if the call failed before it was known.  Work is enqueued on
 * `stream`; the call synchronises it once (to read nnz(C), as aires_spgemm
 * does) and returns with the numeric phase enqueued.
 *
 * Every call on a device shares that device's array, which keeps the last
 * call's contents: calls that overlap on one device (other streams or
 * threads) race and must not be issued.  Counters the kernels need cleared
 * are cleared by each call.
 * Errors: AIRES_E_INVALID_ARG (NULL plan / arrays, negative capacity),
 * AIRES_E_UNSUPPORTED (A or B not on the device), AIRES_E_STATE (plan in
 * use), AIRES_E_CAPACITY (the workspace does not fit the 64 MiB array, or
 * nnz(C) > c_capacity: C.row_ptr and *nnz_out are then valid and the
 * call may be repeated with larger arrays), AIRES_E_HIP.
 */
aires_status aires_spgemm_noalloc(aires_plan *plan, void *stream, int64_t *c_row_ptr, int32_t *c_col_idx,
                                  float *c_vals, int64_t c_capacity, int64_t *nnz_out);

/*
 * aires_stream_tiles -- out-of-core Phase II/III of Algorithm 2 for a
 * host-resident (pinned) A: B is copied to the device once (Phase I); for
 * each tile, its contiguous row_ptr/col/val slices are copied on `h2d` into
 * one of two device slots while the previous tile computes on `compute`;
 * each finished C tile is copied on `d2h` into pinned host memory at the
 * running offset (opts->c_placement == AIRES_MEM_HOST_PINNED) or kept on
 * the device.  The host waits only for each tile's nnz, one tile behind.
 * C's arrays are sized by the plan's C bound; where that bound was only an
 * estimate (AIRES_CBOUND_PAPER_EQ5) and C outgrows it, they are replaced by
 * larger ones (by half again at least) and the entries so far moved over,
 * within the budget when C is on the device.  On return all work has
 * completed and C is valid.
 * Errors: as aires_spgemm, plus AIRES_E_UNSUPPORTED if A is not pinned.
 */
aires_status aires_stream_tiles(aires_plan *plan, void *h2d, void *compute, void *d2h,
                                aires_csr_out *C);

typedef struct aires_stats {
    int64_t ntiles;
    int64_t products;           /* sum of P_i (2 flops each)               */
    int64_t nnz_c;
    int64_t h2d_bytes, d2h_bytes;
    int64_t host_syncs;
    /* milliseconds from HIP events (opts->timing), summed over tiles.
       h2d_ms / d2h_ms: busy time of the copy streams (events around each
       tile's copies, after its waits).  total_ms: the whole call on the
       compute stream, output allocation included.                        */
    double analyze_ms, bin_ms, symbolic_ms, scan_ms, numeric_ms;
    double h2d_ms, d2h_ms, total_ms;
    int64_t numeric_launches;   /* numeric-phase kernel launches           */
    /* milliseconds per kernel kind (index = kind id of the row bins:
       0 empty, 1 dense-wave, 2 dense-block, 3 hash-128, 4 hash-1024,
       5 hash-8192, 6 column windows, 7 split rows, 8 hash-4096; the
       other slots stay 0); [0] symbolic, [1] numeric phase                */
    double kind_ms[2][AIRES_NUM_KINDS];
    /* streamed calls: from the first copy of Phase I to the last copy of
       Phase III (the tile pipeline, without the output allocation)       */
    double pipeline_ms;
    /* max-fill segments: entries of partial rows copied back and sent
       again (8 bytes each, counted in d2h_bytes and h2d_bytes too), and
       the host time spent packing segments into the staging buffers      */
    int64_t resent_bytes;
    double merge_ms;
    /* A in a file: bytes read from it for the tiles and the host time the
       reads took (they run one tile ahead of the copies to the device)    */
    int64_t storage_bytes;
    double storage_ms;
} aires_stats;

/* Activation applied by aires_spmm. */
typedef enum aires_act { AIRES_ACT_NONE = 0, AIRES_ACT_RELU = 1 } aires_act;

/* Kernel family of aires_spmm. */
typedef enum aires_spmm_algo {
    AIRES_SPMM_AUTO = 0,        /* DENSE_TILES when nnz(A) >= m*K/8, K <= 2^20
                                   and ldw < 2^23, else ROWS                 */
    AIRES_SPMM_ROWS = 1,        /* each entry a_ik scales row k of W         */
    AIRES_SPMM_DENSE_TILES = 2  /* 64-row tiles of A densified in LDS, fp32
                                   matrix cores; work ~ m*K*F               */
} aires_spmm_algo;

/*
 * aires_spmm -- Y = act(A * W) for a sparse A and a dense W: the
 * combination step of a GCN layer (Sec. II-A, Eq. 3: the aggregated
 * features times the layer's weights, then the activation sigma, e.g.
 * ReLU), and, with a dense feature matrix in place of W, the aggregation of
 * Eq. 1 (the backward pass of a layer multiplies by the symmetric A_norm
 * the same way).
 *
 * A: CSR descriptor with A->mem == AIRES_MEM_DEVICE (borrowed; rows m =
 * A->nrows, K = A->ncols; canonical: columns in [0, K), strictly increasing
 * per row).  W: device, row-major K x F, row stride ldw >= F elements.
 * Y: device, row-major m x F, row stride ldy >= F, owned by the caller;
 * every element of the m x F block is overwritten (rows of A with no
 * entries give act(0) = 0); columns between F and ldy are untouched.
 * Work is enqueued on `stream` (a hipStream_t); the call allocates nothing
 * and returns once the kernels are enqueued.  Each element is a sum in
 * fp32 over the row's products a_ik * w_kj in an unspecified order.
 * DENSE_TILES also multiplies the row's absent entries, as zeros, with W:
 * for finite W that adds exact zeros and changes nothing, but an Inf or NaN
 * in row k of W then reaches every row of Y, not only rows with an entry
 * in column k.  AUTO assumes W is finite (as layer weights are).
 * Errors: AIRES_E_INVALID_ARG (NULL arrays, ldw < F, ldy < F, bad act or
 * algo), AIRES_E_UNSUPPORTED (A not on the device, F >= 2^31, DENSE_TILES
 * with K > 2^20 or ldw >= 2^23), AIRES_E_HIP.
 */
aires_status aires_spmm(const aires_csr *A, const float *W, int64_t ldw, int64_t F, float *Y, int64_t ldy,
                        aires_act act, aires_spmm_algo algo, void *stream);

/* Statistics of the last aires_spgemm / aires_stream_tiles on the plan. */
aires_status aires_plan_stats(const aires_plan *plan, aires_stats *stats);

/*
 * Per-tile statistics of the last call on the plan: what the paper reports
 * per method (bytes moved between host and GPU and their latency, Sec. V-B)
 * broken down by row block.  Counts are always filled; times need
 * opts->timing (else 0, and the instants -1).  Durations are the busy time
 * of each phase of this tile on its stream.  The instants are milliseconds
 * from the start of the call on the compute stream: the tile's host-to-
 * device copy, its compute (analysis through numeric phase) and its copy of
 * C back (streamed schedule of Algorithm 2; -1 where the tile has none), so
 * that the overlap of tile t+1's copy with tile t's products can be read
 * off directly.
 */
typedef struct aires_tile_stats {
    int64_t r0, r1;             /* rows [r0, r1) of the tile               */
    int64_t products;           /* sum of P_i over the tile                */
    int64_t nnz_c;              /* entries of C in the tile                */
    int64_t h2d_bytes;          /* A bytes copied for the tile             */
    int64_t d2h_bytes;          /* C bytes (row pointers + entries) copied back */
    double analyze_ms, bin_ms, symbolic_ms, scan_ms, numeric_ms;
    double h2d_ms, d2h_ms;
    double h2d_begin_ms, h2d_end_ms;
    double compute_begin_ms, compute_end_ms;
    double d2h_begin_ms, d2h_end_ms;
    int64_t resent_bytes;       /* max-fill: partial-row bytes copied back
                                   after this segment and sent again with
                                   the next one (in d2h_bytes here)        */
    double merge_ms;            /* max-fill: host time packing this
                                   segment's staging buffer                */
    double storage_ms;          /* A in a file: host time reading this
                                   tile's entries                          */
} aires_tile_stats;

/* Errors: AIRES_E_INVALID_ARG (NULL, t out of range), AIRES_E_HIP. */
aires_status aires_plan_tile_stats(const aires_plan *plan, int64_t t, aires_tile_stats *stats);

/* Release C's arrays through the allocator that made them; zeroes *C. */
void aires_csr_out_free(aires_csr_out *C);
void aires_plan_destroy(aires_plan *plan);
const char *aires_status_string(aires_status s);
const char *aires_last_error(void);
int aires_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* AIRES_H */
