// Host-side launch interface of the gfx950 kernels (no HIP types beyond
// hipStream_t / hipError_t).  Rows are tile-local: a kernel sees the tile's
// row pointers starting at its first row, and A's column/value arrays are
// indexed by (row_ptr value - a_base).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aires {
namespace kern {

constexpr int MAX_BINS = 8;

// Kinds of per-row work (see bin_plan in the runtime).
enum Kind : int {
  KIND_EMPTY = 0,       // P_i == 0: empty C row, no launch
  KIND_DENSE_WAVE = 1,  // one wavefront per row, dense LDS row of N slots (N <= 2048)
  KIND_DENSE_BLOCK = 2, // one workgroup per row, dense LDS row of N slots (N <= 16384)
  KIND_HASH_128 = 3,    // one wavefront per row, LDS hash of 128 slots
  KIND_HASH_1024 = 4,   // one wavefront per row, LDS hash of 1024 slots
  KIND_HASH_8192 = 5,   // one workgroup per row, LDS hash of 8192 slots
  KIND_WINDOWS = 6,     // wide rows: per-grain counts, then bitmap-rank column windows
  KIND_DENSE_SPLIT = 7, // heavy rows of a narrow product: runs of A entries per workgroup
  KIND_HASH_4096 = 8,   // one 256-thread workgroup per row, LDS hash of 4096 slots
};
constexpr int NUM_KINDS = 9;

struct BinThresholds {
  int32_t nb;                    // number of bins
  int32_t kind[MAX_BINS];
  int64_t max_p[MAX_BINS];       // bin b holds rows with max_p[b-1] < P_i <= max_p[b]
};

struct Operands {
  const void* arp; int rpa64; int64_t a_base; const int32_t* acol; const float* aval;
  const void* brp; int rpb64; const int32_t* bcol; const float* bval;
  int64_t K, N;
  // Column grains of a wide product: bidx[k*(nG+1) + g] = first position of
  // B_k with column >= g*G, for g in [0, nG]; nullptr when N is narrow.
  const int32_t* bidx; int32_t G; int32_t nG;
  // bmax[k] = max_j |b_kj| for wide products (the bound that lets a window
  // row accumulate in fixed point); nullptr: fp32 accumulation everywhere.
  const float* bmax;
};

struct BinView {
  const int32_t* list;     // tile-local row ids grouped by bin
  const int32_t* binoff;   // [nb+1] offsets into list (device)
  int32_t bin;             // first bin of the view
  int32_t bin_last = -1;   // last bin of the view (-1: same as bin)
  int32_t skip = 0;        // rows at the front of the bin left to another kernel
  __host__ __device__ int32_t last() const { return bin_last < 0 ? bin : bin_last; }
};

struct Outputs {
  int64_t* counts;         // symbolic: nnz of tile row (tile-local index)
  const int64_t* crp;      // numeric: C row pointers, tile-local index
  int32_t* ccol;           // numeric: C arrays, indexed by (crp value - c_base)
  float* cval;
};

// One column window of one wide row: grains [g0, g1), n entries of C,
// written at C position crp[row] + roff.
// Column slabs of the numeric window kernel: one per XCD of the MI355X,
// whose L2 caches are separate.
constexpr int WIN_MAX_SLABS = 8;

struct WinItem {
  int32_t row;
  uint16_t g0, g1;
  int32_t n;
  int32_t roff;
};

struct WindowParams {
  int32_t* gcnt;           // [row * nG + g] entries of C in grain g (per tile)
  int32_t grains_per_count_item;  // grains one symbolic item covers (windows never straddle items)
  int32_t max_grains;      // grains one window may span
  int32_t max_entries;     // entries one window may hold (>= G)
  int32_t pool_words;      // LDS words a window's bitmap (2 per bitmap word) and values (1 per entry) share
  int64_t* item_count;     // [1 + d]: windows of the d-th row of the bins; scanned into offsets
  WinItem* items;          // filled in the numeric sweep
  // zeroed before each window launch (dynamic row scheduling): [0] shared by
  // all workgroups, [1 + x] the rows of the slab bins for column slab x
  int32_t* row_counter;
  int32_t slab_bin;        // first bin whose rows' windows are spread over column slabs (-1: none)
  int32_t nslab;           // column slabs of the numeric launch (1..WIN_MAX_SLABS)
  // Presence bitmaps kept by the symbolic phase for heavy rows (nullptr:
  // none): the words of symbolic item (row, run of grains) start at
  // bm_off[row * items_per_row + item] (-1: not kept), so the numeric phase
  // reads them instead of marking the window from its products.
  uint32_t* bm_cache;
  int64_t bm_cap;                    // words the cache holds
  unsigned long long* bm_top;        // words handed out so far (zeroed once per call)
  int64_t* bm_off;                   // [row * items_per_row + item] per tile
  const int64_t* P;                  // intermediate products per tile row
  int64_t bm_min_products;           // rows with more products keep their bitmaps
  // 1: the windows of those rows are cut at symbolic items, as the symbolic
  // phase planned them; fixed for the call even if the cache is released
  // before the numeric phase (its windows then mark their bits again)
  int32_t item_cut;
};

// P_i per tile row and their total; rows longer than `long_row` entries are
// collected in long_list (count in *long_cnt) and summed by a workgroup each.
hipError_t analyze(const Operands& op, int64_t nrows, int64_t* P, unsigned long long* total,
                   int32_t* long_cnt, int32_t* long_list, hipStream_t s);
hipError_t bin_rows(const int64_t* P, int64_t nrows, const BinThresholds& th,
                    int32_t* cnt_cursor /*2*MAX_BINS zeroed*/, int32_t* binoff,
                    int32_t* list, hipStream_t s);
// phase: 0 symbolic, 1 numeric.  ub_rows: host upper bound on the bin size.
hipError_t run_bin(int kind, int phase, const Operands& op, const BinView& bv,
                   const Outputs& out, int64_t ub_rows, hipStream_t s);
// Dense slots of split rows: cap rows of N presence bits and N fp32 values.
struct SplitWs {
  uint32_t* bm;
  float* acc;
  int64_t cap;
};
// heavy narrow rows (phase 0 symbolic, 1 numeric); rows of the bin beyond
// sw.cap take the one-workgroup-per-row kernel
hipError_t split_rows(int phase, const Operands& op, const BinView& bv, const SplitWs& sw, const Outputs& out,
                      int64_t ub_rows, hipStream_t s);
// wide rows: symbolic grain counts + window plan (counts[row], item_count[1+d])
hipError_t windows_symbolic(const Operands& op, const BinView& bv, const WindowParams& wp,
                            const Outputs& out, int64_t ub_rows, hipStream_t s);
// wide rows: fill the window list (item_count scanned into offsets), then numeric
hipError_t windows_numeric(const Operands& op, const BinView& bv, const WindowParams& wp,
                           const Outputs& out, int64_t ub_rows, int64_t nitems, hipStream_t s);
// The grain index of B and bmax[k] = max_j |b_kj| (NaN if the row holds one).
hipError_t build_window_index(const void* brp, int rpb64, const int32_t* bcol, const float* bval, int64_t K,
                              int32_t G, int32_t nG, int32_t* bidx, float* bmax, hipStream_t s);
// In-place inclusive scan of x[0..n) plus x[-1] (the base): x[i] = x[-1] + sum_{j<=i} x[j].
size_t scan_workspace_bytes(int64_t n);
hipError_t scan_inplace(int64_t* x, int64_t n, void* ws, hipStream_t s);

// Y = act(A * W) for CSR A (m x K) and dense row-major W (ldw) and Y (ldy),
// F columns; relu != 0 applies max(0, .) before the store.  dense != 0
// takes the MFMA dense-tile kernel (K, ldw must satisfy spmm_dense_fits), else
// the entry-gather kernels.
bool spmm_dense_fits(int64_t K, int64_t ldw);
hipError_t spmm(const void* arp, int rpa64, const int32_t* acol, const float* aval, int64_t m, int64_t K,
                const float* W, int64_t ldw, int64_t F, float* Y, int64_t ldy, int relu, int dense, hipStream_t s);

// a_ik = 1/sqrt(r_i r_k) (Eq. 2) for the nnz entries of rows [row0, row0 +
// nrows) of a square CSR: rp holds the whole matrix's row pointers on the
// device, acol/aval are indexed by (entry position - a_base).
hipError_t sym_norm_values(const void* rp, int rp64, int64_t row0, int64_t nrows, int64_t a_base,
                           const int32_t* acol, float* aval, int64_t nnz, hipStream_t s);

size_t lds_bytes(int kind, int phase, int32_t W);
size_t grain_count_lds(int sg, int G);
size_t window_numeric_lds(int pool_words);
constexpr size_t kMaxLds = 160 * 1024;  // LDS of one gfx950 workgroup
// A window's bitmap in LDS: 8-byte words, each with WIN_WORD_BITS presence
// bits (low) and the 16-bit rank of its first set bit (high), so a window
// holds fewer than 65536 entries.
constexpr int WIN_WORD_BITS = 48;
__host__ __device__ constexpr int64_t win_words(int64_t cols) { return (cols + WIN_WORD_BITS - 1) / WIN_WORD_BITS; }
int group_size(int kind);

}  // namespace kern
}  // namespace aires
