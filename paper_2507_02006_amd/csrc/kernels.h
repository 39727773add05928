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
  KIND_DENSE_WAVE = 1,  // one wavefront per row, dense LDS window = N (N <= 2048)
  KIND_DENSE_BLOCK = 2, // one workgroup per (row, column window), window <= 16384
  KIND_HASH_128 = 3,    // one wavefront per row, LDS hash of 128 slots
  KIND_HASH_1024 = 4,   // one wavefront per row, LDS hash of 1024 slots
  KIND_HASH_8192 = 5,   // one workgroup per row, LDS hash of 8192 slots
};

struct BinThresholds {
  int32_t nb;                    // number of bins
  int32_t kind[MAX_BINS];
  int64_t max_p[MAX_BINS];       // bin b holds rows with max_p[b-1] < P_i <= max_p[b]
};

struct Operands {
  const void* arp; int rpa64; int64_t a_base; const int32_t* acol; const float* aval;
  const void* brp; int rpb64; const int32_t* bcol; const float* bval;
  int64_t K, N;
  // column windows (wide products): bidx[w*K + k] = first position of B_k with
  // column >= w*W, for w in [0, nwin]; nullptr for a single window.
  const int32_t* bidx; int32_t W; int32_t nwin;
};

struct BinView {
  const int32_t* list;     // tile-local row ids grouped by bin
  const int32_t* binoff;   // [nb+1] offsets into list (device)
  int32_t bin;
};

struct Outputs {
  int64_t* counts;         // symbolic: nnz of tile row (tile-local index)
  int32_t* wcnt;           // windowed rows: [row*nwin + w] counts, later offsets
  const int64_t* crp;      // numeric: C row pointers, tile-local index
  int32_t* ccol;
  float* cval;
};

hipError_t analyze(const Operands& op, int64_t nrows, int64_t* P,
                   unsigned long long* total, hipStream_t s);
hipError_t bin_rows(const int64_t* P, int64_t nrows, const BinThresholds& th,
                    int32_t* cnt_cursor /*2*MAX_BINS zeroed*/, int32_t* binoff,
                    int32_t* list, hipStream_t s);
// phase: 0 symbolic, 1 numeric.  ub_rows: host upper bound on the bin size.
hipError_t run_bin(int kind, int phase, const Operands& op, const BinView& bv,
                   const Outputs& out, int64_t ub_rows, hipStream_t s);
hipError_t window_rowsum(const BinView& bv, int32_t nwin, int32_t* wcnt, int64_t* counts,
                         int64_t ub_rows, hipStream_t s);
hipError_t build_window_index(const void* brp, int rpb64, const int32_t* bcol, int64_t K,
                              int32_t W, int32_t nwin, int32_t* bidx, hipStream_t s);
// In-place inclusive scan of x[0..n) plus x[-1] (the base): x[i] = x[-1] + sum_{j<=i} x[j].
size_t scan_workspace_bytes(int64_t n);
hipError_t scan_inplace(int64_t* x, int64_t n, void* ws, hipStream_t s);

// LDS bytes one block of a kind needs (0 if unknown)
size_t lds_bytes(int kind, int phase, int32_t W);
int group_size(int kind);

}  // namespace kern
}  // namespace aires
