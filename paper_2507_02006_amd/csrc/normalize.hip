// Values of the normalised adjacency (Sec. II-A, Eq. 2): for a square CSR
// pattern whose rows hold r_x stored entries, a_ik = 1 / sqrt(r_i r_k),
// i.e. D^-1/2 (A + I) D^-1/2 when the pattern is the symmetric adjacency
// with its self-loops.  The library derives these on the device from the
// row pointers instead of copying A's values, which saves a third of the
// bytes a streamed A sends over the host link.
//
// Arithmetic: r_i r_k is exact in double (both below 2^31), IEEE double
// square root and division are correctly rounded, and one rounding to fp32
// follows, so the value is the one a host computes as
// (float)(1.0 / sqrt((double)r_i * r_k)).
#include "kernels.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aires {
namespace kern {
namespace {

constexpr int NB_BLOCK = 256;
constexpr int NB_CHUNK = 2048;  // entries per workgroup step

// last row r in [lo, hi) with rp[r] <= x: for an entry position x that
// row holds it (rp[r] <= x < rp[r + 1]; empty rows are skipped)
template <typename RP>
__device__ __forceinline__ int64_t row_of(const RP* rp, int64_t x, int64_t lo, int64_t hi) {
  while (hi - lo > 1) {
    const int64_t mid = lo + (hi - lo) / 2;
    if ((int64_t)rp[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// Entries of rows [row0, row0 + nrows), NB_CHUNK at a time per workgroup:
// two searches over the row pointers find the rows of the chunk's first and
// last entry, the row pointers between them go to LDS, and each lane finds
// the row of its entry there (a chunk spans at most NB_CHUNK non-empty rows;
// when empty rows make the span longer than LDS holds, the lanes search the
// global row pointers instead).
template <typename RP>
__global__ __launch_bounds__(NB_BLOCK) void k_sym_norm(const RP* rp, int64_t row0, int64_t nrows, int64_t a_base,
                                                       const int32_t* acol, float* aval) {
  __shared__ int64_t srp[NB_CHUNK + 1];
  __shared__ int64_t span[2];
  const int64_t e0 = rp[row0], e1 = rp[row0 + nrows];
  for (int64_t s = e0 + (int64_t)blockIdx.x * NB_CHUNK; s < e1; s += (int64_t)gridDim.x * NB_CHUNK) {
    const int64_t last = s + NB_CHUNK - 1 < e1 ? s + NB_CHUNK - 1 : e1 - 1;
    if (threadIdx.x < 2) span[threadIdx.x] = row_of(rp, threadIdx.x == 0 ? s : last, row0, row0 + nrows);
    __syncthreads();
    const int64_t rs = span[0], rl = span[1];
    const bool staged = rl - rs + 2 <= NB_CHUNK + 1;
    if (staged)
      for (int64_t j = threadIdx.x; j <= rl - rs + 1; j += NB_BLOCK) srp[j] = (int64_t)rp[rs + j];
    __syncthreads();
    for (int64_t e = s + threadIdx.x; e <= last; e += NB_BLOCK) {
      int64_t ri;  // entries of the row that holds e
      if (staged) {
        int64_t lo = 0, hi = rl - rs + 1;  // last j in [0, hi) with srp[j] <= e
        while (hi - lo > 1) {
          const int64_t mid = lo + (hi - lo) / 2;
          if (srp[mid] <= e) lo = mid; else hi = mid;
        }
        ri = srp[lo + 1] - srp[lo];
      } else {
        const int64_t r = row_of(rp, e, rs, rl + 1);
        ri = (int64_t)rp[r + 1] - (int64_t)rp[r];
      }
      const int64_t k = acol[e - a_base];
      const double rk = (double)((int64_t)rp[k + 1] - (int64_t)rp[k]);
      aval[e - a_base] = (float)(1.0 / sqrt((double)ri * rk));
    }
    __syncthreads();  // srp and span are rewritten by the next chunk
  }
}

}  // namespace

hipError_t sym_norm_values(const void* rp, int rp64, int64_t row0, int64_t nrows, int64_t a_base,
                           const int32_t* acol, float* aval, int64_t nnz, hipStream_t s) {
  if (nrows <= 0 || nnz <= 0) return hipSuccess;
  int64_t grid = (nnz + NB_CHUNK - 1) / NB_CHUNK;
  if (grid > 8192) grid = 8192;
  if (rp64)
    hipLaunchKernelGGL((k_sym_norm<int64_t>), dim3((unsigned)grid), dim3(NB_BLOCK), 0, s,
                       static_cast<const int64_t*>(rp), row0, nrows, a_base, acol, aval);
  else
    hipLaunchKernelGGL((k_sym_norm<int32_t>), dim3((unsigned)grid), dim3(NB_BLOCK), 0, s,
                       static_cast<const int32_t*>(rp), row0, nrows, a_base, acol, aval);
  return hipGetLastError();
}

}  // namespace kern
}  // namespace aires
