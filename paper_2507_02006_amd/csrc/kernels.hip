// gfx950 (CDNA4, wave64) kernels for C = A * B with A, B, C in CSR.
//
// The product is the GCN aggregation of Sec. II-A (Eq. 1) with a sparse
// feature operand.  It is not a dense contraction, so nothing here uses
// MFMA: every phase is bound by memory traffic or LDS atomics.
//
// Per row-block tile the runtime launches:
//   analyze      P_i = sum_{k in A_i} nnz(B_k)  (intermediate products)
//   bin_rows     rows grouped by P_i into per-kind work lists
//   symbolic     nnz(C_i) per row (or per (row, column window))
//   scan         C.row_ptr = base + inclusive prefix sum of nnz(C_i)
//   numeric      C_i = sum_k a_ik B_k, written with strictly increasing columns
//
// Accumulators live in LDS:
//   dense window  fp32 slots for a window of W consecutive columns plus a
//                 presence bitmap; compaction walks the bitmap, so the
//                 output comes out sorted with no sort at all.
//   hash          open addressing (linear probing) keyed by column; the
//                 occupied slots are compacted and bitonic-sorted in LDS.
// A product's intermediate terms are spread over the threads of a group by
// a flattened loop: the group loads up to GROUP entries (k, a_ik) of A_i,
// scans the lengths of the matching B rows, and each thread takes every
// GROUP-th term, finding its B row by binary search in the scanned lengths.
// Consecutive threads therefore read consecutive entries of a B row.
#include "kernels.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aires {
namespace kern {
namespace {

constexpr int WAVE = 64;

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Orders LDS traffic between the lanes of one wavefront (they execute in
// lockstep; this stops the compiler from moving LDS accesses across).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
#pragma unroll
  for (int d = 1; d < WAVE; d <<= 1) {
    T u = __shfl_up(v, d, WAVE);
    if (lane_id() >= d) v += u;
  }
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int d = WAVE / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, WAVE);
  return v;
}

// A cooperating group: one wavefront (GROUP == 64) or the whole block.
template <int GROUP, int BLOCK>
struct Group {
  static_assert(GROUP == WAVE || GROUP == BLOCK, "group is a wave or the block");
  static constexpr int NWAVES = GROUP / WAVE;
  int64_t* red;  // NWAVES scratch words in LDS (block groups only)

  __device__ __forceinline__ int t() const { return GROUP == WAVE ? lane_id() : (int)threadIdx.x; }
  __device__ __forceinline__ void sync() const {
    if constexpr (GROUP == WAVE) wave_sync(); else __syncthreads();
  }
  // inclusive scan over the group; *total receives the group sum
  __device__ __forceinline__ int64_t incl_scan(int64_t v, int64_t* total) const {
    int64_t x = wave_incl_scan(v);
    if constexpr (GROUP == WAVE) {
      *total = __shfl(x, WAVE - 1, WAVE);
      return x;
    } else {
      const int w = threadIdx.x / WAVE;
      if (lane_id() == WAVE - 1) red[w] = x;
      __syncthreads();
      int64_t pre = 0, tot = 0;
#pragma unroll
      for (int i = 0; i < NWAVES; ++i) {
        int64_t s = red[i];
        pre += (i < w) ? s : 0;
        tot += s;
      }
      __syncthreads();
      *total = tot;
      return x + pre;
    }
  }
  __device__ __forceinline__ int64_t sum(int64_t v) const {
    int64_t tot;
    incl_scan(v, &tot);
    return tot;
  }
};

template <typename RP>
__device__ __forceinline__ int64_t ld_rp(const void* rp, int64_t i) {
  return (int64_t)static_cast<const RP*>(rp)[i];
}

// ---------------------------------------------------------------- analyze

// P_i for every tile row, 16 lanes per row.
template <typename RA, typename RB>
__global__ __launch_bounds__(256) void k_analyze(const Operands op, int64_t nrows, int64_t* P,
                                                 unsigned long long* total) {
  const int sub = threadIdx.x & 15;
  const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  int64_t s = 0;
  if (row < nrows) {
    const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
    for (int64_t p = ld_rp<RA>(op.arp, row) - op.a_base + sub; p < p1; p += 16) {
      const int64_t k = op.acol[p];
      s += ld_rp<RB>(op.brp, k + 1) - ld_rp<RB>(op.brp, k);
    }
  }
#pragma unroll
  for (int d = 8; d > 0; d >>= 1) s += __shfl_xor(s, d, 16);
  if (row < nrows && sub == 0) P[row] = s;
  int64_t w = (sub == 0) ? s : 0;
  w = wave_sum(w);
  if (lane_id() == 0 && w) atomicAdd(total, (unsigned long long)w);
}

// ----------------------------------------------------------------- binning

__device__ __forceinline__ int bin_of(const BinThresholds& th, int64_t p) {
  int b = 0;
  while (b < th.nb - 1 && p > th.max_p[b]) ++b;
  return b;
}

__global__ __launch_bounds__(256) void k_bin_count(const int64_t* P, int64_t nrows,
                                                   const BinThresholds th, int32_t* cnt) {
  __shared__ int32_t h[MAX_BINS];
  if (threadIdx.x < MAX_BINS) h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nrows) atomicAdd(&h[bin_of(th, P[i])], 1);
  __syncthreads();
  if (threadIdx.x < th.nb && h[threadIdx.x]) atomicAdd(&cnt[threadIdx.x], h[threadIdx.x]);
}

__global__ __launch_bounds__(256) void k_bin_scatter(const int64_t* P, int64_t nrows,
                                                     const BinThresholds th, const int32_t* cnt,
                                                     int32_t* cursor, int32_t* binoff,
                                                     int32_t* list) {
  __shared__ int32_t h[MAX_BINS], off[MAX_BINS + 1], base[MAX_BINS];
  if (threadIdx.x == 0) {
    int32_t s = 0;
    for (int b = 0; b < th.nb; ++b) { off[b] = s; s += cnt[b]; }
    off[th.nb] = s;
    if (blockIdx.x == 0)
      for (int b = 0; b <= th.nb; ++b) binoff[b] = off[b];
  }
  if (threadIdx.x < MAX_BINS) h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int b = 0, r = 0;
  if (i < nrows) {
    b = bin_of(th, P[i]);
    r = atomicAdd(&h[b], 1);
  }
  __syncthreads();
  if (threadIdx.x < th.nb && h[threadIdx.x]) base[threadIdx.x] = atomicAdd(&cursor[threadIdx.x], h[threadIdx.x]);
  __syncthreads();
  if (i < nrows) list[off[b] + base[b] + r] = (int32_t)i;
}

// ---------------------------------------------------- flattened product loop

// Per-group LDS for one chunk of A_i: inclusive term counts, the B position
// of term 0 of each segment (shifted so pos = s_shift[c] + q), and a_ik.
template <int GROUP>
struct Chunk {
  int64_t incl[GROUP];
  int64_t shift[GROUP];
  float av[GROUP];
};

// Calls f(pos, a_ik) for every term of row `row` restricted to window w.
template <typename RA, typename RB, int GROUP, int BLOCK, bool NUM, bool WIDE, typename F>
__device__ __forceinline__ void for_each_term(const Operands& op, const Group<GROUP, BLOCK>& g,
                                              Chunk<GROUP>& ch, int64_t row, int64_t w, F&& f) {
  const int t = g.t();
  const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
  const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
  for (int64_t cb = p0; cb < p1; cb += GROUP) {
    const int64_t p = cb + t;
    int64_t lo = 0, len = 0;
    float av = 0.f;
    if (p < p1) {
      const int64_t k = op.acol[p];
      if constexpr (NUM) av = op.aval[p];
      if constexpr (WIDE) {
        lo = op.bidx[w * op.K + k];
        len = (int64_t)op.bidx[(w + 1) * op.K + k] - lo;
      } else {
        lo = ld_rp<RB>(op.brp, k);
        len = ld_rp<RB>(op.brp, k + 1) - lo;
      }
    }
    int64_t total;
    const int64_t incl = g.incl_scan(len, &total);
    ch.incl[t] = incl;
    ch.shift[t] = lo - (incl - len);
    if constexpr (NUM) ch.av[t] = av;
    g.sync();
    const int nseg = (int)((p1 - cb) < GROUP ? (p1 - cb) : GROUP);
    for (int64_t q = t; q < total; q += GROUP) {
      int a = 0, b = nseg - 1;
      while (a < b) {
        const int mid = (a + b) >> 1;
        if (ch.incl[mid] > q) b = mid; else a = mid + 1;
      }
      f(ch.shift[a] + q, NUM ? ch.av[a] : 0.f);
    }
    g.sync();
  }
}

// -------------------------------------------------------- dense window path

// LDS layout of one group: [bitmap W/32 words][acc W floats if NUM][Chunk][red]
__host__ __device__ constexpr size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

template <int GROUP, bool NUM>
__host__ __device__ constexpr size_t dense_group_bytes(int W) {
  return align16(((size_t)W + 31) / 32 * 4) + (NUM ? align16((size_t)W * 4) : 0) +
         align16(sizeof(Chunk<GROUP>)) + 64;
}

template <typename RA, typename RB, int GROUP, int BLOCK, bool NUM, bool WIDE>
__global__ __launch_bounds__(BLOCK) void k_dense(const Operands op, const BinView bv,
                                                 const Outputs out) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NG = BLOCK / GROUP;
  const int W = WIDE ? op.W : (int)op.N;
  const size_t per = dense_group_bytes<GROUP, NUM>(W);
  const int gi = threadIdx.x / GROUP;
  unsigned char* base = smem + gi * per;
  uint32_t* bm = reinterpret_cast<uint32_t*>(base);
  float* acc = reinterpret_cast<float*>(base + align16(((size_t)W + 31) / 32 * 4));
  Chunk<GROUP>& ch = *reinterpret_cast<Chunk<GROUP>*>(
      base + align16(((size_t)W + 31) / 32 * 4) + (NUM ? align16((size_t)W * 4) : 0));
  Group<GROUP, BLOCK> g;
  g.red = reinterpret_cast<int64_t*>(reinterpret_cast<unsigned char*>(&ch) + align16(sizeof(Chunk<GROUP>)));
  const int t = g.t();
  const int nwd_full = (W + 31) / 32;
  for (int i = t; i < nwd_full; i += GROUP) bm[i] = 0u;
  if constexpr (NUM)
    for (int i = t; i < W; i += GROUP) acc[i] = 0.f;
  g.sync();

  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.bin + 1] - bv.binoff[bv.bin];
  const int64_t nwin = WIDE ? op.nwin : 1;
  const int64_t nitems = cnt * nwin;
  for (int64_t it = (int64_t)blockIdx.x * NG + gi; it < nitems; it += (int64_t)gridDim.x * NG) {
    const int64_t w = it / cnt;          // window-major: one B column slab at a time
    const int64_t row = list[it - w * cnt];
    const int64_t c0 = w * W;
    const int Wn = (int)((op.N - c0) < W ? (op.N - c0) : W);

    for_each_term<RA, RB, GROUP, BLOCK, NUM, WIDE>(op, g, ch, row, w, [&](int64_t pos, float a) {
      const int j = op.bcol[pos] - (int)c0;
      atomicOr(&bm[j >> 5], 1u << (j & 31));
      if constexpr (NUM) atomicAdd(&acc[j], a * op.bval[pos]);
    });

    const int nwd = (Wn + 31) / 32;
    if constexpr (!NUM) {
      int64_t c = 0;
      for (int i = t; i < nwd; i += GROUP) {
        c += __popc(bm[i]);
        bm[i] = 0u;
      }
      c = g.sum(c);
      if (t == 0) {
        if constexpr (WIDE) out.wcnt[row * nwin + w] = (int32_t)c;
        else out.counts[row] = c;
      }
    } else {
      int64_t o0 = out.crp[row];
      if constexpr (WIDE) o0 += out.wcnt[row * nwin + w];
      for (int i0 = 0; i0 < nwd; i0 += GROUP) {
        const int i = i0 + t;
        uint32_t bits = (i < nwd) ? bm[i] : 0u;
        int64_t tot;
        const int64_t c = __popc(bits);
        int64_t o = o0 + g.incl_scan(c, &tot) - c;
        while (bits) {
          const int b = __ffs(bits) - 1;
          bits &= bits - 1;
          const int j = i * 32 + b;
          out.ccol[o] = j + (int)c0;
          out.cval[o] = acc[j];
          acc[j] = 0.f;
          ++o;
        }
        if (i < nwd) bm[i] = 0u;
        o0 += tot;
      }
    }
    g.sync();
  }
}

// -------------------------------------------------------------- hash path

template <int TABLE, int GROUP>
struct HashLds {
  int32_t key[TABLE];
  float val[TABLE];
  Chunk<GROUP> ch;
  int64_t red[GROUP / WAVE + 1];
};

template <int TABLE>
__device__ __forceinline__ uint32_t hslot(int j) {
  constexpr int LOG2 = __builtin_ctz(TABLE);
  return ((uint32_t)j * 2654435761u) >> (32 - LOG2);
}

template <typename RA, typename RB, int TABLE, int GROUP, int BLOCK, bool NUM>
__global__ __launch_bounds__(BLOCK) void k_hash(const Operands op, const BinView bv,
                                                const Outputs out) {
  constexpr int NG = BLOCK / GROUP;
  constexpr int SPT = TABLE / GROUP;   // table slots per thread
  static_assert(TABLE % GROUP == 0, "table divides over the group");
  __shared__ HashLds<TABLE, GROUP> lds[NG];
  const int gi = threadIdx.x / GROUP;
  HashLds<TABLE, GROUP>& L = lds[gi];
  Group<GROUP, BLOCK> g;
  g.red = L.red;
  const int t = g.t();
  for (int i = t; i < TABLE; i += GROUP) {
    L.key[i] = -1;
    if constexpr (NUM) L.val[i] = 0.f;
  }
  g.sync();

  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.bin + 1] - bv.binoff[bv.bin];
  for (int64_t it = (int64_t)blockIdx.x * NG + gi; it < cnt; it += (int64_t)gridDim.x * NG) {
    const int64_t row = list[it];
    int64_t mine = 0;
    for_each_term<RA, RB, GROUP, BLOCK, NUM, false>(op, g, L.ch, row, 0, [&](int64_t pos, float a) {
      const int j = op.bcol[pos];
      uint32_t h = hslot<TABLE>(j);
      for (;;) {
        const int old = atomicCAS(&L.key[h], -1, j);
        if (old == -1 || old == j) {
          if constexpr (NUM) atomicAdd(&L.val[h], a * op.bval[pos]);
          else mine += (old == -1);
          break;
        }
        h = (h + 1) & (TABLE - 1);
      }
    });

    if constexpr (!NUM) {
      const int64_t c = g.sum(mine);
      if (t == 0) out.counts[row] = c;
      for (int i = t; i < TABLE; i += GROUP) L.key[i] = -1;
      g.sync();
    } else {
      // compact the occupied slots to the front of the table
      int32_t kk[SPT];
      float vv[SPT];
      int64_t c = 0;
#pragma unroll
      for (int s = 0; s < SPT; ++s) {
        kk[s] = L.key[s * GROUP + t];
        vv[s] = L.val[s * GROUP + t];
        c += (kk[s] != -1);
      }
      int64_t n;
      int64_t o = g.incl_scan(c, &n) - c;
      g.sync();
#pragma unroll
      for (int s = 0; s < SPT; ++s)
        if (kk[s] != -1) { L.key[o] = kk[s]; L.val[o] = vv[s]; ++o; }
      int n2 = 1;
      while (n2 < n) n2 <<= 1;
      for (int i = (int)n + t; i < n2; i += GROUP) L.key[i] = 0x7fffffff;
      g.sync();
      // bitonic sort of (key, val) pairs in [0, n2)
      for (int k = 2; k <= n2; k <<= 1) {
        for (int jj = k >> 1; jj > 0; jj >>= 1) {
          for (int pi = t; pi < (n2 >> 1); pi += GROUP) {
            const int i = ((pi & ~(jj - 1)) << 1) | (pi & (jj - 1));
            const int l = i | jj;
            const bool asc = (i & k) == 0;
            const int ki = L.key[i], kl = L.key[l];
            if ((ki > kl) == asc) {
              const float vi = L.val[i], vl = L.val[l];
              L.key[i] = kl; L.key[l] = ki;
              L.val[i] = vl; L.val[l] = vi;
            }
          }
          g.sync();
        }
      }
      const int64_t o0 = out.crp[row];
      for (int i = t; i < n; i += GROUP) {
        out.ccol[o0 + i] = L.key[i];
        out.cval[o0 + i] = L.val[i];
      }
      g.sync();
      for (int i = t; i < TABLE; i += GROUP) {
        L.key[i] = -1;
        L.val[i] = 0.f;
      }
      g.sync();
    }
  }
}

// ------------------------------------------------------- windowed row sums

// For each row of a windowed bin: exclusive scan of its window counts in
// place (they become offsets inside the row) and the row total.
__global__ __launch_bounds__(256) void k_window_rowsum(const BinView bv, int32_t nwin,
                                                       int32_t* wcnt, int64_t* counts) {
  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.bin + 1] - bv.binoff[bv.bin];
  for (int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; d < cnt;
       d += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = list[d];
    int32_t* c = wcnt + row * nwin;
    int64_t s = 0;
    for (int w = 0; w < nwin; ++w) {
      const int32_t v = c[w];
      c[w] = (int32_t)s;
      s += v;
    }
    counts[row] = s;
  }
}

// ------------------------------------------------------------ window index

// bidx[w*K + k] = first position p of B_k with bcol[p] >= w*W (or the row
// end), for w in [0, nwin].  One wavefront per B row.
template <typename RB>
__global__ __launch_bounds__(256) void k_window_index(const void* brp, const int32_t* bcol,
                                                      int64_t K, int32_t W, int32_t nwin,
                                                      int32_t* bidx) {
  const int64_t nw = (int64_t)gridDim.x * (blockDim.x / WAVE);
  for (int64_t k = (int64_t)blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE; k < K; k += nw) {
    const int64_t s = ld_rp<RB>(brp, k), e = ld_rp<RB>(brp, k + 1);
    for (int64_t p = s + lane_id(); p < e; p += WAVE) {
      const int wc = bcol[p] / W;
      const int wp = (p == s) ? -1 : bcol[p - 1] / W;
      for (int w = wp + 1; w <= wc; ++w) bidx[(int64_t)w * K + k] = (int32_t)p;
    }
    if (lane_id() == 0) {
      const int wl = (e > s) ? bcol[e - 1] / W : -1;
      for (int w = wl + 1; w <= nwin; ++w) bidx[(int64_t)w * K + k] = (int32_t)e;
    }
  }
}

// -------------------------------------------------------------------- scan

constexpr int SCAN_BLOCK = 1024;
constexpr int SCAN_ITEMS = 4;
constexpr int64_t SCAN_CHUNK = (int64_t)SCAN_BLOCK * SCAN_ITEMS;

__device__ __forceinline__ int64_t block_incl_scan_1024(int64_t v, int64_t* red, int64_t* total) {
  const int w = threadIdx.x / WAVE;
  int64_t x = wave_incl_scan(v);
  if (lane_id() == WAVE - 1) red[w] = x;
  __syncthreads();
  if (w == 0) {
    int64_t r = (lane_id() < SCAN_BLOCK / WAVE) ? red[lane_id()] : 0;
    r = wave_incl_scan(r);
    if (lane_id() < SCAN_BLOCK / WAVE) red[lane_id()] = r;
  }
  __syncthreads();
  const int64_t pre = (w > 0) ? red[w - 1] : 0;
  *total = red[SCAN_BLOCK / WAVE - 1];
  __syncthreads();
  return x + pre;
}

__global__ __launch_bounds__(SCAN_BLOCK) void k_scan_reduce(const int64_t* x, int64_t n, int64_t* bsum) {
  __shared__ int64_t red[SCAN_BLOCK / WAVE];
  const int64_t b0 = (int64_t)blockIdx.x * SCAN_CHUNK;
  int64_t s = 0;
#pragma unroll
  for (int r = 0; r < SCAN_ITEMS; ++r) {
    const int64_t i = b0 + (int64_t)r * SCAN_BLOCK + threadIdx.x;
    if (i < n) s += x[i];
  }
  int64_t tot;
  block_incl_scan_1024(s, red, &tot);
  if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// Exclusive scan of the block sums plus the base x[-1], in one block.
__global__ __launch_bounds__(SCAN_BLOCK) void k_scan_bsums(const int64_t* x, int64_t* bsum, int64_t nb) {
  __shared__ int64_t red[SCAN_BLOCK / WAVE];
  int64_t carry = x[-1];
  for (int64_t b0 = 0; b0 < nb; b0 += SCAN_BLOCK) {
    const int64_t i = b0 + threadIdx.x;
    const int64_t v = (i < nb) ? bsum[i] : 0;
    int64_t tot;
    const int64_t incl = block_incl_scan_1024(v, red, &tot);
    if (i < nb) bsum[i] = carry + incl - v;
    carry += tot;
  }
}

__global__ __launch_bounds__(SCAN_BLOCK) void k_scan_apply(int64_t* x, int64_t n, const int64_t* bsum) {
  __shared__ int64_t red[SCAN_BLOCK / WAVE];
  const int64_t b0 = (int64_t)blockIdx.x * SCAN_CHUNK + (int64_t)threadIdx.x * SCAN_ITEMS;
  int64_t v[SCAN_ITEMS];
  int64_t s = 0;
#pragma unroll
  for (int r = 0; r < SCAN_ITEMS; ++r) {
    const int64_t i = b0 + r;
    v[r] = (i < n) ? x[i] : 0;
    s += v[r];
  }
  int64_t tot;
  int64_t run = block_incl_scan_1024(s, red, &tot) - s + bsum[blockIdx.x];
#pragma unroll
  for (int r = 0; r < SCAN_ITEMS; ++r) {
    const int64_t i = b0 + r;
    run += v[r];
    if (i < n) x[i] = run;
  }
}

// ------------------------------------------------------------- occupancy

int g_num_cus = 0;

int num_cus() {
  if (g_num_cus == 0) {
    int dev = 0;
    (void)hipGetDevice(&dev);
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    g_num_cus = n;
  }
  return g_num_cus;
}

template <typename K>
int64_t grid_for(K kernel, int block, size_t lds, int64_t items_per_block, int64_t ub_items) {
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, block, lds) != hipSuccess || per_cu <= 0)
    per_cu = 1;
  int64_t cap = (int64_t)per_cu * num_cus();
  int64_t need = (ub_items + items_per_block - 1) / items_per_block;
  if (need < 1) need = 1;
  return need < cap ? need : cap;
}

template <typename RA, typename RB, int GROUP, int BLOCK, bool NUM, bool WIDE>
hipError_t launch_dense(const Operands& op, const BinView& bv, const Outputs& out, int64_t ub_rows,
                        hipStream_t s) {
  auto kern = k_dense<RA, RB, GROUP, BLOCK, NUM, WIDE>;
  const int W = WIDE ? op.W : (int)op.N;
  const size_t lds = (BLOCK / GROUP) * dense_group_bytes<GROUP, NUM>(W);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t ub = ub_rows * (WIDE ? op.nwin : 1);
  const int64_t grid = grid_for(kern, BLOCK, lds, BLOCK / GROUP, ub);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(BLOCK), lds, s, op, bv, out);
  return hipGetLastError();
}

template <typename RA, typename RB, int TABLE, int GROUP, int BLOCK, bool NUM>
hipError_t launch_hash(const Operands& op, const BinView& bv, const Outputs& out, int64_t ub_rows,
                       hipStream_t s) {
  auto kern = k_hash<RA, RB, TABLE, GROUP, BLOCK, NUM>;
  const int64_t grid = grid_for(kern, BLOCK, 0, BLOCK / GROUP, ub_rows);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(BLOCK), 0, s, op, bv, out);
  return hipGetLastError();
}

template <typename RA, typename RB, bool NUM>
hipError_t run_bin_t(int kind, const Operands& op, const BinView& bv, const Outputs& out,
                     int64_t ub_rows, hipStream_t s) {
  switch (kind) {
    case KIND_DENSE_WAVE:
      return launch_dense<RA, RB, 64, 256, NUM, false>(op, bv, out, ub_rows, s);
    case KIND_DENSE_BLOCK:
      if (op.bidx) return launch_dense<RA, RB, 512, 512, NUM, true>(op, bv, out, ub_rows, s);
      return launch_dense<RA, RB, 512, 512, NUM, false>(op, bv, out, ub_rows, s);
    case KIND_HASH_128:
      return launch_hash<RA, RB, 128, 64, 256, NUM>(op, bv, out, ub_rows, s);
    case KIND_HASH_1024:
      return launch_hash<RA, RB, 1024, 64, 256, NUM>(op, bv, out, ub_rows, s);
    case KIND_HASH_8192:
      return launch_hash<RA, RB, 8192, 256, 256, NUM>(op, bv, out, ub_rows, s);
    default:
      return hipErrorInvalidValue;
  }
}

template <typename RA, typename RB>
hipError_t run_bin_rp(int kind, int phase, const Operands& op, const BinView& bv, const Outputs& out,
                      int64_t ub_rows, hipStream_t s) {
  return phase ? run_bin_t<RA, RB, true>(kind, op, bv, out, ub_rows, s)
               : run_bin_t<RA, RB, false>(kind, op, bv, out, ub_rows, s);
}

}  // namespace

// ------------------------------------------------------------- host entry

hipError_t analyze(const Operands& op, int64_t nrows, int64_t* P, unsigned long long* total,
                   hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  const int64_t grid = (nrows * 16 + 255) / 256;
  if (op.rpa64) {
    if (op.rpb64) hipLaunchKernelGGL((k_analyze<int64_t, int64_t>), dim3((unsigned)grid), dim3(256), 0, s, op, nrows, P, total);
    else hipLaunchKernelGGL((k_analyze<int64_t, int32_t>), dim3((unsigned)grid), dim3(256), 0, s, op, nrows, P, total);
  } else {
    if (op.rpb64) hipLaunchKernelGGL((k_analyze<int32_t, int64_t>), dim3((unsigned)grid), dim3(256), 0, s, op, nrows, P, total);
    else hipLaunchKernelGGL((k_analyze<int32_t, int32_t>), dim3((unsigned)grid), dim3(256), 0, s, op, nrows, P, total);
  }
  return hipGetLastError();
}

hipError_t bin_rows(const int64_t* P, int64_t nrows, const BinThresholds& th, int32_t* cnt_cursor,
                    int32_t* binoff, int32_t* list, hipStream_t s) {
  const int64_t grid = nrows > 0 ? (nrows + 255) / 256 : 1;
  hipLaunchKernelGGL(k_bin_count, dim3((unsigned)grid), dim3(256), 0, s, P, nrows, th, cnt_cursor);
  hipLaunchKernelGGL(k_bin_scatter, dim3((unsigned)grid), dim3(256), 0, s, P, nrows, th, cnt_cursor,
                     cnt_cursor + MAX_BINS, binoff, list);
  return hipGetLastError();
}

hipError_t run_bin(int kind, int phase, const Operands& op, const BinView& bv, const Outputs& out,
                   int64_t ub_rows, hipStream_t s) {
  if (ub_rows <= 0) return hipSuccess;
  if (op.rpa64) {
    return op.rpb64 ? run_bin_rp<int64_t, int64_t>(kind, phase, op, bv, out, ub_rows, s)
                    : run_bin_rp<int64_t, int32_t>(kind, phase, op, bv, out, ub_rows, s);
  }
  return op.rpb64 ? run_bin_rp<int32_t, int64_t>(kind, phase, op, bv, out, ub_rows, s)
                  : run_bin_rp<int32_t, int32_t>(kind, phase, op, bv, out, ub_rows, s);
}

hipError_t window_rowsum(const BinView& bv, int32_t nwin, int32_t* wcnt, int64_t* counts,
                         int64_t ub_rows, hipStream_t s) {
  if (ub_rows <= 0) return hipSuccess;
  int64_t grid = (ub_rows + 255) / 256;
  if (grid > 4096) grid = 4096;
  hipLaunchKernelGGL(k_window_rowsum, dim3((unsigned)grid), dim3(256), 0, s, bv, nwin, wcnt, counts);
  return hipGetLastError();
}

hipError_t build_window_index(const void* brp, int rpb64, const int32_t* bcol, int64_t K, int32_t W,
                              int32_t nwin, int32_t* bidx, hipStream_t s) {
  if (K <= 0) return hipSuccess;
  int64_t grid = (K + 3) / 4;
  if (grid > 65536) grid = 65536;
  if (rpb64)
    hipLaunchKernelGGL((k_window_index<int64_t>), dim3((unsigned)grid), dim3(256), 0, s, brp, bcol, K, W, nwin, bidx);
  else
    hipLaunchKernelGGL((k_window_index<int32_t>), dim3((unsigned)grid), dim3(256), 0, s, brp, bcol, K, W, nwin, bidx);
  return hipGetLastError();
}

size_t scan_workspace_bytes(int64_t n) {
  const int64_t nb = (n + SCAN_CHUNK - 1) / SCAN_CHUNK;
  return (size_t)(nb > 0 ? nb : 1) * sizeof(int64_t);
}

hipError_t scan_inplace(int64_t* x, int64_t n, void* ws, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = (n + SCAN_CHUNK - 1) / SCAN_CHUNK;
  int64_t* bsum = static_cast<int64_t*>(ws);
  hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)nb), dim3(SCAN_BLOCK), 0, s, x, n, bsum);
  hipLaunchKernelGGL(k_scan_bsums, dim3(1), dim3(SCAN_BLOCK), 0, s, x, bsum, nb);
  hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)nb), dim3(SCAN_BLOCK), 0, s, x, n, bsum);
  return hipGetLastError();
}

size_t lds_bytes(int kind, int phase, int32_t W) {
  switch (kind) {
    case KIND_DENSE_WAVE:
      return 4 * (phase ? dense_group_bytes<64, true>(W) : dense_group_bytes<64, false>(W));
    case KIND_DENSE_BLOCK:
      return phase ? dense_group_bytes<512, true>(W) : dense_group_bytes<512, false>(W);
    case KIND_HASH_128: return 4 * sizeof(HashLds<128, 64>);
    case KIND_HASH_1024: return 4 * sizeof(HashLds<1024, 64>);
    case KIND_HASH_8192: return sizeof(HashLds<8192, 256>);
    default: return 0;
  }
}

int group_size(int kind) {
  switch (kind) {
    case KIND_DENSE_BLOCK: return 512;
    case KIND_HASH_8192: return 256;
    default: return 64;
  }
}

}  // namespace kern
}  // namespace aires
