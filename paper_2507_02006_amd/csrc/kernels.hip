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
//   dense row     fp32 slots for all N columns of a narrow product plus a
//                 presence bitmap; compaction by ballot walks the columns in
//                 order, so the output comes out sorted with no sort at all
//                 (heavy rows: runs of A entries per workgroup, merged in a
//                 dense slot in global memory).
//   hash          open addressing (linear probing) keyed by column; the
//                 occupied slots are compacted and sorted (runs of 16 in
//                 registers, then merge-path rounds in LDS).
//   column window presence bitmap of a window of whole column grains, word
//                 ranks from its popcounts, and a compact fp32 array indexed
//                 by rank (wide products).
// A product's intermediate terms are spread over the threads of a group by
// a flattened loop: the group loads up to GROUP entries (k, a_ik) of A_i and
// scans the lengths of the matching B segments; each wavefront takes an
// equal contiguous share of the terms and maps each term to its segment with
// a segment map of its own.  Consecutive lanes read consecutive entries of a
// B row.
#include "kernels.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

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

// Cross-lane moves by DPP (data-parallel primitives of the GFX9 vector
// ALU, no LDS traffic): row_shr:n = 0x110 + n shifts within rows of 16
// lanes, row_bcast:15 = 0x142 and row_bcast:31 = 0x143 pass the last lane
// of a row (of two rows) on to the rows that ROW_MASK enables, wave_shr:1 =
// 0x138 shifts across the wavefront.  Lanes without a source read 0.
template <int CTRL, int ROW_MASK, typename T>
__device__ __forceinline__ T dpp_move(T x) {
  static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit lanes");
  if constexpr (sizeof(T) == 4) {
    return (T)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROW_MASK, 0xf, false);
  } else {
    const uint64_t u = (uint64_t)x;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, ROW_MASK, 0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, ROW_MASK, 0xf, false);
    return (T)(((uint64_t)hi << 32) | lo);
  }
}

// Inclusive wavefront scan: Hillis-Steele steps 1, 2, 4, 8 inside rows of
// 16 lanes, then the row totals are carried to rows 1 and 3 and to rows 2
// and 3.  OP is + (SUM) or max (for non-negative values).
template <bool SUM, typename T>
__device__ __forceinline__ T wave_scan_op(T v) {
  auto op = [](T a, T b) { return SUM ? a + b : (a > b ? a : b); };
  v = op(v, dpp_move<0x111, 0xf>(v));
  v = op(v, dpp_move<0x112, 0xf>(v));
  v = op(v, dpp_move<0x114, 0xf>(v));
  v = op(v, dpp_move<0x118, 0xf>(v));
  v = op(v, dpp_move<0x142, 0xa>(v));
  v = op(v, dpp_move<0x143, 0xc>(v));
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  return wave_scan_op<true>(v);
}

// The value of lane 63 in every lane.
template <typename T>
__device__ __forceinline__ T wave_last(T x) {
  if constexpr (sizeof(T) == 4) {
    return (T)__builtin_amdgcn_readlane((int)x, WAVE - 1);
  } else {
    const uint64_t u = (uint64_t)x;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, WAVE - 1);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), WAVE - 1);
    return (T)(((uint64_t)hi << 32) | lo);
  }
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
  return wave_last(wave_incl_scan(v));
}

// fp32 sum over the wavefront, in every lane (butterfly over lane pairs).
__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
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
      *total = wave_last(x);
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
  // the same for 32-bit values whose group sum fits 32 bits
  __device__ __forceinline__ int32_t incl_scan32(int32_t v, int32_t* total) const {
    int32_t x = wave_incl_scan(v);
    if constexpr (GROUP == WAVE) {
      *total = wave_last(x);
      return x;
    } else {
      const int w = threadIdx.x / WAVE;
      if (lane_id() == WAVE - 1) red[w] = x;
      __syncthreads();
      int32_t pre = 0, tot = 0;
#pragma unroll
      for (int i = 0; i < NWAVES; ++i) {
        const int32_t s = (int32_t)red[i];
        pre += (i < w) ? s : 0;
        tot += s;
      }
      __syncthreads();
      *total = tot;
      return x + pre;
    }
  }
};

// C is written once and not read back by the kernels: stream it past the
// caches so that B's rows stay resident there.
template <typename T>
__device__ __forceinline__ void store_stream(T* p, T v) {
  __builtin_nontemporal_store(v, p);
}

template <typename RP>
__device__ __forceinline__ int64_t ld_rp(const void* rp, int64_t i) {
  return (int64_t)static_cast<const RP*>(rp)[i];
}

// ---------------------------------------------------------------- analyze

constexpr int64_t kLongRow = 2048;  // longer A rows are summed by a whole workgroup

// P_i for every tile row, 16 lanes per row, rows taken grid-stride; rows
// longer than kLongRow are appended to long_list for k_analyze_long.  The
// total is added once per workgroup.
template <typename RA, typename RB>
__global__ __launch_bounds__(256) void k_analyze(const Operands op, int64_t nrows, int64_t* P,
                                                 unsigned long long* total, int32_t* long_cnt,
                                                 int32_t* long_list) {
  __shared__ int64_t red[256 / WAVE];
  const int sub = threadIdx.x & 15;
  const int64_t nsub = (int64_t)gridDim.x * (blockDim.x / 16);
  int64_t mine = 0;
  for (int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4; row < nrows; row += nsub) {
    int64_t s = 0;
    const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
    const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
    const bool is_long = p1 - p0 > kLongRow;  // uniform over the 16 lanes of the row
    if (is_long) {
      if (sub == 0) long_list[atomicAdd(long_cnt, 1)] = (int32_t)row;
    } else {
      for (int64_t p = p0 + sub; p < p1; p += 64) {
        int64_t k[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) k[u] = (p + 16 * u < p1) ? (int64_t)op.acol[p + 16 * u] : -1;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (k[u] >= 0) s += ld_rp<RB>(op.brp, k[u] + 1) - ld_rp<RB>(op.brp, k[u]);
      }
    }
#pragma unroll
    for (int d = 8; d > 0; d >>= 1) s += __shfl_xor(s, d, 16);
    if (sub == 0 && !is_long) {
      P[row] = s;
      mine += s;
    }
  }
  mine = wave_sum(mine);
  if (lane_id() == 0) red[threadIdx.x / WAVE] = mine;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t t = 0;
    for (int i = 0; i < 256 / WAVE; ++i) t += red[i];
    if (t) atomicAdd(total, (unsigned long long)t);
  }
}

template <typename RA, typename RB>
__global__ __launch_bounds__(1024) void k_analyze_long(const Operands op, int64_t* P,
                                                       unsigned long long* total,
                                                       const int32_t* long_cnt,
                                                       const int32_t* long_list) {
  __shared__ int64_t red[1024 / WAVE];
  const int n = *long_cnt;
  for (int it = blockIdx.x; it < n; it += gridDim.x) {
    const int64_t row = long_list[it];
    const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
    const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
    int64_t s = 0;
    for (int64_t p = p0 + threadIdx.x; p < p1; p += 4 * 1024) {
      int64_t k[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) k[u] = (p + 1024 * u < p1) ? (int64_t)op.acol[p + 1024 * u] : -1;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (k[u] >= 0) s += ld_rp<RB>(op.brp, k[u] + 1) - ld_rp<RB>(op.brp, k[u]);
    }
    s = wave_sum(s);
    if (lane_id() == 0) red[threadIdx.x / WAVE] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
      int64_t t = 0;
      for (int i = 0; i < 1024 / WAVE; ++i) t += red[i];
      P[row] = t;
      if (t) atomicAdd(total, (unsigned long long)t);
    }
    __syncthreads();
  }
}

// ----------------------------------------------------------------- binning

__device__ __forceinline__ int bin_of(const BinThresholds& th, int64_t p) {
  int b = 0;
  while (b < th.nb - 1 && p > th.max_p[b]) ++b;
  return b;
}

// Bins are counted and filled per workgroup over a contiguous range of
// rows, with one global atomic per bin and workgroup.
__device__ __forceinline__ void block_rows(int64_t nrows, int64_t& r0, int64_t& r1) {
  const int64_t per = (nrows + gridDim.x - 1) / gridDim.x;
  r0 = min(nrows, (int64_t)blockIdx.x * per);
  r1 = min(nrows, r0 + per);
}

__global__ __launch_bounds__(256) void k_bin_count(const int64_t* P, int64_t nrows,
                                                   const BinThresholds th, int32_t* cnt) {
  __shared__ int32_t h[MAX_BINS];
  if (threadIdx.x < MAX_BINS) h[threadIdx.x] = 0;
  __syncthreads();
  int64_t r0, r1;
  block_rows(nrows, r0, r1);
  for (int64_t i = r0 + threadIdx.x; i < r1; i += blockDim.x) atomicAdd(&h[bin_of(th, P[i])], 1);
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
  int64_t r0, r1;
  block_rows(nrows, r0, r1);
  for (int64_t i = r0 + threadIdx.x; i < r1; i += blockDim.x) atomicAdd(&h[bin_of(th, P[i])], 1);
  __syncthreads();
  if (threadIdx.x < th.nb) {
    base[threadIdx.x] = h[threadIdx.x] ? atomicAdd(&cursor[threadIdx.x], h[threadIdx.x]) : 0;
    h[threadIdx.x] = 0;
  }
  __syncthreads();
  for (int64_t i = r0 + threadIdx.x; i < r1; i += blockDim.x) {
    const int b = bin_of(th, P[i]);
    list[off[b] + base[b] + atomicAdd(&h[b], 1)] = (int32_t)i;
  }
}

// ---------------------------------------------------- flattened product loop

// Per-group LDS for one chunk of A_i: the B position of term 0 of each
// segment (shifted so pos = shift[c] + q), a_ik, the first term of each
// segment, and per wavefront a segment map of SEG_PER_THREAD * WAVE
// consecutive terms.  A chunk holds fewer than 2^31 terms: segments are at
// most one window or one B row wide and a chunk has at most GROUP of them.
#ifndef AIRES_SEG_PER_THREAD
#define AIRES_SEG_PER_THREAD 8
#endif
constexpr int SEG_PER_THREAD = AIRES_SEG_PER_THREAD;
static_assert(SEG_PER_THREAD % 8 == 0, "segment maps move in 16-byte vectors");

// fp32 add into an LDS slot, returning the slot's previous value.  It is a
// compare-and-swap loop on the slot's bits: on gfx950 the LDS float-add
// atomic issues at roughly a seventh of the rate of the LDS integer atomics
// and compare-swap, and a lane retries only when another lane changed the
// slot between its read and its swap (at least one lane per slot succeeds
// on every round, so the loop ends).  GUESS_EMPTY: the first swap assumes
// the slot still holds +0 instead of reading it first, which saves the read
// where most adds are a slot's first.
template <bool GUESS_EMPTY>
__device__ __forceinline__ float lds_add(float* p, float v) {
  uint32_t* q = reinterpret_cast<uint32_t*>(p);
  uint32_t old = GUESS_EMPTY ? 0u : __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  for (;;) {
    const uint32_t prev = atomicCAS(q, old, __float_as_uint(__uint_as_float(old) + v));
    if (prev == old) return __uint_as_float(old);
    old = prev;
  }
}

template <int GROUP, typename S>
struct Chunk {
  using shift_t = S;  // B positions fit B's row-pointer type
  struct Rec {
    S shift;
    float av;
  };
  Rec rec[GROUP];
  int32_t ex[GROUP + 4];  // GROUP + 1 used; the padding keeps seg 16-byte aligned
  alignas(16) uint16_t seg[GROUP * SEG_PER_THREAD];
};

// Where the terms of a k come from: the whole B row ...
template <typename RB>
struct FullRows {
  const void* brp;
  __device__ __forceinline__ void operator()(int64_t k, int64_t& lo, int64_t& len) const {
    lo = ld_rp<RB>(brp, k);
    len = ld_rp<RB>(brp, k + 1) - lo;
  }
};
// ... or a range each thread already holds for its own k (one chunk) ...
struct HeldRange {
  int64_t lo, len;
  __device__ __forceinline__ void operator()(int64_t, int64_t& l, int64_t& n) const {
    l = lo;
    n = len;
  }
};
// ... or the part of it in a run of column grains (two slabs of the index).
struct GrainRange {
  const int32_t* bidx;  // the grain index, nG + 1 entries per B row
  int32_t stride, g0, g1;
  __device__ __forceinline__ void operator()(int64_t k, int64_t& lo, int64_t& len) const {
    const int32_t* r = bidx + k * stride;
    lo = r[g0];
    len = (int64_t)r[g1] - lo;
  }
};

#ifndef AIRES_UNROLL
#define AIRES_UNROLL 4
#endif
constexpr int UNROLL = AIRES_UNROLL;  // independent B loads each thread keeps in flight

// Segment map of one wavefront's terms [lo, lo + len), len <= WAVE *
// SEG_PER_THREAD: seg_w[x] = the segment holding term lo + x, from the
// first terms ex[c] of segments c < nk (non-decreasing, ex[0] = 0,
// lo < ex[nk]).  The segment holding lo is found with two ballots; each
// later segment starting in the range writes its id at its first term and
// a wavefront max-scan carries ids forward.  No workgroup barrier.
// Returns that segment when it holds the whole range (no map is written:
// long B segments make this common), else -1.
__device__ __forceinline__ int wave_seg_map(const int32_t* ex, int nk, int lo, int len, uint16_t* seg_w) {
  const int l = lane_id();
  wave_sync();  // the previous run's reads of seg_w are done
  const int stride = (nk + WAVE - 1) / WAVE;
  const int cs = l * stride;
  const uint64_t b1 = __ballot(cs < nk && ex[cs] <= lo);
  const int base = (63 - __clzll(b1)) * stride;
  const int c2 = base + l;
  const uint64_t b2 = __ballot(l < stride && c2 < nk && ex[c2] <= lo);
  const int c0 = base + (63 - __clzll(b2));
  if (ex[c0 + 1] >= lo + len) return c0;  // the whole range lies in segment c0: no map
  // each lane's SEG_PER_THREAD entries are moved as 16-byte vectors
  uint4* mine = reinterpret_cast<uint4*>(seg_w + l * SEG_PER_THREAD);
#pragma unroll
  for (int v = 0; v < SEG_PER_THREAD / 8; ++v) mine[v] = make_uint4(0u, 0u, 0u, 0u);
  wave_sync();
  const int hi = lo + len;
  for (int c = c0 + 1 + l; c < nk; c += WAVE) {
    const int e = ex[c];
    if (e >= hi) break;
    if (ex[c + 1] > e) seg_w[e - lo] = (uint16_t)c;
  }
  wave_sync();
  int run[SEG_PER_THREAD];
  int m = c0;
#pragma unroll
  for (int v = 0; v < SEG_PER_THREAD / 8; ++v) {
    const uint4 q = mine[v];
    const uint32_t wv[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      m = max(m, (int)((wv[h >> 1] >> ((h & 1) * 16)) & 0xffffu));
      run[v * 8 + h] = m;
    }
  }
  const int x = wave_scan_op<false>(m);  // segment ids are >= 0
  int before = dpp_move<0x138, 0xf>(x);  // the previous lane's
  if (l == 0) before = c0;
#pragma unroll
  for (int v = 0; v < SEG_PER_THREAD / 8; ++v) {
    uint32_t wv[4];
#pragma unroll
    for (int h = 0; h < 4; ++h)
      wv[h] = (uint32_t)max(before, run[v * 8 + 2 * h]) | ((uint32_t)max(before, run[v * 8 + 2 * h + 1]) << 16);
    mine[v] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
  }
  wave_sync();
  return -1;
}

// Terms of a run of rn each of nw wavefronts takes: an equal share rounded
// up to whole wavefront loads (at most WAVE * SEG_PER_THREAD).
__device__ __forceinline__ int wave_share(int rn, int nw) {
  return ((rn + nw - 1) / nw + WAVE - 1) / WAVE * WAVE;
}

// Calls f(column, a_ik * b_kj) (NUM) or f(column, 0) for every term of A
// entries [p0, p1) (a row or a part of one).  Terms are numbered over the
// chunk's segments; a run of up to GROUP * SEG_PER_THREAD terms is split
// into equal contiguous parts, one per wavefront, whose lane l takes terms
// l, l + WAVE, ..., so consecutive lanes read consecutive entries of a B row.
// P32: B positions fit 32 bits (wide products, nnz(B) < 2^31).
// SMALL_SCAN: a chunk of at most WAVE entries is scanned by the first
// wavefront alone (two workgroup barriers less).
// BATCH: f(j[UR], v[UR], ok[UR]) takes a lane's UR terms at once, with no
// branch per term: a term past the wavefront's share (ok false) repeats the
// lane's first term of the step, so that every read stays in range.
template <int GROUP, int BLOCK, bool NUM, bool P32 = false, int UR = UNROLL, bool SMALL_SCAN = false,
          bool BATCH = false, typename CH, typename SEG, typename F>
__device__ __forceinline__ void for_each_term_in(const Operands& op, const Group<GROUP, BLOCK>& g,
                                                 CH& ch, int64_t p0, int64_t p1, const SEG& seg, F&& f) {
  using S = typename CH::shift_t;
  using PI = std::conditional_t<P32, int32_t, int64_t>;
  constexpr int RUN = GROUP * SEG_PER_THREAD;
  constexpr int WR = WAVE * SEG_PER_THREAD;  // terms of one wavefront per run
  const int t = g.t();
  const int lane = lane_id();
  const int w = t / WAVE;
  uint16_t* seg_w = ch.seg + w * WR;
  for (int64_t cb = p0; cb < p1; cb += GROUP) {
    const int64_t p = cb + t;
    int64_t lo = 0, len = 0;
    float av = 0.f;
    if (p < p1) {
      const int64_t k = op.acol[p];
      if constexpr (NUM) av = op.aval[p];
      seg(k, lo, len);
    }
    int32_t total;  // a chunk holds fewer than 2^31 terms
    const int nk = (int)((p1 - cb) < GROUP ? (p1 - cb) : GROUP);
    if (SMALL_SCAN && GROUP > WAVE && nk <= WAVE) {
      // every A entry of the chunk sits in the first wavefront: its scan
      // alone gives the segment starts (entries past nk are never read; the
      // lanes from nk on write ex[nk] = total)
      if (t < WAVE) {
        const int32_t incl = wave_incl_scan((int32_t)len);
        const int32_t excl = incl - (int32_t)len;
        ch.rec[t].shift = (S)(lo - excl);
        ch.rec[t].av = av;
        ch.ex[t] = excl;
        if (t == WAVE - 1) {
          ch.ex[WAVE] = incl;
          ch.ex[GROUP] = incl;
        }
      }
      g.sync();
      total = ch.ex[GROUP];
    } else {
      const int32_t incl = g.incl_scan32((int32_t)len, &total);
      const int32_t excl = incl - (int32_t)len;
      ch.rec[t].shift = (S)(lo - excl);
      ch.rec[t].av = av;
      ch.ex[t] = excl;
      if (t == 0) ch.ex[GROUP] = total;
      g.sync();
    }
    for (int32_t r0 = 0; r0 < total; r0 += RUN) {
      const int rn = (int)((total - r0) < RUN ? (total - r0) : RUN);
      const int per = wave_share(rn, GROUP / WAVE);
      const int wlo = w * per;
      const int wlen = min(per, rn - wlo);
      if (wlen <= 0) continue;
      const int base = (int)r0 + wlo;
      // the wavefront's terms, each with the record of its segment
      auto terms = [&](auto rec_of) {
        for (int q0 = lane; q0 < wlen; q0 += WAVE * UR) {
          if constexpr (BATCH) {
            PI pos[UR];
            float am[UR];
            bool ok[UR];
#pragma unroll
            for (int u = 0; u < UR; ++u) {
              const int q = q0 + u * WAVE;
              ok[u] = q < wlen;
              const int qc = ok[u] ? q : q0;
              const typename CH::Rec rc = rec_of(qc);
              pos[u] = (PI)rc.shift + base + qc;
              am[u] = rc.av;
            }
            int j[UR];
            float v[UR];
#pragma unroll
            for (int u = 0; u < UR; ++u) {
              j[u] = op.bcol[pos[u]];
              v[u] = NUM ? am[u] * op.bval[pos[u]] : 0.f;
            }
            f(j, v, ok);
          } else {
            PI pos[UR];
            float am[UR];
#pragma unroll
            for (int u = 0; u < UR; ++u) {
              const int q = q0 + u * WAVE;
              pos[u] = -1;
              am[u] = 0.f;
              if (q < wlen) {
                const typename CH::Rec rc = rec_of(q);
                pos[u] = (PI)rc.shift + base + q;
                am[u] = rc.av;
              }
            }
            int j[UR];
            float bv[UR];
#pragma unroll
            for (int u = 0; u < UR; ++u) {
              j[u] = 0;
              bv[u] = 0.f;
              if (pos[u] >= 0) {
                j[u] = op.bcol[pos[u]];
                if constexpr (NUM) bv[u] = op.bval[pos[u]];
              }
            }
#pragma unroll
            for (int u = 0; u < UR; ++u)
              if (pos[u] >= 0) f(j[u], am[u] * bv[u]);
          }
        }
      };
      const int one = wave_seg_map(ch.ex, nk, base, wlen, seg_w);
      if (one >= 0) {
        const typename CH::Rec r1 = ch.rec[one];
        terms([&](int) { return r1; });
      } else {
        terms([&](int q) { return ch.rec[seg_w[q]]; });
      }
    }
    g.sync();
  }
}

// ... over the terms of A entries [p0, p1); the whole row:
template <typename RA, int GROUP, int BLOCK, bool NUM, bool P32 = false, int UR = UNROLL, bool BATCH = false,
          typename CH, typename SEG, typename F>
__device__ __forceinline__ void for_each_term(const Operands& op, const Group<GROUP, BLOCK>& g,
                                              CH& ch, int64_t row, const SEG& seg, F&& f) {
  const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
  const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
  for_each_term_in<GROUP, BLOCK, NUM, P32, UR, false, BATCH>(op, g, ch, p0, p1, seg, static_cast<F&&>(f));
}

// A row with a single A entry is a_ik times B_k: its columns are B_k's
// (sorted, distinct) and each value is the one product added to +0, as the
// accumulation of every other row starts.  Counts (!NUM) or writes (NUM)
// such a row with the group's threads and returns true; false for any other
// row.  The test is the same for every thread of the group.
template <typename RA, typename RB, int GROUP, bool NUM>
__device__ __forceinline__ bool single_entry_row(const Operands& op, const Outputs& out, int64_t row, int t) {
  const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
  const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
  if (p1 - p0 != 1) return false;
  const int64_t k = op.acol[p0];
  const int64_t lo = ld_rp<RB>(op.brp, k);
  const int64_t len = ld_rp<RB>(op.brp, k + 1) - lo;
  if constexpr (!NUM) {
    if (t == 0) out.counts[row] = len;
  } else {
    const float a = op.aval[p0];
    const int64_t o0 = out.crp[row];
    for (int64_t j = t; j < len; j += GROUP) {
      const float prod = a * op.bval[lo + j];
      store_stream(&out.ccol[o0 + j], op.bcol[lo + j]);
      store_stream(&out.cval[o0 + j], 0.f + prod);
    }
  }
  return true;
}

// -------------------------------------------------- dense path (narrow N)

// LDS layout of one group: [bitmap N/32 words][acc N floats if NUM][Chunk][red]
__host__ __device__ constexpr size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

template <int GROUP, bool NUM, typename S>
__host__ __device__ constexpr size_t dense_group_bytes(int W) {
  return align16(((size_t)W + 31) / 32 * 4) + (NUM ? align16((size_t)W * 4) : 0) +
         align16(sizeof(Chunk<GROUP, S>)) + 64;
}

// Narrow products (N <= 16384): a dense fp32 row of N slots plus a presence
// bitmap in LDS per group; compaction walks the bitmap words with a group
// scan of their popcounts, so the row is written with increasing columns.
template <typename RA, typename RB, int GROUP, int BLOCK, bool NUM>
__global__ __launch_bounds__(BLOCK) void k_dense(const Operands op, const BinView bv,
                                                 const Outputs out) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NG = BLOCK / GROUP;
  const int W = (int)op.N;
  const size_t per = dense_group_bytes<GROUP, NUM, RB>(W);
  const int gi = threadIdx.x / GROUP;
  unsigned char* base = smem + gi * per;
  uint32_t* bm = reinterpret_cast<uint32_t*>(base);
  float* acc = reinterpret_cast<float*>(base + align16(((size_t)W + 31) / 32 * 4));
  using CH = Chunk<GROUP, RB>;
  CH& ch = *reinterpret_cast<CH*>(base + align16(((size_t)W + 31) / 32 * 4) + (NUM ? align16((size_t)W * 4) : 0));
  Group<GROUP, BLOCK> g;
  g.red = reinterpret_cast<int64_t*>(reinterpret_cast<unsigned char*>(&ch) + align16(sizeof(CH)));
  const int t = g.t();
  const int nwd = (W + 31) / 32;
  for (int i = t; i < nwd; i += GROUP) bm[i] = 0u;
  if constexpr (NUM)
    for (int i = t; i < W; i += GROUP) acc[i] = 0.f;
  g.sync();

  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.bin + 1] - bv.binoff[bv.bin];
  const FullRows<RB> seg{op.brp};
  for (int64_t it = (int64_t)blockIdx.x * NG + gi + bv.skip; it < cnt; it += (int64_t)gridDim.x * NG) {
    const int64_t row = list[it];
    if (single_entry_row<RA, RB, GROUP, NUM>(op, out, row, t)) continue;
    if constexpr (!NUM) {
      // presence marks are fire-and-forget ORs: a lane's terms go out with
      // no branch per term (a missing term ORs in nothing)
      for_each_term<RA, GROUP, BLOCK, false, false, UNROLL, true>(
          op, g, ch, row, seg, [&](const int (&j)[UNROLL], const float (&)[UNROLL], const bool (&ok)[UNROLL]) {
            for (int u = 0; u < UNROLL; ++u) atomicOr(&bm[j[u] >> 5], ok[u] ? 1u << (j[u] & 31) : 0u);
          });
    } else {
      for_each_term<RA, GROUP, BLOCK, true>(op, g, ch, row, seg, [&](int j, float v) {
        atomicOr(&bm[j >> 5], 1u << (j & 31));
        lds_add<true>(&acc[j], v);
      });
    }
    if constexpr (!NUM) {
      int64_t c = 0;
      for (int i = t; i < nwd; i += GROUP) {
        c += __popc(bm[i]);
        bm[i] = 0u;
      }
      c = g.sum(c);
      if (t == 0) out.counts[row] = c;
    } else {
      // one column per thread per round: present columns get consecutive
      // output slots, so both C arrays are written with coalesced stores
      int64_t o0 = out.crp[row];
      for (int j0 = 0; j0 < W; j0 += GROUP) {
        const int j = j0 + t;
        const bool present = j < W && ((bm[j >> 5] >> (j & 31)) & 1u);
        int64_t before, tot;
        if constexpr (GROUP == WAVE) {
          const uint64_t mask = __ballot(present);
          before = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
          tot = __popcll(mask);
        } else {
          before = g.incl_scan(present ? 1 : 0, &tot) - (present ? 1 : 0);
        }
        if (present) {
          store_stream(&out.ccol[o0 + before], j);
          store_stream(&out.cval[o0 + before], acc[j]);
          acc[j] = 0.f;
        }
        o0 += tot;
      }
      g.sync();
      for (int i = t; i < nwd; i += GROUP) bm[i] = 0u;
    }
    g.sync();
  }
}

// ------------------------------------------- split rows (narrow N, heavy)
//
// The heaviest rows of a narrow product are cut into SPLIT_PARTS runs of
// their A entries, one workgroup per run.  A run accumulates into a dense
// LDS row as above and adds it into the row's dense slot in global memory
// (presence bits by atomic OR, values by atomic add); a wavefront per row
// then counts the slot (symbolic) or writes it out in column order.

constexpr int SPLIT_BLOCK = 512;
constexpr int SPLIT_PARTS = 32;

template <typename RA, typename RB, bool NUM>
__global__ __launch_bounds__(SPLIT_BLOCK) void k_split_parts(const Operands op, const BinView bv,
                                                            const SplitWs sw) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int N = (int)op.N;
  const int nwd = (N + 31) / 32;
  uint32_t* bm = reinterpret_cast<uint32_t*>(smem);
  float* acc = reinterpret_cast<float*>(smem + align16((size_t)nwd * 4));
  using CH = Chunk<SPLIT_BLOCK, RB>;
  CH& ch = *reinterpret_cast<CH*>(smem + align16((size_t)nwd * 4) + (NUM ? align16((size_t)N * 4) : 0));
  Group<SPLIT_BLOCK, SPLIT_BLOCK> g;
  g.red = reinterpret_cast<int64_t*>(reinterpret_cast<unsigned char*>(&ch) + align16(sizeof(CH)));
  const int t = threadIdx.x;
  for (int i = t; i < nwd; i += SPLIT_BLOCK) bm[i] = 0u;
  if constexpr (NUM)
    for (int i = t; i < N; i += SPLIT_BLOCK) acc[i] = 0.f;
  g.sync();
  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = min((int64_t)(bv.binoff[bv.bin + 1] - bv.binoff[bv.bin]), sw.cap);
  const FullRows<RB> seg{op.brp};
  for (int64_t it = blockIdx.x; it < cnt * SPLIT_PARTS; it += gridDim.x) {
    const int64_t d = it / SPLIT_PARTS;
    const int64_t part = it - d * SPLIT_PARTS;
    const int64_t row = list[d];
    const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
    const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
    const int64_t len = (p1 - p0 + SPLIT_PARTS - 1) / SPLIT_PARTS;
    const int64_t q0 = min(p1, p0 + part * len), q1 = min(p1, q0 + len);
    if (q0 < q1) {
      if constexpr (!NUM) {
        for_each_term_in<SPLIT_BLOCK, SPLIT_BLOCK, false, false, UNROLL, false, true>(
            op, g, ch, q0, q1, seg, [&](const int (&j)[UNROLL], const float (&)[UNROLL], const bool (&ok)[UNROLL]) {
              for (int u = 0; u < UNROLL; ++u) atomicOr(&bm[j[u] >> 5], ok[u] ? 1u << (j[u] & 31) : 0u);
            });
      } else {
        for_each_term_in<SPLIT_BLOCK, SPLIT_BLOCK, true>(op, g, ch, q0, q1, seg, [&](int j, float v) {
          atomicOr(&bm[j >> 5], 1u << (j & 31));
          lds_add<true>(&acc[j], v);
        });
      }
    }
    if constexpr (NUM) {
      for (int j = t; j < N; j += SPLIT_BLOCK)
        if ((bm[j >> 5] >> (j & 31)) & 1u) {
          atomicAdd(&sw.acc[d * N + j], acc[j]);
          acc[j] = 0.f;
        }
      __syncthreads();
    }
    for (int w = t; w < nwd; w += SPLIT_BLOCK) {
      const uint32_t x = bm[w];
      if (x) {
        atomicOr(&sw.bm[d * nwd + w], x);
        bm[w] = 0u;
      }
    }
    __syncthreads();
  }
}

// Clears the slots of the rows the parts kernel takes.
__global__ __launch_bounds__(256) void k_split_clear(const BinView bv, SplitWs sw, int32_t N, int num) {
  const int nwd = (N + 31) / 32;
  const int64_t cnt = min((int64_t)(bv.binoff[bv.bin + 1] - bv.binoff[bv.bin]), sw.cap);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < cnt * nwd; i += stride) sw.bm[i] = 0u;
  if (num)
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < cnt * N; i += stride) sw.acc[i] = 0.f;
}

// One wavefront per split row: count its slot, or write it in column order.
template <bool NUM>
__global__ __launch_bounds__(256) void k_split_finish(const BinView bv, const SplitWs sw, int32_t N,
                                                     const Outputs out) {
  const int nwd = (N + 31) / 32;
  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = min((int64_t)(bv.binoff[bv.bin + 1] - bv.binoff[bv.bin]), sw.cap);
  const int64_t nw = (int64_t)gridDim.x * (blockDim.x / WAVE);
  for (int64_t d = (int64_t)blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE; d < cnt; d += nw) {
    const int64_t row = list[d];
    const uint32_t* words = sw.bm + d * nwd;
    if constexpr (!NUM) {
      int64_t c = 0;
      for (int w = lane_id(); w < nwd; w += WAVE) c += __popc(words[w]);
      c = wave_sum(c);
      if (lane_id() == 0) out.counts[row] = c;
    } else {
      int64_t o0 = out.crp[row];
      for (int j0 = 0; j0 < N; j0 += WAVE) {
        const int j = j0 + lane_id();
        const bool present = j < N && ((words[j >> 5] >> (j & 31)) & 1u);
        const uint64_t mask = __ballot(present);
        const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
        if (present) {
          store_stream(&out.ccol[o0 + before], j);
          store_stream(&out.cval[o0 + before], sw.acc[d * N + j]);
        }
        o0 += __popcll(mask);
      }
    }
  }
}

// -------------------------------------------------------------- hash path

template <int TABLE, int GROUP, bool NUM, typename S>
struct HashLds {
  int32_t key[TABLE];
  float val[NUM ? TABLE : 1];
  Chunk<GROUP, S> ch;
  int64_t red[GROUP / WAVE + 1];
};

// Buckets for ordering a hash row's columns: as many as the chunk's segment
// maps hold as 32-bit counters (at most 1024), each 2^shift consecutive
// columns wide so that NB buckets cover [0, N).
__host__ __device__ constexpr int bucket_count(int group) {
  return group * SEG_PER_THREAD / 2 < 1024 ? group * SEG_PER_THREAD / 2 : 1024;
}
__device__ __forceinline__ int bucket_shift(int64_t N, int nb) {
  int sh = 0;
  while (((N - 1) >> sh) >= nb) ++sh;
  return sh;
}

template <int TABLE>
__device__ __forceinline__ uint32_t hslot(int j) {
  constexpr int LOG2 = __builtin_ctz(TABLE);
  return ((uint32_t)j * 2654435761u) >> (32 - LOG2);
}

// Light rows of wide products: open addressing keyed by column (linear
// probing, load <= 1/2 since nnz(C_i) <= P_i <= TABLE/2), then the occupied
// slots are compacted and put in column order by bucket counts and a rank
// within each bucket (a handful of columns per bucket).
template <typename RA, typename RB, int TABLE, int GROUP, int BLOCK, bool NUM>
__global__ __launch_bounds__(BLOCK) void k_hash(const Operands op, const BinView bv,
                                                const Outputs out) {
  constexpr int NG = BLOCK / GROUP;
  constexpr int SPT = TABLE / GROUP;   // table slots per thread
  static_assert(TABLE % GROUP == 0, "table divides over the group");
  __shared__ HashLds<TABLE, GROUP, NUM, RB> lds[NG];
  const int gi = threadIdx.x / GROUP;
  HashLds<TABLE, GROUP, NUM, RB>& L = lds[gi];
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
  const FullRows<RB> seg{op.brp};
  for (int64_t it = (int64_t)blockIdx.x * NG + gi; it < cnt; it += (int64_t)gridDim.x * NG) {
    const int64_t row = list[it];
    if (single_entry_row<RA, RB, GROUP, NUM>(op, out, row, t)) continue;
    int64_t mine = 0;
    for_each_term<RA, GROUP, BLOCK, NUM>(op, g, L.ch, row, seg, [&](int j, float v) {
      uint32_t h = hslot<TABLE>(j);
      for (;;) {
        const int old = atomicCAS(&L.key[h], -1, j);
        if (old == -1 || old == j) {
          if constexpr (NUM) lds_add<true>(&L.val[h], v);
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
      g.sync();
      // order the n compacted pairs by column (the columns are distinct):
      // count them into NB buckets of consecutive columns, place each pair
      // in its bucket's range of the upper half of the table, then give it
      // the rank start(bucket) + (pairs of the bucket with a smaller
      // column) in the lower half (n <= TABLE / 2)
      constexpr int NB = bucket_count(GROUP);
      constexpr int EPT = (TABLE / 2 + GROUP - 1) / GROUP;  // pairs per thread
      int32_t* cnt = reinterpret_cast<int32_t*>(L.ch.seg);   // the chunk's maps are free now
      const int shift = bucket_shift(op.N, NB);
      for (int b = t; b < NB; b += GROUP) cnt[b] = 0;
      g.sync();
      int32_t ek[EPT];
      float ev[EPT];
      int es[EPT];
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int i = t + e * GROUP;
        ek[e] = 0;
        ev[e] = 0.f;
        es[e] = -1;
        if (i < n) {
          ek[e] = L.key[i];
          ev[e] = L.val[i];
          es[e] = atomicAdd(&cnt[ek[e] >> shift], 1);
        }
      }
      g.sync();
      {
        constexpr int BPT = NB / GROUP > 0 ? NB / GROUP : 1;  // buckets per thread
        int c[BPT];
        int32_t sum = 0;
#pragma unroll
        for (int q = 0; q < BPT; ++q) {
          const int b = t * BPT + q;
          c[q] = b < NB ? cnt[b] : 0;
          sum += c[q];
        }
        int32_t tot;
        int32_t run = g.incl_scan32(sum, &tot) - sum;
#pragma unroll
        for (int q = 0; q < BPT; ++q) {
          const int b = t * BPT + q;
          if (b < NB) cnt[b] = run;
          run += c[q];
        }
      }
      g.sync();
      int32_t* hk = L.key + TABLE / 2;
      float* hv = L.val + TABLE / 2;
#pragma unroll
      for (int e = 0; e < EPT; ++e)
        if (es[e] >= 0) {
          const int d = cnt[ek[e] >> shift] + es[e];
          hk[d] = ek[e];
          hv[d] = ev[e];
        }
      g.sync();
#pragma unroll
      for (int e = 0; e < EPT; ++e)
        if (es[e] >= 0) {
          const int b = ek[e] >> shift;
          const int s0 = cnt[b], s1 = b + 1 < NB ? cnt[b + 1] : (int)n;
          int r = s0;
          for (int q = s0; q < s1; ++q) r += hk[q] < ek[e];
          L.key[r] = ek[e];
          L.val[r] = ev[e];
        }
      g.sync();
      const int32_t* ksrc = L.key;
      const float* vsrc = L.val;
      const int64_t o0 = out.crp[row];
      for (int i = t; i < n; i += GROUP) {
        store_stream(&out.ccol[o0 + i], ksrc[i]);
        store_stream(&out.cval[o0 + i], vsrc[i]);
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

// ------------------------------------------------- wide rows: column windows
//
// Wide products (N above the densest LDS row) split the columns into grains
// of G columns.  Symbolic: a workgroup takes a row and, for each run of
// grains (a symbolic item) in column order, sets a presence bitmap, writes
// each grain's popcount and, for heavy rows, keeps the bitmap in global
// memory.  A plan kernel then cuts every row into windows of whole grains
// whose bitmap and values fit one LDS pool (and at most max_entries entries
// and max_grains grains), within one symbolic item where the row's bitmaps
// are kept.  Numeric, per window: the presence bitmap is set from the terms
// (or loaded from the kept one), wavefront scans turn word popcounts into
// ranks, and each term is added into a compact fp32 array at the rank of
// its column; the values are written out, then the column ids, staged at
// their ranks from the bitmap.  LDS grows with the window's entries, not
// its width.

constexpr int WIN_BLOCK = 512;
constexpr int WIN_UNROLL = 2;  // the numeric window kernel keeps fewer loads in flight (registers)
// Largest rounding error (absolute, per entry of C) that a row's fixed-point
// accumulation may carry; rows whose bound exceeds it add in fp32.
constexpr float FIXED_ERR = 1e-6f;

template <typename S>
__host__ __device__ constexpr size_t count_lds_bytes(int sg, int G) {
  return align16((size_t)sg * (G / 32) * 4) + align16((size_t)sg * 4) + align16(sizeof(Chunk<WIN_BLOCK, S>)) + 128 +
         16;  // + the static list offset
}

// Rows whose symbolic bitmaps are kept for the numeric phase (one copy per
// symbolic item, as far as the cache holds them).
__device__ __forceinline__ bool keeps_bitmaps(const WindowParams& wp, int64_t row) {
  return wp.bm_cache && wp.P[row] > wp.bm_min_products;
}

// Rows whose windows never straddle a symbolic item: the rows that keep
// their bitmaps when the cache is there.  The window plan (symbolic phase)
// and its fill (numeric phase) must cut a row alike.
__device__ __forceinline__ bool cuts_at_items(const WindowParams& wp, int64_t row) {
  return wp.item_cut && wp.P[row] > wp.bm_min_products;
}

template <typename RA, typename RB>
__global__ __launch_bounds__(WIN_BLOCK, 8) void k_grain_count(const Operands op, const BinView bv,
                                                           const WindowParams wp) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int64_t s_off, s_row;
  constexpr int64_t CACHE_CHUNK = 65536;  // cache words a workgroup takes from the shared buffer at once
  constexpr int NWV = WIN_BLOCK / WAVE;
  int64_t chunk_cur = 0, chunk_end = 0;   // thread 0: the workgroup's current chunk
  const int SG = wp.grains_per_count_item;
  const int WPG = op.G / 32;  // bitmap words per grain
  const int nwmax = SG * WPG;
  uint32_t* bm = reinterpret_cast<uint32_t*>(smem);
  const size_t bm_bytes = align16((size_t)nwmax * 4);
  using CH = Chunk<WIN_BLOCK, RB>;
  CH& ch = *reinterpret_cast<CH*>(smem + bm_bytes + align16((size_t)SG * 4));
  Group<WIN_BLOCK, WIN_BLOCK> g;
  g.red = reinterpret_cast<int64_t*>(reinterpret_cast<unsigned char*>(&ch) + align16(sizeof(CH)));
  const int t = threadIdx.x;
  const int lane = lane_id(), wv = t / WAVE;
  for (int i = t; i < nwmax; i += WIN_BLOCK) bm[i] = 0u;
  __syncthreads();

  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.last() + 1] - bv.binoff[bv.bin];
  const int64_t ngg = (op.nG + SG - 1) / SG;
  // Workgroups take rows from a shared counter (the heaviest bin first) and
  // walk a row's items in column order.  A row with at most WIN_BLOCK
  // entries keeps one k per thread in a register with the B position where
  // its segment for the current item starts; consecutive items share a
  // grain boundary, so an item needs one index lookup per k (its end),
  // issued while the previous item is counted.
  for (;;) {
    __syncthreads();
    if (t == 0) s_row = atomicAdd(wp.row_counter, 1);
    __syncthreads();
    const int64_t dd = s_row;
    if (dd >= cnt) break;
    const int64_t row = list[cnt - 1 - dd];
    const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
    const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
    const bool short_row = (p1 - p0) <= WIN_BLOCK;
    int32_t k = -1;
    if (short_row && p0 + t < p1) k = op.acol[p0 + t];
    const int32_t* kr = op.bidx + (int64_t)(k >= 0 ? k : 0) * (op.nG + 1);
    int32_t lo = 0, hi_next = 0;
    if (k >= 0) {
      lo = kr[0];
      hi_next = kr[min((int)op.nG, SG)];
    }
    for (int64_t gg = 0; gg < ngg; ++gg) {
      const int g0 = (int)(gg * SG);
      const int g1 = min((int)op.nG, g0 + SG);
      const int c0 = g0 * op.G;
      const int32_t hi = hi_next;
      if (k >= 0 && gg + 1 < ngg) hi_next = kr[min((int)op.nG, g1 + SG)];  // the next item's segment end
      // terms carry absolute columns: bma is the bitmap seen from column 0
      // (c0 is a multiple of 32, so a column's bit index is the same)
      uint32_t* bma = bm - (c0 >> 5);
      // a lane's eight terms at once, with no branch per term (a missing
      // term ORs in nothing): all eight B loads in flight, then the ORs
      auto mark = [&](const int (&j)[8], const float (&)[8], const bool (&ok)[8]) {
#pragma unroll
        for (int u = 0; u < 8; ++u) atomicOr(&bma[j[u] >> 5], ok[u] ? 1u << (j[u] & 31) : 0u);
      };
      // eight B loads in flight per thread: the symbolic loop reads columns only
      if (short_row)
        for_each_term_in<WIN_BLOCK, WIN_BLOCK, false, true, 8, true, true>(
            op, g, ch, p0, p1, HeldRange{lo, (int64_t)hi - lo}, mark);
      else
        for_each_term<RA, WIN_BLOCK, WIN_BLOCK, false, true, 8, true>(op, g, ch, row,
                                                                      GrainRange{op.bidx, op.nG + 1, g0, g1}, mark);
      lo = hi;
      const int nw = (g1 - g0) * WPG;
      int64_t off = -1;
      if (keeps_bitmaps(wp, row)) {
        // heavy row: keep the item's bitmap for the numeric phase, in a slot
        // taken from the workgroup's chunk of the shared cache
        if (t == 0) {
          if (chunk_cur + nw > chunk_end) {
            const int64_t take = max<int64_t>(CACHE_CHUNK, nw);
            chunk_cur = (int64_t)atomicAdd(wp.bm_top, (unsigned long long)take);
            chunk_end = chunk_cur + take;
          }
          const int64_t o = chunk_cur + nw <= wp.bm_cap ? chunk_cur : -1;
          chunk_cur += nw;
          s_off = o;
          wp.bm_off[row * ngg + gg] = o;
        }
        __syncthreads();
        off = s_off;
      } else if (wp.bm_cache && t == 0) {
        wp.bm_off[row * ngg + gg] = -1;
      }
      // one pass over the bitmap: per-grain popcounts (a wavefront per grain,
      // lanes on consecutive words), the copy of a kept bitmap (coalesced)
      // and the clearing for the next item
      if (WPG % (4 * WAVE) == 0) {
        // 16-byte LDS reads and writes (and cache stores): a quarter of the
        // instructions, the same bytes
        uint4* bm4 = reinterpret_cast<uint4*>(bm);
        for (int gi = wv; gi < g1 - g0; gi += NWV) {
          uint32_t c = 0;
          for (int w = gi * (WPG / 4) + lane; w < (gi + 1) * (WPG / 4); w += WAVE) {
            const uint4 x = bm4[w];
            c += __popc(x.x) + __popc(x.y) + __popc(x.z) + __popc(x.w);
            if (off >= 0) reinterpret_cast<uint4*>(wp.bm_cache + off)[w] = x;
            bm4[w] = make_uint4(0u, 0u, 0u, 0u);
          }
          c = wave_sum(c);
          if (lane == 0) wp.gcnt[row * op.nG + g0 + gi] = (int32_t)c;
        }
      } else {
        for (int gi = wv; gi < g1 - g0; gi += NWV) {
          uint32_t c = 0;
          for (int w = gi * WPG + lane; w < (gi + 1) * WPG; w += WAVE) {
            const uint32_t x = bm[w];
            c += __popc(x);
            if (off >= 0) wp.bm_cache[off + w] = x;
            bm[w] = 0u;
          }
          c = wave_sum(c);
          if (lane == 0) wp.gcnt[row * op.nG + g0 + gi] = (int32_t)c;
        }
      }
      __syncthreads();  // the bitmap is clear before the next item's terms
    }
  }
}

// Greedy windows of whole grains (at most max_grains grains and max_entries
// entries; for a row whose symbolic bitmaps are kept, never across a
// symbolic item boundary, a multiple of sg grains, as a window loads its
// bits from one item's copy); empty windows are skipped.  Calls
// f(g0, g1, n, roff).
template <typename F>
__device__ __forceinline__ int64_t plan_windows(const int32_t* gc, int nG, const WindowParams& wp, int gcols,
                                                bool kept, F&& f) {
  const int sg = kept ? wp.grains_per_count_item : nG + 1;
  int64_t roff = 0;
  int g0 = 0;
  while (g0 < nG) {
    int n = gc[g0];
    int g1 = g0 + 1;
    // the window's bitmap (8 bytes per WIN_WORD_BITS columns: bits and rank)
    // and its values share the LDS pool
    while (g1 < nG && g1 - g0 < wp.max_grains && g1 % sg != 0 && n + gc[g1] <= wp.max_entries &&
           2 * win_words((g1 + 1 - g0) * gcols) + n + gc[g1] <= wp.pool_words)
      n += gc[g1++];
    if (n > 0) f(g0, g1, n, roff);
    roff += n;
    g0 = g1;
  }
  return roff;
}

__global__ __launch_bounds__(256) void k_win_plan(const BinView bv, int32_t nG, int32_t gcols, const WindowParams wp,
                                                  int64_t* counts) {
  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.last() + 1] - bv.binoff[bv.bin];
  for (int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; d < cnt; d += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = list[d];
    int64_t nwin = 0;
    counts[row] = plan_windows(wp.gcnt + row * nG, nG, wp, gcols, cuts_at_items(wp, row),
                               [&](int, int, int, int64_t) { ++nwin; });
    wp.item_count[1 + d] = nwin;
  }
}

__global__ __launch_bounds__(256) void k_win_fill(const BinView bv, int32_t nG, int32_t gcols, const WindowParams wp) {
  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.last() + 1] - bv.binoff[bv.bin];
  for (int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; d < cnt; d += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = list[d];
    int64_t o = wp.item_count[d];  // scanned: windows of the rows before d
    plan_windows(wp.gcnt + row * nG, nG, wp, gcols, cuts_at_items(wp, row), [&](int g0, int g1, int n, int64_t roff) {
                   WinItem w;
                   w.row = (int32_t)row;
                   w.g0 = (uint16_t)g0;
                   w.g1 = (uint16_t)g1;
                   w.n = n;
                   w.roff = (int32_t)roff;
                   wp.items[o++] = w;
                 });
  }
}

// A window's LDS: a pool holding the bitmap as 8-byte words of
// WIN_WORD_BITS presence bits with the rank of the word's first set bit in
// the top 16 bits (a term's rank is one 8-byte read), followed by the
// window's fp32 values (a wide window with few entries and a narrow one with
// many use the same pool); then the chunk.

template <typename S>
__host__ __device__ constexpr size_t window_lds_bytes(int pool_words) {
  return align16((size_t)pool_words * 4) + align16(sizeof(Chunk<WIN_BLOCK, S>)) + 128 + 16;  // + the static row slot
}

// Numeric phase of wide rows.  Workgroups take rows from a shared counter
// (the heaviest bin first) and walk each row's windows in column order.
// The rows of the slab bins (the heaviest) are taken once per column slab:
// workgroup b serves slab b mod nslab through that slab's counter and does
// the row's windows whose middle grain lies in the slab, then joins the
// shared counter.  The hardware places workgroup b on XCD b mod 8, so each
// XCD's L2 holds the B segments of one slab of columns rather than of all.
// For a row with at most WIN_BLOCK entries each thread keeps one (k, a_ik)
// of the row in registers with the position where B_k's segment for the
// current window starts; consecutive windows share a grain boundary, so a
// window needs one index lookup per k (its end), issued while the previous
// window is processed.  A window with at most WIN_BLOCK * SEG_PER_THREAD
// terms loads each term once into registers; larger windows make two
// passes over the B segments (one when the symbolic bitmap was kept),
// keeping the row's state in LDS.
template <typename RA, typename RB>
__global__ __launch_bounds__(WIN_BLOCK, 6) void k_win_rows(const Operands op, const BinView bv,
                                                           const WindowParams wp, const Outputs out) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int64_t s_row;
  __shared__ int s_shared;  // this workgroup's slab rows are done
  __shared__ float s_fsum[WIN_BLOCK / WAVE];  // per-wavefront parts of a row's bound
  const int WPG = op.G / 32;  // 32-bit words per grain of a kept symbolic bitmap
  constexpr uint64_t BITS = (uint64_t(1) << WIN_WORD_BITS) - 1u;
  uint64_t* bw = reinterpret_cast<uint64_t*>(smem);  // presence bits | rank of the word's first bit << 48
  using CH = Chunk<WIN_BLOCK, RB>;
  CH& ch = *reinterpret_cast<CH*>(smem + align16((size_t)wp.pool_words * 4));
  Group<WIN_BLOCK, WIN_BLOCK> g;
  g.red = reinterpret_cast<int64_t*>(reinterpret_cast<unsigned char*>(&ch) + align16(sizeof(CH)));
  const int t = threadIdx.x;
  for (int i = t; i < wp.pool_words; i += WIN_BLOCK) reinterpret_cast<uint32_t*>(smem)[i] = 0u;  // pool clear
  constexpr int RUN = WIN_BLOCK * SEG_PER_THREAD;
  const int32_t* list = bv.list + bv.binoff[bv.bin];
  const int64_t cnt = bv.binoff[bv.last() + 1] - bv.binoff[bv.bin];
  // the slab bins are the last of the view: their rows end the list
  const int64_t nslab_rows = wp.slab_bin >= 0 ? bv.binoff[bv.last() + 1] - bv.binoff[wp.slab_bin] : 0;
  const int slab = (int)(blockIdx.x % (unsigned)wp.nslab);
  if (t == 0) s_shared = nslab_rows > 0 ? 0 : 1;

  for (;;) {
    __syncthreads();
    if (t == 0) {
      int64_t v = 0;
      if (!s_shared) {
        v = atomicAdd(wp.row_counter + 1 + slab, 1);
        if (v >= nslab_rows) s_shared = 1;
      }
      if (s_shared) v = nslab_rows + atomicAdd(wp.row_counter, 1);
      s_row = v;
    }
    __syncthreads();
    const int64_t dd = s_row;
    if (dd >= cnt) break;
    const int64_t d = cnt - 1 - dd;  // the heavy bin sits at the end of the list
    const int64_t row = list[d];
    int64_t i0 = wp.item_count[d], i1 = wp.item_count[d + 1];
    if (dd < nslab_rows) {
      // this slab's windows: a run of the row's (column-ordered) windows,
      // counted by each wavefront from their headers, 64 at a time
      int64_t j0 = i0, j1 = i0;
      for (int64_t c = i0; c < i1; c += WAVE) {
        const int64_t q = c + lane_id();
        int sl = wp.nslab;
        if (q < i1) {
          const WinItem w = wp.items[q];
          sl = (int)(((int64_t)w.g0 + w.g1) * wp.nslab / (2 * (int64_t)op.nG));
        }
        j0 += __popcll(__ballot(sl < slab));
        j1 += __popcll(__ballot(sl <= slab));
      }
      i0 = j0;
      i1 = j1;
    }
    const int64_t p0 = ld_rp<RA>(op.arp, row) - op.a_base;
    const int64_t p1 = ld_rp<RA>(op.arp, row + 1) - op.a_base;
    const int64_t rbase = out.crp[row];
    const bool short_row = (p1 - p0) <= WIN_BLOCK;
    int32_t k = -1;  // B positions of a wide product fit 32 bits (nnz(B) < 2^31)
    float a = 0.f;
    if (short_row && p0 + t < p1) {
      k = op.acol[p0 + t];
      a = op.aval[p0 + t];
    }
    // The row's accumulation (uniform over the workgroup, in scalar
    // registers): fixed point where a bound allows, else fp32.
    // S = sum_k |a_ik| max_j |b_kj| bounds every |a_ik b_kj| of the row and
    // every |c_ij|.  With S < 2^e and f = 30 - e, each product scaled by 2^f
    // and rounded to an integer is below 2^30 in magnitude, and so is the sum
    // of an entry's scaled products plus their roundings (at most |A_i| / 2),
    // so adding them in 32-bit two's complement gives that integer sum
    // exactly, whatever the order; the entry's only errors are the roundings
    // of its products, at most 2^-(f+1) each for at most |A_i| products, and
    // the final conversion to fp32.  (S itself is an fp32 sum; with
    // |A_i| < 2^20 its rounding leaves the scaled sums below 2^31.)  Where
    // |A_i| 2^-(f+1) <= FIXED_ERR the
    // adds are plain integer adds (one LDS operation with no return, no
    // retry); otherwise, and for NaN or infinite values, fp32
    // compare-and-swap adds.
    float fx_scale = 0.f, fx_inv = 0.f;  // 0: fp32 adds
    if (op.bmax && i0 < i1) {
      float sv = 0.f;
      if (short_row) {
        if (k >= 0) sv = fabsf(a) * op.bmax[k];
      } else {
        for (int64_t p = p0 + t; p < p1; p += WIN_BLOCK) sv += fabsf(op.aval[p]) * op.bmax[op.acol[p]];
      }
      sv = wave_sum_f32(sv);
      if (lane_id() == 0) s_fsum[t / WAVE] = sv;
      __syncthreads();
      float S = 0.f;
#pragma unroll
      for (int i = 0; i < WIN_BLOCK / WAVE; ++i) S += s_fsum[i];
      int e = 0;
      frexpf(S, &e);
      const int f = min(30 - e, 120);
      if (S <= 1e30f && p1 - p0 < (1 << 20) && (float)(p1 - p0) * ldexpf(1.f, -(f + 1)) <= FIXED_ERR) {
        fx_scale = ldexpf(1.f, f);
        fx_inv = ldexpf(1.f, -f);
      }
      fx_scale = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(fx_scale)));
      fx_inv = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(fx_inv)));
    }
    int32_t cur = 0, nxt_hi = 0;
    int prev_g1 = -1;
    WinItem nextI{};
    if (i0 < i1) {
      nextI = wp.items[i0];
      if (k >= 0) nxt_hi = op.bidx[(int64_t)k * (op.nG + 1) + nextI.g1];
    }
    for (int64_t it = i0; it < i1; ++it) {
      const WinItem I = nextI;
      const int32_t hi = nxt_hi;
      if (it + 1 < i1) {  // next window's header and segment ends, in flight meanwhile
        nextI = wp.items[it + 1];
        if (k >= 0) nxt_hi = op.bidx[(int64_t)k * (op.nG + 1) + nextI.g1];
      }
      const int g0 = I.g0, g1 = I.g1, n = I.n;
      const int c0 = g0 * op.G;
      const int nw32 = (g1 - g0) * WPG;
      const int nw = (int)win_words((int64_t)(g1 - g0) * op.G);
      float* vals = reinterpret_cast<float*>(bw + nw);  // the values follow this window's bitmap
      const int64_t base = rbase + I.roff;
      auto set_bit = [&](int j) {
        const uint32_t dj = (uint32_t)(j - c0);
        const uint32_t w = dj / WIN_WORD_BITS;
        atomicOr(reinterpret_cast<unsigned long long*>(&bw[w]), 1ull << (dj - w * WIN_WORD_BITS));
      };
      // the same with no branch for a term that may be missing (ok false):
      // j is then any column of the window, and nothing is ORed in
      auto set_bit_if = [&](int j, bool ok) {
        const uint32_t dj = (uint32_t)(j - c0);
        const uint32_t w = dj / WIN_WORD_BITS;
        atomicOr(reinterpret_cast<unsigned long long*>(&bw[w]), ok ? 1ull << (dj - w * WIN_WORD_BITS) : 0ull);
      };
      // Heavy rows: the symbolic phase kept the window's bitmap.
      int64_t cached = -1;
      if (keeps_bitmaps(wp, row)) {
        const int SG = wp.grains_per_count_item;
        const int64_t o = wp.bm_off[row * ((op.nG + SG - 1) / SG) + g0 / SG];
        if (o >= 0) cached = o + (int64_t)(g0 % SG) * WPG;
      }
      // the kept bitmap has 32 columns per word from c0 on: a window word is
      // the 48 bits from column 48 w, i.e. of kept words 3w/2 and 3w/2 + 1
      auto load_bits = [&]() {
        __syncthreads();  // the previous window's bitmap is cleared
        for (int w = t; w < nw; w += WIN_BLOCK) {
          const int q = (w * WIN_WORD_BITS) >> 5;
          const uint64_t lo = wp.bm_cache[cached + q];
          const uint64_t hi = q + 1 < nw32 ? wp.bm_cache[cached + q + 1] : 0u;
          bw[w] = ((hi << 32 | lo) >> ((w * WIN_WORD_BITS) & 31)) & BITS;
        }
        __syncthreads();
      };
      auto add_at_rank = [&](int j, float v) {
        const uint32_t dj = (uint32_t)(j - c0);
        const uint32_t w = dj / WIN_WORD_BITS;
        const uint64_t e = bw[w];
        const int rk = (int)(e >> WIN_WORD_BITS) + __popcll(e & ((1ull << (dj - w * WIN_WORD_BITS)) - 1u));
        if (rk < n) {
          if (fx_scale != 0.f)
            atomicAdd(reinterpret_cast<int32_t*>(&vals[rk]), (int32_t)rintf(v * fx_scale));
          else
            lds_add<false>(&vals[rk], v);
        }
      };
      // fixed point with no branch per term: a missing term (ok false, j any
      // column of the window) or a rank past the window's entries adds 0 to
      // slot 0, which changes nothing
      auto add_fixed_if = [&](int j, float v, bool ok) {
        const uint32_t dj = (uint32_t)(j - c0);
        const uint32_t w = dj / WIN_WORD_BITS;
        const uint64_t e = bw[w];
        const int rk = (int)(e >> WIN_WORD_BITS) + __popcll(e & ((1ull << (dj - w * WIN_WORD_BITS)) - 1u));
        const bool in = ok && rk < n;
        atomicAdd(reinterpret_cast<int32_t*>(vals) + (in ? rk : 0), in ? (int32_t)rintf(v * fx_scale) : 0);
      };
      // exclusive popcount prefix over the window's words: each wavefront
      // takes a contiguous share [wa0, wa1), its lanes consecutive words,
      // with one wavefront scan per 64 words and the shares' totals carried
      // in; the share's set bits have the ranks [wr0, wr1)
      constexpr int NWV = WIN_BLOCK / WAVE;
      const int wcw = (nw + NWV * WAVE - 1) / (NWV * WAVE) * WAVE;
      // wavefront-uniform: kept in scalar registers
      const int wa0 = __builtin_amdgcn_readfirstlane(min(nw, (t / WAVE) * wcw));
      const int wa1 = min(nw, wa0 + wcw);
      uint32_t wr0 = 0, wr1 = 0;
      auto word_ranks = [&]() {
        const int lane = lane_id(), wv = t / WAVE;
        uint32_t sw = 0;
        for (int w = wa0 + lane; w < wa1; w += WAVE) sw += __popcll(bw[w]);
        sw = wave_sum(sw);
        if (lane == 0) g.red[wv] = sw;
        __syncthreads();
        uint32_t carry = 0;
        for (int i = 0; i < wv; ++i) carry += (uint32_t)g.red[i];
        wr0 = __builtin_amdgcn_readfirstlane(carry);
        for (int b = wa0; b < wa1; b += WAVE) {
          const int w = b + lane;
          const uint64_t x = w < wa1 ? bw[w] : 0u;
          const uint32_t c = __popcll(x);
          const uint32_t incl = wave_incl_scan(c);
          // only set bits are ranked: empty words stay all zero
          if (c) bw[w] = x | (uint64_t)(carry + incl - c) << WIN_WORD_BITS;
          carry += wave_last(incl);
        }
        wr1 = __builtin_amdgcn_readfirstlane(carry);
        __syncthreads();
      };
      if (short_row) {
        if (k >= 0 && g0 != prev_g1) cur = op.bidx[(int64_t)k * (op.nG + 1) + g0];
        const int32_t len = (k >= 0) ? hi - cur : 0;
        int32_t total;
        const int32_t incl = g.incl_scan32(len, &total);
        const int32_t excl = incl - len;
        ch.rec[t].shift = (RB)(cur - excl);
        ch.rec[t].av = a;
        ch.ex[t] = (int32_t)excl;
        if (t == 0) ch.ex[WIN_BLOCK] = (int32_t)total;
        __syncthreads();
        const int nk = (int)(p1 - p0);
        constexpr int WR = WAVE * SEG_PER_THREAD;  // terms of one wavefront per run
        const int lane = lane_id();
        const int wi = t / WAVE;
        uint16_t* seg_w = ch.seg + wi * WR;
        if (total <= RUN) {
          // every term of the window in registers
          const int per = wave_share((int)total, WIN_BLOCK / WAVE);
          const int wlo = wi * per;
          const int wlen = min(per, (int)total - wlo);
          const int one = wlen > 0 ? wave_seg_map(ch.ex, nk, wlo, wlen, seg_w) : -1;
          int jj[SEG_PER_THREAD];
          float vv[SEG_PER_THREAD];
          // positions first, then every load, then the products: all of the
          // window's B loads are in flight together (a product right after
          // its load would wait for each load in turn)
          auto load_terms = [&](auto rec_of) {
            int32_t pos[SEG_PER_THREAD];
#pragma unroll
            for (int i = 0; i < SEG_PER_THREAD; ++i) {
              const int q = lane + i * WAVE;
              pos[i] = -1;
              vv[i] = 0.f;
              if (q < wlen) {
                const typename CH::Rec rc = rec_of(q);
                pos[i] = (int32_t)rc.shift + wlo + q;
                vv[i] = rc.av;
              }
            }
            float bv[SEG_PER_THREAD];
#pragma unroll
            for (int i = 0; i < SEG_PER_THREAD; ++i) {
              jj[i] = -1;
              bv[i] = 0.f;
              if (pos[i] >= 0) {
                jj[i] = op.bcol[pos[i]];
                bv[i] = op.bval[pos[i]];
              }
            }
#pragma unroll
            for (int i = 0; i < SEG_PER_THREAD; ++i) vv[i] *= bv[i];
          };
          if (one >= 0) {
            const typename CH::Rec r1 = ch.rec[one];
            load_terms([&](int) { return r1; });
          } else {
            load_terms([&](int q) { return ch.rec[seg_w[q]]; });
          }
#pragma unroll
          for (int i = 0; i < SEG_PER_THREAD; ++i)
            if (jj[i] >= 0) set_bit(jj[i]);
          __syncthreads();
          word_ranks();
#pragma unroll
          for (int i = 0; i < SEG_PER_THREAD; ++i)
            if (jj[i] >= 0) add_at_rank(jj[i], vv[i]);
        } else {
          // two passes over runs of the window's terms (one with a kept
          // bitmap); the row's state stays
          if (cached >= 0) {
            load_bits();
            word_ranks();
          }
          for (int pass = cached >= 0 ? 1 : 0; pass < 2; ++pass) {
            for (int32_t r0 = 0; r0 < total; r0 += RUN) {
              const int rn = (int)((total - r0) < RUN ? (total - r0) : RUN);
              const int per = wave_share(rn, WIN_BLOCK / WAVE);
              const int wlo = wi * per;
              const int wlen = min(per, rn - wlo);
              if (wlen <= 0) continue;
              const int base = (int)r0 + wlo;
              auto terms = [&](auto rec_of) {
                for (int q0 = lane; q0 < wlen; q0 += WAVE * WIN_UNROLL) {
                  if (!pass) {
                    // presence bits, with no branch per term: a term past the
                    // share repeats the lane's first one and sets nothing
                    int32_t pp[WIN_UNROLL];
                    bool ok[WIN_UNROLL];
#pragma unroll
                    for (int u = 0; u < WIN_UNROLL; ++u) {
                      const int q = q0 + u * WAVE;
                      ok[u] = q < wlen;
                      const int qc = ok[u] ? q : q0;
                      pp[u] = (int32_t)rec_of(qc).shift + base + qc;
                    }
                    int jb[WIN_UNROLL];
#pragma unroll
                    for (int u = 0; u < WIN_UNROLL; ++u) jb[u] = op.bcol[pp[u]];
#pragma unroll
                    for (int u = 0; u < WIN_UNROLL; ++u) set_bit_if(jb[u], ok[u]);
                    continue;
                  }
                  if (fx_scale != 0.f) {
                    // fixed-point adds, with no branch per term either
                    int32_t pp[WIN_UNROLL];
                    float am[WIN_UNROLL];
                    bool ok[WIN_UNROLL];
#pragma unroll
                    for (int u = 0; u < WIN_UNROLL; ++u) {
                      const int q = q0 + u * WAVE;
                      ok[u] = q < wlen;
                      const int qc = ok[u] ? q : q0;
                      const typename CH::Rec rc = rec_of(qc);
                      pp[u] = (int32_t)rc.shift + base + qc;
                      am[u] = rc.av;
                    }
                    int jb[WIN_UNROLL];
                    float bb[WIN_UNROLL];
#pragma unroll
                    for (int u = 0; u < WIN_UNROLL; ++u) {
                      jb[u] = op.bcol[pp[u]];
                      bb[u] = op.bval[pp[u]];
                    }
#pragma unroll
                    for (int u = 0; u < WIN_UNROLL; ++u) add_fixed_if(jb[u], am[u] * bb[u], ok[u]);
                    continue;
                  }
                  int32_t pos[WIN_UNROLL];
                  float am[WIN_UNROLL];
#pragma unroll
                  for (int u = 0; u < WIN_UNROLL; ++u) {
                    const int q = q0 + u * WAVE;
                    pos[u] = -1;
                    am[u] = 0.f;
                    if (q < wlen) {
                      const typename CH::Rec rc = rec_of(q);
                      pos[u] = (int32_t)rc.shift + base + q;
                      am[u] = rc.av;
                    }
                  }
                  int jv[WIN_UNROLL];
                  float bv2[WIN_UNROLL];
#pragma unroll
                  for (int u = 0; u < WIN_UNROLL; ++u) {
                    jv[u] = 0;
                    bv2[u] = 0.f;
                    if (pos[u] >= 0) {
                      jv[u] = op.bcol[pos[u]];
                      if (pass) bv2[u] = op.bval[pos[u]];
                    }
                  }
#pragma unroll
                  for (int u = 0; u < WIN_UNROLL; ++u) {
                    if (pos[u] < 0) continue;
                    if (pass) add_at_rank(jv[u], am[u] * bv2[u]);
                    else set_bit(jv[u]);
                  }
                }
              };
              const int one = wave_seg_map(ch.ex, nk, base, wlen, seg_w);
              if (one >= 0) {
                const typename CH::Rec r1 = ch.rec[one];
                terms([&](int) { return r1; });
              } else {
                terms([&](int q) { return ch.rec[seg_w[q]]; });
              }
            }
            __syncthreads();
            if (pass == 0) word_ranks();
          }
        }
        cur = hi;
        prev_g1 = g1;
      } else {
        // long row: pass 1 presence bitmap, pass 2 add at the ranks
        const GrainRange seg{op.bidx, op.nG + 1, g0, g1};
        if (cached >= 0)
          load_bits();
        else
          for_each_term<RA, WIN_BLOCK, WIN_BLOCK, false, true, WIN_UNROLL, true>(
              op, g, ch, row, seg,
              [&](const int (&j)[WIN_UNROLL], const float (&)[WIN_UNROLL], const bool (&ok)[WIN_UNROLL]) {
#pragma unroll
                for (int u = 0; u < WIN_UNROLL; ++u) set_bit_if(j[u], ok[u]);
              });
        word_ranks();
        if (fx_scale != 0.f)
          for_each_term<RA, WIN_BLOCK, WIN_BLOCK, true, true, WIN_UNROLL, true>(
              op, g, ch, row, seg,
              [&](const int (&j)[WIN_UNROLL], const float (&v)[WIN_UNROLL], const bool (&ok)[WIN_UNROLL]) {
#pragma unroll
                for (int u = 0; u < WIN_UNROLL; ++u) add_fixed_if(j[u], v[u], ok[u]);
              });
        else
          for_each_term<RA, WIN_BLOCK, WIN_BLOCK, true, true, WIN_UNROLL>(op, g, ch, row, seg,
                                                              [&](int j, float v) { add_at_rank(j, v); });
      }
      __syncthreads();
      // Output, each wavefront on its own share of the bitmap words and so on
      // its own range of ranks (no workgroup barrier): the values out
      // (coalesced); then those value slots take the column ids, written at
      // their ranks from the words (a lane per word), and go out coalesced
      // too, so that C's column array is written in whole lines rather than
      // an entry at a time from the add loops.  A wavefront's LDS operations
      // complete in order, so the slots are read before they are rewritten.
      {
        const int lane = lane_id();
        const int r0 = min((int)wr0, n), r1 = min((int)wr1, n);
        if (fx_inv != 0.f) {
          const int32_t* iv = reinterpret_cast<const int32_t*>(vals);
          for (int kk = r0 + lane; kk < r1; kk += WAVE) store_stream(&out.cval[base + kk], (float)iv[kk] * fx_inv);
        } else {
          for (int kk = r0 + lane; kk < r1; kk += WAVE) store_stream(&out.cval[base + kk], vals[kk]);
        }
        wave_sync();
        int32_t* cid = reinterpret_cast<int32_t*>(vals);
        for (int w = wa0 + lane; w < wa1; w += WAVE) {
          const uint64_t e = bw[w];
          uint64_t b = e & BITS;
          if (!b) continue;  // an empty word holds no rank either
          int r = (int)(e >> WIN_WORD_BITS);
          const int cw = c0 + w * WIN_WORD_BITS;
          do {
            if (r < n) cid[r] = cw + __builtin_ctzll(b);
            ++r;
            b &= b - 1u;
          } while (b);
          bw[w] = 0u;  // ranks too: the next window's values may lie here
        }
        wave_sync();
        for (int kk = r0 + lane; kk < r1; kk += WAVE) {
          store_stream(&out.ccol[base + kk], cid[kk]);
          cid[kk] = 0;  // +0.0f and integer 0 alike: the slots are clear for the next window
        }
      }
    }
  }
}

// ------------------------------------------------------------ window index

// bidx[k*(nwin+1) + g] = first position p of B_k with bcol[p] >= g*W (or
// the row end), for grains g in [0, nwin]; W is the grain width.  A B row's
// entries are contiguous, so the lookups of one k for successive windows
// share cache lines.  One wavefront per B row, a lane per grain, each a
// binary search over the row's sorted columns: the row's index entries are
// written by consecutive lanes.
template <typename RB>
__global__ __launch_bounds__(256) void k_window_index(const void* brp, const int32_t* bcol, const float* bval,
                                                      int64_t K, int32_t W, int32_t nwin,
                                                      int32_t* bidx, float* bmax) {
  const int64_t nw = (int64_t)gridDim.x * (blockDim.x / WAVE);
  for (int64_t k = (int64_t)blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE; k < K; k += nw) {
    const int64_t s = ld_rp<RB>(brp, k), e = ld_rp<RB>(brp, k + 1);
    // max_j |b_kj|: the bits of non-negative floats order as their values,
    // and a NaN's above all of them, so a NaN in the row gives a NaN
    uint32_t mx = 0u;
    for (int64_t q = s + lane_id(); q < e; q += WAVE) mx = max(mx, __float_as_uint(fabsf(bval[q])));
    mx = wave_last(wave_scan_op<false>(mx));
    if (lane_id() == 0) bmax[k] = __uint_as_float(mx);
    for (int w = lane_id(); w <= nwin; w += WAVE) {
      const int64_t c = (int64_t)w * W;  // the grain's first column
      int64_t lo = s, hi = e;
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (bcol[mid] < c)
          lo = mid + 1;
        else
          hi = mid;
      }
      bidx[k * (nwin + 1) + w] = (int32_t)lo;
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

template <typename RA, typename RB, int GROUP, int BLOCK, bool NUM>
hipError_t launch_dense(const Operands& op, const BinView& bv, const Outputs& out, int64_t ub_rows,
                        hipStream_t s) {
  auto kern = k_dense<RA, RB, GROUP, BLOCK, NUM>;
  const size_t lds = (BLOCK / GROUP) * dense_group_bytes<GROUP, NUM, RB>((int)op.N);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t grid = grid_for(kern, BLOCK, lds, BLOCK / GROUP, ub_rows);
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
      return launch_dense<RA, RB, 64, 256, NUM>(op, bv, out, ub_rows, s);
    case KIND_DENSE_BLOCK:
      return launch_dense<RA, RB, 512, 512, NUM>(op, bv, out, ub_rows, s);
    case KIND_HASH_128:
      return launch_hash<RA, RB, 128, 64, 256, NUM>(op, bv, out, ub_rows, s);
    case KIND_HASH_1024:
      return launch_hash<RA, RB, 1024, 64, 256, NUM>(op, bv, out, ub_rows, s);
    case KIND_HASH_4096:
      return launch_hash<RA, RB, 4096, 256, 256, NUM>(op, bv, out, ub_rows, s);
    case KIND_HASH_8192:
      return launch_hash<RA, RB, 8192, 512, 512, NUM>(op, bv, out, ub_rows, s);
    default:
      return hipErrorInvalidValue;
  }
}

template <typename RA, typename RB, bool NUM>
hipError_t split_t(const Operands& op, const BinView& bv, const SplitWs& sw, const Outputs& out,
                   int64_t ub_rows, hipStream_t s) {
  const int64_t cap_rows = std::min<int64_t>(ub_rows, sw.cap);
  int64_t cg = (cap_rows * (((op.N + 31) / 32) + (NUM ? op.N : 0)) + 255) / 256;
  if (cg > 4096) cg = 4096;
  if (cg < 1) cg = 1;
  hipLaunchKernelGGL(k_split_clear, dim3((unsigned)cg), dim3(256), 0, s, bv, sw, (int32_t)op.N, NUM ? 1 : 0);
  auto kern = k_split_parts<RA, RB, NUM>;
  const size_t lds = dense_group_bytes<SPLIT_BLOCK, NUM, RB>((int)op.N);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t grid = grid_for(kern, SPLIT_BLOCK, lds, 1, cap_rows * SPLIT_PARTS);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(SPLIT_BLOCK), lds, s, op, bv, sw);
  int64_t fg = (cap_rows + 3) / 4;
  if (fg > 8192) fg = 8192;
  if (fg < 1) fg = 1;
  hipLaunchKernelGGL((k_split_finish<NUM>), dim3((unsigned)fg), dim3(256), 0, s, bv, sw, (int32_t)op.N, out);
  // rows of the bin beyond the slots: one workgroup each
  if (ub_rows > sw.cap) {
    BinView rest = bv;
    rest.skip = (int32_t)sw.cap;
    hipError_t e = launch_dense<RA, RB, 512, 512, NUM>(op, rest, out, ub_rows - sw.cap, s);
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

template <typename RA, typename RB>
hipError_t split_rp(int phase, const Operands& op, const BinView& bv, const SplitWs& sw, const Outputs& out,
                    int64_t ub_rows, hipStream_t s) {
  return phase ? split_t<RA, RB, true>(op, bv, sw, out, ub_rows, s) : split_t<RA, RB, false>(op, bv, sw, out, ub_rows, s);
}

template <typename RA, typename RB>
hipError_t run_bin_rp(int kind, int phase, const Operands& op, const BinView& bv, const Outputs& out,
                      int64_t ub_rows, hipStream_t s) {
  return phase ? run_bin_t<RA, RB, true>(kind, op, bv, out, ub_rows, s)
               : run_bin_t<RA, RB, false>(kind, op, bv, out, ub_rows, s);
}

template <typename RA, typename RB>
hipError_t win_symbolic_t(const Operands& op, const BinView& bv, const WindowParams& wp,
                          const Outputs& out, int64_t ub_rows, hipStream_t s) {
  auto kern = k_grain_count<RA, RB>;
  const size_t lds = count_lds_bytes<RB>(wp.grains_per_count_item, op.G);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipError_t ez = hipMemsetAsync(wp.row_counter, 0, sizeof(int32_t), s);
  if (ez != hipSuccess) return ez;
  const int64_t grid = grid_for(kern, WIN_BLOCK, lds, 1, ub_rows);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(WIN_BLOCK), lds, s, op, bv, wp);
  int64_t pg = (ub_rows + 255) / 256;
  if (pg > 8192) pg = 8192;
  hipLaunchKernelGGL(k_win_plan, dim3((unsigned)pg), dim3(256), 0, s, bv, op.nG, op.G, wp, out.counts);
  return hipGetLastError();
}

template <typename RA, typename RB>
hipError_t win_numeric_t(const Operands& op, const BinView& bv, const WindowParams& wp,
                         const Outputs& out, int64_t ub_rows, int64_t nitems, hipStream_t s) {
  int64_t pg = (ub_rows + 255) / 256;
  if (pg > 8192) pg = 8192;
  hipLaunchKernelGGL(k_win_fill, dim3((unsigned)pg), dim3(256), 0, s, bv, op.nG, op.G, wp);
  if (nitems <= 0) return hipGetLastError();
  hipError_t ez = hipMemsetAsync(wp.row_counter, 0, sizeof(int32_t) * (1 + WIN_MAX_SLABS), s);
  if (ez != hipSuccess) return ez;
  auto kern = k_win_rows<RA, RB>;
  const size_t lds = window_lds_bytes<RB>(wp.pool_words);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t grid = grid_for(kern, WIN_BLOCK, lds, 1, ub_rows);
  WindowParams wq = wp;
  wq.nslab = (int32_t)(grid < WIN_MAX_SLABS ? grid : WIN_MAX_SLABS);  // every slab has a workgroup
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(WIN_BLOCK), lds, s, op, bv, wq, out);
  return hipGetLastError();
}

}  // namespace

// ------------------------------------------------------------- host entry

#define AIRES_DISPATCH_RP(op, FN, ...)                                                      \
  ((op).rpa64 ? ((op).rpb64 ? FN<int64_t, int64_t>(__VA_ARGS__) : FN<int64_t, int32_t>(__VA_ARGS__)) \
              : ((op).rpb64 ? FN<int32_t, int64_t>(__VA_ARGS__) : FN<int32_t, int32_t>(__VA_ARGS__)))

template <typename RA, typename RB>
static hipError_t analyze_t(const Operands& op, int64_t nrows, int64_t* P, unsigned long long* total,
                            int32_t* long_cnt, int32_t* long_list, hipStream_t s) {
  int64_t grid = (nrows * 16 + 255) / 256;
  if (grid > 8192) grid = 8192;
  hipLaunchKernelGGL((k_analyze<RA, RB>), dim3((unsigned)grid), dim3(256), 0, s, op, nrows, P, total, long_cnt,
                     long_list);
  int64_t lg = nrows / 64 + 1;
  if (lg > 2048) lg = 2048;
  hipLaunchKernelGGL((k_analyze_long<RA, RB>), dim3((unsigned)lg), dim3(1024), 0, s, op, P, total, long_cnt,
                     long_list);
  return hipGetLastError();
}

hipError_t analyze(const Operands& op, int64_t nrows, int64_t* P, unsigned long long* total,
                   int32_t* long_cnt, int32_t* long_list, hipStream_t s) {
  if (nrows <= 0) return hipSuccess;
  return AIRES_DISPATCH_RP(op, analyze_t, op, nrows, P, total, long_cnt, long_list, s);
}

hipError_t bin_rows(const int64_t* P, int64_t nrows, const BinThresholds& th, int32_t* cnt_cursor,
                    int32_t* binoff, int32_t* list, hipStream_t s) {
  int64_t grid = nrows > 0 ? (nrows + 255) / 256 : 1;
  if (grid > 2048) grid = 2048;
  hipLaunchKernelGGL(k_bin_count, dim3((unsigned)grid), dim3(256), 0, s, P, nrows, th, cnt_cursor);
  hipLaunchKernelGGL(k_bin_scatter, dim3((unsigned)grid), dim3(256), 0, s, P, nrows, th, cnt_cursor,
                     cnt_cursor + MAX_BINS, binoff, list);
  return hipGetLastError();
}

hipError_t run_bin(int kind, int phase, const Operands& op, const BinView& bv, const Outputs& out,
                   int64_t ub_rows, hipStream_t s) {
  if (ub_rows <= 0) return hipSuccess;
  return AIRES_DISPATCH_RP(op, run_bin_rp, kind, phase, op, bv, out, ub_rows, s);
}

hipError_t split_rows(int phase, const Operands& op, const BinView& bv, const SplitWs& sw, const Outputs& out,
                      int64_t ub_rows, hipStream_t s) {
  if (ub_rows <= 0) return hipSuccess;
  return AIRES_DISPATCH_RP(op, split_rp, phase, op, bv, sw, out, ub_rows, s);
}

hipError_t windows_symbolic(const Operands& op, const BinView& bv, const WindowParams& wp, const Outputs& out,
                            int64_t ub_rows, hipStream_t s) {
  if (ub_rows <= 0) return hipSuccess;
  return AIRES_DISPATCH_RP(op, win_symbolic_t, op, bv, wp, out, ub_rows, s);
}

hipError_t windows_numeric(const Operands& op, const BinView& bv, const WindowParams& wp, const Outputs& out,
                           int64_t ub_rows, int64_t nitems, hipStream_t s) {
  if (ub_rows <= 0) return hipSuccess;
  return AIRES_DISPATCH_RP(op, win_numeric_t, op, bv, wp, out, ub_rows, nitems, s);
}

hipError_t build_window_index(const void* brp, int rpb64, const int32_t* bcol, const float* bval, int64_t K,
                              int32_t G, int32_t nG, int32_t* bidx, float* bmax, hipStream_t s) {
  if (K <= 0) return hipSuccess;
  int64_t grid = (K + 3) / 4;
  if (grid > 65536) grid = 65536;
  if (rpb64)
    hipLaunchKernelGGL((k_window_index<int64_t>), dim3((unsigned)grid), dim3(256), 0, s, brp, bcol, bval, K, G, nG,
                       bidx, bmax);
  else
    hipLaunchKernelGGL((k_window_index<int32_t>), dim3((unsigned)grid), dim3(256), 0, s, brp, bcol, bval, K, G, nG,
                       bidx, bmax);
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
      return 4 * (phase ? dense_group_bytes<64, true, int64_t>(W) : dense_group_bytes<64, false, int64_t>(W));
    case KIND_DENSE_BLOCK:
    case KIND_DENSE_SPLIT:
      return phase ? dense_group_bytes<512, true, int64_t>(W) : dense_group_bytes<512, false, int64_t>(W);
    case KIND_HASH_128: return 4 * sizeof(HashLds<128, 64, true, int64_t>);
    case KIND_HASH_1024: return 4 * sizeof(HashLds<1024, 64, true, int64_t>);
    case KIND_HASH_4096: return sizeof(HashLds<4096, 256, true, int64_t>);
    case KIND_HASH_8192: return sizeof(HashLds<8192, 512, true, int64_t>);
    default: return 0;
  }
}

size_t grain_count_lds(int sg, int G) { return count_lds_bytes<int64_t>(sg, G); }
size_t window_numeric_lds(int pool_words) {
  return window_lds_bytes<int64_t>(pool_words);
}

int group_size(int kind) {
  switch (kind) {
    case KIND_DENSE_BLOCK: return 512;
    case KIND_DENSE_SPLIT: return SPLIT_BLOCK;
    case KIND_HASH_4096: return 256;
    case KIND_HASH_8192: return 512;
    case KIND_WINDOWS: return WIN_BLOCK;
    default: return 64;
  }
}

}  // namespace kern
}  // namespace aires
