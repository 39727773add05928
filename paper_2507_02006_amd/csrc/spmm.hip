// Sparse-times-dense product Y = act(A * W) on gfx950: the combination step
// of a GCN layer (Sec. II-A, Eq. 3: the aggregated features times the
// layer's weights, then the activation) and, with a dense feature matrix,
// the aggregation of Eq. 1.  A is CSR (32- or 64-bit row pointers), W and
// Y are dense row-major with leading dimensions ldw and ldy.
//
// Rows with at most kHeavy entries take one wavefront: lane l owns V
// consecutive columns of a 64*V-column block, the row's (k, a_ik) pairs are
// read 64 at a time (a lane each) and broadcast with readlane, and several
// rows of W are in flight at a time.  Longer rows
// take a 256-thread workgroup whose four wavefronts split the entries and
// add their partial rows in LDS.  The activation is applied before the
// store; every element of Y is written exactly once.
#include "kernels.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aires {
namespace kern {
namespace {

constexpr int WAVE = 64;
constexpr int SPMM_BLOCK = 256;  // four wavefronts
constexpr int64_t kHeavy = 512;  // longer rows are split over a workgroup

template <typename RP>
__device__ __forceinline__ int64_t rp_at(const void* rp, int64_t i) {
  return (int64_t) static_cast<const RP*>(rp)[i];
}

// V columns of W row k from column c, as one vector load when VEC.
template <int V, bool VEC>
__device__ __forceinline__ void load_w(const float* wr, int c, int F, float (&w)[V]) {
  if constexpr (VEC && V == 8) {
    if (c + V <= F) {
      const float4 a = *reinterpret_cast<const float4*>(wr + c);
      const float4 b = *reinterpret_cast<const float4*>(wr + c + 4);
      w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
      w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
      return;
    }
  } else if constexpr (VEC && V == 4) {
    if (c + V <= F) {
      const float4 a = *reinterpret_cast<const float4*>(wr + c);
      w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
      return;
    }
  } else if constexpr (VEC && V == 2) {
    if (c + V <= F) {
      const float2 a = *reinterpret_cast<const float2*>(wr + c);
      w[0] = a.x; w[1] = a.y;
      return;
    }
  }
#pragma unroll
  for (int v = 0; v < V; ++v) w[v] = c + v < F ? wr[c + v] : 0.f;
}

// acc += a_ik * W[k, c .. c+V) over the entries [p0, p1).  The entries
// come in 64 at a time, one per lane (a coalesced load), and are handed to
// the whole wavefront with readlane, so that U rows of W are in flight per
// step with no scalar load on the path.
template <int V, bool VEC>
__device__ __forceinline__ void row_block(const int32_t* acol, const float* aval, int64_t p0, int64_t p1,
                                          const float* W, int64_t ldw, int c, int F, float (&acc)[V]) {
  constexpr int U = V <= 2 ? 8 : 4;
  const int lane = threadIdx.x % WAVE;
  for (int64_t pb = p0; pb < p1; pb += WAVE) {
    const int cnt = (int)(p1 - pb < WAVE ? p1 - pb : WAVE);
    int kl = 0;
    float al = 0.f;
    if (lane < cnt) {
      kl = acol[pb + lane];
      al = aval[pb + lane];
    }
    int j = 0;
    for (; j + U <= cnt; j += U) {
      float w[U][V];
#pragma unroll
      for (int u = 0; u < U; ++u)
        load_w<V, VEC>(W + (int64_t)__builtin_amdgcn_readlane(kl, j + u) * ldw, c, F, w[u]);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(al), j + u));
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] = fmaf(a, w[u][v], acc[v]);
      }
    }
    for (; j < cnt; ++j) {
      float w[V];
      load_w<V, VEC>(W + (int64_t)__builtin_amdgcn_readlane(kl, j) * ldw, c, F, w);
      const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(al), j));
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = fmaf(a, w[v], acc[v]);
    }
  }
}

template <int V, bool RELU>
__device__ __forceinline__ void store_row(float* yr, int c, int F, const float (&acc)[V]) {
#pragma unroll
  for (int v = 0; v < V; ++v)
    if (c + v < F) yr[c + v] = RELU ? fmaxf(acc[v], 0.f) : acc[v];
}

template <typename RP, int V, bool VEC, bool RELU>
__global__ __launch_bounds__(SPMM_BLOCK) void k_spmm_rows(const void* arp, const int32_t* acol, const float* aval,
                                                           int64_t m, const float* W, int64_t ldw, int F, float* Y,
                                                           int64_t ldy) {
  const int lane = threadIdx.x % WAVE;
  const int64_t nw = (int64_t)gridDim.x * (SPMM_BLOCK / WAVE);
  for (int64_t row = (int64_t)blockIdx.x * (SPMM_BLOCK / WAVE) + threadIdx.x / WAVE; row < m; row += nw) {
    const int64_t p0 = rp_at<RP>(arp, row), p1 = rp_at<RP>(arp, row + 1);
    if (p1 - p0 > kHeavy) continue;  // a workgroup takes it
    for (int cb = 0; cb < F; cb += WAVE * V) {
      const int c = cb + lane * V;
      float acc[V];
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = 0.f;
      row_block<V, VEC>(acol, aval, p0, p1, W, ldw, c, F, acc);
      store_row<V, RELU>(Y + row * ldy, c, F, acc);
    }
  }
}

template <typename RP, int V, bool VEC, bool RELU>
__global__ __launch_bounds__(SPMM_BLOCK) void k_spmm_heavy(const void* arp, const int32_t* acol, const float* aval,
                                                            int64_t m, const float* W, int64_t ldw, int F, float* Y,
                                                            int64_t ldy) {
  constexpr int NWV = SPMM_BLOCK / WAVE;
  __shared__ float part[NWV - 1][WAVE * V];
  const int lane = threadIdx.x % WAVE, wv = threadIdx.x / WAVE;
  for (int64_t row = blockIdx.x; row < m; row += gridDim.x) {
    const int64_t p0 = rp_at<RP>(arp, row), p1 = rp_at<RP>(arp, row + 1);
    if (p1 - p0 <= kHeavy) continue;  // uniform over the workgroup
    const int64_t len = (p1 - p0 + NWV - 1) / NWV;
    const int64_t q0 = p0 + wv * len < p1 ? p0 + wv * len : p1;
    const int64_t q1 = q0 + len < p1 ? q0 + len : p1;
    for (int cb = 0; cb < F; cb += WAVE * V) {
      const int c = cb + lane * V;
      float acc[V];
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = 0.f;
      row_block<V, VEC>(acol, aval, q0, q1, W, ldw, c, F, acc);
      if (wv > 0) {
#pragma unroll
        for (int v = 0; v < V; ++v) part[wv - 1][lane * V + v] = acc[v];
      }
      __syncthreads();
      if (wv == 0) {
#pragma unroll
        for (int i = 0; i < NWV - 1; ++i)
#pragma unroll
          for (int v = 0; v < V; ++v) acc[v] += part[i][lane * V + v];
        store_row<V, RELU>(Y + row * ldy, c, F, acc);
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// Dense tiles on the matrix cores.  When A is dense enough (the aggregated
// features of Eq. 3 typically are), reading one row of W per entry of A
// costs more than a dense product over the zeros: a workgroup takes a
// 64-row x 16*NT-column tile of Y, densifies A's rows 32 columns at a time
// into LDS, stages the matching 32 x 16*NT block of W (transposed, k
// contiguous), and accumulates with v_mfma_f32_32x32x2_f32 (it sustains a
// larger share of the fp32 matrix peak than the 16x16x4 form).  Each
// wavefront owns 32 rows and 8*NT columns (NT/4 blocks of 32) of the tile.
//
// k order: for an 8-wide block of k, lane l (h = l / 32, c = l % 32) reads
// k = 4h .. 4h+3 of its row (A) and of its column (W) as one 16-byte LDS
// load, and the four MFMA steps take those four k's in turn, so every
// product a_ik w_kj meets its partner in the same step.  Absent entries are
// zeros in the tile, and x + 0 * w = x exactly for finite w, so each
// element is still a sum of the row's own products.
//
// Pipeline: LDS holds two chunks.  While the wavefronts multiply chunk c
// from one buffer they write chunk c+1 (loaded during chunk c-1) into the
// other and issue the loads of chunk c+2, so one barrier per chunk
// suffices and the staging work interleaves with the MFMAs.  Every load
// goes through a buffer resource: out-of-range offsets read 0 without
// touching memory, so the loop body has no branches.
constexpr int DT_M = 64;        // rows per tile
constexpr int DT_K = 32;        // k per LDS chunk
constexpr int DT_BLOCK = 256;   // four wavefronts, 16 rows each
constexpr int DT_ENTRIES = DT_K / 4;  // four threads per row: one round of loads covers a chunk
constexpr int NXCD = 8;         // gfx950 hands workgroups round-robin to its 8 XCDs
constexpr int kOutOfRange = INT32_MIN;  // a buffer offset no resource here reaches (reads 0)

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Row layout of a tile chunk in LDS (element k of row r, DT_K per row).
// Padded: rows of DT_K + 4 floats, so the 16-byte operand reads of 16 rows
// fall on distinct banks; column DT_K of each row takes the entries of later
// chunks.  Swizzled (less LDS, used where it buys one more workgroup per
// CU): unpadded rows whose 16-byte groups are permuted by the row's low
// three bits, so eight consecutive rows' reads of one group fall on
// distinct banks; one dump slot per row after the rows.
template <bool SWZ>
struct TileLayout {
  static constexpr int S = SWZ ? DT_K : DT_K + 4;                // floats per row
  static constexpr int A_FLOATS = SWZ ? DT_M * DT_K + DT_M : DT_M * S;
  __device__ static __forceinline__ int at(int r, int k) {
    if constexpr (SWZ) return r * DT_K + ((((k >> 2) ^ (r & 7)) << 2) | (k & 3));
    else return r * S + k;
  }
  __device__ static __forceinline__ int dump(int r) { return SWZ ? DT_M * DT_K + r : r * S + DT_K; }
};

// a wavefront-uniform 64-bit value in scalar registers
__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// raw buffer over `bytes` bytes (gfx9 resource word 3: 32-bit data format)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Occupancy is LDS-bound (two chunks per workgroup): four workgroups per CU
// at NT = 4, three at NT = 8; the register budget is set to match.
template <typename RP, int NT, bool VEC, bool RELU>
__global__ __launch_bounds__(DT_BLOCK, NT > 4 ? 3 : 4) void k_spmm_dense(
    const void* arp, const int32_t* acol, const float* aval, int64_t m, int K, const float* W, int64_t ldw, int F,
    float* Y, int64_t ldy, int64_t nrt, int64_t nct, int64_t ntiles) {
  constexpr int BN = 16 * NT;
  constexpr int WL = NT / 2;  // 16-byte W loads per thread per chunk (32 x BN floats over 256 threads)
  using L = TileLayout<(NT > 4)>;
  __shared__ __align__(16) float As[2][L::A_FLOATS];  // [row][k]
  __shared__ __align__(16) float Wt[2][BN * L::S];    // [column][k]
  constexpr int NB = BN / 64;  // 32-column MFMA blocks per wavefront
  const int t = threadIdx.x, lane = t % WAVE, wv = t / WAVE;
  const int r = t / 4, q = t % 4;             // densify: four threads per row
  const int h = lane / 32, c = lane % 32;     // MFMA operand position
  const int mr = 32 * (wv >> 1), mc = (wv & 1) * (BN / 2);  // the wavefront's rows and columns
  // W staging: the thread takes row wk of the chunk and, for e < WL, the
  // columns wc + 16e .. +3; a row's 64 bytes come from four lanes, and the
  // transposed LDS stores of a wavefront hit 64 distinct banks.
  const int wk = lane % 16 + 16 * (wv & 1);
  const int wc = (wv >> 1) * (BN / 2) + 4 * (lane / 16);
  const int nch = (K + DT_K - 1) / DT_K;
  // The grid is a multiple of 8 blocks, so a block's tiles all have its
  // index mod 8 and stay on its XCD; the column tiles of one row tile are
  // consecutive there and share A's entries through that XCD's L2.
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t x = tile % NXCD, i = tile / NXCD;
    const int64_t rt = (i / nct) * NXCD + x, ct = i % nct;
    if (rt >= nrt) continue;  // uniform over the workgroup
    const int64_t row0 = rt * DT_M;
    const int n0 = (int)ct * BN;
    // A's entries of the tile (< 2^26 of them: K <= 2^20), positions relative to e0
    const int64_t e0 = uniform64(rp_at<RP>(arp, row0));
    const int64_t e1 = uniform64(rp_at<RP>(arp, row0 + DT_M < m ? row0 + DT_M : m));
    const __amdgpu_buffer_rsrc_t rc = make_rsrc(acol + e0, 4 * (e1 - e0));
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(aval + e0, 4 * (e1 - e0));
    // the row's entries as tile-local positions [cur, p1)
    int cur = 0, p1 = 0;
    if (row0 + r < m) {
      cur = (int)(rp_at<RP>(arp, row0 + r) - e0);
      p1 = (int)(rp_at<RP>(arp, row0 + r + 1) - e0);
    }
    int kc[DT_ENTRIES];
    float kv[DT_ENTRIES];
    int nval = 0;  // kc[e] belongs to the row while 4e < nval
    f32x4 w[WL];
    // the row's next 32 entries; nothing here waits for the loads
    auto load_entries = [&]() {
      nval = p1 - cur - q;  // entries of the row at or after this thread's first
      const int off = 4 * (cur + q);
#pragma unroll
      for (int e = 0; e < DT_ENTRIES; ++e) {
        kc[e] = __builtin_amdgcn_raw_buffer_load_b32(rc, off + 16 * e, 0, 0);
        kv[e] = __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(rv, off + 16 * e, 0, 0));
      }
    };
    // this thread's share of rows k0 .. k0+32 of W[:, n0 .. n0+BN): rows
    // past K are outside the resource, columns past F get an out-of-range
    // offset, so both read as zeros (F <= ldw < 2^23 keeps offsets in int)
    auto load_w = [&](int k0) {
      const int rows = K - k0 < DT_K ? (K - k0 > 0 ? K - k0 : 0) : DT_K;
      const __amdgpu_buffer_rsrc_t rw = make_rsrc(W + (int64_t)k0 * ldw + n0, 4 * (int64_t)rows * ldw);
#pragma unroll
      for (int e = 0; e < WL; ++e) {
        const int n = wc + 16 * e;  // column within the tile
        const int base = 4 * (wk * (int)ldw + n);
        if constexpr (VEC) {
          // n0 + n, F and ldw are multiples of 4: the 16 bytes are all
          // columns below F or all past it
          w[e] = __builtin_bit_cast(
              f32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, n0 + n < F ? base : kOutOfRange, 0, 0));
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            w[e][u] = __int_as_float(
                __builtin_amdgcn_raw_buffer_load_b32(rw, n0 + n + u < F ? base + 4 * u : kOutOfRange, 0, 0));
        }
      }
    };
    // chunk k0 from the registers into LDS buffer b
    auto write_chunk = [&](int b, int k0) {
      // zero this thread's quarter of its row; the scatter below runs in the
      // same wavefront after it, and LDS executes a wavefront's accesses in order
#pragma unroll
      for (int e = 0; e < DT_K / 16; ++e)
        *reinterpret_cast<f32x4*>(&As[b][L::at(r, q * (DT_K / 4) + 4 * e)]) = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int e = 0; e < WL; ++e)
#pragma unroll
        for (int u = 0; u < 4; ++u) Wt[b][L::at(wc + 16 * e + u, wk)] = w[e][u];
      // 32 entries cover the 32 columns: every entry of the row in the
      // chunk is here.  Each is stored; one of a later chunk lands in the
      // row's dump slot, which the products never read.
      int n_in = 0;
#pragma unroll
      for (int e = 0; e < DT_ENTRIES; ++e) {
        // a canonical row has no column below k0 left, so this is kc < kend
        const bool in = 4 * e < nval && (unsigned)(kc[e] - k0) < (unsigned)DT_K;
        As[b][in ? L::at(r, kc[e] - k0) : L::dump(r)] = kv[e];
        n_in += in;
      }
      n_in += __shfl_xor(n_in, 1);
      n_in += __shfl_xor(n_in, 2);
      cur += n_in;
    };
    f32x16 acc[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
    if (nch > 0) {
      load_entries();
      load_w(0);
      write_chunk(0, 0);
      load_entries();
      load_w(DT_K);
      __syncthreads();
    }
    for (int ch = 0; ch < nch; ++ch) {
      const int b = ch & 1;
#pragma unroll
      for (int kb = 0; kb < DT_K; kb += 8) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(&As[b][L::at(mr + c, kb + 4 * h)]);
        f32x4 bw[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j)
          bw[j] = *reinterpret_cast<const f32x4*>(&Wt[b][L::at(mc + 32 * j + c, kb + 4 * h)]);
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[s], bw[j][s], acc[j], 0, 0, 0);
      }
      // chunk ch+1 into the other buffer (read last in chunk ch-1, before the
      // barrier), then the loads of chunk ch+2.  Past the last chunk both are
      // harmless: the rows are exhausted and W's rows are out of range.
      write_chunk(b ^ 1, (ch + 1) * DT_K);
      load_entries();
      load_w((ch + 2) * DT_K);
      __syncthreads();
    }
    // register v of block j holds row 8(v/4) + 4h + v%4 of the wavefront's
    // 32, column c of the block
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int col = n0 + mc + 32 * j + c;
      if (col >= F) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t row = row0 + mr + 8 * (v / 4) + 4 * h + v % 4;
        if (row < m) Y[row * ldy + col] = RELU ? fmaxf(acc[j][v], 0.f) : acc[j][v];
      }
    }
  }
}

template <typename RP, int V, bool VEC, bool RELU>
hipError_t spmm_t(const void* arp, const int32_t* acol, const float* aval, int64_t m, const float* W, int64_t ldw,
                  int F, float* Y, int64_t ldy, hipStream_t s) {
  int64_t g1 = (m + SPMM_BLOCK / WAVE - 1) / (SPMM_BLOCK / WAVE);
  if (g1 > 65536) g1 = 65536;
  hipLaunchKernelGGL((k_spmm_rows<RP, V, VEC, RELU>), dim3((unsigned)g1), dim3(SPMM_BLOCK), 0, s, arp, acol, aval,
                     m, W, ldw, F, Y, ldy);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int64_t g2 = m < 2048 ? m : 2048;
  hipLaunchKernelGGL((k_spmm_heavy<RP, V, VEC, RELU>), dim3((unsigned)g2), dim3(SPMM_BLOCK), 0, s, arp, acol, aval,
                     m, W, ldw, F, Y, ldy);
  return hipGetLastError();
}

template <typename RP, int V, bool VEC>
hipError_t spmm_act(int relu, const void* arp, const int32_t* acol, const float* aval, int64_t m, const float* W,
                    int64_t ldw, int F, float* Y, int64_t ldy, hipStream_t s) {
  return relu ? spmm_t<RP, V, VEC, true>(arp, acol, aval, m, W, ldw, F, Y, ldy, s)
              : spmm_t<RP, V, VEC, false>(arp, acol, aval, m, W, ldw, F, Y, ldy, s);
}

template <typename RP>
hipError_t spmm_rp(int relu, const void* arp, const int32_t* acol, const float* aval, int64_t m, const float* W,
                   int64_t ldw, int F, float* Y, int64_t ldy, hipStream_t s) {
  // columns per lane: one 64-lane pass covers up to 512 columns; vector loads
  // when W's rows and the base are aligned to the vector
  const int V = F <= 64 ? 1 : F <= 128 ? 2 : F <= 256 ? 4 : 8;
  const bool vec = V > 1 && ldw % V == 0 && (reinterpret_cast<uintptr_t>(W) % (4 * V)) == 0;
  switch (V) {
    case 1: return spmm_act<RP, 1, false>(relu, arp, acol, aval, m, W, ldw, F, Y, ldy, s);
    case 2: return vec ? spmm_act<RP, 2, true>(relu, arp, acol, aval, m, W, ldw, F, Y, ldy, s)
                       : spmm_act<RP, 2, false>(relu, arp, acol, aval, m, W, ldw, F, Y, ldy, s);
    case 4: return vec ? spmm_act<RP, 4, true>(relu, arp, acol, aval, m, W, ldw, F, Y, ldy, s)
                       : spmm_act<RP, 4, false>(relu, arp, acol, aval, m, W, ldw, F, Y, ldy, s);
    default: return vec ? spmm_act<RP, 8, true>(relu, arp, acol, aval, m, W, ldw, F, Y, ldy, s)
                        : spmm_act<RP, 8, false>(relu, arp, acol, aval, m, W, ldw, F, Y, ldy, s);
  }
}

template <typename RP, int NT, bool VEC>
hipError_t dense_t(int relu, const void* arp, const int32_t* acol, const float* aval, int64_t m, int K,
                   const float* W, int64_t ldw, int F, float* Y, int64_t ldy, hipStream_t s) {
  const int64_t nrt = (m + DT_M - 1) / DT_M, nct = (F + 16 * NT - 1) / (16 * NT);
  const int64_t ntiles = (nrt + NXCD - 1) / NXCD * NXCD * nct;  // a multiple of NXCD
  const int64_t grid = ntiles < 65536 ? ntiles : 65536;          // so is this
  if (relu)
    hipLaunchKernelGGL((k_spmm_dense<RP, NT, VEC, true>), dim3((unsigned)grid), dim3(DT_BLOCK), 0, s, arp, acol,
                       aval, m, K, W, ldw, F, Y, ldy, nrt, nct, ntiles);
  else
    hipLaunchKernelGGL((k_spmm_dense<RP, NT, VEC, false>), dim3((unsigned)grid), dim3(DT_BLOCK), 0, s, arp, acol,
                       aval, m, K, W, ldw, F, Y, ldy, nrt, nct, ntiles);
  return hipGetLastError();
}

template <typename RP>
hipError_t dense_rp(int relu, const void* arp, const int32_t* acol, const float* aval, int64_t m, int K,
                    const float* W, int64_t ldw, int F, float* Y, int64_t ldy, hipStream_t s) {
  const bool vec = ldw % 4 == 0 && F % 4 == 0 && reinterpret_cast<uintptr_t>(W) % 16 == 0;
  if (F > 64)
    return vec ? dense_t<RP, 8, true>(relu, arp, acol, aval, m, K, W, ldw, F, Y, ldy, s)
               : dense_t<RP, 8, false>(relu, arp, acol, aval, m, K, W, ldw, F, Y, ldy, s);
  return vec ? dense_t<RP, 4, true>(relu, arp, acol, aval, m, K, W, ldw, F, Y, ldy, s)
             : dense_t<RP, 4, false>(relu, arp, acol, aval, m, K, W, ldw, F, Y, ldy, s);
}

}  // namespace

bool spmm_dense_fits(int64_t K, int64_t ldw) {
  return K >= 0 && K <= (int64_t(1) << 20) && ldw < (int64_t(1) << 23);
}

hipError_t spmm(const void* arp, int rpa64, const int32_t* acol, const float* aval, int64_t m, int64_t K,
                const float* W, int64_t ldw, int64_t F, float* Y, int64_t ldy, int relu, int dense, hipStream_t s) {
  if (m <= 0 || F <= 0) return hipSuccess;
  if (dense) {
    if (!spmm_dense_fits(K, ldw)) return hipErrorInvalidValue;
    return rpa64 ? dense_rp<int64_t>(relu, arp, acol, aval, m, (int)K, W, ldw, (int)F, Y, ldy, s)
                 : dense_rp<int32_t>(relu, arp, acol, aval, m, (int)K, W, ldw, (int)F, Y, ldy, s);
  }
  return rpa64 ? spmm_rp<int64_t>(relu, arp, acol, aval, m, W, ldw, (int)F, Y, ldy, s)
               : spmm_rp<int32_t>(relu, arp, acol, aval, m, W, ldw, (int)F, Y, ldy, s);
}

}  // namespace kern
}  // namespace aires
