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

}  // namespace

hipError_t spmm(const void* arp, int rpa64, const int32_t* acol, const float* aval, int64_t m, const float* W,
                int64_t ldw, int64_t F, float* Y, int64_t ldy, int relu, hipStream_t s) {
  if (m <= 0 || F <= 0) return hipSuccess;
  return rpa64 ? spmm_rp<int64_t>(relu, arp, acol, aval, m, W, ldw, (int)F, Y, ldy, s)
               : spmm_rp<int32_t>(relu, arp, acol, aval, m, W, ldw, (int)F, Y, ldy, s);
}

}  // namespace kern
}  // namespace aires
