// Host runtime of the library: the C-ABI of aires.h, the RoBW planner
// (Sec. III-A, Algorithm 1; budget split after Eqs. 5-7), in-core execution
// over device-resident tiles, and the out-of-core streaming schedule
// (Sec. III-B, Algorithm 2).
#include "../../include/aires.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <memory>
#include <string>
#include <thread>
#include <vector>

#include <fcntl.h>
#include <unistd.h>

#include "kernels.h"
#include "scratch.h"

using namespace aires;

namespace {

thread_local std::string g_last_error;

aires_status fail(aires_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

#define HIP_TRY(expr)                                                                 \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return fail(AIRES_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));        \
  } while (0)

#define ST_TRY(expr)                       \
  do {                                     \
    aires_status s_ = (expr);              \
    if (s_ != AIRES_OK) return s_;         \
  } while (0)

constexpr int64_t kDenseWaveMaxN = 2048;     // widest dense row one wavefront holds
constexpr int64_t kDenseMaxCols = 16384;     // widest dense row a workgroup holds
// Wide products: a window's bitmap and values share a pool of LDS sized so
// that a numeric workgroup uses 52 KB and three 512-thread workgroups (24
// wavefronts) share a CU; the grain and entry caps rarely bind. A symbolic
// item's bitmap (grains x columns / 8 bytes) stays at 32 KB so that four
// 512-thread counting workgroups share a CU; wider grains mean fewer grain
// steps per item at the same LDS.
constexpr int64_t kGrainCols = 8192;         // column grain of wide products
constexpr int64_t kWindowMaxGrains = 64;     // grains one window may span
constexpr int64_t kWindowMaxEntries = 16384; // C entries one window may hold
constexpr int64_t kWindowPoolBytes = 38912;  // LDS shared by a window's bitmap and values
constexpr int64_t kCountGrains = 24;         // grains one symbolic item covers (four counting workgroups per CU)
constexpr int64_t kBitmapCacheBytes = int64_t(32) << 30;  // symbolic bitmaps kept for heavy rows
constexpr int64_t kStreamTiles = 16;                       // default tile count of a streamed A
constexpr int64_t kMinStreamTileBytes = int64_t(32) << 20;  // ... with at least this much of A per tile
constexpr int64_t kKeepBitmapProducts = 65536;           // rows above this many products keep them
constexpr int64_t kSlabMinProducts = 262144;             // rows above this many products: column slabs
constexpr int64_t kWaveMaxProducts = 8192;   // rows up to this go to one wavefront
constexpr int64_t kSplitMinProducts = 65536; // narrow rows above this are split over workgroups
constexpr int64_t kSplitWsBytes = int64_t(256) << 20;  // their dense slots
constexpr int64_t kHashMaxProducts = 4096;   // = 8192-slot table at load <= 1/2
constexpr int64_t kFixedWorkspace = 4 << 20; // scan partials, counters, slack

int64_t rp_bytes(const aires_csr& M) { return M.rp_type == AIRES_IDX_I64 ? 8 : 4; }
int64_t csr_bytes(const aires_csr& M) { return (M.nrows + 1) * rp_bytes(M) + 8 * M.nnz; }

int64_t host_rp(const aires_csr& M, int64_t i) {
  return M.rp_type == AIRES_IDX_I64 ? static_cast<const int64_t*>(M.row_ptr)[i]
                                    : (int64_t) static_cast<const int32_t*>(M.row_ptr)[i];
}

// --------------------------------------------------------------- allocator

void* default_alloc(void*, size_t bytes, void* stream) {
  void* p = nullptr;
  if (bytes == 0) bytes = 256;
  if (hipMallocAsync(&p, bytes, (hipStream_t)stream) != hipSuccess) {
    (void)hipGetLastError();
    p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
  }
  return p;
}

void default_free(void*, void* p, void* stream) {
  if (!p) return;
  if (hipFreeAsync(p, (hipStream_t)stream) != hipSuccess) {
    (void)hipGetLastError();
    (void)hipFree(p);
  }
}

const aires_allocator kDefaultAllocator = {default_alloc, default_free, nullptr};

// Device allocations of one call, released together (stream-ordered).  The
// pool enforces the plan's device budget (Sec. III-A: the memory constraint
// M): `cap` is what the budget leaves after the borrowed device inputs, and
// `used` counts every byte the call has taken, including blocks handed to
// the caller as C, so a call never holds more than the budget.
struct DevPool {
  aires_allocator a;
  hipStream_t s;
  int64_t cap;      // < 0: no limit
  int64_t used = 0;
  struct Block { void* p; int64_t n; };
  std::vector<Block> live;
  // Arena mode (the allocation-free entry point): blocks are carved, 256-byte
  // aligned, from [arena, arena + cap) and nothing is allocated or freed.
  char* arena = nullptr;
  DevPool(const aires_allocator& al, hipStream_t st, int64_t cap_bytes = -1) : a(al), s(st), cap(cap_bytes) {}
  DevPool(void* base, int64_t bytes, hipStream_t st) : a{}, s(st), cap(bytes), arena(static_cast<char*>(base)) {}
  ~DevPool() { release(); }
  static int64_t round256(int64_t n) { return (n + 255) & ~int64_t(255); }
  bool fits(int64_t bytes) const { return cap < 0 || used + (arena ? round256(bytes) : bytes) <= cap; }
  aires_status get(size_t bytes, void** out) {
    const int64_t n = (int64_t)(bytes ? bytes : 256);
    if (arena) {
      if (!fits(n))
        return fail(AIRES_E_CAPACITY, "the workspace needs more than the %lld-byte fixed scratch array",
                    (long long)cap);
      *out = arena + used;
      used += round256(n);
      return AIRES_OK;
    }
    if (!fits(n))
      return fail(AIRES_E_BUDGET, "device allocation of %lld bytes exceeds the budget (%lld of %lld bytes in use)",
                  (long long)n, (long long)used, (long long)cap);
    void* p = a.alloc(a.ctx, (size_t)n, (void*)s);
    if (!p) return fail(AIRES_E_OOM, "device allocation of %zu bytes failed", bytes);
    live.push_back({p, n});
    used += n;
    *out = p;
    return AIRES_OK;
  }
  template <typename T>
  aires_status get_n(int64_t n, T** out) {
    return get((size_t)std::max<int64_t>(n, 1) * sizeof(T), reinterpret_cast<void**>(out));
  }
  void release() {
    for (const Block& b : live) a.free(a.ctx, b.p, (void*)s);
    live.clear();
  }
  int64_t left() const { return cap < 0 ? INT64_MAX : cap - used; }
  // hand ownership of p to the caller (it still counts against the budget
  // for the rest of the call)
  void detach(void* p) {
    live.erase(std::remove_if(live.begin(), live.end(), [p](const Block& b) { return b.p == p; }), live.end());
  }
  // free p now (stream-ordered) and stop counting it
  void give_back(void* p) {
    if (arena) return;  // carved blocks stay until the call ends
    for (size_t i = 0; i < live.size(); ++i)
      if (live[i].p == p) {
        a.free(a.ctx, p, (void*)s);
        used -= live[i].n;
        live.erase(live.begin() + (long)i);
        return;
      }
  }
};

struct OutOwner {
  aires_allocator a;
  hipStream_t s;
  int host;  // 1: hipHostMalloc'd arrays
};

}  // namespace

// ------------------------------------------------------------------- plan

namespace {

// A's column and value arrays in a file (the storage tier): read per tile
// into pinned staging buffers.  With direct I/O the reads bypass the page
// cache, cover whole 4 KiB blocks around the range and land in a bounce
// buffer of ordinary memory (the runtime's pinned pages cannot be handed to
// the block layer), from which the same threads copy them out.
struct FileSrc {
  int fd = -1;
  bool direct = false;
  int64_t col_off = 0, val_off = 0;
  void* rp_host = nullptr;  // A's row pointers, read at planning (pinned when possible)
  bool rp_pinned = false;
  char* bounce = nullptr;
  size_t bounce_cap = 0;
  ~FileSrc() {
    if (fd >= 0) close(fd);
    if (rp_host) {
      if (rp_pinned) (void)hipHostFree(rp_host);
      else std::free(rp_host);
    }
    std::free(bounce);
  }
};

constexpr int64_t kIoAlign = 4096;

// Opens a file for reading, with direct I/O when asked for and the
// filesystem allows it (else buffered reads).
aires_status open_file_src(const char* path, int direct_io, FileSrc& f) {
  f.fd = open(path, O_RDONLY | (direct_io ? O_DIRECT : 0));
  if (f.fd >= 0 && direct_io) f.direct = true;
  if (f.fd < 0 && direct_io) f.fd = open(path, O_RDONLY);  // no direct I/O on this filesystem
  if (f.fd < 0) return fail(AIRES_E_INVALID_ARG, "cannot open %s: %s", path, strerror(errno));
  return AIRES_OK;
}

// Reads file bytes [off, off + len) into dst; *shift receives where they
// start in dst (always 0 now; kept for the callers' buffer layout).
// Ranges of 8 MiB or more are read by several host threads.
aires_status file_read(FileSrc& f, int64_t off, int64_t len, char* dst, int64_t* shift) {
  const int64_t a0 = f.direct ? off & ~(kIoAlign - 1) : off;
  const int64_t a1 = f.direct ? (off + len + kIoAlign - 1) & ~(kIoAlign - 1) : off + len;
  *shift = 0;
  if (len <= 0) return AIRES_OK;
  const int64_t total = a1 - a0;
  char* buf = dst;
  if (f.direct) {
    if ((size_t)total > f.bounce_cap) {
      std::free(f.bounce);
      f.bounce_cap = (size_t)total;
      f.bounce = static_cast<char*>(std::aligned_alloc((size_t)kIoAlign, f.bounce_cap));
      if (!f.bounce) {
        f.bounce_cap = 0;
        return fail(AIRES_E_OOM, "host allocation of %lld bytes failed", (long long)total);
      }
    }
    buf = f.bounce;
  }
  const int nt = total >= (int64_t(8) << 20) ? 8 : 1;
  std::vector<int> err(nt, 0);
  std::vector<int64_t> got(nt, 0);
  auto part = [&](int i) {
    int64_t lo = total * i / nt, hi = total * (i + 1) / nt;
    if (f.direct) {
      lo &= ~(kIoAlign - 1);
      if (i + 1 < nt) hi &= ~(kIoAlign - 1);
    }
    for (int64_t p = lo; p < hi;) {
      const ssize_t r = pread(f.fd, buf + p, (size_t)(hi - p), (off_t)(a0 + p));
      if (r < 0) { err[i] = errno; return; }
      if (r == 0) break;  // end of file
      p += r;
      got[i] = p - lo;
    }
    if (f.direct) {  // this thread's share of the wanted bytes, out of the bounce buffer
      const int64_t w0 = std::max(lo, off - a0), w1 = std::min(lo + got[i], off - a0 + len);
      if (w1 > w0) std::memcpy(dst + (w0 - (off - a0)), buf + w0, (size_t)(w1 - w0));
    }
  };
  if (nt == 1) {
    part(0);
  } else {
    std::vector<std::thread> th;
    for (int i = 0; i < nt; ++i) th.emplace_back(part, i);
    for (auto& x : th) x.join();
  }
  for (int i = 0; i < nt; ++i)
    if (err[i]) return fail(AIRES_E_INVALID_ARG, "reading A's file failed: %s", strerror(err[i]));
  // the bytes asked for must all be there (a direct read may stop at the
  // end of the file inside the last block)
  int64_t have = 0;
  for (int i = 0; i < nt; ++i) {
    int64_t lo = total * i / nt;
    if (f.direct) lo &= ~(kIoAlign - 1);
    have = std::max(have, lo + got[i]);
  }
  if (have < (off - a0) + len)
    return fail(AIRES_E_INVALID_ARG, "A's file ends before byte %lld", (long long)(off + len));
  return AIRES_OK;
}

}  // namespace

struct aires_plan {
  aires_csr A, B;
  aires_plan_opts opts;
  aires_allocator alloc;
  int64_t budget;
  std::vector<aires_tile> tiles;
  aires_plan_info_t info;
  aires_stats stats;
  int busy = 0;
  std::unique_ptr<FileSrc> file;   // A's entries in a file (aires_tile_plan_file)
  // kernel configuration
  kern::BinThresholds th;
  int wide = 0;
  int32_t G = 0, nG = 0;           // column grains (wide products)
  int32_t win_grains = 0, win_entries = 0, count_grains = 0, win_pool_words = 0;
  int32_t ngg = 0;                 // symbolic items per wide row (runs of count_grains grains)
  int64_t keep_bitmap = 0;         // rows with more products keep their symbolic bitmaps (-1: none)
  int32_t slab_bin = -1;           // first window bin whose rows are split over column slabs (-1: none)
  int split = 0;                   // narrow product with a split-row bin
  int64_t split_cap = 0;           // rows with dense slots for the split bin
  int64_t split_ws = 0;            // bytes of those slots
  // per-tile counts of the last call (products, nnz(C), bytes copied)
  struct TileRun { int64_t products, nnz_c, h2d_bytes, d2h_bytes, resent_bytes; double merge_ms, storage_ms; };
  std::vector<TileRun> trun;
  // per tile, indices into ev of: copy in begin/end, compute begin/end,
  // copy out begin/end (-1: none); times are taken from ev[ev_base]
  enum { T_H2D0, T_H2D1, T_C0, T_C1, T_D2H0, T_D2H1, T_NEV };
  std::vector<std::array<int, T_NEV>> tev;
  int ev_base = -1;
  // timing events of the last call
  std::vector<hipEvent_t> ev;
  struct Mark { int kind; int phase; int a, b; int tile; };  // elapsed(ev[a], ev[b]); tile -1: whole call
  std::vector<Mark> marks;
  ~aires_plan() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  }
};

namespace {

void bin_plan(aires_plan* p) {
  const int64_t N = p->B.ncols;
  const aires_plan_opts& o = p->opts;
  const int64_t dense_max = o.dense_max_cols > 0 ? std::min<int64_t>(o.dense_max_cols, kDenseMaxCols) : kDenseMaxCols;
  const int64_t wave_max = o.wave_max_products > 0 ? o.wave_max_products : kWaveMaxProducts;
  const int64_t split_min = o.split_min_products > 0   ? o.split_min_products
                            : o.split_min_products < 0 ? 0  // < 0: no split rows
                                                       : kSplitMinProducts;
  const int64_t hash_max = o.hash_max_products > 0   ? std::min<int64_t>(o.hash_max_products, kHashMaxProducts)
                           : o.hash_max_products < 0 ? 0  // < 0: no hash bins
                                                     : kHashMaxProducts;
  kern::BinThresholds& th = p->th;
  std::memset(&th, 0, sizeof th);
  int nb = 0;
  auto add = [&](int kind, int64_t maxp) { th.kind[nb] = kind; th.max_p[nb] = maxp; ++nb; };
  add(kern::KIND_EMPTY, 0);
  p->wide = 0;
  p->split = 0;
  if (N <= std::min(kDenseWaveMaxN, dense_max)) {
    // narrow product: every row fits a dense LDS row
    add(kern::KIND_DENSE_WAVE, wave_max);
    if (split_min > 0) {
      add(kern::KIND_DENSE_BLOCK, std::max(wave_max, split_min));
      add(kern::KIND_DENSE_SPLIT, INT64_MAX);
      p->split = 1;
    } else {
      add(kern::KIND_DENSE_BLOCK, INT64_MAX);
    }
  } else {
    // light rows hash in LDS (load factor <= 1/2: nnz(C_i) <= P_i <= slots/2)
    if (hash_max > 0) add(kern::KIND_HASH_128, std::min<int64_t>(hash_max, 64));
    if (hash_max > 64) add(kern::KIND_HASH_1024, std::min<int64_t>(hash_max, 512));
    if (hash_max > 512) add(kern::KIND_HASH_4096, std::min<int64_t>(hash_max, 2048));
    if (hash_max > 2048) add(kern::KIND_HASH_8192, hash_max);
    if (N <= dense_max) {
      add(kern::KIND_DENSE_BLOCK, INT64_MAX);
    } else {
      // window bins, the heavy rows last in the list (processed first): cut
      // where rows start keeping their symbolic bitmaps and where their
      // windows start being spread over column slabs (the bins from there on)
      const int64_t w_lo = std::max<int64_t>(hash_max, 1);
      const int64_t keep = o.keep_bitmap_products == 0 ? kKeepBitmapProducts : o.keep_bitmap_products;
      const int64_t slab_min = o.slab_min_products == 0 ? kSlabMinProducts : o.slab_min_products;
      const int64_t heavy = slab_min > 0 ? slab_min : w_lo << 8;
      int64_t cuts[2] = {keep, heavy};
      if (cuts[0] > cuts[1]) std::swap(cuts[0], cuts[1]);
      const int first_window_bin = nb;
      for (int64_t c : cuts)
        if (c > w_lo && th.max_p[nb - 1] != c) {
          add(kern::KIND_WINDOWS, c);
          if (c == slab_min) p->slab_bin = nb;
        }
      add(kern::KIND_WINDOWS, INT64_MAX);
      if (slab_min > 0 && slab_min <= w_lo) p->slab_bin = first_window_bin;
      p->wide = 1;
      p->G = (int32_t)(o.window_grain_cols > 0 ? o.window_grain_cols : kGrainCols);
      p->nG = (int32_t)((N + p->G - 1) / p->G);
      p->win_grains = (int32_t)(o.window_max_grains > 0 ? o.window_max_grains : kWindowMaxGrains);
      p->win_entries = (int32_t)(o.window_max_entries > 0 ? o.window_max_entries
                                                          : std::max<int64_t>(kWindowMaxEntries, p->G));
      p->count_grains = (int32_t)(o.count_grains > 0 ? o.count_grains : kCountGrains);
      p->win_pool_words = (int32_t)((o.window_pool_bytes > 0 ? o.window_pool_bytes : kWindowPoolBytes) / 4);
      p->ngg = (p->nG + p->count_grains - 1) / p->count_grains;
      p->keep_bitmap = keep;
    }
  }
  th.nb = nb;
}

aires_status check_csr_desc(const aires_csr* M, const char* name, bool need_vals = true) {
  if (!M) return fail(AIRES_E_INVALID_ARG, "%s is NULL", name);
  if (M->nrows < 0 || M->ncols < 0 || M->nnz < 0)
    return fail(AIRES_E_DIM, "%s has a negative size", name);
  if (M->rp_type != AIRES_IDX_I32 && M->rp_type != AIRES_IDX_I64)
    return fail(AIRES_E_INVALID_ARG, "%s.rp_type %d invalid", name, M->rp_type);
  if (M->mem != AIRES_MEM_DEVICE && M->mem != AIRES_MEM_HOST_PINNED && M->mem != AIRES_MEM_HOST)
    return fail(AIRES_E_INVALID_ARG, "%s.mem %d invalid", name, M->mem);
  if (!M->row_ptr) return fail(AIRES_E_INVALID_ARG, "%s.row_ptr is NULL", name);
  if (M->nnz > 0 && (!M->col_idx || (need_vals && !M->vals)))
    return fail(AIRES_E_INVALID_ARG, "%s arrays are NULL", name);
  if (M->ncols > INT32_MAX) return fail(AIRES_E_OVERFLOW, "%s.ncols exceeds int32 column indices", name);
  if (M->rp_type == AIRES_IDX_I32 && M->nnz > INT32_MAX)
    return fail(AIRES_E_OVERFLOW, "%s.nnz needs int64 row pointers", name);
  return AIRES_OK;
}

aires_status validate_host(const aires_csr& M, const char* name, bool check_vals = true) {
  if (host_rp(M, 0) != 0) return fail(AIRES_E_INVALID_CSR, "%s.row_ptr[0] != 0", name);
  if (host_rp(M, M.nrows) != M.nnz) return fail(AIRES_E_INVALID_CSR, "%s.row_ptr[nrows] != nnz", name);
  for (int64_t i = 0; i < M.nrows; ++i) {
    const int64_t a = host_rp(M, i), b = host_rp(M, i + 1);
    if (b < a) return fail(AIRES_E_INVALID_CSR, "%s.row_ptr decreases at row %lld", name, (long long)i);
    for (int64_t q = a; q < b; ++q) {
      const int32_t c = M.col_idx[q];
      if (c < 0 || c >= M.ncols)
        return fail(AIRES_E_INVALID_CSR, "%s column %d out of range in row %lld", name, c, (long long)i);
      if (q > a && c <= M.col_idx[q - 1])
        return fail(AIRES_E_INVALID_CSR, "%s columns not strictly increasing in row %lld", name, (long long)i);
      if (check_vals && !std::isfinite(M.vals[q]))
        return fail(AIRES_E_INVALID_CSR, "%s has a non-finite value", name);
    }
  }
  return AIRES_OK;
}

// P_i on the host: A and B.rp in host memory; multithreaded over row ranges.
// n int64 values left uninitialised: the parallel passes that fill them
// also touch their pages first.
struct I64Array {
  std::unique_ptr<int64_t[]> v;
  int64_t n = 0;
  void alloc(int64_t k) {
    v.reset(new int64_t[(size_t)std::max<int64_t>(k, 1)]);
    n = k;
  }
  void clear() {
    v.reset();
    n = 0;
  }
  bool empty() const { return n == 0; }
  int64_t& operator[](size_t i) { return v[i]; }
  const int64_t& operator[](size_t i) const { return v[i]; }
};

// Runs fn(lo, hi, t) over [0, n) cut into contiguous ranges, one per host
// thread t < nt (up to 16 threads; one below 2^16 items).
template <typename Fn>
int parallel_ranges(int64_t n, Fn fn) {
  int nt = (int)std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  if (n < 65536) nt = 1;
  if (nt == 1) {
    fn((int64_t)0, n, 0);
    return 1;
  }
  std::vector<std::thread> th;
  for (int t = 0; t < nt; ++t) th.emplace_back([&, t]() { fn(n * t / nt, n * (t + 1) / nt, t); });
  for (auto& x : th) x.join();
  return nt;
}

// nnz(B_k) for every row of a device-resident B (rows hold at most N < 2^31
// entries), from its row pointers copied to the host
aires_status host_row_lengths(const aires_csr& B, std::vector<int32_t>& len, int64_t* max_len) {
  const int64_t K = B.nrows;
  len.resize((size_t)K);
  std::vector<int64_t> brp((size_t)K + 1);
  if (B.rp_type == AIRES_IDX_I64) {
    HIP_TRY(hipMemcpy(brp.data(), B.row_ptr, brp.size() * 8, hipMemcpyDeviceToHost));
  } else {
    std::vector<int32_t> tmp(brp.size());
    HIP_TRY(hipMemcpy(tmp.data(), B.row_ptr, tmp.size() * 4, hipMemcpyDeviceToHost));
    for (size_t i = 0; i < tmp.size(); ++i) brp[i] = tmp[i];
  }
  int64_t mx = 0;
  for (int64_t k = 0; k < K; ++k) {
    len[(size_t)k] = (int32_t)(brp[(size_t)k + 1] - brp[(size_t)k]);
    mx = std::max<int64_t>(mx, len[(size_t)k]);
  }
  *max_len = mx;
  return AIRES_OK;
}

// C bound per row, u_i = min(N, P_i) with P_i = sum over A_i of nnz(B_k):
// its total, its running sum when cpre is given (cpre[0] = 0, m + 1
// entries; u_i is parked in cpre[i + 1] and summed in place), and the
// number of rows with P_i > lim.  The gather of nnz(B_k) is random over B's rows: the
// lengths are read from the narrowest table that holds them (a byte each
// for feature matrices), each thread requests them a fixed distance ahead
// of their use, and a row stops once its sum reaches N, or max(N, lim + 1)
// if it could pass lim (|A_i| * max_k nnz(B_k) > lim): min(N, P_i) and
// P_i > lim stay exact.
template <typename L>
void host_bounds_t(const aires_csr& A, const int64_t* arp, const L* len, int64_t max_len, int64_t N, int64_t lim,
                   I64Array* cpre, int64_t* total, int64_t* above) {
  constexpr int64_t kAhead = 64;
  const int64_t m = A.nrows;
  const int32_t* col = A.col_idx;
  if (cpre) {
    cpre->alloc(m + 1);
    (*cpre)[0] = 0;
  }
  int64_t* u_out = cpre ? &(*cpre)[1] : nullptr;
  std::vector<int64_t> part(17, 0), cnt(17, 0);
  const int nt = parallel_ranges(m, [&](int64_t lo, int64_t hi, int t) {
    int64_t sum = 0, c = 0;
    const int64_t qend = arp[hi];
    const int64_t heavy_stop = lim < INT64_MAX ? std::max(N, lim + 1) : N;
    for (int64_t i = lo; i < hi; ++i) {
      int64_t P = 0;
      const int64_t stop = (arp[i + 1] - arp[i]) * max_len > lim ? heavy_stop : N;
      for (int64_t q = arp[i]; q < arp[i + 1] && P < stop; ++q) {
        if (q + kAhead < qend) __builtin_prefetch(len + col[q + kAhead], 0, 0);
        P += len[col[q]];
      }
      const int64_t u = std::min<int64_t>(N, P);
      if (u_out) u_out[i] = u;
      sum += u;
      c += P > lim;
    }
    part[(size_t)t + 1] = sum;
    cnt[(size_t)t] = c;
  });
  for (int t = 0; t < nt; ++t) part[(size_t)t + 1] += part[(size_t)t];
  if (u_out) {
    parallel_ranges(m, [&](int64_t lo, int64_t hi, int t) {
      int64_t run = part[(size_t)t];
      for (int64_t i = lo; i < hi; ++i) {
        run += u_out[i];
        u_out[i] = run;
      }
    });
  }
  *total = part[(size_t)nt];
  int64_t a = 0;
  for (int t = 0; t < nt; ++t) a += cnt[(size_t)t];
  *above = a;
}

// B's row lengths in the narrowest table that holds them (max_len known),
// read from B's row pointers in host memory or from lenB when B is on the
// device (its row pointers were copied to the host to measure them)
void host_bounds(const aires_csr& A, const int64_t* arp, const aires_csr& B, const std::vector<int32_t>& lenB,
                 int64_t max_len, int64_t N, int64_t lim, I64Array* cpre, int64_t* total, int64_t* above) {
  const int64_t K = B.nrows;
  auto narrow = [&](auto tag) {
    using L = decltype(tag);
    std::vector<L> t((size_t)K);
    auto fill = [&](const auto* r) {
      parallel_ranges(K, [&, r](int64_t lo, int64_t hi, int) {
        for (int64_t k = lo; k < hi; ++k) t[(size_t)k] = (L)(r[k + 1] - r[k]);
      });
    };
    if (B.mem == AIRES_MEM_DEVICE) {
      parallel_ranges(K, [&](int64_t lo, int64_t hi, int) {
        for (int64_t k = lo; k < hi; ++k) t[(size_t)k] = (L)lenB[(size_t)k];
      });
    } else if (B.rp_type == AIRES_IDX_I64) {
      fill(static_cast<const int64_t*>(B.row_ptr));
    } else {
      fill(static_cast<const int32_t*>(B.row_ptr));
    }
    host_bounds_t(A, arp, t.data(), max_len, N, lim, cpre, total, above);
  };
  if (max_len <= 255) narrow(uint8_t{});
  else if (max_len <= 65535) narrow(uint16_t{});
  else narrow(int32_t{});
}

// max_k nnz(B_k) from B's row pointers
aires_status host_max_row_length(const aires_csr& B, int64_t* max_len) {
  const int64_t K = B.nrows;
  if (B.mem == AIRES_MEM_DEVICE) {
    std::vector<int32_t> len;
    return host_row_lengths(B, len, max_len);
  }
  std::vector<int64_t> mx(16, 0);
  auto scan = [&](const auto* r) {
    return parallel_ranges(K, [&, r](int64_t lo, int64_t hi, int t) {
      int64_t x = 0;
      for (int64_t k = lo; k < hi; ++k) x = std::max<int64_t>(x, (int64_t)r[k + 1] - (int64_t)r[k]);
      mx[(size_t)t] = x;
    });
  };
  const int nt = B.rp_type == AIRES_IDX_I64 ? scan(static_cast<const int64_t*>(B.row_ptr))
                                            : scan(static_cast<const int32_t*>(B.row_ptr));
  *max_len = K > 0 ? *std::max_element(mx.begin(), mx.begin() + nt) : 0;
  return AIRES_OK;
}

// u_i = min(N, nnz(A_i) * max_len) from A's row pointers alone: its total,
// and its running sum when cpre is given (a second pass recomputes u_i)
void host_row_bounds(const aires_csr& A, const int64_t* arp, int64_t max_len, int64_t N, I64Array* cpre,
                     int64_t* total) {
  const int64_t m = A.nrows;
  auto u_of = [&](int64_t i) -> int64_t {
    const int64_t len = arp[i + 1] - arp[i];
    return len > 0 && max_len > N / len ? N : std::min<int64_t>(N, len * max_len);
  };
  std::vector<int64_t> part(17, 0);
  const int nt = parallel_ranges(m, [&](int64_t lo, int64_t hi, int t) {
    int64_t sum = 0;
    for (int64_t i = lo; i < hi; ++i) sum += u_of(i);
    part[(size_t)t + 1] = sum;
  });
  for (int t = 0; t < nt; ++t) part[(size_t)t + 1] += part[(size_t)t];
  *total = part[(size_t)nt];
  if (!cpre) return;
  cpre->alloc(m + 1);
  (*cpre)[0] = 0;
  int64_t* run_out = &(*cpre)[1];
  parallel_ranges(m, [&](int64_t lo, int64_t hi, int t) {
    int64_t run = part[(size_t)t];
    for (int64_t i = lo; i < hi; ++i) {
      run += u_of(i);
      run_out[i] = run;
    }
  });
}

aires_status host_row_ptr(const aires_csr& M, std::vector<int64_t>& out) {
  out.resize((size_t)M.nrows + 1);
  if (M.mem == AIRES_MEM_DEVICE) {
    if (M.rp_type == AIRES_IDX_I64) {
      HIP_TRY(hipMemcpy(out.data(), M.row_ptr, out.size() * 8, hipMemcpyDeviceToHost));
    } else {
      std::vector<int32_t> tmp(out.size());
      HIP_TRY(hipMemcpy(tmp.data(), M.row_ptr, tmp.size() * 4, hipMemcpyDeviceToHost));
      for (size_t i = 0; i < tmp.size(); ++i) out[i] = tmp[i];
    }
  } else {
    parallel_ranges(M.nrows + 1, [&](int64_t lo, int64_t hi, int) {
      if (M.rp_type == AIRES_IDX_I64) {
        std::memcpy(out.data() + lo, static_cast<const int64_t*>(M.row_ptr) + lo, (size_t)(hi - lo) * 8);
      } else {
        const int32_t* r = static_cast<const int32_t*>(M.row_ptr);
        for (int64_t i = lo; i < hi; ++i) out[(size_t)i] = r[i];
      }
    });
  }
  return AIRES_OK;
}

}  // namespace

extern "C" {

int aires_abi_version(void) { return AIRES_ABI_VERSION; }

const char* aires_last_error(void) { return g_last_error.c_str(); }

const char* aires_status_string(aires_status s) {
  switch (s) {
    case AIRES_OK: return "AIRES_OK";
    case AIRES_E_INVALID_ARG: return "AIRES_E_INVALID_ARG";
    case AIRES_E_INVALID_CSR: return "AIRES_E_INVALID_CSR";
    case AIRES_E_DIM: return "AIRES_E_DIM";
    case AIRES_E_BUDGET: return "AIRES_E_BUDGET";
    case AIRES_E_OVERFLOW: return "AIRES_E_OVERFLOW";
    case AIRES_E_OOM: return "AIRES_E_OOM";
    case AIRES_E_HIP: return "AIRES_E_HIP";
    case AIRES_E_STATE: return "AIRES_E_STATE";
    case AIRES_E_UNSUPPORTED: return "AIRES_E_UNSUPPORTED";
    case AIRES_E_CAPACITY: return "AIRES_E_CAPACITY";
  }
  return "AIRES_E_UNKNOWN";
}

aires_status aires_plan_opts_default(aires_plan_opts* o) {
  if (!o) return fail(AIRES_E_INVALID_ARG, "opts is NULL");
  std::memset(o, 0, sizeof *o);
  o->struct_size = sizeof(aires_plan_opts);
  o->c_placement = AIRES_MEM_DEVICE;
  o->c_bound = AIRES_CBOUND_PRODUCTS;
  return AIRES_OK;
}

}  // extern "C"

namespace {

// The planner.  file != nullptr: A's entries are in that file (A->col_idx
// and A->vals are NULL; its row pointers are in host memory); the plan
// takes the file over when it succeeds.
aires_status plan_impl(const aires_csr* A, const aires_csr* B, uint64_t hbm_budget, const aires_plan_opts* opts,
                       aires_plan** out, std::unique_ptr<FileSrc>* file) {
  if (!out) return fail(AIRES_E_INVALID_ARG, "out is NULL");
  if (opts && opts->struct_size != sizeof(aires_plan_opts))
    return fail(AIRES_E_INVALID_ARG, "opts.struct_size %u != %zu", opts->struct_size, sizeof(aires_plan_opts));
  const bool a_sym_norm = opts && opts->a_values == AIRES_AVALUES_SYM_NORM;
  if (file) {
    if (!A || !A->row_ptr || A->nrows < 0 || A->ncols < 0 || A->nnz < 0)
      return fail(AIRES_E_INVALID_ARG, "A's descriptor is incomplete");
  } else {
    ST_TRY(check_csr_desc(A, "A", !a_sym_norm));
  }
  ST_TRY(check_csr_desc(B, "B"));
  if (opts && opts->a_values != AIRES_AVALUES_GIVEN && opts->a_values != AIRES_AVALUES_SYM_NORM)
    return fail(AIRES_E_INVALID_ARG, "opts.a_values %d invalid", opts->a_values);
  if (a_sym_norm && A->nrows != A->ncols)
    return fail(AIRES_E_DIM, "a_values = SYM_NORM needs a square A (%lld x %lld)", (long long)A->nrows,
                (long long)A->ncols);
  if (A->ncols != B->nrows)
    return fail(AIRES_E_DIM, "A.ncols (%lld) != B.nrows (%lld)", (long long)A->ncols, (long long)B->nrows);
  if (A->nrows > INT32_MAX - 1) return fail(AIRES_E_OVERFLOW, "A.nrows exceeds int32 row ids");
  aires_plan_opts o;
  aires_plan_opts_default(&o);
  if (opts) {
    if (opts->struct_size != sizeof(aires_plan_opts))
      return fail(AIRES_E_INVALID_ARG, "opts.struct_size %u != %zu", opts->struct_size, sizeof(aires_plan_opts));
    o = *opts;
  }
  if (o.c_placement != AIRES_MEM_DEVICE && o.c_placement != AIRES_MEM_HOST_PINNED)
    return fail(AIRES_E_INVALID_ARG, "opts.c_placement %d invalid", o.c_placement);
  if (o.c_bound < AIRES_CBOUND_PRODUCTS || o.c_bound > AIRES_CBOUND_ROWS)
    return fail(AIRES_E_INVALID_ARG, "opts.c_bound %d invalid", o.c_bound);
  if (o.max_tile_rows < 0 || o.max_tile_bytes < 0 || o.m_a_bytes < 0 || o.bitmap_cache_bytes < 0)
    return fail(AIRES_E_INVALID_ARG, "negative tile or cache cap");
  if (o.segmentation != AIRES_SEG_ROBW && o.segmentation != AIRES_SEG_MAXFILL)
    return fail(AIRES_E_INVALID_ARG, "opts.segmentation %d invalid", o.segmentation);
  if (o.segmentation == AIRES_SEG_MAXFILL &&
      (A->mem != AIRES_MEM_HOST_PINNED || a_sym_norm || o.m_a_bytes > 0 || o.max_tile_rows > 0))
    return fail(AIRES_E_UNSUPPORTED,
                "max-fill segments need A in pinned host memory with given values (and no Algorithm 1 "
                "planning mode or row cap)");
  if (file && (o.segmentation != AIRES_SEG_ROBW || o.c_bound == AIRES_CBOUND_PRODUCTS || o.validate ||
               o.m_a_bytes > 0))
    return fail(AIRES_E_UNSUPPORTED,
                "a file-backed A is planned from its row pointers alone: row blocks with c_bound ROWS, DENSE "
                "or PAPER_EQ5, no validation, no Algorithm 1 planning mode");
  if (o.validate) {
    if (A->mem != AIRES_MEM_DEVICE) ST_TRY(validate_host(*A, "A", !a_sym_norm));
    if (B->mem != AIRES_MEM_DEVICE) ST_TRY(validate_host(*B, "B"));
  }

  const int a_streamed = A->mem != AIRES_MEM_DEVICE;
  const int c_on_host = o.c_placement == AIRES_MEM_HOST_PINNED;
  if (!a_streamed && c_on_host)
    return fail(AIRES_E_UNSUPPORTED, "C in host memory needs A in host memory (streamed tiles)");

  int64_t budget = (int64_t)hbm_budget;
  if (budget == 0) {
    size_t fr = 0, tot = 0;
    HIP_TRY(hipMemGetInfo(&fr, &tot));
    budget = (int64_t)fr;
  }

  auto* p = new aires_plan();
  p->A = *A;
  p->B = *B;
  p->opts = o;
  p->alloc = o.allocator ? *o.allocator : kDefaultAllocator;
  p->budget = budget;
  bin_plan(p);
  const int64_t m = A->nrows, K = A->ncols, N = B->ncols;
  const int64_t sA = rp_bytes(*A);
  std::memset(&p->info, 0, sizeof p->info);
  p->info.m = m;
  p->info.k = K;
  p->info.n = N;
  p->info.budget = budget;
  p->info.b_bytes = csr_bytes(*B);
  p->info.a_bytes = csr_bytes(*A);
  p->info.a_streamed = a_streamed;
  p->info.c_on_host = c_on_host;
  p->info.c_bound_entries = -1;

  if (p->wide) {
    if (p->G < 32 || p->G % 32 || p->G > (1 << 20) || p->win_entries < p->G || p->win_entries > 65535 ||
        p->win_grains < 1 || p->count_grains < 1 ||
        kern::window_numeric_lds(p->win_pool_words) > kern::kMaxLds ||
        2 * kern::win_words(p->G) + p->G > p->win_pool_words ||  // one full grain fits the pool
        kern::grain_count_lds(p->count_grains, p->G) > kern::kMaxLds || p->nG > 65535 ||
        (int64_t)p->count_grains * p->G * kern::group_size(kern::KIND_WINDOWS) >= (int64_t(1) << 31)) {
      aires_status st = fail(AIRES_E_INVALID_ARG,
                             "window options out of range (grain %d, windows of %d grains / %d entries, "
                             "%d grains per count item, %d grains)",
                             p->G, p->win_grains, p->win_entries, p->count_grains, p->nG);
      delete p;
      return st;
    }
    if (B->nnz > INT32_MAX) {
      delete p;
      return fail(AIRES_E_UNSUPPORTED, "column windows need nnz(B) < 2^31");
    }
  }
  const int64_t nG = p->wide ? p->nG : 0;
  const int64_t index_bytes = p->wide ? 4 * (nG + 2) * K : 0;  // grain index and max |b| per B row

  // A's row pointers on the host as int64 (in place when they already are)
  std::vector<int64_t> arp_own;
  const int64_t* arp = nullptr;
  aires_status st = AIRES_OK;
  if (A->mem != AIRES_MEM_DEVICE && A->rp_type == AIRES_IDX_I64) {
    arp = static_cast<const int64_t*>(A->row_ptr);
  } else {
    st = host_row_ptr(*A, arp_own);
    if (st != AIRES_OK) { delete p; return st; }
    arp = arp_own.data();
  }

  // Per-row and per-tile bytes of one tile slot.
  // ws per row: P_i (8) + bin list (4) + window counts (4 per window) + C row
  // pointer of the tile (8, streamed only).
  I64Array cu;    // C bound per row (entries), for the bounds built row by row
  I64Array cpre;  // running sum of the C bound when C is placed in host memory
  int64_t split_rows = -1;    // rows above the split threshold (when P_i is computed)
  int64_t resident = p->info.b_bytes + kFixedWorkspace + index_bytes;
  // (+ per-grain counts and per-row window counts of wide products)
  int64_t per_row_ws = 8 + 4 + (p->wide ? 4 * nG + 8 : 0);
  // derived values of a streamed A need all of A's row pointers on the device
  if (a_streamed && a_sym_norm) resident += (m + 1) * sA;
  if (!a_streamed) {
    // A and C.row_ptr resident; products, bin lists and window bookkeeping
    // for all rows (the numeric sweep of a tile reads its rows' products
    // after the symbolic sweep of every tile)
    resident += p->info.a_bytes + 8 * (m + 1) + (8 + 4 + (p->wide ? 4 * nG + 8 + 8 * p->ngg : 0)) * m;
    per_row_ws = 0;
  } else if (o.m_a_bytes == 0) {
    // C bound per row for the C slots (or for a device-resident C)
    if (o.c_bound == AIRES_CBOUND_PRODUCTS) {
      std::vector<int32_t> lenB;  // B on the device only
      int64_t max_len = 0;
      st = B->mem == AIRES_MEM_DEVICE ? host_row_lengths(*B, lenB, &max_len) : host_max_row_length(*B, &max_len);
      if (st != AIRES_OK) { delete p; return st; }
      const int64_t lim = p->split ? p->th.max_p[p->th.nb - 2] : INT64_MAX;
      host_bounds(*A, arp, *B, lenB, max_len, N, lim, c_on_host ? &cpre : nullptr, &p->info.c_bound_entries,
                  &split_rows);
    } else if (o.c_bound == AIRES_CBOUND_ROWS) {
      int64_t max_len = 0;
      st = host_max_row_length(*B, &max_len);
      if (st != AIRES_OK) { delete p; return st; }
      host_row_bounds(*A, arp, max_len, N, c_on_host ? &cpre : nullptr, &p->info.c_bound_entries);
    } else if (o.c_bound == AIRES_CBOUND_DENSE) {
      cu.alloc(m);
      for (int64_t i = 0; i < m; ++i) cu[(size_t)i] = N;
      p->info.c_bound_entries = m * N;
    } else {
      // Eq. 5 with alpha_A read as dense value bytes: M_C = 12 nnzA (1 + N/m + rho_B),
      // shared out over rows in proportion to their A entries.
      const double rhoB = (K > 0 && N > 0) ? (double)B->nnz / ((double)K * (double)N) : 0.0;
      const double mc_entries = 12.0 * (double)A->nnz * (1.0 + (m ? (double)N / (double)m : 0.0) + rhoB) / 8.0;
      cu.alloc(m);
      int64_t tot = 0;
      for (int64_t i = 0; i < m; ++i) {
        const double share = A->nnz ? mc_entries * (double)(arp[i + 1] - arp[i]) / (double)A->nnz : 0.0;
        cu[(size_t)i] = std::min<int64_t>(N, (int64_t)std::ceil(share));
        tot += cu[(size_t)i];
      }
      p->info.c_bound_entries = tot;
    }
    if (!c_on_host) resident += 8 * p->info.c_bound_entries + 8 * (m + 1);
  }
  if (p->split) {
    // dense slots of the split rows, shared by all tiles (their kernels run
    // on one stream): as many as rows above the split threshold when P_i is
    // known on the host, else as many as fit kSplitWsBytes
    const int64_t per = 4 * ((N + 31) / 32 + N);
    int64_t rows = std::min<int64_t>(m, std::max<int64_t>(1, kSplitWsBytes / per));
    if (split_rows >= 0)  // P_i known: rows above the upper end of the bin before the split bin
      rows = std::min(split_rows, std::max<int64_t>(1, kSplitWsBytes / per));
    if (o.split_max_rows > 0) rows = std::min(rows, o.split_max_rows);
    p->split_cap = rows;
    p->split_ws = rows * per;
    resident += p->split_ws;
  }

  const int nslots = a_streamed ? 2 : 1;
  int64_t tile_budget;
  if (o.m_a_bytes > 0) {
    tile_budget = o.m_a_bytes;
  } else {
    if (resident >= budget) {
      delete p;
      return fail(AIRES_E_BUDGET, "budget %lld bytes cannot hold the resident %lld bytes", (long long)budget,
                  (long long)resident);
    }
    tile_budget = (budget - resident) / nslots;
  }
  p->info.tile_budget = tile_budget;

  // bytes of a slot holding rows [r0, r1)
  auto slot_bytes = [&](int64_t r0, int64_t r1) -> int64_t {
    const int64_t k = r1 - r0, q = arp[r1] - arp[r0];
    if (o.m_a_bytes > 0) return (k + 1) * sA + 8 * q;  // calcMem of Algorithm 1
    int64_t b = k * per_row_ws;
    if (a_streamed) {
      b += (k + 1) * sA + 8 * q;
      if (c_on_host) {
        int64_t c = 0;
        for (int64_t i = r0; i < r1; ++i) c += cu[(size_t)i];
        b += 8 * c + 8 * (k + 1);
      }
    }
    return b;
  };
  // Greedy maximal blocks of whole rows (Algorithm 1).  Costs grow with
  // every added row, so the longest feasible block is found by doubling
  // and bisection; this yields exactly the linear scan's blocks.
  if (a_streamed && c_on_host && o.m_a_bytes == 0 && cpre.empty()) {
    cpre.alloc(m + 1);
    cpre[0] = 0;
    for (int64_t i = 0; i < m; ++i) cpre[(size_t)i + 1] = cpre[(size_t)i] + cu[(size_t)i];
  }
  if (!(a_streamed && c_on_host && o.m_a_bytes == 0)) cpre.clear();
  auto slot_bytes_fast = [&](int64_t r0, int64_t r1) -> int64_t {
    if (cpre.empty()) return slot_bytes(r0, r1);
    const int64_t k = r1 - r0, q = arp[r1] - arp[r0];
    return k * per_row_ws + (k + 1) * sA + 8 * q + 8 * (cpre[(size_t)r1] - cpre[(size_t)r0]) + 8 * (k + 1);
  };
  // Streamed A with no cap given: about kStreamTiles tiles, so that the
  // copies of one tile overlap the products of another (Algorithm 2)
  int64_t max_tile_bytes = o.max_tile_bytes;
  if (a_streamed && max_tile_bytes == 0 && o.m_a_bytes == 0)
    max_tile_bytes = std::max<int64_t>(p->info.a_bytes / kStreamTiles, kMinStreamTileBytes);
  int64_t part_budget = tile_budget;  // the budget the partition is cut under
  // (the tile-bytes cap sets the pipeline's grain: a row above it, which
  // cannot be divided, is a tile of its own)
  auto fits = [&](int64_t r0, int64_t r1) -> bool {
    if (o.max_tile_rows > 0 && r1 - r0 > o.max_tile_rows) return false;
    if (max_tile_bytes > 0 && r1 - r0 > 1 && (r1 - r0 + 1) * sA + 8 * (arp[r1] - arp[r0]) > max_tile_bytes)
      return false;
    return slot_bytes_fast(r0, r1) <= part_budget;
  };
  // The two slots of a streamed A are sized by the largest row count, the
  // largest number of entries sent and the largest C bound over all tiles,
  // which need not come from one tile: if those maxima together pass the
  // slot budget, the partition is redone under a budget smaller by the
  // excess.
  int64_t peak_slot = 0;
  for (int pass = 0;; ++pass) {
  p->tiles.clear();
  peak_slot = 0;
  int64_t r0 = 0;
  if (o.segmentation == AIRES_SEG_MAXFILL) {
    // Max-fill segments: from the first row not yet multiplied, as many of
    // A's entries as the slot holds, wherever that ends.  Entries [E, E + q)
    // are sent; rows [r0, r1) are complete in them (r1 the last row whose
    // end is at or before E + q); the head of row r1 goes back and opens
    // the next segment.  A segment's slot holds its q entries and the rows'
    // pointers, workspace and C bound, as a row block's does.
    auto last_row = [&](int64_t e) {  // largest r with arp[r] <= e
      return (int64_t)(std::upper_bound(arp, arp + m + 1, e) - arp) - 1;
    };
    auto seg_fits = [&](int64_t s0, int64_t e, int64_t q) -> bool {
      const int64_t s1 = std::min(m, last_row(e + q));
      if (s1 <= s0) return true;  // no complete row yet: the cost so far is below a row's
      if (max_tile_bytes > 0 && (s1 - s0 + 1) * sA + 8 * q > max_tile_bytes) return false;
      return slot_bytes_fast(s0, s1) + 8 * (e + q - arp[s1]) <= part_budget;
    };
    const int64_t nnzA = arp[m];
    while (r0 < m) {
      const int64_t E = arp[r0];
      const int64_t rest = nnzA - E;
      int64_t lo = 0, hi = rest + 1;  // seg_fits(lo); the largest q in [0, rest] that fits
      if (seg_fits(r0, E, rest)) {
        lo = rest;
      } else {
        while (hi - lo > 1) {
          const int64_t mid = lo + (hi - lo) / 2;
          if (seg_fits(r0, E, mid)) lo = mid; else hi = mid;
        }
      }
      int64_t q = lo;
      int64_t r1 = q == rest ? m : std::min(m, last_row(E + q));
      if (r1 <= r0) {
        // not one whole row under the tile-bytes cap: the segment is row r0
        // alone if its slot fits the budget (a row is never divided)
        const int64_t need = slot_bytes_fast(r0, r0 + 1);
        if (need > part_budget) {
          delete p;
          return fail(AIRES_E_BUDGET, "row %lld alone needs %lld bytes; a segment slot has %lld", (long long)r0,
                      (long long)need, (long long)part_budget);
        }
        q = arp[r0 + 1] - E;
        r1 = r0 + 1;
      }
      aires_tile t;
      t.r0 = r0;
      t.r1 = r1;
      t.nnz0 = E;
      t.nnz1 = arp[r1];
      t.sent_nnz1 = E + q;
      t.a_bytes = (r1 - r0 + 1) * sA + 8 * q;
      t.c_bound_entries = cpre.empty() ? -1 : cpre[(size_t)r1] - cpre[(size_t)r0];
      t.tile_bytes = slot_bytes_fast(r0, r1) + 8 * (E + q - arp[r1]);
      peak_slot = std::max(peak_slot, t.tile_bytes);
      p->tiles.push_back(t);
      r0 = r1;
    }
  }
  while (r0 < m) {
    if (!fits(r0, r0 + 1)) {
      const int64_t need = slot_bytes_fast(r0, r0 + 1);
      delete p;
      return fail(AIRES_E_BUDGET, "row %lld alone needs %lld bytes; a tile slot has %lld", (long long)r0,
                  (long long)need, (long long)part_budget);
    }
    int64_t lo = r0 + 1, step = 1;  // fits(r0, lo)
    int64_t hi = -1;                // first end that does not fit
    while (true) {
      const int64_t cand = std::min(m, r0 + step * 2);
      if (cand == lo) break;
      if (fits(r0, cand)) {
        lo = cand;
        if (cand == m) break;
        step *= 2;
      } else {
        hi = cand;
        break;
      }
    }
    if (hi > 0) {
      while (hi - lo > 1) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (fits(r0, mid)) lo = mid; else hi = mid;
      }
    }
    aires_tile t;
    t.r0 = r0;
    t.r1 = lo;
    t.nnz0 = arp[r0];
    t.nnz1 = arp[lo];
    t.a_bytes = (lo - r0 + 1) * sA + 8 * (t.nnz1 - t.nnz0);
    t.c_bound_entries = cpre.empty() ? -1 : cpre[(size_t)lo] - cpre[(size_t)r0];
    t.tile_bytes = slot_bytes_fast(r0, lo);
    t.sent_nnz1 = t.nnz1;
    peak_slot = std::max(peak_slot, t.tile_bytes);
    p->tiles.push_back(t);
    r0 = lo;
  }
  if (!a_streamed || o.m_a_bytes > 0) break;  // one slot sized by its rows alone
  int64_t mk = 0, mq = 0, mc = 0;
  for (const aires_tile& t : p->tiles) {
    mk = std::max(mk, t.r1 - t.r0);
    mq = std::max(mq, t.sent_nnz1 - t.nnz0);
    mc = std::max(mc, t.c_bound_entries);
  }
  const int64_t need = mk * per_row_ws + (mk + 1) * sA + 8 * mq + (c_on_host ? 8 * mc + 8 * (mk + 1) : 0);
  peak_slot = std::max(peak_slot, need);
  if (need <= tile_budget) break;
  if (pass >= 32 || part_budget <= need - tile_budget) {
    delete p;
    return fail(AIRES_E_BUDGET, "tile slots of %lld bytes cannot hold the largest tile parts (%lld bytes)",
                (long long)tile_budget, (long long)need);
  }
  part_budget -= need - tile_budget;
  }
  p->info.ntiles = (int64_t)p->tiles.size();
  p->info.part_budget = part_budget;
  p->info.peak_bytes = resident + nslots * peak_slot;
  if (file) {
    p->file = std::move(*file);
    p->info.a_in_file = 1;
  }
  std::memset(&p->stats, 0, sizeof p->stats);
  *out = p;
  return AIRES_OK;
}

}  // namespace

extern "C" {

aires_status aires_tile_plan(const aires_csr* A, const aires_csr* B, uint64_t hbm_budget,
                             const aires_plan_opts* opts, aires_plan** out) {
  return plan_impl(A, B, hbm_budget, opts, out, nullptr);
}

aires_status aires_tile_plan_file(const aires_file_csr* A, const aires_csr* B, uint64_t hbm_budget,
                                  const aires_plan_opts* opts, aires_plan** out) {
  if (!A || !A->path || !out) return fail(AIRES_E_INVALID_ARG, "NULL argument");
  if (A->nrows < 0 || A->ncols < 0 || A->nnz < 0) return fail(AIRES_E_DIM, "A has a negative size");
  if (A->rp_type != AIRES_IDX_I32 && A->rp_type != AIRES_IDX_I64)
    return fail(AIRES_E_INVALID_ARG, "A.rp_type %d invalid", A->rp_type);
  if (A->rp_type == AIRES_IDX_I32 && A->nnz > INT32_MAX)
    return fail(AIRES_E_OVERFLOW, "A.nnz needs int64 row pointers");
  if (A->ncols > INT32_MAX) return fail(AIRES_E_OVERFLOW, "A.ncols exceeds int32 column indices");
  if (A->row_ptr_offset < 0 || A->col_idx_offset < 0 || A->vals_offset < 0)
    return fail(AIRES_E_INVALID_ARG, "negative file offset");
  auto f = std::make_unique<FileSrc>();
  ST_TRY(open_file_src(A->path, A->direct_io, *f));
  f->col_off = A->col_idx_offset;
  f->val_off = A->vals_offset;
  // A's row pointers to host memory (pinned where a device is present:
  // each tile copies its slice from them)
  const int64_t s = A->rp_type == AIRES_IDX_I64 ? 8 : 4;
  const int64_t rp_len = (A->nrows + 1) * s;
  const size_t cap = (size_t)(rp_len + 2 * kIoAlign);
  if (hipHostMalloc(&f->rp_host, cap, hipHostMallocDefault) == hipSuccess) {
    f->rp_pinned = true;
  } else {
    (void)hipGetLastError();
    f->rp_host = std::aligned_alloc((size_t)kIoAlign, (cap + kIoAlign - 1) / kIoAlign * kIoAlign);
    if (!f->rp_host) return fail(AIRES_E_OOM, "host allocation of %zu bytes failed", cap);
  }
  int64_t shift = 0;
  ST_TRY(file_read(*f, A->row_ptr_offset, rp_len, static_cast<char*>(f->rp_host), &shift));
  if (shift) std::memmove(f->rp_host, static_cast<char*>(f->rp_host) + shift, (size_t)rp_len);
  aires_csr a{};
  a.nrows = A->nrows;
  a.ncols = A->ncols;
  a.nnz = A->nnz;
  a.rp_type = A->rp_type;
  a.mem = AIRES_MEM_HOST_PINNED;
  a.row_ptr = f->rp_host;
  const int64_t last = s == 8 ? static_cast<const int64_t*>(f->rp_host)[A->nrows]
                              : (int64_t) static_cast<const int32_t*>(f->rp_host)[A->nrows];
  const int64_t first = s == 8 ? static_cast<const int64_t*>(f->rp_host)[0]
                               : (int64_t) static_cast<const int32_t*>(f->rp_host)[0];
  if (first != 0 || last != A->nnz) return fail(AIRES_E_INVALID_CSR, "A's row pointers in the file do not end at nnz");
  return plan_impl(&a, B, hbm_budget, opts, out, &f);
}

aires_status aires_plan_info(const aires_plan* plan, aires_plan_info_t* info) {
  if (!plan || !info) return fail(AIRES_E_INVALID_ARG, "NULL argument");
  *info = plan->info;
  return AIRES_OK;
}

aires_status aires_plan_info_get(const aires_plan* plan, aires_plan_info_t* info) { return aires_plan_info(plan, info); }

aires_status aires_plan_tile(const aires_plan* plan, int64_t t, aires_tile* tile) {
  if (!plan || !tile) return fail(AIRES_E_INVALID_ARG, "NULL argument");
  if (t < 0 || t >= (int64_t)plan->tiles.size()) return fail(AIRES_E_INVALID_ARG, "tile %lld out of range", (long long)t);
  *tile = plan->tiles[(size_t)t];
  return AIRES_OK;
}

void aires_plan_destroy(aires_plan* plan) { delete plan; }

aires_status aires_csr_read_file(const aires_file_csr* M, int32_t mem, const aires_allocator* alloc, void* stream,
                                 int64_t chunk_bytes, aires_csr_out* out, aires_read_stats* st) {
  if (!M || !M->path || !out) return fail(AIRES_E_INVALID_ARG, "NULL argument");
  if (mem != AIRES_MEM_DEVICE && mem != AIRES_MEM_HOST_PINNED)
    return fail(AIRES_E_INVALID_ARG, "mem %d: AIRES_MEM_DEVICE or AIRES_MEM_HOST_PINNED", mem);
  if (M->nrows < 0 || M->ncols < 0 || M->nnz < 0) return fail(AIRES_E_DIM, "the matrix has a negative size");
  if (M->rp_type != AIRES_IDX_I32 && M->rp_type != AIRES_IDX_I64)
    return fail(AIRES_E_INVALID_ARG, "rp_type %d invalid", M->rp_type);
  if (M->rp_type == AIRES_IDX_I32 && M->nnz > INT32_MAX) return fail(AIRES_E_OVERFLOW, "nnz needs int64 row pointers");
  if (M->ncols > INT32_MAX) return fail(AIRES_E_OVERFLOW, "ncols exceeds int32 column indices");
  if (M->row_ptr_offset < 0 || M->col_idx_offset < 0 || M->vals_offset < 0)
    return fail(AIRES_E_INVALID_ARG, "negative file offset");
  if (chunk_bytes < 0) return fail(AIRES_E_INVALID_ARG, "negative chunk size");
  const int64_t chunk = chunk_bytes > 0 ? (chunk_bytes + kIoAlign - 1) / kIoAlign * kIoAlign : int64_t(64) << 20;
  const auto t0 = std::chrono::steady_clock::now();
  double read_ms = 0;
  FileSrc f;
  ST_TRY(open_file_src(M->path, M->direct_io, f));
  auto timed_read = [&](int64_t off, int64_t len, char* dst) {
    const auto r0 = std::chrono::steady_clock::now();
    int64_t shift = 0;
    const aires_status s = file_read(f, off, len, dst, &shift);
    read_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - r0).count();
    return s;
  };
  // row pointers: read, checked (0 .. nnz, non-decreasing) and widened to int64
  const int64_t n = M->nrows, nnz = M->nnz, s = M->rp_type == AIRES_IDX_I64 ? 8 : 4;
  std::vector<char> rpf((size_t)((n + 1) * s));
  ST_TRY(timed_read(M->row_ptr_offset, (n + 1) * s, rpf.data()));
  std::vector<int64_t> rp((size_t)n + 1);
  std::vector<int64_t> first_drop(17, INT64_MAX);  // per host thread: the first row whose pointer decreases
  parallel_ranges(n + 1, [&](int64_t lo, int64_t hi, int t) {
    for (int64_t i = lo; i < hi; ++i)
      rp[(size_t)i] = s == 8 ? reinterpret_cast<const int64_t*>(rpf.data())[i]
                             : (int64_t) reinterpret_cast<const int32_t*>(rpf.data())[i];
    const int64_t prev = lo > 0 ? (s == 8 ? reinterpret_cast<const int64_t*>(rpf.data())[lo - 1]
                                          : (int64_t) reinterpret_cast<const int32_t*>(rpf.data())[lo - 1])
                                : INT64_MIN;
    for (int64_t i = lo; i < hi; ++i)
      if (rp[(size_t)i] < (i > lo ? rp[(size_t)i - 1] : prev)) {
        first_drop[(size_t)t] = i - 1;
        break;
      }
  });
  if (rp[0] != 0 || rp[(size_t)n] != nnz) return fail(AIRES_E_INVALID_CSR, "row pointers do not run from 0 to nnz");
  const int64_t drop = *std::min_element(first_drop.begin(), first_drop.end());
  if (drop != INT64_MAX) return fail(AIRES_E_INVALID_CSR, "row pointers decrease at row %lld", (long long)drop);
  const hipStream_t hs = (hipStream_t)stream;
  const aires_allocator a = alloc ? *alloc : kDefaultAllocator;
  const bool host = mem == AIRES_MEM_HOST_PINNED;
  int64_t* d_rp = nullptr;
  int32_t* d_col = nullptr;
  float* d_val = nullptr;
  char* stage[2] = {nullptr, nullptr};
  hipEvent_t ev[2] = {nullptr, nullptr};
  auto release = [&](bool keep_out) {
    for (int i = 0; i < 2; ++i) {
      if (stage[i]) (void)hipHostFree(stage[i]);
      if (ev[i]) (void)hipEventDestroy(ev[i]);
    }
    if (keep_out) return;
    void* arr[3] = {d_rp, d_col, d_val};
    for (void* q : arr) {
      if (!q) continue;
      if (host) (void)hipHostFree(q);
      else a.free(a.ctx, q, (void*)hs);
    }
  };
  auto get = [&](int64_t bytes, void** q) {
    bytes = std::max<int64_t>(bytes, 4);  // an empty array is still a block of its own
    if (host) {
      if (hipHostMalloc(q, (size_t)bytes, hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        *q = nullptr;
      }
    } else {
      *q = a.alloc(a.ctx, (size_t)bytes, (void*)hs);
    }
    return *q ? AIRES_OK : fail(AIRES_E_OOM, "allocation of %lld bytes failed", (long long)bytes);
  };
  aires_status rc = get(8 * (n + 1), reinterpret_cast<void**>(&d_rp));
  if (rc == AIRES_OK) rc = get(4 * nnz, reinterpret_cast<void**>(&d_col));
  if (rc == AIRES_OK) rc = get(4 * nnz, reinterpret_cast<void**>(&d_val));
  if (rc != AIRES_OK) {
    release(false);
    return rc;
  }
  int64_t bytes = (n + 1) * s;
  if (host) {
    // straight into the caller's pinned arrays
    std::memcpy(d_rp, rp.data(), (size_t)(8 * (n + 1)));
    if (nnz > 0) rc = timed_read(M->col_idx_offset, 4 * nnz, reinterpret_cast<char*>(d_col));
    if (rc == AIRES_OK && nnz > 0) rc = timed_read(M->vals_offset, 4 * nnz, reinterpret_cast<char*>(d_val));
    bytes += 8 * nnz;
  } else {
    // two pinned staging buffers: chunk c + 1 is read from the file while
    // chunk c is copied to the device
    auto hip_ok = [&](hipError_t e, const char* what) {
      if (e == hipSuccess) return AIRES_OK;
      (void)hipGetLastError();
      return fail(AIRES_E_HIP, "%s: %s", what, hipGetErrorString(e));
    };
    for (int i = 0; i < 2 && rc == AIRES_OK; ++i) {
      rc = hip_ok(hipHostMalloc(reinterpret_cast<void**>(&stage[i]), (size_t)chunk, hipHostMallocDefault), "hipHostMalloc");
      if (rc == AIRES_OK) rc = hip_ok(hipEventCreateWithFlags(&ev[i], hipEventDisableTiming), "hipEventCreate");
    }
    int64_t c = 0;
    auto send = [&](const char* src_host, int64_t len, char* dst_dev, int64_t file_off) {
      for (int64_t o = 0; o < len && rc == AIRES_OK; o += chunk, ++c) {
        const int64_t l = std::min(chunk, len - o);
        char* buf = stage[c & 1];
        if (c >= 2) rc = hip_ok(hipEventSynchronize(ev[c & 1]), "hipEventSynchronize");  // its last copy is done
        if (rc != AIRES_OK) break;
        if (src_host) std::memcpy(buf, src_host + o, (size_t)l);
        else rc = timed_read(file_off + o, l, buf);
        if (rc == AIRES_OK) rc = hip_ok(hipMemcpyAsync(dst_dev + o, buf, (size_t)l, hipMemcpyHostToDevice, hs), "hipMemcpyAsync");
        if (rc == AIRES_OK) rc = hip_ok(hipEventRecord(ev[c & 1], hs), "hipEventRecord");
      }
    };
    if (rc == AIRES_OK) send(reinterpret_cast<const char*>(rp.data()), 8 * (n + 1), reinterpret_cast<char*>(d_rp), 0);
    if (rc == AIRES_OK) send(nullptr, 4 * nnz, reinterpret_cast<char*>(d_col), M->col_idx_offset);
    if (rc == AIRES_OK) send(nullptr, 4 * nnz, reinterpret_cast<char*>(d_val), M->vals_offset);
    const aires_status sync = hip_ok(hipStreamSynchronize(hs), "hipStreamSynchronize");  // staging is freed next
    if (rc == AIRES_OK) rc = sync;
    bytes += 8 * nnz;
  }
  if (rc != AIRES_OK) {
    release(false);
    return rc;
  }
  release(true);
  std::memset(out, 0, sizeof *out);
  out->nrows = n;
  out->ncols = M->ncols;
  out->nnz = nnz;
  out->row_ptr = d_rp;
  out->col_idx = d_col;
  out->vals = d_val;
  out->mem = mem;
  out->_owner = new OutOwner{a, hs, host ? 1 : 0};
  if (st) {
    st->bytes_read = bytes;
    st->read_ms = read_ms;
    st->total_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  }
  return AIRES_OK;
}

}  // extern "C"

// ------------------------------------------------------------- execution

namespace {

struct Timer {
  aires_plan* p;
  hipStream_t s;
  bool on;
  int tile = -1;  // tile the next marks belong to
  int record() {
    if (!on) return -1;
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) { on = false; return -1; }
    (void)hipEventRecord(e, s);
    p->ev.push_back(e);
    return (int)p->ev.size() - 1;
  }
  // event e as moment `which` of the current tile (first setting wins for
  // a beginning, last for an end)
  void at(int which, int e) {
    if (!on || e < 0 || tile < 0 || (size_t)tile >= p->tev.size()) return;
    int& slot = p->tev[(size_t)tile][(size_t)which];
    const bool begin = which == aires_plan::T_H2D0 || which == aires_plan::T_C0 || which == aires_plan::T_D2H0;
    if (!begin || slot < 0) slot = e;
  }
  void mark(int kind, int phase, int a, int b) {
    if (on && a >= 0 && b >= 0) p->marks.push_back({kind, phase, a, b, tile});
  }
};

void reset_timing(aires_plan* p) {
  for (hipEvent_t e : p->ev) (void)hipEventDestroy(e);
  p->ev.clear();
  p->marks.clear();
}

// 32-bit words of B's grain index, bidx[k * (nG + 1) + g], followed by
// max_j |b_kj| per B row (fp32), both built once per call for wide products.
int64_t index_words(const aires_plan* p) { return ((int64_t)p->nG + 2) * p->B.nrows; }

float* index_bmax(const aires_plan* p, int32_t* bidx) {
  return reinterpret_cast<float*>(bidx + ((int64_t)p->nG + 1) * p->B.nrows);
}

kern::Operands tile_operands(const aires_plan* p, const void* arp, int64_t a_base, const int32_t* acol,
                             const float* aval, const void* brp, const int32_t* bcol, const float* bval,
                             const int32_t* bidx) {
  kern::Operands op;
  op.arp = arp;
  op.rpa64 = p->A.rp_type == AIRES_IDX_I64;
  op.a_base = a_base;
  op.acol = acol;
  op.aval = aval;
  op.brp = brp;
  op.rpb64 = p->B.rp_type == AIRES_IDX_I64;
  op.bcol = bcol;
  op.bval = bval;
  op.K = p->B.nrows;
  op.N = p->B.ncols;
  op.bidx = p->wide ? bidx : nullptr;
  op.G = p->G;
  op.nG = p->nG;
  // max |b| per B row, stored after the grain index (index_words)
  op.bmax = p->wide && bidx ? reinterpret_cast<const float*>(bidx + ((int64_t)p->nG + 1) * p->B.nrows) : nullptr;
  return op;
}

// Phase markers for the stats: kinds >= 100 are whole phases.
enum { PH_ANALYZE = 100, PH_BIN, PH_SYMBOLIC, PH_SCAN, PH_NUMERIC, PH_H2D, PH_D2H, PH_TOTAL, PH_INDEX,
       PH_PIPELINE };

// Device workspace of one tile (tile-local rows).
struct TileWs {
  int64_t* P = nullptr;          // [n] intermediate products per row
  int32_t* list = nullptr;       // [n] rows grouped by bin (long-row list during analysis)
  int32_t* binoff = nullptr;     // [MAX_BINS + 1]
  int32_t* cntcur = nullptr;     // [2 * MAX_BINS + 1] bin counts, cursors, long-row count
  int32_t* gcnt = nullptr;       // [n * nG] entries per (row, grain)     (wide)
  int64_t* icount = nullptr;     // [n + 1] windows per bin row, scanned  (wide)
  kern::WinItem* items = nullptr;
  int64_t nitems = 0;            // host copy of icount[n]
  int32_t* wcounter = nullptr;   // row counters of the window kernels (shared, then one per column slab)
  void* scan_ws = nullptr;
  kern::SplitWs split{nullptr, nullptr, 0};  // dense slots of split rows (shared by all tiles)
  int64_t* bm_off = nullptr;     // [n * ngg] kept bitmaps of the symbolic items (wide, in-core)
  uint32_t* bm_cache = nullptr;  // shared bitmap cache (nullptr: none)
  int64_t bm_cap = 0;
  unsigned long long* bm_top = nullptr;
  bool item_cut = false;          // the call started with a bitmap cache (window cuts of kept rows)
};

// with_list_gcnt: the per-row arrays (products, bin list, grain and window
// counts) for n rows; without, the caller points them into arrays of its own
aires_status alloc_tile_ws(aires_plan* p, DevPool& ws, int64_t n, bool with_list_gcnt, TileWs& w) {
  if (with_list_gcnt) {
    ST_TRY(ws.get_n(n, &w.P));
    ST_TRY(ws.get_n(n, &w.list));
    if (p->wide) {
      ST_TRY(ws.get_n(n * (int64_t)p->nG, &w.gcnt));
      ST_TRY(ws.get_n(n + 1, &w.icount));
    }
    ST_TRY(ws.get_n(kern::MAX_BINS + 1, &w.binoff));
  }
  ST_TRY(ws.get_n(2 * kern::MAX_BINS + 1, &w.cntcur));
  ST_TRY(ws.get_n(1 + kern::WIN_MAX_SLABS, &w.wcounter));
  ST_TRY(ws.get(kern::scan_workspace_bytes(n), &w.scan_ws));
  return AIRES_OK;
}

aires_status alloc_split_ws(aires_plan* p, DevPool& ws, kern::SplitWs& sw) {
  sw = kern::SplitWs{nullptr, nullptr, 0};
  if (!p->split) return AIRES_OK;
  const int64_t N = p->B.ncols;
  int64_t cap = p->split_cap;
  if (ws.arena) {
    // a fixed workspace gives slots to as many split rows as fit in what is
    // left of it; the other rows of the bin take a workgroup each
    const int64_t per = 4 * ((N + 31) / 32) + 4 * N;
    cap = std::min(cap, (ws.left() - 1024) / per);
    if (cap < 1) return fail(AIRES_E_CAPACITY, "no room for a split-row slot in the fixed scratch array");
  }
  ST_TRY(ws.get_n(cap * ((N + 31) / 32), &sw.bm));
  ST_TRY(ws.get_n(cap * N, &sw.acc));
  sw.cap = cap;
  return AIRES_OK;
}

kern::WindowParams window_params(const aires_plan* p, const TileWs& w) {
  kern::WindowParams wp;
  wp.gcnt = w.gcnt;
  wp.grains_per_count_item = p->count_grains;
  wp.max_grains = p->win_grains;
  wp.max_entries = p->win_entries;
  wp.pool_words = p->win_pool_words;
  wp.item_count = w.icount;
  wp.items = w.items;
  wp.row_counter = w.wcounter;
  wp.bm_cache = w.bm_cache;
  wp.bm_cap = w.bm_cap;
  wp.bm_top = w.bm_top;
  wp.bm_off = w.bm_off;
  wp.P = w.P;
  wp.bm_min_products = p->keep_bitmap;
  wp.item_cut = w.item_cut ? 1 : 0;
  wp.slab_bin = p->slab_bin;
  wp.nslab = 1;  // set at the numeric launch from its grid
  return wp;
}

// analyze + bin + symbolic + scan of one tile; counts land in crp[1..n] and
// are scanned in place on top of crp[0].  Wide rows also get their window
// counts scanned into w.icount.
aires_status tile_symbolic(aires_plan* p, const kern::Operands& op, int64_t n, TileWs& w, int64_t* crp,
                           unsigned long long* prod_total, hipStream_t s, Timer& tm) {
  const int e0 = tm.record();
  tm.at(aires_plan::T_C0, e0);
  HIP_TRY(hipMemsetAsync(w.cntcur, 0, sizeof(int32_t) * (2 * kern::MAX_BINS + 1), s));
  HIP_TRY(kern::analyze(op, n, w.P, prod_total, w.cntcur + 2 * kern::MAX_BINS, w.list, s));
  const int e1 = tm.record();
  HIP_TRY(kern::bin_rows(w.P, n, p->th, w.cntcur, w.binoff, w.list, s));
  HIP_TRY(hipMemsetAsync(crp + 1, 0, sizeof(int64_t) * (size_t)std::max<int64_t>(n, 0), s));
  if (p->wide) HIP_TRY(hipMemsetAsync(w.icount, 0, sizeof(int64_t) * (size_t)(n + 1), s));
  const int e2 = tm.record();
  kern::Outputs out{};
  out.counts = crp + 1;
  for (int b = 0; b < p->th.nb; ++b) {
    const int kind = p->th.kind[b];
    if (kind == kern::KIND_EMPTY) continue;
    kern::BinView bv{w.list, w.binoff, b};
    const int ka = tm.record();
    if (kind == kern::KIND_WINDOWS) {
      // all window bins (consecutive) as one range
      while (bv.last() + 1 < p->th.nb && p->th.kind[bv.last() + 1] == kern::KIND_WINDOWS) bv.bin_last = bv.last() + 1;
      HIP_TRY(kern::windows_symbolic(op, bv, window_params(p, w), out, n, s));
      b = bv.last();
    } else if (kind == kern::KIND_DENSE_SPLIT) {
      HIP_TRY(kern::split_rows(0, op, bv, w.split, out, n, s));
    } else {
      HIP_TRY(kern::run_bin(kind, 0, op, bv, out, n, s));
    }
    tm.mark(kind, 0, ka, tm.record());
  }
  const int e3 = tm.record();
  HIP_TRY(kern::scan_inplace(crp + 1, n, w.scan_ws, s));
  if (p->wide) HIP_TRY(kern::scan_inplace(w.icount + 1, n, w.scan_ws, s));
  const int e4 = tm.record();
  tm.mark(PH_ANALYZE, 0, e0, e1);
  tm.mark(PH_BIN, 0, e1, e2);
  tm.mark(PH_SYMBOLIC, 0, e2, e3);
  tm.mark(PH_SCAN, 0, e3, e4);
  return AIRES_OK;
}

aires_status tile_numeric(aires_plan* p, const kern::Operands& op, int64_t n, const TileWs& w, const int64_t* crp,
                          int32_t* ccol, float* cval, int64_t c_base, hipStream_t s, Timer& tm) {
  kern::Outputs out{};
  out.crp = crp;
  out.ccol = ccol - c_base;
  out.cval = cval - c_base;
  const int e0 = tm.record();
  for (int b = 0; b < p->th.nb; ++b) {
    const int kind = p->th.kind[b];
    if (kind == kern::KIND_EMPTY) continue;
    kern::BinView bv{w.list, w.binoff, b};
    const int ka = tm.record();
    if (kind == kern::KIND_WINDOWS) {
      while (bv.last() + 1 < p->th.nb && p->th.kind[bv.last() + 1] == kern::KIND_WINDOWS) bv.bin_last = bv.last() + 1;
      HIP_TRY(kern::windows_numeric(op, bv, window_params(p, w), out, n, w.nitems, s));
      b = bv.last();
    } else if (kind == kern::KIND_DENSE_SPLIT) {
      HIP_TRY(kern::split_rows(1, op, bv, w.split, out, n, s));
    } else {
      HIP_TRY(kern::run_bin(kind, 1, op, bv, out, n, s));
    }
    tm.mark(kind, 1, ka, tm.record());
    p->stats.numeric_launches++;
  }
  const int e1 = tm.record();
  tm.mark(PH_NUMERIC, 1, e0, e1);
  tm.at(aires_plan::T_C1, e1);
  return AIRES_OK;
}

// Device bytes of the caller's inputs that the call reads in place; the
// budget covers them, so the library's own allocations get the rest.
int64_t borrowed_device_bytes(const aires_plan* p) {
  int64_t b = 0;
  if (p->A.mem == AIRES_MEM_DEVICE) {
    b += (p->A.nrows + 1) * rp_bytes(p->A) + 4 * p->A.nnz;
    if (p->opts.a_values != AIRES_AVALUES_SYM_NORM) b += 4 * p->A.nnz;
  }
  if (p->B.mem == AIRES_MEM_DEVICE) b += csr_bytes(p->B);
  return b;
}

aires_status begin_call(aires_plan* p, aires_csr_out* C) {
  if (!p || !C) return fail(AIRES_E_INVALID_ARG, "NULL argument");
  if (p->busy) return fail(AIRES_E_STATE, "plan is in use");
  if (C->row_ptr || C->col_idx || C->vals || C->_owner)
    return fail(AIRES_E_STATE, "output descriptor is not zeroed (free it first)");
  std::memset(&p->stats, 0, sizeof p->stats);
  p->stats.ntiles = (int64_t)p->tiles.size();
  p->trun.assign(p->tiles.size(), aires_plan::TileRun{0, 0, 0, 0, 0, 0.0, 0.0});
  reset_timing(p);
  std::array<int, aires_plan::T_NEV> none;
  none.fill(-1);
  p->tev.assign(p->tiles.size(), none);
  p->ev_base = -1;
  return AIRES_OK;
}

// C arrays the caller owns (the allocation-free entry point).
struct CallerC {
  int64_t* row_ptr;
  int32_t* col;
  float* val;
  int64_t capacity;
  int64_t* nnz_out;
};

// In-core call (device-resident A and B).  Workspace comes from `ws`: the
// plan's allocator under its budget, or a fixed arena.  C is allocated and
// handed to *C, or written into the caller's arrays (cc != nullptr).
aires_status spgemm_device_in(aires_plan* p, hipStream_t s, DevPool& ws, aires_csr_out* C, const CallerC* cc) {
  const int64_t m = p->A.nrows, K = p->B.nrows, N = p->B.ncols;
  const int64_t sA = rp_bytes(p->A);
  Timer tm{p, s, p->opts.timing != 0};
  const int e_total0 = tm.record();
  p->ev_base = e_total0;
  int64_t max_rows = 1;
  for (const auto& t : p->tiles) max_rows = std::max(max_rows, t.r1 - t.r0);
  const int64_t nt = (int64_t)p->tiles.size();

  // Workspace: P, counters and scan partials are reused by every tile; row
  // lists, bin offsets and window bookkeeping persist from the symbolic
  // sweep to the numeric sweep (tile regions of whole-matrix arrays).
  int64_t* crp = nullptr;
  if (cc) crp = cc->row_ptr;
  else ST_TRY(ws.get_n(m + 1, &crp));
  TileWs shared;
  ST_TRY(alloc_tile_ws(p, ws, max_rows, false, shared));
  int32_t *list = nullptr, *binoff = nullptr, *gcnt = nullptr, *bidx = nullptr;
  int64_t* icount = nullptr;
  unsigned long long* prod = nullptr;
  ST_TRY(ws.get_n(m, &list));
  // products per row for all rows: the numeric sweep of tile t reads the
  // values its symbolic sweep wrote (which rows keep their bitmaps), after
  // the symbolic sweeps of the later tiles
  int64_t* P_all = nullptr;
  ST_TRY(ws.get_n(m, &P_all));
  ST_TRY(ws.get_n(nt * (kern::MAX_BINS + 1), &binoff));
  ST_TRY(ws.get_n(nt, &prod));  // intermediate products of each tile
  // A's values: given, or derived from its pattern (Eq. 2) into the workspace
  const float* avals = p->A.vals;
  if (p->opts.a_values == AIRES_AVALUES_SYM_NORM && p->A.nnz > 0) {
    float* v = nullptr;
    ST_TRY(ws.get_n(p->A.nnz, &v));
    HIP_TRY(kern::sym_norm_values(p->A.row_ptr, p->A.rp_type == AIRES_IDX_I64, 0, m, 0, p->A.col_idx, v, p->A.nnz,
                                  s));
    avals = v;
  }
  int64_t* bm_off = nullptr;
  uint32_t* bm_cache = nullptr;
  unsigned long long* bm_top = nullptr;
  int64_t bm_cap = 0;
  if (p->wide) {
    ST_TRY(ws.get_n(m * (int64_t)p->nG, &gcnt));
    ST_TRY(ws.get_n(m + nt, &icount));
    ST_TRY(ws.get_n(index_words(p), &bidx));
    if (p->keep_bitmap >= 0 && !ws.arena) {
      ST_TRY(ws.get_n(m * (int64_t)p->ngg, &bm_off));
      ST_TRY(ws.get_n(1, &bm_top));
      // The kept bitmaps are a cache: they take up to a fifth of the budget
      // the plan leaves free; items that do not fit are marked again by the
      // numeric phase, and the cache is dropped if C then does not fit.
      const int64_t spare = p->budget - p->info.peak_bytes;
      const int64_t cache_max = p->opts.bitmap_cache_bytes > 0 ? p->opts.bitmap_cache_bytes : kBitmapCacheBytes;
      bm_cap = spare > 0 ? std::min<int64_t>(spare / 5, cache_max) / (int64_t)sizeof(uint32_t) : 0;
      const int64_t words_all = m * (int64_t)p->nG * (p->G / 32);  // every row's bitmaps
      if (words_all / std::max<int64_t>(m, 1) == (int64_t)p->nG * (p->G / 32)) bm_cap = std::min(bm_cap, words_all);
      if (bm_cap > 0 && ws.get_n(bm_cap, &bm_cache) != AIRES_OK) {
        bm_cache = nullptr;
        bm_cap = 0;
      }
    }
  }
  const bool item_cut = bm_cache != nullptr;  // kept for the call, even if the cache is released later
  ST_TRY(alloc_split_ws(p, ws, shared.split));
  auto tile_ws = [&](int64_t t) {
    const aires_tile& T = p->tiles[(size_t)t];
    TileWs w = shared;
    w.P = P_all + T.r0;
    w.item_cut = item_cut;
    w.list = list + T.r0;
    w.binoff = binoff + t * (kern::MAX_BINS + 1);
    if (p->wide) {
      w.gcnt = gcnt + T.r0 * (int64_t)p->nG;
      w.icount = icount + T.r0 + t;
      if (bm_cache) {
        w.bm_cache = bm_cache;
        w.bm_cap = bm_cap;
        w.bm_top = bm_top;
        w.bm_off = bm_off + T.r0 * (int64_t)p->ngg;
      }
    }
    return w;
  };
  HIP_TRY(hipMemsetAsync(crp, 0, sizeof(int64_t), s));
  HIP_TRY(hipMemsetAsync(prod, 0, sizeof(unsigned long long) * (size_t)std::max<int64_t>(nt, 1), s));
  if (bm_cache) HIP_TRY(hipMemsetAsync(bm_top, 0, sizeof(unsigned long long), s));
  if (p->wide) {
    const int ea = tm.record();
    HIP_TRY(kern::build_window_index(p->B.row_ptr, p->B.rp_type == AIRES_IDX_I64, p->B.col_idx, p->B.vals, K, p->G,
                                     p->nG, bidx, index_bmax(p, bidx), s));
    tm.mark(PH_INDEX, 0, ea, tm.record());
  }

  // Sweep 1: symbolic phase of every tile; C.row_ptr grows tile by tile.
  for (int64_t t = 0; t < nt; ++t) {
    const aires_tile& T = p->tiles[(size_t)t];
    TileWs w = tile_ws(t);
    const void* arp = static_cast<const char*>(p->A.row_ptr) + T.r0 * sA;
    kern::Operands op = tile_operands(p, arp, 0, p->A.col_idx, avals, p->B.row_ptr, p->B.col_idx,
                                      p->B.vals, bidx);
    tm.tile = (int)t;
    ST_TRY(tile_symbolic(p, op, T.r1 - T.r0, w, crp + T.r0, prod + t, s, tm));
  }
  tm.tile = -1;
  // The one host synchronisation: nnz(C) (and the window count of every
  // tile) decide the allocations.  Host buffer: [0, nt) products per tile,
  // [nt, 2nt) C.row_ptr at each tile's end, [2nt, 3nt) windows per tile.
  std::vector<int64_t> hostbuf(3 * (size_t)std::max<int64_t>(nt, 1));
  int64_t* hb = hostbuf.data();
  int64_t* hb_end = hb + nt;
  int64_t* hb_win = hb + 2 * nt;
  if (nt > 0) HIP_TRY(hipMemcpyAsync(hb, prod, sizeof(int64_t) * (size_t)nt, hipMemcpyDeviceToHost, s));
  for (int64_t t = 0; t < nt; ++t) {
    const aires_tile& T = p->tiles[(size_t)t];
    HIP_TRY(hipMemcpyAsync(hb_end + t, crp + T.r1, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    if (p->wide)
      HIP_TRY(hipMemcpyAsync(hb_win + t, icount + T.r0 + t + (T.r1 - T.r0), sizeof(int64_t), hipMemcpyDeviceToHost,
                             s));
  }
  HIP_TRY(hipStreamSynchronize(s));
  const int64_t nnz = nt > 0 ? hb_end[nt - 1] : 0;
  if (cc && cc->nnz_out) *cc->nnz_out = nnz;
  p->stats.host_syncs = 1;
  p->stats.nnz_c = nnz;
  for (int64_t t = 0; t < nt; ++t) {
    p->stats.products += hb[t];
    p->trun[(size_t)t].products = hb[t];
    p->trun[(size_t)t].nnz_c = hb_end[t] - (t > 0 ? hb_end[t - 1] : 0);
  }
  kern::WinItem* items = nullptr;
  std::vector<int64_t> item_base((size_t)nt + 1, 0);
  if (p->wide)
    for (int64_t t = 0; t < nt; ++t) item_base[(size_t)t + 1] = item_base[(size_t)t] + hb_win[t];
  // C and the window list next to everything the call holds must fit the
  // budget; the kept bitmaps are a cache and go first if they do not
  const int64_t need = 8 * std::max<int64_t>(nnz, 1) + (int64_t)sizeof(kern::WinItem) *
                                                          (p->wide ? std::max<int64_t>(item_base[(size_t)nt], 1) : 0);
  if (bm_cache && !ws.fits(need)) {
    // the numeric phase then marks every window from the products
    ws.give_back(bm_cache);
    bm_cache = nullptr;
    bm_cap = 0;
  }
  int32_t* ccol = nullptr;
  float* cval = nullptr;
  if (cc) {
    if (nnz > cc->capacity)
      return fail(AIRES_E_CAPACITY, "C has %lld entries; the caller's arrays hold %lld (C.row_ptr is written)",
                  (long long)nnz, (long long)cc->capacity);
    ccol = cc->col;
    cval = cc->val;
  } else {
    if (!ws.fits(need))
      return fail(AIRES_E_BUDGET,
                  "C needs %lld bytes (and its window list %lld); the budget of %lld bytes leaves %lld",
                  (long long)(8 * nnz), (long long)(need - 8 * nnz), (long long)p->budget,
                  (long long)(ws.cap - ws.used));
    ST_TRY(ws.get_n(nnz, &ccol));
    ST_TRY(ws.get_n(nnz, &cval));
  }
  if (p->wide) ST_TRY(ws.get_n(item_base[(size_t)nt], &items));

  // Sweep 2: numeric phase of every tile.
  for (int64_t t = 0; t < nt; ++t) {
    const aires_tile& T = p->tiles[(size_t)t];
    TileWs w = tile_ws(t);
    if (p->wide) {
      w.items = items + item_base[(size_t)t];
      w.nitems = hb_win[t];
    }
    const void* arp = static_cast<const char*>(p->A.row_ptr) + T.r0 * sA;
    kern::Operands op = tile_operands(p, arp, 0, p->A.col_idx, avals, p->B.row_ptr, p->B.col_idx,
                                      p->B.vals, bidx);
    tm.tile = (int)t;
    ST_TRY(tile_numeric(p, op, T.r1 - T.r0, w, crp + T.r0, ccol, cval, 0, s, tm));
  }
  tm.tile = -1;
  tm.mark(PH_TOTAL, 0, e_total0, tm.record());
  if (cc) return AIRES_OK;

  // hand C to the caller
  ws.detach(crp);
  ws.detach(ccol);
  ws.detach(cval);
  auto* own = new OutOwner{p->alloc, s, 0};
  C->nrows = m;
  C->ncols = N;
  C->nnz = nnz;
  C->row_ptr = crp;
  C->col_idx = ccol;
  C->vals = cval;
  C->mem = AIRES_MEM_DEVICE;
  C->_owner = own;
  return AIRES_OK;  // ws releases the workspace stream-ordered on s
}

aires_status spgemm_device(aires_plan* p, hipStream_t s, aires_csr_out* C) {
  DevPool ws(p->alloc, s, p->budget - borrowed_device_bytes(p));
  return spgemm_device_in(p, s, ws, C, nullptr);
}

// Out-of-core schedule (Algorithm 2): B resident (Phase I), A tiles
// double-buffered host->device (Phase II), C tiles device->host (Phase III).
aires_status stream_impl(aires_plan* p, hipStream_t sh, hipStream_t sc, hipStream_t sd, aires_csr_out* C) {
  const aires_csr& A = p->A;
  const aires_csr& B = p->B;
  const int64_t m = A.nrows, K = B.nrows, N = B.ncols;
  const int64_t sA = rp_bytes(A), sB = rp_bytes(B);
  const int c_on_host = p->opts.c_placement == AIRES_MEM_HOST_PINNED;
  if (A.mem != AIRES_MEM_HOST_PINNED) return fail(AIRES_E_UNSUPPORTED, "streaming needs A in pinned host memory");
  if (B.mem == AIRES_MEM_HOST) return fail(AIRES_E_UNSUPPORTED, "B in pageable host memory");
  if (p->info.c_bound_entries < 0) return fail(AIRES_E_STATE, "plan has no C bound (Algorithm 1 planning mode)");
  Timer tm{p, sc, p->opts.timing != 0};
  const int e_total0 = tm.record();
  p->ev_base = e_total0;
  DevPool ws(p->alloc, sc, p->budget - borrowed_device_bytes(p));
  const int64_t nt = (int64_t)p->tiles.size();
  const bool maxfill = p->opts.segmentation == AIRES_SEG_MAXFILL;
  FileSrc* file = p->file.get();
  int64_t max_rows = 1, max_q = 1, max_cb = 1, max_carry = 1;
  for (const auto& t : p->tiles) {
    max_rows = std::max(max_rows, t.r1 - t.r0);
    max_q = std::max(max_q, t.sent_nnz1 - t.nnz0);
    max_cb = std::max(max_cb, t.c_bound_entries);
    max_carry = std::max(max_carry, t.sent_nnz1 - t.nnz1);
  }
  int64_t cap = p->info.c_bound_entries;  // grows when the bound was only an estimate (Eq. 5)

  // output arrays
  int64_t* C_rp = nullptr;
  int32_t* C_col = nullptr;
  float* C_val = nullptr;
  struct HostBufs {
    std::vector<void*> v;
    ~HostBufs() { for (void* x : v) (void)hipHostFree(x); }
  } hb;
  // Destroyed first on every exit: no copy or kernel may still touch the
  // workspace or host buffers when they are released.
  struct Drain {
    hipStream_t a, b, c;
    ~Drain() { (void)hipStreamSynchronize(a); (void)hipStreamSynchronize(b); (void)hipStreamSynchronize(c); }
  } drain{sh, sc, sd};
  if (c_on_host) {
    HIP_TRY(hipHostMalloc((void**)&C_rp, sizeof(int64_t) * (size_t)(m + 1), hipHostMallocDefault));
    hb.v.push_back(C_rp);
    HIP_TRY(hipHostMalloc((void**)&C_col, sizeof(int32_t) * (size_t)std::max<int64_t>(cap, 1), hipHostMallocDefault));
    hb.v.push_back(C_col);
    HIP_TRY(hipHostMalloc((void**)&C_val, sizeof(float) * (size_t)std::max<int64_t>(cap, 1), hipHostMallocDefault));
    hb.v.push_back(C_val);
  } else {
    ST_TRY(ws.get_n(m + 1, &C_rp));
    ST_TRY(ws.get_n(cap, &C_col));
    ST_TRY(ws.get_n(cap, &C_val));
  }

  // Phase I: B resident on the device
  const void* brp = B.row_ptr;
  const int32_t* bcol = B.col_idx;
  const float* bval = B.vals;
  void *d_brp = nullptr, *d_bcol = nullptr, *d_bval = nullptr;
  if (B.mem != AIRES_MEM_DEVICE) {
    ST_TRY(ws.get((size_t)(K + 1) * sB, &d_brp));
    ST_TRY(ws.get((size_t)std::max<int64_t>(B.nnz, 1) * 4, &d_bcol));
    ST_TRY(ws.get((size_t)std::max<int64_t>(B.nnz, 1) * 4, &d_bval));
  }

  // two slots of everything a tile needs on the device
  struct Slot {
    void* arp; int32_t* acol; float* aval;
    TileWs w;
    int64_t* crp; int32_t* ccol; float* cval; int64_t ccap;
    int64_t icap;
  } slot[2];
  int32_t* bidx = nullptr;
  unsigned long long* prod = nullptr;
  int64_t* running = nullptr;
  ST_TRY(ws.get_n(nt, &prod));  // intermediate products of each tile
  ST_TRY(ws.get_n(1, &running));
  if (p->wide) ST_TRY(ws.get_n(index_words(p), &bidx));
  kern::SplitWs split{nullptr, nullptr, 0};
  ST_TRY(alloc_split_ws(p, ws, split));
  for (int s = 0; s < 2; ++s) {
    Slot& S = slot[s];
    S = Slot{};
    ST_TRY(ws.get((size_t)(max_rows + 1) * sA, &S.arp));
    ST_TRY(ws.get_n(max_q, &S.acol));
    ST_TRY(ws.get_n(max_q, &S.aval));
    ST_TRY(alloc_tile_ws(p, ws, max_rows, true, S.w));
    S.w.split = split;
    ST_TRY(ws.get_n(max_rows + 1, &S.crp));
    if (c_on_host) {
      ST_TRY(ws.get_n(max_cb, &S.ccol));
      ST_TRY(ws.get_n(max_cb, &S.cval));
      S.ccap = max_cb;
    }
  }
  // max-fill segments: two pinned staging buffers a segment is packed into
  // (the head of the partial row returned by the previous segment, then
  // the new entries) and the pinned buffer the partial row returns to
  int32_t* stage_col[2] = {nullptr, nullptr};
  float* stage_val[2] = {nullptr, nullptr};
  int32_t* carry_col = nullptr;
  float* carry_val = nullptr;
  // (A in a file: the staging buffers take each tile's entries as read,
  // with room for the whole 4 KiB blocks of direct reads)
  int64_t shift_col[2] = {0, 0}, shift_val[2] = {0, 0};
  if (maxfill || file) {
    const size_t sb = sizeof(int32_t) * (size_t)max_q + (file ? 2 * kIoAlign : 0);
    for (int b = 0; b < 2; ++b) {
      HIP_TRY(hipHostMalloc((void**)&stage_col[b], sb, hipHostMallocDefault));
      hb.v.push_back(stage_col[b]);
      HIP_TRY(hipHostMalloc((void**)&stage_val[b], sb, hipHostMallocDefault));
      hb.v.push_back(stage_val[b]);
    }
  }
  if (maxfill) {
    HIP_TRY(hipHostMalloc((void**)&carry_col, sizeof(int32_t) * (size_t)max_carry, hipHostMallocDefault));
    hb.v.push_back(carry_col);
    HIP_TRY(hipHostMalloc((void**)&carry_val, sizeof(float) * (size_t)max_carry, hipHostMallocDefault));
    hb.v.push_back(carry_val);
  }
  int64_t* cnt_host = nullptr;  // pinned per-tile (running nnz, windows, products)
  HIP_TRY(hipHostMalloc((void**)&cnt_host, sizeof(int64_t) * 3 * (size_t)std::max<int64_t>(nt, 1), hipHostMallocDefault));
  hb.v.push_back(cnt_host);
  HIP_TRY(hipMemsetAsync(prod, 0, sizeof(unsigned long long) * (size_t)std::max<int64_t>(nt, 1), sc));
  HIP_TRY(hipMemsetAsync(running, 0, sizeof(int64_t), sc));

  std::vector<hipEvent_t> evs;
  struct EvGuard {
    std::vector<hipEvent_t>& v;
    ~EvGuard() { for (hipEvent_t e : v) (void)hipEventDestroy(e); }
  } eg{evs};
  auto mkev = [&](hipEvent_t* e) -> aires_status {
    HIP_TRY(hipEventCreateWithFlags(e, hipEventDisableTiming));
    evs.push_back(*e);
    return AIRES_OK;
  };
  std::vector<hipEvent_t> ev_in(nt), ev_cnt(nt), ev_done(nt), ev_carry(maxfill ? nt : 0);
  hipEvent_t ev_cfree[2] = {nullptr, nullptr};
  for (int64_t t = 0; t < nt; ++t) {
    ST_TRY(mkev(&ev_in[(size_t)t]));
    ST_TRY(mkev(&ev_cnt[(size_t)t]));
    ST_TRY(mkev(&ev_done[(size_t)t]));
    if (maxfill) ST_TRY(mkev(&ev_carry[(size_t)t]));
  }
  ST_TRY(mkev(&ev_cfree[0]));
  ST_TRY(mkev(&ev_cfree[1]));
  hipEvent_t ev_ws;  // workspace allocations (on sc) complete before h2d uses them
  ST_TRY(mkev(&ev_ws));
  HIP_TRY(hipEventRecord(ev_ws, sc));
  HIP_TRY(hipStreamWaitEvent(sh, ev_ws, 0));
  Timer th{p, sh, tm.on}, td{p, sd, tm.on};  // copy-stream busy time
  const int e_pipe0 = th.record();
  if (B.mem != AIRES_MEM_DEVICE) {
    const int eb0 = th.record();
    HIP_TRY(hipMemcpyAsync(d_brp, B.row_ptr, (size_t)(K + 1) * sB, hipMemcpyHostToDevice, sh));
    HIP_TRY(hipMemcpyAsync(d_bcol, B.col_idx, (size_t)B.nnz * 4, hipMemcpyHostToDevice, sh));
    HIP_TRY(hipMemcpyAsync(d_bval, B.vals, (size_t)B.nnz * 4, hipMemcpyHostToDevice, sh));
    th.mark(PH_H2D, 0, eb0, th.record());
    p->stats.h2d_bytes += (K + 1) * sB + 8 * B.nnz;
    brp = d_brp;
    bcol = (const int32_t*)d_bcol;
    bval = (const float*)d_bval;
  }

  // Derived values (Eq. 2): all of A's row pointers stay on the device (they
  // give every row's length); a tile then sends only its column indices.
  const bool sym_norm = p->opts.a_values == AIRES_AVALUES_SYM_NORM;
  void* d_arp_all = nullptr;
  if (sym_norm) {
    ST_TRY(ws.get((size_t)(m + 1) * sA, &d_arp_all));
    HIP_TRY(hipEventRecord(ev_ws, sc));
    HIP_TRY(hipStreamWaitEvent(sh, ev_ws, 0));
    const int ea = th.record();
    HIP_TRY(hipMemcpyAsync(d_arp_all, A.row_ptr, (size_t)(m + 1) * sA, hipMemcpyHostToDevice, sh));
    th.mark(PH_H2D, 0, ea, th.record());
    p->stats.h2d_bytes += (m + 1) * sA;
  }

  // Max-fill: pack segment t into its staging buffer on the host: the head
  // of the partial row segment t-1 returned (waited for here), then A's
  // new entries.  The buffer's previous copy (segment t-2) must be done.
  auto pack_segment = [&](int64_t t) -> aires_status {
    const aires_tile& T = p->tiles[(size_t)t];
    const int b = (int)(t % 2);
    if (t >= 2) HIP_TRY(hipEventSynchronize(ev_in[(size_t)t - 2]));
    int64_t c = 0;
    if (t >= 1) {
      const aires_tile& Tp = p->tiles[(size_t)t - 1];
      c = Tp.sent_nnz1 - Tp.nnz1;  // == T.nnz0 .. Tp.sent_nnz1
      if (c > 0) {
        HIP_TRY(hipEventSynchronize(ev_carry[(size_t)t - 1]));
        p->stats.host_syncs++;
      }
    }
    const auto t0 = std::chrono::steady_clock::now();
    const int64_t q = T.sent_nnz1 - T.nnz0;
    if (c > 0) {
      std::memcpy(stage_col[b], carry_col, sizeof(int32_t) * (size_t)c);
      std::memcpy(stage_val[b], carry_val, sizeof(float) * (size_t)c);
    }
    parallel_ranges(q - c, [&](int64_t lo, int64_t hi, int) {
      std::memcpy(stage_col[b] + c + lo, A.col_idx + T.nnz0 + c + lo, sizeof(int32_t) * (size_t)(hi - lo));
      std::memcpy(stage_val[b] + c + lo, A.vals + T.nnz0 + c + lo, sizeof(float) * (size_t)(hi - lo));
    });
    const double ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    p->stats.merge_ms += ms;
    p->trun[(size_t)t].merge_ms = ms;
    return AIRES_OK;
  };

  // A in a file: read tile t's entries into its staging buffer (the
  // buffer's previous copy, tile t-2's, must be done)
  auto read_tile = [&](int64_t t) -> aires_status {
    const aires_tile& T = p->tiles[(size_t)t];
    const int b = (int)(t % 2);
    if (t >= 2) HIP_TRY(hipEventSynchronize(ev_in[(size_t)t - 2]));
    const auto t0 = std::chrono::steady_clock::now();
    const int64_t q = T.nnz1 - T.nnz0;
    ST_TRY(file_read(*file, file->col_off + 4 * T.nnz0, 4 * q, reinterpret_cast<char*>(stage_col[b]), &shift_col[b]));
    p->stats.storage_bytes += 4 * q;
    if (!sym_norm) {
      ST_TRY(file_read(*file, file->val_off + 4 * T.nnz0, 4 * q, reinterpret_cast<char*>(stage_val[b]),
                       &shift_val[b]));
      p->stats.storage_bytes += 4 * q;
    }
    const double ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    p->stats.storage_ms += ms;
    p->trun[(size_t)t].storage_ms = ms;
    return AIRES_OK;
  };

  auto issue_h2d = [&](int64_t t) -> aires_status {
    const aires_tile& T = p->tiles[(size_t)t];
    Slot& S = slot[t % 2];
    if (maxfill) ST_TRY(pack_segment(t));
    if (file) ST_TRY(read_tile(t));
    if (t >= 2) HIP_TRY(hipStreamWaitEvent(sh, ev_done[(size_t)t - 2], 0));
    th.tile = (int)t;
    const int ea = th.record();
    th.at(aires_plan::T_H2D0, ea);
    const int64_t k = T.r1 - T.r0, q = T.sent_nnz1 - T.nnz0;
    const int32_t* src_col = maxfill ? stage_col[t % 2] : A.col_idx + T.nnz0;
    const float* src_val = maxfill ? stage_val[t % 2] : A.vals + T.nnz0;
    if (file) {
      src_col = reinterpret_cast<const int32_t*>(reinterpret_cast<const char*>(stage_col[t % 2]) + shift_col[t % 2]);
      src_val = reinterpret_cast<const float*>(reinterpret_cast<const char*>(stage_val[t % 2]) + shift_val[t % 2]);
    }
    if (!sym_norm)
      HIP_TRY(hipMemcpyAsync(S.arp, static_cast<const char*>(A.row_ptr) + T.r0 * sA, (size_t)(k + 1) * sA,
                             hipMemcpyHostToDevice, sh));
    if (q > 0) {
      HIP_TRY(hipMemcpyAsync(S.acol, src_col, (size_t)q * 4, hipMemcpyHostToDevice, sh));
      if (!sym_norm) HIP_TRY(hipMemcpyAsync(S.aval, src_val, (size_t)q * 4, hipMemcpyHostToDevice, sh));
    }
    HIP_TRY(hipEventRecord(ev_in[(size_t)t], sh));
    const int eb = th.record();
    th.mark(PH_H2D, 0, ea, eb);
    th.at(aires_plan::T_H2D1, eb);
    const int64_t bytes = sym_norm ? 4 * q : (k + 1) * sA + 8 * q;
    p->stats.h2d_bytes += bytes;
    p->trun[(size_t)t].h2d_bytes = bytes;
    if (maxfill && T.sent_nnz1 > T.nnz1) {
      // the partial last row goes back to host memory (it is sent again,
      // packed in front of the next segment)
      const int64_t c = T.sent_nnz1 - T.nnz1, off = T.nnz1 - T.nnz0;
      const int ec = th.record();
      HIP_TRY(hipMemcpyAsync(carry_col, S.acol + off, (size_t)c * 4, hipMemcpyDeviceToHost, sh));
      HIP_TRY(hipMemcpyAsync(carry_val, S.aval + off, (size_t)c * 4, hipMemcpyDeviceToHost, sh));
      HIP_TRY(hipEventRecord(ev_carry[(size_t)t], sh));
      th.mark(PH_D2H, 0, ec, th.record());
      p->stats.d2h_bytes += 8 * c;
      p->stats.resent_bytes += 8 * c;
      p->trun[(size_t)t].d2h_bytes += 8 * c;
      p->trun[(size_t)t].resent_bytes = 8 * c;
    }
    th.tile = -1;
    return AIRES_OK;
  };

  if (nt > 0) ST_TRY(issue_h2d(0));
  if (nt > 1) ST_TRY(issue_h2d(1));
  if (p->wide && nt > 0) {
    HIP_TRY(hipStreamWaitEvent(sc, ev_in[0], 0));  // B is resident once tile 0 arrived
    HIP_TRY(kern::build_window_index(brp, B.rp_type == AIRES_IDX_I64, bcol, bval, K, p->G, p->nG, bidx,
                                     index_bmax(p, bidx), sc));
  }
  int64_t base = 0;
  for (int64_t t = 0; t < nt; ++t) {
    const aires_tile& T = p->tiles[(size_t)t];
    Slot& S = slot[t % 2];
    const int64_t k = T.r1 - T.r0;
    HIP_TRY(hipStreamWaitEvent(sc, ev_in[(size_t)t], 0));
    if (t >= 2 && c_on_host) HIP_TRY(hipStreamWaitEvent(sc, ev_cfree[t % 2], 0));
    const void* tile_rp = S.arp;
    if (sym_norm) {
      tile_rp = static_cast<const char*>(d_arp_all) + T.r0 * sA;
      HIP_TRY(kern::sym_norm_values(d_arp_all, A.rp_type == AIRES_IDX_I64, T.r0, k, T.nnz0, S.acol, S.aval,
                                    T.nnz1 - T.nnz0, sc));
    }
    kern::Operands op = tile_operands(p, tile_rp, T.nnz0, S.acol, S.aval, brp, bcol, bval, bidx);
    // running base of C.row_ptr for this tile: crp[0] = total so far
    HIP_TRY(hipMemcpyAsync(S.crp, running, sizeof(int64_t), hipMemcpyDeviceToDevice, sc));
    tm.tile = (int)t;
    ST_TRY(tile_symbolic(p, op, k, S.w, S.crp, prod + t, sc, tm));
    HIP_TRY(hipMemcpyAsync(running, S.crp + k, sizeof(int64_t), hipMemcpyDeviceToDevice, sc));
    HIP_TRY(hipMemcpyAsync(cnt_host + 3 * t, S.crp + k, sizeof(int64_t), hipMemcpyDeviceToHost, sc));
    if (p->wide)
      HIP_TRY(hipMemcpyAsync(cnt_host + 3 * t + 1, S.w.icount + k, sizeof(int64_t), hipMemcpyDeviceToHost, sc));
    HIP_TRY(hipMemcpyAsync(cnt_host + 3 * t + 2, prod + t, sizeof(int64_t), hipMemcpyDeviceToHost, sc));
    HIP_TRY(hipEventRecord(ev_cnt[(size_t)t], sc));
    HIP_TRY(hipEventSynchronize(ev_cnt[(size_t)t]));
    p->stats.host_syncs++;
    const int64_t end = cnt_host[3 * t];
    const int64_t nnz_t = end - base;
    p->trun[(size_t)t].nnz_c = nnz_t;
    p->trun[(size_t)t].products = cnt_host[3 * t + 2];
    if (end > cap) {
      // The C bound was an estimate (Eq. 5 mode) and C's arrays are full:
      // move the entries so far into larger ones (by half again at least).
      const int64_t ncap = std::max<int64_t>(end, cap + cap / 2);
      if (c_on_host) {
        HIP_TRY(hipStreamSynchronize(sd));  // earlier tiles' copies into C have landed
        int32_t* nc = nullptr;
        float* nv = nullptr;
        HIP_TRY(hipHostMalloc((void**)&nc, sizeof(int32_t) * (size_t)ncap, hipHostMallocDefault));
        hb.v.push_back(nc);
        HIP_TRY(hipHostMalloc((void**)&nv, sizeof(float) * (size_t)ncap, hipHostMallocDefault));
        hb.v.push_back(nv);
        std::memcpy(nc, C_col, sizeof(int32_t) * (size_t)base);
        std::memcpy(nv, C_val, sizeof(float) * (size_t)base);
        for (void* old : {(void*)C_col, (void*)C_val}) {
          hb.v.erase(std::remove(hb.v.begin(), hb.v.end(), old), hb.v.end());
          (void)hipHostFree(old);
        }
        C_col = nc;
        C_val = nv;
      } else {
        int32_t* nc = nullptr;
        float* nv = nullptr;
        ST_TRY(ws.get_n(ncap, &nc));
        ST_TRY(ws.get_n(ncap, &nv));
        if (base > 0) {  // after the earlier tiles' numeric kernels on sc
          HIP_TRY(hipMemcpyAsync(nc, C_col, sizeof(int32_t) * (size_t)base, hipMemcpyDeviceToDevice, sc));
          HIP_TRY(hipMemcpyAsync(nv, C_val, sizeof(float) * (size_t)base, hipMemcpyDeviceToDevice, sc));
        }
        ws.give_back(C_col);
        ws.give_back(C_val);
        C_col = nc;
        C_val = nv;
      }
      cap = ncap;
    }
    if (c_on_host && nnz_t > S.ccap) {
      // the bound was an estimate (Eq. 5 mode): grow this slot, within the budget
      HIP_TRY(hipStreamWaitEvent(sc, ev_cfree[t % 2], 0));
      ws.give_back(S.ccol);
      ws.give_back(S.cval);
      S.ccol = nullptr;
      S.cval = nullptr;
      ST_TRY(ws.get_n(nnz_t, &S.ccol));
      ST_TRY(ws.get_n(nnz_t, &S.cval));
      S.ccap = nnz_t;
    }
    if (p->wide) {
      S.w.nitems = cnt_host[3 * t + 1];
      if (S.w.nitems > S.icap) {
        if (S.w.items) ws.give_back(S.w.items);
        S.w.items = nullptr;
        // grow geometrically while the budget allows, else to the exact need
        const int64_t want = std::max<int64_t>(S.w.nitems, 2 * S.icap);
        const int64_t grow = ws.fits((int64_t)sizeof(kern::WinItem) * want) ? want : S.w.nitems;
        ST_TRY(ws.get_n(grow, &S.w.items));
        S.icap = grow;
      }
    }
    if (c_on_host) {
      ST_TRY(tile_numeric(p, op, k, S.w, S.crp, S.ccol, S.cval, base, sc, tm));
    } else {
      ST_TRY(tile_numeric(p, op, k, S.w, S.crp, C_col, C_val, 0, sc, tm));
    }
    tm.tile = -1;
    HIP_TRY(hipEventRecord(ev_done[(size_t)t], sc));
    // Phase III for this tile
    if (c_on_host) {
      HIP_TRY(hipStreamWaitEvent(sd, ev_done[(size_t)t], 0));
      td.tile = (int)t;
      const int ea = td.record();
      td.at(aires_plan::T_D2H0, ea);
      HIP_TRY(hipMemcpyAsync(C_rp + T.r0 + 1, S.crp + 1, sizeof(int64_t) * (size_t)k, hipMemcpyDeviceToHost, sd));
      if (nnz_t > 0) {
        HIP_TRY(hipMemcpyAsync(C_col + base, S.ccol, sizeof(int32_t) * (size_t)nnz_t, hipMemcpyDeviceToHost, sd));
        HIP_TRY(hipMemcpyAsync(C_val + base, S.cval, sizeof(float) * (size_t)nnz_t, hipMemcpyDeviceToHost, sd));
      }
      HIP_TRY(hipEventRecord(ev_cfree[t % 2], sd));
      const int eb = td.record();
      td.mark(PH_D2H, 0, ea, eb);
      td.at(aires_plan::T_D2H1, eb);
      td.tile = -1;
      p->stats.d2h_bytes += 8 * k + 8 * nnz_t;
      p->trun[(size_t)t].d2h_bytes += 8 * k + 8 * nnz_t;
    } else {
      HIP_TRY(hipMemcpyAsync(C_rp + T.r0 + 1, S.crp + 1, sizeof(int64_t) * (size_t)k, hipMemcpyDeviceToDevice, sc));
    }
    base = end;
    if (t + 2 < nt) ST_TRY(issue_h2d(t + 2));
  }
  // the pipeline ends with the last copy: join the copy streams into sc
  hipEvent_t ev_end[2];
  ST_TRY(mkev(&ev_end[0]));
  ST_TRY(mkev(&ev_end[1]));
  HIP_TRY(hipEventRecord(ev_end[0], sh));
  HIP_TRY(hipEventRecord(ev_end[1], sd));
  HIP_TRY(hipStreamWaitEvent(sc, ev_end[0], 0));
  HIP_TRY(hipStreamWaitEvent(sc, ev_end[1], 0));
  {
    const int e_end = tm.record();
    tm.mark(PH_PIPELINE, 0, e_pipe0, e_end);
    tm.mark(PH_TOTAL, 0, e_total0, e_end);
  }
  HIP_TRY(hipStreamSynchronize(sd));
  HIP_TRY(hipStreamSynchronize(sh));
  for (int64_t t = 0; t < nt; ++t) p->stats.products += p->trun[(size_t)t].products;
  p->stats.nnz_c = base;
  if (c_on_host) C_rp[0] = 0;
  else HIP_TRY(hipMemsetAsync(C_rp, 0, sizeof(int64_t), sc));

  auto* own = new OutOwner{p->alloc, sc, c_on_host};
  if (c_on_host) {
    hb.v.erase(std::remove(hb.v.begin(), hb.v.end(), (void*)C_rp), hb.v.end());
    hb.v.erase(std::remove(hb.v.begin(), hb.v.end(), (void*)C_col), hb.v.end());
    hb.v.erase(std::remove(hb.v.begin(), hb.v.end(), (void*)C_val), hb.v.end());
  } else {
    ws.detach(C_rp);
    ws.detach(C_col);
    ws.detach(C_val);
  }
  C->nrows = m;
  C->ncols = N;
  C->nnz = base;
  C->row_ptr = C_rp;
  C->col_idx = C_col;
  C->vals = C_val;
  C->mem = c_on_host ? AIRES_MEM_HOST_PINNED : AIRES_MEM_DEVICE;
  C->_owner = own;
  HIP_TRY(hipStreamSynchronize(sc));
  return AIRES_OK;
}

}  // namespace

extern "C" {

aires_status aires_spgemm(aires_plan* plan, void* stream, aires_csr_out* C) {
  ST_TRY(begin_call(plan, C));
  if (plan->A.mem != AIRES_MEM_DEVICE) {
    hipStream_t sh = nullptr, sd = nullptr;
    HIP_TRY(hipStreamCreateWithFlags(&sh, hipStreamNonBlocking));
    if (hipStreamCreateWithFlags(&sd, hipStreamNonBlocking) != hipSuccess) {
      (void)hipStreamDestroy(sh);
      return fail(AIRES_E_HIP, "hipStreamCreate failed");
    }
    plan->busy = 1;
    aires_status st = stream_impl(plan, sh, (hipStream_t)stream, sd, C);
    plan->busy = 0;
    (void)hipStreamSynchronize(sh);
    (void)hipStreamSynchronize(sd);
    (void)hipStreamDestroy(sh);
    (void)hipStreamDestroy(sd);
    return st;
  }
  if (plan->B.mem != AIRES_MEM_DEVICE)
    return fail(AIRES_E_UNSUPPORTED, "device-resident A needs device-resident B");
  plan->busy = 1;
  aires_status st = spgemm_device(plan, (hipStream_t)stream, C);
  plan->busy = 0;
  return st;
}

aires_status aires_spgemm_noalloc(aires_plan* plan, void* stream, int64_t* c_row_ptr, int32_t* c_col_idx,
                                  float* c_vals, int64_t c_capacity, int64_t* nnz_out) {
  if (nnz_out) *nnz_out = -1;
  if (!plan || !c_row_ptr) return fail(AIRES_E_INVALID_ARG, "NULL plan or C.row_ptr");
  if (c_capacity < 0) return fail(AIRES_E_INVALID_ARG, "negative C capacity");
  if (c_capacity > 0 && (!c_col_idx || !c_vals)) return fail(AIRES_E_INVALID_ARG, "NULL C arrays");
  if (plan->A.mem != AIRES_MEM_DEVICE || plan->B.mem != AIRES_MEM_DEVICE)
    return fail(AIRES_E_UNSUPPORTED, "the allocation-free call needs A and B on the device");
  if (plan->busy) return fail(AIRES_E_STATE, "plan is in use");
  void* base = nullptr;
  HIP_TRY(aires::scratch_address(&base));
  std::memset(&plan->stats, 0, sizeof plan->stats);
  plan->stats.ntiles = (int64_t)plan->tiles.size();
  plan->trun.assign(plan->tiles.size(), aires_plan::TileRun{0, 0, 0, 0, 0, 0.0, 0.0});
  reset_timing(plan);
  std::array<int, aires_plan::T_NEV> none;
  none.fill(-1);
  plan->tev.assign(plan->tiles.size(), none);
  plan->ev_base = -1;
  // no timing events: the call creates no runtime objects either
  const int32_t timing = plan->opts.timing;
  plan->opts.timing = 0;
  plan->busy = 1;
  DevPool ws(base, kScratchBytes, (hipStream_t)stream);
  CallerC cc{c_row_ptr, c_col_idx, c_vals, c_capacity, nnz_out};
  aires_status st = spgemm_device_in(plan, (hipStream_t)stream, ws, nullptr, &cc);
  plan->busy = 0;
  plan->opts.timing = timing;
  return st;
}

aires_status aires_stream_tiles(aires_plan* plan, void* h2d, void* compute, void* d2h, aires_csr_out* C) {
  ST_TRY(begin_call(plan, C));
  plan->busy = 1;
  aires_status st = stream_impl(plan, (hipStream_t)h2d, (hipStream_t)compute, (hipStream_t)d2h, C);
  plan->busy = 0;
  return st;
}

aires_status aires_spmm(const aires_csr* A, const float* W, int64_t ldw, int64_t F, float* Y, int64_t ldy,
                        aires_act act, aires_spmm_algo algo, void* stream) {
  ST_TRY(check_csr_desc(A, "A"));
  if (A->mem != AIRES_MEM_DEVICE) return fail(AIRES_E_UNSUPPORTED, "aires_spmm needs A on the device");
  if (F < 0 || F >= (int64_t(1) << 31)) return fail(AIRES_E_UNSUPPORTED, "F = %lld out of range", (long long)F);
  if (act != AIRES_ACT_NONE && act != AIRES_ACT_RELU) return fail(AIRES_E_INVALID_ARG, "act %d invalid", (int)act);
  if (algo != AIRES_SPMM_AUTO && algo != AIRES_SPMM_ROWS && algo != AIRES_SPMM_DENSE_TILES)
    return fail(AIRES_E_INVALID_ARG, "algo %d invalid", (int)algo);
  if (algo == AIRES_SPMM_DENSE_TILES && !kern::spmm_dense_fits(A->ncols, ldw) && A->nrows > 0 && F > 0)
    return fail(AIRES_E_UNSUPPORTED, "dense tiles need K <= 2^20 and ldw < 2^23 (K = %lld, ldw = %lld)",
                (long long)A->ncols, (long long)ldw);
  if (A->nrows == 0 || F == 0) return AIRES_OK;
  if (ldw < F || ldy < F) return fail(AIRES_E_INVALID_ARG, "ldw %lld / ldy %lld below F %lld", (long long)ldw,
                                      (long long)ldy, (long long)F);
  if (!Y || !A->row_ptr || (A->nnz > 0 && (!W || !A->col_idx || !A->vals)))
    return fail(AIRES_E_INVALID_ARG, "NULL array");
  // dense tiles do m*K*F multiply-adds against nnz*F gathered rows: worth it
  // from about one entry in eight (measured on 512-column aggregates)
  bool dense = algo == AIRES_SPMM_DENSE_TILES;
  if (algo == AIRES_SPMM_AUTO)
    dense = kern::spmm_dense_fits(A->ncols, ldw) && (double)A->nnz * 8.0 >= (double)A->nrows * (double)A->ncols;
  if (dense && !W && A->ncols > 0) return fail(AIRES_E_INVALID_ARG, "NULL W (dense tiles read W)");
  HIP_TRY(kern::spmm(A->row_ptr, A->rp_type == AIRES_IDX_I64, A->col_idx, A->vals, A->nrows, A->ncols, W, ldw, F,
                     Y, ldy, act == AIRES_ACT_RELU, dense, (hipStream_t)stream));
  return AIRES_OK;
}

aires_status aires_plan_stats(const aires_plan* plan, aires_stats* stats) {
  if (!plan || !stats) return fail(AIRES_E_INVALID_ARG, "NULL argument");
  *stats = plan->stats;
  if (!plan->ev.empty()) {
    HIP_TRY(hipEventSynchronize(plan->ev.back()));
    for (const auto& mk : plan->marks) {
      float ms = 0.f;
      HIP_TRY(hipEventElapsedTime(&ms, plan->ev[(size_t)mk.a], plan->ev[(size_t)mk.b]));
      switch (mk.kind) {
        case PH_ANALYZE: stats->analyze_ms += ms; break;
        case PH_BIN: stats->bin_ms += ms; break;
        case PH_SYMBOLIC: stats->symbolic_ms += ms; break;
        case PH_SCAN: stats->scan_ms += ms; break;
        case PH_NUMERIC: stats->numeric_ms += ms; break;
        case PH_H2D: stats->h2d_ms += ms; break;
        case PH_D2H: stats->d2h_ms += ms; break;
        case PH_TOTAL: stats->total_ms += ms; break;
        case PH_PIPELINE: stats->pipeline_ms += ms; break;
        default:
          if (mk.kind >= 0 && mk.kind < AIRES_NUM_KINDS) stats->kind_ms[mk.phase][mk.kind] += ms;
          break;
      }
    }
  }
  return AIRES_OK;
}

aires_status aires_plan_tile_stats(const aires_plan* plan, int64_t t, aires_tile_stats* ts) {
  if (!plan || !ts) return fail(AIRES_E_INVALID_ARG, "NULL argument");
  if (t < 0 || t >= (int64_t)plan->tiles.size()) return fail(AIRES_E_INVALID_ARG, "tile %lld out of range", (long long)t);
  std::memset(ts, 0, sizeof *ts);
  ts->h2d_begin_ms = ts->h2d_end_ms = ts->compute_begin_ms = ts->compute_end_ms = ts->d2h_begin_ms =
      ts->d2h_end_ms = -1.0;
  const aires_tile& T = plan->tiles[(size_t)t];
  ts->r0 = T.r0;
  ts->r1 = T.r1;
  if ((size_t)t < plan->trun.size()) {
    const auto& r = plan->trun[(size_t)t];
    ts->products = r.products;
    ts->nnz_c = r.nnz_c;
    ts->h2d_bytes = r.h2d_bytes;
    ts->d2h_bytes = r.d2h_bytes;
    ts->resent_bytes = r.resent_bytes;
    ts->merge_ms = r.merge_ms;
    ts->storage_ms = r.storage_ms;
  }
  if (!plan->ev.empty()) {
    HIP_TRY(hipEventSynchronize(plan->ev.back()));
    for (const auto& mk : plan->marks) {
      if (mk.tile != (int)t) continue;
      float ms = 0.f;
      HIP_TRY(hipEventElapsedTime(&ms, plan->ev[(size_t)mk.a], plan->ev[(size_t)mk.b]));
      switch (mk.kind) {
        case PH_ANALYZE: ts->analyze_ms += ms; break;
        case PH_BIN: ts->bin_ms += ms; break;
        case PH_SYMBOLIC: ts->symbolic_ms += ms; break;
        case PH_SCAN: ts->scan_ms += ms; break;
        case PH_NUMERIC: ts->numeric_ms += ms; break;
        case PH_H2D: ts->h2d_ms += ms; break;
        case PH_D2H: ts->d2h_ms += ms; break;
        default: break;
      }
    }
    if (plan->ev_base >= 0 && (size_t)t < plan->tev.size()) {
      double* at[aires_plan::T_NEV] = {&ts->h2d_begin_ms, &ts->h2d_end_ms, &ts->compute_begin_ms,
                                       &ts->compute_end_ms, &ts->d2h_begin_ms, &ts->d2h_end_ms};
      for (int i = 0; i < aires_plan::T_NEV; ++i) {
        const int e = plan->tev[(size_t)t][(size_t)i];
        *at[i] = -1.0;
        if (e < 0) continue;
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, plan->ev[(size_t)plan->ev_base], plan->ev[(size_t)e]));
        *at[i] = ms;
      }
    }
  }
  return AIRES_OK;
}

void aires_csr_out_free(aires_csr_out* C) {
  if (!C) return;
  auto* own = static_cast<OutOwner*>(C->_owner);
  if (own) {
    if (own->host) {
      if (C->row_ptr) (void)hipHostFree(C->row_ptr);
      if (C->col_idx) (void)hipHostFree(C->col_idx);
      if (C->vals) (void)hipHostFree(C->vals);
    } else {
      if (C->row_ptr) own->a.free(own->a.ctx, C->row_ptr, (void*)own->s);
      if (C->col_idx) own->a.free(own->a.ctx, C->col_idx, (void*)own->s);
      if (C->vals) own->a.free(own->a.ctx, C->vals, (void*)own->s);
    }
    delete own;
  }
  std::memset(C, 0, sizeof *C);
}

}  // extern "C"
