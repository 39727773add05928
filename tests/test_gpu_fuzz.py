"""GPU parity over seeded random cases: random shapes with heavy-tailed row
lengths (hub rows in A, long rows in B), random row-pointer widths, and a
random valid combination of the plan options that pick the kernel paths
(dense rows, split rows, the four hash tiers, column windows with their
grain, pool, entry and item sizes, kept symbolic bitmaps and a too-small
bitmap cache, column slabs, tiling).  Each case is compared with the oracle:
structure bit-exact, values bit-exact for integer inputs (every product and
partial sum is exact in fp32) and within 1e-5 * (1 + |ref|) otherwise."""
import sys

import numpy as np
import pytest

import oracle
import workloads
from workloads import CSR

pytestmark = pytest.mark.gpu

TOL = 1e-5
CASES = 160


@pytest.fixture(scope="module")
def torch_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    return torch


def heavy_tailed_csr(rng, m, n, mean_len, ints, rp64):
    """Rows of Pareto-distributed lengths (capped at n) with distinct random
    columns; a few rows are hubs."""
    lens = np.minimum(n, (rng.pareto(1.3, size=m) * mean_len).astype(np.int64))
    hubs = rng.random(m) < 0.01
    lens[hubs] = np.minimum(n, rng.integers(n // 4 + 1, n + 1, size=int(hubs.sum())))
    cols = [np.sort(rng.choice(n, size=int(k), replace=False)) if k else np.zeros(0, np.int64) for k in lens]
    col = np.concatenate(cols).astype(np.int32) if m else np.zeros(0, np.int32)
    rp = np.zeros(m + 1, np.int64)
    rp[1:] = np.cumsum(lens)
    nnz = int(rp[-1])
    val = (rng.integers(-4, 5, size=nnz) if ints else rng.uniform(-1, 1, size=nnz)).astype(np.float32)
    return CSR(m, n, rp if rp64 else rp.astype(np.int32), col, val)


def draw_options(rng, N):
    o = {}
    if rng.random() < 0.3:
        o["dense_max_cols"] = int(rng.choice([32, 96, 512, 2048]))
    if rng.random() < 0.5:
        o["hash_max_products"] = int(rng.choice([-1, 64, 512, 2048, 4096]))
    if rng.random() < 0.4:
        o["wave_max_products"] = int(rng.choice([1, 16, 256]))
    if rng.random() < 0.3:
        o["split_min_products"] = int(rng.choice([-1, 1, 500]))
        if rng.random() < 0.5:
            o["split_max_rows"] = int(rng.integers(1, 8))
    # column windows: a grain of 32..2048 columns, windows of 1..6 grains and
    # G..4G entries, symbolic items of 1..8 grains, sometimes a small pool
    G = int(rng.choice([32, 64, 96, 256, 1024, 2048]))
    o["window_grain_cols"] = G
    o["window_max_grains"] = int(rng.integers(1, 7))
    o["window_max_entries"] = int(min(65535, G * rng.integers(1, 5)))
    o["count_grains"] = int(rng.integers(1, 9))
    if rng.random() < 0.3:
        words = 2 * ((G + 47) // 48) + G  # one full grain
        o["window_pool_bytes"] = int(4 * (words + rng.integers(0, 2 * words)))
    o["keep_bitmap_products"] = int(rng.choice([0, 1, -1, 100]))
    if o["keep_bitmap_products"] != -1 and rng.random() < 0.3:
        o["bitmap_cache_bytes"] = int(rng.choice([4096, 65536]))
    o["slab_min_products"] = int(rng.choice([0, 1, -1, 50, 2000]))
    return o


def case(seed):
    rng = np.random.default_rng(1_000_003 * seed + 17)
    m = int(rng.integers(1, 2500))
    K = int(rng.integers(1, 1500))
    N = int(rng.choice([1, 17, 100, 333, 700, 2049, 5000, 40000]))
    ints = bool(rng.random() < 0.5)
    A = heavy_tailed_csr(rng, m, K, float(rng.uniform(0.5, 12)), ints, bool(rng.random() < 0.3))
    B = heavy_tailed_csr(rng, K, N, float(rng.uniform(0.5, 20)), ints, bool(rng.random() < 0.3))
    opts = draw_options(rng, N)
    tiles = int(rng.choice([0, 0, max(1, m // 3)]))
    return A, B, ints, opts, tiles


@pytest.mark.parametrize("seed", range(CASES))
def test_random_case(torch_gpu, seed):
    import paper_2507_02006_amd as aires
    A, B, ints, opts, tiles = case(seed)
    print("[gpu-case] fuzz seed=%d m=%d K=%d N=%d nnzA=%d nnzB=%d ints=%s tiles=%d opts=%s" %
          (seed, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, ints, tiles, opts), flush=True)
    sys.stdout.flush()
    ref = oracle.spgemm(A, B)
    dA, dB = aires.to_device(A), aires.to_device(B)
    with aires.tile_plan(dA, dB, 0, max_tile_rows=tiles, **opts) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        st = aires.plan_stats(plan)
    rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(rp - rp[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    assert st["products"] == ref.products and st["nnz_c"] == ref.nnz
    if ints:
        assert np.array_equal(val, ref.val), "integer values differ"
    else:
        err = np.abs(val.astype(np.float64) - ref.val.astype(np.float64))
        bad = err > TOL * (1 + np.abs(ref.val.astype(np.float64)))
        assert not bad.any(), "values differ at %d entries, max err %g" % (bad.sum(), err.max())


STREAMED = 64
NOALLOC = 32


def check_values(val, ref, ints):
    if ints:
        assert np.array_equal(val, ref.val), "integer values differ"
    else:
        err = np.abs(val.astype(np.float64) - ref.val.astype(np.float64))
        bad = err > TOL * (1 + np.abs(ref.val.astype(np.float64)))
        assert not bad.any(), "values differ at %d entries, max err %g" % (bad.sum(), err.max())


@pytest.mark.parametrize("seed", range(STREAMED))
def test_random_streamed_case(torch_gpu, seed):
    """A in pinned host memory, streamed in 2..5 row blocks with double-
    buffered copies; B on the device or in pinned memory; C returned in
    pinned host or device memory; C bound from the products or from the row
    pointers; random path options as above."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B, ints, opts, _ = case(1000 + seed)
    rng = np.random.default_rng(7_000 + seed)
    c_on_host = bool(rng.random() < 0.5)
    c_bound = B_.CBOUND_ROWS if rng.random() < 0.5 else B_.CBOUND_PRODUCTS
    b_pinned = bool(rng.random() < 0.5)
    tiles = max(1, A.nrows // int(rng.integers(2, 6)))
    print("[gpu-case] fuzz streamed seed=%d m=%d K=%d N=%d nnzA=%d nnzB=%d ints=%s tiles=%d c_on_host=%s "
          "c_bound=%d b_pinned=%s opts=%s" % (seed, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, ints, tiles, c_on_host,
                                              c_bound, b_pinned, opts), flush=True)
    ref = oracle.spgemm(A, B)
    dB = aires.to_pinned(B) if b_pinned else aires.to_device(B)
    with aires.tile_plan(aires.to_pinned(A), dB, 1 << 34, c_on_host=c_on_host, c_bound=c_bound,
                         max_tile_rows=tiles, **opts) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        if c_on_host:
            rp, col, val = C.rp.copy(), C.col.copy(), C.val.copy()
            C.free()
        else:
            rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(rp - rp[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    check_values(val, ref, ints)


@pytest.mark.parametrize("seed", range(NOALLOC))
def test_random_noalloc_case(torch_gpu, seed):
    """The allocation-free entry point on random cases (C arrays with room
    to spare; nothing is written past nnz(C))."""
    import paper_2507_02006_amd as aires
    A, B, ints, opts, tiles = case(2000 + seed)
    print("[gpu-case] fuzz noalloc seed=%d m=%d K=%d N=%d nnzA=%d nnzB=%d ints=%s tiles=%d opts=%s" %
          (seed, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, ints, tiles, opts), flush=True)
    ref = oracle.spgemm(A, B)
    dA, dB = aires.to_device(A), aires.to_device(B)
    with aires.tile_plan(dA, dB, 0, max_tile_rows=tiles, **opts) as plan:
        rp = torch_gpu.full((A.nrows + 1,), -1, dtype=torch_gpu.int64, device="cuda")
        cap = ref.nnz + 17
        col = torch_gpu.full((cap,), -1, dtype=torch_gpu.int32, device="cuda")
        val = torch_gpu.zeros((cap,), dtype=torch_gpu.float32, device="cuda")
        try:
            nnz = aires.spgemm_noalloc(plan, rp, col, val)
        except aires.AiresError as e:
            from paper_2507_02006_amd import _binding as B_
            if e.status == B_.E_CAPACITY and "workspace" in str(e):
                pytest.skip("workspace beyond the fixed array: %s" % e)
            raise
        torch_gpu.cuda.synchronize()
    assert nnz == ref.nnz
    assert np.all(col[nnz:].cpu().numpy() == -1)
    rpn = rp.cpu().numpy()
    assert np.array_equal(rpn - rpn[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col[:nnz].cpu().numpy(), ref.col), "col_idx differs"
    check_values(val[:nnz].cpu().numpy(), ref, ints)


MAXFILL = 32
FILES = 16


@pytest.mark.parametrize("seed", range(MAXFILL))
def test_random_maxfill_case(torch_gpu, seed):
    """Max-fill segments (ending inside rows; the partial row is copied back
    and sent again with the next segment) of a pinned A, in slots of a
    random size, C on the host or the device."""
    import paper_2507_02006_amd as aires
    A, B, ints, opts, _ = case(3000 + seed)
    rng = np.random.default_rng(9_000 + seed)
    c_on_host = bool(rng.random() < 0.5)
    slot = max(4096, int(A.nbytes() // int(rng.integers(2, 9))))
    print("[gpu-case] fuzz maxfill seed=%d m=%d K=%d N=%d nnzA=%d nnzB=%d ints=%s slot=%d c_on_host=%s opts=%s" %
          (seed, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, ints, slot, c_on_host, opts), flush=True)
    ref = oracle.spgemm(A, B)
    with aires.tile_plan(aires.to_pinned(A), aires.to_device(B), 1 << 34, c_on_host=c_on_host, max_tile_bytes=slot,
                         segmentation="maxfill", **opts) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        if c_on_host:
            rp, col, val = C.rp.copy(), C.col.copy(), C.val.copy()
            C.free()
        else:
            rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(rp - rp[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    check_values(val, ref, ints)


@pytest.mark.parametrize("seed", range(FILES))
def test_random_file_case(torch_gpu, tmp_path, seed):
    """A (and, for half the cases, B) in files: A's tiles read per tile with
    direct or buffered I/O, B read whole into HBM first; row-pointer C bound."""
    import paper_2507_02006_amd as aires
    A, B, ints, opts, _ = case(4000 + seed)
    rng = np.random.default_rng(11_000 + seed)
    c_on_host = bool(rng.random() < 0.5)
    direct = bool(rng.random() < 0.5)
    b_file = bool(rng.random() < 0.5)
    slot = max(4096, int(A.nbytes() // int(rng.integers(2, 6))))
    print("[gpu-case] fuzz file seed=%d m=%d K=%d N=%d nnzA=%d nnzB=%d ints=%s slot=%d c_on_host=%s direct=%s "
          "b_file=%s opts=%s" % (seed, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, ints, slot, c_on_host, direct,
                                 b_file, opts), flush=True)
    ref = oracle.spgemm(A, B)
    ma = workloads.write_csr_file(str(tmp_path / "a.csr"), A)
    if b_file:
        mb = workloads.write_csr_file(str(tmp_path / "b.csr"), B)
        mb["direct_io"] = direct
        Bd, _ = aires.read_csr_file(mb, mem="device", chunk_bytes=int(rng.choice([4096, 1 << 20])))
        dB = (B.nrows, B.ncols, Bd.rp, Bd.col, Bd.val)
    else:
        dB = aires.to_pinned(B)
    with aires.tile_plan_file(ma, dB, 1 << 34, c_on_host=c_on_host, direct_io=direct, max_tile_bytes=slot) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        if c_on_host:
            rp, col, val = C.rp.copy(), C.col.copy(), C.val.copy()
            C.free()
        else:
            rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(rp - rp[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    check_values(val, ref, ints)


SPMM = 48


@pytest.mark.parametrize("seed", range(SPMM))
def test_random_spmm_case(torch_gpu, seed):
    """The combination step Y = act(A * W) (aires_spmm) on random shapes
    with heavy-tailed rows, a random feature width, kernel family, ReLU,
    row strides, offsets and row-pointer width, held to the fp32 summation
    bound (bit-exact for integer inputs) by the spmm tests' own checker."""
    from test_gpu_spmm import check as spmm_check
    rng = np.random.default_rng(13_000 + seed)
    m = int(rng.integers(1, 3000))
    K = int(rng.integers(1, 2000))
    ints = bool(rng.random() < 0.4)
    rp64 = bool(rng.random() < 0.3)
    A = heavy_tailed_csr(rng, m, K, float(rng.uniform(0.5, 30)), ints, False)
    F = int(rng.choice([1, 3, 16, 63, 64, 65, 128, 200, 256, 511, 700]))
    W = (rng.integers(-4, 5, size=(K, F)) if ints else rng.uniform(-1, 1, size=(K, F))).astype(np.float32)
    spmm_check(torch_gpu, A, W, relu=bool(rng.random() < 0.5), rp64=rp64, ldw_pad=int(rng.choice([0, 0, 3, 64])),
               ldy_pad=int(rng.choice([0, 0, 5])), w_offset=int(rng.choice([0, 0, 1, 3])), exact=ints,
               name="fuzz spmm seed=%d" % seed, algo=str(rng.choice(["auto", "rows", "dense_tiles"])),
               a_offset=int(rng.choice([0, 0, 1, 2])))


WIDE = 32


def sparse_wide_csr(rng, m, n, mean_len, ints, rp64):
    """Like heavy_tailed_csr for a very wide n: columns drawn with
    replacement and made distinct (rows a little shorter than drawn)."""
    lens = np.minimum(n, (rng.pareto(1.3, size=m) * mean_len).astype(np.int64))
    hubs = rng.random(m) < 0.01
    lens[hubs] = np.minimum(n, rng.integers(1000, 20000, size=int(hubs.sum())))
    cols = [np.unique(rng.integers(0, n, size=int(k))) for k in lens]
    lens = np.array([len(c) for c in cols], np.int64)
    col = np.concatenate(cols).astype(np.int32) if m else np.zeros(0, np.int32)
    rp = np.zeros(m + 1, np.int64)
    rp[1:] = np.cumsum(lens)
    nnz = int(rp[-1])
    val = (rng.integers(-4, 5, size=nnz) if ints else rng.uniform(-1, 1, size=nnz)).astype(np.float32)
    return CSR(m, n, rp if rp64 else rp.astype(np.int32), col, val)


def case_wide(seed):
    rng = np.random.default_rng(5_000_011 * seed + 3)
    m = int(rng.integers(1, 2000))
    K = int(rng.integers(1, 3000))
    N = int(rng.choice([131072, 1048576]))
    ints = bool(rng.random() < 0.5)
    A = heavy_tailed_csr(rng, m, K, float(rng.uniform(1, 30)), ints, bool(rng.random() < 0.3))
    B = sparse_wide_csr(rng, K, N, float(rng.uniform(5, 200)), ints, bool(rng.random() < 0.3))
    o = {"window_grain_cols": int(rng.choice([4096, 8192])), "count_grains": int(rng.choice([16, 32])),
         "keep_bitmap_products": int(rng.choice([0, 1, -1, 20000])),
         "slab_min_products": int(rng.choice([0, 1, -1, 20000]))}
    if rng.random() < 0.5:
        o["hash_max_products"] = int(rng.choice([-1, 512, 2048, 4096]))
    tiles = int(rng.choice([0, 0, max(1, m // 3)]))
    return A, B, ints, o, tiles


@pytest.mark.parametrize("seed", range(WIDE))
def test_random_wide_case(torch_gpu, seed):
    """Products of 2^17 or 2^20 columns with default-like windows (grains of
    4096 or 8192 columns, items of 16 or 32 grains), kept bitmaps, column
    slabs and tiles drawn at random; hub rows in A and long rows in B."""
    import paper_2507_02006_amd as aires
    A, B, ints, opts, tiles = case_wide(seed)
    print("[gpu-case] fuzz wide seed=%d m=%d K=%d N=%d nnzA=%d nnzB=%d ints=%s tiles=%d opts=%s" %
          (seed, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, ints, tiles, opts), flush=True)
    ref = oracle.spgemm(A, B)
    dA, dB = aires.to_device(A), aires.to_device(B)
    with aires.tile_plan(dA, dB, 0, max_tile_rows=tiles, **opts) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        st = aires.plan_stats(plan)
    rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(rp - rp[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    assert st["products"] == ref.products and st["nnz_c"] == ref.nnz
    check_values(val, ref, ints)


BUDGET = 40


@pytest.mark.parametrize("seed", range(BUDGET))
def test_random_budget_case(torch_gpu, seed):
    """A device budget of the caller's device inputs (which the budget
    covers), the planner's 4 MiB of fixed slack, and 0 to 1.5 times what a
    first call measured at the allocator, in core or with A streamed from
    pinned memory: the call either returns the oracle's C with the
    allocator's peak within the budget, or fails with AIRES_E_BUDGET (at
    planning or after the symbolic phase) leaving nothing allocated."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B, ints, opts, tiles = case(5000 + seed)
    rng = np.random.default_rng(17_000 + seed)
    streamed = bool(rng.random() < 0.5)
    c_on_host = streamed and bool(rng.random() < 0.5)
    f = float(rng.uniform(0.0, 1.5))
    ref = oracle.spgemm(A, B)
    dA = aires.to_pinned(A) if streamed else aires.to_device(A)
    dB = aires.to_device(B)
    inputs = B.nbytes() + (0 if streamed else A.nbytes())
    kw = dict(opts, max_tile_rows=tiles, c_on_host=c_on_host)
    probe = B_.TorchAllocator(0)
    with aires.tile_plan(dA, dB, 1 << 36, allocator=probe, **kw) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        if c_on_host:
            C.free()
        del C
    need = probe.peak
    budget = inputs + (4 << 20) + int(f * need)
    print("[gpu-case] fuzz budget seed=%d m=%d K=%d N=%d streamed=%s c_on_host=%s need=%d budget=%d (%.2f x) opts=%s" %
          (seed, A.nrows, A.ncols, B.ncols, streamed, c_on_host, need, budget, f, kw), flush=True)
    alloc = B_.TorchAllocator(0)
    try:
        with aires.tile_plan(dA, dB, budget, allocator=alloc, **kw) as plan:
            C = aires.spgemm(plan)
            torch_gpu.cuda.synchronize()
            if c_on_host:
                rp, col, val = C.rp.copy(), C.col.copy(), C.val.copy()
                C.free()
            else:
                rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    except aires.AiresError as e:
        torch_gpu.cuda.synchronize()
        assert e.status == B_.E_BUDGET, str(e)
        assert alloc.cur == 0 and not alloc.live, "blocks left after %s" % e
        print("[gpu-case] refused: %s" % e, flush=True)
        return
    print("[gpu-case] ran: allocator peak %d of %d" % (alloc.peak, budget - inputs), flush=True)
    assert alloc.peak <= budget - inputs, "allocator peak %d over the budget's %d" % (alloc.peak, budget - inputs)
    assert np.array_equal(rp - rp[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    check_values(val, ref, ints)


WIDE_STREAMED = 16


@pytest.mark.parametrize("seed", range(WIDE_STREAMED))
def test_random_wide_streamed_case(torch_gpu, seed):
    """The wide cases above with A streamed from pinned host memory in 2..5
    row blocks (windows and column slabs per tile), C on the host or the
    device."""
    import paper_2507_02006_amd as aires
    A, B, ints, opts, _ = case_wide(100 + seed)
    rng = np.random.default_rng(19_000 + seed)
    c_on_host = bool(rng.random() < 0.5)
    tiles = max(1, A.nrows // int(rng.integers(2, 6)))
    print("[gpu-case] fuzz wide streamed seed=%d m=%d K=%d N=%d nnzA=%d nnzB=%d ints=%s tiles=%d c_on_host=%s opts=%s" %
          (seed, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, ints, tiles, c_on_host, opts), flush=True)
    ref = oracle.spgemm(A, B)
    with aires.tile_plan(aires.to_pinned(A), aires.to_device(B), 1 << 36, c_on_host=c_on_host, max_tile_rows=tiles,
                         **opts) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        if c_on_host:
            rp, col, val = C.rp.copy(), C.col.copy(), C.val.copy()
            C.free()
        else:
            rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(rp - rp[0], ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    check_values(val, ref, ints)
