"""GPU parity: the HIP path through the C-ABI against the CPU oracle.

Bar: C.row_ptr and C.col_idx bit-exact; values within
|c - ref| <= 1e-5 * (1 + |ref|) (fp32 accumulation in any order).  Every
kernel path is forced on its own through the plan options, on seeded
inputs shaped like the five aggregation workloads (scaled down so the
oracle finishes in seconds, spanning several tiles/windows and ragged
tails), plus edge cases, and every row of all five workloads at full size
(the oracle over row chunks on the host's threads)."""
import json
import os
import sys
import zlib

import numpy as np
import pytest

import fullcheck
import oracle
import workloads
from workloads import CSR

pytestmark = pytest.mark.gpu

TOL = 1e-5


@pytest.fixture(scope="module")
def torch_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    return torch


def say(msg):
    print("[gpu-case] " + msg, flush=True)
    sys.stdout.flush()


def run(torch, A, B, budget=0, **kw):
    import paper_2507_02006_amd as aires
    dA, dB = aires.to_device(A), aires.to_device(B)
    with aires.tile_plan(dA, dB, budget, timing=True, **kw) as plan:
        C = aires.spgemm(plan)
        torch.cuda.synchronize()
        st = aires.plan_stats(plan)
        ntiles = aires.plan_info(plan).ntiles
    return C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), st, ntiles


def assert_match(rp, col, val, ref, r0=0):
    assert rp.dtype == np.int64
    base = rp[0]
    assert np.array_equal(rp - base, ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    err = np.abs(val.astype(np.float64) - ref.val.astype(np.float64))
    bad = err > TOL * (1 + np.abs(ref.val.astype(np.float64)))
    assert not bad.any(), "values differ at %d entries, max err %g" % (bad.sum(), err.max())


def check(torch, A, B, name, **kw):
    say("%s m=%d K=%d N=%d nnzA=%d nnzB=%d opts=%s" % (name, A.nrows, A.ncols, B.ncols, A.nnz, B.nnz, kw))
    ref = oracle.spgemm(A, B)
    rp, col, val, st, nt = run(torch, A, B, **kw)
    assert_match(rp, col, val, ref)
    assert st["products"] == ref.products
    assert st["nnz_c"] == ref.nnz
    return st, nt, ref


# ------------------------------------------------------------ golden / tiny

def test_hand_4x4(torch_gpu, golden_dir):
    g = json.load(open(os.path.join(golden_dir, "hand_4x4.json")))
    mk = lambda d: CSR(d["nrows"], d["ncols"], np.array(d["rp"], np.int32), np.array(d["col"], np.int32),
                       np.array(d["val"], np.float32))
    A, B = mk(g["A"]), mk(g["B"])
    for kw in ({}, {"wave_max_products": 1}):
        rp, col, val, st, _ = run(torch_gpu, A, B, **kw)
        assert rp.tolist() == g["C"]["rp"] and col.tolist() == g["C"]["col"]
        assert val.tolist() == g["C"]["val"]


PATHS = {
    # narrow N (<= 2048): wavefront rows, workgroup rows
    "dense_wave": dict(),
    "dense_block": dict(wave_max_products=1),
    # wide N forced through tiny column grains: grain counts, windows of whole
    # grains (several grains, ragged last grain), per-lane grain popcounts
    "windows_only": dict(dense_max_cols=64, hash_max_products=-1, window_grain_cols=64,
                         window_max_grains=2, window_max_entries=64, count_grains=3),
    "hash128_then_windows": dict(dense_max_cols=96, hash_max_products=64, window_grain_cols=32,
                                 window_max_grains=3, window_max_entries=40, count_grains=2),
    "hash1024_then_windows": dict(dense_max_cols=128, hash_max_products=512, window_grain_cols=128,
                                  window_max_grains=1, window_max_entries=128, count_grains=1),
    "hash8192_then_windows": dict(dense_max_cols=160, hash_max_products=4096, window_grain_cols=96,
                                  window_max_grains=4, window_max_entries=200, count_grains=5),
    "hash4096_then_windows": dict(dense_max_cols=160, hash_max_products=2048, window_grain_cols=96,
                                  window_max_grains=4, window_max_entries=200, count_grains=5),
    # windows cut by the shared LDS pool (bitmap words + values), not by the
    # grain or entry caps: a wide sparse window or a narrow dense one
    "windows_pool": dict(dense_max_cols=64, hash_max_products=-1, window_grain_cols=64,
                         window_max_grains=16, window_max_entries=1000, count_grains=8,
                         window_pool_bytes=4 * 100),
    # the numeric kernel's column slabs: every window row's windows spread
    # over the slabs (one per XCD; several slabs get none of a row's
    # windows), then only rows above 50 products, the rest from the shared
    # counter, with every window row keeping its symbolic bitmaps
    "windows_slabs": dict(dense_max_cols=64, hash_max_products=-1, window_grain_cols=64,
                          window_max_grains=2, window_max_entries=64, count_grains=3, slab_min_products=1),
    "windows_slabs_kept": dict(dense_max_cols=64, hash_max_products=-1, window_grain_cols=64,
                               window_max_grains=2, window_max_entries=64, count_grains=3,
                               keep_bitmap_products=1, slab_min_products=50),
    # 2048 < N <= 16384 handled as narrow: hash bins then workgroup dense rows
    "narrow_block_hash": dict(dense_max_cols=200, hash_max_products=512),
    # narrow rows split over workgroups (dense slots in global memory); then
    # with too few slots, the rest of the bin one workgroup per row
    "dense_split": dict(wave_max_products=1, split_min_products=1),
    "dense_split_capped": dict(wave_max_products=1, split_min_products=1, split_max_rows=7),
}


@pytest.mark.parametrize("path", list(PATHS))
def test_each_path_integer_values_exact(torch_gpu, path):
    """Integer values: every product and partial sum is exact in fp32, so
    values are bit-exact whatever the summation order."""
    rng = np.random.default_rng(zlib.crc32(path.encode()))
    A = workloads.random_csr(rng, 700, 300, 0.03, values="int")
    B = workloads.random_csr(rng, 300, 333, 0.05, values="int")
    say("int-exact %s" % path)
    ref = oracle.spgemm(A, B)
    rp, col, val, st, _ = run(torch_gpu, A, B, **PATHS[path])
    assert np.array_equal(rp, ref.rp) and np.array_equal(col, ref.col)
    assert np.array_equal(val, ref.val)


# wide products whose rows all go to column windows (plain, cut by the LDS
# pool, and over column slabs with kept bitmaps)
FIXED_PATHS = ["windows_only", "windows_pool", "windows_slabs_kept"]


def ones_and_tiny(rng, m, K, N, a_per_row, a_val, tiny, signed=False):
    """A: m rows of a_per_row distinct columns of K, every value a_val.
    B: K rows of about N/2 random columns of N, each value 1.0 with
    probability 1/4, else `tiny`; every row holds at least one 1.0.
    signed: every value of A and B takes a random sign."""
    arp = np.arange(m + 1, dtype=np.int32) * a_per_row
    acol = np.concatenate([np.sort(rng.choice(K, a_per_row, replace=False)) for _ in range(m)]).astype(np.int32)
    A = CSR(m, K, arp, acol, np.full(m * a_per_row, a_val, np.float32))
    if signed:
        A.val[rng.random(len(A.val)) < 0.5] *= -1
    rows, vals = [], []
    for _ in range(K):
        c = np.sort(rng.choice(N, N // 2, replace=False)).astype(np.int32)
        v = np.where(rng.random(len(c)) < 0.25, 1.0, tiny).astype(np.float32)
        v[rng.integers(len(c))] = 1.0
        rows.append(c)
        vals.append(v)
    brp = np.zeros(K + 1, np.int32)
    brp[1:] = np.cumsum([len(c) for c in rows])
    bval = np.concatenate(vals)
    if signed:
        bval[rng.random(len(bval)) < 0.5] *= -1
    return A, CSR(K, N, brp, np.concatenate(rows), bval)


# (A rows, K, entries per A row, their value, B's small value): short rows,
# and rows longer than a numeric workgroup (512 entries)
FIXED_SHAPES = {"short": (300, 96, 24, 1.0, 2.0 ** -24), "short12": (300, 96, 12, 1.0, 2.0 ** -24),
                "long": (40, 1024, 600, 2.0 ** -10, 2.0 ** -20), "signed": (300, 96, 24, 1.0, 2.0 ** -24)}


@pytest.mark.parametrize("shape", list(FIXED_SHAPES))
@pytest.mark.parametrize("path", FIXED_PATHS)
def test_window_rows_fixed_point_exact(torch_gpu, path, shape):
    """Window rows whose bound allows it accumulate in fixed point.  Short:
    24 entries of 1 per A row, B values 1 or 2^-24; the row's bound is
    S = 24 < 2^5, so products are scaled by 2^25 (rounding error bound
    24 * 2^-26 < 1e-6); with 12 entries, S = 12 and scale 2^26.  Long: 600
    entries of 2^-10, B values 1 or 2^-20; S = 600 * 2^-10 < 2^0, scale
    2^30 (error bound 600 * 2^-31).  Signed: the short shape with random
    signs (negative products, sums that cancel to zero).  Every
    product is then an exact multiple of the scale's unit, the integer sum
    is exact and its one rounding to fp32 equals the oracle's fp64 sum
    (exact for these products too) rounded once: values bit-exact.  Summed
    in fp32 instead, a small term added to a partial sum many times larger
    is lost."""
    m, K, per, a_val, tiny = FIXED_SHAPES[shape]
    rng = np.random.default_rng(zlib.crc32((path + shape).encode()) + 1)
    A, B = ones_and_tiny(rng, m, K, 333, per, a_val, tiny, signed=shape == "signed")
    say("fixed-point exact %s %s" % (path, shape))
    ref = oracle.spgemm(A, B, f64=True)
    exact = ref.val64.astype(np.float32)  # the exact sums rounded once to fp32
    rp, col, val, st, _ = run(torch_gpu, A, B, **PATHS[path])
    assert np.array_equal(rp - rp[0], ref.rp) and np.array_equal(col, ref.col)
    assert np.array_equal(val, exact), "fixed-point sums differ from the exactly rounded ones at %d entries" % (
        (val != exact).sum())


@pytest.mark.parametrize("path", FIXED_PATHS)
def test_window_rows_fp32_where_bound_fails(torch_gpu, path):
    """Rows whose bound leaves too few fractional bits stay in fp32: an A row
    with one entry of 2^20 has S > 2^20, so a fixed-point scale would be at
    most 2^9 and would flush entries made only of 2^-24 products to zero.
    All values are positive (no cancellation), so fp32 sums in any order
    are within 24 * 2^-24 of the exact ones relative to each entry."""
    rng = np.random.default_rng(zlib.crc32(path.encode()) + 2)
    A, B = ones_and_tiny(rng, 300, 96, 333, 24, 1.0, 2.0 ** -24)
    A.val[A.rp[:-1]] = 2.0 ** 20  # each row's first entry
    say("fp32 fallback %s" % path)
    ref = oracle.spgemm(A, B, f64=True)
    rp, col, val, st, _ = run(torch_gpu, A, B, **PATHS[path])
    assert np.array_equal(rp - rp[0], ref.rp) and np.array_equal(col, ref.col)
    rel = np.abs(val.astype(np.float64) - ref.val64) / np.abs(ref.val64)
    assert rel.max() <= 2e-6, "relative error %g" % rel.max()


@pytest.mark.parametrize("path", list(PATHS))
def test_each_path_cfg1(torch_gpu, path):
    A, B = workloads.workload(1)
    check(torch_gpu, A, B, "cfg1/" + path, **PATHS[path])


# --------------------------------------------------- scaled workload shapes

def test_cfg2_scaled(torch_gpu):
    A, B = workloads.workload(2, n=32768)
    check(torch_gpu, A, B, "cfg2 n=32768")


def test_cfg3_scaled_wide(torch_gpu):
    """A*A with N = 40000 > 16384: hash bins plus 3 column windows (ragged)."""
    A, B = workloads.workload(3, n=40000)
    st, _, _ = check(torch_gpu, A, B, "cfg3 n=40000")
    assert st["kind_ms"]["numeric"]["windows"] > 0


@pytest.mark.parametrize("keep", [1, -1])
def test_cfg3_scaled_kept_bitmaps(torch_gpu, keep):
    """Symbolic bitmaps kept for every wide row (keep=1) or for none (-1);
    small windows so that windows of more than one run of terms occur."""
    A, B = workloads.workload(3, n=40000)
    check(torch_gpu, A, B, "cfg3 n=40000 keep_bitmap_products=%d" % keep, keep_bitmap_products=keep,
          window_grain_cols=4096, window_max_grains=8, window_max_entries=16384, count_grains=4)


@pytest.mark.parametrize("cache_bytes", [256 << 10, 4 << 20])
def test_cfg3_scaled_partial_bitmap_cache(torch_gpu, cache_bytes):
    """Kept bitmaps for every wide row, but a cache far too small for them
    (items of 4 grains of 4096 columns: 2 KB each, about 2 * 10^4 of them):
    the first items to claim cache chunks keep their bitmaps, the rest are
    marked again from their terms in the numeric phase, in the same launch."""
    A, B = workloads.workload(3, n=40000)
    check(torch_gpu, A, B, "cfg3 n=40000 bitmap cache %d bytes" % cache_bytes, keep_bitmap_products=1,
          bitmap_cache_bytes=cache_bytes, window_grain_cols=4096, window_max_grains=8, window_max_entries=16384,
          count_grains=4)


@pytest.mark.parametrize("slab,keep", [(1, 0), (20000, 1), (-1, 0)])
def test_cfg3_scaled_column_slabs(torch_gpu, slab, keep):
    """Windows of the rows above `slab` products spread over the numeric
    kernel's column slabs (1: every window row; -1: none), with 1024-column
    grains so that a row has windows in every slab; kept bitmaps from the
    default threshold or for every row."""
    A, B = workloads.workload(3, n=40000)
    check(torch_gpu, A, B, "cfg3 n=40000 slabs above %d products, keep %d" % (slab, keep),
          slab_min_products=slab, keep_bitmap_products=keep, window_grain_cols=1024, window_max_grains=3,
          window_max_entries=1024, count_grains=5)


def test_cfg3_scaled_small_windows(torch_gpu):
    """Many windows per row: 1024-column grains, windows of <= 4 grains and
    <= 1024 entries, 8 grains per symbolic item (64-word grains: wave sums)."""
    A, B = workloads.workload(3, n=40000)
    check(torch_gpu, A, B, "cfg3 n=40000 small windows", window_grain_cols=2048, window_max_grains=4,
          window_max_entries=2048, count_grains=8)
    check(torch_gpu, A, B, "cfg3 n=40000 1024-col grains", window_grain_cols=1024, window_max_grains=3,
          window_max_entries=1024, count_grains=5)


def test_cfg3_scaled_wide_grains(torch_gpu):
    """8192-column grains (256 bitmap words per grain) with symbolic items of
    2 grains over 5 grains (a ragged last item) and windows of <= 2 grains."""
    A, B = workloads.workload(3, n=40000)
    check(torch_gpu, A, B, "cfg3 n=40000 8192-col grains", window_grain_cols=8192, window_max_grains=2,
          window_max_entries=8192, count_grains=2)


def test_cfg3_scaled_narrow_block(torch_gpu):
    """A*A with 2048 < N <= 16384: hash bins plus single-window workgroup rows."""
    A, B = workloads.workload(3, n=12000)
    check(torch_gpu, A, B, "cfg3 n=12000")


def test_cfg4_scaled(torch_gpu):
    A, B = workloads.workload(4, n=65536)
    check(torch_gpu, A, B, "cfg4 n=65536")
    st, _, _ = check(torch_gpu, A, B, "cfg4 n=65536 split rows", split_min_products=4096)
    assert st["kind_ms"]["numeric"]["split"] > 0


def test_cfg5_scaled_int64_rowptr(torch_gpu):
    A, B = workloads.workload(5, n=50000)
    assert A.rp.dtype == np.int64
    check(torch_gpu, A, B, "cfg5 n=50000 (int64 A.row_ptr)")


def test_int64_rowptr_B(torch_gpu):
    A, B = workloads.workload(1, n=3000)
    B64 = CSR(B.nrows, B.ncols, B.rp.astype(np.int64), B.col, B.val)
    check(torch_gpu, A, B64, "int64 B.row_ptr")


# ----------------------------------------------------------------- tiling

def test_tiled_equals_untiled(torch_gpu):
    A, B = workloads.workload(2, n=20000)
    st1, n1, ref = check(torch_gpu, A, B, "cfg2 untiled")
    st2, n2, _ = check(torch_gpu, A, B, "cfg2 tiled", max_tile_rows=3001)
    assert n1 == 1 and n2 == 7


def test_tiled_wide(torch_gpu):
    A, B = workloads.workload(3, n=30000)
    check(torch_gpu, A, B, "cfg3 tiled wide", max_tile_rows=4099)


@pytest.mark.parametrize("keep", [1, 0])
def test_tiled_wide_kept_bitmaps(torch_gpu, keep):
    """In-core tiles with kept symbolic bitmaps: every tile's symbolic phase
    runs before any numeric phase, and a tile's numeric phase must decide
    which rows keep their bitmaps (and so where their windows are cut) from
    its own rows' products, not from the tile symbolised last.  Items of 2
    grains of 1024 columns and windows of up to 6 grains make the two cuts
    differ."""
    A, B = workloads.workload(3, n=30000)
    check(torch_gpu, A, B, "cfg3 tiled wide, kept bitmaps above %d products" % keep, max_tile_rows=7001,
          keep_bitmap_products=keep, window_grain_cols=1024, window_max_grains=6, window_max_entries=4096,
          count_grains=2)


def test_kept_bitmaps_cache_released(torch_gpu):
    """A budget whose slack, after the plan's peak, is 1.1 times C: the
    kept-bitmap cache (a fifth of the slack) is released after the symbolic
    phase so that C fits, and the numeric phase marks every window again,
    cut where the symbolic phase planned the cuts."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(3, n=30000)
    ref = oracle.spgemm(A, B)
    kw = dict(keep_bitmap_products=1, window_grain_cols=1024, window_max_grains=6, window_max_entries=4096,
              count_grains=2)
    dA, dB = aires.to_device(A), aires.to_device(B)
    with aires.tile_plan(dA, dB, 1 << 36, **kw) as plan:
        peak = aires.plan_info(plan).peak_bytes
    for slack in (1.1, 1.25):
        budget = peak + int(slack * 8 * ref.nnz) + (1 << 20)
        say("cache released: budget %d = peak %d + %.2f x C" % (budget, peak, slack))
        rp, col, val, st, _ = run(torch_gpu, A, B, budget, **kw)
        assert_match(rp, col, val, ref)


def test_streamed_tiles_host_c(torch_gpu):
    """A in pinned host memory, double-buffered tiles, C tiles copied to
    pinned host memory at the running offset (Algorithm 2, Phases I-III)."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(5, n=60000)
    ref = oracle.spgemm(A, B)
    pA, pB = aires.to_pinned(A), aires.to_pinned(B)
    budget = B.nbytes() + (4 << 20) + 2 * 1_500_000
    say("streamed cfg5 n=60000 budget=%d" % budget)
    with aires.tile_plan(pA, pB, budget, c_on_host=True, timing=True) as plan:
        info = aires.plan_info(plan)
        C = aires.spgemm(plan)
        st = aires.plan_stats(plan)
        assert info.ntiles >= 3
        assert info.c_bound_entries == int(np.minimum(oracle.products(A, B), B.ncols).sum())
        assert C.on_host
        assert_match(C.rp, C.col, C.val, ref)
        assert st["host_syncs"] == info.ntiles
        # each tile copies its own k+1 row pointers: one shared word per boundary
        assert st["h2d_bytes"] == A.nbytes() + B.nbytes() + 8 * (info.ntiles - 1)
        C.free()


@pytest.mark.parametrize("F", [16, 32, 256])
def test_streamed_feature_sizes(torch_gpu, F):
    """The streamed schedule across feature widths (the feature-size study
    runs F = 16 ... 256): out-of-core-shaped graph, features of width F at
    the same density, A in pinned host memory, C tiles to pinned host
    memory, a budget that forces several tiles; every entry against the
    oracle."""
    import paper_2507_02006_amd as aires
    A, _ = workloads.workload(5, n=60000)
    B = workloads.features(60000, F, 0.10, seed=1000 + F)
    ref = oracle.spgemm(A, B)
    pA, pB = aires.to_pinned(A), aires.to_pinned(B)
    budget = B.nbytes() + (4 << 20) + 2 * 1_500_000 + 8 * int(np.minimum(oracle.products(A, B), F).sum()) // 3
    say("streamed cfg5-shaped n=60000 F=%d budget=%d" % (F, budget))
    with aires.tile_plan(pA, pB, budget, c_on_host=True, timing=True) as plan:
        info = aires.plan_info(plan)
        assert info.ntiles >= 3
        C = aires.spgemm(plan)
        assert C.on_host
        assert_match(C.rp, C.col, C.val, ref)
        st = aires.plan_stats(plan)
        assert st["products"] == ref.products and st["nnz_c"] == ref.nnz
        C.free()


def test_streamed_tiles_device_c(torch_gpu):
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(4, n=40000)
    ref = oracle.spgemm(A, B)
    pA = aires.to_pinned(A)
    dB = aires.to_device(B)
    budget = B.nbytes() + (4 << 20) + 8 * 40001 + 8 * int(np.minimum(oracle.products(A, B), 128).sum()) \
        + 2 * 400_000
    say("streamed cfg4 n=40000 device C")
    with aires.tile_plan(pA, dB, budget) as plan:
        assert aires.plan_info(plan).ntiles >= 2
        # exact bound with B's row lengths read from its device row pointers
        assert aires.plan_info(plan).c_bound_entries == int(np.minimum(oracle.products(A, B), B.ncols).sum())
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)


def test_streamed_wide(torch_gpu):
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(3, n=20000)
    ref = oracle.spgemm(A, B)
    say("streamed wide cfg3 n=20000")
    for slab in (0, 1):
        with aires.tile_plan(aires.to_pinned(A), aires.to_device(B), 1 << 34, c_on_host=True, max_tile_rows=5000,
                             dense_max_cols=4096, window_grain_cols=4096, slab_min_products=slab) as plan:
            C = aires.spgemm(plan)
            assert_match(C.rp, C.col, C.val, ref)
            C.free()


# ------------------------------------------------------------- edge cases

def _csr(m, n, rows):
    rp = np.zeros(m + 1, np.int32)
    col, val = [], []
    for i, r in enumerate(rows):
        for j, v in r:
            col.append(j)
            val.append(v)
        rp[i + 1] = len(col)
    return CSR(m, n, rp, np.array(col, np.int32), np.array(val, np.float32))


def test_edge_empty_operands(torch_gpu):
    A = _csr(5, 4, [[]] * 5)
    B = workloads.random_csr(np.random.default_rng(0), 4, 7, 0.5)
    check(torch_gpu, A, B, "empty A")
    check(torch_gpu, B, _csr(7, 3, [[]] * 7), "empty B")
    check(torch_gpu, _csr(0, 4, []), B, "zero rows")


def test_edge_single_row_and_column(torch_gpu):
    rng = np.random.default_rng(2)
    check(torch_gpu, workloads.random_csr(rng, 1, 50, 0.5), workloads.random_csr(rng, 50, 1, 0.5), "1x50*50x1")
    check(torch_gpu, workloads.random_csr(rng, 300, 1, 0.5), workloads.random_csr(rng, 1, 900, 0.5), "outer")


def test_edge_hub_row(torch_gpu):
    """One row touching every B row: the heaviest row of the tile."""
    rng = np.random.default_rng(3)
    B = workloads.random_csr(rng, 5000, 512, 0.05)
    A = _csr(3, 5000, [[(k, 1.0) for k in range(5000)], [], [(7, 2.0)]])
    check(torch_gpu, A, B, "hub row narrow")
    B2 = workloads.random_csr(rng, 5000, 40000, 0.0005)
    check(torch_gpu, A, B2, "hub row wide")
    check(torch_gpu, A, B2, "hub row wide, kept bitmaps", keep_bitmap_products=1)
    check(torch_gpu, A, B2, "hub row wide, no kept bitmaps", keep_bitmap_products=-1)
    # three rows: a numeric grid of three workgroups, so three column slabs
    check(torch_gpu, A, B2, "hub row wide, column slabs", slab_min_products=1)


def test_edge_stored_zeros_kept(torch_gpu):
    A = _csr(2, 2, [[(0, 1.0), (1, 1.0)], [(0, 0.0)]])
    B = _csr(2, 3, [[(0, 1.0), (2, 5.0)], [(0, -1.0)]])
    rp, col, val, _, _ = run(torch_gpu, A, B)
    assert rp.tolist() == [0, 2, 4] and col.tolist() == [0, 2, 0, 2]
    assert val.tolist() == [0.0, 5.0, 0.0, 0.0]


@pytest.mark.parametrize("N", [4, 20000])
def test_edge_single_entry_rows_signed_zeros(torch_gpu, N):
    """Rows with a single A entry are written as a_ik times B_k: each value
    is still one product added to +0, so a product that is -0 comes out +0
    as in the oracle (bit patterns compared), in the dense (N = 4) and the
    hash (N = 20000) kernels."""
    A = _csr(3, 2, [[(0, -1.0)], [(1, 2.0)], [(0, 1.0), (1, 1.0)]])
    B = _csr(2, N, [[(0, 0.0), (3, 4.0)], [(0, -0.0), (2, 1.5)]])
    ref = oracle.spgemm(A, B)
    rp, col, val, _, _ = run(torch_gpu, A, B)
    assert rp.tolist() == ref.rp.tolist() and col.tolist() == ref.col.tolist()
    assert np.array_equal(val.view(np.uint32), ref.val.view(np.uint32)), (val, ref.val)
    assert not np.signbit(val[0]) and not np.signbit(val[2])


def test_determinism_of_structure(torch_gpu):
    A, B = workloads.workload(3, n=20000)
    r1 = run(torch_gpu, A, B)
    r2 = run(torch_gpu, A, B)
    assert np.array_equal(r1[0], r2[0]) and np.array_equal(r1[1], r2[1])
    assert np.allclose(r1[2], r2[2], rtol=1e-5, atol=1e-6)


# ------------------------------------------------- full size, every row

def device_bytes(*Ms):
    return sum(M.nbytes() for M in Ms)


def full_check(torch, A, B, name, budget=0, **kw):
    """The bench's launch configuration (one tile, default options) or the
    given plan options; every row of C against the oracle (row chunks over
    host threads); the allocator's measured peak within the budget."""
    import paper_2507_02006_amd as aires
    say("%s full size: planning and running" % name)
    dA, dB = aires.to_device(A), aires.to_device(B)
    with aires.tile_plan(dA, dB, budget, timing=True, **kw) as plan:
        info = aires.plan_info(plan)
        C = aires.spgemm(plan)
        torch.cuda.synchronize()
        st = aires.plan_stats(plan)
        ts = aires.plan_tile_stats(plan)
        peak = plan.allocator.peak
    say("%s: %d tiles, nnz(C) = %d, products = %d, %.1f ms; allocator peak %.2f GB" %
        (name, info.ntiles, st["nnz_c"], st["products"], st["total_ms"], peak / 1e9))
    assert peak + device_bytes(A, B) <= info.budget
    assert sum(t["products"] for t in ts) == st["products"]
    assert sum(t["nnz_c"] for t in ts) == st["nnz_c"] == C.nnz
    rp = C.rp.cpu().numpy()
    res = fullcheck.verify(A, B, rp, fullcheck.device_fetch(C), say=say)
    say("%s: every row verified (%d chunks, %d threads, max rel err %.2e)" %
        (name, res["chunks"], res["threads"], res["max_rel_err"]))
    assert res["products"] == st["products"]
    del C
    return info, st, ts


def test_cfg2_full(torch_gpu):
    A, B = workloads.workload(2)
    full_check(torch_gpu, A, B, "cfg2")


@pytest.mark.slow
def test_cfg3_full(torch_gpu):
    """The square product at full size (9.7 G entries of C, 77.6 GB in HBM):
    every row against the oracle."""
    A, B = workloads.workload(3)
    full_check(torch_gpu, A, B, "cfg3")


@pytest.mark.slow
def test_cfg4_full_tiled(torch_gpu):
    """8,388,608-node aggregation under a 64 GB budget, cut into row-block
    tiles by a tile cap (Algorithm 1), device-resident operands; every row."""
    say("cfg4 full size: generating")
    A, B = workloads.workload(4, verbose=True)
    info, st, ts = full_check(torch_gpu, A, B, "cfg4", budget=64 << 30, max_tile_bytes=256 << 20)
    assert info.ntiles >= 4
    assert [(t["r0"], t["r1"]) for t in ts][-1][1] == A.nrows


@pytest.mark.slow
def test_cfg5_full_streamed(torch_gpu):
    """68M-node aggregation, A (int64 row_ptr) and X in pinned host memory,
    32 GB device budget: row-block tiles stream host to HBM double-buffered
    and C tiles return to pinned host memory (Algorithm 2).  Every row of C
    against the oracle; the device bytes the library held, measured at its
    allocator, within the budget; the copies of tile t+1 overlap the
    products of tile t (HIP event instants per tile)."""
    import paper_2507_02006_amd as aires
    torch = torch_gpu
    hold = []

    def pinned(n, rp_dtype):
        def out(nnz):
            rp = torch.empty(n + 1, dtype=rp_dtype, pin_memory=True)
            col = torch.empty(max(nnz, 1), dtype=torch.int32, pin_memory=True)[:nnz]
            val = torch.empty(max(nnz, 1), dtype=torch.float32, pin_memory=True)[:nnz]
            hold.append((rp, col, val))
            return rp.numpy(), col.numpy(), val.numpy()
        return out

    n = workloads.CONFIGS[5]["n"]
    say("cfg5 full size: generating into pinned memory")
    A, B = workloads.workload(5, out_a=pinned(n, torch.int64), out_b=pinned(n, torch.int32), verbose=True)
    assert A.rp.dtype == np.int64
    tA = (A.nrows, A.ncols) + hold[0]
    tB = (B.nrows, B.ncols) + hold[1]
    say("cfg5 nnzA=%d nnzB=%d" % (A.nnz, B.nnz))
    budget = 32 << 30
    with aires.tile_plan(tA, tB, budget, c_on_host=True, max_tile_bytes=768 << 20, timing=True) as plan:
        info = aires.plan_info(plan)
        say("cfg5 plan: %d tiles, peak %.2f GB of %d GB" % (info.ntiles, info.peak_bytes / 1e9, 32))
        assert info.a_streamed and info.c_on_host and info.ntiles >= 8
        assert info.peak_bytes <= budget
        C = aires.spgemm(plan)
        st = aires.plan_stats(plan)
        ts = aires.plan_tile_stats(plan)
        peak = plan.allocator.peak
        compute_ms = sum(st[k] for k in ("analyze_ms", "bin_ms", "symbolic_ms", "scan_ms", "numeric_ms"))
        say("cfg5 streamed: nnzC=%d total_ms=%.1f pipeline_ms=%.1f h2d_ms=%.1f compute_ms=%.1f d2h_ms=%.1f "
            "h2d=%.2fGB d2h=%.2fGB allocator peak %.2f GB" %
            (st["nnz_c"], st["total_ms"], st["pipeline_ms"], st["h2d_ms"], compute_ms, st["d2h_ms"],
             st["h2d_bytes"] / 1e9, st["d2h_bytes"] / 1e9, peak / 1e9))
        # A and X live in host memory: every device byte is the library's
        assert 0 < peak <= budget
        assert st["host_syncs"] == info.ntiles
        assert st["h2d_bytes"] == A.nbytes() + B.nbytes() + 8 * (info.ntiles - 1)
        assert sum(t["h2d_bytes"] for t in ts) == A.nbytes() + 8 * (info.ntiles - 1)
        assert sum(t["d2h_bytes"] for t in ts) == st["d2h_bytes"]
        assert sum(t["products"] for t in ts) == st["products"]
        assert sum(t["nnz_c"] for t in ts) == st["nnz_c"]
        # Algorithm 2's overlap, read from the event instants: tile t+1's
        # copy begins before tile t's products end, and the copies of C
        # trail the tile that made them
        for t in range(info.ntiles - 1):
            assert ts[t + 1]["h2d_begin_ms"] < ts[t]["compute_end_ms"], t
            assert ts[t]["d2h_begin_ms"] >= ts[t]["compute_end_ms"] - 1e-3, t
        assert st["pipeline_ms"] < 0.9 * (st["h2d_ms"] + compute_ms + st["d2h_ms"])
        assert C.on_host
        res = fullcheck.verify(A, B, C.rp, fullcheck.host_fetch(C), say=say)
        say("cfg5: every row verified (%d chunks, %d threads, max rel err %.2e)" %
            (res["chunks"], res["threads"], res["max_rel_err"]))
        assert res["products"] == st["products"]
        C.free()


# ------------------------------------------- values derived from the pattern (Eq. 2)

def _identity(n, scale=1.0):
    return CSR(n, n, np.arange(n + 1, dtype=np.int32), np.arange(n, dtype=np.int32), np.full(n, scale, np.float32))


# C = A * (2^64 I): the rows' bound (>= 2^44 here) leaves fixed point no
# fractional bits, so the product runs in fp32, where an entry made of one
# product is exact; the power-of-two scale is exact too.
CARRIER = 2.0 ** 64


@pytest.mark.parametrize("n", [20000, 1048576])
def test_sym_norm_values_bitwise(torch_gpu, n):
    """a_values='sym_norm': C = A_norm * (2^64 I) gives 2^64 / sqrt(r_i r_j)
    bit for bit (double arithmetic, one rounding to fp32) with A's own values
    not passed at all, against the oracle's Eq. 2 (oracle.sym_norm) on the
    square workload's graph scaled and at full size."""
    import paper_2507_02006_amd as aires
    A, _ = workloads.workload(3, n=n)
    dA = aires.to_device(A)
    say("sym_norm values n=%d nnz=%d" % (n, A.nnz))
    with aires.tile_plan(dA[:4] + (None,), aires.to_device(_identity(A.ncols, CARRIER)), 0,
                         a_values="sym_norm") as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(rp, A.rp.astype(np.int64))
    assert np.array_equal(col, A.col)
    want = oracle.sym_norm(A.rp, A.col) * np.float32(CARRIER)
    assert np.array_equal(val.view(np.uint32), want.view(np.uint32))


def test_sym_norm_values_sparse_rows(torch_gpu):
    """Derived values when runs of empty rows make a 2048-entry chunk span
    more rows than the kernel stages in LDS (its global-search branch):
    C = A_norm * (2^64 I) against the oracle's Eq. 2 scaled alike."""
    import paper_2507_02006_amd as aires
    rng = np.random.default_rng(31)
    m = 200000
    full = np.arange(0, m, 97)  # non-empty rows; columns only among them
    lens = np.zeros(m, np.int64)
    lens[full] = rng.integers(1, 60, len(full))
    cols = [np.sort(rng.choice(full, int(L), replace=False)) for L in lens[full]]
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    col = np.concatenate(cols).astype(np.int32)
    A = CSR(m, m, rp, col, np.zeros(len(col), np.float32))
    want = oracle.sym_norm(rp, col) * np.float32(CARRIER)
    dA = aires.to_device(A)
    say("sym_norm sparse rows m=%d nnz=%d" % (m, len(col)))
    with aires.tile_plan(dA[:4] + (None,), aires.to_device(_identity(m, CARRIER)), 0,
                         a_values="sym_norm") as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        c_col, c_val = C.col.cpu().numpy(), C.val.cpu().numpy()
    assert np.array_equal(c_col, col)
    assert np.array_equal(c_val.view(np.uint32), want.view(np.uint32))


def test_sym_norm_incore_equals_given(torch_gpu):
    """In-core tiles with derived values: the same structure as with the
    given values and both within the bar of the oracle (the order of the
    fp32 sums in LDS differs from run to run, so values are not compared
    bit for bit; the derived values themselves are, above)."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(2, n=8192)
    dA, dB = aires.to_device(A), aires.to_device(B)
    say("sym_norm in-core cfg2 n=8192")
    out = []
    for mode, a in (("given", dA), ("sym_norm", dA[:4] + (None,))):
        with aires.tile_plan(a, dB, 0, a_values=mode, max_tile_rows=3001) as plan:
            C = aires.spgemm(plan)
            torch_gpu.cuda.synchronize()
            out.append((C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()))
    ref = oracle.spgemm(A, B)
    for rp, col, val in out:
        assert_match(rp, col, val, ref)
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])


def test_sym_norm_streamed_equals_given(torch_gpu):
    """Streamed tiles with derived values: A's row pointers cross the host
    link once and each tile sends only its column indices; the structure
    equals that of the given values and both meet the oracle's bar."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(5, n=60000)
    pA, pB = aires.to_pinned(A), aires.to_pinned(B)
    budget = B.nbytes() + (4 << 20) + 8 * (A.nrows + 1) + 2 * 1_500_000
    say("sym_norm streamed cfg5 n=60000 budget=%d" % budget)
    out = []
    for mode, a in (("given", pA), ("sym_norm", pA[:4] + (None,))):
        with aires.tile_plan(a, pB, budget, c_on_host=True, timing=True, a_values=mode) as plan:
            info = aires.plan_info(plan)
            C = aires.spgemm(plan)
            st = aires.plan_stats(plan)
            assert info.ntiles >= 3
            out.append((C.rp.copy(), C.col.copy(), C.val.copy()))
            C.free()
    assert st["h2d_bytes"] == 8 * (A.nrows + 1) + 4 * A.nnz + B.nbytes()
    ref = oracle.spgemm(A, B)
    for rp, col, val in out:
        assert_match(rp, col, val, ref)
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])


def test_sym_norm_streamed_device_c(torch_gpu):
    """Derived values with a streamed A and C kept in device memory (the
    schedule with no copies back), against the oracle on the generator's
    values; two tiles or more under the budget."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(4, n=40000)
    ref = oracle.spgemm(A, B)
    pA = aires.to_pinned(A)
    dB = aires.to_device(B)
    budget = B.nbytes() + (4 << 20) + 8 * 40001 + 8 * int(np.minimum(oracle.products(A, B), 128).sum()) \
        + 4 * 40001 + 2 * 400_000
    say("sym_norm streamed cfg4 n=40000 device C")
    with aires.tile_plan(pA[:4] + (None,), dB, budget, a_values="sym_norm", timing=True) as plan:
        assert aires.plan_info(plan).ntiles >= 2
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        st = aires.plan_stats(plan)
        assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)
    assert st["h2d_bytes"] == 4 * (A.nrows + 1) + 4 * A.nnz


def test_streamed_rows_bound(torch_gpu):
    """Streamed tiles planned with the gather-free C bound (c_bound = ROWS):
    the same C as the oracle."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B = workloads.workload(5, n=60000)
    ref = oracle.spgemm(A, B)
    pA, pB = aires.to_pinned(A), aires.to_pinned(B)
    # P_i is not computed on the host, so the split rows' slots take their cap
    budget = B.nbytes() + (24 << 20) + 2 * 3_000_000
    say("streamed cfg5 n=60000 rows bound budget=%d" % budget)
    with aires.tile_plan(pA, pB, budget, c_on_host=True, c_bound=B_.CBOUND_ROWS) as plan:
        assert aires.plan_info(plan).ntiles >= 3
        C = aires.spgemm(plan)
        assert_match(C.rp, C.col, C.val, ref)
        C.free()


# ------------------------------------- max-fill segments (the unaligned baseline)

@pytest.mark.parametrize("c_on_host", [True, False])
def test_maxfill_streamed(torch_gpu, c_on_host):
    """Segments filled to their slot that end inside rows (Sec. III-A's
    unaligned scheme): the same C as the oracle and as row blocks; every
    partial row is copied back and sent again, which the byte counts show
    exactly."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(5, n=60000)
    ref = oracle.spgemm(A, B)
    pA, pB = aires.to_pinned(A), aires.to_pinned(B)
    budget = 1 << 32
    say("max-fill streamed cfg5 n=60000 c_on_host=%s" % c_on_host)
    out = {}
    for seg in ("maxfill", "robw"):
        with aires.tile_plan(pA, pB, budget, c_on_host=c_on_host, timing=True, max_tile_bytes=300_000,
                             segmentation=seg) as plan:
            tiles = aires.plan_tiles(plan)
            C = aires.spgemm(plan)
            torch_gpu.cuda.synchronize()
            st = aires.plan_stats(plan)
            ts = aires.plan_tile_stats(plan)
            if c_on_host:
                got = (C.rp.copy(), C.col.copy(), C.val.copy())
                C.free()
            else:
                got = (C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy())
        assert_match(*got, ref)
        out[seg] = (tiles, st, ts)
    tiles, st, ts = out["maxfill"]
    nt = len(tiles)
    carried = sum(t["sent_nnz1"] - t["nnz1"] for t in tiles)
    assert nt >= 10 and carried > 0
    assert st["resent_bytes"] == 8 * carried
    assert st["h2d_bytes"] == A.nbytes() + B.nbytes() + 8 * (nt - 1) + 8 * carried
    assert sum(t["resent_bytes"] for t in ts) == 8 * carried
    assert st["merge_ms"] > 0 and all(t["merge_ms"] >= 0 for t in ts)
    assert st["host_syncs"] == nt + sum(1 for t in tiles[:-1] if t["sent_nnz1"] > t["nnz1"])
    assert out["robw"][1]["resent_bytes"] == 0 and out["robw"][1]["merge_ms"] == 0


def test_maxfill_streamed_wide(torch_gpu):
    """Max-fill segments of a wide product (column windows), C to host."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(3, n=20000)
    ref = oracle.spgemm(A, B)
    say("max-fill streamed wide cfg3 n=20000")
    with aires.tile_plan(aires.to_pinned(A), aires.to_device(B), 1 << 34, c_on_host=True, max_tile_bytes=120_000,
                         dense_max_cols=4096, window_grain_cols=4096, segmentation="maxfill") as plan:
        assert aires.plan_info(plan).ntiles >= 5
        C = aires.spgemm(plan)
        assert_match(C.rp, C.col, C.val, ref)
        C.free()


@pytest.mark.parametrize("c_on_host", [True, False])
def test_streamed_eq5_bound_grows(torch_gpu, c_on_host):
    """The paper's Eq. 5 estimate as the C bound undershoots the square
    product's C many times over: C's arrays grow as tiles complete and the
    result still equals the oracle's."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B = workloads.workload(3, n=20000)
    ref = oracle.spgemm(A, B)
    say("streamed Eq. 5 bound, square n=20000, c_on_host=%s" % c_on_host)
    with aires.tile_plan(aires.to_pinned(A), aires.to_device(B), 1 << 34, c_on_host=c_on_host, timing=True,
                         c_bound=B_.CBOUND_PAPER_EQ5, max_tile_bytes=100_000, dense_max_cols=4096,
                         window_grain_cols=4096) as plan:
        info = aires.plan_info(plan)
        assert info.ntiles >= 4 and info.c_bound_entries * 4 < ref.nnz
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        if c_on_host:
            assert_match(C.rp, C.col, C.val, ref)
            C.free()
        else:
            assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)


# ------------------------------------------------------- A on storage (a file)

@pytest.mark.parametrize("direct,c_on_host,values", [(1, True, "given"), (0, False, "given"), (1, True, "sym_norm")])
def test_storage_tier_streamed(torch_gpu, tmp_path, direct, c_on_host, values):
    """A's arrays in a file: each tile is read into pinned staging (direct
    I/O or the page cache), then streamed as from pinned memory; the same C
    as the oracle, and every byte of A read exactly once."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B = workloads.workload(5, n=60000)
    ref = oracle.spgemm(A, B)
    meta = workloads.write_csr_file(str(tmp_path / "a.csr"), A)
    budget = B.nbytes() + (24 << 20) + 8 * (A.nrows + 1) + 2 * 3_000_000
    say("storage tier cfg5 n=60000 direct=%d c_on_host=%s values=%s" % (direct, c_on_host, values))
    with aires.tile_plan_file(meta, aires.to_pinned(B), budget if c_on_host else 1 << 32, c_on_host=c_on_host,
                              timing=True, direct_io=bool(direct), max_tile_bytes=200_000, a_values=values) as plan:
        info = aires.plan_info(plan)
        assert info.a_in_file and info.ntiles >= 5
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        st = aires.plan_stats(plan)
        ts = aires.plan_tile_stats(plan)
        if c_on_host:
            assert_match(C.rp, C.col, C.val, ref)
            C.free()
        else:
            assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)
    per_entry = 8 if values == "given" else 4
    assert st["storage_bytes"] == per_entry * A.nnz
    assert st["storage_ms"] > 0 and sum(t["storage_ms"] for t in ts) == pytest.approx(st["storage_ms"])
    if values == "given":
        assert st["h2d_bytes"] == A.nbytes() + B.nbytes() + 8 * (info.ntiles - 1)


# ----------------------------------------------- B on storage (a file) too

@pytest.mark.parametrize("which,mem,direct,chunk", [("features", "device", 1, 1 << 20), ("features", "device", 0, 0),
                                                     ("graph", "device", 1, 4096), ("features", "pinned", 1, 0),
                                                     ("graph", "pinned", 0, 0), ("empty", "device", 1, 0),
                                                     ("empty", "pinned", 0, 0)])
def test_read_csr_file(torch_gpu, tmp_path, which, mem, direct, chunk):
    """A CSR read whole from a file (aires_csr_read_file) into device or
    pinned memory, in chunks through two pinned staging buffers (1 MiB:
    several chunks and a ragged last one; 4 KiB: many): row pointers widened
    to int64, every array equal to what was written, bitwise."""
    import paper_2507_02006_amd as aires
    A, X = workloads.workload(5, n=60000)
    M = X if which == "features" else workloads.workload(1)[0] if which == "graph" else \
        workloads.CSR(5, 9, np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    meta = workloads.write_csr_file(str(tmp_path / "m.csr"), M)
    meta["direct_io"] = bool(direct)
    say("read_csr_file %s mem=%s direct=%d chunk=%d nnz=%d" % (which, mem, direct, chunk, M.nnz))
    out, st = aires.read_csr_file(meta, mem=mem, chunk_bytes=chunk)
    if mem == "device":
        torch_gpu.cuda.synchronize()
        rp, col, val = out.rp.cpu().numpy(), out.col.cpu().numpy(), out.val.cpu().numpy()
    else:
        rp, col, val = out.rp.copy(), out.col.copy(), out.val.copy()
        out.free()
    assert rp.dtype == np.int64 and np.array_equal(rp, M.rp.astype(np.int64))
    assert np.array_equal(col, M.col) and np.array_equal(val.view(np.int32), M.val.view(np.int32))
    assert st["bytes_read"] == M.rp.nbytes + 8 * M.nnz and st["total_ms"] >= st["read_ms"] >= 0


@pytest.mark.parametrize("c_on_host", [True, False])
def test_storage_tier_both_ways(torch_gpu, tmp_path, c_on_host):
    """A and B both in files: B read once into device memory before the
    tiles (aires_csr_read_file), A's tiles read from their file and streamed
    (aires_tile_plan_file); the same C as the oracle."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(5, n=60000)
    ref = oracle.spgemm(A, B)
    ma = workloads.write_csr_file(str(tmp_path / "a.csr"), A)
    mb = workloads.write_csr_file(str(tmp_path / "b.csr"), B)
    say("storage tier, A and B in files, cfg5 n=60000 c_on_host=%s" % c_on_host)
    Bd, st = aires.read_csr_file(mb, mem="device", chunk_bytes=1 << 20)
    dB = (B.nrows, B.ncols, Bd.rp, Bd.col, Bd.val)
    budget = B.nbytes() + 8 * (B.nrows + 1) + (24 << 20) + 8 * (A.nrows + 1) + 2 * 3_000_000
    with aires.tile_plan_file(ma, dB, budget if c_on_host else 1 << 32, c_on_host=c_on_host,
                              max_tile_bytes=200_000) as plan:
        assert aires.plan_info(plan).ntiles >= 5
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        if c_on_host:
            assert_match(C.rp, C.col, C.val, ref)
            C.free()
        else:
            assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)
