"""GPU parity of the combination step Y = act(A * W) (aires_spmm, Sec. II-A
Eq. 3) through the C-ABI against the oracle's double-precision product.

Bar: every entry within the fp32 summation error bound of the GPU's
arbitrary order with fused multiply-adds,
    |y - y64| <= (n_i + 2) * 2^-24 * sum_k |a_ik w_kj| + 2^-24 * |y64|,
where n_i is the number of stored entries of row i (the standard bound
gamma_n for a sum of n_i rounded terms, plus the final rounding); exact
(bit-equal to the integer product) when every value is a small integer.
Both kernel families are held to it: the entry gather ("rows") and the
densified tiles on the matrix cores ("dense_tiles"), whose extra products
with absent entries are exact zeros for finite W."""
import numpy as np
import pytest

import oracle
import workloads
from workloads import CSR

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
ALGOS = ["rows", "dense_tiles"]


@pytest.fixture(scope="module")
def torch_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    return torch


def say(msg):
    print("[gpu-case] " + msg, flush=True)


def dev_csr(torch, A, rp64=False, a_offset=0):
    """A on the device; a_offset > 0 starts its column and value arrays that
    many elements into their allocations (off 16-byte alignment for 1-3)."""
    rp = A.rp.astype(np.int64 if rp64 else np.int32)
    col = torch.zeros(A.nnz + a_offset, dtype=torch.int32, device="cuda")[a_offset:]
    val = torch.zeros(A.nnz + a_offset, dtype=torch.float32, device="cuda")[a_offset:]
    col.copy_(torch.from_numpy(A.col.astype(np.int32)))
    val.copy_(torch.from_numpy(A.val.astype(np.float32)))
    return (A.nrows, A.ncols, torch.from_numpy(rp).cuda(), col, val)


def check(torch, A, W, relu=False, rp64=False, ldw_pad=0, ldy_pad=0, w_offset=0, exact=False, name="",
          algo="auto", a_offset=0):
    import paper_2507_02006_amd as aires
    say("%s algo=%s m=%d K=%d F=%d relu=%d rp64=%d pads=(%d,%d) off=%d a_off=%d" % (
        name, algo, A.nrows, A.ncols, W.shape[1], relu, rp64, ldw_pad, ldy_pad, w_offset, a_offset))
    K, F = W.shape
    buf = torch.zeros(K * (F + ldw_pad) + w_offset + 1, dtype=torch.float32, device="cuda")
    Wd = buf[w_offset:w_offset + K * (F + ldw_pad)].view(K, F + ldw_pad)[:, :F]
    Wd.copy_(torch.from_numpy(W))
    ybuf = torch.full((A.nrows, F + ldy_pad), 7.0, dtype=torch.float32, device="cuda")
    Y = aires.spmm(dev_csr(torch, A, rp64, a_offset), Wd, relu=relu, out=ybuf[:, :F], algo=algo)
    torch.cuda.synchronize()
    y = Y.cpu().numpy().astype(np.float64)
    if ldy_pad:
        assert np.all(ybuf[:, F:].cpu().numpy() == 7.0), "columns past F were written"
    ref, refabs = oracle.spmm(A, W, relu=relu)
    if exact:
        assert np.array_equal(y, ref), name
        return
    n = np.diff(A.rp.astype(np.int64))[:, None]
    tol = (n + 2) * U * refabs + U * np.abs(ref)
    err = np.abs(y - ref)
    bad = err > tol
    assert not bad.any(), "%s: %d entries over the bound, worst %g" % (name, bad.sum(), (err - tol).max())


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("F", [1, 7, 64, 65, 100, 128, 129, 200, 256, 512, 700])
def test_widths(torch_gpu, F, algo):
    """Rows: one wavefront pass covers 64*V columns (V = 1, 2, 4, 8); 700
    takes two passes; F not a multiple of the vector takes the scalar tail.
    Dense tiles: 64- or 128-column tiles, ragged in m (300), K (90) and F."""
    rng = np.random.default_rng(F)
    A = workloads.random_csr(rng, 300, 90, 0.05)
    W = rng.uniform(-1, 1, (90, F)).astype(np.float32)
    check(torch_gpu, A, W, name="width %d" % F, algo=algo)


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("relu", [False, True])
def test_integer_values_exact(torch_gpu, relu, algo):
    """Small integers: every product and partial sum is exact in fp32, so Y
    equals the integer product whatever the order."""
    rng = np.random.default_rng(5)
    Ad = rng.integers(-3, 4, (257, 129)) * (rng.random((257, 129)) < 0.1)
    A = CSR(257, 129, *_csr_parts(Ad))
    W = rng.integers(-3, 4, (129, 96)).astype(np.float32)
    check(torch_gpu, A, W, relu=relu, exact=True, name="integer relu=%d" % relu, algo=algo)


def _csr_parts(D):
    rows, cols = np.nonzero(D)
    rp = np.zeros(D.shape[0] + 1, dtype=np.int64)
    np.add.at(rp, rows + 1, 1)
    return np.cumsum(rp).astype(np.int32), cols.astype(np.int32), D[rows, cols].astype(np.float32)


@pytest.mark.parametrize("algo", ALGOS)
def test_heavy_rows_split_over_a_workgroup(torch_gpu, algo):
    """Rows above 512 entries take the workgroup kernel (four wavefronts
    and an LDS reduction); mixed with light and empty rows.  For dense
    tiles, rows with more than 32 entries in a 64-column chunk take several
    load rounds."""
    rng = np.random.default_rng(7)
    K = 3000
    lens = np.array([0, 3, 513, 512, 2999, 0, 1, 1500, 700, 5] * 4)
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    col = np.concatenate([np.sort(rng.choice(K, L, replace=False)) for L in lens]).astype(np.int32)
    val = rng.uniform(-1, 1, len(col)).astype(np.float32)
    A = CSR(len(lens), K, rp, col, val)
    for F in (64, 256, 600):
        W = rng.uniform(-1, 1, (K, F)).astype(np.float32)
        check(torch_gpu, A, W, relu=True, name="heavy F=%d" % F, algo=algo)


@pytest.mark.parametrize("algo", ALGOS)
def test_strides_offsets_and_rp64(torch_gpu, algo):
    """Row strides above F (padding untouched), a W base that is not
    vector-aligned (scalar loads), and 64-bit row pointers."""
    rng = np.random.default_rng(8)
    A = workloads.random_csr(rng, 200, 70, 0.1)
    W = rng.uniform(-1, 1, (70, 256)).astype(np.float32)
    check(torch_gpu, A, W, ldw_pad=3, ldy_pad=5, name="pads", algo=algo)
    check(torch_gpu, A, W, ldw_pad=4, name="aligned pad", algo=algo)
    check(torch_gpu, A, W, w_offset=1, name="unaligned W", algo=algo)
    check(torch_gpu, A, W, rp64=True, relu=True, name="rp64", algo=algo)
    for off in (1, 2, 4):  # A's arrays off 16-byte alignment (single-entry loads), then back on it
        check(torch_gpu, A, W, a_offset=off, name="A offset %d" % off, algo=algo)


def test_edges(torch_gpu):
    import paper_2507_02006_amd as aires
    torch = torch_gpu
    rng = np.random.default_rng(9)
    E = CSR(6, 10, np.zeros(7, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    W = rng.uniform(-1, 1, (10, 33)).astype(np.float32)
    for algo in ALGOS:
        check(torch, E, W, name="all rows empty", algo=algo)
    check(torch, CSR(5, 0, np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32)),
          np.zeros((0, 20), np.float32), name="K = 0", algo="dense_tiles")
    Y = aires.spmm(dev_csr(torch, CSR(0, 10, np.zeros(1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))),
                   torch.from_numpy(W).cuda())
    assert Y.shape == (0, 33)
    A = workloads.random_csr(rng, 8, 10, 0.5)
    Y = aires.spmm(dev_csr(torch, A), torch.zeros((10, 0), device="cuda"))
    assert Y.shape == (8, 0)
    with pytest.raises(ValueError):
        aires.spmm(dev_csr(torch, A), torch.zeros((11, 4), device="cuda"))
    with pytest.raises(ValueError):
        aires.spmm(dev_csr(torch, A), torch.zeros((10, 4), device="cuda"), algo="gemm")


@pytest.mark.parametrize("density", [0.3, 1.0])
def test_dense_tiles_dense_rows(torch_gpu, density):
    """Fully dense and 30 % rows: 64 entries per 64-column chunk (two load
    rounds of 32 and a third that finds the chunk's end), K not a multiple
    of 64, several column tiles on the XCD-ordered grid."""
    rng = np.random.default_rng(int(density * 10))
    A = workloads.random_csr(rng, 517, 333, density)
    for F in (48, 300):
        W = rng.uniform(-1, 1, (333, F)).astype(np.float32)
        check(torch_gpu, A, W, relu=True, name="dense rows %.1f F=%d" % (density, F), algo="dense_tiles")
        check(torch_gpu, A, W, name="dense rows %.1f F=%d A offset 1" % (density, F), algo="dense_tiles",
              a_offset=1)


def test_dense_tiles_grid_loop(torch_gpu):
    """More tiles than the grid (65536 blocks): the second sweep of the
    persistent loop, checked on sampled rows and the last rows (1 075 200
    rows, one entry each, K = 16, F = 512: 67200 tiles)."""
    import paper_2507_02006_amd as aires
    torch = torch_gpu
    rng = np.random.default_rng(12)
    m, K, F = 1075200, 16, 512
    rp = np.arange(m + 1, dtype=np.int32)
    col = (np.arange(m) * 7 % K).astype(np.int32)
    val = rng.integers(-4, 5, m).astype(np.float32)
    A = CSR(m, K, rp, col, val)
    W = rng.integers(-8, 9, (K, F)).astype(np.float32)
    say("grid loop m=%d K=%d F=%d" % (m, K, F))
    Y = aires.spmm(dev_csr(torch, A), torch.from_numpy(W).cuda(), algo="dense_tiles")
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([rng.integers(0, m, 2000), np.arange(m - 3000, m)]))
    y = Y[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    sub = CSR(len(rows), K, np.arange(len(rows) + 1, dtype=np.int32), col[rows], val[rows])
    ref, _ = oracle.spmm(sub, W)
    assert np.array_equal(y, ref)


def test_gcn_layer_on_aggregated_features(torch_gpu):
    """A GCN layer H' = relu((A_norm X) W) (Eqs. 1-3): the aggregation from
    aires_spgemm, then the combination on its CSR output (int64 row
    pointers), against the oracle on the oracle's aggregation."""
    import paper_2507_02006_amd as aires
    torch = torch_gpu
    A, X = workloads.workload(2, n=8192)  # cfg2 scaled down: F_in = 512 features at 5 %
    rng = np.random.default_rng(10)
    W = rng.uniform(-0.5, 0.5, (X.ncols, 64)).astype(np.float32)
    say("gcn layer m=%d nnzA=%d F_in=%d F_out=64" % (A.nrows, A.nnz, X.ncols))
    with aires.tile_plan(aires.to_device(A), aires.to_device(X), 0) as plan:
        C = aires.spgemm(plan)
        Wd = torch.from_numpy(W).cuda()
        H = aires.spmm((C.nrows, C.ncols, C.rp, C.col, C.val), Wd, relu=True)
        torch.cuda.synchronize()
        h = H.cpu().numpy().astype(np.float64)
    Co = oracle.spgemm(A, X)
    ref, refabs = oracle.spmm(CSR(Co.r1 - Co.r0, Co.ncols, Co.rp, Co.col, Co.val), W, relu=True)
    # C itself differs from the oracle's by at most 1e-5 (1 + |c|) per entry
    n = np.diff(Co.rp)[:, None]
    cabs, _ = oracle.spmm(CSR(Co.r1 - Co.r0, Co.ncols, Co.rp, Co.col, np.abs(Co.val)), np.abs(W))
    tol = (n + 2) * U * refabs + U * np.abs(ref) + 1e-5 * (np.abs(W).sum(0)[None, :] + cabs)
    assert np.all(np.abs(h - ref) <= tol)


@pytest.mark.slow
@pytest.mark.parametrize("algo", ALGOS)
def test_full_cfg2_combination_sampled(torch_gpu, algo):
    """The combination step at the size the bench times: relu(C W) with C
    the aggregate of the full cfg2 (262144 x 512, 39.2 M entries) from
    aires_spgemm and W 512 x 256, checked on sampled rows and the heaviest
    rows against the oracle's product of the oracle's aggregate rows."""
    import paper_2507_02006_amd as aires
    torch = torch_gpu
    A, X = workloads.workload(2)
    rng = np.random.default_rng(21)
    W = rng.uniform(-0.05, 0.05, (X.ncols, 256)).astype(np.float32)
    say("full cfg2 combination algo=%s" % algo)
    with aires.tile_plan(aires.to_device(A), aires.to_device(X), 0) as plan:
        C = aires.spgemm(plan)
        H = aires.spmm((C.nrows, C.ncols, C.rp, C.col, C.val), torch.from_numpy(W).cuda(), relu=True, algo=algo)
        torch.cuda.synchronize()
        crow = np.diff(C.rp.cpu().numpy())
        rows = np.unique(np.concatenate([rng.choice(A.nrows, 200, replace=False), np.argsort(crow)[-5:],
                                         [0, A.nrows - 1]]))
        h = H[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    for r, hr in zip(rows, h):
        Co = oracle.spgemm(A, X, int(r), int(r) + 1)
        row = CSR(1, Co.ncols, Co.rp, Co.col, Co.val)
        ref, refabs = oracle.spmm(row, W, relu=True)
        cabs, _ = oracle.spmm(CSR(1, Co.ncols, Co.rp, Co.col, np.abs(Co.val)), np.abs(W))
        n = len(Co.col)
        tol = (n + 2) * U * refabs + U * np.abs(ref) + 1e-5 * (np.abs(W).sum(0)[None, :] + cabs)
        assert np.all(np.abs(hr[None, :] - ref) <= tol), "row %d" % r
