"""Pins for the CPU oracle: each test ties the oracle to something other
than itself (dense products, hand-worked examples, closed forms of the
normalised operator, invariants, brute force, an independent library and
the standard summation error bound).  CPU only."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads
from workloads import CSR


def from_dense(D, pattern=None, rp64=False):
    """CSR of a dense array; `pattern` (bool) fixes the stored positions so
    stored zeros can be represented."""
    D = np.asarray(D, dtype=np.float32)
    mask = (D != 0) if pattern is None else np.asarray(pattern, dtype=bool)
    rows, cols = np.nonzero(mask)
    rp = np.zeros(D.shape[0] + 1, dtype=np.int64)
    np.add.at(rp, rows + 1, 1)
    rp = np.cumsum(rp)
    return CSR(D.shape[0], D.shape[1], rp if rp64 else rp.astype(np.int32),
               cols.astype(np.int32), D[rows, cols].astype(np.float32))


def to_dense(P, nrows):
    D = np.zeros((nrows, P.ncols), dtype=np.float64)
    S = np.zeros((nrows, P.ncols), dtype=bool)
    for i in range(nrows):
        cols = P.col[P.rp[i]:P.rp[i + 1]]
        D[i, cols] = P.val[P.rp[i]:P.rp[i + 1]]
        S[i, cols] = True
    return D, S


def pattern_dense(M):
    S = np.zeros((M.nrows, M.ncols), dtype=bool)
    rp = M.rp.astype(np.int64)
    for i in range(M.nrows):
        S[i, M.col[rp[i]:rp[i + 1]]] = True
    return S


def check_canonical(P):
    rp = P.rp
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0) and rp[-1] == len(P.col)
    for i in range(len(rp) - 1):
        c = P.col[rp[i]:rp[i + 1]]
        assert np.all(np.diff(c) > 0)


# ---------------------------------------------------------------- golden

def test_hand_4x4(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "hand_4x4.json")))
    mk = lambda d: CSR(d["nrows"], d["ncols"], np.array(d["rp"], np.int32),
                       np.array(d["col"], np.int32), np.array(d["val"], np.float32))
    A, B = mk(g["A"]), mk(g["B"])
    C = oracle.spgemm(A, B)
    assert C.rp.tolist() == g["C"]["rp"]
    assert C.col.tolist() == g["C"]["col"]
    assert C.val.tolist() == g["C"]["val"]          # exact: small integers/halves
    assert oracle.products(A, B).tolist() == g["P_rows"]
    assert C.products == sum(g["P_rows"])
    # the cancelled entry (3, 1) is stored with value 0
    assert C.col[C.rp[3]] == 1 and C.val[C.rp[3]] == 0.0


# ------------------------------------------------------------ dense pins

@pytest.mark.parametrize("density", [0.0, 0.05, 0.3, 1.0])
@pytest.mark.parametrize("seed", range(6))
def test_dense_integer_products(density, seed):
    """Integer values in [-4, 4]: every product and partial sum is exact in
    fp32, so values must equal the dense product bit for bit; the structure
    must equal the boolean product of the patterns (not the nonzero pattern
    of the numeric result)."""
    rng = np.random.default_rng(seed)
    m, K, N = rng.integers(1, 33, size=3)
    A = workloads.random_csr(rng, m, K, density, values="int")
    B = workloads.random_csr(rng, K, N, max(density, 0.1), values="int")
    C = oracle.spgemm(A, B)
    check_canonical(C)
    Da = np.zeros((m, K)); Db = np.zeros((K, N))
    Sa, Sb = pattern_dense(A), pattern_dense(B)
    Da[Sa] = A.val; Db[Sb] = B.val      # nonzero() order == CSR order
    Dc, Sc = to_dense(C, m)
    assert np.array_equal(Sc, (Sa.astype(np.int64) @ Sb.astype(np.int64)) > 0)
    assert np.array_equal(Dc, Da @ Db)


def test_stored_zero_inputs_keep_structure():
    """A stored 0.0 in A still contributes its B row to the structure."""
    A = from_dense([[0.0, 1.0]], pattern=[[True, True]])
    B = from_dense([[2.0, 0.0, 0.0], [0.0, 0.0, 3.0]])
    C = oracle.spgemm(A, B)
    assert C.col.tolist() == [0, 2]
    assert C.val.tolist() == [0.0, 3.0]


def test_brute_force_structure():
    """Tiny random patterns: enumerate every (i, k, j) triple directly."""
    rng = np.random.default_rng(7)
    for _ in range(200):
        m, K, N = rng.integers(1, 7, size=3)
        A = workloads.random_csr(rng, m, K, rng.random())
        B = workloads.random_csr(rng, K, N, rng.random())
        Sa, Sb = pattern_dense(A), pattern_dense(B)
        want = [sorted({j for k in range(K) if Sa[i, k] for j in range(N) if Sb[k, j]})
                for i in range(m)]
        C = oracle.spgemm(A, B)
        got = [C.col[C.rp[i]:C.rp[i + 1]].tolist() for i in range(m)]
        assert got == want
        P = oracle.products(A, B)
        assert P.tolist() == [sum(int(Sb[k].sum()) for k in range(K) if Sa[i, k]) for i in range(m)]


def test_scipy_cross_check():
    """Independent library product on continuous random data (no exact
    cancellations, so scipy's pruning of zero sums does not arise)."""
    sp = pytest.importorskip("scipy.sparse")
    rng = np.random.default_rng(11)
    A = workloads.random_csr(rng, 150, 120, 0.05)
    B = workloads.random_csr(rng, 120, 90, 0.08)
    C = oracle.spgemm(A, B)
    SA = sp.csr_matrix((A.val, A.col, A.rp), shape=(150, 120))
    SB = sp.csr_matrix((B.val, B.col, B.rp), shape=(120, 90))
    SC = (SA.astype(np.float64) @ SB.astype(np.float64)).tocsr()
    SC.sort_indices()
    assert np.array_equal(SC.indptr, C.rp)
    assert np.array_equal(SC.indices, C.col)
    np.testing.assert_allclose(C.val, SC.data, rtol=1e-5, atol=1e-6)


def test_fp64_error_bound():
    """|c32 - c64| <= gamma_n * sum|a b| with n = |A_i| (the standard bound
    for a sum of n rounded products; c64 is exact up to 2^-53 here since
    products of binary32 values are exact in binary64)."""
    A, B = workloads.workload(1)
    C = oracle.spgemm(A, B, f64=True)
    u = 2.0 ** -24
    n = np.repeat(A.row_lengths(), np.diff(C.rp)).astype(np.float64)
    gamma = n * u / (1 - n * u)
    err = np.abs(C.val.astype(np.float64) - C.val64)
    assert np.all(err <= gamma * C.abs64 + 1e-300)
    assert np.all(np.abs(C.val64) <= C.abs64 * (1 + 1e-12))


# --------------------------------------------------------- closed forms

def _sym_graph(n, edges):
    """Normalised A+I of an undirected graph given as an edge list, with
    values computed independently in numpy (1/sqrt(d_i d_j), fp64 -> fp32)."""
    S = np.eye(n, dtype=bool)
    for u, v in edges:
        S[u, v] = S[v, u] = True
    d = S.sum(1).astype(np.float64)
    V = np.where(S, 1.0 / np.sqrt(np.outer(d, d)), 0.0).astype(np.float32)
    return from_dense(V, pattern=S)


def test_edgeless_graph_is_identity():
    rng = np.random.default_rng(3)
    X = workloads.random_csr(rng, 64, 40, 0.2)
    A = _sym_graph(64, [])
    C = oracle.spgemm(A, X)
    assert np.array_equal(C.rp, X.rp.astype(np.int64))
    assert np.array_equal(C.col, X.col)
    assert np.array_equal(C.val.view(np.uint32), X.val.view(np.uint32))


@pytest.mark.parametrize("n", [2, 4, 8, 16])
def test_complete_graph_averages(n):
    """K_n with self-loops: every degree is n, so A_norm = J/n exactly when n
    is a power of two, and every row of C is (1/n) * sum_k X_k (exact for
    small integer X)."""
    A = _sym_graph(n, [(u, v) for u in range(n) for v in range(u + 1, n)])
    assert np.all(A.val == np.float32(1.0 / n))
    rng = np.random.default_rng(n)
    X = workloads.random_csr(rng, n, 12, 0.4, values="int")
    C = oracle.spgemm(A, X)
    Dx = np.zeros((n, 12)); Dx[pattern_dense(X)] = X.val
    want = Dx.sum(0) / n
    Dc, Sc = to_dense(C, n)
    col_any = pattern_dense(X).any(0)
    for i in range(n):
        assert np.array_equal(Sc[i], col_any)
        assert np.array_equal(Dc[i], np.where(col_any, want, 0.0))


def test_cycle_values_are_one_third():
    n = 9
    A = _sym_graph(n, [(i, (i + 1) % n) for i in range(n)])
    assert np.all(A.row_lengths() == 3)
    assert np.all(A.val == np.float32(1.0 / 3.0))
    # C = A * I equals A bitwise
    C = oracle.spgemm(A, from_dense(np.eye(n)))
    assert np.array_equal(C.val.view(np.uint32), A.val.view(np.uint32))


def test_identities_and_permutations():
    rng = np.random.default_rng(5)
    M = workloads.random_csr(rng, 30, 30, 0.2)
    I = from_dense(np.eye(30))
    for C in (oracle.spgemm(I, M), oracle.spgemm(M, I)):
        assert np.array_equal(C.col, M.col)
        assert np.array_equal(C.val.view(np.uint32), M.val.view(np.uint32))
    perm = rng.permutation(30)
    Pm = from_dense(np.eye(30)[perm])          # row i of Pm*M is row perm[i] of M
    C = oracle.spgemm(Pm, M)
    for i in range(30):
        s = slice(M.rp[perm[i]], M.rp[perm[i] + 1])
        assert np.array_equal(C.col[C.rp[i]:C.rp[i + 1]], M.col[s])
        assert np.array_equal(C.val[C.rp[i]:C.rp[i + 1]].view(np.uint32),
                              M.val[s].view(np.uint32))


# ------------------------------------------------------------ invariants

@pytest.fixture(scope="module")
def cfg1():
    A, B = workloads.workload(1)
    return A, B, oracle.spgemm(A, B)


def test_bounds_and_canonical(cfg1):
    A, B, C = cfg1
    assert oracle.validate(CSR(A.nrows, B.ncols, C.rp, C.col, C.val)) == 0
    P = oracle.products(A, B)
    nnz_row = np.diff(C.rp)
    assert np.all(nnz_row <= np.minimum(P, B.ncols))
    assert C.nnz <= P.sum() and C.products == P.sum()


def test_isolated_rows_copy_features(cfg1):
    """A row whose only entry is its self-loop (degree 1, value 1.0)
    reproduces the feature row bitwise."""
    A, B, C = cfg1
    iso = np.nonzero(A.row_lengths() == 1)[0]
    assert len(iso) > 100
    for i in iso[:200]:
        assert A.col[A.rp[i]] == i and A.val[A.rp[i]] == 1.0
        s = slice(B.rp[i], B.rp[i + 1])
        assert np.array_equal(C.col[C.rp[i]:C.rp[i + 1]], B.col[s])
        assert np.array_equal(C.val[C.rp[i]:C.rp[i + 1]].view(np.uint32), B.val[s].view(np.uint32))


def test_tiled_equals_untiled(cfg1):
    A, B, C = cfg1
    rng = np.random.default_rng(1)
    for _ in range(5):
        cuts = np.sort(rng.choice(np.arange(1, A.nrows), size=rng.integers(1, 12), replace=False))
        bounds = [0, *cuts.tolist(), A.nrows]
        parts = [oracle.spgemm(A, B, r0, r1) for r0, r1 in zip(bounds[:-1], bounds[1:])]
        T = oracle.concat(parts)
        assert np.array_equal(T.rp, C.rp) and np.array_equal(T.col, C.col)
        assert np.array_equal(T.val.view(np.uint32), C.val.view(np.uint32))


def test_square_of_symmetric_is_symmetric():
    """A*A of a symmetric A: entry (i, j) and (j, i) sum the same terms
    a_ik a_kj = a_jk a_ki in the same ascending-k order -> bitwise equal."""
    A = workloads.rmat_sym(2048, 8, seed=21)
    C = oracle.spgemm(A, A)
    D = np.zeros((2048, 2048), dtype=np.float32)
    S = np.zeros((2048, 2048), dtype=bool)
    rows = np.repeat(np.arange(2048), np.diff(C.rp))
    D[rows, C.col] = C.val
    S[rows, C.col] = True
    assert np.array_equal(S, S.T)
    assert np.array_equal(D.view(np.uint32), D.T.view(np.uint32))


def test_power_of_two_scaling(cfg1):
    A, B, C = cfg1
    A4 = CSR(A.nrows, A.ncols, A.rp, A.col, (A.val * np.float32(4)).astype(np.float32))
    B8 = CSR(B.nrows, B.ncols, B.rp, B.col, (B.val / np.float32(8)).astype(np.float32))
    C2 = oracle.spgemm(A4, B8)
    assert np.array_equal(C2.col, C.col)
    assert np.array_equal(C2.val, (C.val * np.float32(0.5)).astype(np.float32))


def test_rp64_inputs_match_rp32(cfg1):
    A, B, C = cfg1
    A64 = CSR(A.nrows, A.ncols, A.rp.astype(np.int64), A.col, A.val)
    C2 = oracle.spgemm(A64, B)
    assert np.array_equal(C2.val.view(np.uint32), C.val.view(np.uint32))


def test_empty_operands():
    A = CSR(5, 4, np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    B = workloads.random_csr(np.random.default_rng(0), 4, 7, 0.5)
    C = oracle.spgemm(A, B)
    assert C.nnz == 0 and C.rp.tolist() == [0] * 6
    C = oracle.spgemm(B, CSR(7, 3, np.zeros(8, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32)))
    assert C.nnz == 0


def test_validate_codes():
    ok = CSR(2, 3, np.array([0, 1, 2]), np.array([0, 2], np.int32), np.ones(2, np.float32))
    assert oracle.validate(ok) == 0
    assert oracle.validate(CSR(2, 3, np.array([1, 1, 2]), ok.col, ok.val)) == 1
    assert oracle.validate(CSR(2, 3, np.array([0, 2, 1]), ok.col, ok.val)) == 2
    assert oracle.validate(CSR(2, 3, np.array([0, 1, 3]), ok.col, ok.val)) == 3
    assert oracle.validate(CSR(2, 3, ok.rp, np.array([0, 3], np.int32), ok.val)) == 4
    assert oracle.validate(CSR(1, 3, np.array([0, 2]), np.array([2, 1], np.int32), ok.val)) == 5


# ---------------------------------------------------------------- RoBW

def test_robw_hand(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "robw_hand.json")))
    rp = np.array(g["rp"])
    for case in g["cases"]:
        if case["tiles"] is None:
            with pytest.raises(oracle.BudgetError):
                oracle.robw(rp, g["rp_bytes"], case["M_A"])
        else:
            assert [list(t) for t in oracle.robw(rp, g["rp_bytes"], case["M_A"])] == case["tiles"]


def _calc_mem(rp, r0, r1, s):
    return (r1 - r0 + 1) * s + 8 * int(rp[r1] - rp[r0])


@pytest.mark.parametrize("seed", range(20))
def test_robw_partition_fit_maximal(seed):
    """The greedy partition is the unique one whose blocks partition the
    rows, each fit M_A, and each (but the last) would overflow with its next
    row -- so these three properties pin it completely."""
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 300))
    lens = rng.integers(0, 50, size=m) * (rng.random(m) < 0.9)
    rp = np.concatenate([[0], np.cumsum(lens)])
    s = int(rng.choice([4, 8]))
    M_A = int(_calc_mem(rp, 0, 1, s) + rng.integers(0, 2000)) if m else 100
    need = max(_calc_mem(rp, i, i + 1, s) for i in range(m))
    if need > M_A:
        with pytest.raises(oracle.BudgetError):
            oracle.robw(rp, s, M_A)
        return
    tiles = oracle.robw(rp, s, M_A)
    assert tiles[0][0] == 0 and tiles[-1][1] == m
    for (a, b), (c, _) in zip(tiles[:-1], tiles[1:]):
        assert b == c
    for a, b in tiles:
        assert b > a and _calc_mem(rp, a, b, s) <= M_A
    for a, b in tiles[:-1]:
        assert _calc_mem(rp, a, b + 1, s) > M_A


# ------------------------------------------------------------ generator

def test_generator_properties():
    A = workloads.rmat_sym(4096, 16, seed=1)
    assert oracle.validate(A) == 0
    S = pattern_dense(A)
    assert np.array_equal(S, S.T) and np.all(np.diag(S))
    d = A.row_lengths().astype(np.float64)
    rows = np.repeat(np.arange(4096), A.row_lengths())
    want = (1.0 / np.sqrt(d[rows] * d[A.col])).astype(np.float32)
    assert np.array_equal(A.val, want)
    A2 = workloads.rmat_sym(4096, 16, seed=1)
    assert np.array_equal(A.col, A2.col) and np.array_equal(A.val, A2.val)
    assert not np.array_equal(workloads.rmat_sym(4096, 16, seed=2).rp, A.rp)
    X = workloads.features(4096, 256, 0.1, seed=1001)
    assert oracle.validate(X) == 0
    assert abs(X.nnz / (4096 * 256) - 0.1) < 0.005
    assert X.val.min() >= -1.0 and X.val.max() <= 1.0


# --------------------------------------- combination step (Eq. 3): A * W

def test_spmm_identity_and_relu():
    """A = I: Y = W exactly; with the activation, Y = max(W, 0)."""
    rng = np.random.default_rng(11)
    W = rng.standard_normal((37, 19)).astype(np.float32)
    I = from_dense(np.eye(37))
    Y, Ya = oracle.spmm(I, W)
    assert np.array_equal(Y, W.astype(np.float64))
    assert np.array_equal(Ya, np.abs(W).astype(np.float64))
    Yr, _ = oracle.spmm(I, W, relu=True)
    assert np.array_equal(Yr, np.maximum(W, 0).astype(np.float64))


@pytest.mark.parametrize("density", [0.0, 0.05, 0.3, 1.0])
def test_spmm_integer_matches_integer_matmul(density):
    """Small integers: every product and partial sum is exact in double, so
    Y equals the exact integer product of the dense operands."""
    rng = np.random.default_rng(int(density * 100) + 3)
    Ad = rng.integers(-4, 5, (23, 31)) * (rng.random((23, 31)) < density)
    W = rng.integers(-4, 5, (31, 45))
    A = from_dense(Ad.astype(np.float32), pattern=(Ad != 0))
    Y, Ya = oracle.spmm(A, W.astype(np.float32))
    assert np.array_equal(Y, (Ad.astype(np.int64) @ W.astype(np.int64)).astype(np.float64))
    assert np.array_equal(Ya, (np.abs(Ad).astype(np.int64) @ np.abs(W).astype(np.int64)).astype(np.float64))
    Yr, _ = oracle.spmm(A, W.astype(np.float32), relu=True)
    assert np.all(Yr >= 0) and np.array_equal(Yr, np.maximum(Y, 0))


def test_spmm_permutation_empty_rows_and_average():
    rng = np.random.default_rng(12)
    W = rng.standard_normal((16, 9)).astype(np.float32)
    perm = rng.permutation(16)
    Y, _ = oracle.spmm(from_dense(np.eye(16)[perm]), W)           # row i = W[perm[i]]
    assert np.array_equal(Y, W[perm].astype(np.float64))
    E = CSR(5, 16, np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    Y, Ya = oracle.spmm(E, W, relu=True)                           # empty rows: act(0) = 0
    assert np.array_equal(Y, np.zeros((5, 9))) and np.array_equal(Ya, np.zeros((5, 9)))
    # K_16 with self-loops: A_norm = J/16 exactly, so every row is the mean of W's rows
    A = _sym_graph(16, [(u, v) for u in range(16) for v in range(u + 1, 16)])
    Wi = rng.integers(-8, 9, (16, 9)).astype(np.float32)
    Y, _ = oracle.spmm(A, Wi)
    assert np.array_equal(Y, np.tile(Wi.astype(np.float64).sum(0) / 16, (16, 1)))


def test_spmm_brute_force_triples():
    """Tiny random inputs: the sum over stored (i, k) entries of a_ik w_kj
    enumerated directly."""
    rng = np.random.default_rng(13)
    for trial in range(20):
        m, K, F = rng.integers(1, 7, 3)
        Ad = rng.standard_normal((m, K)) * (rng.random((m, K)) < 0.5)
        A = from_dense(Ad.astype(np.float32), pattern=(Ad != 0))
        W = rng.standard_normal((K, F)).astype(np.float32)
        want = np.zeros((m, F))
        rp = A.rp.astype(np.int64)
        for i in range(m):
            for p in range(rp[i], rp[i + 1]):
                for j in range(F):
                    want[i, j] += float(A.val[p]) * float(W[A.col[p], j])
        Y, _ = oracle.spmm(A, W)
        assert np.allclose(Y, want, rtol=0, atol=1e-12)


def test_spmm_gcn_layer_composes():
    """A GCN layer H' = relu((A_norm X) W) from the two oracle products
    equals relu(A_norm (X W)) up to double rounding (associativity)."""
    rng = np.random.default_rng(14)
    A = _sym_graph(40, [tuple(e) for e in rng.integers(0, 40, (60, 2)) if e[0] != e[1]])
    X = workloads.random_csr(rng, 40, 24, 0.3)
    W = rng.standard_normal((24, 8)).astype(np.float32)
    C = oracle.spgemm(A, X, f64=True)
    Cd = CSR(40, 24, C.rp, C.col, C.val)
    H1, _ = oracle.spmm(Cd, W, relu=True)
    Dx = np.zeros((40, 24)); Dx[pattern_dense(X)] = X.val
    Da = np.zeros((40, 40)); Da[pattern_dense(A)] = A.val
    H2 = np.maximum(Da @ (Dx @ W.astype(np.float64)), 0)
    assert np.allclose(H1, H2, rtol=1e-5, atol=1e-6)


def test_sym_norm_closed_forms():
    """Eq. 2 from a pattern with its self-loops (oracle.sym_norm), against
    values worked by hand: the complete graph on 8 vertices gives 1/8
    everywhere (exact); a 6-cycle, three entries per row, gives fl32(1/3) =
    0.333333343...; a star with 3 leaves gives 1/4 at the centre's loop,
    1/sqrt(8) = 0.353553385... on its edges and 1/2 at the leaves' loops; an
    isolated vertex (its loop alone) gives 1.  Then the generator's own
    values for the tiny workload's graph, computed there independently."""
    n = 8
    v = oracle.sym_norm(np.arange(0, n * n + 1, n), np.tile(np.arange(n), n))
    assert np.all(v == np.float32(0.125))
    cyc = [sorted({(i - 1) % 6, i, (i + 1) % 6}) for i in range(6)]
    v = oracle.sym_norm(np.arange(0, 19, 3), np.array(sum(cyc, []), np.int32))
    assert np.all(v.view(np.uint32) == np.uint32(0x3EAAAAAB))
    star_rp = np.array([0, 4, 6, 8, 10, 11])
    star_col = np.array([0, 1, 2, 3, 0, 1, 0, 2, 0, 3, 4], np.int32)
    e = np.float32(0.35355338)
    want = np.array([0.25, e, e, e, e, 0.5, e, 0.5, e, 0.5, 1.0], np.float32)
    assert np.array_equal(oracle.sym_norm(star_rp, star_col), want)
    A, _ = workloads.workload(1)
    assert np.array_equal(oracle.sym_norm(A.rp, A.col).view(np.uint32), A.val.view(np.uint32))
