"""The whole-matrix verifier used at full size (CPU): it accepts the
oracle's own product computed in different row blocks, and rejects a C with
a planted mistake in its row pointers, a column, or a value just outside
the bar."""
import numpy as np
import pytest

import fullcheck
import oracle
import workloads


def _fetch(ref):
    return lambda s, e: (ref.col[s:e].copy(), ref.val[s:e].copy())


@pytest.fixture(scope="module")
def case():
    A, B = workloads.workload(3, n=3000)
    ref = oracle.concat([oracle.spgemm(A, B, r0, r1) for r0, r1 in ((0, 1234), (1234, 2999), (2999, 3000))])
    return A, B, ref


def test_chunks_cover_rows():
    rp = np.array([0, 5, 5, 100, 101, 101, 300], np.int64)
    for t in (1, 3, 50, 1000):
        ch = fullcheck.chunks(rp, t)
        assert ch[0][0] == 0 and ch[-1][1] == 6
        assert all(a[1] == b[0] for a, b in zip(ch, ch[1:]))
        assert all(r1 > r0 for r0, r1 in ch)


def test_accepts_the_oracle(case):
    A, B, ref = case
    res = fullcheck.verify(A, B, ref.rp, _fetch(ref), target_entries=4000, threads=4)
    assert res["nnz"] == ref.nnz and res["products"] == ref.products and res["chunks"] > 10
    assert res["max_rel_err"] == 0.0


def test_rejects_planted_mistakes(case):
    A, B, ref = case
    i = ref.nnz // 2
    rp = ref.rp.copy()
    row = int(np.searchsorted(rp, i, side="right")) - 1
    rp[row + 1] += 1  # one entry moved to the next row
    with pytest.raises(AssertionError, match="row_ptr"):
        fullcheck.verify(A, B, rp, _fetch(ref), target_entries=4000, threads=4)
    col = ref.col.copy()
    col[i] += 1
    with pytest.raises(AssertionError, match="col_idx"):
        fullcheck.verify(A, B, ref.rp, lambda s, e: (col[s:e], ref.val[s:e]), target_entries=4000, threads=4)
    val = ref.val.astype(np.float64)
    val[i] += 1.5e-5 * (1 + abs(val[i]))
    val = val.astype(np.float32)
    with pytest.raises(AssertionError, match="value at entry %d" % i):
        fullcheck.verify(A, B, ref.rp, lambda s, e: (ref.col[s:e], val[s:e]), target_entries=4000, threads=4)
    # within the bar: accepted
    ok = (ref.val.astype(np.float64) * (1 + 2e-6)).astype(np.float32)
    fullcheck.verify(A, B, ref.rp, lambda s, e: (ref.col[s:e], ok[s:e]), target_entries=4000, threads=4)
