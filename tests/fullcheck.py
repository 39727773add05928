"""Whole-matrix verification of a product C = A * B against the oracle, in
row chunks spread over host threads (test infrastructure).

Every row of C is checked: the rows are cut into chunks of about
`target_entries` entries of C (by C's own row pointers); for each chunk
the oracle computes the same rows (Gustavson, Eq. 1) and the chunk's
entries of C are fetched from wherever C lives.  Row pointers (rebased to
the chunk) and column indices must be identical; every value must satisfy
|c - ref| <= tol * (1 + |ref|).  The oracle runs outside the GIL (a plain C
call through ctypes), so the chunks proceed in parallel.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
from workloads import CSR


def host_threads(limit: int = 16) -> int:
    """Threads for the oracle: this process's CPUs, at most `limit`."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(limit, n))


def _wide_rp(M) -> CSR:
    """The same matrix with int64 row pointers (the oracle's width), so that
    no oracle call converts them again."""
    if M.rp.dtype == np.int64:
        return M
    return CSR(M.nrows, M.ncols, M.rp.astype(np.int64), M.col, M.val)


def chunks(c_rp: np.ndarray, target_entries: int, max_rows: int = 1 << 22):
    """Consecutive row ranges [r0, r1) covering all rows, each with about
    target_entries entries of C (a single longer row is a chunk of its own)
    and at most max_rows rows."""
    m = len(c_rp) - 1
    out = []
    r0 = 0
    while r0 < m:
        want = c_rp[r0] + target_entries
        r1 = int(np.searchsorted(c_rp, want, side="right")) - 1
        r1 = max(r0 + 1, min(r1, m, r0 + max_rows))
        out.append((r0, r1))
        r0 = r1
    return out


def verify(A, B, c_rp: np.ndarray, fetch, tol: float = 1e-5, target_entries: int = 1 << 25,
           threads: int | None = None, say=None) -> dict:
    """Check every row of C.  `c_rp` is C's int64 row-pointer array (host);
    fetch(s, e) returns (col, val) numpy arrays of C's entries [s, e).
    Returns counts; raises AssertionError naming the first bad chunk."""
    A64, B64 = _wide_rp(A), _wide_rp(B)
    c_rp = np.asarray(c_rp)
    assert c_rp.dtype == np.int64 and len(c_rp) == A.nrows + 1
    assert c_rp[0] == 0, "C.row_ptr[0] = %d" % c_rp[0]
    parts = chunks(c_rp, target_entries)
    threads = threads or host_threads()

    def one(rg):
        r0, r1 = rg
        ref = oracle.spgemm(A64, B64, r0, r1)
        rp = c_rp[r0:r1 + 1] - c_rp[r0]
        if not np.array_equal(rp, ref.rp):
            bad = int(np.argmax(rp != ref.rp))
            return "rows [%d, %d): row_ptr differs first at row %d" % (r0, r1, r0 + max(bad - 1, 0)), 0, 0
        s, e = int(c_rp[r0]), int(c_rp[r1])
        col, val = fetch(s, e)
        if not np.array_equal(col, ref.col):
            bad = int(np.argmax(col != ref.col))
            row = r0 + int(np.searchsorted(ref.rp, bad, side="right")) - 1
            return "rows [%d, %d): col_idx differs at entry %d (row %d)" % (r0, r1, s + bad, row), 0, 0
        step = 1 << 22
        worst = 0.0
        for q in range(0, e - s, step):
            v = val[q:q + step].astype(np.float64)
            r = ref.val[q:q + step].astype(np.float64)
            err = np.abs(v - r)
            lim = tol * (1.0 + np.abs(r))
            if not np.all(err <= lim):
                bad = q + int(np.argmax(err > lim))
                row = r0 + int(np.searchsorted(ref.rp, bad, side="right")) - 1
                return ("rows [%d, %d): value at entry %d (row %d, col %d): %r vs oracle %r"
                        % (r0, r1, s + bad, row, int(ref.col[bad]), float(val[bad]), float(ref.val[bad]))), 0, 0
            if len(err):
                worst = max(worst, float((err / (1.0 + np.abs(r))).max()))
        return None, ref.products, worst

    products = 0
    worst = 0.0
    with ThreadPoolExecutor(threads) as ex:
        for i, (msg, p, w) in enumerate(ex.map(one, parts)):
            assert msg is None, msg
            products += p
            worst = max(worst, w)
            if say and (i + 1) % max(1, len(parts) // 8) == 0:
                say("verified %d of %d chunks" % (i + 1, len(parts)))
    return {"rows": A.nrows, "nnz": int(c_rp[-1]), "chunks": len(parts), "products": products,
            "threads": threads, "max_rel_err": worst}


def device_fetch(C):
    """fetch(s, e) for a C whose col/val are device torch tensors."""
    def f(s, e):
        return C.col[s:e].cpu().numpy(), C.val[s:e].cpu().numpy()
    return f


def host_fetch(C):
    """fetch(s, e) for a C in (pinned) host memory as numpy arrays."""
    def f(s, e):
        return C.col[s:e], C.val[s:e]
    return f
