"""ORACLE -- test infrastructure only (tests, the smoke check and the
benchmark's CPU-baseline leg).  The GPU library never imports it.

Python front end to ``oracle.c``: a serial CPU Gustavson sparse product
(Sec. II-A, Eq. 1, with both operands compressed), the per-row
intermediate-product counts, the sparse-times-dense combination product of
a GCN layer (Eq. 3, in double), the RoBW row-block partition of Algorithm 1
(Sec. III-A) and a canonical-CSR validator.  Matrices are any object with
``nrows, ncols, rp, col, val`` numpy attributes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# -ffp-contract=off: every product and every sum rounds to binary32 (no FMA).
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC"]


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        lib.oracle_spgemm.restype = vp
        lib.oracle_spgemm.argtypes = [i64, vp, vp, vp, vp, vp, vp, i64, i64, ci]
        lib.oracle_result_free.restype = None
        lib.oracle_result_free.argtypes = [vp]
        lib.oracle_result_nnz.restype = i64
        lib.oracle_result_nnz.argtypes = [vp]
        lib.oracle_result_products.restype = i64
        lib.oracle_result_products.argtypes = [vp]
        lib.oracle_result_export.restype = None
        lib.oracle_result_export.argtypes = [vp, vp, vp, vp, vp, vp]
        lib.oracle_products.restype = i64
        lib.oracle_products.argtypes = [vp, vp, vp, i64, i64, vp]
        lib.oracle_robw.restype = i64
        lib.oracle_robw.argtypes = [i64, vp, i64, i64, vp, i64]
        lib.oracle_validate.restype = ci
        lib.oracle_validate.argtypes = [i64, i64, i64, vp, vp]
        lib.oracle_spmm.restype = None
        lib.oracle_spmm.argtypes = [i64, vp, vp, vp, vp, i64, i64, ctypes.c_int, vp, vp]
        lib.oracle_sym_norm.restype = None
        lib.oracle_sym_norm.argtypes = [i64, vp, vp, vp]
        _lib = lib
    return _lib


def _rp64(rp: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(rp, dtype=np.int64)


def _c(a: np.ndarray, dt) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dt)


@dataclass
class Product:
    """Rows [r0, r1) of C: rp is int64 and starts at 0."""
    r0: int
    r1: int
    ncols: int
    rp: np.ndarray
    col: np.ndarray
    val: np.ndarray
    products: int
    val64: np.ndarray | None = None
    abs64: np.ndarray | None = None

    @property
    def nnz(self) -> int:
        return int(self.rp[-1])


def spgemm(A, B, r0: int = 0, r1: int | None = None, f64: bool = False) -> Product:
    """Rows [r0, r1) of C = A * B, in the fixed ascending-k fp32 order."""
    if A.ncols != B.nrows:
        raise ValueError("inner dimensions differ: %d vs %d" % (A.ncols, B.nrows))
    lib = _load()
    r1 = A.nrows if r1 is None else r1
    if not (0 <= r0 <= r1 <= A.nrows):
        raise ValueError("bad row range")
    arp, brp = _rp64(A.rp), _rp64(B.rp)
    acol, aval = _c(A.col, np.int32), _c(A.val, np.float32)
    bcol, bval = _c(B.col, np.int32), _c(B.val, np.float32)
    h = lib.oracle_spgemm(int(B.ncols), arp.ctypes.data, acol.ctypes.data, aval.ctypes.data,
                          brp.ctypes.data, bcol.ctypes.data, bval.ctypes.data,
                          int(r0), int(r1), 1 if f64 else 0)
    if not h:
        raise MemoryError("oracle_spgemm failed")
    try:
        nnz = int(lib.oracle_result_nnz(h))
        rp = np.empty(r1 - r0 + 1, dtype=np.int64)
        col = np.empty(nnz, dtype=np.int32)
        val = np.empty(nnz, dtype=np.float32)
        v64 = np.empty(nnz, dtype=np.float64) if f64 else None
        a64 = np.empty(nnz, dtype=np.float64) if f64 else None
        lib.oracle_result_export(h, rp.ctypes.data, col.ctypes.data, val.ctypes.data,
                                 v64.ctypes.data if f64 else None,
                                 a64.ctypes.data if f64 else None)
        prods = int(lib.oracle_result_products(h))
    finally:
        lib.oracle_result_free(h)
    return Product(r0, r1, B.ncols, rp, col, val, prods, v64, a64)


def spmm(A, W: np.ndarray, relu: bool = False) -> tuple[np.ndarray, np.ndarray]:
    """Y = act(A * W) in double (Sec. II-A, Eq. 3) and the sums of |a_ik w_kj|
    for each entry: A a CSR, W a float32 (A.ncols x F) array."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    if W.ndim != 2 or W.shape[0] != A.ncols:
        raise ValueError("W must be (A.ncols x F)")
    lib = _load()
    m, F = A.nrows, W.shape[1]
    arp, acol, aval = _rp64(A.rp), _c(A.col, np.int32), _c(A.val, np.float32)
    Y = np.empty((m, F), dtype=np.float64)
    Ya = np.empty((m, F), dtype=np.float64)
    if m and F:
        lib.oracle_spmm(int(m), arp.ctypes.data, acol.ctypes.data, aval.ctypes.data, W.ctypes.data, int(F), int(F),
                        1 if relu else 0, Y.ctypes.data, Ya.ctypes.data)
    return Y, Ya


def sym_norm(rp: np.ndarray, col: np.ndarray) -> np.ndarray:
    """The values of the normalised adjacency (Sec. II-A, Eq. 2) of a square
    pattern whose self-loops are stored: a_ij = 1/sqrt(r_i r_j), r_i the
    stored entries of row i, in double, rounded once to float32."""
    lib = _load()
    rp64, c = _rp64(rp), _c(col, np.int32)
    m = len(rp64) - 1
    out = np.empty(len(c), dtype=np.float32)
    if len(c):
        lib.oracle_sym_norm(int(m), rp64.ctypes.data, c.ctypes.data, out.ctypes.data)
    return out


def products(A, B, r0: int = 0, r1: int | None = None) -> np.ndarray:
    """P_i = sum over stored k of A_i of nnz(B_k), int64, for rows [r0, r1)."""
    lib = _load()
    r1 = A.nrows if r1 is None else r1
    arp, brp, acol = _rp64(A.rp), _rp64(B.rp), _c(A.col, np.int32)
    P = np.empty(r1 - r0, dtype=np.int64)
    lib.oracle_products(arp.ctypes.data, acol.ctypes.data, brp.ctypes.data,
                        int(r0), int(r1), P.ctypes.data)
    return P


class BudgetError(Exception):
    pass


def robw(rp: np.ndarray, rp_bytes: int, M_A: int) -> list[tuple[int, int]]:
    """Algorithm 1 row blocks [(r0, r1), ...] with calcMem(k,q)=(k+1)*rp_bytes+8q."""
    lib = _load()
    rp = _rp64(rp)
    m = len(rp) - 1
    starts = np.empty(max(m, 1), dtype=np.int64)
    n = int(lib.oracle_robw(m, rp.ctypes.data, int(rp_bytes), int(M_A), starts.ctypes.data,
                            len(starts)))
    if n == -1:
        raise BudgetError("a single row exceeds M_A=%d" % M_A)
    if n < 0:
        raise RuntimeError("oracle_robw failed: %d" % n)
    s = [int(x) for x in starts[:n]]
    return [(s[t], s[t + 1] if t + 1 < n else m) for t in range(n)]


def validate(M) -> int:
    """0 if M is canonical CSR, else the oracle's positive error code."""
    lib = _load()
    rp = _rp64(M.rp)
    col = _c(M.col, np.int32)
    if len(rp) != M.nrows + 1:
        return 3
    return int(lib.oracle_validate(int(M.nrows), int(M.ncols), int(len(col)),
                                   rp.ctypes.data, col.ctypes.data))


def concat(parts: list[Product]) -> Product:
    """Join consecutive row-range results (rp rebased by the running nnz)."""
    rp = [np.zeros(1, dtype=np.int64)]
    base = 0
    for p in parts:
        rp.append(p.rp[1:] + base)
        base += p.nnz
    return Product(parts[0].r0, parts[-1].r1, parts[0].ncols, np.concatenate(rp),
                   np.concatenate([p.col for p in parts]), np.concatenate([p.val for p in parts]),
                   sum(p.products for p in parts))
