"""Seeded synthetic inputs shared by the oracle tests and the GPU path.

This package builds inputs only; it holds none of the sparse-product
arithmetic.  The arrays it returns are plain numpy CSR triples.

Workloads follow the GCN aggregation setting of the paper (Sec. II-A,
Eqs. 1-2): a symmetric R-MAT graph with self-loops whose stored values are
1/sqrt(d_i d_j) (the D^-1/2 (A+I) D^-1/2 normalisation), times a sparse
feature matrix with uniformly random positions and U[-1, 1) values.  The
paper's SuiteSparse graphs are not used; these power-law graphs stand in
for them.
"""
from __future__ import annotations

import ctypes
import os
import sys
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libgen.so")

RMAT_ABCD = (0.57, 0.19, 0.19, 0.05)


def build(force: bool = True) -> str:
    """Compile the generator with gcc (OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        i64, u64, dbl, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
        lib.rmat_build.restype = vp
        lib.rmat_build.argtypes = [i64, dbl, dbl, dbl, dbl, u64, ctypes.c_int]
        for f in ("rmat_nnz", "rmat_samples", "rmat_self_samples"):
            getattr(lib, f).restype = i64
            getattr(lib, f).argtypes = [vp]
        lib.rmat_export.restype = None
        lib.rmat_export.argtypes = [vp, vp, ctypes.c_int, vp, vp]
        lib.rmat_free.restype = None
        lib.rmat_free.argtypes = [vp]
        lib.feat_count.restype = i64
        lib.feat_count.argtypes = [i64, i64, dbl, u64, vp]
        lib.feat_fill.restype = None
        lib.feat_fill.argtypes = [i64, i64, dbl, u64, vp, vp, vp]
        _lib = lib
    return _lib


@dataclass
class CSR:
    """A CSR matrix held as numpy arrays (row_ptr int32 or int64)."""
    nrows: int
    ncols: int
    rp: np.ndarray
    col: np.ndarray
    val: np.ndarray

    @property
    def nnz(self) -> int:
        return int(self.rp[-1]) if len(self.rp) else 0

    def row_lengths(self) -> np.ndarray:
        return np.diff(self.rp.astype(np.int64))

    def nbytes(self) -> int:
        return self.rp.nbytes + self.col.nbytes + self.val.nbytes


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def rmat_sym(n: int, avg_deg: float, seed: int, rp64: bool = False,
             abcd=RMAT_ABCD, out=None, verbose: bool = False) -> CSR:
    """Symmetric R-MAT graph, self-loops added, values 1/sqrt(d_i d_j) in fp32.

    ``out`` may supply preallocated (rp, col, val) buffers (e.g. pinned host
    memory viewed as numpy) of the right sizes; otherwise numpy allocates.
    ``verbose`` prints a line to stderr as each generation stage ends.
    """
    lib = _load()
    a, b, c, _ = abcd
    h = lib.rmat_build(int(n), float(avg_deg), a, b, c, int(seed), int(bool(verbose)))
    if not h:
        raise MemoryError("rmat_build failed for n=%d" % n)
    try:
        nnz = int(lib.rmat_nnz(h))
        if not rp64 and nnz >= 2**31:
            raise OverflowError("nnz %d needs int64 row_ptr" % nnz)
        if out is None:
            rp = np.empty(n + 1, dtype=np.int64 if rp64 else np.int32)
            col = np.empty(max(nnz, 1), dtype=np.int32)[:nnz]
            val = np.empty(max(nnz, 1), dtype=np.float32)[:nnz]
        else:
            rp, col, val = out(nnz)
        lib.rmat_export(h, _ptr(rp), 1 if rp64 else 0, _ptr(col), _ptr(val))
    finally:
        lib.rmat_free(h)
    return CSR(n, n, rp, col, val)


def features(n: int, F: int, rho: float, seed: int, rp64: bool = False, out=None,
             verbose: bool = False) -> CSR:
    """n x F sparse features: each entry present w.p. rho, value U[-1, 1) as fp32."""
    lib = _load()
    lens = np.empty(n, dtype=np.int64)
    nnz = int(lib.feat_count(int(n), int(F), float(rho), int(seed), _ptr(lens)))
    if verbose:
        print("[gen] features %dx%d counted: nnz %d" % (n, F, nnz), file=sys.stderr, flush=True)
    rp64_tmp = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lens, out=rp64_tmp[1:])
    if out is None:
        col = np.empty(max(nnz, 1), dtype=np.int32)[:nnz]
        val = np.empty(max(nnz, 1), dtype=np.float32)[:nnz]
        rp = rp64_tmp if rp64 else rp64_tmp.astype(np.int32)
    else:
        rp, col, val = out(nnz)
        rp[:] = rp64_tmp if rp64 else rp64_tmp.astype(np.int32)
    lib.feat_fill(int(n), int(F), float(rho), int(seed), _ptr(rp64_tmp), _ptr(col), _ptr(val))
    return CSR(n, F, rp, col, val)


# The five aggregation workloads.  Each is (graph n, target degree D,
# feature width F or None for the square product A*A, density rho,
# row_ptr width of A).
CONFIGS = {
    1: dict(name="tiny-gcn-agg", n=4096, deg=16, F=256, rho=0.10, rp64=False),
    2: dict(name="mid-gcn-agg", n=262144, deg=32, F=512, rho=0.05, rp64=False),
    3: dict(name="two-hop-square", n=1048576, deg=16, F=None, rho=None, rp64=False),
    4: dict(name="large-gcn-agg", n=8388608, deg=24, F=128, rho=0.10, rp64=False),
    5: dict(name="out-of-core-gcn-agg", n=68000000, deg=22, F=64, rho=0.10, rp64=True),
}


def workload(cfg: int, n: int | None = None, out_a=None, out_b=None, verbose: bool = False):
    """Return (A, B) for workload ``cfg``; ``n`` overrides the node count
    (same degree, width and density) for scaled-down parity cases."""
    c = CONFIGS[cfg]
    nn = c["n"] if n is None else int(n)
    A = rmat_sym(nn, c["deg"], seed=cfg, rp64=c["rp64"], out=out_a, verbose=verbose)
    if c["F"] is None:
        return A, A
    B = features(nn, c["F"], c["rho"], seed=1000 + cfg, out=out_b, verbose=verbose)
    return A, B


def random_csr(rng: np.random.Generator, m: int, n: int, density: float,
               values: str = "uniform", rp64: bool = False) -> CSR:
    """Small random CSR with sorted unique columns, for unit tests.

    values: "uniform" U[-1,1) fp32, "int" integers in [-4, 4] (exact in
    fp32 for small products), "ones".
    """
    mask = rng.random((m, n)) < density
    rows, cols = np.nonzero(mask)
    if values == "int":
        v = rng.integers(-4, 5, size=len(rows)).astype(np.float32)
    elif values == "ones":
        v = np.ones(len(rows), dtype=np.float32)
    else:
        v = rng.uniform(-1, 1, size=len(rows)).astype(np.float32)
    rp = np.zeros(m + 1, dtype=np.int64)
    np.add.at(rp, rows + 1, 1)
    rp = np.cumsum(rp)
    return CSR(m, n, rp if rp64 else rp.astype(np.int32), cols.astype(np.int32), v)


def write_csr_file(path: str, M: CSR, align: int = 4096) -> dict:
    """Write M's three CSR arrays as raw arrays into one file, each starting
    at a multiple of `align` bytes; returns the descriptor fields of
    aires_file_csr (path, sizes, row-pointer width, byte offsets)."""
    offs = {}
    pos = 0
    with open(path, "wb") as f:
        for name, arr in (("row_ptr_offset", M.rp), ("col_idx_offset", M.col), ("vals_offset", M.val)):
            pad = (-pos) % align
            if pad:
                f.write(b"\0" * pad)
                pos += pad
            offs[name] = pos
            a = np.ascontiguousarray(arr)
            f.write(memoryview(a).cast("B"))
            pos += a.nbytes
    return dict(path=path, nrows=M.nrows, ncols=M.ncols, nnz=M.nnz, rp_dtype=str(M.rp.dtype), **offs)

