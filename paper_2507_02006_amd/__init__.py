"""MI355X (gfx950) out-of-core CSR x CSR product for GCN aggregation, after
AIRES (arXiv 2507.02006): C = A * B over row block-wise (RoBW) tiles
(Sec. III-A, Algorithm 1) under a device budget, with B resident and A
tiles streamed from pinned host memory when they do not fit (Sec. III-B,
Algorithm 2).

Python names mirror the C-ABI of include/aires.h:
  tile_plan(A, B, hbm_budget, ...)  -> Plan       (aires_tile_plan)
  spgemm(plan, stream=None)         -> Output     (aires_spgemm)
  stream_tiles(plan, ...)           -> Output     (aires_stream_tiles)
  plan_info / plan_tile / plan_stats
A and B are (nrows, ncols, row_ptr, col_idx, vals) tuples or objects with
those attributes (``nrows, ncols, rp, col, val``); arrays are device torch
tensors, pinned host torch tensors, or numpy arrays (planning only).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

from . import _binding as B_

__all__ = ["tile_plan", "tile_plan_file", "read_csr_file", "spgemm", "spmm", "stream_tiles", "plan_info",
           "plan_tile", "plan_stats", "plan_tile_stats", "spgemm_noalloc", "Plan", "Output", "AiresError",
           "to_device", "to_pinned"]

AiresError = B_.AiresError


def _parts(M):
    if isinstance(M, tuple):
        return M
    return (M.nrows, M.ncols, M.rp, M.col, M.val)


class Plan:
    """An aires_plan plus references keeping its borrowed inputs alive."""

    def __init__(self, handle, A, B, allocator, opts):
        self.handle = handle
        self._inputs = (A, B)
        self.allocator = allocator
        self.opts = opts

    def close(self):
        if self.handle:
            B_.load().aires_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001 -- interpreter shutdown
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()


def _opts(lib, **kw):
    o = B_.PlanOpts()
    B_.check(lib.aires_plan_opts_default(ctypes.byref(o)), "aires_plan_opts_default")
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def tile_plan_file(A, B, hbm_budget: int = 0, *, c_on_host: bool = True, c_bound: int = B_.CBOUND_ROWS,
                   timing: bool = False, max_tile_bytes: int = 0, a_values: str = "given", direct_io: bool = True,
                   torch_allocator: bool = True, device: int = 0) -> Plan:
    """Plan C = A * B with A's arrays in a file (aires_tile_plan_file).  A is
    a dict with nrows, ncols, nnz, rp_dtype ("int32"/"int64"), path and the
    byte offsets row_ptr_offset, col_idx_offset, vals_offset (as written by
    ``workloads.write_csr_file``); B as for tile_plan.  The plan streams:
    each tile is read from the file into pinned staging, then sent."""
    lib = B_.load()
    path = A["path"].encode()
    fa = B_.FileCsr(int(A["nrows"]), int(A["ncols"]), int(A["nnz"]),
                    B_.IDX_I64 if A["rp_dtype"] == "int64" else B_.IDX_I32, int(bool(direct_io)), path,
                    int(A["row_ptr_offset"]), int(A["col_idx_offset"]), int(A["vals_offset"]))
    b = B_.make_csr(*_parts(B))
    if a_values not in ("given", "sym_norm"):
        raise ValueError("a_values must be 'given' or 'sym_norm'")
    o = _opts(lib, c_placement=B_.MEM_HOST_PINNED if c_on_host else B_.MEM_DEVICE, c_bound=c_bound,
              timing=int(timing), max_tile_bytes=max_tile_bytes,
              a_values=B_.AVALUES_SYM_NORM if a_values == "sym_norm" else B_.AVALUES_GIVEN)
    alloc = B_.TorchAllocator(device) if torch_allocator else None
    if alloc is not None:
        o.allocator = ctypes.pointer(alloc.struct)
    h = ctypes.c_void_p()
    B_.check(lib.aires_tile_plan_file(ctypes.byref(fa), ctypes.byref(b), int(hbm_budget), ctypes.byref(o),
                                      ctypes.byref(h)), "aires_tile_plan_file")
    return Plan(h.value, (fa, path), B, alloc, o)


def _file_csr(F) -> B_.FileCsr:
    return B_.FileCsr(int(F["nrows"]), int(F["ncols"]), int(F["nnz"]),
                      B_.IDX_I64 if F["rp_dtype"] == "int64" else B_.IDX_I32, int(bool(F.get("direct_io", True))),
                      F["path"].encode(), int(F["row_ptr_offset"]), int(F["col_idx_offset"]), int(F["vals_offset"]))


def read_csr_file(F, mem: str = "device", chunk_bytes: int = 0, stream=None, device: int = 0):
    """A CSR held in a file (a dict as for ``tile_plan_file``, optionally
    with ``direct_io``) read whole into device memory (torch tensors from
    torch's allocator) or pinned host memory (numpy views owned by the
    library) through aires_csr_read_file.  Returns (Output, stats dict)."""
    if mem not in ("device", "pinned"):
        raise ValueError("mem must be 'device' or 'pinned'")
    lib = B_.load()
    fc = _file_csr(F)
    out, st = B_.CsrOut(), B_.ReadStats()
    alloc = B_.TorchAllocator(device) if mem == "device" else None
    B_.check(lib.aires_csr_read_file(ctypes.byref(fc), B_.MEM_DEVICE if mem == "device" else B_.MEM_HOST_PINNED,
                                     ctypes.byref(alloc.struct) if alloc else None, _stream_handle(stream),
                                     int(chunk_bytes), ctypes.byref(out), ctypes.byref(st)), "aires_csr_read_file")
    return Output(out, alloc), {"bytes_read": st.bytes_read, "read_ms": st.read_ms, "total_ms": st.total_ms}


def tile_plan(A, B, hbm_budget: int = 0, *, validate: bool = False, c_on_host: bool = False,
              c_bound: int = B_.CBOUND_PRODUCTS, timing: bool = False, max_tile_rows: int = 0,
              max_tile_bytes: int = 0, m_a_bytes: int = 0, dense_max_cols: int = 0,
              hash_max_products: int = 0, wave_max_products: int = 0, window_grain_cols: int = 0,
              window_max_grains: int = 0, window_max_entries: int = 0, count_grains: int = 0,
              keep_bitmap_products: int = 0, split_min_products: int = 0, split_max_rows: int = 0,
              window_pool_bytes: int = 0, bitmap_cache_bytes: int = 0, slab_min_products: int = 0,
              a_values: str = "given", segmentation: str = "robw",
              torch_allocator: bool = True, allocator=None, device: int = 0) -> Plan:
    """Plan C = A * B under a device budget (aires_tile_plan).  a_values:
    "given" (A's values) or "sym_norm" (a_ik = 1/sqrt(r_i r_k) of A's
    pattern, Eq. 2, derived on the device; A's vals may then be None).
    segmentation: "robw" (row blocks, Algorithm 1) or "maxfill" (segments
    filled to the slot that may end inside a row: the partial row is copied
    back, packed on the host with the next segment and sent again).
    ``allocator``: an object with a ctypes ``struct`` (``_binding.Allocator``)
    such as a ``_binding.TorchAllocator``; by default a TorchAllocator
    (``torch_allocator``) or the library's own hipMallocAsync."""
    lib = B_.load()
    a = B_.make_csr(*_parts(A))
    b = B_.make_csr(*_parts(B))
    o = B_.PlanOpts()
    B_.check(lib.aires_plan_opts_default(ctypes.byref(o)), "aires_plan_opts_default")
    o.validate = int(validate)
    o.c_placement = B_.MEM_HOST_PINNED if c_on_host else B_.MEM_DEVICE
    o.c_bound = c_bound
    o.timing = int(timing)
    o.max_tile_rows = max_tile_rows
    o.max_tile_bytes = max_tile_bytes
    o.m_a_bytes = m_a_bytes
    o.dense_max_cols = dense_max_cols
    o.hash_max_products = hash_max_products
    o.wave_max_products = wave_max_products
    o.window_grain_cols = window_grain_cols
    o.window_max_grains = window_max_grains
    o.window_max_entries = window_max_entries
    o.count_grains = count_grains
    o.keep_bitmap_products = keep_bitmap_products
    o.slab_min_products = slab_min_products
    o.split_min_products = split_min_products
    o.split_max_rows = split_max_rows
    o.window_pool_bytes = window_pool_bytes
    o.bitmap_cache_bytes = bitmap_cache_bytes
    if a_values not in ("given", "sym_norm"):
        raise ValueError("a_values must be 'given' or 'sym_norm'")
    o.a_values = B_.AVALUES_SYM_NORM if a_values == "sym_norm" else B_.AVALUES_GIVEN
    if segmentation not in ("robw", "maxfill"):
        raise ValueError("segmentation must be 'robw' or 'maxfill'")
    o.segmentation = B_.SEG_MAXFILL if segmentation == "maxfill" else B_.SEG_ROBW
    alloc = allocator
    if alloc is None and torch_allocator and (a.mem == B_.MEM_DEVICE or b.mem != B_.MEM_HOST):
        alloc = B_.TorchAllocator(device)
    if alloc is not None:
        o.allocator = ctypes.pointer(alloc.struct)
    h = ctypes.c_void_p()
    B_.check(lib.aires_tile_plan(ctypes.byref(a), ctypes.byref(b), int(hbm_budget), ctypes.byref(o),
                                 ctypes.byref(h)), "aires_tile_plan")
    return Plan(h.value, A, B, alloc, o)


@dataclass
class Info:
    ntiles: int
    m: int
    k: int
    n: int
    budget: int
    b_bytes: int
    a_bytes: int
    tile_budget: int
    peak_bytes: int
    c_bound_entries: int
    a_streamed: bool
    c_on_host: bool
    part_budget: int
    a_in_file: bool
    _pad1: int = 0


def plan_info(plan: Plan) -> Info:
    i = B_.PlanInfo()
    B_.check(B_.load().aires_plan_info(plan.handle, ctypes.byref(i)), "aires_plan_info")
    return Info(*(getattr(i, f) for f, _ in B_.PlanInfo._fields_))


def plan_tile(plan: Plan, t: int) -> dict:
    x = B_.Tile()
    B_.check(B_.load().aires_plan_tile(plan.handle, int(t), ctypes.byref(x)), "aires_plan_tile")
    return {f: getattr(x, f) for f, _ in B_.Tile._fields_}


def plan_tiles(plan: Plan) -> list[dict]:
    return [plan_tile(plan, t) for t in range(plan_info(plan).ntiles)]


def plan_stats(plan: Plan) -> dict:
    s = B_.Stats()
    B_.check(B_.load().aires_plan_stats(plan.handle, ctypes.byref(s)), "aires_plan_stats")
    d = {f: getattr(s, f) for f, _ in B_.Stats._fields_ if f != "kind_ms"}
    d["kind_ms"] = {ph: {B_.KIND_NAMES[k]: s.kind_ms[p][k] for k in range(len(B_.KIND_NAMES))}
                    for p, ph in enumerate(("symbolic", "numeric"))}
    return d


def plan_tile_stats(plan: Plan, t: int | None = None):
    """Per-tile counts, phase times and begin/end instants of the last call
    (aires_plan_tile_stats): one dict, or a list over all tiles."""
    if t is None:
        return [plan_tile_stats(plan, i) for i in range(plan_info(plan).ntiles)]
    x = B_.TileStats()
    B_.check(B_.load().aires_plan_tile_stats(plan.handle, int(t), ctypes.byref(x)), "aires_plan_tile_stats")
    return {f: getattr(x, f) for f, _ in B_.TileStats._fields_}


class Output:
    """C in CSR.  Device results are torch tensors owned by torch's
    allocator; host results are numpy views of pinned memory owned by the
    library until free() (or garbage collection)."""

    def __init__(self, out: B_.CsrOut, allocator):
        self.nrows, self.ncols, self.nnz = out.nrows, out.ncols, out.nnz
        self.on_host = out.mem == B_.MEM_HOST_PINNED
        self._out = out
        if self.on_host or allocator is None:
            if self.on_host:
                import numpy as np
                self.rp = np.ctypeslib.as_array(ctypes.cast(out.row_ptr, ctypes.POINTER(ctypes.c_int64)),
                                                (self.nrows + 1,))
                n = max(self.nnz, 0)
                if n:
                    self.col = np.ctypeslib.as_array(ctypes.cast(out.col_idx, ctypes.POINTER(ctypes.c_int32)), (n,))
                    self.val = np.ctypeslib.as_array(ctypes.cast(out.vals, ctypes.POINTER(ctypes.c_float)), (n,))
                else:
                    self.col = np.zeros(0, np.int32)
                    self.val = np.zeros(0, np.float32)
            else:
                raise RuntimeError("device output without the torch allocator is not wrapped")
        else:
            import torch
            self.rp = allocator.take(out.row_ptr, torch.int64, self.nrows + 1)
            self.col = allocator.take(out.col_idx, torch.int32, self.nnz)
            self.val = allocator.take(out.vals, torch.float32, self.nnz)
            B_.load().aires_csr_out_free(ctypes.byref(self._out))  # registry already released

    def free(self):
        if self._out is not None and self._out._owner:
            self.rp = self.col = self.val = None
            B_.load().aires_csr_out_free(ctypes.byref(self._out))
        self._out = None

    def __del__(self):
        try:
            if self.on_host:
                self.free()
        except Exception:  # noqa: BLE001
            pass


def _stream_handle(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


_SPMM_ALGOS = {"auto": 0, "rows": 1, "dense_tiles": 2}


def spmm(A, W, relu: bool = False, out=None, stream=None, algo: str = "auto"):
    """Y = act(A * W) (aires_spmm): A a device CSR (a tuple as from
    ``to_device``, or an ``Output`` of ``spgemm``), W a dense device float32
    matrix with A.ncols rows (row stride W.stride(0)); act is ReLU when
    ``relu``.  ``algo``: "auto", "rows" (entry gather) or "dense_tiles"
    (densified 64-row tiles on the matrix cores).  Returns Y (m x F
    float32, a new tensor unless ``out`` is given); valid once ``stream``
    reaches the enqueued kernels."""
    import torch
    if algo not in _SPMM_ALGOS:
        raise ValueError("algo must be one of %s" % sorted(_SPMM_ALGOS))
    m, k, rp, col, val = _parts(A)
    if W.dim() != 2 or W.dtype != torch.float32 or W.stride(1) != 1 or W.shape[0] != k:
        raise ValueError("W must be a float32 (A.ncols x F) matrix with unit column stride")
    F = int(W.shape[1])
    if out is None:
        out = torch.empty((m, F), dtype=torch.float32, device=W.device)
    if out.dim() != 2 or out.shape[0] != m or out.shape[1] != F or out.stride(1) != 1 or out.dtype != torch.float32:
        raise ValueError("out must be a float32 (m x F) matrix with unit column stride")
    a = B_.make_csr(m, k, rp, col, val)
    B_.check(B_.load().aires_spmm(ctypes.byref(a), W.data_ptr(), W.stride(0), F, out.data_ptr(), out.stride(0),
                                  B_.ACT_RELU if relu else B_.ACT_NONE, _SPMM_ALGOS[algo],
                                  _stream_handle(stream)), "aires_spmm")
    return out


def spgemm(plan: Plan, stream=None) -> Output:
    """C = A * B (aires_spgemm).  Work is enqueued on ``stream`` (torch's
    current stream by default); C is valid once that stream reaches it."""
    out = B_.CsrOut()
    B_.check(B_.load().aires_spgemm(plan.handle, _stream_handle(stream), ctypes.byref(out)), "aires_spgemm")
    return Output(out, plan.allocator)


def spgemm_noalloc(plan: Plan, rp, col, val, stream=None) -> int:
    """C = A * B into caller-owned device tensors (aires_spgemm_noalloc):
    rp int64 (m + 1), col int32 and val float32 of equal length (C's
    capacity).  The library allocates nothing (its workspace is a fixed
    per-device array).  Returns nnz(C); raises AiresError (AIRES_E_CAPACITY
    when C or the workspace does not fit)."""
    import torch
    if rp.dtype != torch.int64 or col.dtype != torch.int32 or val.dtype != torch.float32:
        raise TypeError("expected int64 rp, int32 col, float32 val")
    if col.numel() != val.numel() or not (rp.is_cuda and col.is_cuda and val.is_cuda):
        raise ValueError("col and val must be device tensors of equal length")
    nnz = ctypes.c_int64(-1)
    st = B_.load().aires_spgemm_noalloc(plan.handle, _stream_handle(stream), rp.data_ptr(),
                                        col.data_ptr() if col.numel() else None,
                                        val.data_ptr() if val.numel() else None, int(col.numel()),
                                        ctypes.byref(nnz))
    if st != B_.OK:
        err = B_.AiresError(st, "aires_spgemm_noalloc")
        err.nnz = nnz.value
        raise err
    return nnz.value


def stream_tiles(plan: Plan, h2d=None, compute=None, d2h=None) -> Output:
    """Out-of-core C = A * B with A in pinned host memory (aires_stream_tiles)."""
    import torch
    h2d = h2d or torch.cuda.Stream()
    d2h = d2h or torch.cuda.Stream()
    out = B_.CsrOut()
    B_.check(B_.load().aires_stream_tiles(plan.handle, _stream_handle(h2d), _stream_handle(compute),
                                          _stream_handle(d2h), ctypes.byref(out)), "aires_stream_tiles")
    return Output(out, plan.allocator)


def to_device(M, device="cuda"):
    """Copy a numpy CSR (nrows, ncols, rp, col, val) to device torch tensors."""
    import torch
    n, k, rp, col, val = _parts(M)
    return (n, k, torch.from_numpy(rp).to(device), torch.from_numpy(col).to(device),
            torch.from_numpy(val).to(device))


def to_pinned(M):
    import torch
    n, k, rp, col, val = _parts(M)
    return (n, k, torch.from_numpy(rp).pin_memory(), torch.from_numpy(col).pin_memory(),
            torch.from_numpy(val).pin_memory())
