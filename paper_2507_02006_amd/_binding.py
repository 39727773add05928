"""ctypes binding of libaires.so: argument marshalling only.

Every step of the product runs in the library's HIP kernels.  PyTorch
supplies device memory (through the allocator callbacks below, which hand
out blocks of torch's caching allocator) and streams.  There is no CPU
fallback: if the library is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libaires.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "aires.h")

c_i32, c_i64, c_u32, c_u64, c_vp, c_dbl, c_sz = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                                 ctypes.c_uint64, ctypes.c_void_p, ctypes.c_double,
                                                 ctypes.c_size_t)

# enums of aires.h
OK, E_INVALID_ARG, E_INVALID_CSR, E_DIM, E_BUDGET, E_OVERFLOW, E_OOM, E_HIP, E_STATE, \
    E_UNSUPPORTED, E_CAPACITY = 0, -1, -2, -3, -4, -5, -6, -7, -8, -9, -10
IDX_I32, IDX_I64 = 0, 1
MEM_DEVICE, MEM_HOST_PINNED, MEM_HOST = 0, 1, 2
CBOUND_PRODUCTS, CBOUND_DENSE, CBOUND_PAPER_EQ5, CBOUND_ROWS = 0, 1, 2, 3
KIND_NAMES = ["empty", "dense_wave", "dense_block", "hash_128", "hash_1024", "hash_8192", "windows", "split",
              "hash_4096"]
NUM_KINDS = 16  # kind_ms slots per phase
ABI_VERSION = 5  # AIRES_ABI_VERSION of the header these structures mirror


class Csr(ctypes.Structure):
    _fields_ = [("nrows", c_i64), ("ncols", c_i64), ("nnz", c_i64), ("rp_type", c_i32), ("mem", c_i32),
                ("row_ptr", c_vp), ("col_idx", c_vp), ("vals", c_vp)]


class CsrOut(ctypes.Structure):
    _fields_ = [("nrows", c_i64), ("ncols", c_i64), ("nnz", c_i64), ("row_ptr", c_vp), ("col_idx", c_vp),
                ("vals", c_vp), ("mem", c_i32), ("_reserved", c_i32), ("_owner", c_vp)]


ALLOC_FN = ctypes.CFUNCTYPE(c_vp, c_vp, c_sz, c_vp)
FREE_FN = ctypes.CFUNCTYPE(None, c_vp, c_vp, c_vp)


class Allocator(ctypes.Structure):
    _fields_ = [("alloc", ALLOC_FN), ("free", FREE_FN), ("ctx", c_vp)]


class PlanOpts(ctypes.Structure):
    _fields_ = [("struct_size", c_u32), ("validate", c_i32), ("c_placement", c_i32), ("c_bound", c_i32),
                ("timing", c_i32), ("_pad0", c_i32), ("max_tile_rows", c_i64), ("max_tile_bytes", c_i64),
                ("m_a_bytes", c_i64), ("allocator", ctypes.POINTER(Allocator)), ("dense_max_cols", c_i64),
                ("hash_max_products", c_i64), ("wave_max_products", c_i64), ("window_grain_cols", c_i64),
                ("window_max_grains", c_i64), ("window_max_entries", c_i64), ("count_grains", c_i64),
                ("keep_bitmap_products", c_i64), ("split_min_products", c_i64),
                ("split_max_rows", c_i64), ("window_pool_bytes", c_i64), ("a_values", c_i32),
                ("segmentation", c_i32), ("bitmap_cache_bytes", c_i64),
                ("slab_min_products", c_i64)]


class PlanInfo(ctypes.Structure):
    _fields_ = [(n, c_i64) for n in ("ntiles", "m", "k", "n", "budget", "b_bytes", "a_bytes", "tile_budget",
                                     "peak_bytes", "c_bound_entries")] + \
               [("a_streamed", c_i32), ("c_on_host", c_i32), ("part_budget", c_i64), ("a_in_file", c_i32),
                ("_pad1", c_i32)]


class Tile(ctypes.Structure):
    _fields_ = [(n, c_i64) for n in ("r0", "r1", "nnz0", "nnz1", "a_bytes", "c_bound_entries", "tile_bytes",
                                     "sent_nnz1")]


class Stats(ctypes.Structure):
    _fields_ = [(n, c_i64) for n in ("ntiles", "products", "nnz_c", "h2d_bytes", "d2h_bytes", "host_syncs")] + \
               [(n, c_dbl) for n in ("analyze_ms", "bin_ms", "symbolic_ms", "scan_ms", "numeric_ms", "h2d_ms",
                                     "d2h_ms", "total_ms")] + \
               [("numeric_launches", c_i64), ("kind_ms", (c_dbl * NUM_KINDS) * 2), ("pipeline_ms", c_dbl),
                ("resent_bytes", c_i64), ("merge_ms", c_dbl), ("storage_bytes", c_i64), ("storage_ms", c_dbl)]


class TileStats(ctypes.Structure):
    _fields_ = [(n, c_i64) for n in ("r0", "r1", "products", "nnz_c", "h2d_bytes", "d2h_bytes")] + \
               [(n, c_dbl) for n in ("analyze_ms", "bin_ms", "symbolic_ms", "scan_ms", "numeric_ms", "h2d_ms",
                                     "d2h_ms", "h2d_begin_ms", "h2d_end_ms", "compute_begin_ms",
                                     "compute_end_ms", "d2h_begin_ms", "d2h_end_ms")] + \
               [("resent_bytes", c_i64), ("merge_ms", c_dbl), ("storage_ms", c_dbl)]


class FileCsr(ctypes.Structure):
    _fields_ = [("nrows", c_i64), ("ncols", c_i64), ("nnz", c_i64), ("rp_type", c_i32), ("direct_io", c_i32),
                ("path", ctypes.c_char_p), ("row_ptr_offset", c_i64), ("col_idx_offset", c_i64),
                ("vals_offset", c_i64)]


class ReadStats(ctypes.Structure):
    _fields_ = [("bytes_read", c_i64), ("read_ms", c_dbl), ("total_ms", c_dbl)]


_lib = None


def declared_symbols() -> list[str]:
    """Function names declared in include/aires.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(aires_[a-z_0-9]+)\s*\(", text)))


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libaires.so is not built (run __graft_entry__.build()); "
                           "there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    sig = {
        "aires_abi_version": (ctypes.c_int, []),
        "aires_last_error": (ctypes.c_char_p, []),
        "aires_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "aires_plan_opts_default": (ctypes.c_int, [P(PlanOpts)]),
        "aires_tile_plan": (ctypes.c_int, [P(Csr), P(Csr), c_u64, P(PlanOpts), P(c_vp)]),
        "aires_tile_plan_file": (ctypes.c_int, [P(FileCsr), P(Csr), c_u64, P(PlanOpts), P(c_vp)]),
        "aires_csr_read_file": (ctypes.c_int, [P(FileCsr), c_i32, c_vp, c_vp, c_i64, P(CsrOut), P(ReadStats)]),
        "aires_plan_info": (ctypes.c_int, [c_vp, P(PlanInfo)]),
        "aires_plan_info_get": (ctypes.c_int, [c_vp, P(PlanInfo)]),
        "aires_plan_tile_stats": (ctypes.c_int, [c_vp, c_i64, P(TileStats)]),
        "aires_plan_tile": (ctypes.c_int, [c_vp, c_i64, P(Tile)]),
        "aires_spgemm": (ctypes.c_int, [c_vp, c_vp, P(CsrOut)]),
        "aires_spgemm_noalloc": (ctypes.c_int, [c_vp, c_vp, c_vp, c_vp, c_vp, c_i64, P(c_i64)]),
        "aires_stream_tiles": (ctypes.c_int, [c_vp, c_vp, c_vp, c_vp, P(CsrOut)]),
        "aires_plan_stats": (ctypes.c_int, [c_vp, P(Stats)]),
        "aires_csr_out_free": (None, [P(CsrOut)]),
        "aires_plan_destroy": (None, [c_vp]),
        "aires_spmm": (ctypes.c_int, [P(Csr), c_vp, c_i64, c_i64, c_vp, c_i64, ctypes.c_int, ctypes.c_int,
                                       c_vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    # the structures above follow one version of include/aires.h
    if lib.aires_abi_version() != ABI_VERSION:
        raise RuntimeError("libaires.so has ABI version %d, this binding expects %d (rebuild it)"
                           % (lib.aires_abi_version(), ABI_VERSION))
    _lib = lib
    return lib


ACT_NONE, ACT_RELU = 0, 1
SPMM_AUTO, SPMM_ROWS, SPMM_DENSE_TILES = 0, 1, 2
AVALUES_GIVEN, AVALUES_SYM_NORM = 0, 1
SEG_ROBW, SEG_MAXFILL = 0, 1


class AiresError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        self.status = status
        msg = lib.aires_status_string(status).decode()
        detail = lib.aires_last_error().decode()
        super().__init__("%s: %s (%s)" % (where, msg, detail))


def check(status: int, where: str) -> None:
    if status != OK:
        raise AiresError(status, where)


# ----------------------------------------------------------- descriptors

def _mem_of(x) -> int:
    if isinstance(x, np.ndarray):
        return MEM_HOST
    import torch
    if x.is_cuda:
        return MEM_DEVICE
    return MEM_HOST_PINNED if x.is_pinned() else MEM_HOST


def _ptr(x) -> int:
    if isinstance(x, np.ndarray):
        return x.ctypes.data if x.size else 0
    return x.data_ptr()


def _dtype_name(x) -> str:
    return str(x.dtype).replace("torch.", "")


def make_csr(nrows: int, ncols: int, rp, col, val) -> Csr:
    """Descriptor over caller arrays (numpy, pinned or device torch tensors).
    All three arrays must live in the same memory and be contiguous."""
    arrays = (rp, col) if val is None else (rp, col, val)
    mems = {_mem_of(x) for x in arrays}
    if len(mems) != 1:
        raise ValueError("row_ptr, col_idx and vals must live in the same memory")
    rpt = _dtype_name(rp)
    if rpt not in ("int32", "int64") or _dtype_name(col) != "int32" or \
            (val is not None and _dtype_name(val) != "float32"):
        raise TypeError("expected int32/int64 row_ptr, int32 col_idx, float32 vals")
    for x in arrays:
        if not (x.flags["C_CONTIGUOUS"] if isinstance(x, np.ndarray) else x.is_contiguous()):
            raise ValueError("arrays must be contiguous")
    nnz = int(col.shape[0])
    return Csr(int(nrows), int(ncols), nnz, IDX_I64 if rpt == "int64" else IDX_I32, mems.pop(),
               _ptr(rp) or None, _ptr(col) or None, (_ptr(val) or None) if val is not None else None)


# -------------------------------------------------------------- allocator

class TorchAllocator:
    """Device memory for the library from torch's caching allocator.  Blocks
    are uint8 tensors kept alive in a registry until the library frees them
    (or Python takes them over as output views).

    Each block is allocated with the library's stream (the callback's
    `stream` argument) as torch's current stream.  torch's cache keeps a
    freed block for later allocations on that same stream only, so when the
    library frees a block while its kernels on that stream may still read
    it, the block cannot be handed to work on any other stream."""

    def __init__(self, device: int = 0):
        import torch
        self.torch = torch
        self.device = device
        self.live: dict[int, object] = {}
        self._alloc = ALLOC_FN(self._alloc_cb)
        self._free = FREE_FN(self._free_cb)
        self.struct = Allocator(self._alloc, self._free, None)
        self.peak = 0
        self.cur = 0
        self.calls = 0
        self._streams: dict[int, object] = {}

    def _stream_of(self, handle):
        """The torch stream object for a hipStream_t handle."""
        torch = self.torch
        h = int(handle or 0)
        cur = torch.cuda.current_stream(self.device)
        if cur.cuda_stream == h:
            return cur
        if h == 0:
            return torch.cuda.default_stream(self.device)
        s = self._streams.get(h)
        if s is None:
            s = torch.cuda.ExternalStream(h, device=self.device)
            self._streams[h] = s
        return s

    def _alloc_cb(self, ctx, nbytes, stream):
        self.calls += 1
        try:
            with self.torch.cuda.stream(self._stream_of(stream)):
                t = self.torch.empty(int(nbytes), dtype=self.torch.uint8, device="cuda:%d" % self.device)
        except Exception:  # noqa: BLE001 -- out of memory is reported as NULL
            return None
        p = t.data_ptr()
        self.live[p] = t
        self.cur += int(nbytes)
        self.peak = max(self.peak, self.cur)
        return p

    def _free_cb(self, ctx, ptr, stream):
        t = self.live.pop(ptr, None)
        if t is not None:
            self.cur -= t.numel()

    def take(self, ptr: int, dtype, n: int):
        """Take ownership of a library block as a typed tensor view."""
        t = self.live.pop(ptr)
        self.cur -= t.numel()
        esz = self.torch.empty(0, dtype=dtype).element_size()
        return t[: max(n, 0) * esz].view(dtype)
