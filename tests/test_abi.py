"""C-ABI checks that need no GPU: the library loads, exports every symbol
its header declares, reports errors, and plans RoBW tiles (host inputs)."""
import ctypes
import re
import json
import os
import subprocess

import numpy as np
import pytest

import oracle
import workloads
import paper_2507_02006_amd as aires
from paper_2507_02006_amd import _binding as B_


def test_exports_every_declared_symbol():
    lib = B_.load()
    syms = B_.declared_symbols()
    assert len(syms) >= 12
    for s in syms:
        assert hasattr(lib, s), s
    out = subprocess.run(["nm", "-D", "--defined-only", B_.LIB_PATH], capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    assert set(syms) <= exported


def test_version_and_strings():
    lib = B_.load()
    assert lib.aires_abi_version() == 5
    # the binding's structures, the header and the library agree on the version
    hdr = open(B_.HEADER).read()
    assert int(re.search(r"#define AIRES_ABI_VERSION (\d+)", hdr).group(1)) == B_.ABI_VERSION == 5
    assert int(re.search(r"#define AIRES_NUM_KINDS (\d+)", hdr).group(1)) == B_.NUM_KINDS
    assert lib.aires_status_string(0) == b"AIRES_OK"
    assert lib.aires_status_string(B_.E_BUDGET) == b"AIRES_E_BUDGET"
    assert lib.aires_status_string(-99) == b"AIRES_E_UNKNOWN"
    o = B_.PlanOpts()
    assert lib.aires_plan_opts_default(ctypes.byref(o)) == 0
    assert o.struct_size == ctypes.sizeof(B_.PlanOpts)
    assert lib.aires_plan_opts_default(None) == B_.E_INVALID_ARG


def _host(M):
    return (M.nrows, M.ncols, M.rp, M.col, M.val)


def test_state_and_query_errors():
    """AIRES_E_STATE for an output descriptor that is not zeroed (checked
    before any device work), plan queries under their current names, and
    per-tile statistics of a plan that has not run (no GPU needed: a
    planning-only plan over host inputs)."""
    lib = B_.load()
    rng = np.random.default_rng(5)
    A = workloads.random_csr(rng, 40, 30, 0.2)
    Bm = workloads.random_csr(rng, 30, 9, 0.2)
    with aires.tile_plan(_host(A), _host(Bm), 1 << 30, m_a_bytes=200) as plan:
        info = aires.plan_info(plan)
        i2 = B_.PlanInfo()
        assert lib.aires_plan_info_get(plan.handle, ctypes.byref(i2)) == 0
        assert i2.ntiles == info.ntiles > 1
        assert lib.aires_plan_info(None, ctypes.byref(i2)) == B_.E_INVALID_ARG
        ts = aires.plan_tile_stats(plan)
        assert len(ts) == info.ntiles
        assert [(t["r0"], t["r1"]) for t in ts] == [(t["r0"], t["r1"]) for t in aires.plan_tiles(plan)]
        assert all(t["products"] == 0 and t["compute_begin_ms"] == -1.0 for t in ts)
        x = B_.TileStats()
        assert lib.aires_plan_tile_stats(plan.handle, info.ntiles, ctypes.byref(x)) == B_.E_INVALID_ARG
        assert lib.aires_plan_tile_stats(plan.handle, -1, ctypes.byref(x)) == B_.E_INVALID_ARG
        dummy = (ctypes.c_int64 * 4)()
        out = B_.CsrOut()
        out.row_ptr = ctypes.cast(dummy, ctypes.c_void_p)
        assert lib.aires_spgemm(plan.handle, None, ctypes.byref(out)) == B_.E_STATE
        assert b"not zeroed" in lib.aires_last_error()
        assert lib.aires_stream_tiles(plan.handle, None, None, None, ctypes.byref(out)) == B_.E_STATE


def test_error_paths():
    lib = B_.load()
    rng = np.random.default_rng(0)
    A = workloads.random_csr(rng, 20, 10, 0.3)
    Bm = workloads.random_csr(rng, 11, 7, 0.3)
    with pytest.raises(aires.AiresError) as e:
        aires.tile_plan(_host(A), _host(Bm), 1 << 30)
    assert e.value.status == B_.E_DIM
    Bm = workloads.random_csr(rng, 10, 7, 0.3)
    with pytest.raises(aires.AiresError) as e:
        aires.tile_plan(_host(A), _host(Bm), 1000)
    assert e.value.status == B_.E_BUDGET
    bad = workloads.random_csr(rng, 10, 7, 0.5)
    bad.col[:2] = [3, 3] if bad.rp[1] >= 2 else bad.col[:2]
    col = bad.col.copy()
    r = int(np.argmax(np.diff(bad.rp) >= 2))
    col[bad.rp[r]:bad.rp[r] + 2] = [5, 2]          # decreasing columns in row r
    with pytest.raises(aires.AiresError) as e:
        aires.tile_plan(_host(A), (10, 7, bad.rp, col, bad.val), 1 << 30, validate=True)
    assert e.value.status == B_.E_INVALID_CSR
    # NULL handles and a wrong struct_size
    a = B_.make_csr(*_host(A))
    h = ctypes.c_void_p()
    assert lib.aires_tile_plan(None, ctypes.byref(a), 1 << 30, None, ctypes.byref(h)) == B_.E_INVALID_ARG
    o = B_.PlanOpts()
    lib.aires_plan_opts_default(ctypes.byref(o))
    o.struct_size = 3
    b = B_.make_csr(*_host(Bm))
    assert lib.aires_tile_plan(ctypes.byref(a), ctypes.byref(b), 1 << 30, ctypes.byref(o), ctypes.byref(h)) \
        == B_.E_INVALID_ARG
    assert b"struct_size" in lib.aires_last_error()
    # device-resident A with C on the host is not a supported combination
    assert h.value is None


def test_algorithm1_hand_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "robw_hand.json")))
    rp = np.array(g["rp"], np.int32)
    A = (4, 4, rp, np.array([0, 2, 1, 3, 0, 3], np.int32), np.ones(6, np.float32))
    Bm = (4, 4, np.array([0, 2, 4, 5, 7], np.int32), np.array([1, 3, 0, 3, 2, 1, 3], np.int32),
          np.ones(7, np.float32))
    for case in g["cases"]:
        if case["tiles"] is None:
            with pytest.raises(aires.AiresError) as e:
                aires.tile_plan(A, Bm, 1 << 30, m_a_bytes=case["M_A"])
            assert e.value.status == B_.E_BUDGET
            continue
        with aires.tile_plan(A, Bm, 1 << 30, m_a_bytes=case["M_A"]) as p:
            got = [[t["r0"], t["r1"]] for t in aires.plan_tiles(p)]
        assert got == case["tiles"]


@pytest.mark.parametrize("seed", range(12))
def test_algorithm1_matches_oracle(seed):
    """The library's bisection planner yields the blocks of the oracle's
    literal linear greedy (Algorithm 1)."""
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 3000))
    rp64 = bool(seed % 2)
    A = workloads.random_csr(rng, m, 50, rng.uniform(0.01, 0.3), rp64=rp64)
    Bm = workloads.random_csr(rng, 50, 30, 0.2)
    s = 8 if rp64 else 4
    need = max((2 * s + 8 * int(A.rp[i + 1] - A.rp[i])) for i in range(m))
    M_A = int(need + rng.integers(0, 5000))
    want = oracle.robw(A.rp, s, M_A)
    with aires.tile_plan(_host(A), _host(Bm), 1 << 40, m_a_bytes=M_A) as p:
        got = [(t["r0"], t["r1"]) for t in aires.plan_tiles(p)]
        info = aires.plan_info(p)
    assert got == want
    assert info.ntiles == len(want)


def _slot_bytes(A, P, N, r0, r1, s, per_row_ws=12):
    """Documented per-slot bytes for a host-resident A with C placed in host
    memory: tile workspace + A slices + C bound (min(N, P_i) entries)."""
    k = r1 - r0
    q = int(A.rp[r1] - A.rp[r0])
    cb = int(np.minimum(P[r0:r1], N).sum())
    return k * per_row_ws + (k + 1) * s + 8 * q + 8 * cb + 8 * (k + 1)


@pytest.mark.parametrize("seed", range(6))
def test_streamed_plan_invariants(seed):
    """Host-resident A, C in host memory: tiles partition the rows, each slot
    fits the tile budget (checked against the documented cost model with
    P_i from the oracle), and each block is maximal."""
    rng = np.random.default_rng(100 + seed)
    A, Bm = workloads.workload(1, n=1024 + 200 * seed)
    P = oracle.products(A, Bm)
    budget = Bm.nbytes() + (4 << 20) + int(rng.integers(2, 6)) * 200_000
    with aires.tile_plan(_host(A), _host(Bm), budget, c_on_host=True) as p:
        info = aires.plan_info(p)
        tiles = aires.plan_tiles(p)
    assert info.a_streamed and info.c_on_host
    assert info.c_bound_entries == int(np.minimum(P, Bm.ncols).sum())
    assert info.tile_budget == (budget - (Bm.nbytes() + (4 << 20))) // 2
    assert tiles[0]["r0"] == 0 and tiles[-1]["r1"] == A.nrows
    for t0, t1 in zip(tiles[:-1], tiles[1:]):
        assert t0["r1"] == t1["r0"]
    for t in tiles:
        sb = _slot_bytes(A, P, Bm.ncols, t["r0"], t["r1"], 4)
        assert t["tile_bytes"] == sb and sb <= info.part_budget <= info.tile_budget
        assert t["c_bound_entries"] == int(np.minimum(P[t["r0"]:t["r1"]], Bm.ncols).sum())
    for t in tiles[:-1]:
        assert _slot_bytes(A, P, Bm.ncols, t["r0"], t["r1"] + 1, 4) > info.part_budget
    # the two slots hold the largest row count, entry count and C bound of
    # any tiles together (row pointers 4 B, 12 B of row workspace, 8 B of C
    # row pointer per row, 8 B per entry and per C bound entry)
    mk = max(t["r1"] - t["r0"] for t in tiles)
    mq = max(t["nnz1"] - t["nnz0"] for t in tiles)
    mc = max(t["c_bound_entries"] for t in tiles)
    assert mk * 12 + (mk + 1) * 4 + 8 * mq + 8 * mc + 8 * (mk + 1) <= info.tile_budget
    assert len(tiles) > 1


def test_tile_caps():
    A, Bm = workloads.workload(1, n=1000)
    with aires.tile_plan(_host(A), _host(Bm), 1 << 40, c_on_host=True, max_tile_rows=128) as p:
        tiles = aires.plan_tiles(p)
    assert [t["r1"] - t["r0"] for t in tiles] == [128] * 7 + [104]


def test_eq5_bound_mode():
    """Eq. 5 of the paper, read with alpha_A as the dense value bytes of A:
    M_C = 12 nnz(A) (1 + N/m + rho_B) bytes, i.e. M_C/8 entries."""
    A, Bm = workloads.workload(1, n=1024)
    with aires.tile_plan(_host(A), _host(Bm), 1 << 40, c_on_host=True, c_bound=B_.CBOUND_PAPER_EQ5) as p:
        info = aires.plan_info(p)
    rho = Bm.nnz / (Bm.nrows * Bm.ncols)
    mc = 12 * A.nnz * (1 + Bm.ncols / A.nrows + rho) / 8
    assert abs(info.c_bound_entries - mc) <= A.nrows + 1   # per-row ceil, capped at N


@pytest.mark.parametrize("N,row_max", [(8, 40), (300, 300), (70000, 70000)])
def test_streamed_c_bound_exact(N, row_max):
    """The planner's C bound is sum_i min(N, P_i) with P_i from the oracle,
    whatever the width of B's row lengths (byte, 16-bit, 32-bit tables) and
    with rows that reach N after a few entries (the bound pass stops
    summing a row there) next to rows that do not."""
    rng = np.random.default_rng(N)
    K, m = 400, 70000
    lens = rng.integers(0, row_max + 1, K)
    lens[:3] = [row_max, 0, 1]
    cols = [np.sort(rng.choice(N, min(int(L), N), replace=False)) for L in lens]
    brp = np.concatenate([[0], np.cumsum([len(c) for c in cols])]).astype(np.int64)
    Bm = workloads.CSR(K, N, brp.astype(np.int32), np.concatenate(cols).astype(np.int32),
                       np.ones(int(brp[-1]), np.float32))
    alen = rng.integers(0, 6, m)
    alen[:5] = [0, 1, K, 2, 50]
    acol = np.concatenate([np.sort(rng.choice(K, int(L), replace=False)) for L in alen]).astype(np.int32)
    arp = np.concatenate([[0], np.cumsum(alen)]).astype(np.int32)
    A = workloads.CSR(m, K, arp, acol, np.ones(len(acol), np.float32))
    P = oracle.products(A, Bm)
    with aires.tile_plan(_host(A), _host(Bm), 1 << 40, c_on_host=True) as p:
        info = aires.plan_info(p)
        tiles = aires.plan_tiles(p)
    assert info.c_bound_entries == int(np.minimum(P, N).sum())
    for t in tiles:
        assert t["c_bound_entries"] == int(np.minimum(P[t["r0"]:t["r1"]], N).sum())
    # C on the device: the plan needs (and keeps) only the total
    with aires.tile_plan(_host(A), _host(Bm), 1 << 40) as p:
        assert aires.plan_info(p).c_bound_entries == int(np.minimum(P, N).sum())
        assert all(t["c_bound_entries"] == -1 for t in aires.plan_tiles(p))


def test_sym_norm_plan():
    """a_values='sym_norm': A's values may be absent; a streamed plan keeps
    all of A's row pointers on the device (counted in the budget); A must be
    square."""
    A, Bm = workloads.workload(1, n=1024)
    budget = Bm.nbytes() + (4 << 20) + 600_000
    hA = _host(A)
    with aires.tile_plan(hA[:4] + (None,), _host(Bm), budget, c_on_host=True, a_values="sym_norm") as p:
        info = aires.plan_info(p)
    assert info.tile_budget == (budget - (Bm.nbytes() + (4 << 20) + 4 * (A.nrows + 1))) // 2
    with pytest.raises(aires.AiresError):
        aires.tile_plan(_host(Bm)[:4] + (None,), _host(workloads.random_csr(np.random.default_rng(1), 256, 7, 0.3)),
                        1 << 30, c_on_host=True, a_values="sym_norm")
    with pytest.raises(ValueError):
        aires.tile_plan(hA, _host(Bm), budget, c_on_host=True, a_values="normalised")


def test_spmm_argument_errors():
    """aires_spmm rejects bad arguments before touching the device: unknown
    activation or kernel family, W/Y strides below F, an A outside device
    memory, and dense tiles past their K and ldw limits."""
    lib = B_.load()
    fake = 1 << 40  # never dereferenced: every case fails validation first

    def call(A, ldw=64, F=64, ldy=64, act=B_.ACT_NONE, algo=B_.SPMM_AUTO):
        return lib.aires_spmm(ctypes.byref(A), fake, ldw, F, fake, ldy, act, algo, None)

    def csr(m=10, k=20, mem=B_.MEM_DEVICE):
        return B_.Csr(m, k, 5, B_.IDX_I32, mem, fake, fake, fake)

    assert call(csr(), act=5) == -1
    assert call(csr(), algo=7) == -1
    assert call(csr(), ldw=63) == -1
    assert call(csr(), ldy=10) == -1
    assert call(csr(mem=B_.MEM_HOST)) == -9
    assert call(csr(k=(1 << 20) + 1), algo=B_.SPMM_DENSE_TILES) == -9
    assert "dense tiles" in lib.aires_last_error().decode()
    assert call(csr(), ldw=1 << 23, algo=B_.SPMM_DENSE_TILES) == -9
    assert call(csr(), F=1 << 31) == -9


@pytest.mark.parametrize("N", [8, 256, 5000])
def test_streamed_rows_bound(N):
    """c_bound = ROWS: u_i = min(N, nnz(A_i) * max_k nnz(B_k)) from the row
    pointers alone; never below the exact bound min(N, P_i)."""
    rng = np.random.default_rng(N + 7)
    A = workloads.random_csr(rng, 70000, 300, 0.01)
    Bm = workloads.random_csr(rng, 300, N, min(1.0, 40.0 / N))
    alen = np.diff(A.rp.astype(np.int64))
    maxlen = int(np.diff(Bm.rp.astype(np.int64)).max())
    want = np.minimum(N, alen * maxlen)
    with aires.tile_plan(_host(A), _host(Bm), 1 << 40, c_on_host=True, c_bound=B_.CBOUND_ROWS) as p:
        info = aires.plan_info(p)
        tiles = aires.plan_tiles(p)
    assert info.c_bound_entries == int(want.sum())
    for t in tiles:
        assert t["c_bound_entries"] == int(want[t["r0"]:t["r1"]].sum())
    assert info.c_bound_entries >= int(np.minimum(oracle.products(A, Bm), N).sum())
    with aires.tile_plan(_host(A), _host(Bm), 1 << 40, c_bound=B_.CBOUND_ROWS) as p:
        assert aires.plan_info(p).c_bound_entries == int(want.sum())
        assert all(t["c_bound_entries"] == -1 for t in aires.plan_tiles(p))


def _pinned_desc(M):
    """A descriptor labelled pinned host memory over numpy arrays: planning
    reads host arrays only, so no device is needed to plan a streamed A."""
    d = B_.make_csr(M.nrows, M.ncols, M.rp, M.col, M.val)
    d.mem = B_.MEM_HOST_PINNED
    return d


def _plan_tiles(A, Bm, budget, **opts):
    lib = B_.load()
    o = B_.PlanOpts()
    lib.aires_plan_opts_default(ctypes.byref(o))
    for k, v in opts.items():
        setattr(o, k, v)
    a, b = _pinned_desc(A), _pinned_desc(Bm)
    h = ctypes.c_void_p()
    st = lib.aires_tile_plan(ctypes.byref(a), ctypes.byref(b), int(budget), ctypes.byref(o), ctypes.byref(h))
    if st != 0:
        raise aires.AiresError(st, "aires_tile_plan")
    info = B_.PlanInfo()
    lib.aires_plan_info(h, ctypes.byref(info))
    tiles = []
    for t in range(info.ntiles):
        x = B_.Tile()
        lib.aires_plan_tile(h, t, ctypes.byref(x))
        tiles.append({f: getattr(x, f) for f, _ in B_.Tile._fields_})
    lib.aires_plan_destroy(h)
    return info, tiles


def test_maxfill_segments_hand_example(golden_dir):
    """Max-fill segments of the 4x4 hand example (row lengths 2, 0, 2, 2;
    int32 row pointers) under a 40-byte cap on a segment's A bytes,
    (k + 1) * 4 + 8 q: entries [0, 3) (rows 0-1 complete, one entry of
    row 2 sent ahead), then [2, 5) (row 2 again, one entry of row 3 ahead),
    then [4, 6).  Row blocks under the same cap cut the same rows.  Under a
    cap below one row, every such row is a segment (a tile) of its own."""
    g = json.load(open(os.path.join(golden_dir, "hand_4x4.json")))
    mk = lambda d: workloads.CSR(d["nrows"], d["ncols"], np.array(d["rp"], np.int32), np.array(d["col"], np.int32),
                                 np.array(d["val"], np.float32))
    A, Bm = mk(g["A"]), mk(g["B"])
    _, seg = _plan_tiles(A, Bm, 1 << 30, max_tile_bytes=40, segmentation=B_.SEG_MAXFILL)
    assert [(t["r0"], t["r1"], t["nnz0"], t["nnz1"], t["sent_nnz1"]) for t in seg] == \
        [(0, 2, 0, 2, 3), (2, 3, 2, 4, 5), (3, 4, 4, 6, 6)]
    _, rb = _plan_tiles(A, Bm, 1 << 30, max_tile_bytes=40)
    assert [(t["r0"], t["r1"], t["nnz1"], t["sent_nnz1"]) for t in rb] == [(0, 2, 2, 2), (2, 3, 4, 4), (3, 4, 6, 6)]
    # a 23-byte cap is below every non-empty row (2 * 4 + 8 * 2 = 24 bytes):
    # such a row is a segment of its own, never divided; the empty row 1
    # goes with the head of row 2, which is sent again with the rest of it
    _, seg = _plan_tiles(A, Bm, 1 << 30, max_tile_bytes=23, segmentation=B_.SEG_MAXFILL)
    assert [(t["r0"], t["r1"], t["nnz0"], t["nnz1"], t["sent_nnz1"]) for t in seg] == \
        [(0, 1, 0, 2, 2), (1, 2, 2, 2, 3), (2, 3, 2, 4, 4), (3, 4, 4, 6, 6)]
    _, rb = _plan_tiles(A, Bm, 1 << 30, max_tile_bytes=23)
    assert [(t["r0"], t["r1"]) for t in rb] == [(0, 1), (1, 2), (2, 3), (3, 4)]  # rows 1-2: 12 + 16 > 23


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_maxfill_segments_fill_and_cover(seed):
    """On random row lengths (empty rows included): segments start where
    the previous one's complete rows end, cover every row once, send every
    entry at least once (the partial rows twice), end inside the next row
    unless they end the matrix, and are full: one more entry would pass
    the cap."""
    rng = np.random.default_rng(seed)
    m = 400
    lens = rng.integers(0, 30, m)
    lens[rng.random(m) < 0.2] = 0
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    col = np.concatenate([np.sort(rng.choice(50, int(L), replace=False)) for L in lens]).astype(np.int32)
    A = workloads.CSR(m, 50, rp, col, np.ones(len(col), np.float32))
    Bm = workloads.random_csr(rng, 50, 20, 0.2)
    cap = 600
    _, seg = _plan_tiles(A, Bm, 1 << 30, max_tile_bytes=cap, segmentation=B_.SEG_MAXFILL)
    assert seg[0]["r0"] == 0 and seg[-1]["r1"] == m and seg[-1]["sent_nnz1"] == rp[-1]
    for a, b in zip(seg, seg[1:]):
        assert b["r0"] == a["r1"] and b["nnz0"] == a["nnz1"] == rp[a["r1"]]
    for t in seg:
        r0, r1, q = t["r0"], t["r1"], t["sent_nnz1"] - t["nnz0"]
        assert r1 > r0 and t["nnz0"] == rp[r0] and t["nnz1"] == rp[r1]
        assert (r1 - r0 + 1) * 4 + 8 * q <= cap
        if t is not seg[-1]:
            assert rp[r1] <= t["sent_nnz1"] < rp[r1 + 1]  # ends inside row r1
            # one more entry: either past the cap, or it would complete more rows
            r1x = int(np.searchsorted(rp, t["sent_nnz1"] + 1, side="right")) - 1
            assert (r1x - r0 + 1) * 4 + 8 * (q + 1) > cap


def _plan_file(meta, Bm, budget, **opts):
    lib = B_.load()
    o = B_.PlanOpts()
    lib.aires_plan_opts_default(ctypes.byref(o))
    for k, v in opts.items():
        setattr(o, k, v)
    fa = B_.FileCsr(meta["nrows"], meta["ncols"], meta["nnz"], B_.IDX_I64 if meta["rp_dtype"] == "int64" else
                    B_.IDX_I32, int(meta.get("direct_io", 0)), meta["path"].encode(), meta["row_ptr_offset"],
                    meta["col_idx_offset"], meta["vals_offset"])
    b = _pinned_desc(Bm)
    h = ctypes.c_void_p()
    st = lib.aires_tile_plan_file(ctypes.byref(fa), ctypes.byref(b), int(budget), ctypes.byref(o), ctypes.byref(h))
    if st != 0:
        raise aires.AiresError(st, "aires_tile_plan_file")
    info = B_.PlanInfo()
    lib.aires_plan_info(h, ctypes.byref(info))
    tiles = []
    for t in range(info.ntiles):
        x = B_.Tile()
        lib.aires_plan_tile(h, t, ctypes.byref(x))
        tiles.append({f: getattr(x, f) for f, _ in B_.Tile._fields_})
    lib.aires_plan_destroy(h)
    return info, tiles


@pytest.mark.parametrize("rp64", [False, True])
def test_file_plan_equals_memory_plan(tmp_path, rp64):
    """A's arrays in a file (aligned raw arrays): the planner reads its row
    pointers and cuts the same row blocks, with the same C bound, as for
    the same A in host memory; direct I/O or not."""
    A, Bm = workloads.workload(5, n=6000)
    if not rp64:
        A = workloads.CSR(A.nrows, A.ncols, A.rp.astype(np.int32), A.col, A.val)
    meta = workloads.write_csr_file(str(tmp_path / "a.csr"), A)
    kw = dict(c_placement=B_.MEM_HOST_PINNED, c_bound=B_.CBOUND_ROWS, max_tile_bytes=40_000)
    budget = Bm.nbytes() + (16 << 20)
    info_m, tiles_m = _plan_tiles(A, Bm, budget, **kw)
    for direct in (0, 1):
        info_f, tiles_f = _plan_file(dict(meta, direct_io=direct), Bm, budget, **kw)
        assert tiles_f == tiles_m and len(tiles_f) > 5
        assert info_f.a_in_file == 1 and info_m.a_in_file == 0
        assert info_f.c_bound_entries == info_m.c_bound_entries and info_f.peak_bytes == info_m.peak_bytes


def test_file_plan_errors(tmp_path):
    A, Bm = workloads.workload(5, n=3000)
    meta = workloads.write_csr_file(str(tmp_path / "a.csr"), A)
    budget = Bm.nbytes() + (16 << 20)
    rows = dict(c_placement=B_.MEM_HOST_PINNED, c_bound=B_.CBOUND_ROWS)
    with pytest.raises(aires.AiresError) as e:  # the exact bound needs A's columns
        _plan_file(meta, Bm, budget, c_placement=B_.MEM_HOST_PINNED)
    assert e.value.status == B_.E_UNSUPPORTED
    with pytest.raises(aires.AiresError) as e:
        _plan_file(dict(meta, path=str(tmp_path / "missing")), Bm, budget, **rows)
    assert e.value.status == B_.E_INVALID_ARG
    with pytest.raises(aires.AiresError) as e:  # row pointers that do not end at nnz
        _plan_file(dict(meta, nnz=meta["nnz"] + 1), Bm, budget, **rows)
    assert e.value.status == B_.E_INVALID_CSR
    short = tmp_path / "short.csr"
    short.write_bytes((tmp_path / "a.csr").read_bytes()[:meta["row_ptr_offset"] + 100])
    with pytest.raises(aires.AiresError) as e:
        _plan_file(dict(meta, path=str(short)), Bm, budget, **rows)
    assert e.value.status == B_.E_INVALID_ARG and "ends before" in str(e.value)
    with pytest.raises(aires.AiresError) as e:
        _plan_file(meta, Bm, budget, segmentation=B_.SEG_MAXFILL, **rows)
    assert e.value.status == B_.E_UNSUPPORTED


def test_read_csr_file_errors(tmp_path):
    """aires_csr_read_file's argument and file checks, all taken before any
    device work; *out is left as it was."""
    lib = B_.load()
    A, _ = workloads.workload(5, n=3000)
    meta = workloads.write_csr_file(str(tmp_path / "a.csr"), A)

    def call(m=meta, mem=B_.MEM_DEVICE, chunk=0, null=False):
        out = B_.CsrOut()
        out.nnz = -7
        fc = None if null else aires._file_csr(m)
        st = lib.aires_csr_read_file(ctypes.byref(fc) if fc is not None else None, mem, None, None, chunk,
                                     ctypes.byref(out), None)
        assert out.nnz == -7 and not out.row_ptr
        return st, lib.aires_last_error()

    assert call(null=True)[0] == B_.E_INVALID_ARG
    assert call(mem=B_.MEM_HOST)[0] == B_.E_INVALID_ARG            # pageable host memory is not offered
    assert call(chunk=-1)[0] == B_.E_INVALID_ARG
    assert call(dict(meta, nrows=-1))[0] == B_.E_DIM
    assert call(dict(meta, path=str(tmp_path / "missing")))[0] == B_.E_INVALID_ARG
    st, msg = call(dict(meta, nnz=meta["nnz"] + 1))                # row pointers that do not end at nnz
    assert st == B_.E_INVALID_CSR and b"0 to nnz" in msg
    short = tmp_path / "short.csr"
    short.write_bytes((tmp_path / "a.csr").read_bytes()[:meta["row_ptr_offset"] + 100])
    st, msg = call(dict(meta, path=str(short)))
    assert st == B_.E_INVALID_ARG and b"ends before" in msg
    # row pointers 0, 3, 2, 4: a decreasing step
    bad = workloads.CSR(3, 5, np.array([0, 3, 2, 4], np.int32), np.array([0, 1, 2, 3], np.int32),
                        np.ones(4, np.float32))
    mb = workloads.write_csr_file(str(tmp_path / "bad.csr"), bad)
    st, msg = call(mb)
    assert st == B_.E_INVALID_CSR and b"decrease" in msg
