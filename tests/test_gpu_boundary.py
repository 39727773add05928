"""GPU checks of the C-ABI's contract beyond the numbers: the device budget
(the memory constraint M of Sec. III-A) measured at the allocator, failure
and rollback paths (AIRES_E_OOM, AIRES_E_BUDGET, AIRES_E_STATE), a call on
a stream other than torch's current one, and the per-tile statistics of the
row-block schedule (Algorithm 2)."""
import ctypes
import sys

import numpy as np
import pytest

import oracle
import workloads

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


def assert_match(rp, col, val, ref):
    assert np.array_equal(rp, ref.rp), "row_ptr differs"
    assert np.array_equal(col, ref.col), "col_idx differs"
    err = np.abs(val.astype(np.float64) - ref.val.astype(np.float64))
    assert np.all(err <= TOL * (1 + np.abs(ref.val.astype(np.float64)))), "values differ"


class FailingAllocator:
    """torch-backed allocator whose n-th request returns NULL."""

    def __init__(self, fail_at):
        from paper_2507_02006_amd import _binding as B_
        self.inner = B_.TorchAllocator(0)
        self.fail_at = fail_at
        self.calls = 0
        self._alloc = B_.ALLOC_FN(self._alloc_cb)
        self.struct = B_.Allocator(self._alloc, self.inner._free, None)
        self.take = self.inner.take

    def _alloc_cb(self, ctx, nbytes, stream):
        self.calls += 1
        if self.calls == self.fail_at:
            return None
        return self.inner._alloc_cb(ctx, nbytes, stream)


@pytest.mark.parametrize("wide", [False, True])
def test_oom_rolls_back(torch_gpu, wide):
    """The allocator refuses its n-th request, for every n the call makes:
    AIRES_E_OOM, and every block taken before it is handed back."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B = workloads.workload(3 if wide else 2, n=6000)
    dA, dB = aires.to_device(A), aires.to_device(B)
    kw = dict(dense_max_cols=1024, window_grain_cols=1024) if wide else {}
    probe = B_.TorchAllocator(0)
    with aires.tile_plan(dA, dB, 0, allocator=probe, max_tile_rows=2500, **kw) as plan:
        aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
    ncalls = probe.calls
    say("oom rollback wide=%s: %d allocations per call" % (wide, ncalls))
    assert ncalls >= 8
    ref = oracle.spgemm(A, B)
    optional = 0
    for n in range(1, ncalls + 1):
        fa = FailingAllocator(n)
        with aires.tile_plan(dA, dB, 0, allocator=fa, max_tile_rows=2500, **kw) as plan:
            try:
                C = aires.spgemm(plan)
            except aires.AiresError as e:
                torch_gpu.cuda.synchronize()
                assert e.status == B_.E_OOM, (n, str(e))
                assert fa.inner.cur == 0 and not fa.inner.live, n
                continue
            # the one optional request (the cache of kept symbolic bitmaps
            # of wide rows) may be refused: the call goes on without it
            torch_gpu.cuda.synchronize()
            optional += 1
            assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)
            del C
    assert optional <= (1 if wide else 0)
    # the plan still works afterwards with a good allocator
    with aires.tile_plan(dA, dB, 0, max_tile_rows=2500, **kw) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)


def test_budget_too_small_for_c(torch_gpu):
    """A budget that holds the workspace but not the exact C: AIRES_E_BUDGET
    after the symbolic phase, nothing left allocated; the measured peak of a
    successful call under a budget just above its need stays within it."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B = workloads.workload(2, n=16384)
    ref = oracle.spgemm(A, B)
    dA, dB = aires.to_device(A), aires.to_device(B)
    inputs = A.nbytes() + B.nbytes()
    probe = B_.TorchAllocator(0)
    with aires.tile_plan(dA, dB, 0, allocator=probe) as plan:
        aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
    need = probe.peak
    c_bytes = 8 * ref.nnz
    say("budget: need %d bytes of which C %d" % (need, c_bytes))
    tight = B_.TorchAllocator(0)
    with aires.tile_plan(dA, dB, inputs + need - c_bytes // 2, allocator=tight) as plan:
        with pytest.raises(aires.AiresError) as e:
            aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
    assert e.value.status == B_.E_BUDGET and b"C needs" in str(e.value).encode()
    assert tight.cur == 0 and not tight.live
    ok = B_.TorchAllocator(0)
    with aires.tile_plan(dA, dB, inputs + need, allocator=ok) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        assert ok.peak <= need
        assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)


def test_plan_in_use(torch_gpu):
    """A second call on a plan while its first call runs (here: from inside
    the first call's allocator) is refused with AIRES_E_STATE; the first
    call still completes correctly."""
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    A, B = workloads.workload(1, n=2048)
    ref = oracle.spgemm(A, B)
    dA, dB = aires.to_device(A), aires.to_device(B)
    seen = []

    class Reentrant(B_.TorchAllocator):
        plan = None

        def _alloc_cb(self, ctx, nbytes, stream):
            if self.plan is not None and not seen:
                out = B_.CsrOut()
                seen.append(B_.load().aires_spgemm(self.plan.handle, stream, ctypes.byref(out)))
                seen.append(B_.load().aires_last_error())
            return super()._alloc_cb(ctx, nbytes, stream)

    al = Reentrant(0)
    with aires.tile_plan(dA, dB, 0, allocator=al) as plan:
        al.plan = plan
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        assert seen[0] == B_.E_STATE and b"in use" in seen[1]
        assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)


@pytest.mark.parametrize("wide", [False, True])
def test_side_stream(torch_gpu, wide):
    """spgemm on a stream that is not torch's current one, followed at once
    by allocations and writes on the current stream: the library's blocks
    belong to its own stream, so the writes cannot land in its workspace."""
    import paper_2507_02006_amd as aires
    torch = torch_gpu
    A, B = workloads.workload(3 if wide else 2, n=20000)
    ref = oracle.spgemm(A, B)
    dA, dB = aires.to_device(A), aires.to_device(B)
    kw = dict(dense_max_cols=4096, window_grain_cols=4096) if wide else {}
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    for rep in range(3):
        with aires.tile_plan(dA, dB, 0, **kw) as plan:
            C = aires.spgemm(plan, stream=side)
            junk = [torch.full((1 << 20,), -7.0, device="cuda") for _ in range(64)]
            side.synchronize()
            torch.cuda.synchronize()
            del junk
            with torch.cuda.stream(side):
                rp, col, val = C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy()
            assert_match(rp, col, val, ref)
            del C


def test_tile_stats_in_core(torch_gpu):
    """Per-tile statistics of an in-core tiled call: counts add up to the
    call's, each tile's products and nnz(C) equal the oracle's for its rows,
    and its phases were timed."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(2, n=20000)
    P = oracle.products(A, B)
    ref = oracle.spgemm(A, B)
    with aires.tile_plan(aires.to_device(A), aires.to_device(B), 0, timing=True, max_tile_rows=3001) as plan:
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        st = aires.plan_stats(plan)
        ts = aires.plan_tile_stats(plan)
    assert len(ts) == 7
    for t in ts:
        assert t["products"] == int(P[t["r0"]:t["r1"]].sum())
        assert t["nnz_c"] == int(ref.rp[t["r1"]] - ref.rp[t["r0"]])
        assert t["h2d_bytes"] == 0 and t["d2h_bytes"] == 0
        assert t["symbolic_ms"] > 0 and t["numeric_ms"] > 0
        assert 0 <= t["compute_begin_ms"] < t["compute_end_ms"]
        assert t["h2d_begin_ms"] == -1.0 and t["d2h_begin_ms"] == -1.0
    assert sum(t["products"] for t in ts) == st["products"] == int(P.sum())
    assert sum(t["numeric_ms"] for t in ts) == pytest.approx(st["numeric_ms"], rel=1e-6, abs=1e-6)


@pytest.mark.parametrize("c_on_host", [True, False])
def test_streamed_budget_and_tiles(torch_gpu, c_on_host):
    """Streamed tiles under a tight budget: the device bytes the library
    held, measured at its allocator, stay within the budget (B in pinned
    host memory, so every device byte is the library's); per-tile bytes
    and counts add up; each tile's copy in precedes its compute, whose end
    precedes its copy of C back, and tile t+1's copy begins before tile t's
    products end."""
    import paper_2507_02006_amd as aires
    A, B = workloads.workload(5, n=60000)
    ref = oracle.spgemm(A, B)
    P = oracle.products(A, B)
    pA, pB = aires.to_pinned(A), aires.to_pinned(B)
    cb = int(np.minimum(P, B.ncols).sum())
    budget = B.nbytes() + (4 << 20) + (0 if c_on_host else 8 * (A.nrows + 1) + 8 * cb) + 2 * 1_500_000
    say("streamed budget c_on_host=%s budget=%d" % (c_on_host, budget))
    with aires.tile_plan(pA, pB, budget, c_on_host=c_on_host, timing=True) as plan:
        info = aires.plan_info(plan)
        C = aires.spgemm(plan)
        torch_gpu.cuda.synchronize()
        st = aires.plan_stats(plan)
        ts = aires.plan_tile_stats(plan)
        peak = plan.allocator.peak
        if c_on_host:
            assert_match(C.rp, C.col, C.val, ref)
            C.free()
        else:
            assert_match(C.rp.cpu().numpy(), C.col.cpu().numpy(), C.val.cpu().numpy(), ref)
    say("streamed: %d tiles, allocator peak %d of budget %d" % (info.ntiles, peak, budget))
    assert info.ntiles >= 3
    assert 0 < peak <= budget
    assert sum(t["h2d_bytes"] for t in ts) == A.nbytes() + 8 * (info.ntiles - 1)
    assert sum(t["d2h_bytes"] for t in ts) == st["d2h_bytes"]
    for t in ts:
        assert t["products"] == int(P[t["r0"]:t["r1"]].sum())
        assert t["nnz_c"] == int(ref.rp[t["r1"]] - ref.rp[t["r0"]])
        assert t["h2d_end_ms"] <= t["compute_begin_ms"] + 1e-3
        if c_on_host:
            assert t["compute_end_ms"] <= t["d2h_begin_ms"] + 1e-3
            assert t["d2h_bytes"] == 8 * (t["r1"] - t["r0"]) + 8 * t["nnz_c"]
        else:
            assert t["d2h_begin_ms"] == -1.0
    for t in range(info.ntiles - 1):
        assert ts[t + 1]["h2d_begin_ms"] < ts[t]["compute_end_ms"], t
