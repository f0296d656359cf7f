"""The C-ABI contract on the GPU: call order, transactional errors,
determinism of the overlapped schedule, and flush / resume."""
import numpy as np
import pytest

from paper_2205_04702_amd import workload as wl
from paper_2205_04702_amd import scratchpipe as spm

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def harness():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_harness
    return gpu_harness


def _say(msg):
    print(msg, flush=True)


def _small():
    return wl.custom(rows=[1500, 2500], dim=32, batch=24, pooling=[3, 2], slots=[300, 260],
                     lookahead=2, steps=16, dist=("zipf", 1.0), seed=31)


def test_call_order_is_enforced(harness):
    import torch
    w = _small()
    _say("case call order")
    host = harness.fresh_host(w)
    batches = harness.make_inputs(w)
    ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, w.lookahead, host, w.batch, w.nnz)
    out = torch.zeros((w.tables * w.batch, w.dim), device="cuda:0")
    g = torch.zeros_like(out)
    try:
        with pytest.raises(spm.SPError) as e:
            ctx.forward(0, out)
        assert e.value.status == spm.SP_ERR_SEQUENCE
        t = ctx.plan(batches[0:3])
        with pytest.raises(spm.SPError) as e:
            ctx.plan(batches[1:4])
        assert e.value.status == spm.SP_ERR_SEQUENCE
        with pytest.raises(spm.SPError) as e:
            ctx.backward_update(t, g, 0.1)
        assert e.value.status == spm.SP_ERR_SEQUENCE
        ctx.forward(t, out)
        with pytest.raises(spm.SPError) as e:
            ctx.forward(t, out)
        assert e.value.status == spm.SP_ERR_SEQUENCE
        with pytest.raises(spm.SPError) as e:
            ctx.backward_update(t + 1, g, 0.1)
        assert e.value.status == spm.SP_ERR_SEQUENCE
        ctx.backward_update(t, g, 0.1)
        with pytest.raises(spm.SPError) as e:
            ctx.plan(batches[1:7])  # more than lookahead + 1 + SP_MAX_AHEAD batches
        assert e.value.status == spm.SP_ERR_INVALID_ARG
        assert ctx.plan(batches[1:4]) == 1
    finally:
        ctx.close()
        host.close()


def _bad_ids(batch, w, table, row):
    ids, off = batch[0].copy(), batch[1]
    ids[int(off[table * w.batch])] = row
    return ids, off


def _big_batch(w):
    """Table 0: every bag row 0; table 1: one bag with slots+5 distinct rows."""
    big_rows = np.arange(w.slots[1] + 5, dtype=np.int32)
    ids = np.concatenate([np.zeros(w.batch * 3, np.int32), big_rows])
    off = np.concatenate([np.arange(0, 3 * w.batch + 1, 3),
                          np.full(w.batch, 3 * w.batch + big_rows.size)]).astype(np.int32)
    return ids, off


def _fat_table(w, n):
    """Table 0: n IDs in its first bag, the other bags empty; table 1: one ID per bag."""
    ids = np.concatenate([np.arange(n, dtype=np.int32) % w.rows[0], np.zeros(w.batch, np.int32)])
    off = np.concatenate([[0], np.full(w.batch - 1, n), n + np.arange(1, w.batch + 1)])
    return ids, off.astype(np.int32)


@pytest.mark.parametrize("lookahead,bound", [(0, 0), (2, 0), (0, 512), (2, 512)])
def test_rejected_plans_leave_state_unchanged(harness, lookahead, bound):
    """Rejected plans (row out of range, negative row, offsets not increasing,
    more misses than unheld slots, and with a bound on IDs per table a table
    above it) change nothing: continuing afterwards matches the oracle, which
    saw only the accepted plans.  New content enters through the window's last
    batch, the one seen for the first time.  bound 512 sorts each table in LDS."""
    import torch
    from oracle import oracle
    w = wl.custom(rows=[1500, 2500], dim=32, batch=24, pooling=[3, 2], slots=[300, 260],
                  lookahead=lookahead, steps=16, dist=("zipf", 1.0), seed=31)
    _say(f"case transactional errors L={lookahead} bound={bound}")
    batches = harness.make_inputs(w)
    host = harness.fresh_host(w)
    ref = [wl.init_table(w, t) for t in range(w.tables)]
    planner = oracle.Planner(w.rows, w.slots)
    ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, w.lookahead, host, w.batch, 4096,
                          max_table_ids=bound)
    out = torch.zeros((w.tables * w.batch, w.dim), device="cuda:0")
    L = w.lookahead
    try:
        for u in range(w.steps):
            win = batches[u:min(u + L, w.steps - 1) + 1]
            if u in (3, 7, 11):
                tail = win[-1]
                bad_windows = [
                    win[:-1] + [_bad_ids(tail, w, 1, w.rows[1])],          # row out of range
                    win[:-1] + [_bad_ids(tail, w, 0, -3)],                  # negative row
                    win[:-1] + [(tail[0], tail[1][::-1].copy())],          # offsets decreasing
                ] + ([win[:-1] + [_fat_table(w, bound + 1)]] if bound else [])  # over the bound
                for bw in bad_windows:
                    with pytest.raises(spm.SPError) as e:
                        ctx.plan(bw)
                    assert e.value.status == spm.SP_ERR_INVALID_ARG
                if L == 0:
                    big = _big_batch(w)
                    with pytest.raises(spm.SPError) as e:
                        ctx.plan([big])
                    assert e.value.status == spm.SP_ERR_CAPACITY
                    with pytest.raises(oracle.PlanError):
                        planner.plan([big], w.batch)
            t = ctx.plan(win)
            p = planner.plan(win, w.batch)
            harness.compare_plan(u, ctx.debug_plan(t, int(win[0][0].size)), p, w.tables, w.batch)
            ctx.forward(t, out)
            g = wl.grads(w, u)
            ctx.backward_update(t, torch.from_numpy(g).to("cuda:0"), w.lr)
            oracle.train_step(ref, *batches[u], w.batch, g, w.lr)
        ctx.flush()
        for t in range(w.tables):
            assert harness.row_rel_err(host[t], ref[t]).max() <= harness.REL_TOL
    finally:
        ctx.close()
        host.close()


@pytest.mark.parametrize("ahead", [1, 2])
def test_bad_prepared_batch_fails_the_plan_that_holds_it(harness, ahead):
    """A batch handed over early as a prepared-ahead batch is read once.  Bad
    content in it does not affect the plans it was handed to before it enters
    a hold window; the first plan whose window holds it is rejected whatever is
    passed, and a retry with good content re-reads it.  Continuing matches the
    oracle."""
    import torch
    from oracle import oracle
    w = wl.custom(rows=[1500, 2500], dim=32, batch=24, pooling=[3, 2], slots=[300, 260],
                  lookahead=2, steps=14, dist=("zipf", 1.0), seed=37)
    _say(f"case bad prepared-ahead batch, {ahead} ahead")
    batches = harness.make_inputs(w)
    host = harness.fresh_host(w)
    ref = [wl.init_table(w, t) for t in range(w.tables)]
    planner = oracle.Planner(w.rows, w.slots)
    ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, w.lookahead, host, w.batch, 4096)
    out = torch.zeros((w.tables * w.batch, w.dim), device="cuda:0")
    L, n = w.lookahead, w.steps
    try:
        for u in range(n):
            held = batches[u:min(u + L, n - 1) + 1]
            extra = [batches[q] for q in range(u + L + 1, u + L + 1 + ahead) if q < n]
            bad_q = 4 + L + ahead  # handed over last (and bad) at step 4
            if u == 4:
                extra[-1] = _bad_ids(extra[-1], w, 1, w.rows[1] + 7)
            if u == bad_q - L:  # first plan whose window holds it
                with pytest.raises(spm.SPError) as e:
                    ctx.plan(held + extra)
                assert e.value.status == spm.SP_ERR_INVALID_ARG
            t = ctx.plan(held + extra)
            p = planner.plan(held, w.batch)
            harness.compare_plan(u, ctx.debug_plan(t, int(held[0][0].size)), p, w.tables, w.batch)
            ctx.forward(t, out)
            g = wl.grads(w, u)
            ctx.backward_update(t, torch.from_numpy(g).to("cuda:0"), w.lr)
            oracle.train_step(ref, *batches[u], w.batch, g, w.lr)
        ctx.flush()
        for t in range(w.tables):
            assert harness.row_rel_err(host[t], ref[t]).max() <= harness.REL_TOL
    finally:
        ctx.close()
        host.close()


def test_overlapped_equals_serialized_bit_for_bit(harness):
    """The overlapped schedule (plan of the next batch while this one trains,
    fills and write-backs on side streams) gives exactly the tables of a run
    with a device synchronisation after every call, of runs with batches
    handed over early, of a run that waits on events instead of stream values,
    and of a second run."""
    w = wl.custom(rows=[3000, 5000, 2000], dim=64, batch=64, pooling=[4, 6, 2],
                  slots=[800, 1200, 500], lookahead=3, steps=30, dist=("zipf", 1.05), seed=41)
    _say("case overlap vs serialised")
    batches = harness.make_inputs(w)
    results = []
    for flags, ahead in ((0, 0), (spm.SP_FLAG_DEBUG_SYNC, 0), (0, 1), (0, 2),
                         (spm.SP_FLAG_EVENT_WAITS, 2), (0, 0)):
        host = harness.fresh_host(w)
        harness.run_gpu(w, batches, host, flags=flags, prepare_ahead=ahead)
        results.append([host[t].copy() for t in range(w.tables)])
        host.close()
    for r in results[1:]:
        for x, y in zip(results[0], r):
            assert np.array_equal(x, y)


def test_cached_equals_all_resident_bit_for_bit(harness):
    """The GPU's arithmetic order does not depend on which rows are cached."""
    w = wl.custom(rows=[2000, 3000], dim=32, batch=48, pooling=3, slots=[400, 600], lookahead=1,
                  steps=25, dist=("zipf", 0.9), seed=43)
    full = wl.custom(rows=[2000, 3000], dim=32, batch=48, pooling=3, slots=[2000, 3000],
                     lookahead=1, steps=25, dist=("zipf", 0.9), seed=43)
    _say("case cached vs resident")
    batches = harness.make_inputs(w)
    out = []
    for cfg in (w, full):
        host = harness.fresh_host(cfg)
        st = harness.run_gpu(cfg, batches, host)
        out.append(([host[t].copy() for t in range(cfg.tables)], st))
        host.close()
    assert out[0][1]["evictions"] > 0 and out[1][1]["evictions"] == 0
    for x, y in zip(out[0][0], out[1][0]):
        assert np.array_equal(x, y)


def test_flush_destroy_and_resume_is_bit_identical(harness):
    """Checkpoint = flushed host tables; a new context over them continues
    exactly as an uninterrupted run."""
    w = wl.custom(rows=[2500, 1800], dim=32, batch=32, pooling=[3, 4], slots=[500, 450],
                  lookahead=2, steps=24, dist=("zipf", 1.1), seed=47)
    _say("case resume")
    batches = harness.make_inputs(w)
    a = harness.fresh_host(w)
    harness.run_gpu(w, batches, a)
    b = harness.fresh_host(w)
    harness.run_gpu(w, batches, b, first=0, last=11)
    snapshot = [b[t].copy() for t in range(w.tables)]
    harness.run_gpu(w, batches, b, first=11, last=w.steps)
    for t in range(w.tables):
        assert np.array_equal(a[t], b[t])
        assert not np.array_equal(snapshot[t], b[t])
    a.close()
    b.close()


def test_stats_account_for_every_lookup(harness):
    w = _small()
    _say("case stats")
    batches = harness.make_inputs(w)
    host = harness.fresh_host(w)
    st = harness.run_gpu(w, batches, host, flags=spm.SP_FLAG_TIMING)
    host.close()
    assert st["plans"] == st["updates"] == w.steps
    assert st["lookups"] == sum(int(b[0].size) for b in batches)
    assert st["hits"] + st["misses"] == st["unique"]
    assert st["bytes_fill"] == st["misses"] * w.dim * 4
    assert st["evictions"] <= st["misses"]
    assert st["timed_forward"] == w.steps and st["ms_forward"] > 0
    assert st["min_capacity_margin"] >= 0


def test_timing_can_be_sampled_per_step(harness):
    """sp_set_flags switches kernel timing for the calls that follow; timed
    launch counts match the sampled steps and the trained tables do not depend
    on which steps were timed."""
    import torch
    w = _small()
    _say("case sampled timing")
    batches = harness.make_inputs(w)
    L = w.lookahead
    results = []
    for every in (0, 3):
        host = harness.fresh_host(w)
        ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, L, host, w.batch, 4096)
        out = torch.zeros((w.tables * w.batch, w.dim), device="cuda:0")
        try:
            for u in range(w.steps):
                if every:
                    ctx.set_flags(spm.SP_FLAG_TIMING if u % every == 0 else 0)
                t = ctx.plan(batches[u:min(u + L + 1, w.steps - 1) + 1])
                ctx.forward(t, out)
                ctx.backward_update(t, torch.from_numpy(wl.grads(w, u)).to("cuda:0"), w.lr)
            st = ctx.stats()
            ctx.flush()
        finally:
            ctx.close()
        n_timed = len(range(0, w.steps, every)) if every else 0
        assert st["timed_forward"] == n_timed and st["timed_backward"] == n_timed
        assert st["timed_plan"] == n_timed
        results.append([host[t].copy() for t in range(w.tables)])
        host.close()
    with pytest.raises(spm.SPError) as e:
        spm.sp_set_flags(0, 0)
    for x, y in zip(*results):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("fill", ["mapped", "staged"])
def test_allocation_failure_is_reported_and_cleaned_up(harness, fill, monkeypatch):
    """SP_FAIL_ALLOC_AFTER=n makes the allocation after the first n of sp_create fail:
    every such failure must come back as SP_ERR_OOM (no context, nothing leaked: the
    same create then succeeds), whichever allocation it hits."""
    import ctypes as C
    w = wl.custom(rows=[2000, 3000], dim=16, batch=16, pooling=2, slots=[200, 300],
                  lookahead=2, steps=4, seed=5)
    host = harness.fresh_host(w, fill)
    L = spm.load()
    rows = (C.c_int64 * 2)(*w.rows)
    slots = (C.c_int64 * 2)(*w.slots)
    tabs = (C.c_void_p * 2)(*host.ptrs)
    cfg = spm.sp_config(num_tables=2, rows=rows, dim=16, slots=slots, lookahead=2,
                        host_tables=tabs, max_batch=16, max_ids=64, flags=0, device=0,
                        fill=spm.FILLS[fill])
    try:
        failures = 0
        for n in (0, 1, 7, 30, 60, 90, 10_000):
            monkeypatch.setenv("SP_FAIL_ALLOC_AFTER", str(n))
            h = C.c_void_p()
            st = L.sp_create(C.byref(cfg), C.byref(h))
            if st == spm.SP_OK:  # n above the allocations the create makes
                assert h.value
                L.sp_destroy(h)
                continue
            failures += 1
            assert st == spm.SP_ERR_OOM and not h.value
            assert "injected" in spm.sp_last_error(None)
        assert failures >= 5
        monkeypatch.delenv("SP_FAIL_ALLOC_AFTER")
        ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, w.lookahead, host, max_batch=16,
                              max_ids=64, fill=fill)
        ctx.close()
    finally:
        host.close()


@pytest.mark.parametrize("hold_past", [0, 1])
def test_window_length_changes(harness, hold_past):
    """Windows that shorten and lengthen from step to step: a window shorter
    than what earlier plans held makes the plan rebuild every hold, and a
    longer one has several batches enter the hold window at once.  Every plan
    must equal the oracle's for the same windows, and the tables its
    training."""
    import torch
    from oracle import oracle
    w = wl.custom(rows=[1500, 2500, 900], dim=32, batch=24, pooling=[3, 2, 4],
                  slots=[420, 380, 300], lookahead=3, steps=26, dist=("zipf", 1.0), seed=53)
    _say(f"case window length changes, hold_past {hold_past}")
    batches = harness.make_inputs(w)
    host = harness.fresh_host(w)
    ref = [wl.init_table(w, t) for t in range(w.tables)]
    planner = oracle.Planner(w.rows, w.slots)
    ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, w.lookahead, host, w.batch, 4096,
                          hold_past=hold_past)
    out = torch.zeros((w.tables * w.batch, w.dim), device="cuda:0")
    n = len(batches)
    # window lengths (1 .. lookahead + 1): drops below what was held, regrowth
    lengths = [4, 4, 1, 1, 4, 2, 4, 4, 3, 1, 4, 4, 2, 2, 4, 1, 3, 4, 4, 1, 4, 4, 4, 2, 4, 4]
    try:
        for u in range(w.steps):
            win = batches[u:min(u + lengths[u], n)]
            t = ctx.plan(win)
            p = planner.plan(win, w.batch, past=batches[max(0, u - hold_past):u])
            harness.compare_plan(u, ctx.debug_plan(t, int(win[0][0].size)), p, w.tables, w.batch)
            ctx.forward(t, out)
            g = wl.grads(w, u)
            ctx.backward_update(t, torch.from_numpy(g).to("cuda:0"), w.lr)
            oracle.train_step(ref, *batches[u], w.batch, g, w.lr)
            _say(f"  step {u} window {len(win)} done")
        ctx.flush()
        for t in range(w.tables):
            assert harness.row_rel_err(host[t], ref[t]).max() <= harness.REL_TOL
    finally:
        ctx.close()
        host.close()
