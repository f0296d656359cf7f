"""Parity of the HIP planner's prefetch mode (needs an MI355X).

With prefetch each plan also fills the rows of the next batch of its window
that are neither cached nor in the planned batch: an earlier fill of future
misses, which the multi-stage overlap of Sec. IV-C allows.  Plans (the miss
list with the planned batch's misses then the prefetched rows per table, the
victims, old rows and last uses, hits, slots) must match the oracle planner run
in the same mode bit for bit; outputs and tables within 1e-5 per row as in the
other parity tests.
"""
import pytest

from paper_2205_04702_amd import workload as wl

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


@pytest.mark.parametrize("policy", ["lru", "lfu", "random"])
def test_tiny_all_steps(harness, policy):
    """4 x 20k x 32, B=128, 4 IDs per bag, 2048 slots, lookahead 2, 50 steps."""
    w = wl.get_workload("tiny")
    _say(f"case prefetch tiny policy {policy}")
    r = harness.run_parity(w, policy=policy, seed=5, prefetch=True)
    st = r["stats"]
    assert st["evictions"] > 0 and st["prefetched"] > 0


def test_ragged_and_empty_bags_general_ingest(harness):
    """Ragged bags with empty ones, sorted by the general (multi-launch) ingest path."""
    w = wl.custom(rows=[3000, 5000], dim=16, batch=64, pooling=[3, 5], slots=[700, 900],
                  lookahead=2, steps=20, dist=(("zipf", 1.05), ("uniform",)), seed=6)
    batches = [wl.ragged_batch(w, s, max_len=8, empty_frac=0.25) for s in range(w.steps)]
    _say("case prefetch ragged general ingest")
    r = harness.run_parity(w, batches, prefetch=True, max_table_ids=0)
    assert r["stats"]["prefetched"] > 0


def test_no_lookahead_means_no_prefetch(harness):
    w = wl.custom(rows=[4000] * 2, dim=32, batch=64, pooling=4, slots=[600] * 2, lookahead=0,
                  steps=20, dist=("zipf", 1.05), seed=7)
    _say("case prefetch lookahead 0")
    r = harness.run_parity(w, prefetch=True)
    assert r["stats"]["prefetched"] == 0 and r["stats"]["evictions"] > 0


def test_past_window_and_prepared_batches(harness):
    """A past window of 2 (its batches follow the hold window in the query) and two
    batches handed over early from device memory."""
    w = wl.custom(rows=[50_000] * 3, dim=32, batch=128, pooling=4, slots=[4096] * 3,
                  lookahead=2, steps=30, dist=("zipf", 1.05), seed=4)
    _say("case prefetch past window 2")
    r = harness.run_parity(w, hold_past=2, prepare_ahead=2, device_ids=True, prefetch=True)
    assert r["stats"]["prefetched"] > 0 and r["stats"]["evictions"] > 0


def test_large_victim_sets(harness):
    """Over 2048 victims per table per plan (own and prefetched misses together): the
    victims are ordered by the global radix sort."""
    w = wl.custom(rows=[1_000_000] * 2, dim=16, batch=1024, pooling=4, slots=[30_000] * 2,
                  lookahead=1, steps=12, dist=("uniform",), seed=8)
    _say("case prefetch large victim sets")
    r = harness.run_parity(w, seed=3, sync_each_step=False, prefetch=True)
    st = r["stats"]
    assert st["evictions"] > 4 * 2 * 2048 and st["prefetched"] > 0


def test_zipf_8x1M_sampled(harness):
    """The benchmark workload with prefetch, driven as the benchmark drives it, 40 steps."""
    w = wl.get_workload("zipf-8x1M")
    _say("case prefetch zipf-8x1M")
    sample = [0, 1, 2, 13, 25, 38, 39]
    r = harness.run_sampled_parity(w, 40, check_plan_steps=sample, check_fwd_steps=sample,
                                   say=_say, prefetch=True)
    _say(f"zipf-8x1M prefetch: worst fwd {r['worst_fwd']:.2e} table {r['worst_table']:.2e} "
         f"misses {r['stats']['misses']} prefetched {r['stats']['prefetched']}")


def test_overlapped_equals_serialized_bit_for_bit(harness):
    """With prefetch the forward and update of a batch run beside its plan's fill: the
    overlapped schedule gives exactly the tables of runs synchronised after every call,
    with batches handed over early, and waiting on events instead of stream values."""
    import numpy as np
    from paper_2205_04702_amd import scratchpipe as spm
    w = wl.custom(rows=[3000, 5000, 2000], dim=64, batch=64, pooling=[4, 6, 2],
                  slots=[900, 1400, 600], lookahead=3, steps=30, dist=("zipf", 1.05), seed=41)
    _say("case prefetch overlap vs serialised")
    batches = harness.make_inputs(w)
    results = []
    for flags, ahead in ((0, 0), (spm.SP_FLAG_DEBUG_SYNC, 0), (0, 2), (spm.SP_FLAG_EVENT_WAITS, 2)):
        host = harness.fresh_host(w)
        st = harness.run_gpu(w, batches, host, flags=flags, prepare_ahead=ahead, prefetch=True)
        assert st["prefetched"] > 0 and st["evictions"] > 0
        results.append([host[t].copy() for t in range(w.tables)])
        host.close()
    for r in results[1:]:
        for x, y in zip(results[0], r):
            assert np.array_equal(x, y)


def test_capacity_error_from_the_prefetched_rows_changes_nothing(harness):
    """A next batch whose new rows do not fit beside the planned batch's is rejected
    (SP_ERR_CAPACITY) as the oracle rejects it; continuing with the regular window then
    matches the oracle, which saw only the accepted plans."""
    import numpy as np
    import torch
    from oracle import oracle
    from paper_2205_04702_amd import scratchpipe as spm
    w = wl.custom(rows=[1500, 2500], dim=32, batch=24, pooling=[3, 2], slots=[300, 260],
                  lookahead=1, steps=12, dist=("zipf", 1.0), seed=31)
    _say("case prefetch capacity error")
    batches = harness.make_inputs(w)
    host = harness.fresh_host(w)
    ref = [wl.init_table(w, t) for t in range(w.tables)]
    planner = oracle.Planner(w.rows, w.slots, prefetch=True)
    ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, w.lookahead, host, w.batch, 4096, prefetch=True)
    # table 1 of the substitute next batch: one bag of slots + 5 distinct rows
    big_rows = np.arange(1000, 1000 + w.slots[1] + 5, dtype=np.int32)
    big_ids = np.concatenate([np.zeros(w.batch * 3, np.int32), big_rows])
    big_off = np.concatenate([np.arange(0, 3 * w.batch + 1, 3),
                              np.full(w.batch, 3 * w.batch + big_rows.size)]).astype(np.int32)
    out = torch.zeros((w.tables * w.batch, w.dim), device="cuda:0")
    try:
        for u in range(w.steps):
            win = batches[u:min(u + 1, w.steps - 1) + 1]
            if u in (2, 6) and len(win) == 2:
                with pytest.raises(spm.SPError) as e:
                    ctx.plan([win[0], (big_ids, big_off)])
                assert e.value.status == spm.SP_ERR_CAPACITY
                with pytest.raises(oracle.PlanError):
                    planner.plan([win[0], (big_ids, big_off)], w.batch)
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


# ----------------------------------------------------------------------------- deeper prefetch

@pytest.mark.parametrize("depth", [2, 3, 4])
def test_deeper_prefetch_every_step(harness, depth):
    """Prefetch depth d: each plan also fills the rows of its next d batches that are
    neither cached nor in an earlier window batch, successor by successor."""
    w = wl.custom(rows=[6000, 9000, 4000], dim=32, batch=64, pooling=[4, 3, 5],
                  slots=[2500, 3000, 2200], lookahead=4, steps=30,
                  dist=(("zipf", 1.05), ("uniform",), ("zipf", 1.2)), seed=60 + depth)
    _say(f"case prefetch depth {depth}")
    r = harness.run_parity(w, prefetch=depth, prepare_ahead=2)
    st = r["stats"]
    assert st["prefetched"] > 0 and st["evictions"] > 0


@pytest.mark.parametrize("policy", ["lfu", "random"])
def test_deeper_prefetch_policies_past_window_device_ids(harness, policy):
    w = wl.custom(rows=[40_000] * 2, dim=16, batch=96, pooling=4, slots=[5000] * 2,
                  lookahead=3, steps=24, dist=("zipf", 1.05), seed=71)
    _say(f"case prefetch depth 3 policy {policy} past 1")
    r = harness.run_parity(w, prefetch=3, policy=policy, seed=9, hold_past=1, prepare_ahead=2,
                           device_ids=True, sync_each_step=False, check_fwd_steps=[0, 12, 23])
    assert r["stats"]["prefetched"] > 0


def test_deeper_prefetch_ragged_general_ingest_large_victims(harness):
    """Ragged and empty bags on the general ingest path, and over 2048 victims per
    table (the global victim sort), at depth 2."""
    w = wl.custom(rows=[800_000, 500_000], dim=16, batch=1024, pooling=[4, 3],
                  slots=[40_000, 30_000], lookahead=2, steps=10, dist=("uniform",), seed=72)
    batches = [wl.ragged_batch(w, s, max_len=7, empty_frac=0.2) for s in range(w.steps)]
    _say("case prefetch depth 2 ragged large")
    r = harness.run_parity(w, batches, prefetch=2, max_table_ids=0, sync_each_step=False,
                           check_fwd_steps=[0, 9])
    assert r["stats"]["prefetched"] > 2 * 2048


def test_deeper_prefetch_overlapped_and_staged_equal_serialized(harness):
    """Depth 3: the overlapped schedule, the serialised one, event waits and the staged
    fill give bit-identical tables."""
    import numpy as np
    from paper_2205_04702_amd import scratchpipe as spm
    w = wl.custom(rows=[3000, 5000, 2000], dim=64, batch=64, pooling=[4, 6, 2],
                  slots=[1400, 2000, 900], lookahead=3, steps=30, dist=("zipf", 1.05), seed=73)
    _say("case prefetch depth 3 overlap vs serialised vs staged")
    batches = harness.make_inputs(w)
    results = []
    for flags, ahead, fill in ((0, 0, "mapped"), (spm.SP_FLAG_DEBUG_SYNC, 0, "mapped"),
                               (spm.SP_FLAG_EVENT_WAITS, 2, "mapped"), (0, 2, "staged")):
        host = harness.fresh_host(w, fill)
        st = harness.run_gpu(w, batches, host, flags=flags, prepare_ahead=ahead, prefetch=3,
                             fill=fill)
        assert st["prefetched"] > 0 and st["evictions"] > 0
        results.append([host[t].copy() for t in range(w.tables)])
        host.close()
    for r in results[1:]:
        for x, y in zip(results[0], r):
            assert np.array_equal(x, y)
