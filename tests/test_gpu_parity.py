"""Parity of the HIP scratchpad against the CPU oracle (needs an MI355X).

Plans (dedup, hits, misses, victims, slot maps) must match the oracle bit for
bit; pooled outputs and final tables must match per row within 1e-5 relative
(max-norm), and rows never gathered must be bit-identical.
"""
import numpy as np
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


@pytest.mark.parametrize("bound", ["auto", 0])
def test_tiny_all_steps(harness, bound):
    """4 x 20k x 32, B=128, 4 IDs per bag, 2048 slots, lookahead 2, 50 steps; tables
    sorted in LDS (bound: the batches' own) and by the general multi-launch path (0)."""
    w = wl.get_workload("tiny")
    _say(f"case tiny {w.describe()} bound {bound}")
    r = harness.run_parity(w, max_table_ids=bound)
    st = r["stats"]
    assert st["plans"] == 50 and st["misses"] > 0 and st["evictions"] > 0
    # the Hit-Map (16384 entries for 8192 slots) passes 70% use within a few steps
    # of about 2000 misses each, so plans are checked across its rebuilds
    assert st["hash_rebuilds"] > 0
    _say(f"tiny worst fwd {r['worst_fwd']:.2e} table {r['worst_table']:.2e} stats {st}")


@pytest.mark.parametrize("dim", [4, 8, 16, 64, 128, 256])
def test_every_row_width(harness, dim):
    w = wl.custom(rows=[3000, 5000], dim=dim, batch=40, pooling=[3, 5], slots=[600, 900],
                  lookahead=2, steps=20, dist=(("zipf", 1.05), ("uniform",)), seed=dim)
    _say(f"case dim={dim}")
    harness.run_parity(w)


def test_ragged_bags_with_empty_bags(harness):
    w = wl.custom(rows=[4000, 2500, 6000], dim=32, batch=64, pooling=4, slots=[1500, 1200, 1800],
                  lookahead=3, steps=25, dist=("zipf", 1.1), seed=5)
    batches = harness.make_inputs(w, ragged=9)
    _say("case ragged")
    harness.run_parity(w, batches)


def test_long_zipf_runs_split_into_chunks(harness):
    """A few very hot rows: runs much longer than one backward chunk."""
    w = wl.custom(rows=[500], dim=64, batch=512, pooling=16, slots=[400], lookahead=1, steps=12,
                  dist=("zipf", 1.6), seed=2)
    _say("case hot rows")
    harness.run_parity(w)


def test_no_lookahead(harness):
    w = wl.custom(rows=[2000, 3000], dim=32, batch=32, pooling=4, slots=[200, 300], lookahead=0,
                  steps=25, dist=("zipf", 0.9), seed=8)
    _say("case lookahead 0")
    harness.run_parity(w)


def test_all_resident(harness):
    w = wl.custom(rows=[1000, 1500], dim=32, batch=32, pooling=4, slots=[1000, 1500], lookahead=2,
                  steps=20, seed=9)
    _say("case all resident")
    r = harness.run_parity(w)
    assert r["stats"]["evictions"] == 0


def test_single_table_single_slot_pressure(harness):
    """Capacity exactly tight: every batch of one ID per bag, one bag, one slot."""
    w = wl.custom(rows=[7], dim=8, batch=1, pooling=1, slots=[1], lookahead=0, steps=30, seed=4)
    _say("case one slot")
    harness.run_parity(w)


@pytest.mark.parametrize("device_ids,ahead", [(False, 1), (True, 1), (True, 2)])
def test_prepared_ahead_batch_changes_nothing(harness, device_ids, ahead):
    """Passing the batches after the window (prepared early, not held) gives the
    same plans and tables as the plain window."""
    w = wl.custom(rows=[2500, 4000], dim=64, batch=40, pooling=[4, 2], slots=[500, 600],
                  lookahead=2, steps=20, dist=("zipf", 1.0), seed=21)
    _say(f"case prepared-ahead device_ids={device_ids} ahead={ahead}")
    a = harness.run_parity(w, return_tables=True)
    b = harness.run_parity(w, prepare_ahead=ahead, device_ids=device_ids, return_tables=True)
    for x, y in zip(a["tables"], b["tables"]):
        assert np.array_equal(x, y)


def test_device_resident_ids_match_host_ids(harness):
    w = wl.custom(rows=[3000, 3000], dim=32, batch=48, pooling=3, slots=[700, 700], lookahead=2,
                  steps=15, dist=("zipf", 1.0), seed=12)
    _say("case device ids")
    a = harness.run_parity(w, return_tables=True)
    b = harness.run_parity(w, device_ids=True, return_tables=True)
    for x, y in zip(a["tables"], b["tables"]):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("shape", ["ragged", "8192-ids", "8192-bags", "skewed-rows"])
def test_ingest_in_lds_matches_general_path(harness, shape):
    """Batches whose tables fit one workgroup are sorted and deduplicated in LDS, one
    launch per batch, several workgroups per table, each over a range of the table's
    rows; the general path uses several launches over the whole batch.  Both must give
    the oracle's plans, and bit-identical tables.  Edge cases: ragged and empty bags,
    tables at the 8192-ID limit with hot runs split into chunks, 8192 bags, and every
    ID of a table in its first row range (one workgroup holds all 8192) beside a table
    with fewer rows than there are ranges."""
    if shape == "skewed-rows":
        w = wl.custom(rows=[200_000, 5, 50_000], dim=16, batch=1024, pooling=8,
                      slots=[20_000, 5, 5_000], lookahead=1, steps=6, dist=("zipf", 1.1),
                      seed=20)
        batches = []
        for ids, off in harness.make_inputs(w):
            ids = ids.copy()
            ids[:1024 * 8] %= 9000  # table 0: rows below 9000 only
            batches.append((ids, off))
    elif shape == "ragged":
        w = wl.custom(rows=[900, 1400, 700], dim=16, batch=64, pooling=3, slots=[600, 800, 500],
                      lookahead=2, steps=14, seed=17)
        batches = [wl.ragged_batch(w, s, 7, empty_frac=0.25) for s in range(w.steps)]
    elif shape == "8192-ids":
        w = wl.custom(rows=[200_000] * 2, dim=16, batch=1024, pooling=8, slots=[20_000] * 2,
                      lookahead=1, steps=6, dist=("zipf", 1.1), seed=18)
        batches = harness.make_inputs(w)
    else:
        w = wl.custom(rows=[100_000] * 2, dim=8, batch=8192, pooling=1, slots=[20_000] * 2,
                      lookahead=1, steps=6, dist=("zipf", 1.05), seed=19)
        batches = harness.make_inputs(w)
    _say(f"case ingest paths {shape} bound {harness.table_bound(w, batches)}")
    assert harness.table_bound(w, batches) <= 8192
    a = harness.run_parity(w, batches, return_tables=True)
    b = harness.run_parity(w, batches, return_tables=True, max_table_ids=0)
    for x, y in zip(a["tables"], b["tables"]):
        assert np.array_equal(x, y)


def test_zipf_8x1M_full_size(harness):
    """The benchmark workload at full size: 8 x 1M x 64, B=1024, 8 IDs per bag,
    100k slots per table, lookahead 3, 200 steps.  Plans checked at sampled
    steps, forward outputs at sampled steps, all final tables in full."""
    w = wl.get_workload("zipf-8x1M")
    _say(f"case zipf-8x1M {w.describe()}")
    sample = [0, 1, 2, 3, 50, 101, 150, 198, 199]
    # as the benchmark drives it: IDs in device memory, the two batches after
    # the window handed over early (read after sp_plan returns); the IDs of
    # held batches are overwritten once their plan has returned
    r = harness.run_parity(w, check_plan_steps=sample, check_fwd_steps=sample,
                           sync_each_step=False, prepare_ahead=2, device_ids=True,
                           overwrite_held_ids=True)
    st = r["stats"]
    assert st["plans"] == 200 and st["evictions"] > 0
    _say(f"zipf-8x1M worst fwd {r['worst_fwd']:.2e} table {r['worst_table']:.2e} "
         f"misses {st['misses']} evictions {st['evictions']} rebuilds {st['hash_rebuilds']}")
