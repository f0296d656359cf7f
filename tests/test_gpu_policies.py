"""Parity of the HIP planner's LFU and random replacement policies and of its past
window (needs an MI355X).

LRU is the default policy and LFU and random eviction the alternatives named
in the sensitivity study (Sec. VI-E); the past window holds the rows of batches
planned before the current one (Sec. IV-C).  Plans must match the oracle
planner, run with the same policy, seed and past window, bit for bit; outputs
and tables within 1e-5 per row as in the LRU parity tests.
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


@pytest.mark.parametrize("policy", ["lfu", "random"])
def test_tiny_all_steps(harness, policy):
    """4 x 20k x 32, B=128, 4 IDs per bag, 2048 slots, lookahead 2, 50 steps."""
    w = wl.get_workload("tiny")
    _say(f"case tiny policy {policy}")
    r = harness.run_parity(w, policy=policy, seed=5)
    assert r["stats"]["evictions"] > 0


@pytest.mark.parametrize("policy", ["lru", "lfu", "random"])
@pytest.mark.parametrize("past", [1, 3])
def test_past_window(harness, policy, past):
    """Three Zipf tables of 50k rows, 4096 slots, lookahead 2, the two batches after the
    window handed over early from device memory (the ring then also keeps the past)."""
    w = wl.custom(rows=[50_000] * 3, dim=32, batch=128, pooling=4, slots=[4096] * 3,
                  lookahead=2, steps=40, dist=("zipf", 1.05), seed=4)
    _say(f"case past window {past} policy {policy}")
    r = harness.run_parity(w, policy=policy, hold_past=past, seed=2, prepare_ahead=2,
                           device_ids=True)
    assert r["stats"]["evictions"] > 0


@pytest.mark.parametrize("policy", ["lru", "lfu", "random"])
def test_large_victim_sets(harness, policy):
    """Over 2048 victims per table per plan: the victims are ordered by one global radix
    sort on (table, priority) instead of per table in LDS."""
    w = wl.custom(rows=[1_000_000] * 2, dim=16, batch=1024, pooling=4, slots=[20_000] * 2,
                  lookahead=1, steps=12, dist=("uniform",), seed=8)
    _say(f"case large victim sets policy {policy}")
    r = harness.run_parity(w, policy=policy, seed=3, sync_each_step=False)
    st = r["stats"]
    assert st["evictions"] > 4 * 2 * 2048


@pytest.mark.parametrize("policy", ["lfu", "random"])
def test_zipf_8x1M_sampled(harness, policy):
    """The benchmark workload (8 x 1M x 64, B=1024, 8 IDs per bag, 100k slots, lookahead 3)
    under the other policies, driven as the benchmark drives it, for 40 steps."""
    w = wl.get_workload("zipf-8x1M")
    _say(f"case zipf-8x1M policy {policy}")
    sample = [0, 1, 2, 13, 25, 38, 39]
    r = harness.run_sampled_parity(w, 40, check_plan_steps=sample, check_fwd_steps=sample,
                                   say=_say, policy=policy, seed=1)
    _say(f"zipf-8x1M {policy}: worst fwd {r['worst_fwd']:.2e} table {r['worst_table']:.2e} "
         f"misses {r['stats']['misses']} evictions {r['stats']['evictions']}")


def test_hold_mask_fragment_of_the_paper(harness):
    """The worked fragment of Sec. IV-D through the C ABI with a past window of three
    batches: 3010 misses and 7089 hits in the second cycle, nothing is evicted before
    the fifth cycle, whose miss evicts 2021; plans bit-exact against the oracle."""
    import numpy as np
    from tests.test_oracle_holdmask import CYCLES
    w = wl.custom(rows=[10_000], dim=8, batch=1, pooling=2, slots=[3], lookahead=0, steps=5,
                  seed=3)
    _say("case hold-mask fragment, past window 3")
    r = harness.run_parity(w, list(CYCLES), hold_past=3, max_table_ids=0)
    assert r["stats"]["evictions"] == 1 and r["stats"]["misses"] == 4


def test_hold_mask_fragment_fourth_cycle_miss_is_a_capacity_error(harness):
    import torch
    from paper_2205_04702_amd import scratchpipe as spm
    from tests.test_oracle_holdmask import CYCLES, one_bag
    w = wl.custom(rows=[10_000], dim=8, batch=1, pooling=2, slots=[3], lookahead=0, steps=5,
                  seed=3)
    _say("case hold-mask fragment, fourth-cycle miss")
    host = harness.fresh_host(w)
    ctx = spm.ScratchPipe(w.rows, w.dim, w.slots, 0, host, max_batch=1, max_ids=4, hold_past=3)
    out = torch.zeros((1, w.dim), device="cuda:0")
    try:
        for b in CYCLES[:3]:
            t = ctx.plan([b])
            ctx.forward(t, out)
            ctx.backward_update(t, torch.zeros((1, w.dim), device="cuda:0"), 0.01)
        with pytest.raises(spm.SPError) as e:
            ctx.plan([one_bag(4444)])
        assert e.value.status == spm.SP_ERR_CAPACITY
    finally:
        ctx.close()
        host.close()
