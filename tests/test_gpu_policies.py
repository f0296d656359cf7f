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
