"""Pin of the past-window hold against the worked fragment of Sec. IV-D.

The paper's figure (missing from the text) follows IDs through the Hit-Map and
the hold mask; the text states the outcome: the first mini-batch uses IDs 7089
and 2021; the second mini-batch's IDs 3010 and 7089 are a miss and a hit when
the Hit-Map is queried in the second cycle; and E[2021], whose hold mask has
aged to zero after the fourth cycle (a mask of three past batches, Algorithm 1),
is the victim chosen in the fifth cycle.  In this repository's reading the past
window is hold_past = 3 batches before the planned one, with no look-forward
(lookahead 0) and a Storage of three slots, so that a fifth-cycle miss has
exactly one unheld slot to take.  The slot positions in the figure are not
recoverable; the trace below pins the hits, the misses and which row is evicted
when, which is what the text fixes."""
import numpy as np
import pytest

from paper_2205_04702_amd import workload as wl


def one_bag(*ids):
    return np.array(ids, np.int32), np.array([0, len(ids)], np.int32)


CYCLES = [one_bag(7089, 2021), one_bag(3010, 7089), one_bag(7089), one_bag(3010), one_bag(4444)]


def plan_all(oracle, batches, past):
    planner = oracle.Planner([10_000], [3])
    out = []
    for u, b in enumerate(batches):
        out.append(planner.plan([b], 1, past=batches[max(0, u - past):u]))
    return out


def test_second_batch_sees_a_miss_and_a_hit(oracle):
    p = plan_all(oracle, CYCLES[:2], past=3)
    assert p[0].u_row.tolist() == [2021, 7089] and not p[0].hit.any()
    assert p[1].u_row.tolist() == [3010, 7089]
    assert p[1].hit.tolist() == [0, 1]               # 3010 misses, 7089 hits (cycle 2)
    assert p[1].m_row.tolist() == [3010]


def test_2021_is_evicted_in_the_fifth_cycle(oracle):
    p = plan_all(oracle, CYCLES, past=3)
    for u in range(4):
        assert p[u].n_evict == 0                     # nothing leaves before the fifth cycle
    assert p[4].m_row.tolist() == [4444]
    assert p[4].v_old_row.tolist() == [2021]         # E[2021] is the victim (cycle 5)
    assert p[4].n_evict == 1


def test_with_a_fourth_cycle_miss_2021_is_still_held(oracle):
    """A miss in the fourth cycle finds every slot held (2021's mask has not aged to
    zero yet: batch 1 is among the three past batches), so the plan fails for
    capacity; with a past window of two batches the same miss evicts 2021."""
    batches = CYCLES[:3] + [one_bag(4444)]
    planner = oracle.Planner([10_000], [3])
    for u in range(3):
        planner.plan([batches[u]], 1, past=batches[max(0, u - 3):u])
    with pytest.raises(oracle.PlanError) as e:
        planner.plan([batches[3]], 1, past=batches[0:3])
    assert e.value.status == oracle.ERR_CAPACITY
    p = plan_all(oracle, batches, past=2)
    assert p[3].v_old_row.tolist() == [2021]


def test_cached_training_on_the_fragment_equals_uncached(oracle):
    w = wl.custom(rows=[10_000], dim=4, batch=1, pooling=2, slots=[3], lookahead=0, steps=5,
                  seed=3)
    plain = [wl.init_table(w, 0)]
    host = [plain[0].copy()]
    sim = oracle.CachedSimulator(host, [3])
    for u, b in enumerate(CYCLES):
        g = wl.grads(w, u)
        o1 = oracle.train_step(plain, *b, 1, g, 0.05, want_out=True)
        _, o2 = sim.step([b], 1, g, 0.05, want_out=True, past=CYCLES[max(0, u - 3):u])
        assert np.array_equal(o1, o2)
    sim.flush()
    assert np.array_equal(plain[0], host[0])
