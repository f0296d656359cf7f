"""Pins for the oracle planner's other replacement policies and its past window.

LRU is the default replacement policy and random eviction and LFU are the
alternatives the evaluation names (Sec. VI-E); Algorithm 1 keeps rows of the
batches still in flight from being evicted (the past window, Sec. IV-C and
IV-D).  Nothing here re-implements the planner.  Each plan is checked against
what the definitions fix, recomputed outside it:
  * the random policy's generator reproduces SplitMix64's published outputs,
    and the slots it evicts are spread uniformly over the candidates
    (chi-square);
  * LFU evicts the unheld slots with the fewest uses, where a slot's uses are
    counted here from the batch history: the plans since its row was placed
    whose batch contains that row;
  * a trace worked out by hand where LRU and LFU choose differently;
  * with a past window no evicted row belongs to a past batch, and the
    capacity check counts the past holds;
  * every other plan property of the LRU pins (dedup, hits, residency, the
    Hit-Map update) holds under each policy;
  * scratchpad training under every policy and past window equals uncached
    training bit for bit (Sec. II-D: caching does not change the result).
"""
import itertools
import json
import os

import numpy as np
import pytest

from paper_2205_04702_amd import workload as wl
from tests.test_oracle_planner import capacity_short, check_plan, snapshot

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _one(rows):
    """A single-table, single-bag batch holding `rows`."""
    return (np.array(rows, np.int32), np.array([0, len(rows)], np.int32))


class UseCounter:
    """Uses of every slot counted from the plan history, not from planner state."""

    def __init__(self, planner):
        self.planner = planner
        self.placed = [dict() for _ in range(planner.T)]  # slot -> (row, plan that placed it)
        self.rows_of = []                                   # plan -> [set of rows per table]

    def counts(self, t, u):
        S = int(self.planner.slots[t])
        c = np.zeros(S, np.int64)
        for s, (row, f) in self.placed[t].items():
            c[s] = sum(row in self.rows_of[q][t] for q in range(f, u))
        return c

    def record(self, p, batch, B):
        ids, off = batch
        self.rows_of.append([set(int(r) for r in ids[int(off[t * B]):int(off[(t + 1) * B])])
                             for t in range(self.planner.T)])
        u = len(self.rows_of) - 1
        base = self.planner.slot_base
        for i in range(p.m_row.size):
            t = int(p.m_table[i])
            self.placed[t][int(p.v_slot[i]) - int(base[t])] = (int(p.m_row[i]), u)


def priorities(oracle, planner, pre, uses, u):
    """Each table's slot priorities before plan u under the planner's policy."""
    if planner.policy == "lru":
        return None
    if planner.policy == "lfu":
        return [uses.counts(t, u) for t in range(planner.T)]
    base = planner.slot_base
    return [np.array([oracle.random_priority(planner.seed, u, int(base[t]) + s, int(pre[t][1][s]))
                      for s in range(int(planner.slots[t]))], np.int64)
            for t in range(planner.T)]


def run_policy(oracle, w, batches, policy, past=0, seed=0):
    """Plan every batch, checking each plan; returns False at the first capacity failure."""
    planner = oracle.Planner(w.rows, w.slots, policy, seed)
    uses = UseCounter(planner)
    n = len(batches)
    for u in range(n):
        win = [batches[q] for q in range(u, min(u + w.lookahead, n - 1) + 1)]
        back = [batches[q] for q in range(max(0, u - past), u)]
        pre = snapshot(planner)
        short = capacity_short(planner, pre, win + back, w.batch)
        prio = priorities(oracle, planner, pre, uses, u)
        try:
            p = planner.plan(win, w.batch, past=back)
        except oracle.PlanError as e:
            assert e.status == oracle.ERR_CAPACITY and short
            assert planner.step == u
            for a, b in zip(pre, snapshot(planner)):
                for x, y in zip(a, b):
                    assert np.array_equal(x, y), "a failed plan changed state"
            return False
        assert not short
        check_plan(planner, pre, snapshot(planner), win + back, w.batch, p, u, prio)
        uses.record(p, batches[u], w.batch)
        if policy == "lfu":  # the planner's own counts agree with the history
            for t in range(w.tables):
                assert np.array_equal(planner.uses(t), uses.counts(t, u + 1))
    return True


# ------------------------------------------------------------------- generator

def test_splitmix64_reproduces_published_outputs(oracle):
    g = json.load(open(os.path.join(GOLDEN, "splitmix64_seed0.json")))
    got = [oracle.splitmix64_nth(g["seed"], n) for n in range(1, len(g["outputs_hex"]) + 1)]
    assert got == [int(h, 16) for h in g["outputs_hex"]]
    assert got[0] - (1 << 64) == g["java_splittable_random_0_next_long"]


def test_random_priority_range_and_freshness(oracle):
    assert oracle.random_priority(0, 5, 7, -1) == 0  # a never-used slot goes first
    vals = [oracle.random_priority(3, u, g, 0) for u in range(4) for g in range(2000)]
    assert min(vals) >= 1 and max(vals) <= 1 << 24
    a = [oracle.random_priority(3, 0, g, 0) for g in range(2000)]
    b = [oracle.random_priority(3, 1, g, 0) for g in range(2000)]
    c = [oracle.random_priority(4, 0, g, 0) for g in range(2000)]
    assert a != b and a != c  # fresh per plan and per seed
    # the draw does not depend on the slot's last use once it is occupied
    assert oracle.random_priority(3, 2, 11, 0) == oracle.random_priority(3, 2, 11, 1)
    # 24-bit draws: top and bottom halves equally likely
    top = sum(v - 1 >= 1 << 23 for v in vals)
    assert abs(top - len(vals) / 2) < 4 * np.sqrt(len(vals) / 4)


def test_random_eviction_is_uniform_over_candidates(oracle):
    """20 occupied, unheld slots and one miss per plan: each slot is evicted about equally."""
    S, n = 20, 4000
    planner = oracle.Planner([n + S], [S], "random", seed=1)
    hits = np.zeros(S, np.int64)
    for u in range(n):
        p = planner.plan([_one([u])], 1)
        if u >= S:
            assert p.n_evict == 1
            hits[int(p.v_slot[0])] += 1
        else:
            assert int(p.v_slot[0]) == u and p.n_evict == 0  # free slots first, in order
    exp = hits.sum() / S
    chi2 = float(((hits - exp) ** 2 / exp).sum())
    assert chi2 < 60.0, (chi2, hits)  # 19 degrees of freedom; 60 is p < 1e-5
    # LRU on the same trace cycles through the slots in order
    lru = oracle.Planner([n + S], [S], "lru")
    order = [int(lru.plan([_one([u])], 1).v_slot[0]) for u in range(3 * S)]
    assert order == list(range(S)) * 3


def test_random_policy_depends_on_the_seed(oracle):
    w = wl.custom(rows=[200], dim=2, batch=4, pooling=2, slots=[20], lookahead=1, steps=30,
                  seed=5)
    batches = [wl.batch(w, s) for s in range(w.steps)]
    runs = []
    for seed in (0, 0, 1):
        planner = oracle.Planner(w.rows, w.slots, "random", seed)
        runs.append([planner.plan(batches[u:u + 2], w.batch).v_slot.tolist() for u in range(29)])
    assert runs[0] == runs[1] and runs[0] != runs[2]


# ------------------------------------------------------------------------- LFU

def test_lfu_hand_trace(oracle):
    """Three slots, no look-forward.  Plans: {0,1,2} {0,1} {0,1} {2} {3} {4}.
    Before plan 4, slots 0/1/2 hold rows 0/1/2 with uses 3/3/2 and last uses 2/2/3.
    LFU evicts row 2 (fewest uses); LRU evicts row 0 (oldest, slot 0 before slot 1).
    Before plan 5, row 3 in slot 2 has one use: LFU evicts it; LRU evicts row 1."""
    trace = [[0, 1, 2], [0, 1], [0, 1], [2], [3], [4]]
    lfu, lru = oracle.Planner([10], [3], "lfu"), oracle.Planner([10], [3], "lru")
    a = [lfu.plan([_one(b)], 1) for b in trace]
    b = [lru.plan([_one(b)], 1) for b in trace]
    assert [p.v_slot.tolist() for p in a[:3]] == [[0, 1, 2], [], []]
    assert a[4].v_old_row.tolist() == [2] and a[4].v_slot.tolist() == [2]
    assert a[5].v_old_row.tolist() == [3] and a[5].v_slot.tolist() == [2]
    assert b[4].v_old_row.tolist() == [0] and b[5].v_old_row.tolist() == [1]
    assert lfu.uses(0).tolist() == [3, 3, 1]


@pytest.mark.parametrize("policy", ["lfu", "random"])
@pytest.mark.parametrize("case", range(6))
def test_random_runs_hold_every_property(oracle, policy, case):
    rng = np.random.default_rng(300 + case)
    T = int(rng.integers(1, 4))
    rows = [int(rng.integers(20, 120)) for _ in range(T)]
    L = int(rng.integers(0, 4))
    B = int(rng.integers(2, 7))
    P = [int(rng.integers(1, 4)) for _ in range(T)]
    slots = [min(r, (L + 1) * B * p + int(rng.integers(0, 20))) for r, p in zip(rows, P)]
    dist = tuple(("zipf", 1.1) if rng.random() < 0.5 else ("uniform",) for _ in range(T))
    w = wl.custom(rows=rows, dim=4, batch=B, pooling=P, slots=slots, lookahead=L, steps=25,
                  dist=dist, seed=case)
    batches = [wl.batch(w, s) for s in range(w.steps)]
    assert run_policy(oracle, w, batches, policy, seed=case)


@pytest.mark.parametrize("policy", ["lru", "lfu", "random"])
def test_exhaustive_tiny_spaces(oracle, policy):
    """Every sequence of three single-table batches over 3 rows (bags of 1-2 IDs), every
    slot count, with and without look-forward and past window (LRU without a past window
    is covered by the LRU pins): each plan satisfies every property or fails for capacity
    exactly when the independent count says it must."""
    bags = [(a,) for a in range(3)] + list(itertools.product(range(3), repeat=2))
    combos = ((0, 1), (1, 1)) if policy == "lru" else ((0, 0), (1, 1))
    runs = failed = 0
    for seq in itertools.product(bags, repeat=3):
        batches = [_one(list(b)) for b in seq]
        for S in (1, 2, 3):
            for L, past in combos:
                w = wl.custom(rows=[3], dim=1, batch=1, pooling=1, slots=[S], lookahead=L,
                              steps=3)
                failed += not run_policy(oracle, w, batches, policy, past=past, seed=7)
                runs += 1
    assert runs == 12 ** 3 * 6 and 0 < failed < runs


# ------------------------------------------------------------------ past window

def test_past_window_hand_trace(oracle):
    """Two slots: plan 0 caches rows 0 and 1; plan 1 misses row 2.  Without a past window
    LRU evicts row 0 (slot 0); holding batch 0 leaves no candidate, a capacity failure."""
    b0, b1 = _one([0, 1]), _one([2])
    p = oracle.Planner([5], [2])
    p.plan([b0], 1)
    assert p.plan([b1], 1).v_old_row.tolist() == [0]
    q = oracle.Planner([5], [2])
    q.plan([b0], 1)
    with pytest.raises(oracle.PlanError) as e:
        q.plan([b1], 1, past=[b0])
    assert e.value.status == oracle.ERR_CAPACITY and q.step == 1
    # three slots: the free one is used and rows 0 and 1 stay
    r = oracle.Planner([5], [3])
    r.plan([b0], 1)
    assert r.plan([b1], 1, past=[b0]).v_slot.tolist() == [2]


@pytest.mark.parametrize("policy", ["lru", "lfu", "random"])
@pytest.mark.parametrize("past", [1, 3])
def test_past_window_runs_hold_every_property(oracle, policy, past):
    w = wl.custom(rows=[80, 120], dim=4, batch=5, pooling=[2, 3], slots=[45, 70], lookahead=2,
                  steps=30, dist=(("zipf", 1.05), ("uniform",)), seed=21)
    batches = [wl.batch(w, s) for s in range(w.steps)]
    assert run_policy(oracle, w, batches, policy, past=past, seed=3)


# ---------------------------------------------------------------- training result

@pytest.mark.parametrize("policy,past", [("lfu", 0), ("random", 0), ("lru", 2), ("lfu", 1),
                                         ("random", 3)])
def test_cached_training_equals_uncached_bit_for_bit(oracle, policy, past):
    w = wl.custom(rows=[100, 150], dim=6, batch=5, pooling=[2, 3], slots=[40, 60], lookahead=1,
                  steps=30, dist=(("zipf", 1.05), ("uniform",)), seed=11)
    batches = [wl.ragged_batch(w, s, 5) for s in range(w.steps)]
    plain = [wl.init_table(w, t) for t in range(w.tables)]
    host = [t.copy() for t in plain]
    sim = oracle.CachedSimulator(host, w.slots, policy=policy, seed=9)
    for u in range(w.steps):
        g = wl.grads(w, u)
        o_plain = oracle.train_step(plain, *batches[u], w.batch, g, w.lr, want_out=True)
        _, o_sim = sim.step(batches[u:u + 2], w.batch, g, w.lr, want_out=True,
                            past=batches[max(0, u - past):u])
        assert np.array_equal(o_plain, o_sim)
    sim.flush()
    for t in range(w.tables):
        assert np.array_equal(plain[t], host[t])
    assert sim.writebacks > 0
