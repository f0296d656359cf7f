"""Pins for the oracle's reference planner (O2) and cached simulator (O3).

Nothing here re-implements the planner.  Each plan is checked against
properties that the paper or plain set arithmetic fixes, recomputed from the
state snapshot taken before the plan:
  * dedup equals numpy's unique (library routine);
  * hit <=> the row was cached before the plan (Hit-Map query, Algorithm 1);
  * every row of the planned batch is cached after the plan ("always hits",
    Sec. IV-A);
  * no evicted row belongs to any window batch (hold window, Sec. IV-C);
  * victims are exactly the |M| smallest unheld slots by (last_use, slot), given
    to the misses in that order (LRU ChooseVictim, Sec. VI-E);
  * Hit-Map and slot map stay mutually inverse; untouched slots are unchanged;
  * with slots >= rows nothing is ever evicted and the misses are exactly the
    first touches (closed form);
  * scratchpad training equals uncached training bit for bit (Sec. II-D,
    opening of Sec. VI).
"""
import itertools

import numpy as np
import pytest

from paper_2205_04702_amd import workload as wl


def snapshot(planner):
    return [planner.state(t) for t in range(planner.T)]


def check_plan(planner, pre, post, window, B, p, u, prio=None):
    """Verify plan p (already applied: pre -> post) against the stated properties.

    window holds every batch whose rows are held (the planned one first); prio[t]
    gives each slot's eviction priority before the plan (default: last use, LRU)."""
    ids, off = window[0]
    T = planner.T
    base = planner.slot_base
    u_off = m_off = 0
    for t in range(T):
        kos0, lu0, sor0 = pre[t]
        kos1, lu1, sor1 = post[t]
        S = int(planner.slots[t])
        j0, j1 = int(off[t * B]), int(off[(t + 1) * B])
        rows_b = np.asarray(ids[j0:j1])
        U, inv = np.unique(rows_b, return_inverse=True)
        nU = U.size
        assert np.array_equal(p.u_table[u_off:u_off + nU], np.full(nU, t))
        assert np.array_equal(p.u_row[u_off:u_off + nU], U)
        assert np.array_equal(p.inv[j0:j1], u_off + inv)
        hit = sor0[U] >= 0
        assert np.array_equal(p.hit[u_off:u_off + nU].astype(bool), hit)
        miss = U[~hit]
        k = miss.size
        assert np.array_equal(p.m_table[m_off:m_off + k], np.full(k, t))
        assert np.array_equal(p.m_row[m_off:m_off + k], miss)

        win_rows = set()
        for wi, wo in window:
            win_rows.update(int(r) for r in wi[int(wo[t * B]):int(wo[(t + 1) * B])])
        held = {int(sor0[r]) for r in win_rows if sor0[r] >= 0}
        pr = lu0 if prio is None else prio[t]
        cand = sorted((int(pr[s]), s) for s in range(S) if s not in held)
        victims = [int(v) - int(base[t]) for v in p.v_slot[m_off:m_off + k]]
        assert len(set(victims)) == k
        # exactly the k smallest unheld slots by (priority, slot), in that order
        assert [(int(pr[v]), v) for v in victims] == cand[:k]
        assert np.array_equal(p.v_old_row[m_off:m_off + k], kos0[victims])
        assert np.array_equal(p.v_old_use[m_off:m_off + k], lu0[victims])
        for old in kos0[victims]:
            assert old < 0 or int(old) not in win_rows, "evicted a held row"
        # post-state: placements, evictions, residency, recency
        for i, v in enumerate(victims):
            assert kos1[v] == miss[i] and sor1[miss[i]] == v
            if kos0[v] >= 0:
                assert sor1[kos0[v]] == -1
        local = p.slot_of[j0:j1] - int(base[t])
        assert np.array_equal(kos1[local], rows_b), "a row of the batch is not cached"
        assert np.array_equal(p.slot_u[u_off:u_off + nU] - int(base[t]), sor1[U])
        touched = np.zeros(S, bool)
        touched[sor1[U]] = True
        assert np.all(lu1[touched] == u)
        assert np.array_equal(lu1[~touched], lu0[~touched])
        changed = np.ones(S, bool)
        changed[victims] = False
        assert np.array_equal(kos1[changed], kos0[changed])
        occ = np.nonzero(kos1 >= 0)[0]
        assert np.array_equal(sor1[kos1[occ]], occ)
        assert int((sor1 >= 0).sum()) == occ.size
        u_off += nU
        m_off += k
    assert u_off == p.u_row.size and m_off == p.m_row.size
    assert p.n_evict == int((p.v_old_row >= 0).sum())


def capacity_short(planner, pre, window, B):
    """Independent count: does some table have more misses than unheld slots?"""
    ids, off = window[0]
    for t in range(planner.T):
        kos0, lu0, sor0 = pre[t]
        U = np.unique(ids[int(off[t * B]):int(off[(t + 1) * B])])
        nmiss = int((sor0[U] < 0).sum())
        win_rows = set()
        for wi, wo in window:
            win_rows.update(int(r) for r in wi[int(wo[t * B]):int(wo[(t + 1) * B])])
        held = {int(sor0[r]) for r in win_rows if sor0[r] >= 0}
        if nmiss > int(planner.slots[t]) - len(held):
            return True
    return False


def run_checked(oracle, w, batches, expect_capacity_ok=True):
    planner = oracle.Planner(w.rows, w.slots)
    n = len(batches)
    for u in range(n):
        win = [batches[q] for q in range(u, min(u + w.lookahead, n - 1) + 1)]
        pre = snapshot(planner)
        short = capacity_short(planner, pre, win, w.batch)
        try:
            p = planner.plan(win, w.batch)
        except oracle.PlanError as e:
            assert e.status == oracle.ERR_CAPACITY and short
            post = snapshot(planner)
            for a, b in zip(pre, post):
                for x, y in zip(a, b):
                    assert np.array_equal(x, y), "a failed plan changed state"
            assert planner.step == u
            return False
        assert not short
        check_plan(planner, pre, snapshot(planner), win, w.batch, p, u)
    return True


@pytest.mark.parametrize("case", range(8))
def test_random_runs_hold_every_property(oracle, case):
    rng = np.random.default_rng(100 + case)
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
    assert run_checked(oracle, w, batches)


def test_ragged_and_empty_bags(oracle):
    w = wl.custom(rows=[40, 60], dim=4, batch=6, pooling=2, slots=[40, 60], lookahead=2,
                  steps=12, seed=3)
    batches = [wl.ragged_batch(w, s, max_len=4, empty_frac=0.3) for s in range(w.steps)]
    w2 = wl.custom(rows=[40, 60], dim=4, batch=6, pooling=2, slots=[30, 45], lookahead=2,
                   steps=12, seed=3)
    assert run_checked(oracle, w, batches)
    assert run_checked(oracle, w2, batches)


def degenerate_batches(w):
    """Batches without any ID (alone, and two in a row, so that the planned batch
    and the batch entering the window are empty in turn), a batch with some tables
    without IDs, and a batch of one ID, between ordinary ones."""
    kinds = {3: ((), None), 5: ((1,), None), 7: ((), None), 8: ((), None), 10: (None, 1)}
    return [wl.thinned_batch(w, s, *kinds.get(s, (None, None))) for s in range(w.steps)]


@pytest.mark.parametrize("L", [0, 1, 2])
def test_empty_batches_and_tables(oracle, L):
    """Zero IDs planned, held or entering the window: every property holds, an
    empty batch has no unique keys and no misses, and training through the
    scratchpad equals uncached training bit for bit."""
    w = wl.custom(rows=[50, 70, 40], dim=4, batch=5, pooling=[3, 2, 2], slots=[30, 40, 25],
                  lookahead=L, steps=14, seed=21)
    batches = degenerate_batches(w)
    assert [int(b[0].size) for b in batches][3] == 0 and batches[10][0].size == 1
    assert run_checked(oracle, w, batches)
    planner = oracle.Planner(w.rows, w.slots)
    for u in range(w.steps):
        p = planner.plan(batches[u:u + L + 1], w.batch)
        if batches[u][0].size == 0:
            assert len(p.u_row) == 0 and len(p.m_row) == 0 and p.n_evict == 0
    plain = [wl.init_table(w, t) for t in range(w.tables)]
    host = [t.copy() for t in plain]
    sim = oracle.CachedSimulator(host, w.slots)
    for u in range(w.steps):
        g = wl.grads(w, u)
        o_plain = oracle.train_step(plain, *batches[u], w.batch, g, w.lr, want_out=True)
        _, o_sim = sim.step(batches[u:u + L + 1], w.batch, g, w.lr, want_out=True)
        assert np.array_equal(o_plain, o_sim)
        if batches[u][0].size == 0:
            assert not o_sim.any()
    sim.flush()
    for t in range(w.tables):
        assert np.array_equal(plain[t], host[t])
    assert sim.writebacks > 0


def test_exhaustive_tiny_spaces(oracle):
    """Every sequence of three single-table batches over 3 rows (B=1, bags of 1-2 IDs),
    every slot count and lookahead 0-2: each plan either satisfies every property or
    fails for capacity exactly when the independent count says it must."""
    bags = [(a,) for a in range(3)] + list(itertools.product(range(3), repeat=2))
    runs = failed = 0
    for seq in itertools.product(bags, repeat=3):
        batches = [(np.array(b, np.int32), np.array([0, len(b)], np.int32)) for b in seq]
        for S in (1, 2, 3):
            for L in (0, 1, 2):
                w = wl.custom(rows=[3], dim=1, batch=1, pooling=1, slots=[S], lookahead=L,
                              steps=3)
                ok = run_checked(oracle, w, batches)
                runs += 1
                failed += not ok
    assert runs == 12 ** 3 * 9 and 0 < failed < runs


def test_enough_slots_means_no_eviction_and_compulsory_misses(oracle):
    """slots >= rows: the misses of step u are exactly the rows never seen before."""
    w = wl.custom(rows=[50, 80], dim=2, batch=8, pooling=3, slots=[50, 80], lookahead=2,
                  steps=15, dist=("zipf", 1.0), seed=9)
    planner = oracle.Planner(w.rows, w.slots)
    batches = [wl.batch(w, s) for s in range(w.steps)]
    seen = [set() for _ in range(w.tables)]
    for u in range(w.steps):
        p = planner.plan(batches[u:u + w.lookahead + 1], w.batch)
        ids, off = batches[u]
        expect = []
        for t in range(w.tables):
            rows = set(int(r) for r in ids[off[t * w.batch]:off[(t + 1) * w.batch]])
            expect += [(t, r) for r in sorted(rows - seen[t])]
            seen[t] |= rows
        assert list(zip(p.m_table.tolist(), p.m_row.tolist())) == expect
        assert p.n_evict == 0


def test_capacity_error_changes_nothing_and_exact_fit_succeeds(oracle):
    # one table, 4 slots; batch of 5 distinct rows cannot fit
    planner = oracle.Planner([10], [4])
    ok = (np.array([0, 1, 2, 3], np.int32), np.array([0, 4], np.int32))
    big = (np.array([4, 5, 6, 7, 8], np.int32), np.array([0, 5], np.int32))
    planner.plan([ok], 1)
    pre = snapshot(planner)
    with pytest.raises(oracle.PlanError) as e:
        planner.plan([big], 1)
    assert e.value.status == oracle.ERR_CAPACITY
    assert all(np.array_equal(x, y) for a, b in zip(pre, snapshot(planner)) for x, y in zip(a, b))
    assert planner.step == 1
    # misses == unheld slots exactly: batch {4,5} with window holding rows 0,1 -> 2 candidates
    exact = (np.array([4, 5], np.int32), np.array([0, 2], np.int32))
    hold = (np.array([0, 1], np.int32), np.array([0, 2], np.int32))
    p = planner.plan([exact, hold], 1)
    assert sorted(p.v_old_row.tolist()) == [2, 3]
    # one more miss than unheld slots fails
    pre = snapshot(planner)
    three = (np.array([6, 7, 8], np.int32), np.array([0, 3], np.int32))
    hold2 = (np.array([0, 4], np.int32), np.array([0, 2], np.int32))
    with pytest.raises(oracle.PlanError):
        planner.plan([three, hold2], 1)
    assert planner.step == 2


def test_invalid_ids_are_rejected_without_change(oracle):
    planner = oracle.Planner([10, 10], [5, 5])
    good = (np.array([1, 2, 3], np.int32), np.array([0, 1, 3], np.int32))
    planner.plan([good], 1)
    pre = snapshot(planner)
    for bad in [(np.array([1, 2, 10], np.int32), np.array([0, 1, 3], np.int32)),
                (np.array([1, -1, 3], np.int32), np.array([0, 1, 3], np.int32)),
                (np.array([1, 2, 3], np.int32), np.array([0, 2, 1], np.int32))]:
        with pytest.raises(oracle.PlanError) as e:
            planner.plan([good, bad], 1)
        assert e.value.status == oracle.ERR_INVALID
    assert all(np.array_equal(x, y) for a, b in zip(pre, snapshot(planner)) for x, y in zip(a, b))


@pytest.mark.parametrize("name,slots,L,ragged", [
    ("small-cache", [24, 30], 1, False),
    ("no-lookahead", [16, 20], 0, False),
    ("deep-window", [60, 70], 3, False),
    ("ragged", [40, 50], 2, True),
    ("all-resident", [100, 150], 2, False),
])
def test_cached_training_equals_uncached_bit_for_bit(oracle, name, slots, L, ragged):
    w = wl.custom(rows=[100, 150], dim=6, batch=5, pooling=[2, 3], slots=slots, lookahead=L,
                  steps=30, dist=(("zipf", 1.05), ("uniform",)), seed=11)
    batches = [wl.ragged_batch(w, s, 5) if ragged else wl.batch(w, s) for s in range(w.steps)]
    plain = [wl.init_table(w, t) for t in range(w.tables)]
    host = [t.copy() for t in plain]
    sim = oracle.CachedSimulator(host, w.slots)
    for u in range(w.steps):
        g = wl.grads(w, u)
        o_plain = oracle.train_step(plain, *batches[u], w.batch, g, w.lr, want_out=True)
        _, o_sim = sim.step(batches[u:u + L + 1], w.batch, g, w.lr, want_out=True)
        assert np.array_equal(o_plain, o_sim)
    sim.flush()
    for t in range(w.tables):
        assert np.array_equal(plain[t], host[t])
    if name != "all-resident":
        assert sim.writebacks > 0


def test_worst_case_storage_closed_form():
    """Sec. VI-D: 8 tables x 20 gathers x 2048 x 128 dims x 4 B x 6 batches = 960 MiB."""
    from paper_2205_04702_amd.scratchpipe import worst_case_scratchpad_bytes
    b = worst_case_scratchpad_bytes(tables=8, pooling=20, batch=2048, dim=128, window=6)
    assert b == 8 * 20 * 2048 * 128 * 4 * 6 == 1_006_632_960 == 960 * 2 ** 20
