"""The seeded input generator: determinism, shapes and distributions."""
import numpy as np

from paper_2205_04702_amd import workload as wl


def test_batches_are_deterministic_and_independent_of_order():
    w = wl.get_workload("tiny")
    a = wl.batch(w, 7)
    _ = wl.batch(w, 3)
    b = wl.batch(w, 7)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert not np.array_equal(wl.batch(w, 8)[0], a[0])
    assert np.array_equal(wl.grads(w, 2), wl.grads(w, 2))


def test_shapes_ranges_and_csr():
    w = wl.get_workload("tiny")
    ids, off = wl.batch(w, 0)
    assert ids.dtype == np.int32 and off.dtype == np.int32
    assert ids.size == w.nnz == w.batch * sum(w.pooling)
    assert off.size == w.tables * w.batch + 1 and off[0] == 0 and off[-1] == ids.size
    for t in range(w.tables):
        seg = ids[off[t * w.batch]:off[(t + 1) * w.batch]]
        assert seg.min() >= 0 and seg.max() < w.rows[t]
    g = wl.grads(w, 0)
    assert g.shape == (w.tables, w.batch, w.dim) and g.dtype == np.float32
    tab = wl.init_table(w, 0)
    assert tab.dtype == np.float32 and tab.min() >= -0.05 and tab.max() < 0.05


def test_zipf_rank_frequencies():
    """Rank-1 frequency of Zipf(alpha) over R rows is 1/H(R, alpha)."""
    w = wl.custom(rows=[1000], dim=4, batch=1, pooling=200_000, slots=[1000], lookahead=0,
                  steps=1, dist=("zipf", 1.05), seed=4)
    ids = wl.table_ids(w, 0, 0)
    counts = np.bincount(ids, minlength=1000)
    h = (np.arange(1, 1001, dtype=np.float64) ** -1.05).sum()
    top = np.sort(counts)[::-1]
    assert abs(top[0] / ids.size - 1 / h) < 0.01
    assert abs(top[1] / ids.size - 2 ** -1.05 / h) < 0.01
    # the hottest row is the permutation's first entry, not row 0
    assert np.argmax(counts) == wl._row_permutation(4, 0, 1000)[0]


def test_ragged_batches_have_empty_bags():
    w = wl.custom(rows=[50, 60], dim=4, batch=40, pooling=3, slots=[50, 60], lookahead=1, steps=2)
    ids, off = wl.ragged_batch(w, 0, max_len=5, empty_frac=0.25)
    lens = np.diff(off)
    assert (lens == 0).any() and lens.max() <= 5 and off[-1] == ids.size


def test_named_workload_sizes():
    c2 = wl.get_workload("zipf-8x1M")
    assert (c2.tables, c2.rows[0], c2.dim, c2.batch, c2.pooling[0]) == (8, 1_000_000, 64, 1024, 8)
    assert c2.slots[0] == 100_000 and c2.lookahead == 3 and c2.steps == 200
    c3 = wl.get_workload("zipf-26x4M")
    assert c3.slots[0] == 200_000 and c3.grad_sigma == 0.1
    mx = wl.get_workload("mixed")
    assert mx.tables == 64 and all(1 <= p <= 80 for p in mx.pooling)
    assert all(1000 <= r <= 2e7 for r in mx.rows) and all(s <= r for s, r in zip(mx.slots, mx.rows))
    assert sum(mx.slots) * 64 * 4 <= 40e9


def test_thinned_batch_keeps_a_prefix_of_each_bag_of_the_kept_tables():
    w = wl.get_workload("tiny")
    B = w.batch
    full_ids, full_off = wl.batch(w, 4)
    for tables, max_ids in [((), None), ((1, 3), None), (None, 1), ((0, 2), 300), (None, None)]:
        ids, off = wl.thinned_batch(w, 4, tables, max_ids)
        assert ids.dtype == np.int32 and off.dtype == np.int32
        assert off.size == w.tables * B + 1 and off[0] == 0 and off[-1] == ids.size
        assert np.all(np.diff(off) >= 0)
        kept = 0
        for g in range(w.tables * B):
            t = g // B
            full = full_ids[full_off[g]:full_off[g + 1]]
            got = ids[off[g]:off[g + 1]]
            if tables is not None and t not in tables:
                assert got.size == 0
            else:
                assert np.array_equal(got, full[:got.size])
                room = full.size if max_ids is None else min(full.size, max(max_ids - kept, 0))
                assert got.size == room
            kept += got.size
        if max_ids is not None:
            assert ids.size == min(max_ids, sum(
                int(full_off[(t + 1) * B] - full_off[t * B]) for t in range(w.tables)
                if tables is None or t in tables))
    ids, off = wl.thinned_batch(w, 4)
    assert np.array_equal(ids, full_ids) and np.array_equal(off, full_off)
