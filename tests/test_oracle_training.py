"""Pins for the oracle's uncached trainer (O1): forward pooling, gradient
coalescing and the SGD update, checked against values fixed outside the oracle."""
import json
import os

import numpy as np
import pytest
import torch

from paper_2205_04702_amd import workload as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tables(rng, T, R, D):
    return [rng.standard_normal((R, D)).astype(np.float32) for _ in range(T)]


def test_paper_two_bag_example(oracle):
    """Sec. II-B, Fig. 2: rows {0,4} and {0,2,5}; row 0 receives G[0]+G[1]."""
    g = json.load(open(os.path.join(GOLDEN, "paper_two_bag_example.json")))
    table = np.array(g["table"], np.float32)
    ids = np.array(g["ids"], np.int32)
    off = np.array(g["bag_off"], np.int32)
    out = oracle.forward([table], ids, off, B=2)
    assert np.array_equal(out, np.array(g["expected_out"], np.float32))
    oracle.backward_sgd([table], ids, off, 2, np.array(g["grad"], np.float32), g["lr"])
    assert np.array_equal(table, np.array(g["expected_table"], np.float32))


def _torch_reference(tables, ids, off, B, grad, lr):
    """Library routine: embedding_bag(sum) + autograd + a manual SGD step."""
    T = len(tables)
    outs, new = [], []
    for t in range(T):
        w = torch.tensor(tables[t], dtype=torch.float64, requires_grad=True)
        j0, j1 = int(off[t * B]), int(off[(t + 1) * B])
        idx = torch.tensor(ids[j0:j1], dtype=torch.int64)
        offs = torch.tensor(off[t * B:(t + 1) * B] - j0, dtype=torch.int64)
        o = torch.nn.functional.embedding_bag(idx, w, offs, mode="sum", include_last_offset=False)
        o.backward(torch.tensor(grad[t], dtype=torch.float64))
        outs.append(o.detach().numpy())
        with torch.no_grad():
            new.append((w - float(np.float32(lr)) * w.grad).numpy())
    return np.concatenate(outs), new


@pytest.mark.parametrize("seed", range(6))
def test_against_torch_embedding_bag(oracle, seed):
    rng = np.random.default_rng(seed)
    T, R, D, B = 3, int(rng.integers(5, 40)), int(rng.choice([1, 4, 8, 12])), int(rng.integers(1, 9))
    w = wl.custom(rows=[R] * T, dim=D, batch=B, pooling=3, slots=R, lookahead=0, steps=1,
                  seed=seed)
    ids, off = wl.ragged_batch(w, 0, max_len=6, empty_frac=0.2)
    tables = _tables(rng, T, R, D)
    grad = rng.standard_normal((T, B, D)).astype(np.float32)
    ref_out, ref_tab = _torch_reference(tables, ids, off, B, grad, 0.01)
    out = oracle.forward(tables, ids, off, B)
    # fp64 accumulation rounded once: equal to the fp64 library result rounded to fp32
    assert np.array_equal(out, ref_out.astype(np.float32))
    oracle.backward_sgd(tables, ids, off, B, grad, 0.01)
    for t in range(T):
        np.testing.assert_allclose(tables[t], ref_tab[t], rtol=1e-6, atol=1e-7)


def test_duplicates_inside_a_bag_count_twice(oracle):
    table = np.array([[1.0, 2.0], [3.0, 4.0]], np.float32)
    ids = np.array([1, 1, 0], np.int32)
    off = np.array([0, 3], np.int32)
    out = oracle.forward([table.copy()], ids, off, 1)
    assert np.array_equal(out, [[7.0, 10.0]])
    oracle.backward_sgd([table], ids, off, 1, np.array([[1.0, -1.0]], np.float32), 0.25)
    assert np.array_equal(table, [[0.75, 2.25], [2.5, 4.5]])


def test_empty_bags_give_zero_and_touch_nothing(oracle):
    table = np.arange(8, dtype=np.float32).reshape(4, 2)
    ids = np.array([2], np.int32)
    off = np.array([0, 0, 1, 1], np.int32)  # bags: {}, {2}, {}
    out = oracle.forward([table.copy()], ids, off, 3)
    assert np.array_equal(out, [[0, 0], [4, 5], [0, 0]])
    before = table.copy()
    oracle.backward_sgd([table], ids, off, 3, np.ones((3, 2), np.float32), 1.0)
    assert np.array_equal(table[[0, 1, 3]], before[[0, 1, 3]])
    assert np.array_equal(table[2], before[2] - 1.0)


def test_tables_are_independent(oracle):
    """Training T tables together equals training each alone (per-table reduction)."""
    rng = np.random.default_rng(7)
    w = wl.custom(rows=[30, 50], dim=4, batch=5, pooling=[2, 3], slots=[30, 50], lookahead=0,
                  steps=1)
    ids, off = wl.batch(w, 0)
    tabs = [rng.standard_normal((r, 4)).astype(np.float32) for r in w.rows]
    grad = rng.standard_normal((2, 5, 4)).astype(np.float32)
    joint = [t.copy() for t in tabs]
    out = oracle.train_step(joint, ids, off, 5, grad, 0.1, want_out=True)
    for t in range(2):
        j0, j1 = int(off[t * 5]), int(off[(t + 1) * 5])
        single = [tabs[t].copy()]
        o = oracle.train_step(single, ids[j0:j1], off[t * 5:(t + 1) * 5 + 1] - j0, 5,
                              grad[t:t + 1], 0.1, want_out=True)
        assert np.array_equal(o, out[t * 5:(t + 1) * 5])
        assert np.array_equal(single[0], joint[t])


def test_forward_sees_previous_update(oracle):
    """Two steps on one row: step 2's forward reads the row after step 1's update."""
    table = np.array([[1.0]], np.float32)
    ids, off = np.array([0], np.int32), np.array([0, 1], np.int32)
    o1 = oracle.train_step([table], ids, off, 1, np.array([[2.0]], np.float32), 0.5, True)
    o2 = oracle.train_step([table], ids, off, 1, np.array([[2.0]], np.float32), 0.5, True)
    assert o1[0, 0] == 1.0 and o2[0, 0] == 0.0 and table[0, 0] == -1.0
