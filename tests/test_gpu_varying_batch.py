"""Batch sizes that differ within one window (a short last batch of an epoch, a
batch of one sample, a batch of none) on the GPU (needs an MI355X)."""
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


def _shrink(w, ids, off, b):
    """The first b bags of every table of a batch of w.batch bags, as a batch of b
    bags (for the GPU) and as a batch of w.batch bags whose later bags are empty
    (for the oracle, whose planner takes one batch size per window: the keys and
    their positions are the same, so the plans are)."""
    T, B = w.tables, w.batch
    lens = np.diff(off.astype(np.int64)).reshape(T, B).copy()
    lens[:, b:] = 0
    keep = np.zeros(ids.size, dtype=bool)
    for g in np.nonzero(lens.reshape(-1))[0]:
        keep[int(off[g]):int(off[g + 1])] = True
    kept = ids[keep].astype(np.int32)
    pad_off = np.zeros(T * B + 1, np.int64)
    np.cumsum(lens.reshape(-1), out=pad_off[1:])
    small_off = np.zeros(T * b + 1, np.int64)
    np.cumsum(lens[:, :b].reshape(-1), out=small_off[1:])
    return (kept, small_off.astype(np.int32)), (kept, pad_off.astype(np.int32))


@pytest.mark.parametrize("device_ids,bound", [(False, "auto"), (True, 0)],
                         ids=["host-ids-lds-ingest", "device-ids-general-ingest"])
def test_batch_sizes_vary_within_the_window(harness, device_ids, bound):
    import torch
    from oracle import oracle
    from paper_2205_04702_amd.scratchpipe import ScratchPipe

    dev = torch.device("cuda:0")
    w = wl.custom(rows=[3000, 5000, 4000], dim=32, batch=48, pooling=[3, 2, 4],
                  slots=[420, 300, 560], lookahead=2, steps=16,
                  dist=(("zipf", 1.05), ("uniform",), ("zipf", 1.2)), seed=9)
    T, B, D, L = w.tables, w.batch, w.dim, w.lookahead
    sizes = [48, 17, 48, 1, 48, 0, 30, 48, 48, 5, 48, 0, 0, 48, 33, 48]
    gpu_b, ora_b = [], []
    for s, b in enumerate(sizes):
        g_b, o_b = _shrink(w, *wl.batch(w, s), b)
        gpu_b.append(g_b)
        ora_b.append(o_b)
    src = gpu_b
    if device_ids:
        src = [(torch.from_numpy(i).to(dev), torch.from_numpy(o).to(dev)) for i, o in gpu_b]
    print(f"case batch sizes {sizes} device_ids {device_ids} bound {bound}", flush=True)

    host = harness.fresh_host(w)
    ref = [wl.init_table(w, t) for t in range(T)]
    planner = oracle.Planner(w.rows, w.slots)
    touched = [np.zeros(r, bool) for r in w.rows]
    sp = ScratchPipe(w.rows, D, w.slots, L, host, max_batch=B,
                     max_ids=max(int(i.size) for i, _ in gpu_b),
                     max_table_ids=harness.table_bound(w, ora_b) if bound == "auto" else 0)
    worst = 0.0
    try:
        n = len(sizes)
        for u in range(n):
            win = list(range(u, min(u + L, n - 1) + 1))
            ahead = [q for q in range(u + L + 1, u + L + 3) if q < n]
            tk = sp.plan([src[q] for q in win + ahead])
            assert tk == u
            p = planner.plan([ora_b[q] for q in win], B)
            harness.compare_plan(u, sp.debug_plan(tk, max(int(gpu_b[u][0].size), 1)), p, T, B)
            b = sizes[u]
            out = torch.full((T * b, D), float("nan"), dtype=torch.float32, device=dev)
            sp.forward(tk, out)
            g = wl.grads(w, u)                      # [T][B][D]; rows past b belong to empty bags
            gd = torch.from_numpy(np.ascontiguousarray(g[:, :b])).to(dev)
            sp.backward_update(tk, gd, w.lr)
            ids, off = ora_b[u]
            o_ref = oracle.train_step(ref, ids, off, B, g, w.lr, want_out=True)
            for t in range(T):
                touched[t][ids[off[t * B]:off[(t + 1) * B]]] = True
            torch.cuda.synchronize()
            assert not o_ref.reshape(T, B, D)[:, b:].any()  # the padding bags are empty
            if b == 0:
                continue  # no output rows
            got = out.cpu().numpy().reshape(T, b, D)
            exp = o_ref.reshape(T, B, D)[:, :b]
            e = harness.row_rel_err(got.reshape(-1, D), exp.reshape(-1, D))
            worst = max(worst, float(e.max(initial=0.0)))
            assert e.max(initial=0.0) <= harness.REL_TOL, f"step {u}: forward rel err {e.max()}"
        sp.flush()
        st = sp.stats()
    finally:
        sp.close()
    assert st["plans"] == len(sizes) and st["evictions"] > 0
    for t in range(T):
        assert np.array_equal(host[t][~touched[t]], ref[t][~touched[t]])
        e = harness.row_rel_err(host[t][touched[t]], ref[t][touched[t]])
        assert e.max(initial=0.0) <= harness.REL_TOL, f"table {t}: row rel err {e.max()}"
    host.close()
    print(f"batch sizes worst fwd {worst:.2e} evictions {st['evictions']}", flush=True)
