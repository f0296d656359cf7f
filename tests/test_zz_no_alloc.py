"""sp_backward_update_static, the entry point that allocates nothing: its split runs'
partial sums live in a fixed per-GPU device array.  Through the C ABI it must give
exactly what sp_backward_update gives, on two calls in a row (the second with a
smaller batch), and reject a ticket whose partial sums do not fit, changing nothing."""
import ctypes as C

import numpy as np
import pytest

from paper_2205_04702_amd import scratchpipe as sp
from paper_2205_04702_amd import workload as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch, torch.device("cuda:0")


def _batches():
    """Two batches of one table of hot rows (runs longer than one 16-position chunk,
    so partial sums are used): B=96 then a smaller B=24."""
    rng = np.random.default_rng(7)
    out = []
    for B, P in ((96, 12), (24, 12)):
        ids = (rng.zipf(1.3, size=B * P) % 300).astype(np.int32)
        off = (np.arange(B + 1, dtype=np.int64) * P).astype(np.int32)
        out.append((ids, off, B))
    return out


def _train(torch, dev, use_static):
    from tests import gpu_harness
    w = wl.custom(rows=[300], dim=64, batch=96, pooling=12, slots=[300], lookahead=0, steps=2,
                  seed=3)
    host = gpu_harness.fresh_host(w)
    L = sp.load()
    ctx = sp.ScratchPipe(w.rows, w.dim, w.slots, 0, host, max_batch=96, max_ids=96 * 12)
    outs = []
    try:
        stream = torch.cuda.current_stream().cuda_stream
        for u, (ids, off, B) in enumerate(_batches()):
            tk = ctx.plan([(ids, off)])
            out = torch.zeros((B, w.dim), device=dev)
            ctx.forward(tk, out)
            g = torch.from_numpy(wl.grads(wl.custom(rows=[300], dim=64, batch=B, pooling=12,
                                                    slots=[300], lookahead=0, steps=2, seed=u),
                                          u)).to(dev)
            fn = L.sp_backward_update_static if use_static else L.sp_backward_update
            st = fn(ctx.handle, tk, g.data_ptr(), C.c_float(0.05), stream)
            assert st == sp.SP_OK, sp.sp_last_error(ctx.handle)
            torch.cuda.synchronize()
            outs.append((out.cpu().numpy(), g.cpu().numpy()))
        ctx.flush()
        return host[0].copy(), outs, ctx.stats()
    finally:
        ctx.close()
        host.close()


def test_static_matches_backward_update_twice(torch_dev):
    torch, dev = torch_dev
    a_tab, a_outs, a_st = _train(torch, dev, use_static=False)
    b_tab, b_outs, b_st = _train(torch, dev, use_static=True)
    assert a_st["chunks"] > 0 and b_st["chunks"] == a_st["chunks"]
    for (ao, ag), (bo, bg) in zip(a_outs, b_outs):
        assert np.array_equal(ao, bo) and np.array_equal(ag, bg)
    assert np.array_equal(a_tab, b_tab)
    # and the oracle's uncached training agrees within the per-row tolerance
    from oracle import oracle
    from tests import gpu_harness
    w = wl.custom(rows=[300], dim=64, batch=96, pooling=12, slots=[300], lookahead=0, steps=2,
                  seed=3)
    ref = [wl.init_table(w, 0)]
    for (ids, off, B), (_, g) in zip(_batches(), b_outs):
        oracle.train_step(ref, ids, off, B, g.reshape(1, B, 64), 0.05)
    assert gpu_harness.row_rel_err(b_tab, ref[0]).max() <= gpu_harness.REL_TOL


def test_static_rejects_a_ticket_above_the_array(torch_dev):
    """32 MiB holds 32768 chunks of 256 floats: a batch of 40000 distinct keys with a
    split run has more; the call fails and sp_backward_update then succeeds."""
    torch, dev = torch_dev
    from tests import gpu_harness
    n = 40_000
    w = wl.custom(rows=[60_000], dim=256, batch=1, pooling=n + 40, slots=[60_000], lookahead=0,
                  steps=1, seed=5)
    ids = np.concatenate([np.arange(n, dtype=np.int32), np.full(40, 7, np.int32)])
    off = np.array([0, ids.size], np.int32)
    host = gpu_harness.fresh_host(w)
    ctx = sp.ScratchPipe(w.rows, w.dim, w.slots, 0, host, max_batch=1, max_ids=ids.size)
    try:
        tk = ctx.plan([(ids, off)])
        out = torch.zeros((1, 256), device=dev)
        ctx.forward(tk, out)
        g = torch.ones((1, 256), device=dev)
        with pytest.raises(sp.SPError) as e:
            ctx.backward_update_static(tk, g, 0.01)
        assert e.value.status == sp.SP_ERR_INVALID_ARG
        assert "backward chunks" in str(e.value)
        ctx.backward_update(tk, g, 0.01)
        ctx.flush()
        assert ctx.stats()["updates"] == 1
    finally:
        ctx.close()
        host.close()
