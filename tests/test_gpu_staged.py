"""The staged fill on the GPU: host threads gather each plan's missing rows from
ordinary (pageable) host tables into pinned staging, copies take them to the device
piece by piece, and the move kernel writes them into their slots ([Collect],
[Exchange] and [Insert] of Sec. IV-B).  Plans must match the oracle bit for bit,
outputs and tables within 1e-5 per row, and the tables must be bit-identical to the
zero-copy fill's."""
import numpy as np
import pytest

from paper_2205_04702_amd import scratchpipe as sp
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


def test_tiny_staged_matches_oracle_and_mapped(harness):
    w = wl.get_workload("tiny")
    _say("case staged tiny")
    a = harness.run_parity(w, fill="staged", return_tables=True)
    b = harness.run_parity(w, fill="mapped", return_tables=True)
    assert a["stats"]["evictions"] > 0
    for x, y in zip(a["tables"], b["tables"]):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("dim", [4, 64, 256])
def test_staged_every_row_width_ragged(harness, dim):
    """Ragged and empty bags, the general ingest path, IDs from host memory; no
    synchronisation between steps, so the fill thread runs behind the caller."""
    w = wl.custom(rows=[4000, 2500, 6000], dim=dim, batch=64, pooling=4,
                  slots=[1500, 1200, 1800], lookahead=3, steps=25, dist=("zipf", 1.1),
                  seed=30 + dim)
    batches = harness.make_inputs(w, ragged=9)
    _say(f"case staged ragged dim {dim}")
    harness.run_parity(w, batches, fill="staged", sync_each_step=False, max_table_ids=0,
                       check_fwd_steps=[0, 12, 24])


@pytest.mark.parametrize("bound", ["auto", 0])
def test_staged_device_ids_handed_over_ahead(harness, bound):
    """IDs in device memory, the two batches after the window handed over ahead and no
    synchronisation between steps: batches prepared ahead are read after sp_plan has
    returned, and once a plan that holds a batch has returned its IDs are overwritten
    with an out-of-range row, which the library must never see.  Both ingest paths (in
    LDS, and general); the tables must equal the host-ID run's bit for bit."""
    w = wl.custom(rows=[6000, 9000, 4000], dim=32, batch=64, pooling=6,
                  slots=[1500, 2000, 1200], lookahead=2, steps=30, dist=("zipf", 1.05),
                  seed=43)
    _say(f"case staged device IDs bound {bound}")
    a = harness.run_parity(w, fill="staged", device_ids=True, prepare_ahead=2,
                           sync_each_step=False, max_table_ids=bound, return_tables=True,
                           check_fwd_steps=[0, 15, 29], overwrite_held_ids=True)
    b = harness.run_parity(w, fill="staged", prepare_ahead=2, sync_each_step=False,
                           max_table_ids=bound, return_tables=True, check_fwd_steps=[29])
    assert a["stats"]["evictions"] > 0
    for x, y in zip(a["tables"], b["tables"]):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("device_ids,static", [(False, False), (True, False), (True, True)],
                         ids=["host-ids", "device-ids", "device-ids-static-backward"])
def test_staged_sorts_deferred_behind_the_update(harness, device_ids, static):
    """SP_FLAG_DEFER_SORTS: the batches prepared ahead are sorted behind each update,
    as they are by default behind a large write-back; with the allocation-free backward
    they are left to the next plan.  Device IDs of held batches are overwritten once
    their plan returns.  Plans, sampled outputs and tables must match the oracle."""
    w = wl.custom(rows=[6000, 9000, 4000], dim=32, batch=64, pooling=6,
                  slots=[1500, 2000, 1200], lookahead=2, steps=30, dist=("zipf", 1.05),
                  seed=47)
    _say(f"case staged deferred sorts device_ids={device_ids} static={static}")
    r = harness.run_parity(w, fill="staged", device_ids=device_ids, prepare_ahead=2,
                           sync_each_step=False, flags=sp.SP_FLAG_DEFER_SORTS,
                           static_backward=static, overwrite_held_ids=device_ids,
                           check_fwd_steps=[0, 15, 29])
    assert r["stats"]["evictions"] > 0


@pytest.mark.parametrize("prefetch", [False, True])
def test_staged_prefetch_and_past_window(harness, prefetch):
    w = wl.custom(rows=[3000, 5000], dim=32, batch=48, pooling=[3, 5], slots=[900, 1400],
                  lookahead=2, steps=24, dist=("zipf", 1.05), seed=41)
    _say(f"case staged prefetch={prefetch} hold_past 1")
    harness.run_parity(w, fill="staged", prefetch=prefetch, hold_past=1, prepare_ahead=2,
                       sync_each_step=False, check_fwd_steps=[0, 11, 23])


def test_staged_large_misses_span_several_pieces(harness):
    """More missing rows per plan than one host-to-device piece (8 MiB of rows)."""
    w = wl.custom(rows=[400_000, 300_000], dim=128, batch=2048, pooling=12,
                  slots=[40_000, 30_000], lookahead=1, steps=6, dist=("uniform",), seed=43)
    _say("case staged large fills")
    r = harness.run_parity(w, fill="staged", sync_each_step=False, check_fwd_steps=[0, 5],
                           prepare_ahead=2)
    assert r["stats"]["misses"] > 3 * (8 << 20) // (4 * 128)


def test_staged_poison_flag(harness):
    """SP_FLAG_POISON: Storage starts as NaN and spent staging is set to NaN; a
    correct schedule never lets either reach an output or a table."""
    w = wl.custom(rows=[3000, 2000], dim=32, batch=40, pooling=[4, 3], slots=[500, 450],
                  lookahead=2, steps=20, dist=("zipf", 1.0), seed=44)
    for fill in ("staged", "mapped"):
        _say(f"case poison {fill}")
        harness.run_parity(w, fill=fill, flags=sp.SP_FLAG_POISON, sync_each_step=False)


def test_sync_lands_every_writeback(harness):
    """sp_sync: afterwards the host tables hold every row evicted so far, and
    training continues as if nothing happened (same tables as without it)."""
    import torch
    w = wl.custom(rows=[3000], dim=16, batch=32, pooling=4, slots=[300], lookahead=1,
                  steps=16, dist=("uniform",), seed=45)
    batches = harness.make_inputs(w)
    dev = torch.device("cuda:0")
    res = []
    for with_sync in (False, True):
        host = harness.fresh_host(w, "staged")
        ctx = sp.ScratchPipe(w.rows, w.dim, w.slots, w.lookahead, host, max_batch=w.batch,
                             max_ids=max(int(b[0].size) for b in batches), fill="staged")
        out = torch.zeros((w.tables * w.batch, w.dim), device=dev)
        for u in range(w.steps):
            tk = ctx.plan([batches[q] for q in range(u, min(u + 1, w.steps - 1) + 1)])
            ctx.forward(tk, out)
            ctx.backward_update(tk, torch.from_numpy(wl.grads(w, u)).to(dev), w.lr)
            if with_sync and u == 9:
                ctx.sync()
                st = ctx.stats()
                assert st["evictions"] > 0
                assert st["bytes_writeback"] == st["evictions"] * w.dim * 4
        ctx.flush()
        res.append(host[0].copy())
        ctx.close()
        host.close()
    assert np.array_equal(res[0], res[1])
