"""Batches without IDs, tables without IDs and a one-ID batch on the GPU (needs an
MI355X): planned, held, entering the window and prepared ahead, on both ingest
paths, with host and device IDs, the staged fill, prefetch, a past window and
the random policy.  Plans must match the oracle bit for bit, empty batches'
outputs must be zeros, and tables must match within 1e-5 per row."""
import pytest

from paper_2205_04702_amd import scratchpipe as sp
from paper_2205_04702_amd import workload as wl

pytestmark = pytest.mark.gpu

# step -> (tables kept, most IDs kept): two empty batches in a row make the
# planned batch and the batch entering the window empty in turn
KINDS = {3: ((), None), 5: ((1, 3), None), 7: ((), None), 8: ((), None), 10: (None, 1)}


@pytest.fixture(scope="module")
def harness():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_harness
    return gpu_harness


@pytest.mark.parametrize("case", [
    dict(max_table_ids="auto", prepare_ahead=2),
    dict(max_table_ids=0, device_ids=True),
    dict(fill="staged", prepare_ahead=2, flags=sp.SP_FLAG_DEFER_SORTS),
    dict(prefetch=1, prepare_ahead=2),
    dict(hold_past=2, prepare_ahead=2),
    dict(policy="random", seed=5, max_table_ids=0),
], ids=["lds-host-ids", "general-device-ids", "staged-deferred", "prefetch", "past-window",
        "random-policy"])
def test_empty_batches_and_tables(harness, case):
    w = wl.get_workload("tiny")
    batches = [wl.thinned_batch(w, s, *KINDS.get(s, (None, None))) for s in range(16)]
    assert [b[0].size for b in batches][3] == 0 and batches[10][0].size == 1
    print(f"case zero sizes {case}", flush=True)
    r = harness.run_parity(w, batches, **case)
    st = r["stats"]
    assert st["plans"] == 16 and st["evictions"] > 0
    print(f"zero sizes worst fwd {r['worst_fwd']:.2e} table {r['worst_table']:.2e}", flush=True)
