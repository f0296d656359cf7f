"""The largest keys the library accepts, on the GPU (needs an MI355X): 64 tables,
the last of 2^25 rows, so keys use all 31 bits and table 63's last row is key
2^31 - 1; table 0's row 0 is key 0.  Both are in every batch beside uniform
IDs, through both ingest paths, with host and device IDs."""
import pytest

from paper_2205_04702_amd import workload as wl

pytestmark = pytest.mark.gpu

TOP = 1 << 25  # most rows of one table


@pytest.fixture(scope="module")
def harness():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_harness
    return gpu_harness


def max_key_batches(w):
    B = w.batch
    out = []
    for s in range(w.steps):
        ids, off = wl.batch(w, s)
        ids = ids.copy()
        a = int(off[63 * B])
        ids[a:a + 3] = [TOP - 1, TOP - 2, 0]  # table 63: the top key, its neighbour, row 0
        ids[int(off[0])] = 0                  # key 0
        out.append((ids, off))
    return out


@pytest.mark.parametrize("bound,device_ids", [("auto", False), (0, True)],
                         ids=["lds-ingest-host-ids", "general-ingest-device-ids"])
def test_largest_keys(harness, bound, device_ids):
    w = wl.custom(rows=[200] * 63 + [TOP], dim=4, batch=16, pooling=[1] * 63 + [4],
                  slots=[80] * 63 + [300], lookahead=2, steps=12, dist=("uniform",), seed=31)
    batches = max_key_batches(w)
    print(f"case largest keys bound {bound} device_ids {device_ids}", flush=True)
    r = harness.run_parity(w, batches, max_table_ids=bound, device_ids=device_ids)
    st = r["stats"]
    assert st["evictions"] > 0 and st["hits"] > 0
    print(f"largest keys worst fwd {r['worst_fwd']:.2e} table {r['worst_table']:.2e} "
          f"evictions {st['evictions']}", flush=True)
