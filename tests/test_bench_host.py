"""Host-side behaviour of bench.py that needs no GPU: the one-GPU refusal and the
CPU-baseline leg (the oracle trainer, timed on a bounded sample)."""
import os
import re
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def _run_bench(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, BENCH] + args, capture_output=True, text=True,
                          timeout=120, env=env, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run_bench(["--gpus", "2", "--steps", "1", "--warmup", "0"])
    assert r.returncode == 2, r.stderr[-500:]
    assert "one GPU" in r.stderr and r.stdout == ""
    # launched as one of several ranks (torch.distributed.run sets WORLD_SIZE)
    r = _run_bench(["--steps", "1", "--warmup", "0"], {"WORLD_SIZE": "4"})
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_cpu_baseline_trains_the_workload_with_the_oracle(oracle):
    sys.path.insert(0, ROOT)
    import bench
    from paper_2205_04702_amd import workload as wl

    w = wl.get_workload("tiny")
    batches = [wl.batch(w, s) for s in range(8)]
    tables = [wl.init_table(w, t) for t in range(w.tables)]
    res = bench.cpu_baseline(w, tables, batches, seconds=0.05)

    assert res["kind"] == "oracle" and res["unit"] == "samples/s" and res["value"] > 0
    assert 1 <= res["cores"] <= w.tables and res["affinity_cpus"] >= 1
    m = re.match(r"steps 1\.\.(\d+) of " + re.escape(w.name) + r", all 4 tables", res["sample"])
    assert m, res["sample"]
    n = int(m.group(1))
    assert 1 <= n <= len(batches) - 1

    # The timed work is the whole step: the tables it leaves equal step 0 (its
    # untimed sizing run) and steps 1..n of the oracle, applied to fresh tables.
    ref = [wl.init_table(w, t) for t in range(w.tables)]
    for s in range(n + 1):
        ids, off = batches[s]
        oracle.train_step(ref, ids, off, w.batch, wl.grads(w, s), w.lr)
    for a, b in zip(tables, ref):
        assert np.array_equal(a, b)
    assert not np.array_equal(ref[0], wl.init_table(w, 0))
