"""Embedding-training throughput of the HIP scratchpad on one MI355X.

One step = sp_plan (window ingest, dedup, Hit-Map query, hold, LRU victims,
commit, miss fill and evicted-row write-back) + sp_forward (pooled gather) +
sp_backward_update (gradient coalescing and in-place SGD) for one mini-batch
of the synthetic workload.  Batch IDs and upstream gradients are generated
before timing and are resident in HBM when the timed region starts; the
embedding tables live in pinned host memory and only the scratchpad is in HBM.

Prints one JSON line (rank 0).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_bytes(w, n_unique: float, n_chunks: float) -> dict:
    """Algorithmic HBM bytes per launch of the forward and backward kernels.

    forward  (unique-bound): each unique row read once, slot_of, bag offsets,
             pooled output written.
    backward: each unique row read and written once, each bag gradient read
             once, sorted bag index per position, per-run offsets / first
             chunk / slot, chunk->run map.
    """
    T, B, D = w.tables, w.batch, w.dim
    nnz = w.nnz
    row = 4 * D
    fwd = n_unique * row + nnz * 4 + (T * B + 1) * 4 + T * B * row
    fwd_req = nnz * row + nnz * 4 + (T * B + 1) * 4 + T * B * row
    bwd = 2 * n_unique * row + T * B * row + nnz * 4 + n_unique * 12 + n_chunks * 4
    return {"forward": fwd, "forward_requested": fwd_req, "backward": bwd}


def traffic_from_profile(kernel: str, src_hash: str, workload: str):
    """HBM bytes per launch measured by rocprofv3 counters, if a summary for the
    current kernel source exists under profiles/ (keyed by the --workload name)."""
    p = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
        e = d.get(workload, {}).get(kernel)
        if e and e.get("source_sha256") == src_hash:
            return float(e["bytes_per_launch"])
    except Exception:
        return None
    return None


def access_ceiling(w, n_rows: int) -> dict | None:
    """Bare random-row read-modify-write, random-row gather and sequential copy at the
    workload's shape (Storage slots, distinct rows per step, row width, bags), timed by
    the ceiling probe built beside the library.  The fraction of these that a training
    kernel reaches says how close it is to what HBM gives its access pattern."""
    import subprocess
    exe = os.path.join(ROOT, "paper_2205_04702_amd", "ceiling")
    if not os.path.exists(exe):
        log("[bench] no ceiling probe built; skipping it")
        return None
    cmd = [exe, str(sum(w.slots)), str(max(1, n_rows)), str(w.dim), str(w.tables * w.batch), "1024"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    if r.returncode != 0:
        log(f"[bench] ceiling probe failed ({r.returncode}): {r.stderr.strip()}")
        return None
    return json.loads(r.stdout.strip().splitlines()[-1])


def cpu_baseline(w, seconds: float = 15.0, max_steps: int | None = None) -> dict:
    """The uncached CPU oracle trainer on the same inputs, bounded in time."""
    from oracle import oracle
    from paper_2205_04702_amd import workload as wl
    tables = [wl.init_table(w, t) for t in range(w.tables)]
    cores = min(oracle.max_threads(), w.tables)
    # one step to size the sample
    ids, off = wl.batch(w, 0)
    g = wl.grads(w, 0)
    t0 = time.perf_counter()
    oracle.train_step(tables, ids, off, w.batch, g, w.lr, want_out=True)
    one = time.perf_counter() - t0
    n = max(1, min(int(seconds / max(one, 1e-6)), max_steps or w.steps))
    inputs = [(wl.batch(w, s), wl.grads(w, s)) for s in range(1, n + 1)]
    t0 = time.perf_counter()
    for (ids, off), g in inputs:
        oracle.train_step(tables, ids, off, w.batch, g, w.lr, want_out=True)
    dt = time.perf_counter() - t0
    return {"value": round(w.batch * n / dt, 1), "unit": "samples/s", "cores": cores,
            "kind": "oracle",
            "sample": f"steps 1..{n} of {w.name} (forward + coalesced SGD, fp64 accumulation, "
                      f"OpenMP over tables), input generation excluded"}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="zipf-8x1M")
    ap.add_argument("--tables", type=int, default=0, metavar="N",
                    help="run only the workload's first N tables (one GPU's share when the "
                         "pinned host tables of the whole workload exceed what one process maps)")
    ap.add_argument("--policy", choices=["lru", "lfu", "random"], default="lru",
                    help="replacement policy (LRU is the method's default)")
    ap.add_argument("--hold-past", type=int, default=0, metavar="P",
                    help="also hold the rows of the P batches planned before each plan")
    ap.add_argument("--prefetch", action="store_true",
                    help="each plan also fills the next batch's missing rows")
    ap.add_argument("--host-ids", action="store_true",
                    help="hand the batch IDs over from host memory (PCIe-inclusive variant)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-timing", action="store_true", help="do not time kernels with events")
    ap.add_argument("--time-every", type=int, default=8, metavar="K",
                    help="time the kernels of every K-th step with events (the rest run untimed)")
    ap.add_argument("--event-waits", action="store_true",
                    help="wait on events instead of stream values (for profilers that run one "
                         "dispatch at a time, such as counter collection)")
    ap.add_argument("--serialize", action="store_true",
                    help="synchronise the device at the end of every call, so each kernel runs "
                         "alone (kernel times without overlap; throughput is then not the "
                         "pipelined one)")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the access-pattern ceiling probe run after the timed region")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="after the timed region, run a plain elementwise copy (torch.neg) of MIB "
                         "MiB three times: the reference kernel for scaling HBM byte counters")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the scratchpad path has no multi-GPU mode "
              "(tables would shard across GPUs, one context per GPU)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2205_04702_amd import workload as wl
    from paper_2205_04702_amd import scratchpipe as sp

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    w = wl.get_workload(args.workload)
    if args.tables > 0:
        import dataclasses
        n = args.tables
        w = dataclasses.replace(w, name=f"{w.name}-first{n}", rows=w.rows[:n],
                                pooling=w.pooling[:n], dist=w.dist[:n], slots=w.slots[:n])
    W, K, L = args.warmup, args.steps, w.lookahead
    ahead = sp.SP_MAX_AHEAD
    nb = W + K + L + 1 + ahead  # the window of the last step plus the batches prepared after it
    log(f"[bench] workload {w.name}: generating {nb} batches and {W + K} gradient tensors")
    t0 = time.perf_counter()
    host_batches = [wl.batch(w, s) for s in range(nb)]
    if args.host_ids:
        batches = host_batches
    else:
        batches = [(torch.from_numpy(i).to(dev), torch.from_numpy(o).to(dev)) for i, o in host_batches]
    grads = [torch.from_numpy(wl.grads(w, s)).to(dev) for s in range(W + K)]
    host = sp.HostTables(w.rows, w.dim)
    # tables are independent streams: fill them on a few threads (numpy's
    # generators release the GIL)
    import concurrent.futures as cf
    with cf.ThreadPoolExecutor(max_workers=max(1, min(16, w.tables, os.cpu_count() or 1))) as ex:
        list(ex.map(lambda t: wl.init_table(w, t, out=host[t]), range(w.tables)))
    log(f"[bench] inputs ready in {time.perf_counter() - t0:.1f}s")

    timed = not args.no_timing
    every = max(1, args.time_every)
    base_flags = ((sp.SP_FLAG_EVENT_WAITS if args.event_waits else 0)
                  | (sp.SP_FLAG_DEBUG_SYNC if args.serialize else 0))
    ctx = sp.ScratchPipe(w.rows, w.dim, w.slots, L, host, max_batch=w.batch, max_ids=w.nnz,
                         flags=base_flags, policy=args.policy, hold_past=args.hold_past,
                         prefetch=args.prefetch,
                         max_table_ids=w.batch * max(w.pooling))
    out = torch.empty((w.tables * w.batch, w.dim), dtype=torch.float32, device=dev)

    host_s = [0.0, 0.0, 0.0]  # host time inside plan / forward / backward calls
    stream = torch.cuda.current_stream().cuda_stream  # forward and backward run here

    def step(u):
        # hold window u..u+L, plus the next batches handed over early for sorting;
        # kernel events on a sample of the steps only (they cost host time)
        base = base_flags
        if timed:
            ctx.set_flags(base | (sp.SP_FLAG_TIMING if u % every == 0 else 0))
        elif base:
            ctx.set_flags(base)
        t0 = time.perf_counter()
        tk = ctx.plan([batches[q] for q in range(u, min(u + L + ahead, nb - 1) + 1)])
        t1 = time.perf_counter()
        ctx.forward(tk, out, stream)
        t2 = time.perf_counter()
        ctx.backward_update(tk, grads[u], w.lr, stream)
        t3 = time.perf_counter()
        host_s[0] += t1 - t0
        host_s[1] += t2 - t1
        host_s[2] += t3 - t2

    for u in range(W):
        step(u)
    torch.cuda.synchronize()
    s0 = ctx.stats()
    log(f"[bench] warmup {W} steps done")
    torch.cuda.synchronize()
    host_s[:] = [0.0, 0.0, 0.0]
    t0 = time.perf_counter()
    for u in range(W, W + K):
        step(u)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    s1 = ctx.stats()
    if args.calibrate_copy > 0:
        x = torch.ones(args.calibrate_copy << 18, dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        for _ in range(3):
            torch.neg(x, out=y)  # reads and writes MIB MiB
        torch.cuda.synchronize()
        del x, y
    ctx.close()
    host.close()
    log(f"[bench] timed {K} steps in {dt:.3f}s")

    d = {k: s1[k] - s0[k] for k in s1 if isinstance(s1[k], (int, float))}
    n_unique = d["unique"] / max(d["plans"], 1)
    samples_per_s = w.batch * K / dt
    res = {
        "metric": "embedding-train samples/sec at 1 MI355X; achieved HBM GB/s vs peak",
        "value": round(samples_per_s, 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(dt * 1e3 / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {**w.describe(), "ids": "host" if args.host_ids else "hbm",
                   **({"policy": args.policy} if args.policy != "lru" else {}),
                   **({"hold_past": args.hold_past} if args.hold_past else {}),
                   **({"serialized": True} if args.serialize else {}),
                   **({"prefetch": True} if args.prefetch else {})},
    }
    # the planned batches' own misses; with prefetch, fills also cover the next batches
    detail = {"miss_rate": round((d["misses"] - d.get("prefetched", 0)) / max(d["unique"], 1), 4),
              "fills_per_step": round(d["misses"] / K, 1),
              "unique_per_step": round(n_unique, 1),
              "evictions_per_step": round(d["evictions"] / K, 1),
              "prefetched_per_step": round(d.get("prefetched", 0) / K, 1),
              "fill_GBps": round(d["bytes_fill"] / dt / 1e9, 3),
              "writeback_GBps": round(d["bytes_writeback"] / dt / 1e9, 3),
              "host_ms_per_step": {"plan": round(host_s[0] * 1e3 / K, 4),
                                   "forward": round(host_s[1] * 1e3 / K, 4),
                                   "backward": round(host_s[2] * 1e3 / K, 4),
                                   **{k[8:]: round(d[k] / K, 4) for k in d if k.startswith("host_ms_")}}}
    if not args.no_timing and d["timed_forward"] > 0:
        # kernel execution times from start/stop events of the launches themselves
        fwd_ms = d["ms_forward"] / d["timed_forward"]
        bwd_ms = d["ms_backward"] / max(d["timed_backward"], 1)
        n_chunks = d["chunks"] / max(d["updates"], 1)
        kb = kernel_bytes(w, n_unique, n_chunks)
        fwd_gbs = kb["forward"] / (fwd_ms * 1e-3) / 1e9
        bwd_gbs = kb["backward"] / (bwd_ms * 1e-3) / 1e9
        detail.update({"forward_ms": round(fwd_ms, 5), "backward_ms": round(bwd_ms, 5),
                       "combine_ms": round(d["ms_combine"] / max(d["timed_combine"], 1), 5),
                       "combine_launches": d["timed_combine"],
                       "plan_ms": round(d["ms_plan"] / max(d["timed_plan"], 1), 5),
                       "fill_ms": round(d["ms_fill"] / max(d["timed_fill"], 1), 5),
                       "ingest_ms": round(d["ms_ingest"] / max(d["timed_ingest"], 1), 5),
                       "query_ms": round(d["ms_query"] / max(d["timed_query"], 1), 5),
                       "chunks_per_step": round(n_chunks, 1),
                       "forward_GBps_unique": round(fwd_gbs, 1),
                       "forward_GBps_requested": round(kb["forward_requested"] / (fwd_ms * 1e-3) / 1e9, 1),
                       "backward_GBps": round(bwd_gbs, 1)})
        # the fill is bound by the host link, not by HBM: its misses' rows
        # cross the link once per fill (timed with the same events)
        fill_ms = d["ms_fill"] / max(d["timed_fill"], 1)
        if fill_ms > 0:
            link = d["bytes_fill"] / max(d["plans"], 1) / (fill_ms * 1e-3) / 1e9
            detail["host_link"] = {"kernel": "k_move", "achieved_GBps": round(link, 1),
                                   "nominal_GBps": 64.0, "unit": "GB/s host to device",
                                   "frac_nominal": round(link / 64.0, 3)}
        src = open(os.path.join(ROOT, "paper_2205_04702_amd", "csrc", "k_train.hip"), "rb").read()
        src_hash = hashlib.sha256(src).hexdigest()
        dom = "forward" if fwd_ms >= bwd_ms else "backward"
        ach = fwd_gbs if dom == "forward" else bwd_gbs
        name = "k_forward" if dom == "forward" else "k_backward"
        tr = traffic_from_profile(name, src_hash, args.workload if not args.tables else w.name)
        res["roofline"] = {"bound": "hbm", "kernel": name,
                           "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": tr,
                           "bytes_per_launch": int(kb[dom]),
                           "ms_per_launch": round(fwd_ms if dom == "forward" else bwd_ms, 5)}
    if not args.no_ceiling and "roofline" in res:
        ceil = access_ceiling(w, int(round(n_unique)))
        if ceil:
            detail["ceiling"] = ceil
            pat = "gather" if res["roofline"]["kernel"] == "k_forward" else "rmw"
            c_gbs = ceil[pat]["GBps"]
            res["roofline"]["pattern_ceiling"] = {
                "pattern": pat, "GBps": c_gbs, "frac": round(res["roofline"]["achieved"] / c_gbs, 4),
                "copy_GBps": ceil["copy"]["GBps"]}
    res["detail"] = detail
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle")
        res["cpu_baseline"] = cpu_baseline(w, seconds=args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
