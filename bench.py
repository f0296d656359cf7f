"""Embedding-training throughput of the HIP scratchpad on one MI355X.

One step = sp_plan (window ingest, dedup, Hit-Map query, hold, LRU victims,
commit, miss fill and evicted-row write-back) + sp_forward (pooled gather) +
sp_backward_update (gradient coalescing and in-place SGD) for one mini-batch
of the synthetic workload.  The embedding tables live in host memory and only
the scratchpad is in HBM.  The batches' IDs and the upstream gradients are
generated in device memory before timing.  A second timed region then runs
the next steps with the IDs handed over from host memory (copied to the
device every step) and reports that rate beside the first.

Before the timed steps the scratchpad is filled until every slot holds a row
(untimed fill-up steps, so the timed steps evict and write back as in steady
state), then `--warmup` more untimed steps run.  The timed region is
bracketed by a device synchronisation and sp_sync (every write-back of the
steps so far has landed in the host tables) on both sides.

The default workload is the largest one: 26 tables x 10M rows x 128 (133 GB
of host tables, batch 4096, pooling 40, Zipf 0.9, 200k slots per table,
lookahead 4), with the staged fill (host gather into pinned staging, then
copies), since one process can pin only about 64 GiB.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
HOST_LINK_NOMINAL_GBS = 64.0  # PCIe Gen5 x16, per direction
STAGED_ABOVE_BYTES = 8 << 30  # tables above this use the staged fill by default


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
    current kernel source exists under profiles/ (keyed by the workload name)."""
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


def link_rates(mib: int = 1024, piece_mib: int = 32) -> dict:
    """The host link as this step uses it: host-to-device and device-to-host copies
    of `mib` MiB between pinned host memory and HBM, in pieces of `piece_mib` MiB as
    the library issues them, each direction alone and both at once on two streams
    (GB/s)."""
    import torch
    n, p = mib << 20, piece_mib << 20
    h_in = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    h_out = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    d_in = torch.empty(n, dtype=torch.uint8, device="cuda")
    d_out = torch.empty(n, dtype=torch.uint8, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()

    def h2d():
        with torch.cuda.stream(s1):
            for o in range(0, n, p):
                d_in[o:o + p].copy_(h_in[o:o + p], non_blocking=True)

    def d2h():
        with torch.cuda.stream(s2):
            for o in range(0, n, p):
                h_out[o:o + p].copy_(d_out[o:o + p], non_blocking=True)

    def seconds(*fs):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for f in fs:
            f()
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    seconds(h2d, d2h)  # first use of the buffers
    a, b, c = seconds(h2d), seconds(d2h), seconds(h2d, d2h)
    return {"h2d_alone_GBps": round(n / a / 1e9, 2), "d2h_alone_GBps": round(n / b / 1e9, 2),
            "both_GBps": round(2 * n / c / 1e9, 2)}


def link_rates_in_child():
    """link_rates() in a fresh child process.  In this one the library's four
    streams and the caller's already share the GPU's four hardware queues, and the
    two copy streams could land on one queue and run one after the other."""
    import subprocess
    r = subprocess.run([sys.executable, os.path.abspath(__file__), "--link-rates-only"],
                       capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        log(f"[bench] host-link probe failed: {r.stderr.strip()[-300:]}")
        return None
    return json.loads(r.stdout.strip().splitlines()[-1])


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, tables, batches, seconds: float) -> dict:
    """The uncached CPU oracle trainer on the same workload and tables, bounded in
    time (input generation excluded)."""
    from oracle import oracle
    from paper_2205_04702_amd import workload as wl
    cores = min(oracle.max_threads(), w.tables)
    ids, off = batches[0]
    g = wl.grads(w, 0)
    t0 = time.perf_counter()
    oracle.train_step(tables, ids, off, w.batch, g, w.lr, want_out=True)
    one = time.perf_counter() - t0
    n = max(1, min(int(seconds / max(one, 1e-6)), len(batches) - 1))
    inputs = [(batches[s], wl.grads(w, s)) for s in range(1, n + 1)]
    t0 = time.perf_counter()
    for (ids, off), g in inputs:
        oracle.train_step(tables, ids, off, w.batch, g, w.lr, want_out=True)
    dt = time.perf_counter() - t0
    return {"value": round(w.batch * n / dt, 1), "unit": "samples/s", "cores": cores,
            "kind": "oracle",
            "sample": f"steps 1..{n} of {w.name}, all {w.tables} tables (forward + coalesced "
                      f"SGD, fp64 accumulation, OpenMP over tables, {cores} threads), input "
                      f"generation excluded",
            "affinity_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model()}


def main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="zipf-26x10M")
    ap.add_argument("--tables", type=int, default=0, metavar="N",
                    help="run only the workload's first N tables")
    ap.add_argument("--fill", choices=["auto", "mapped", "staged"], default="auto",
                    help="how missing rows reach HBM: zero-copy from pinned, mapped tables, or "
                         "host gather into pinned staging then copies (auto: staged when the "
                         "tables exceed 8 GiB; measured faster on 26x4M and the mixed "
                         "workload, and the only way for tables beyond what one process pins)")
    ap.add_argument("--ids", choices=["host", "hbm"], default="hbm",
                    help="hand the batch IDs over from device memory (resident in HBM before "
                         "the timed region) or from host memory, copied over the host link "
                         "every step as the method's planner does")
    ap.add_argument("--no-host-ids-rate", action="store_true",
                    help="with --ids hbm, skip the second timed region that hands the same "
                         "workload's next batches over from host memory")
    ap.add_argument("--fillup", type=int, default=-1, metavar="N",
                    help="untimed steps before the warm-up (-1: until every slot holds a row, "
                         "none when the slots hold every table)")
    ap.add_argument("--policy", choices=["lru", "lfu", "random"], default="lru",
                    help="replacement policy (LRU is the method's default)")
    ap.add_argument("--hold-past", type=int, default=0, metavar="P",
                    help="also hold the rows of the P batches planned before each plan")
    ap.add_argument("--prefetch", type=int, default=0, metavar="D",
                    help="each plan also fills the missing rows of the next D batches")
    ap.add_argument("--ahead", type=int, default=-1, metavar="N",
                    help="batches after the hold window handed over early for sorting "
                         "(-1: SP_MAX_AHEAD)")
    ap.add_argument("--general-ingest", action="store_true",
                    help="promise no bound on IDs per table, so batches are sorted by the "
                         "multi-launch path even where one workgroup per table would do")
    ap.add_argument("--no-huge-pages", action="store_true",
                    help="staged fill: do not advise the host tables for transparent huge pages")
    ap.add_argument("--no-link-probe", action="store_true",
                    help="skip the host-link measurement after the timed region")
    ap.add_argument("--link-rates-only", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-timing", action="store_true", help="do not time kernels with events")
    ap.add_argument("--time-every", type=int, default=0, metavar="K",
                    help="time the kernels of every K-th step with events (0: every step when "
                         "a step moves more than 100 MB, else every 8th)")
    ap.add_argument("--event-waits", action="store_true",
                    help="wait on events instead of stream values (for profilers that run one "
                         "dispatch at a time, such as counter collection)")
    ap.add_argument("--serialize", action="store_true",
                    help="synchronise the device at the end of every call, so each kernel runs "
                         "alone (kernel times without overlap; throughput is then not the "
                         "pipelined one)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="after the timed region, run a plain elementwise copy (torch.neg) of MIB "
                         "MiB three times: the reference kernel for scaling HBM byte counters")
    args = ap.parse_args()
    if args.link_rates_only:  # the child of link_rates_in_child
        print(json.dumps(link_rates()), flush=True)
        return

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
    table_bytes = sum(w.rows) * w.dim * 4
    fill = args.fill if args.fill != "auto" else (
        "staged" if table_bytes > STAGED_ABOVE_BYTES else "mapped")
    evicts = sum(w.slots) < sum(w.rows)
    if args.fillup >= 0:
        fillup_max = args.fillup
    else:
        # enough steps to place a row in every slot at the first batch's miss count
        fillup_max = 0 if not evicts else 200
    W, K, L = args.warmup, args.steps, w.lookahead
    ahead = sp.SP_MAX_AHEAD if args.ahead < 0 else min(args.ahead, sp.SP_MAX_AHEAD)
    nsteps = fillup_max + W + K
    nb_needed = lambda steps: steps + L + 1 + ahead  # noqa: E731  (windows of the last step)

    t0 = time.perf_counter()
    host = sp.host_tables(w.rows, w.dim, fill, huge_pages=not args.no_huge_pages)
    # tables are independent streams: fill them on threads (numpy's generators
    # release the GIL)
    with cf.ThreadPoolExecutor(max_workers=max(1, min(16, w.tables, os.cpu_count() or 1))) as ex:
        list(ex.map(lambda t: wl.init_table(w, t, out=host[t]), range(w.tables)))
    log(f"[bench] workload {w.name}: {table_bytes / 1e9:.1f} GB of {fill} host tables "
        f"ready in {time.perf_counter() - t0:.1f}s")

    # batches are generated as the steps need them, outside the timed region
    host_batches: list = []
    dev_batches: list = []
    pool = cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1))

    def ensure_batches(n, chunk=1):
        if n <= len(host_batches):
            return
        n = max(n, len(host_batches) + chunk)
        new = list(pool.map(lambda s: wl.batch(w, s), range(len(host_batches), n)))
        host_batches.extend(new)
        if args.ids == "hbm":
            dev_batches.extend((torch.from_numpy(i).to(dev), torch.from_numpy(o).to(dev))
                               for i, o in new)

    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    grads: list = []

    def ensure_grads(n):
        while len(grads) < n:
            g = torch.randn((w.tables * w.batch, w.dim), generator=gen, device=dev)
            if w.grad_sigma != 1.0:
                g *= w.grad_sigma
            grads.append(g)

    every = args.time_every or (1 if w.nnz * w.dim * 4 > 100e6 else 8)
    timed = not args.no_timing
    base_flags = ((sp.SP_FLAG_EVENT_WAITS if args.event_waits else 0)
                  | (sp.SP_FLAG_DEBUG_SYNC if args.serialize else 0))
    ctx = sp.ScratchPipe(w.rows, w.dim, w.slots, L, host, max_batch=w.batch, max_ids=w.nnz,
                         flags=base_flags, policy=args.policy, hold_past=args.hold_past,
                         prefetch=args.prefetch, fill=fill,
                         max_table_ids=0 if args.general_ingest else w.batch * max(w.pooling))
    out = torch.empty((w.tables * w.batch, w.dim), dtype=torch.float32, device=dev)

    host_s = [0.0, 0.0, 0.0]  # host time inside plan / forward / backward calls
    stream = torch.cuda.current_stream().cuda_stream  # forward and backward run here
    src = dev_batches if args.ids == "hbm" else host_batches

    def step(u, last_batch):
        # hold window u..u+L, plus the next batches handed over early for sorting;
        # kernel events on a sample of the steps only (they cost host time)
        if timed:
            ctx.set_flags(base_flags | (sp.SP_FLAG_TIMING if u % every == 0 else 0))
        elif base_flags:
            ctx.set_flags(base_flags)
        t0 = time.perf_counter()
        tk = ctx.plan([src[q] for q in range(u, min(u + L + ahead, last_batch) + 1)])
        t1 = time.perf_counter()
        ctx.forward(tk, out, stream)
        t2 = time.perf_counter()
        ctx.backward_update(tk, grads[u], w.lr, stream)
        t3 = time.perf_counter()
        host_s[0] += t1 - t0
        host_s[1] += t2 - t1
        host_s[2] += t3 - t2

    # ---- untimed: fill-up until every slot holds a row, then warm-up
    t0 = time.perf_counter()
    u = 0
    fillup = 0
    total_slots = sum(w.slots)
    while fillup < fillup_max:
        ensure_batches(nb_needed(u + 1), chunk=16)
        ensure_grads(u + 1)
        step(u, len(host_batches) - 1)
        u += 1
        fillup += 1
        if ctx.stats()["misses"] >= total_slots:
            break
    log(f"[bench] fill-up: {fillup} steps ({time.perf_counter() - t0:.1f}s)")
    host_region = args.ids == "hbm" and not args.no_host_ids_rate
    n_timed = K + (W + K if host_region else 0)
    ensure_batches(nb_needed(u + W + n_timed))
    ensure_grads(u + W + n_timed)
    last = len(host_batches) - 1
    for _ in range(W):
        step(u, last)
        u += 1
    torch.cuda.synchronize()
    ctx.sync()
    s0 = ctx.stats()
    log(f"[bench] warmup {W} steps done")
    host_s[:] = [0.0, 0.0, 0.0]
    first_timed = u
    t0 = time.perf_counter()
    for _ in range(K):
        step(u, last)
        u += 1
    torch.cuda.synchronize()
    ctx.sync()
    dt = time.perf_counter() - t0
    s1 = ctx.stats()
    host_s_timed = list(host_s)
    host_rate = None
    if host_region:
        # the next K steps with the IDs handed over from host memory: the rate
        # that includes their copy over the host link every step (after W more
        # untimed steps with them)
        src = host_batches
        for _ in range(W):
            step(u, last)
            u += 1
        torch.cuda.synchronize()
        ctx.sync()
        s1h = ctx.stats()
        first_host = u
        t0 = time.perf_counter()
        for _ in range(K):
            step(u, last)
            u += 1
        torch.cuda.synchronize()
        ctx.sync()
        dth = time.perf_counter() - t0
        s2 = ctx.stats()
        host_rate = {"value": round(w.batch * K / dth, 1), "unit": "samples/s",
                     "ms_per_step": round(dth * 1e3 / K, 4),
                     "timed_steps": [first_host, first_host + K - 1],
                     "evictions_per_step": round((s2["evictions"] - s1h["evictions"]) / K, 1),
                     # later steps: where the budget holds every table, fewer
                     # rows are seen for the first time, so fewer miss
                     "miss_rate": round((s2["misses"] - s1h["misses"]
                                         - (s2.get("prefetched", 0) - s1h.get("prefetched", 0)))
                                        / max(s2["unique"] - s1h["unique"], 1), 4),
                     "ids": "host memory, copied to the device every step"}
        log(f"[bench] timed {K} more steps with host IDs in {dth:.3f}s")
    if args.calibrate_copy > 0:
        x = torch.ones(args.calibrate_copy << 18, dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        for _ in range(3):
            torch.neg(x, out=y)  # reads and writes MIB MiB
        torch.cuda.synchronize()
        del x, y
    ctx.close()
    log(f"[bench] timed {K} steps in {dt:.3f}s")
    host_s[:] = host_s_timed

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
        "config": {**w.describe(), "ids": args.ids, "fill": fill,
                   **({"host_pages": "4k" if args.no_huge_pages else "huge (advised)"}
                      if fill == "staged" else {}),
                   "timed_steps": [first_timed, first_timed + K - 1], "fillup_steps": fillup,
                   **({"policy": args.policy} if args.policy != "lru" else {}),
                   **({"hold_past": args.hold_past} if args.hold_past else {}),
                   **({"serialized": True} if args.serialize else {}),
                   **({"prefetch": args.prefetch} if args.prefetch else {})},
    }
    # the planned batches' own misses; with prefetch, fills also cover later batches
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
    if timed and d["timed_forward"] > 0:
        # kernel execution times from start/stop events of the launches themselves
        fwd_ms = d["ms_forward"] / d["timed_forward"]
        bwd_ms = d["ms_backward"] / max(d["timed_backward"], 1)
        cmb_ms = d["ms_combine"] / max(d["timed_combine"], 1)
        n_chunks = d["chunks"] / max(d["updates"], 1)
        kb = kernel_bytes(w, n_unique, n_chunks)
        src_hash = hashlib.sha256(open(os.path.join(ROOT, "paper_2205_04702_amd", "csrc",
                                                    "k_train.hip"), "rb").read()).hexdigest()
        wname = w.name if args.tables else args.workload
        kern = {}
        for name, key, ms in (("k_forward", "forward", fwd_ms), ("k_backward", "backward", bwd_ms)):
            gbs = kb[key] / (ms * 1e-3) / 1e9
            tr = traffic_from_profile(name, src_hash, wname)
            kern[name] = {"achieved": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
                          "bytes_per_launch": int(kb[key]), "ms_per_launch": round(ms, 5),
                          "traffic": tr}
            if tr:  # the counted bytes (scaled FETCH_SIZE + WRITE_SIZE) over the same time
                kern[name]["traffic_GBps"] = round(tr / (ms * 1e-3) / 1e9, 1)
                kern[name]["traffic_frac"] = round(tr / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        kern["k_forward"]["requested_GBps"] = round(kb["forward_requested"] / (fwd_ms * 1e-3) / 1e9, 1)
        # the dominant kernel: the one with more time per step
        dom = "k_forward" if fwd_ms >= bwd_ms else "k_backward"
        res["roofline"] = {"bound": "hbm", "kernel": dom, "achieved": kern[dom]["achieved"],
                           "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": kern[dom]["frac"],
                           "traffic": kern[dom]["traffic"],
                           "bytes_per_launch": kern[dom]["bytes_per_launch"],
                           "ms_per_launch": kern[dom]["ms_per_launch"],
                           "kernels": kern, "timed_launches": int(d["timed_forward"])}
        detail.update({"combine_ms": round(cmb_ms, 5), "combine_launches": d["timed_combine"],
                       "plan_ms": round(d["ms_plan"] / max(d["timed_plan"], 1), 5),
                       "fill_ms": round(d["ms_fill"] / max(d["timed_fill"], 1), 5),
                       "ingest_ms": round(d["ms_ingest"] / max(d["timed_ingest"], 1), 5),
                       "query_ms": round(d["ms_query"] / max(d["timed_query"], 1), 5),
                       "chunks_per_step": round(n_chunks, 1)})
        # the host link: fills host -> device (the zero-copy move kernel, or the
        # staged fill's copies), write-backs device -> host over the whole step
        fill_ms = (d["ms_h2d"] / max(d["timed_h2d"], 1)) if fill == "staged" else \
            d["ms_fill"] / max(d["timed_fill"], 1)
        link = {"unit": "GB/s", "nominal_GBps": HOST_LINK_NOMINAL_GBS,
                "h2d_bytes_per_step": int(d["bytes_fill"] / K),
                "d2h_bytes_per_step": int(d["bytes_writeback"] / K),
                "h2d_step_average_GBps": round(d["bytes_fill"] / dt / 1e9, 2),
                "d2h_step_average_GBps": round(d["bytes_writeback"] / dt / 1e9, 2)}
        if fill_ms > 0:
            g = d["bytes_fill"] / max(d["plans"], 1) / (fill_ms * 1e-3) / 1e9
            link.update({"h2d_during_fill_GBps": round(g, 2),
                         "h2d_fill_span_ms": round(fill_ms, 4),
                         "h2d_span": "host-to-device copies of gathered rows" if fill == "staged"
                         else "zero-copy move kernel"})
        if not args.no_link_probe:
            # the step's floor on this link: its bytes in each direction at that
            # direction's rate, and both together at the rate of both at once
            r = link_rates_in_child()
            if r:
                h, o = link["h2d_bytes_per_step"], link["d2h_bytes_per_step"]
                bound = max(h / r["h2d_alone_GBps"], o / r["d2h_alone_GBps"],
                            (h + o) / r["both_GBps"]) / 1e6
                link.update({"measured": r, "bound_ms_per_step": round(bound, 3),
                             "step_frac_of_bound": round(bound / (dt * 1e3 / K), 4)})
        detail["host_link"] = link
    if host_rate:
        detail["host_ids_rate"] = host_rate
    res["detail"] = detail
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on the same tables")
        res["cpu_baseline"] = cpu_baseline(w, host.arrays, host_batches, args.cpu_seconds)
    host.close()
    pool.shutdown()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
