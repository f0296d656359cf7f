"""Drive the HIP scratchpad and the CPU oracle side by side on the same inputs."""
from __future__ import annotations

import numpy as np

from oracle import oracle
from paper_2205_04702_amd import workload as wl
from paper_2205_04702_amd.scratchpipe import SP_MAX_AHEAD, ScratchPipe, host_tables

PLAN_FIELDS = ("u_table", "u_row", "inv", "hit", "m_table", "m_row", "v_slot", "v_old_row",
               "v_old_use", "slot_u", "slot_of")
REL_TOL = 1e-5  # per-row max |gpu - ref| / max |ref|


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per row: infinity-norm of the difference over infinity-norm of the reference."""
    got = got.reshape(ref.shape[0], -1).astype(np.float64)
    ref = ref.reshape(ref.shape[0], -1).astype(np.float64)
    den = np.abs(ref).max(axis=1)
    num = np.abs(got - ref).max(axis=1)
    return np.where(den > 0, num / np.where(den > 0, den, 1), num)


def compare_plan(step, dump, ref, T, B):
    for f in PLAN_FIELDS:
        a = np.asarray(dump[f])
        b = np.asarray(getattr(ref, f))
        if f == "hit":
            a, b = a.astype(np.uint8), b.astype(np.uint8)
        assert a.shape == b.shape, f"step {step}: {f} shape {a.shape} vs {b.shape}"
        if not np.array_equal(a, b):
            bad = np.nonzero(a != b)[0][:5]
            raise AssertionError(f"step {step}: plan field {f} differs at {bad.tolist()}: "
                                 f"gpu {a[bad].tolist()} oracle {b[bad].tolist()}")
    assert dump["n_evict"] == ref.n_evict, f"step {step}: evictions {dump['n_evict']} vs {ref.n_evict}"


def table_bound(w, batches):
    """The most IDs any one table has in any of the batches."""
    B = w.batch
    return max(int(np.max(np.diff(np.asarray(off)[::B]))) for _, off in batches) if batches else 0


def _bound(w, batches, max_table_ids):
    return table_bound(w, batches) if max_table_ids == "auto" else int(max_table_ids)


def run_gpu(w, batches, host, first=0, last=None, flags=0, prepare_ahead=0, policy="lru",
            hold_past=0, seed=0, max_table_ids="auto", prefetch=False, fill="mapped"):
    """Train batches[first:last] on the GPU only (fresh context over `host`), then flush.
    prepare_ahead: how many batches after each window to hand over for early sorting."""
    import torch
    dev = torch.device("cuda:0")
    n = len(batches)
    last = n if last is None else last
    T, B, D, L = w.tables, w.batch, w.dim, w.lookahead
    max_ids = max(int(b[0].size) for b in batches)
    sp = ScratchPipe(w.rows, D, w.slots, L, host, max_batch=B, max_ids=max(max_ids, 1), flags=flags,
                     policy=policy, hold_past=hold_past, seed=seed,
                     max_table_ids=_bound(w, batches, max_table_ids), prefetch=prefetch, fill=fill)
    try:
        out = torch.zeros((T * B, D), dtype=torch.float32, device=dev)
        for u in range(first, last):
            idx = list(range(u, min(u + L, last - 1) + 1))
            idx += [q for q in range(u + L + 1, u + L + 1 + int(prepare_ahead)) if q < last]
            ticket = sp.plan([batches[q] for q in idx])
            sp.forward(ticket, out)
            sp.backward_update(ticket, torch.from_numpy(wl.grads(w, u)).to(dev), w.lr)
        sp.flush()
        return sp.stats()
    finally:
        sp.close()


def fresh_host(w, fill="mapped"):
    host = host_tables(w.rows, w.dim, fill)
    for t in range(w.tables):
        wl.init_table(w, t, out=host[t])
    return host


def make_inputs(w, steps=None, ragged=None):
    n = w.steps if steps is None else steps
    if ragged:
        batches = [wl.ragged_batch(w, s, ragged) for s in range(n)]
    else:
        batches = [wl.batch(w, s) for s in range(n)]
    return batches


def run_parity(w, batches=None, *, check_plan_steps="all", check_fwd_steps="all", flags=0,
               device_ids=False, ref_tables=None, sync_each_step=True, compare_tables=True,
               return_tables=False, steps=None, prepare_ahead=0, policy="lru", hold_past=0,
               seed=0, max_table_ids="auto", prefetch=False, fill="mapped",
               overwrite_held_ids=False, static_backward=False):
    """Train w on the GPU and with the oracle; assert parity; return a summary.

    prepare_ahead: also hand the GPU that many batches after the window
    (prepared in advance, not held); the oracle always sees the plain window.
    policy, hold_past, seed: replacement policy and past window of both planners.
    max_table_ids: the bound handed to the library ("auto": the batches' own maximum,
    which sorts tables of up to 8192 IDs in LDS; 0: no bound, the general path).
    prefetch: both planners also fill the next batch's missing rows.
    fill: how the GPU brings missing rows in ("mapped" or "staged").
    overwrite_held_ids: with device_ids, set every ID of the batches a plan held to
    an out-of-range row once the plan returns (the library must not read a batch
    again once a plan that holds it has returned).
    static_backward: update through the allocation-free sp_backward_update_static."""
    import torch
    dev = torch.device("cuda:0")
    if batches is None:
        batches = make_inputs(w, steps)
    n = len(batches)
    T, B, D, L = w.tables, w.batch, w.dim, w.lookahead
    max_ids = max(int(b[0].size) for b in batches)
    host = host_tables(w.rows, D, fill)
    for t in range(T):
        wl.init_table(w, t, out=host[t])
    ref = ref_tables if ref_tables is not None else [wl.init_table(w, t) for t in range(T)]
    planner = oracle.Planner(w.rows, w.slots, policy, seed, prefetch)
    touched = [np.zeros(r, bool) for r in w.rows]
    dev_batches = None
    if device_ids:
        dev_batches = [(torch.from_numpy(i).to(dev), torch.from_numpy(o).to(dev)) for i, o in batches]
    plan_set = set(range(n)) if check_plan_steps == "all" else set(check_plan_steps)
    fwd_set = set(range(n)) if check_fwd_steps == "all" else set(check_fwd_steps)
    worst_fwd = 0.0
    sp = ScratchPipe(w.rows, D, w.slots, L, host, max_batch=B, max_ids=max(max_ids, 1), flags=flags,
                     policy=policy, hold_past=hold_past, seed=seed,
                     max_table_ids=_bound(w, batches, max_table_ids), prefetch=prefetch, fill=fill)
    try:
        out = torch.zeros((T * B, D), dtype=torch.float32, device=dev)
        for u in range(n):
            win_idx = list(range(u, min(u + L, n - 1) + 1))
            src = dev_batches if device_ids else batches
            gpu_idx = win_idx + [q for q in range(u + L + 1, u + L + 1 + int(prepare_ahead))
                                 if q < n]
            ticket = sp.plan([src[q] for q in gpu_idx])
            assert ticket == u
            if device_ids and overwrite_held_ids:
                for q in win_idx:
                    dev_batches[q][0].fill_(0x7FFFFFFF)
            p = planner.plan([batches[q] for q in win_idx], B,
                             past=batches[max(0, u - hold_past):u])
            if u in plan_set:
                compare_plan(u, sp.debug_plan(ticket, max(int(batches[u][0].size), 1)), p, T, B)
            sp.forward(ticket, out)
            g = wl.grads(w, u)
            gd = torch.from_numpy(g).to(dev)
            (sp.backward_update_static if static_backward else sp.backward_update)(ticket, gd, w.lr)
            ids, off = batches[u]
            o_ref = oracle.train_step(ref, ids, off, B, g, w.lr, want_out=u in fwd_set)
            for t in range(T):
                touched[t][ids[off[t * B]:off[(t + 1) * B]]] = True
            if u in fwd_set:
                torch.cuda.synchronize()
                e = row_rel_err(out.cpu().numpy(), o_ref)
                worst_fwd = max(worst_fwd, float(e.max(initial=0.0)))
                assert e.max(initial=0.0) <= REL_TOL, f"step {u}: forward rel err {e.max()}"
            elif sync_each_step:
                torch.cuda.synchronize()
        sp.flush()
        stats = sp.stats()
    finally:
        sp.close()
    worst_tab = 0.0
    if compare_tables:
        for t in range(T):
            got, exp = host[t], ref[t]
            assert np.array_equal(got[~touched[t]], exp[~touched[t]]), f"table {t}: untouched rows changed"
            e = row_rel_err(got[touched[t]], exp[touched[t]])
            worst_tab = max(worst_tab, float(e.max(initial=0.0)))
            assert e.max(initial=0.0) <= REL_TOL, f"table {t}: row rel err {e.max()}"
    tables = [host[t].copy() for t in range(T)] if return_tables else None
    host.close()
    return {"stats": stats, "worst_fwd": worst_fwd, "worst_table": worst_tab, "tables": tables}


# ----------------------------------------------------------------------------- full-size configs

def touched_rows(w, batches, steps):
    """Per table: sorted unique rows read by batches[0:steps], the only rows training touches."""
    T, B = w.tables, w.batch
    out = []
    for t in range(T):
        parts = [b[0][int(b[1][t * B]):int(b[1][(t + 1) * B])] for b in batches[:steps]]
        out.append(np.unique(np.concatenate(parts)) if parts else np.zeros(0, np.int32))
    return out


def row_values(t, rows, dim):
    """Deterministic values in [-0.05, 0.05) for (table, row, column); cheap to make for a
    few rows of a huge table (full initialisation of 100+ GB would dominate the test)."""
    r = np.asarray(rows, dtype=np.int64)[:, None]
    c = np.arange(dim, dtype=np.int64)[None, :]
    h = (r * 2654435761 + c * 40503 + (t + 1) * 977) % 2003
    return ((h - 1001) * (0.05 / 1002)).astype(np.float32)


def run_sampled_parity(w, steps, *, check_plan_steps, check_fwd_steps, say=print, policy="lru",
                       hold_past=0, seed=0, max_table_ids="auto", prefetch=False, fill="mapped",
                       host_ids=False):
    """A full-size workload driven as the benchmark drives it (the SP_MAX_AHEAD batches
    after the window handed over early; IDs in device memory, or host memory with host_ids) for
    `steps` steps.

    Only rows that the trained batches read are initialised (plus sentinel rows elsewhere);
    the oracle trains compact copies of exactly those rows (uncached training touches no
    other row, so its arithmetic is the same).  Checks: plans bit-exact against the
    reference planner at `check_plan_steps`, forward outputs at `check_fwd_steps`, every
    touched row after flush, and sentinel rows unchanged."""
    import time
    import torch
    dev = torch.device("cuda:0")
    T, B, D, L = w.tables, w.batch, w.dim, w.lookahead
    t0 = time.perf_counter()
    ahead = SP_MAX_AHEAD
    batches = [wl.batch(w, s) for s in range(steps + L + ahead)]
    rows = touched_rows(w, batches, steps)
    say(f"  inputs {time.perf_counter() - t0:.1f}s, touched rows {sum(r.size for r in rows)}")
    host = host_tables(w.rows, D, fill)
    ref = []
    sentinels = []
    for t in range(T):
        v = row_values(t, rows[t], D)
        host[t][rows[t]] = v
        ref.append(v.copy())
        cand = np.linspace(0, w.rows[t] - 1, num=min(w.rows[t], 512), dtype=np.int64)
        s = np.setdiff1d(cand, rows[t])
        host[t][s] = row_values(t + 1000, s, D)
        sentinels.append(s)
    say(f"  host tables ready {time.perf_counter() - t0:.1f}s")

    def compact(u):
        ids, off = batches[u]
        parts = []
        for t in range(T):
            seg = ids[int(off[t * B]):int(off[(t + 1) * B])]
            parts.append(np.searchsorted(rows[t], seg).astype(np.int32))
        return np.concatenate(parts), off

    dev_batches = batches if host_ids else \
        [(torch.from_numpy(i).to(dev), torch.from_numpy(o).to(dev)) for i, o in batches]
    planner = oracle.Planner(w.rows, w.slots, policy, seed, prefetch)
    max_ids = max(int(b[0].size) for b in batches)
    sp = ScratchPipe(w.rows, D, w.slots, L, host, max_batch=B, max_ids=max_ids, policy=policy,
                     hold_past=hold_past, seed=seed,
                     max_table_ids=_bound(w, batches, max_table_ids), prefetch=prefetch, fill=fill)
    worst_fwd = 0.0
    try:
        out = torch.zeros((T * B, D), dtype=torch.float32, device=dev)
        for u in range(steps):
            ticket = sp.plan([dev_batches[q] for q in range(u, u + L + 1 + ahead)])
            p = planner.plan([batches[q] for q in range(u, u + L + 1)], B,
                             past=batches[max(0, u - hold_past):u])
            if u in check_plan_steps:
                compare_plan(u, sp.debug_plan(ticket, int(batches[u][0].size)), p, T, B)
            sp.forward(ticket, out)
            g = wl.grads(w, u)
            sp.backward_update(ticket, torch.from_numpy(g).to(dev), w.lr)
            cid, off = compact(u)
            o_ref = oracle.train_step(ref, cid, off, B, g, w.lr, want_out=u in check_fwd_steps)
            if u in check_fwd_steps:
                torch.cuda.synchronize()
                e = row_rel_err(out.cpu().numpy(), o_ref)
                worst_fwd = max(worst_fwd, float(e.max(initial=0.0)))
                assert e.max(initial=0.0) <= REL_TOL, f"step {u}: forward rel err {e.max()}"
            say(f"  step {u} done {time.perf_counter() - t0:.1f}s")
        sp.flush()
        stats = sp.stats()
    finally:
        sp.close()
    worst_tab = 0.0
    try:
        for t in range(T):
            e = row_rel_err(host[t][rows[t]], ref[t])
            worst_tab = max(worst_tab, float(e.max(initial=0.0)))
            assert e.max(initial=0.0) <= REL_TOL, f"table {t}: row rel err {e.max()}"
            s = sentinels[t]
            assert np.array_equal(host[t][s], row_values(t + 1000, s, D)), f"table {t}: sentinel changed"
    finally:
        host.close()
    say(f"  checked {time.perf_counter() - t0:.1f}s")
    return {"stats": stats, "worst_fwd": worst_fwd, "worst_table": worst_tab}
