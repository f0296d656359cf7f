"""Python binding of the scratchpad C ABI (include/scratchpipe.h).

Argument marshalling only: every step of planning, filling, forward and
backward runs in the HIP library.  There is no fallback; if the library is not
built, loading fails with an error.  PyTorch supplies device memory and the
stream (torch.cuda.current_stream()) for forward/backward.
"""
from __future__ import annotations

import ctypes as C
import mmap
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# SCRATCHPIPE_LIB selects another build of the library (for comparing builds)
LIB_PATH = os.environ.get("SCRATCHPIPE_LIB") or os.path.join(_HERE, "libscratchpipe.so")

SP_OK = 0
SP_ERR_INVALID_ARG = -1
SP_ERR_OOM = -2
SP_ERR_CAPACITY = -3
SP_ERR_SEQUENCE = -4
SP_ERR_HIP = -5
SP_ERR_STATE = -6
SP_FLAG_DEBUG_SYNC = 0x1
SP_FLAG_TIMING = 0x2
SP_FLAG_EVENT_WAITS = 0x4
SP_FLAG_POISON = 0x8
SP_FLAG_DEFER_SORTS = 0x10
SP_FILL_MAPPED = 0
SP_FILL_STAGED = 1
FILLS = {"mapped": SP_FILL_MAPPED, "staged": SP_FILL_STAGED}
SP_MAX_AHEAD = 2  # batches after the hold window that sp_plan sorts early
SP_MAX_HOLD_PAST = 4
POLICIES = {"lru": 0, "lfu": 1, "random": 2}  # SP_POLICY_*

_NAMES = {SP_ERR_INVALID_ARG: "SP_ERR_INVALID_ARG", SP_ERR_OOM: "SP_ERR_OOM",
          SP_ERR_CAPACITY: "SP_ERR_CAPACITY", SP_ERR_SEQUENCE: "SP_ERR_SEQUENCE",
          SP_ERR_HIP: "SP_ERR_HIP", SP_ERR_STATE: "SP_ERR_STATE"}


class SPError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_NAMES.get(status, status)}: {msg}")
        self.status = status


class sp_config(C.Structure):
    _fields_ = [("num_tables", C.c_int32), ("rows", C.POINTER(C.c_int64)), ("dim", C.c_int32),
                ("slots", C.POINTER(C.c_int64)), ("lookahead", C.c_int32),
                ("host_tables", C.POINTER(C.c_void_p)), ("max_batch", C.c_int32),
                ("max_ids", C.c_int64), ("flags", C.c_uint32), ("device", C.c_int32),
                ("policy", C.c_int32), ("hold_past", C.c_int32), ("seed", C.c_uint64),
                ("max_table_ids", C.c_int64), ("prefetch", C.c_int32), ("fill", C.c_int32)]


class sp_batch(C.Structure):
    _fields_ = [("batch", C.c_int32), ("nnz", C.c_int64), ("ids", C.c_void_p),
                ("bag_off", C.c_void_p), ("on_device", C.c_int32)]


_STAT_I64 = ["plans", "updates", "lookups", "unique", "hits", "misses", "evictions", "bytes_fill",
             "bytes_writeback", "hash_rebuilds", "chunks", "min_capacity_margin", "device_bytes",
             "pinned_bytes"]
_STAT_F64 = ["ms_forward", "ms_backward", "ms_combine", "ms_plan", "ms_fill"]
_STAT_CNT = ["timed_forward", "timed_backward", "timed_combine", "timed_plan", "timed_fill"]


_STAT_HOST = ["host_ms_ingest", "host_ms_query", "host_ms_wait", "host_ms_commit", "host_ms_mover"]
_STAT_F64B = ["ms_ingest", "ms_query"]
_STAT_CNTB = ["timed_ingest", "timed_query"]
_STAT_HOSTB = ["host_ms_inputs"]
_STAT_I64B = ["prefetched"]
_STAT_F64C = ["host_ms_gather", "host_ms_fill_join", "ms_h2d"]
_STAT_I64C = ["timed_h2d"]


class sp_stats(C.Structure):
    _fields_ = ([(n, C.c_int64) for n in _STAT_I64] + [(n, C.c_double) for n in _STAT_F64]
                + [(n, C.c_int64) for n in _STAT_CNT] + [(n, C.c_double) for n in _STAT_HOST]
                + [(n, C.c_double) for n in _STAT_F64B] + [(n, C.c_int64) for n in _STAT_CNTB]
                + [(n, C.c_double) for n in _STAT_HOSTB] + [(n, C.c_int64) for n in _STAT_I64B]
                + [(n, C.c_double) for n in _STAT_F64C] + [(n, C.c_int64) for n in _STAT_I64C])


_DUMP_I32 = ["u_table", "u_row", "inv", "m_table", "m_row", "v_slot", "v_old_row", "v_old_use",
             "slot_u", "slot_of"]


class sp_plan_dump(C.Structure):
    _fields_ = ([(n, C.POINTER(C.c_int32)) for n in _DUMP_I32] + [("hit", C.POINTER(C.c_uint8))]
                + [(n, C.c_int64) for n in ("n_unique", "n_miss", "n_evict", "nnz")])


_lib = None


def load():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2205_04702_amd/build.py")
        L = C.CDLL(LIB_PATH)
        h = C.c_void_p
        L.sp_create.argtypes = [C.POINTER(sp_config), C.POINTER(h)]
        L.sp_plan.argtypes = [h, C.POINTER(sp_batch), C.c_int32, C.POINTER(C.c_int64)]
        L.sp_forward.argtypes = [h, C.c_int64, C.c_void_p, C.c_void_p]
        L.sp_backward_update.argtypes = [h, C.c_int64, C.c_void_p, C.c_float, C.c_void_p]
        L.sp_backward_update_static.argtypes = [h, C.c_int64, C.c_void_p, C.c_float, C.c_void_p]
        L.sp_flush.argtypes = [h]
        L.sp_sync.argtypes = [h]
        L.sp_get_stats.argtypes = [h, C.POINTER(sp_stats)]
        L.sp_set_flags.argtypes = [h, C.c_uint32]
        L.sp_debug_plan.argtypes = [h, C.c_int64, C.POINTER(sp_plan_dump)]
        L.sp_destroy.argtypes = [h]
        L.sp_destroy.restype = None
        L.sp_last_error.argtypes = [h]
        L.sp_last_error.restype = C.c_char_p
        L.sp_host_alloc.argtypes = [C.c_size_t, C.POINTER(C.c_void_p)]
        L.sp_host_free.argtypes = [C.c_void_p]
        L.sp_host_free.restype = None
        for n in ("sp_create", "sp_plan", "sp_forward", "sp_backward_update",
                  "sp_backward_update_static", "sp_flush", "sp_sync",
                  "sp_get_stats", "sp_set_flags", "sp_debug_plan", "sp_host_alloc"):
            getattr(L, n).restype = C.c_int32
        _lib = L
    return _lib


def _check(st: int, handle=None):
    if st != SP_OK:
        msg = load().sp_last_error(handle)
        raise SPError(st, msg.decode() if msg else "")


# ----------------------------------------------------------------------------- C-ABI names

def sp_host_alloc(nbytes: int) -> int:
    p = C.c_void_p()
    _check(load().sp_host_alloc(nbytes, C.byref(p)))
    return p.value


def sp_host_free(ptr: int) -> None:
    load().sp_host_free(ptr)


def sp_create(cfg: sp_config) -> int:
    h = C.c_void_p()
    _check(load().sp_create(C.byref(cfg), C.byref(h)))
    return h.value


def sp_plan(handle: int, window, n: int) -> int:
    t = C.c_int64(-1)
    _check(load().sp_plan(handle, window, n, C.byref(t)), handle)
    return t.value


def sp_forward(handle: int, ticket: int, d_out: int, stream: int) -> None:
    _check(load().sp_forward(handle, ticket, d_out, stream), handle)


def sp_backward_update(handle: int, ticket: int, d_grad: int, lr: float, stream: int) -> None:
    _check(load().sp_backward_update(handle, ticket, d_grad, C.c_float(lr), stream), handle)


def sp_backward_update_static(handle: int, ticket: int, d_grad: int, lr: float,
                              stream: int) -> None:
    _check(load().sp_backward_update_static(handle, ticket, d_grad, C.c_float(lr), stream), handle)


def sp_flush(handle: int) -> None:
    _check(load().sp_flush(handle), handle)


def sp_sync(handle: int) -> None:
    _check(load().sp_sync(handle), handle)


def sp_get_stats(handle: int) -> dict:
    s = sp_stats()
    _check(load().sp_get_stats(handle, C.byref(s)), handle)
    return {n: getattr(s, n) for n, _ in sp_stats._fields_}


def sp_set_flags(handle: int, flags: int) -> None:
    _check(load().sp_set_flags(handle, flags), handle)


def sp_debug_plan(handle: int, ticket: int, nnz_cap: int, miss_cap: int | None = None) -> dict:
    """miss_cap: room for the miss arrays (in prefetch mode the nnz of the planned and
    the next batch together); nnz_cap by default."""
    cap = max(int(nnz_cap), 1)
    mcap = max(int(miss_cap if miss_cap is not None else nnz_cap), 1)
    misses = ("m_table", "m_row", "v_slot", "v_old_row", "v_old_use")
    arrays = {n: np.empty(mcap if n in misses else cap, np.int32) for n in _DUMP_I32}
    hit = np.empty(cap, np.uint8)
    d = sp_plan_dump()
    for n in _DUMP_I32:
        setattr(d, n, arrays[n].ctypes.data_as(C.POINTER(C.c_int32)))
    d.hit = hit.ctypes.data_as(C.POINTER(C.c_uint8))
    _check(load().sp_debug_plan(handle, ticket, C.byref(d)), handle)
    nU, nM, nnz = d.n_unique, d.n_miss, d.nnz
    out = {n: arrays[n][:nU].copy() for n in ("u_table", "u_row", "slot_u")}
    out["hit"] = hit[:nU].copy()
    out.update({n: arrays[n][:nM].copy() for n in ("m_table", "m_row", "v_slot", "v_old_row",
                                                  "v_old_use")})
    out.update({n: arrays[n][:nnz].copy() for n in ("inv", "slot_of")})
    out["n_evict"] = d.n_evict
    return out


def sp_destroy(handle: int) -> None:
    if handle:
        load().sp_destroy(handle)


def sp_last_error(handle=None) -> str:
    m = load().sp_last_error(handle)
    return m.decode() if m else ""


def worst_case_scratchpad_bytes(tables, pooling, batch, dim, window) -> int:
    """Storage needed when no ID of the window's batches repeats (Sec. VI-D):
    tables x IDs per table per sample x batch x row bytes x window batches."""
    return int(tables) * int(pooling) * int(batch) * int(dim) * 4 * int(window)


# ----------------------------------------------------------------------------- convenience

class HostTables:
    """fp32 tables in pinned, device-mapped host memory, exposed as numpy arrays."""

    def __init__(self, rows, dim: int):
        self.ptrs, self.arrays = [], []
        try:
            for r in rows:
                n = int(r) * dim
                p = sp_host_alloc(n * 4)
                self.ptrs.append(p)
                buf = (C.c_float * n).from_address(p)
                self.arrays.append(np.ctypeslib.as_array(buf).reshape(int(r), dim))
        except Exception:
            self.close()
            raise

    def __getitem__(self, t):
        return self.arrays[t]

    def __len__(self):
        return len(self.arrays)

    def close(self):
        self.arrays = []
        for p in self.ptrs:
            sp_host_free(p)
        self.ptrs = []


class PageableTables:
    """fp32 host tables in ordinary (pageable) memory, for the staged fill, allocated
    lazily by the OS (pages appear when first written).  With huge_pages (the
    default) each table is an anonymous mapping advised for transparent huge pages
    before any page is touched: the fill's host threads read and write rows at
    random places in the tables, and 2 MB pages take most address translations off
    that path.  Where the kernel does not allow it the advice changes nothing."""

    def __init__(self, rows, dim: int, huge_pages: bool = True):
        self._maps = []
        self.arrays = []
        for r in rows:
            n = int(r) * dim
            if huge_pages and hasattr(mmap, "MADV_HUGEPAGE"):
                m = mmap.mmap(-1, max(4 * n, 1), flags=mmap.MAP_PRIVATE | mmap.MAP_ANONYMOUS)
                try:
                    m.madvise(mmap.MADV_HUGEPAGE)
                except OSError:
                    pass
                self._maps.append(m)
                self.arrays.append(np.frombuffer(m, dtype=np.float32, count=n).reshape(int(r), dim))
            else:
                self.arrays.append(np.empty((int(r), dim), dtype=np.float32))
        self.ptrs = [int(a.ctypes.data) for a in self.arrays]

    def __getitem__(self, t):
        return self.arrays[t]

    def __len__(self):
        return len(self.arrays)

    def close(self):
        self.arrays = []
        self.ptrs = []
        for m in self._maps:
            try:
                m.close()
            except BufferError:  # an array of it is still referenced: freed with it
                pass
        self._maps = []


def host_tables(rows, dim: int, fill: str = "mapped", huge_pages: bool = True):
    """Host tables for a context: pinned and device-mapped for the mapped fill,
    ordinary memory (in transparent huge pages unless huge_pages is false) for the
    staged fill."""
    return PageableTables(rows, dim, huge_pages) if fill == "staged" else HostTables(rows, dim)


def _ptr(x) -> int:
    if x is None:
        return 0
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    return int(x.ctypes.data)


def _on_device(x) -> int:
    return int(bool(getattr(x, "is_cuda", False)))


def _stream_handle(stream) -> int:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return int(getattr(stream, "cuda_stream", stream) or 0)


class ScratchPipe:
    """One scratchpad context over host tables (see include/scratchpipe.h).

    policy: "lru", "lfu" or "random"; hold_past: earlier batches held as well;
    seed: the random policy's stream; max_table_ids: 0 or the most IDs any one
    table has in a batch (a promise that is checked); prefetch: depth d (True =
    1): plans also fill the missing rows of their next d batches; fill:
    "mapped" (zero-copy from pinned, device-mapped tables, HostTables) or
    "staged" (host gather, then copies; any host tables, PageableTables)."""

    def __init__(self, rows, dim, slots, lookahead, host_tables, max_batch, max_ids,
                 flags: int = 0, device: int = 0, policy: str = "lru", hold_past: int = 0,
                 seed: int = 0, max_table_ids: int = 0, prefetch=0,
                 fill: str = "mapped"):
        self.T = len(rows)
        self.prefetch = int(prefetch)  # depth (True = 1)
        self.max_ids = int(max_ids)
        self.dim = dim
        self._rows = (C.c_int64 * self.T)(*[int(r) for r in rows])
        self._slots = (C.c_int64 * self.T)(*[int(s) for s in slots])
        self._tabs = (C.c_void_p * self.T)(*host_tables.ptrs)
        cfg = sp_config(num_tables=self.T, rows=self._rows, dim=dim, slots=self._slots,
                        lookahead=lookahead, host_tables=self._tabs, max_batch=max_batch,
                        max_ids=max_ids, flags=flags, device=device, policy=POLICIES[policy],
                        hold_past=hold_past, seed=seed, max_table_ids=max_table_ids,
                        prefetch=self.prefetch, fill=FILLS[fill])
        self.handle = sp_create(cfg)
        self._desc_cache = {}

    def _describe(self, ids, off) -> sp_batch:
        B = (len(off) - 1) // self.T
        nnz = int(ids.shape[0])
        return sp_batch(batch=B, nnz=nnz, ids=_ptr(ids) if nnz else None, bag_off=_ptr(off),
                        on_device=_on_device(ids))

    def plan(self, window) -> int:
        """window: [(ids, bag_off), ...] as int32 numpy arrays or int32 device tensors.

        Device tensors must hold their batch already (synchronise the stream that
        wrote them first: the library reads them on its own stream) and stay
        unchanged until a plan that holds the batch (window index <= lookahead)
        has returned."""
        n = len(window)
        arr = (sp_batch * n)()
        keep = []
        for i, (ids, off) in enumerate(window):
            if hasattr(ids, "data_ptr"):
                # device tensors: descriptors cached per tensor pair (the cache
                # holds the tensors, so their addresses stay valid)
                key = (id(ids), id(off))
                hit = self._desc_cache.get(key)
                if hit is None:
                    if len(self._desc_cache) >= 64:
                        self._desc_cache.pop(next(iter(self._desc_cache)))
                    hit = (self._describe(ids, off), ids, off)
                    self._desc_cache[key] = hit
                arr[i] = hit[0]
            else:
                ids = np.ascontiguousarray(ids, dtype=np.int32)
                off = np.ascontiguousarray(off, dtype=np.int32)
                keep.append((ids, off))
                arr[i] = self._describe(ids, off)
        return sp_plan(self.handle, arr, n)

    def forward(self, ticket: int, out, stream=None) -> None:
        sp_forward(self.handle, ticket, _ptr(out), _stream_handle(stream))

    def backward_update(self, ticket: int, grad, lr: float, stream=None) -> None:
        sp_backward_update(self.handle, ticket, _ptr(grad), lr, _stream_handle(stream))

    def backward_update_static(self, ticket: int, grad, lr: float, stream=None) -> None:
        sp_backward_update_static(self.handle, ticket, _ptr(grad), lr, _stream_handle(stream))

    def flush(self) -> None:
        sp_flush(self.handle)

    def sync(self) -> None:
        sp_sync(self.handle)

    def stats(self) -> dict:
        return sp_get_stats(self.handle)

    def set_flags(self, flags: int) -> None:
        sp_set_flags(self.handle, flags)

    def debug_plan(self, ticket: int, nnz: int) -> dict:
        # prefetch mode: misses of the planned batch and its successors (each at most max_ids)
        return sp_debug_plan(self.handle, ticket, nnz, nnz + self.prefetch * self.max_ids)

    def close(self) -> None:
        if getattr(self, "handle", None):
            sp_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
