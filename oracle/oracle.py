"""Python face of the CPU oracle.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product library.

  forward / backward_sgd / train_step   uncached embedding-bag SGD (O1)
  Planner                               reference scratchpad planner (O2), with the
                                        LRU, LFU and random replacement policies
                                        (Sec. VI-E) and an optional past window
  CachedSimulator                       O2's plans applied to a CPU copy of the
                                        scratchpad, trained with O1's arithmetic (O3)

The method's claim is that training through the scratchpad gives exactly the
result of uncached training (Sec. II-D and the opening of Sec. VI); O3 must
therefore reproduce O1's tables bit for bit.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIB selects another build (the sanitizer build of the CPU checks)
_LIB_PATH = os.environ.get("ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

OK, ERR_INVALID, ERR_CAPACITY = 0, -1, -3
POLICIES = {"lru": 0, "lfu": 1, "random": 2}  # replacement policies of Sec. VI-E

_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = C.CDLL(_LIB_PATH)
        L.orc_forward.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_void_p, _i32p, _i32p, _f32p]
        L.orc_backward_sgd.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_void_p, _i32p, _i32p,
                                       _f32p, C.c_float]
        L.orc_max_threads.restype = C.c_int
        L.orc_planner_create.restype = C.c_void_p
        L.orc_planner_create.argtypes = [C.c_int32, _i64p, _i64p, C.c_int32, C.c_uint64]
        L.orc_splitmix64_nth.restype = C.c_uint64
        L.orc_splitmix64_nth.argtypes = [C.c_uint64, C.c_uint64]
        L.orc_random_priority.restype = C.c_uint32
        L.orc_random_priority.argtypes = [C.c_uint64, C.c_int32, C.c_int64, C.c_int32]
        L.orc_planner_destroy.argtypes = [C.c_void_p]
        L.orc_planner_step.argtypes = [C.c_void_p]
        L.orc_planner_step.restype = C.c_int32
        L.orc_planner_state.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                        C.c_void_p]
        L.orc_planner_plan_pf.restype = C.c_int32
        L.orc_planner_plan_pf.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_int32,
                                          C.c_int32, _i32p, _i32p, _i32p, _u8p, _i32p, _i32p,
                                          _i32p, _i32p, _i32p, _i32p, _i32p, _i64p]
        L.orc_planner_plan.restype = C.c_int32
        L.orc_planner_plan.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_int32,
                                       _i32p, _i32p, _i32p, _u8p, _i32p, _i32p, _i32p, _i32p,
                                       _i32p, _i32p, _i32p, _i64p]
        _lib = L
    return _lib


def max_threads() -> int:
    return int(lib().orc_max_threads())


def splitmix64_nth(seed: int, n: int) -> int:
    """Output number n (n >= 1) of SplitMix64 started from state `seed`."""
    return int(lib().orc_splitmix64_nth(C.c_uint64(seed), C.c_uint64(n)))


def random_priority(seed: int, u: int, g: int, last_use: int) -> int:
    """Random-eviction priority of global slot g at plan u (0 for a never-used slot)."""
    return int(lib().orc_random_priority(C.c_uint64(seed), u, g, last_use))


def _ptr_array(arrays):
    arr = (C.c_void_p * len(arrays))()
    for i, a in enumerate(arrays):
        arr[i] = a.ctypes.data
    return arr


def _check_tables(tables, D):
    for t in tables:
        assert t.dtype == np.float32 and t.flags.c_contiguous and t.ndim == 2 and t.shape[1] == D


# ----------------------------------------------------------------------------- O1

def forward(tables, ids, bag_off, B: int) -> np.ndarray:
    """Pooled forward of one batch: float32 [T*B, D]."""
    D = tables[0].shape[1]
    _check_tables(tables, D)
    out = np.empty((len(tables) * B, D), dtype=np.float32)
    lib().orc_forward(len(tables), B, D, _ptr_array(tables), np.ascontiguousarray(ids, np.int32),
                      np.ascontiguousarray(bag_off, np.int32), out)
    return out


def backward_sgd(tables, ids, bag_off, B: int, grad, lr: float) -> None:
    """Coalesce the bag gradients per row and apply W -= lr*g in place."""
    D = tables[0].shape[1]
    _check_tables(tables, D)
    g = np.ascontiguousarray(grad, dtype=np.float32).reshape(len(tables) * B, D)
    lib().orc_backward_sgd(len(tables), B, D, _ptr_array(tables),
                           np.ascontiguousarray(ids, np.int32),
                           np.ascontiguousarray(bag_off, np.int32), g, C.c_float(lr))


def train_step(tables, ids, bag_off, B: int, grad, lr: float, want_out: bool = False):
    out = forward(tables, ids, bag_off, B) if want_out else None
    backward_sgd(tables, ids, bag_off, B, grad, lr)
    return out


# ----------------------------------------------------------------------------- O2

class PlanResult:
    """One plan's decisions; field meanings follow orc_planner_plan."""

    __slots__ = ("u_table", "u_row", "inv", "hit", "m_table", "m_row", "v_slot", "v_old_row",
                 "v_old_use", "slot_u", "slot_of", "n_evict", "n_prefetch")

    def keys(self):
        return [s for s in self.__slots__ if s not in ("n_evict", "n_prefetch")]


class Planner:
    """Reference planner (O2).  plan() returns a PlanResult or raises PlanError.

    policy: "lru" (the default of Sec. VI-E), "lfu" or "random"; seed feeds the
    random policy's draws.  prefetch: depth d (True = 1): each plan also fills the
    rows of the first d successor batches of its window that are neither cached
    nor in an earlier batch of the window (orc_planner_plan_pf); they follow the
    planned batch's misses, per table, batch by batch.
    """

    def __init__(self, rows, slots, policy: str = "lru", seed: int = 0, prefetch=0):
        self.T = len(rows)
        self.rows = np.asarray(rows, dtype=np.int64)
        self.slots = np.asarray(slots, dtype=np.int64)
        self.slot_base = np.concatenate([[0], np.cumsum(self.slots)]).astype(np.int64)
        self.policy, self.seed = policy, int(seed)
        self.prefetch = int(prefetch)
        self._h = lib().orc_planner_create(self.T, self.rows, self.slots, POLICIES[policy],
                                           C.c_uint64(self.seed))

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.orc_planner_destroy(h)

    @property
    def step(self) -> int:
        return int(lib().orc_planner_step(self._h))

    def state(self, t: int):
        kos = np.empty(int(self.slots[t]), np.int32)
        lu = np.empty(int(self.slots[t]), np.int32)
        sor = np.empty(int(self.rows[t]), np.int32)
        lib().orc_planner_state(self._h, t, kos.ctypes.data, lu.ctypes.data, sor.ctypes.data, None)
        return kos, lu, sor

    def uses(self, t: int):
        """Per-slot use counts of table t (the LFU frequency)."""
        n = np.empty(int(self.slots[t]), np.int32)
        lib().orc_planner_state(self._h, t, None, None, None, n.ctypes.data)
        return n

    def plan(self, window, B: int, past=()) -> PlanResult:
        """window: list of (ids, bag_off) for the planned batch and its visible successors;
        past: earlier batches whose cached rows are held as well (the past window)."""
        npf = min(self.prefetch, len(window) - 1)  # successors in the look-forward window
        window = list(window) + list(past)
        ids_l = [np.ascontiguousarray(w[0], np.int32) for w in window]
        off_l = [np.ascontiguousarray(w[1], np.int32) for w in window]
        nnz = int(off_l[0][-1])
        cap = max(nnz, 1)
        mcap = cap + sum(int(ids_l[w].size) for w in range(1, npf + 1))
        r = PlanResult()
        r.u_table, r.u_row, r.inv = (np.empty(cap, np.int32) for _ in range(3))
        r.hit = np.empty(cap, np.uint8)
        r.slot_u, r.slot_of = np.empty(cap, np.int32), np.empty(cap, np.int32)
        (r.m_table, r.m_row, r.v_slot, r.v_old_row,
         r.v_old_use) = (np.empty(mcap, np.int32) for _ in range(5))
        counts = np.zeros(4, np.int64)
        if npf == 0:
            st = lib().orc_planner_plan(self._h, len(window), _ptr_array(ids_l), _ptr_array(off_l),
                                        B, r.u_table, r.u_row, r.inv, r.hit, r.m_table, r.m_row,
                                        r.v_slot, r.v_old_row, r.v_old_use, r.slot_u, r.slot_of,
                                        counts)
        else:
            st = lib().orc_planner_plan_pf(self._h, len(window), _ptr_array(ids_l),
                                           _ptr_array(off_l), B, npf, r.u_table,
                                           r.u_row, r.inv, r.hit, r.m_table, r.m_row, r.v_slot,
                                           r.v_old_row, r.v_old_use, r.slot_u, r.slot_of, counts)
        if st != OK:
            raise PlanError(st)
        nU, nM = int(counts[0]), int(counts[1])
        r.n_prefetch = int(counts[3])
        for f in ("u_table", "u_row", "hit", "slot_u"):
            setattr(r, f, getattr(r, f)[:nU].copy())
        for f in ("m_table", "m_row", "v_slot", "v_old_row", "v_old_use"):
            setattr(r, f, getattr(r, f)[:nM].copy())
        r.inv, r.slot_of = r.inv[:nnz].copy(), r.slot_of[:nnz].copy()
        r.n_evict = int(counts[2])
        return r


class PlanError(RuntimeError):
    def __init__(self, status):
        super().__init__({ERR_INVALID: "invalid input", ERR_CAPACITY: "capacity"}.get(status, status))
        self.status = status


# ----------------------------------------------------------------------------- O3

class CachedSimulator:
    """Scratchpad training on the CPU: O2 decides, O1's arithmetic trains.

    host_tables are the authoritative copies of rows not in the scratchpad;
    they are modified in place (write-backs, flush).
    """

    def __init__(self, host_tables, slots, check_residency: bool = True, policy: str = "lru",
                 seed: int = 0, prefetch=0):
        self.host = host_tables
        self.D = host_tables[0].shape[1]
        rows = [t.shape[0] for t in host_tables]
        self.planner = Planner(rows, slots, policy, seed, prefetch)
        self.storage = np.zeros((int(self.planner.slot_base[-1]), self.D), np.float32)
        self.check = check_residency
        self.writebacks = 0

    def _views(self):
        b = self.planner.slot_base
        return [self.storage[b[t]:b[t + 1]] for t in range(len(self.host))]

    def step(self, window, B: int, grad, lr: float, want_out: bool = False, past=()):
        p = self.planner.plan(window, B, past)
        base = self.planner.slot_base
        # write back evicted rows (they were trained, so they are dirty), then fill misses
        for i in range(p.m_row.size):
            t, v, old = int(p.m_table[i]), int(p.v_slot[i]), int(p.v_old_row[i])
            if old >= 0:
                self.host[t][old] = self.storage[v]
                self.writebacks += 1
            self.storage[v] = self.host[t][p.m_row[i]]
        ids, off = window[0]
        T = len(self.host)
        local = p.slot_of.astype(np.int64)
        for t in range(T):
            j0, j1 = int(off[t * B]), int(off[(t + 1) * B])
            local[j0:j1] -= base[t]
        local = local.astype(np.int32)
        if self.check:
            for t in range(T):
                j0, j1 = int(off[t * B]), int(off[(t + 1) * B])
                kos, _, _ = self.planner.state(t)
                assert np.array_equal(kos[local[j0:j1]], np.asarray(ids[j0:j1])), "not resident"
        out = train_step(self._views(), local, off, B, grad, lr, want_out)
        return p, out

    def flush(self):
        base = self.planner.slot_base
        for t in range(len(self.host)):
            kos, _, _ = self.planner.state(t)
            occ = np.nonzero(kos >= 0)[0]
            self.host[t][kos[occ]] = self.storage[base[t] + occ]
