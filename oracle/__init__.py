"""CPU oracle of the multi-signal growing-network iteration — TEST INFRASTRUCTURE.

This package defines the results the HIP path is checked against.  It shares no code
with the product package and never imports it.  Only ``tests/``, the smoke check and the
CPU-baseline leg of ``bench.py`` may use it.

The arithmetic lives in ``gsn_oracle.c`` (plain sequential C, see its header for the
paper passages each step follows and the readings of points the paper leaves open).
This module only marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liborc.so")

OK = 0
E_INVAL = -1
E_CAPACITY = -2
E_STATE = -4


class _Params(ctypes.Structure):
    _fields_ = [
        ("eps_b", ctypes.c_float),
        ("eps_n", ctypes.c_float),
        ("max_age", ctypes.c_int32),
        ("err_alpha", ctypes.c_float),
        ("err_beta", ctypes.c_float),
        ("n_max", ctypes.c_int32),
        ("e_max", ctypes.c_int32),
        ("m_max", ctypes.c_int32),
        ("lock_mode", ctypes.c_int32),
        ("key_mode", ctypes.c_int32),
    ]


@dataclass
class Params:
    """Learning rates (Eq. adaptation), edge aging limit, GNG error factors, capacities."""
    eps_b: float = 0.05
    eps_n: float = 0.0006
    max_age: int = 50
    err_alpha: float = 0.5
    err_beta: float = 0.995
    n_max: int = 1024
    e_max: int = 4096
    m_max: int = 1024
    lock_mode: int = 0   # 0: lock set {b, s} + N(b); 1: winner only, sequential update;
    #                      2: lock set, greedy in key order
    key_mode: int = 0    # 0: (bits(d1) << 32) | j; 1: j (arrival order)

    def c(self) -> _Params:
        return _Params(self.eps_b, self.eps_n, self.max_age, self.err_alpha, self.err_beta,
                       self.n_max, self.e_max, self.m_max, self.lock_mode, self.key_mode)


class _Schedule(ctypes.Structure):
    _fields_ = [
        ("m_cap", ctypes.c_int32),
        ("fixed_m", ctypes.c_int32),
        ("insert_every", ctypes.c_int64),
        ("qe_window", ctypes.c_int64),
        ("max_signals", ctypes.c_int64),
        ("qe_threshold", ctypes.c_float),
        ("seed", ctypes.c_uint64),
    ]


class _ScheduleResult(ctypes.Structure):
    _fields_ = [
        ("iterations", ctypes.c_int64),
        ("signals", ctypes.c_int64),
        ("accepted", ctypes.c_int64),
        ("inserted", ctypes.c_int64),
        ("qe", ctypes.c_double),
        ("converged", ctypes.c_int32),
        ("n_units", ctypes.c_int32),
        ("n_edges", ctypes.c_int64),
    ]


@dataclass
class Schedule:
    """The growing-network schedule (Sec. 3.1 level of parallelism, GNG insertion, stop on
    the quantization error); see the header of gsn_oracle.c."""
    m_cap: int = 8192
    fixed_m: int = 0
    insert_every: int = 100
    qe_window: int = 8192
    max_signals: int = 1 << 20
    qe_threshold: float = 0.0
    seed: int = 0

    def c(self) -> _Schedule:
        return _Schedule(self.m_cap, self.fixed_m, self.insert_every, self.qe_window,
                         self.max_signals, self.qe_threshold, self.seed)


class _Grid(ctypes.Structure):
    _fields_ = [("lo", ctypes.c_float * 3), ("h", ctypes.c_float), ("dims", ctypes.c_int32 * 3)]


def _grid(lo, h, dims) -> _Grid:
    g = _Grid()
    for a in range(3):
        g.lo[a] = float(lo[a])
        g.dims[a] = int(dims[a])
    g.h = float(h)
    return g


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i32 = ctypes.c_int32
    lib.orc_create.argtypes = [ctypes.POINTER(_Params), i32, P, ctypes.POINTER(P)]
    lib.orc_destroy.argtypes = [P]
    lib.orc_destroy.restype = None
    lib.orc_find_winners.argtypes = [P, P, i32, P, P, P, P, i32]
    lib.orc_resolve_conflicts.argtypes = [P, i32, P, P, P, P]
    lib.orc_adapt.argtypes = [P, P, i32, P, P, P, P]
    lib.orc_update_edges.argtypes = [P, i32, P, P, P]
    lib.orc_grow.argtypes = [P, i32, i32]
    lib.orc_sizes.argtypes = [P, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_int64)]
    lib.orc_status.argtypes = [P]
    lib.orc_export.argtypes = [P, P, P, P, P]
    lib.orc_import.argtypes = [P, i32, P, P, i32, P]
    lib.orc_age.argtypes = [P, i32, i32]
    lib.orc_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
    lib.orc_splitmix64.restype = ctypes.c_uint64
    lib.orc_schedule_m.argtypes = [i32, i32, i32]
    lib.orc_schedule_m.restype = i32
    lib.orc_run_schedule.argtypes = [P, P, ctypes.c_int64, ctypes.POINTER(_Schedule),
                                     ctypes.POINTER(_ScheduleResult), i32]
    lib.orc_run_schedule.restype = ctypes.c_int
    lib.orc_grid_cell.argtypes = [ctypes.POINTER(_Grid), ctypes.c_float, ctypes.c_float,
                                  ctypes.c_float, P]
    lib.orc_grid_cell.restype = None
    lib.orc_find_winners_grid.argtypes = [P, ctypes.POINTER(_Grid), P, i32, P, P, P, P, P, i32]
    lib.orc_find_winners_grid.restype = ctypes.c_int
    for f in ("orc_create", "orc_find_winners", "orc_resolve_conflicts", "orc_adapt",
              "orc_update_edges", "orc_grow", "orc_sizes", "orc_status", "orc_export",
              "orc_import", "orc_age"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


def splitmix64(seed: int, counter: int) -> int:
    """Output number `counter` (1, 2, ...) of SplitMix64 started at `seed`."""
    return int(_load().orc_splitmix64(seed & (2**64 - 1), counter & (2**64 - 1)))


def schedule_m(n: int, m_cap: int, fixed_m: int = 0) -> int:
    return int(_load().orc_schedule_m(n, m_cap, fixed_m))


def grid_cell(lo, h, dims, point) -> tuple:
    """Cell coordinates of a point in the index grid (see gsn_oracle.c)."""
    c = np.zeros(3, np.int32)
    _load().orc_grid_cell(ctypes.byref(_grid(lo, h, dims)), float(point[0]), float(point[1]),
                          float(point[2]), ctypes.c_void_p(c.ctypes.data))
    return tuple(int(v) for v in c)


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


def _soa(xyz, dtype=np.float32) -> np.ndarray:
    """Accept (3, n) SoA or (n, 3) AoS point arrays; return contiguous SoA (3, n)."""
    a = np.asarray(xyz, dtype=dtype)
    if a.ndim != 2:
        raise ValueError("expected a 2-D point array")
    if a.shape[0] != 3 and a.shape[1] == 3:
        a = a.T
    return np.ascontiguousarray(a)


class OracleError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what} failed with code {code}")
        self.code = code


def _check(rc: int, what: str):
    if rc != OK:
        raise OracleError(rc, what)


class Oracle:
    """One network state and the five steps of the multi-signal iteration."""

    def __init__(self, params: Params, init_xyz, threads: int = 1):
        lib = _load()
        self.params = params
        self.threads = int(threads)
        xyz = _soa(init_xyz)
        n0 = xyz.shape[1]
        h = ctypes.c_void_p()
        _check(lib.orc_create(ctypes.byref(params.c()), n0, _ptr(xyz), ctypes.byref(h)),
               "orc_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            _load().orc_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- steps ----
    def find_winners(self, sig):
        """sig: (3, m) float32.  Returns winner, second (int32), d1, d2 (float32)."""
        s = _soa(sig)
        m = s.shape[1]
        w = np.empty(m, np.int32)
        sc = np.empty(m, np.int32)
        d1 = np.empty(m, np.float32)
        d2 = np.empty(m, np.float32)
        _check(_load().orc_find_winners(self._h, _ptr(s), m, _ptr(w), _ptr(sc), _ptr(d1),
                                        _ptr(d2), self.threads), "orc_find_winners")
        return w, sc, d1, d2

    def find_winners_grid(self, sig, lo, h, dims):
        """The indexed search of the paper's "Indexed" implementation on every signal.
        Returns winner, second, d1, d2 and the number of signals that fell back to the
        exhaustive search."""
        s = _soa(sig)
        m = s.shape[1]
        w = np.empty(m, np.int32)
        sc = np.empty(m, np.int32)
        d1 = np.empty(m, np.float32)
        d2 = np.empty(m, np.float32)
        fb = ctypes.c_int32()
        _check(_load().orc_find_winners_grid(self._h, ctypes.byref(_grid(lo, h, dims)), _ptr(s),
                                             m, _ptr(w), _ptr(sc), _ptr(d1), _ptr(d2),
                                             ctypes.byref(fb), self.threads),
               "orc_find_winners_grid")
        return w, sc, d1, d2, fb.value

    def resolve_conflicts(self, winner, second, d1):
        w = np.ascontiguousarray(winner, np.int32)
        s = np.ascontiguousarray(second, np.int32)
        d = np.ascontiguousarray(d1, np.float32)
        acc = np.zeros(w.shape[0], np.uint8)
        _check(_load().orc_resolve_conflicts(self._h, w.shape[0], _ptr(w), _ptr(s), _ptr(d),
                                             _ptr(acc)), "orc_resolve_conflicts")
        return acc

    def adapt(self, sig, winner, second, d1, accepted):
        s = _soa(sig)
        w = np.ascontiguousarray(winner, np.int32)
        sc = np.ascontiguousarray(second, np.int32)
        d = np.ascontiguousarray(d1, np.float32)
        a = np.ascontiguousarray(accepted, np.uint8)
        _check(_load().orc_adapt(self._h, _ptr(s), s.shape[1], _ptr(w), _ptr(sc), _ptr(d),
                                 _ptr(a)), "orc_adapt")

    def update_edges(self, winner, second, accepted):
        w = np.ascontiguousarray(winner, np.int32)
        sc = np.ascontiguousarray(second, np.int32)
        a = np.ascontiguousarray(accepted, np.uint8)
        _check(_load().orc_update_edges(self._h, w.shape[0], _ptr(w), _ptr(sc), _ptr(a)),
               "orc_update_edges")

    def grow(self, iteration: int, insert_every: int):
        _check(_load().orc_grow(self._h, int(iteration), int(insert_every)), "orc_grow")

    def iterate(self, sig, iteration: int = 0, insert_every: int = 0, grow: bool = False):
        """One whole iteration; returns (winner, second, d1, d2, accepted)."""
        w, s, d1, d2 = self.find_winners(sig)
        acc = self.resolve_conflicts(w, s, d1)
        self.adapt(sig, w, s, d1, acc)
        self.update_edges(w, s, acc)
        if grow:
            self.grow(iteration, insert_every)
        return w, s, d1, d2, acc

    # ---------------------------------------------------------------- state ----
    def sizes(self):
        n = ctypes.c_int32()
        e = ctypes.c_int64()
        _check(_load().orc_sizes(self._h, ctypes.byref(n), ctypes.byref(e)), "orc_sizes")
        return n.value, e.value

    def status(self) -> int:
        return _load().orc_status(self._h)

    def export(self):
        """Returns dict(xyz=(3,n) f32, err=(n,) f32, edges=(3,E) i32 sorted (u<v), orphan)."""
        n, e = self.sizes()
        xyz = np.empty((3, n), np.float32)
        err = np.empty(n, np.float32)
        edges = np.empty((3, e), np.int32)
        orphan = np.empty(n, np.uint8)
        _check(_load().orc_export(self._h, _ptr(xyz), _ptr(err), _ptr(edges), _ptr(orphan)),
               "orc_export")
        return {"xyz": xyz, "err": err, "edges": edges, "orphan": orphan}

    def import_state(self, xyz, err=None, edges=None):
        x = _soa(xyz)
        n = x.shape[1]
        e = (np.zeros((3, 0), np.int32) if edges is None
             else np.ascontiguousarray(np.asarray(edges, np.int32).reshape(3, -1)))
        er = None if err is None else np.ascontiguousarray(err, np.float32)
        _check(_load().orc_import(self._h, n, _ptr(x), _ptr(er), e.shape[1], _ptr(e)),
               "orc_import")

    def age(self, u: int, v: int) -> int:
        return _load().orc_age(self._h, int(u), int(v))

    def run_schedule(self, cloud, schedule: Schedule) -> dict:
        """Whole iterations under the growing-network schedule from the current state."""
        c = _soa(cloud)
        r = _ScheduleResult()
        _check(_load().orc_run_schedule(self._h, _ptr(c), c.shape[1],
                                        ctypes.byref(schedule.c()), ctypes.byref(r),
                                        self.threads), "orc_run_schedule")
        return {f: getattr(r, f) for f, _ in _ScheduleResult._fields_}
