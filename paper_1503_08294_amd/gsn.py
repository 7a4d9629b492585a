"""Thin Python binding of libgsn (include/gsn.h).

Argument marshalling only: every step of the iteration runs in the HIP kernels of
``libgsn.so``.  Device buffers are torch tensors on the current HIP device; the stream
passed to the library is torch's current stream unless one is given.  The functions keep
the C names; ``Network`` bundles a handle with its workspace for convenience.

Importing this module fails loudly when the library has not been built: there is no
fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgsn.so")

GSN_OK = 0
GSN_E_INVAL = -1
GSN_E_CAPACITY = -2
GSN_E_HIP = -3
GSN_E_STATE = -4

GSN_TUNE_SPLIT = 1
GSN_TUNE_VARIANT = 2
GSN_TUNE_GRID_ROUNDS = 3
GSN_TUNE_GRAB = 4
GSN_TUNE_REBUCKET = 5
GSN_MAX_SPLIT = 64

GSN_T_FIND_SCAN = 0
GSN_T_FIND = 1
GSN_T_RESOLVE = 2
GSN_T_ADAPT = 3
GSN_T_EDGES = 4
GSN_T_UPDATE = 5
GSN_T_COUNT = 6

GSN_LOCK_SET = 0
GSN_LOCK_WINNER = 1
GSN_LOCK_SET_GREEDY = 2
GSN_KEY_DIST_INDEX = 0
GSN_KEY_INDEX = 1

GSN_NOALLOC_SCRATCH_BYTES = 32 << 20
GSN_MAX_LOOP = 4096
GSN_GRAPH_CACHE = 4

GSN_STAT_ROUNDS = 0
GSN_STAT_ROUNDS_MAX = 1
GSN_STAT_UPDATES = 2
GSN_STAT_CLEAR = 3
GSN_STAT_RESOLVED = 4
GSN_STAT_ACCEPTED = 5
GSN_STAT_LOOP_RECORDS = 6

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                      "(hipcc --offload-arch=gfx950); there is no fallback path")

_lib = ctypes.CDLL(LIB_PATH)


class gsn_params(ctypes.Structure):
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


class gsn_grid(ctypes.Structure):
    _fields_ = [("lo", ctypes.c_float * 3), ("h", ctypes.c_float), ("dims", ctypes.c_int32 * 3),
                ("exact", ctypes.c_int32)]


def make_grid(lo, h, dims, exact=False) -> gsn_grid:
    g = gsn_grid()
    for a in range(3):
        g.lo[a] = float(lo[a])
        g.dims[a] = int(dims[a])
    g.h = float(h)
    g.exact = 1 if exact else 0
    return g


class gsn_schedule(ctypes.Structure):
    _fields_ = [
        ("m_cap", ctypes.c_int32),
        ("fixed_m", ctypes.c_int32),
        ("insert_every", ctypes.c_int64),
        ("qe_window", ctypes.c_int64),
        ("max_signals", ctypes.c_int64),
        ("qe_threshold", ctypes.c_float),
        ("seed", ctypes.c_uint64),
    ]


class gsn_schedule_result(ctypes.Structure):
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


_P = ctypes.c_void_p
_I = ctypes.c_int32
_sig = {
    "gsn_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(gsn_params)]),
    "gsn_create": (ctypes.c_int, [ctypes.POINTER(gsn_params), _P, ctypes.c_size_t, _I, _P, _P,
                                  ctypes.POINTER(_P)]),
    "gsn_find_winners": (ctypes.c_int, [_P, _P, _I, _P, _P, _P, _P, _P]),
    "gsn_grid_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(gsn_grid), _I, _I]),
    "gsn_find_winners_grid": (ctypes.c_int, [_P, ctypes.POINTER(gsn_grid), _P, ctypes.c_size_t,
                                             _P, _I, _P, _P, _P, _P, _P]),
    "gsn_find_winners_grid_noalloc": (ctypes.c_int, [_P, ctypes.POINTER(gsn_grid), _P, _I, _P,
                                                     _P, _P, _P, _P]),
    "gsn_resolve_conflicts": (ctypes.c_int, [_P, _I, _P, _P, _P, _P, _P]),
    "gsn_adapt": (ctypes.c_int, [_P, _P, _I, _P, _P, _P, _P, _P]),
    "gsn_update_edges": (ctypes.c_int, [_P, _I, _P, _P, _P, _P]),
    "gsn_iterate": (ctypes.c_int, [_P, _P, _I, _P, _P, _P, _P, _P, _P]),
    "gsn_update": (ctypes.c_int, [_P, _P, _I, _P, _P, _P, _P, _P]),
    "gsn_iterate_loop": (ctypes.c_int, [_P, _P, _I, _I, _P, _P, _P, _P, _P, _P]),
    "gsn_grow": (ctypes.c_int, [_P, _I, _I, _P]),
    "gsn_run_schedule": (ctypes.c_int, [_P, _P, ctypes.c_int64, ctypes.POINTER(gsn_schedule),
                                        ctypes.POINTER(gsn_schedule_result), _P]),
    "gsn_sizes": (ctypes.c_int, [_P, ctypes.POINTER(_I), ctypes.POINTER(_I), _P]),
    "gsn_export": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "gsn_import": (ctypes.c_int, [_P, _I, _P, _P, _I, _P, _P]),
    "gsn_check": (ctypes.c_int, [_P, _P]),
    "gsn_destroy": (None, [_P]),
    "gsn_tune": (ctypes.c_int, [_P, _I, _I]),
    "gsn_timing_enable": (ctypes.c_int, [_P, _I]),
    "gsn_timing_select": (ctypes.c_int, [_P, ctypes.c_uint32]),
    "gsn_timing_read": (ctypes.c_int, [_P, _I, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(_I)]),
    "gsn_stat": (ctypes.c_int, [_P, _I, ctypes.POINTER(ctypes.c_int64), _P]),
}
for _name, (_res, _args) in _sig.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_sig)


class GsnError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what} returned {code}")
        self.code = code


def _check(rc: int, what: str) -> int:
    if rc != GSN_OK:
        raise GsnError(rc, what)
    return rc


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else stream)


def _dev(t: torch.Tensor | None, dtype, n: int | None = None, what: str = "tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if n is not None and t.numel() < n:
        raise ValueError(f"{what} holds {t.numel()} elements, needs {n}")
    return ctypes.c_void_p(t.data_ptr())


def make_params(eps_b=0.05, eps_n=0.0006, max_age=50, err_alpha=0.5, err_beta=0.995,
                n_max=1024, e_max=4096, m_max=1024, lock_mode=GSN_LOCK_SET,
                key_mode=GSN_KEY_DIST_INDEX) -> gsn_params:
    return gsn_params(eps_b, eps_n, max_age, err_alpha, err_beta, n_max, e_max, m_max,
                      lock_mode, key_mode)


# ------------------------------------------------------------- C-named calls ----

def gsn_workspace_bytes(params: gsn_params) -> int:
    return int(_lib.gsn_workspace_bytes(ctypes.byref(params)))


def gsn_create(params: gsn_params, workspace: torch.Tensor, init_xyz: torch.Tensor,
               stream=None) -> ctypes.c_void_p:
    """init_xyz: (3, n0) float32 SoA, device or host tensor."""
    if init_xyz.dtype != torch.float32 or not init_xyz.is_contiguous() or init_xyz.dim() != 2 \
            or init_xyz.shape[0] != 3:
        raise ValueError("init_xyz must be a contiguous (3, n0) float32 tensor")
    h = ctypes.c_void_p()
    _check(_lib.gsn_create(ctypes.byref(params), _dev(workspace, torch.uint8),
                           workspace.numel(), init_xyz.shape[1],
                           ctypes.c_void_p(init_xyz.data_ptr()), _stream(stream),
                           ctypes.byref(h)), "gsn_create")
    return h


def gsn_find_winners(net, sig, m, winner, second, d1, d2, stream=None):
    return _check(_lib.gsn_find_winners(
        net, _dev(sig, torch.float32, 3 * m, "sig"), m, _dev(winner, torch.int32, m, "winner"),
        _dev(second, torch.int32, m, "second"), _dev(d1, torch.float32, m, "d1"),
        _dev(d2, torch.float32, m, "d2"), _stream(stream)), "gsn_find_winners")


def gsn_resolve_conflicts(net, m, winner, second, d1, accepted, stream=None):
    return _check(_lib.gsn_resolve_conflicts(
        net, m, _dev(winner, torch.int32, m, "winner"), _dev(second, torch.int32, m, "second"),
        _dev(d1, torch.float32, m, "d1"), _dev(accepted, torch.uint8, m, "accepted"),
        _stream(stream)), "gsn_resolve_conflicts")


def gsn_adapt(net, sig, m, winner, second, d1, accepted, stream=None):
    return _check(_lib.gsn_adapt(
        net, _dev(sig, torch.float32, 3 * m, "sig"), m, _dev(winner, torch.int32, m, "winner"),
        _dev(second, torch.int32, m, "second"), _dev(d1, torch.float32, m, "d1"),
        _dev(accepted, torch.uint8, m, "accepted"), _stream(stream)), "gsn_adapt")


def gsn_update_edges(net, m, winner, second, accepted, stream=None):
    return _check(_lib.gsn_update_edges(
        net, m, _dev(winner, torch.int32, m, "winner"), _dev(second, torch.int32, m, "second"),
        _dev(accepted, torch.uint8, m, "accepted"), _stream(stream)), "gsn_update_edges")


def gsn_grow(net, iteration: int, insert_every: int, stream=None):
    return _check(_lib.gsn_grow(net, iteration, insert_every, _stream(stream)), "gsn_grow")


def gsn_sizes(net, stream=None):
    n = ctypes.c_int32()
    e = ctypes.c_int32()
    _check(_lib.gsn_sizes(net, ctypes.byref(n), ctypes.byref(e), _stream(stream)), "gsn_sizes")
    return n.value, e.value


def gsn_export(net, stream=None) -> dict:
    """State as host tensors: xyz (3, N) f32, err (N,) f32, edges (3, E) i32 (u < v, sorted)."""
    n, e = gsn_sizes(net, stream)
    xyz = torch.empty((3, n), dtype=torch.float32)
    err = torch.empty(n, dtype=torch.float32)
    edges = torch.empty((3, e), dtype=torch.int32)
    _check(_lib.gsn_export(net, ctypes.c_void_p(xyz.data_ptr()), ctypes.c_void_p(err.data_ptr()),
                           ctypes.c_void_p(edges.data_ptr()), _stream(stream)), "gsn_export")
    return {"xyz": xyz, "err": err, "edges": edges}


def gsn_import(net, xyz: torch.Tensor, err: torch.Tensor | None = None,
               edges: torch.Tensor | None = None, stream=None):
    xyz = xyz.contiguous()
    n = xyz.shape[1]
    if edges is None:
        edges = torch.zeros((3, 0), dtype=torch.int32)
    edges = edges.to(torch.int32).contiguous()
    err_p = None if err is None else ctypes.c_void_p(err.contiguous().data_ptr())
    return _check(_lib.gsn_import(net, n, ctypes.c_void_p(xyz.data_ptr()), err_p,
                                  edges.shape[1], ctypes.c_void_p(edges.data_ptr()),
                                  _stream(stream)), "gsn_import")


def gsn_check(net, stream=None) -> int:
    return int(_lib.gsn_check(net, _stream(stream)))


def gsn_destroy(net):
    _lib.gsn_destroy(net)


def gsn_tune(net, key: int, value: int):
    return _check(_lib.gsn_tune(net, key, value), "gsn_tune")


def gsn_timing_enable(net, enable: bool):
    return _check(_lib.gsn_timing_enable(net, 1 if enable else 0), "gsn_timing_enable")


def gsn_timing_select(net, mask: int):
    return _check(_lib.gsn_timing_select(net, mask), "gsn_timing_select")


def gsn_timing_read(net, which: int):
    ms = ctypes.c_double()
    cnt = ctypes.c_int32()
    _check(_lib.gsn_timing_read(net, which, ctypes.byref(ms), ctypes.byref(cnt)),
           "gsn_timing_read")
    return ms.value, cnt.value


def gsn_grid_workspace_bytes(grid: gsn_grid, n_max: int, m_max: int) -> int:
    return int(_lib.gsn_grid_workspace_bytes(ctypes.byref(grid), n_max, m_max))


def gsn_find_winners_grid(net, grid: gsn_grid, grid_ws: torch.Tensor, sig: torch.Tensor, m: int,
                          winner, second, d1, d2, stream=None):
    _check(_lib.gsn_find_winners_grid(net, ctypes.byref(grid), _dev(grid_ws, torch.uint8),
                                      grid_ws.numel(), _dev(sig, torch.float32, 3 * m, "sig"),
                                      m, _dev(winner, torch.int32, m, "winner"),
                                      _dev(second, torch.int32, m, "second"),
                                      _dev(d1, torch.float32, m, "d1"),
                                      _dev(d2, torch.float32, m, "d2"), _stream(stream)),
           "gsn_find_winners_grid")


def gsn_find_winners_grid_noalloc(net, grid: gsn_grid, sig: torch.Tensor, m: int, winner,
                                  second, d1, d2, stream=None):
    _check(_lib.gsn_find_winners_grid_noalloc(net, ctypes.byref(grid),
                                              _dev(sig, torch.float32, 3 * m, "sig"), m,
                                              _dev(winner, torch.int32, m, "winner"),
                                              _dev(second, torch.int32, m, "second"),
                                              _dev(d1, torch.float32, m, "d1"),
                                              _dev(d2, torch.float32, m, "d2"), _stream(stream)),
           "gsn_find_winners_grid_noalloc")


def gsn_iterate(net, sig: torch.Tensor, m: int, winner, second, d1, d2, accepted,
                stream=None):
    _check(_lib.gsn_iterate(net, _dev(sig, torch.float32, 3 * m, "sig"), m,
                            _dev(winner, torch.int32, m, "winner"),
                            _dev(second, torch.int32, m, "second"),
                            _dev(d1, torch.float32, m, "d1"), _dev(d2, torch.float32, m, "d2"),
                            _dev(accepted, torch.uint8, m, "accepted"), _stream(stream)),
           "gsn_iterate")


def gsn_update(net, sig: torch.Tensor, m: int, winner, second, d1, accepted, stream=None):
    _check(_lib.gsn_update(net, _dev(sig, torch.float32, 3 * m, "sig"), m,
                           _dev(winner, torch.int32, m, "winner"),
                           _dev(second, torch.int32, m, "second"),
                           _dev(d1, torch.float32, m, "d1"),
                           _dev(accepted, torch.uint8, m, "accepted"), _stream(stream)),
           "gsn_update")


def gsn_iterate_loop(net, sigs: torch.Tensor, m: int, count: int, winner, second, d1, d2,
                     accepted, stream=None):
    _check(_lib.gsn_iterate_loop(net, _dev(sigs, torch.float32, 3 * m * count, "sigs"), m,
                                 count, _dev(winner, torch.int32, m, "winner"),
                                 _dev(second, torch.int32, m, "second"),
                                 _dev(d1, torch.float32, m, "d1"),
                                 _dev(d2, torch.float32, m, "d2"),
                                 _dev(accepted, torch.uint8, m, "accepted"), _stream(stream)),
           "gsn_iterate_loop")


def make_schedule(m_cap=8192, fixed_m=0, insert_every=100, qe_window=8192,
                  max_signals=1 << 20, qe_threshold=0.0, seed=0) -> gsn_schedule:
    return gsn_schedule(m_cap, fixed_m, insert_every, qe_window, max_signals, qe_threshold,
                        seed)


def gsn_run_schedule(net, cloud: torch.Tensor, schedule: gsn_schedule, stream=None) -> dict:
    """cloud: device SoA (3, P) float32.  Returns the result fields as a dict."""
    if cloud.dim() != 2 or cloud.shape[0] != 3:
        raise ValueError("cloud must be (3, P)")
    p = _dev(cloud, torch.float32, what="cloud")
    r = gsn_schedule_result()
    _check(_lib.gsn_run_schedule(net, p, cloud.shape[1], ctypes.byref(schedule),
                                 ctypes.byref(r), _stream(stream)), "gsn_run_schedule")
    return {f: getattr(r, f) for f, _ in gsn_schedule_result._fields_}


def gsn_stat(net, key: int, stream=None) -> int:
    v = ctypes.c_int64()
    _check(_lib.gsn_stat(net, key, ctypes.byref(v), _stream(stream)), "gsn_stat")
    return v.value


# ------------------------------------------------------------------ convenience ----

class PreparedIterate:
    """Pre-marshalled gsn_iterate calls over a fixed list of signal batches (see
    Network.prepare_iterate).  The tensors must stay alive and unchanged in shape."""

    def __init__(self, net, sigs):
        b = net.buf
        self._net = net
        self._keep = list(sigs)
        m = self._keep[0].shape[1]
        outs = [_dev(b.winner, torch.int32, m, "winner"), _dev(b.second, torch.int32, m, "second"),
                _dev(b.d1, torch.float32, m, "d1"), _dev(b.d2, torch.float32, m, "d2"),
                _dev(b.accepted, torch.uint8, m, "accepted")]
        st = _stream(net.stream)
        self._args = []
        for sig in self._keep:
            if sig.shape[1] != m:
                raise ValueError("every batch must hold the same number of signals")
            self._args.append((net.h, _dev(sig, torch.float32, 3 * m, "sig"), m, *outs, st))
        self.m = m

    def __len__(self):
        return len(self._args)

    def __call__(self, t: int):
        rc = _lib.gsn_iterate(*self._args[t])
        if rc != GSN_OK:
            raise GsnError(rc, "gsn_iterate")


@dataclass
class Buffers:
    """Per-iteration device buffers for up to m_max signals."""
    winner: torch.Tensor
    second: torch.Tensor
    d1: torch.Tensor
    d2: torch.Tensor
    accepted: torch.Tensor

    @staticmethod
    def make(m_max: int, device) -> "Buffers":
        return Buffers(torch.empty(m_max, dtype=torch.int32, device=device),
                       torch.empty(m_max, dtype=torch.int32, device=device),
                       torch.empty(m_max, dtype=torch.float32, device=device),
                       torch.empty(m_max, dtype=torch.float32, device=device),
                       torch.empty(m_max, dtype=torch.uint8, device=device))


class Network:
    """A handle with its workspace and per-iteration buffers (all torch device memory)."""

    def __init__(self, params: gsn_params, init_xyz: torch.Tensor, device="cuda",
                 stream=None):
        self.params = params
        self.device = torch.device(device)
        size = gsn_workspace_bytes(params)
        if size == 0:
            raise GsnError(GSN_E_INVAL, "gsn_workspace_bytes")
        # over-allocate so the start can be aligned to 256 bytes
        self._ws_raw = torch.empty(size + 256, dtype=torch.uint8, device=self.device)
        off = (-self._ws_raw.data_ptr()) % 256
        self.workspace = self._ws_raw[off:off + size]
        self.stream = stream
        self.h = gsn_create(params, self.workspace, init_xyz.contiguous(), stream)
        self.buf = Buffers.make(params.m_max, self.device)

    def close(self):
        if getattr(self, "h", None):
            gsn_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def find_winners(self, sig: torch.Tensor):
        m = sig.shape[1]
        b = self.buf
        gsn_find_winners(self.h, sig, m, b.winner, b.second, b.d1, b.d2, self.stream)
        return b.winner[:m], b.second[:m], b.d1[:m], b.d2[:m]

    def grid_workspace(self, grid: gsn_grid) -> torch.Tensor:
        """A 256-byte aligned device buffer for gsn_find_winners_grid with this grid."""
        size = gsn_grid_workspace_bytes(grid, self.params.n_max, self.params.m_max)
        if size == 0:
            raise GsnError(GSN_E_INVAL, "gsn_grid_workspace_bytes")
        raw = torch.empty(size + 256, dtype=torch.uint8, device=self.device)
        off = (-raw.data_ptr()) % 256
        ws = raw[off:off + size]
        ws._raw = raw  # keep the allocation alive with the view
        return ws

    def find_winners_grid(self, sig: torch.Tensor, grid: gsn_grid, grid_ws: torch.Tensor):
        m = sig.shape[1]
        b = self.buf
        gsn_find_winners_grid(self.h, grid, grid_ws, sig, m, b.winner, b.second, b.d1, b.d2,
                              self.stream)
        return b.winner[:m], b.second[:m], b.d1[:m], b.d2[:m]

    def find_winners_grid_noalloc(self, sig: torch.Tensor, grid: gsn_grid):
        m = sig.shape[1]
        b = self.buf
        gsn_find_winners_grid_noalloc(self.h, grid, sig, m, b.winner, b.second, b.d1, b.d2,
                                      self.stream)
        return b.winner[:m], b.second[:m], b.d1[:m], b.d2[:m]

    def resolve_conflicts(self, m, winner=None, second=None, d1=None):
        b = self.buf
        gsn_resolve_conflicts(self.h, m, b.winner if winner is None else winner,
                              b.second if second is None else second,
                              b.d1 if d1 is None else d1, b.accepted, self.stream)
        return b.accepted[:m]

    def adapt(self, sig, winner=None, second=None, d1=None, accepted=None):
        m = sig.shape[1]
        b = self.buf
        gsn_adapt(self.h, sig, m, b.winner if winner is None else winner,
                  b.second if second is None else second, b.d1 if d1 is None else d1,
                  b.accepted if accepted is None else accepted, self.stream)

    def update_edges(self, m, winner=None, second=None, accepted=None):
        b = self.buf
        gsn_update_edges(self.h, m, b.winner if winner is None else winner,
                         b.second if second is None else second,
                         b.accepted if accepted is None else accepted, self.stream)

    def iterate(self, sig: torch.Tensor):
        """find -> resolve -> adapt -> update_edges on one batch (device SoA (3, m)), in one
        gsn_iterate call."""
        m = sig.shape[1]
        b = self.buf
        gsn_iterate(self.h, sig, m, b.winner, b.second, b.d1, b.d2, b.accepted, self.stream)
        return b.winner[:m], b.second[:m], b.d1[:m], b.d2[:m], b.accepted[:m]

    def update(self, sig: torch.Tensor, winner=None, second=None, d1=None):
        """resolve -> adapt -> update_edges after a find, fused as in gsn_iterate (one
        gsn_update call); returns the acceptance."""
        m = sig.shape[1]
        b = self.buf
        gsn_update(self.h, sig, m, b.winner if winner is None else winner,
                   b.second if second is None else second, b.d1 if d1 is None else d1,
                   b.accepted, self.stream)
        return b.accepted[:m]

    def iterate_loop(self, sigs: torch.Tensor):
        """One iteration per batch of ``sigs`` (a contiguous device (T, 3, m) tensor) in one
        gsn_iterate_loop call (recorded into a HIP graph once, replayed afterwards); returns
        the last iteration's outputs."""
        count, _, m = sigs.shape
        b = self.buf
        gsn_iterate_loop(self.h, sigs, m, count, b.winner, b.second, b.d1, b.d2, b.accepted,
                         self.stream)
        return b.winner[:m], b.second[:m], b.d1[:m], b.d2[:m], b.accepted[:m]

    def prepare_iterate(self, sigs):
        """gsn_iterate arguments for each batch of ``sigs`` (device SoA (3, m) tensors, or a
        (T, 3, m) tensor), validated and marshalled once; calling the result with t makes
        the one gsn_iterate call of batch t.  For timed loops where the per-call argument
        checks would cost more host time than the call itself."""
        return PreparedIterate(self, sigs)

    def iterate_steps(self, sig: torch.Tensor):
        """The same iteration through the four separate calls."""
        m = sig.shape[1]
        self.find_winners(sig)
        self.resolve_conflicts(m)
        self.adapt(sig)
        self.update_edges(m)
        b = self.buf
        return b.winner[:m], b.second[:m], b.d1[:m], b.d2[:m], b.accepted[:m]

    def grow(self, iteration: int, insert_every: int):
        gsn_grow(self.h, iteration, insert_every, self.stream)

    def sizes(self):
        return gsn_sizes(self.h, self.stream)

    def export(self):
        return gsn_export(self.h, self.stream)

    def import_state(self, xyz, err=None, edges=None):
        gsn_import(self.h, xyz, err, edges, self.stream)

    def check(self) -> int:
        return gsn_check(self.h, self.stream)

    def tune(self, key: int, value: int):
        gsn_tune(self.h, key, value)

    def stat(self, key: int) -> int:
        return gsn_stat(self.h, key, self.stream)

    def run_schedule(self, cloud: torch.Tensor, schedule: gsn_schedule) -> dict:
        return gsn_run_schedule(self.h, cloud.contiguous(), schedule, self.stream)
