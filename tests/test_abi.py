"""The C ABI library: it loads, exports every symbol include/gsn.h declares, and rejects
bad arguments on the host before touching a device (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gsn.h")
LIB = os.path.join(ROOT, "paper_1503_08294_amd", "libgsn.so")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gsn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    return ctypes.CDLL(LIB)


def test_every_declared_symbol_is_exported(lib):
    names = declared()
    for n in ("gsn_create", "gsn_find_winners", "gsn_resolve_conflicts", "gsn_adapt",
              "gsn_update_edges", "gsn_grow", "gsn_destroy"):
        assert n in names
    for n in names:
        assert hasattr(lib, n), n


def test_binding_covers_the_header():
    from paper_1503_08294_amd import gsn
    assert sorted(gsn.EXPORTED) == declared()
    for n in declared():
        assert callable(getattr(gsn, n))


def test_host_side_validation(lib):
    from paper_1503_08294_amd.gsn import gsn_params, make_params
    lib.gsn_workspace_bytes.restype = ctypes.c_size_t
    lib.gsn_workspace_bytes.argtypes = [ctypes.POINTER(gsn_params)]
    good = make_params(n_max=1000, e_max=4000, m_max=256)
    size = lib.gsn_workspace_bytes(ctypes.byref(good))
    assert size > 12 * 1000 and size % 256 == 0
    # the winner lock needs room for one insertion at the winner and one at the second of
    # every survivor in both adjacency buffers (col and age)
    winner = make_params(n_max=1000, e_max=4000, m_max=256, lock_mode=1)
    assert lib.gsn_workspace_bytes(ctypes.byref(winner)) >= size + 4 * 4 * 2 * 256
    for bad in (make_params(eps_b=1.5), make_params(eps_n=-0.1), make_params(max_age=-1),
                make_params(n_max=1), make_params(m_max=0), make_params(e_max=-1),
                make_params(lock_mode=3), make_params(key_mode=-1),
                make_params(err_alpha=1.5), make_params(err_alpha=-0.5),
                make_params(err_beta=1.01), make_params(err_beta=float("nan")),
                make_params(lock_mode=1, e_max=2**30 - 1, m_max=2**20)):
        assert lib.gsn_workspace_bytes(ctypes.byref(bad)) == 0
    P = ctypes.c_void_p
    lib.gsn_create.argtypes = [ctypes.POINTER(gsn_params), P, ctypes.c_size_t, ctypes.c_int32,
                               P, P, ctypes.POINTER(P)]
    h = P()
    fake = P(1 << 20)   # never dereferenced: every call below fails validation first
    bad = make_params(eps_b=2.0)
    assert lib.gsn_create(ctypes.byref(bad), fake, size, 10, fake, None, ctypes.byref(h)) == -1
    assert lib.gsn_create(ctypes.byref(good), P(0), size, 10, fake, None, ctypes.byref(h)) == -1
    assert lib.gsn_create(ctypes.byref(good), P((1 << 20) + 4), size, 10, fake, None,
                          ctypes.byref(h)) == -1                      # misaligned
    assert lib.gsn_create(ctypes.byref(good), fake, size - 256, 10, fake, None,
                          ctypes.byref(h)) == -2                      # too small
    assert lib.gsn_create(ctypes.byref(good), fake, size, 1001, fake, None,
                          ctypes.byref(h)) == -1                      # n0 > n_max
    assert lib.gsn_create(ctypes.byref(good), fake, size, 10, P(0), None,
                          ctypes.byref(h)) == -1                      # no positions
    for name, nargs in (("gsn_find_winners", 8), ("gsn_resolve_conflicts", 7),
                        ("gsn_adapt", 8), ("gsn_update_edges", 6), ("gsn_grow", 4),
                        ("gsn_iterate", 9), ("gsn_iterate_loop", 10),
                        ("gsn_check", 2), ("gsn_tune", 3), ("gsn_timing_enable", 2),
                        ("gsn_timing_select", 2)):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        args = [P(0)] + [0] * (nargs - 1)
        f.argtypes = [P] + [ctypes.c_int64] * (nargs - 1)
        assert f(*args) == -1, name
