"""Pins of the oracle's indexed search (the hash index of the paper's "Indexed"
implementation, Sec. 3.1: cubes of fixed side over a box holding the signals; winner and
second searched in the signal's cube and its 26 neighbours; the exhaustive search when that
fails).  Pinned by hand cases, by the special case where the 27 cubes hold every unit (the
exhaustive result), and by a float32 brute force on tiny inputs."""
import numpy as np
import pytest

import oracle


def net(units):
    p = oracle.Params(n_max=max(units.shape[1], 2) + 4, e_max=16, m_max=4096)
    return oracle.Oracle(p, np.ascontiguousarray(units, np.float32))


def test_cell_of_a_point():
    lo, h, dims = (0.0, 0.0, 0.0), 0.5, (4, 4, 4)
    assert oracle.grid_cell(lo, h, dims, (0.49, 0.0, 1.99)) == (0, 0, 3)
    assert oracle.grid_cell(lo, h, dims, (0.5, 1.0, 1.5)) == (1, 2, 3)
    # outside the box: the border cells
    assert oracle.grid_cell(lo, h, dims, (-3.0, 100.0, 2.0)) == (0, 3, 3)
    assert oracle.grid_cell((-1.0, -1.0, -1.0), 0.25, (8, 8, 8), (0.0, -0.75, 0.99)) == (4, 1, 7)


def test_one_cube_holding_everything_is_the_exhaustive_search():
    rng = np.random.default_rng(0)
    units = rng.standard_normal((3, 300)).astype(np.float32)
    sig = rng.standard_normal((3, 500)).astype(np.float32)
    o = net(units)
    ex = o.find_winners(sig)
    for dims in ((1, 1, 1), (3, 3, 3), (2, 3, 1)):
        # a box of side 3 h around the data; with at most 3 cubes per axis every unit is
        # within one cube of every signal
        g = o.find_winners_grid(sig, (-10.0, -10.0, -10.0), 20.0 / 3, dims)
        for a, b in zip(ex, g[:4]):
            np.testing.assert_array_equal(a, b)
        assert g[4] == 0


def test_a_nearer_unit_outside_the_cubes_is_not_found():
    # a line of cubes of side 1 and a signal at x = 0.95 (cube 0); units at x = 1.2 (cube
    # 1, inside the 27 cubes), -0.2 (clamped into cube 0, inside) and 2.05 (cube 2,
    # outside).  The unit at 2.05 (distance 1.1) is nearer than the one at -0.2 (1.15).
    units = np.array([[1.2, -0.2, 2.05], [0, 0, 0], [0, 0, 0]], np.float32)
    o = net(units)
    sig = np.array([[0.95], [0.0], [0.0]], np.float32)
    w, s, d1, d2, fb = o.find_winners_grid(sig, (0.0, -0.5, -0.5), 1.0, (4, 1, 1))
    assert (w[0], s[0], fb) == (0, 1, 0)            # the unit at 2.05 (index 2) is not seen
    ew, es, _, _ = o.find_winners(sig)
    assert (ew[0], es[0]) == (0, 2)                  # the exhaustive second is index 2


def test_fewer_than_two_candidates_fall_back_to_the_exhaustive_search():
    units = np.array([[0.1, 5.5, 7.5], [0, 0, 0], [0, 0, 0]], np.float32)
    o = net(units)
    sig = np.array([[0.2, 7.0], [0.0, 0.0], [0.0, 0.0]], np.float32)
    w, s, d1, d2, fb = o.find_winners_grid(sig, (0.0, -0.5, -0.5), 1.0, (8, 1, 1))
    # signal 0 (cube 0) sees only unit 0 (cubes 0-1); signal 1 (cube 7) sees only unit 2
    # (unit 1 is in cube 5): both fall back to the exhaustive search
    assert fb == 2
    ew, es, ed1, ed2 = o.find_winners(sig)
    np.testing.assert_array_equal(w, ew)
    np.testing.assert_array_equal(s, es)
    np.testing.assert_array_equal(d1, ed1)


def brute(units, sig, lo, h, dims):
    inv = np.float32(1.0) / np.float32(h)

    def cells(p):
        c = np.empty(p.shape, np.int64)
        for a in range(3):
            t = (p[a] - np.float32(lo[a])) * inv
            t = t.astype(np.float32)
            ca = np.where(t >= 0, np.floor(t), 0).astype(np.int64)
            c[a] = np.clip(ca, 0, dims[a] - 1)
        return c

    cu, cs = cells(units), cells(sig)
    out = []
    fb = 0
    for j in range(sig.shape[1]):
        dx = sig[0, j] - units[0]
        dy = sig[1, j] - units[1]
        dz = sig[2, j] - units[2]
        d = ((dx * dx + dy * dy) + dz * dz).astype(np.float32)
        near = np.all(np.abs(cu - cs[:, j:j + 1]) <= 1, axis=0)
        cand = np.nonzero(near)[0]
        if cand.size < 2:
            cand = np.arange(units.shape[1])
            fb += 1
        order = sorted(cand, key=lambda i: (d[i], i))
        out.append((order[0], order[1], d[order[0]], d[order[1]]))
    return out, fb


@pytest.mark.parametrize("seed,h", [(1, 0.3), (2, 0.15), (3, 0.6), (4, 0.05)])
def test_brute_force_on_small_random_inputs(seed, h):
    rng = np.random.default_rng(seed)
    units = rng.uniform(-1, 1, (3, 120)).astype(np.float32)
    sig = rng.uniform(-1.1, 1.1, (3, 200)).astype(np.float32)   # some outside the box
    lo, dims = (-1.0, -1.0, -1.0), tuple(int(np.ceil(2.0 / h)) for _ in range(3))
    o = net(units)
    w, s, d1, d2, fb = o.find_winners_grid(sig, lo, h, dims)
    want, wfb = brute(units, sig, lo, h, dims)
    assert fb == wfb
    for j, (a, b, da, db) in enumerate(want):
        assert (w[j], s[j], d1[j], d2[j]) == (a, b, da, db), j


def test_invalid_grids_are_rejected():
    o = net(np.zeros((3, 4), np.float32))
    sig = np.zeros((3, 2), np.float32)
    for lo, h, dims in (((0, 0, 0), 0.0, (2, 2, 2)), ((0, 0, 0), -1.0, (2, 2, 2)),
                        ((0, 0, 0), 1.0, (0, 2, 2))):
        with pytest.raises(oracle.OracleError):
            o.find_winners_grid(sig, lo, h, dims)
