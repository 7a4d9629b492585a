"""Pins of the oracle's find-winners step (Sec. 2.1 step 2, Sec. 2.2 step 2: for each
signal, the nearest and second-nearest units by exhaustive search, k = 2).

Independent checks, none of which reuses the oracle's scan:
  * float64 brute force: where the exact distances leave clear gaps, the winner and second
    must be the exact nearest two, and d1, d2 must be the binary32 distances within the
    rounding bound of five operations;
  * selection by a full lexicographic sort of (distance, index), which pins the tie rule;
  * closed-form special cases (a signal on a unit, two units, symmetric ties, duplicates);
  * invariants d1 <= d2, winner != second; independence of the thread count.
"""
import numpy as np
import pytest

import oracle

U = 2.0 ** -24


def make(units, m_max=4096, **kw):
    units = np.asarray(units, np.float32)
    if units.shape[0] != 3:
        units = units.T
    p = oracle.Params(n_max=max(2, units.shape[1]), e_max=8 * units.shape[1] + 8,
                      m_max=m_max, **kw)
    return oracle.Oracle(p, units)


def exact_d(units, sig):
    """(m, N) float64 squared distances from the binary32 inputs (exact up to 1 ulp of
    float64, far below every margin used here)."""
    u = np.asarray(units, np.float64)
    s = np.asarray(sig, np.float64)
    return ((s[:, :, None] - u[:, None, :]) ** 2).sum(axis=0)


@pytest.mark.parametrize("seed,n,m", [(0, 2, 1), (1, 3, 7), (2, 64, 64), (3, 1000, 256),
                                      (4, 3000, 97)])
def test_matches_float64_brute_force_where_gaps_are_clear(seed, n, m):
    rng = np.random.default_rng(seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    sig = rng.standard_normal((3, m)).astype(np.float32)
    w, s, d1, d2 = make(units).find_winners(sig)
    D = exact_d(units, sig)
    order = np.argsort(D, axis=1, kind="stable")
    rows = np.arange(m)
    e1, e2 = D[rows, order[:, 0]], D[rows, order[:, 1]]
    e3 = D[rows, order[:, 2]] if n > 2 else np.full(m, np.inf)
    # binary32 result of 5 rounded operations on non-negative terms: |d - D| <= 5u D / (1-5u)
    tol = 6 * U
    clear = (e2 - e1 > 4 * tol * e2) & ((e3 == np.inf) | (e3 - e2 > 4 * tol * e3))
    assert clear.mean() > 0.9
    np.testing.assert_array_equal(w[clear], order[clear, 0])
    np.testing.assert_array_equal(s[clear], order[clear, 1])
    np.testing.assert_allclose(d1.astype(np.float64), D[rows, w], rtol=tol, atol=1e-38)
    np.testing.assert_allclose(d2.astype(np.float64), D[rows, s], rtol=tol, atol=1e-38)


def fp32_distances(units, sig):
    """binary32 distances evaluated by numpy, one rounding per array operation."""
    u = np.asarray(units, np.float32)
    s = np.asarray(sig, np.float32)
    dx = s[0][:, None] - u[0][None, :]
    dy = s[1][:, None] - u[1][None, :]
    dz = s[2][:, None] - u[2][None, :]
    return (dx * dx + dy * dy) + dz * dz


@pytest.mark.parametrize("seed,n,m,grid", [(5, 50, 200, 4), (6, 500, 300, 3),
                                           (7, 17, 64, 1)])
def test_tie_rule_matches_lexicographic_sort(seed, n, m, grid):
    """Units and signals on a coarse integer grid produce many exact ties; the winner and
    second must be the first two entries of a lexicographic sort on (d, index)."""
    rng = np.random.default_rng(seed)
    units = rng.integers(-grid, grid + 1, (3, n)).astype(np.float32)
    sig = rng.integers(-grid, grid + 1, (3, m)).astype(np.float32)
    w, s, d1, d2 = make(units).find_winners(sig)
    D = fp32_distances(units, sig)
    idx = np.arange(n)
    for j in range(m):
        order = np.lexsort((idx, D[j]))
        assert (w[j], s[j]) == (order[0], order[1])
        assert d1[j] == D[j, order[0]] and d2[j] == D[j, order[1]]


def test_invariants_and_thread_independence():
    rng = np.random.default_rng(11)
    units = rng.standard_normal((3, 4000)).astype(np.float32)
    sig = rng.standard_normal((3, 1000)).astype(np.float32)
    o = make(units)
    a = o.find_winners(sig)
    o.threads = 4
    b = o.find_winners(sig)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    w, s, d1, d2 = a
    assert np.all(w != s)
    assert np.all(d1 <= d2)
    assert np.all((w >= 0) & (w < 4000) & (s >= 0) & (s < 4000))


def test_signal_on_a_unit_gives_zero_distance():
    rng = np.random.default_rng(3)
    units = rng.standard_normal((3, 100)).astype(np.float32)
    sig = units[:, [5, 17, 99]].copy()
    w, s, d1, d2 = make(units).find_winners(sig)
    np.testing.assert_array_equal(w, [5, 17, 99])
    assert np.all(d1 == 0.0) and not np.any(np.signbit(d1))
    assert np.all(d2 > 0.0)


def test_two_units():
    units = np.array([[0.0, 3.0], [0.0, 0.0], [0.0, 0.0]], np.float32)
    sig = np.array([[1.0, 2.0, 1.5], [0.0, 0.0, 0.0], [0.0, 0.0, 0.0]], np.float32)
    w, s, d1, d2 = make(units).find_winners(sig)
    np.testing.assert_array_equal(w, [0, 1, 0])      # 1.5 is equidistant: lower index
    np.testing.assert_array_equal(s, [1, 0, 1])
    np.testing.assert_array_equal(d1, np.float32([1.0, 1.0, 2.25]))
    np.testing.assert_array_equal(d2, np.float32([4.0, 4.0, 2.25]))


def test_symmetric_tie_and_duplicates():
    # units at -e_x, +e_x, a duplicate of +e_x, and a far unit; signal at the origin
    units = np.array([[-1, 1, 1, 5], [0, 0, 0, 0], [0, 0, 0, 0]], np.float32)
    sig = np.array([[0.0, 1.0], [0.0, 0.0], [0.0, 0.0]], np.float32)
    w, s, d1, d2 = make(units).find_winners(sig)
    assert (w[0], s[0], d1[0], d2[0]) == (0, 1, 1.0, 1.0)
    # a signal on the duplicated unit: both copies at distance 0, lower index wins
    assert (w[1], s[1], d1[1], d2[1]) == (1, 2, 0.0, 0.0)


def test_hand_worked_single_signal():
    """Units (0,0,0), (1,0,0), (0,2,0); signal (0.4,0,0): squared distances 0.16, 0.36,
    4.16, so b = 0 and s = 1."""
    units = np.array([[0, 1, 0], [0, 0, 2], [0, 0, 0]], np.float32)
    sig = np.array([[0.4], [0.0], [0.0]], np.float32)
    w, s, d1, d2 = make(units).find_winners(sig)
    assert (w[0], s[0]) == (0, 1)
    assert abs(float(d1[0]) - 0.16) < 1e-7 and abs(float(d2[0]) - 0.36) < 1e-7


def test_argument_errors():
    o = make(np.zeros((3, 1), np.float32).repeat(2, axis=1))
    with pytest.raises(oracle.OracleError):
        o.find_winners(np.zeros((3, 5000), np.float32))   # m > m_max
    one = oracle.Oracle(oracle.Params(n_max=4, e_max=4, m_max=4), np.zeros((3, 1), np.float32))
    with pytest.raises(oracle.OracleError):
        one.find_winners(np.zeros((3, 1), np.float32))    # fewer than two units
    w, s, d1, d2 = o.find_winners(np.zeros((3, 0), np.float32))
    assert w.shape == (0,)
