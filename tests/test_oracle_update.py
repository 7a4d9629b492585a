"""Pins of the oracle's update steps: conflict resolution (Sec. 2.2, collision kinds and
the implicit lock), adaptation (Sec. 2.1, Eq. adaptation with eta = 1 iff connected), the
edge update (Sec. 2.1 step 3 and its aging footnote) and growth (Sec. 2.1, GNG insertion
near the unit of largest error; removal of units left without edges).
"""
import numpy as np
import pytest

import oracle
from pins import SingleSignalGNG, keys, lock_sets, pairwise_accepted


def net(units, edges=None, err=None, m_max=512, **kw):
    units = np.asarray(units, np.float32)
    if units.shape[0] != 3:
        units = units.T
    n = units.shape[1]
    p = oracle.Params(n_max=kw.pop("n_max", n + 8), e_max=kw.pop("e_max", 8 * n + 16),
                      m_max=m_max, **kw)
    o = oracle.Oracle(p, units)
    if edges is not None or err is not None:
        o.import_state(units, err, None if edges is None else np.asarray(edges, np.int32))
    return o


def random_graph(rng, n, e):
    pairs = set()
    while len(pairs) < e:
        u, v = rng.integers(0, n, 2)
        if u != v:
            pairs.add((min(u, v), max(u, v)))
    pairs = sorted(pairs)
    ages = rng.integers(0, 6, len(pairs))
    return np.array([[p[0] for p in pairs], [p[1] for p in pairs], ages], np.int32)


# ----------------------------------------------------------------- resolve -------

@pytest.mark.parametrize("seed,n,e,m", [(0, 30, 40, 25), (1, 200, 500, 120), (2, 12, 0, 40),
                                        (3, 500, 1400, 300)])
def test_resolve_matches_pairwise_definition(seed, n, e, m):
    rng = np.random.default_rng(seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    edges = random_graph(rng, n, e)
    o = net(units, edges)
    sig = rng.standard_normal((3, m)).astype(np.float32)
    w, s, d1, _ = o.find_winners(sig)
    acc = o.resolve_conflicts(w, s, d1)
    np.testing.assert_array_equal(acc, pairwise_accepted(edges, n, w, s, d1))
    # accepted lock sets are pairwise disjoint, and the smallest key always survives
    L = lock_sets(edges, n, w, s)
    seen = set()
    for j in np.flatnonzero(acc):
        assert not (L[j] & seen)
        seen |= L[j]
    assert acc[int(np.argmin(keys(d1, m)))] == 1


def test_resolve_hand_cases():
    # 4 units on a line, no edges; signals 0 and 1 share winner 0 -> smaller d1 survives
    units = np.array([[0, 1, 10, 11], [0, 0, 0, 0], [0, 0, 0, 0]], np.float32)
    o = net(units)
    w = np.array([0, 0, 2], np.int32)
    s = np.array([1, 1, 3], np.int32)
    acc = o.resolve_conflicts(w, s, np.float32([0.5, 0.25, 0.5]))
    np.testing.assert_array_equal(acc, [0, 1, 1])
    # equal distance: the lower signal index survives
    acc = o.resolve_conflicts(w, s, np.float32([0.25, 0.25, 0.5]))
    np.testing.assert_array_equal(acc, [1, 0, 1])
    # a single signal is always accepted
    np.testing.assert_array_equal(o.resolve_conflicts(w[:1], s[:1], np.float32([9.0])), [1])
    # different winners but a shared second: conflict
    acc = o.resolve_conflicts(np.int32([0, 2]), np.int32([1, 1]), np.float32([1.0, 2.0]))
    np.testing.assert_array_equal(acc, [1, 0])


def test_resolve_neighbourhood_conflict():
    # path 0-1-2-3; winners 0 and 2 (seconds 4 and 5): N(0) = {1}, N(2) = {1, 3} meet at 1
    units = np.zeros((3, 6), np.float32)
    edges = np.array([[0, 1, 2], [1, 2, 3], [0, 0, 0]], np.int32)
    o = net(units, edges)
    acc = o.resolve_conflicts(np.int32([0, 2]), np.int32([4, 5]), np.float32([3.0, 1.0]))
    np.testing.assert_array_equal(acc, [0, 1])


def test_resolve_rejects_bad_indices():
    o = net(np.zeros((3, 4), np.float32))
    with pytest.raises(oracle.OracleError):
        o.resolve_conflicts(np.int32([0]), np.int32([0]), np.float32([0]))
    with pytest.raises(oracle.OracleError):
        o.resolve_conflicts(np.int32([4]), np.int32([0]), np.float32([0]))


# ------------------------------------------------------------------- adapt -------

def test_single_signal_hand_worked():
    """Units (0,0,0), (1,0,0), (0,2,0); signal (0.4,0,0); eps_b = 0.5, eps_n = 0.25.
    b = 0 moves half way to 0.2; s = 1 moves a quarter of the way: 1 + 0.25 (0.4 - 1) =
    0.85; unit 2 stays; edge {0, 1} is created at age 0."""
    units = np.array([[0, 1, 0], [0, 0, 2], [0, 0, 0]], np.float32)
    o = net(units, eps_b=0.5, eps_n=0.25)
    sig = np.float32([[0.4], [0.0], [0.0]])
    w, s, d1, d2, acc = o.iterate(sig)
    st = o.export()
    assert (w[0], s[0], acc[0]) == (0, 1, 1)
    assert st["xyz"][0, 0] == np.float32(0.2)       # 0.4f * 0.5 is exact
    assert abs(float(st["xyz"][0, 1]) - 0.85) < 1e-7
    np.testing.assert_array_equal(st["xyz"][:, 2], units[:, 2])
    np.testing.assert_array_equal(st["xyz"][1:, :2], units[1:, :2])
    np.testing.assert_array_equal(st["edges"], [[0], [1], [0]])
    # error: d1 = 0.16 accumulated on the winner, then decayed by beta
    assert abs(float(st["err"][0]) - 0.16 * 0.995) < 1e-7 and st["err"][1] == 0


def test_adapt_moves_exactly_the_lock_sets():
    rng = np.random.default_rng(5)
    n, m = 300, 150
    units = rng.standard_normal((3, n)).astype(np.float32)
    edges = random_graph(rng, n, 600)
    o = net(units, edges, eps_b=0.05, eps_n=0.0006)
    sig = rng.standard_normal((3, m)).astype(np.float32)
    w, s, d1, d2, acc = o.iterate(sig)
    after = o.export()["xyz"]
    L = lock_sets(edges, n, w, s)
    moved = set().union(*[L[j] for j in np.flatnonzero(acc)])
    untouched = np.array(sorted(set(range(n)) - moved))
    np.testing.assert_array_equal(after[:, untouched], units[:, untouched])
    x64 = units.astype(np.float64)
    for j in np.flatnonzero(acc):
        b = w[j]
        # the winner moves eps_b of the way to its signal (one rounding per operation)
        expect = x64[:, b] + 0.05 * (sig[:, j].astype(np.float64) - x64[:, b])
        np.testing.assert_allclose(after[:, b], expect, rtol=0, atol=4e-7)
        for v in L[j] - {int(b)}:
            expect = x64[:, v] + np.float64(np.float32(0.0006)) * (sig[:, j] - x64[:, v])
            np.testing.assert_allclose(after[:, v], expect, rtol=0, atol=4e-7)


def test_zero_learning_rates_do_not_move_units():
    rng = np.random.default_rng(6)
    units = rng.standard_normal((3, 50)).astype(np.float32)
    o = net(units, random_graph(rng, 50, 80), eps_b=0.0, eps_n=0.0)
    for _ in range(3):
        o.iterate(rng.standard_normal((3, 20)).astype(np.float32))
    np.testing.assert_array_equal(o.export()["xyz"], units)


# ------------------------------------------------------------------- edges -------

def test_edge_aging_reset_and_pruning_hand_worked():
    # star around 0: edges {0,1} age 5, {0,2} age 3, {0,3} age 0; {1,2} age 7 (not at 0)
    units = np.array([[0, 1, -1, 0, 5], [0, 0, 0, 1, 5], [0, 0, 0, 0, 5]], np.float32)
    edges = np.array([[0, 0, 0, 1], [1, 2, 3, 2], [5, 3, 0, 7]], np.int32)
    o = net(units, edges, max_age=5)
    # b = 0, s = 3 (existing edge): everything at 0 ages, {0,3} resets, {0,1} reaches 6 > 5
    o.update_edges(np.int32([0]), np.int32([3]), np.uint8([1]))
    st = o.export()
    np.testing.assert_array_equal(st["edges"], [[0, 0, 1], [2, 3, 2], [4, 0, 7]])
    assert st["orphan"].sum() == 0        # unit 1 still has {1,2}
    # b = 4 (isolated), s = 2: new edge {2,4} at age 0
    o.update_edges(np.int32([4]), np.int32([2]), np.uint8([1]))
    st = o.export()
    np.testing.assert_array_equal(st["edges"], [[0, 0, 1, 2], [2, 3, 2, 4], [4, 0, 7, 0]])
    # rejected signals change nothing
    o.update_edges(np.int32([0]), np.int32([1]), np.uint8([0]))
    np.testing.assert_array_equal(o.export()["edges"], st["edges"])


def test_pruning_marks_orphans_and_grow_removes_them():
    # path 3-0-1, unit 2 never connected; {0,1} at age 9 with max_age 9: ages to 10 and goes
    units = np.array([[0, 1, 2, 3], [0, 0, 0, 0], [0, 0, 0, 0]], np.float32)
    edges = np.array([[0, 0], [1, 3], [9, 0]], np.int32)
    err = np.float32([1, 2, 3, 4])
    o = net(units, edges, err, max_age=9)
    o.update_edges(np.int32([0]), np.int32([3]), np.uint8([1]))
    st = o.export()
    np.testing.assert_array_equal(st["orphan"], [0, 1, 0, 0])
    np.testing.assert_array_equal(st["edges"], [[0], [3], [0]])
    o.grow(iteration=1, insert_every=0)
    st = o.export()
    assert o.sizes() == (3, 1)
    # unit 1 removed: 2 -> 1, 3 -> 2 (never-connected unit 2 stays)
    np.testing.assert_array_equal(st["xyz"][0], [0, 2, 3])
    np.testing.assert_array_equal(st["err"], [1, 3, 4])
    np.testing.assert_array_equal(st["edges"], [[0], [2], [0]])


def test_grow_inserts_between_largest_error_units():
    # path 0-1-2-3 with errors; q = 2 (largest), f = argmax err over {1, 3} = 3
    units = np.array([[0, 1, 2, 4], [0, 0, 0, 0], [0, 0, 0, 0]], np.float32)
    edges = np.array([[0, 1, 2], [1, 2, 3], [4, 2, 7]], np.int32)
    err = np.float32([1.0, 5.0, 8.0, 6.0])
    o = net(units, edges, err, err_alpha=0.5)
    o.grow(iteration=10, insert_every=10)
    st = o.export()
    assert o.sizes() == (5, 4)
    np.testing.assert_array_equal(st["xyz"][:, 4], [3.0, 0.0, 0.0])   # midpoint of 2 and 3
    np.testing.assert_array_equal(st["err"], np.float32([1.0, 5.0, 4.0, 3.0, 4.0]))
    np.testing.assert_array_equal(st["edges"], [[0, 1, 2, 3], [1, 2, 4, 4], [4, 2, 0, 0]])
    # not a multiple of the interval: nothing happens
    o.grow(iteration=11, insert_every=10)
    assert o.sizes() == (5, 4)


def test_grow_tie_rules_and_skip_when_isolated():
    units = np.zeros((3, 4), np.float32)
    # equal errors everywhere: q = 0; its neighbours {1, 3} tie: f = 1
    o = net(units, np.array([[0, 0], [1, 3], [0, 0]], np.int32), np.float32([2, 2, 2, 2]))
    o.grow(iteration=1, insert_every=1)
    np.testing.assert_array_equal(o.export()["edges"], [[0, 0, 1], [3, 4, 4], [0, 0, 0]])
    # q without neighbours: no insertion
    o = net(units, np.array([[1], [2], [0]], np.int32), np.float32([9, 1, 1, 1]))
    o.grow(iteration=1, insert_every=1)
    assert o.sizes() == (4, 1)


def test_capacity_errors_are_reported():
    units = np.zeros((3, 6), np.float32)
    o = net(units, e_max=1)
    with pytest.raises(oracle.OracleError) as e:
        o.update_edges(np.int32([0, 2]), np.int32([1, 3]), np.uint8([1, 1]))
    assert e.value.code == oracle.E_CAPACITY
    assert o.status() == oracle.E_CAPACITY


# ----------------------------------------------------------- m = 1 reduction -------

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_one_signal_per_iteration_is_the_single_signal_algorithm(seed):
    """Sec. 2.2 with m = 1 is the basic iteration of Sec. 2.1, step by step."""
    rng = np.random.default_rng(seed)
    n = 40
    units = rng.standard_normal((3, n)).astype(np.float32)
    edges = random_graph(rng, n, 60)
    edges[2] = rng.integers(0, 4, edges.shape[1])
    o = net(units, edges, eps_b=0.2, eps_n=0.05, max_age=3, m_max=1)
    ref = SingleSignalGNG(units, edges, eps_b=0.2, eps_n=0.05, max_age=3)
    for _ in range(60):
        xi = rng.standard_normal((3, 1)).astype(np.float32)
        w, s, d1, d2, acc = o.iterate(xi)
        b, sc, db = ref.step(xi[:, 0])
        assert (w[0], s[0], acc[0]) == (b, sc, 1) and d1[0] == db
        st = o.export()
        np.testing.assert_array_equal(st["xyz"], ref.w.T)
        np.testing.assert_array_equal(st["edges"], ref.edges())
