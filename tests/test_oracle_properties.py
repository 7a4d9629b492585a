"""Property checks of the oracle over random tiny networks and several iterations,
including forced ties (duplicated units, signals on units, integer grids).  After every
iteration:
  * winner / second are the first two of a lexicographic sort on (d, index);
  * the accepted mask equals the pairwise definition of the survivor rule;
  * units outside every accepted lock set are bitwise unchanged;
  * every accepted winner-second edge exists at age 0, the edge list is canonical;
  * no edge at an accepted winner is older than max_age; other edges keep their ages.
"""
import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from pins import lock_sets, pairwise_accepted
from test_oracle_find_winners import fp32_distances


@st.composite
def scenario(draw):
    n = draw(st.integers(2, 40))
    m = draw(st.integers(1, 40))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    grid = draw(st.sampled_from([0, 2, 5]))        # 0: continuous coordinates
    max_age = draw(st.integers(0, 6))
    return n, m, seed, grid, max_age


def coords(rng, shape, grid):
    if grid:
        return rng.integers(-grid, grid + 1, shape).astype(np.float32)
    return rng.standard_normal(shape).astype(np.float32)


@settings(max_examples=60, deadline=None)
@given(scenario())
def test_iteration_invariants(sc):
    n, m, seed, grid, max_age = sc
    rng = np.random.default_rng(seed)
    units = coords(rng, (3, n), grid)
    if n > 3:
        units[:, 1] = units[:, 0]                   # a duplicated unit
    p = oracle.Params(eps_b=0.3, eps_n=0.1, max_age=max_age, n_max=n, e_max=4 * n * n,
                      m_max=m)
    o = oracle.Oracle(p, units)
    for _ in range(4):
        before = o.export()
        sig = coords(rng, (3, m), grid)
        if m > 2:
            sig[:, 0] = before["xyz"][:, 0]         # a signal exactly on a unit
        w, s, d1, d2, acc = o.iterate(sig)
        after = o.export()
        D = fp32_distances(before["xyz"], sig)
        idx = np.arange(n)
        for j in range(m):
            order = np.lexsort((idx, D[j]))
            assert (w[j], s[j]) == (order[0], order[1])
        np.testing.assert_array_equal(acc, pairwise_accepted(before["edges"], n, w, s, d1))
        L = lock_sets(before["edges"], n, w, s)
        touched = set().union(set(), *[L[j] for j in np.flatnonzero(acc)])
        winners = {int(w[j]) for j in np.flatnonzero(acc)}
        for u in set(range(n)) - touched:
            np.testing.assert_array_equal(after["xyz"][:, u], before["xyz"][:, u])
        e = after["edges"]
        assert np.all(e[0] < e[1])
        pairs = list(zip(e[0].tolist(), e[1].tolist()))
        assert pairs == sorted(set(pairs))
        age = {(u, v): a for u, v, a in zip(*e.tolist())}
        for j in np.flatnonzero(acc):
            b, c = int(w[j]), int(s[j])
            assert age[(min(b, c), max(b, c))] == 0
        old = {(u, v): a for u, v, a in zip(*before["edges"].tolist())}
        for (u, v), a in age.items():
            if u in winners or v in winners:
                assert a <= max_age
            elif (u, v) in old:
                assert a == old[(u, v)]
