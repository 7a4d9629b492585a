"""Pins of the greedy lock-set rule (lock_mode 2): the lock sets {b, s} + N(b) of the
lock-set reading of Sec. 2.2, with signals taken in key order and accepted iff their lock
set is disjoint from those accepted before them (R10's one round re-admits nobody).

The result is pinned by its characterization rather than by a second copy of the loop:
a set of signals whose lock sets are pairwise disjoint and such that every other signal
meets the lock set of an accepted signal of smaller key is unique (by induction over the
key order) and is what the greedy order yields."""
import numpy as np
import pytest

import oracle

from test_oracle_paper_lock import random_graph


def make(units, edges, lock_mode, key_mode=0, m_max=512):
    n = units.shape[1]
    o = oracle.Oracle(oracle.Params(n_max=n + 8, e_max=8 * n + 16, m_max=m_max,
                                    lock_mode=lock_mode, key_mode=key_mode), units)
    if edges is not None:
        o.import_state(units, None, edges)
    return o


def lock_sets(edges, n, w, s):
    nb = [set() for _ in range(n)]
    for u, v in zip(edges[0], edges[1]):
        nb[u].add(v)
        nb[v].add(u)
    return [{int(w[j]), int(s[j])} | nb[int(w[j])] for j in range(len(w))]


def key(d1, j, key_mode):
    return j if key_mode == 1 else (int(np.float32(d1).view(np.uint32)) << 32) | j


@pytest.mark.parametrize("key_mode", [0, 1])
@pytest.mark.parametrize("seed,n,e,m", [(0, 30, 40, 40), (1, 100, 200, 150), (2, 400, 900, 500),
                                        (3, 15, 0, 30)])
def test_greedy_is_the_unique_key_ordered_maximal_set(seed, n, e, m, key_mode):
    rng = np.random.default_rng(seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    edges = random_graph(rng, n, e)
    o = make(units, edges, 2, key_mode)
    sig = rng.standard_normal((3, m)).astype(np.float32)
    w, s, d1, d2 = o.find_winners(sig)
    acc = o.resolve_conflicts(w, s, d1)
    L = lock_sets(edges, n, w, s)
    keys = [key(d1[j], j, key_mode) for j in range(m)]
    A = [j for j in range(m) if acc[j]]
    for a in range(len(A)):                       # pairwise disjoint
        for b in range(a + 1, len(A)):
            assert not (L[A[a]] & L[A[b]])
    for j in range(m):                            # every rejected one is blocked by an
        if not acc[j]:                            # accepted one of smaller key
            assert any(L[j] & L[k] and keys[k] < keys[j] for k in A)
    # the one-round rule accepts a subset
    one = make(units, edges, 0, key_mode).resolve_conflicts(w, s, d1)
    assert np.all(acc[one == 1] == 1)
    assert acc.sum() >= one.sum()


def test_a_chain_of_three():
    # units on a line 0 - 1 - 2 - 3 - 4 - 5, edges between neighbours; three signals whose
    # lock sets form a chain: A meets B, B meets C, A and C are disjoint, keys A < B < C
    units = np.array([[0, 1, 2, 3, 4, 5, 10, 11], [0] * 8, [0] * 8], np.float32)
    edges = np.array([[0, 1, 2, 3, 4], [1, 2, 3, 4, 5], [0] * 5], np.int32)
    w = np.array([0, 2, 4], np.int32)     # A locks {0, 1}, B {2, 1, 3}, C {4, 3, 5}
    s = np.array([1, 3, 5], np.int32)
    d1 = np.array([0.1, 0.2, 0.3], np.float32)
    assert make(units, edges, 0).resolve_conflicts(w, s, d1).tolist() == [1, 0, 0]
    assert make(units, edges, 2).resolve_conflicts(w, s, d1).tolist() == [1, 0, 1]


def test_the_update_is_the_lock_set_update_of_the_greedy_survivors():
    rng = np.random.default_rng(8)
    n = 200
    units = rng.standard_normal((3, n)).astype(np.float32)
    edges = random_graph(rng, n, 500)
    g = make(units, edges, 2)
    r = make(units, edges, 0)
    for it in range(5):
        sig = rng.standard_normal((3, 300)).astype(np.float32)
        w, s, d1, d2, acc = g.iterate(sig)
        r.adapt(sig, w, s, d1, acc)              # lock-set update fed with the same survivors
        r.update_edges(w, s, acc)
        a, b = g.export(), r.export()
        for f in ("xyz", "err", "edges"):
            np.testing.assert_array_equal(a[f], b[f], err_msg=f"iteration {it} {f}")
