"""Independent definitions used to pin the oracle (test helpers, not an implementation of
the multi-signal iteration).

* ``pairwise_accepted``: the survivor rule written as its definition over all pairs of
  signals (O(m^2)), not as the claim/check pass the oracle uses.
* ``SingleSignalGNG``: the textbook single-signal step of Sec. 2.1 (one signal: find the
  two nearest units, connect or reset them, age the winner's edges, move the winner and its
  neighbours, drop edges that are too old, remove units left without edges), with the
  adjacency held as a Python dict of frozensets.  With m = 1 the multi-signal iteration of
  Sec. 2.2 must reduce to exactly this.
"""
from __future__ import annotations

import numpy as np


def neighbours(edges: np.ndarray, n: int):
    """edges (3, E) -> list of sets of neighbours."""
    nb = [set() for _ in range(n)]
    for u, v in zip(edges[0], edges[1]):
        nb[int(u)].add(int(v))
        nb[int(v)].add(int(u))
    return nb


def keys(d1, m):
    bits = np.asarray(d1, np.float32).view(np.uint32).astype(np.uint64)
    return (bits << np.uint64(32)) | np.arange(m, dtype=np.uint64)


def lock_sets(edges, n, winner, second):
    nb = neighbours(edges, n)
    return [({int(b), int(s)} | nb[int(b)]) for b, s in zip(winner, second)]


def pairwise_accepted(edges, n, winner, second, d1):
    """j survives iff no other signal k with a smaller key has a lock set meeting L_j."""
    m = len(winner)
    L = lock_sets(edges, n, winner, second)
    k = keys(d1, m)
    acc = np.ones(m, np.uint8)
    for j in range(m):
        for i in range(m):
            if i != j and k[i] < k[j] and (L[i] & L[j]):
                acc[j] = 0
                break
    return acc


class SingleSignalGNG:
    """One signal at a time (Sec. 2.1), positions as float32 scalars."""

    def __init__(self, xyz, edges=None, eps_b=0.05, eps_n=0.0006, max_age=50):
        self.w = np.asarray(xyz, np.float32).T.copy()      # (n, 3)
        self.age = {}
        if edges is not None:
            for u, v, a in zip(*edges):
                self.age[frozenset((int(u), int(v)))] = int(a)
        self.eps_b, self.eps_n, self.max_age = np.float32(eps_b), np.float32(eps_n), max_age

    def nbrs(self, u):
        return sorted(next(iter(e - {u})) for e in self.age if u in e)

    def step(self, xi):
        xi = np.asarray(xi, np.float32)
        n = self.w.shape[0]
        d = [((xi[0] - self.w[i, 0]) * (xi[0] - self.w[i, 0])
              + (xi[1] - self.w[i, 1]) * (xi[1] - self.w[i, 1]))
             + (xi[2] - self.w[i, 2]) * (xi[2] - self.w[i, 2]) for i in range(n)]
        order = sorted(range(n), key=lambda i: (d[i], i))
        b, s = order[0], order[1]
        self.apply(b, s, xi)
        return b, s, d[b]

    def apply(self, b, s, xi):
        """The update half of the step for a given winner b and second s."""
        xi = np.asarray(xi, np.float32)
        nb_before = self.nbrs(b)
        for v in nb_before:
            self.age[frozenset((b, v))] += 1
        self.age[frozenset((b, s))] = 0
        for u, eps in [(b, self.eps_b)] + [(v, self.eps_n) for v in sorted(set(nb_before) | {s})]:
            for c in range(3):
                t = np.float32(xi[c] - self.w[u, c])
                t = np.float32(eps * t)
                self.w[u, c] = np.float32(self.w[u, c] + t)
        old = [e for e, a in self.age.items() if b in e and a > self.max_age]
        for e in old:
            del self.age[e]

    def edges(self):
        out = sorted((min(e), max(e), a) for e, a in self.age.items())
        return np.array(out, np.int32).T.reshape(3, -1)
