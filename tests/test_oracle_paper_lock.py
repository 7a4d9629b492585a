"""The paper's own collision rule (Sec. 2.2): an implicit lock on the winner unit, the first
incoming signal of each winner survives and the others are discarded; the survivors update
the network one after another.  Pinned against the textbook single-signal step of Sec. 2.1
(``pins.SingleSignalGNG``, a dict-of-edges implementation written independently of the
oracle), applied survivor by survivor with the snapshot's winners and seconds."""
import numpy as np
import pytest

import oracle
from pins import SingleSignalGNG

pytestmark = pytest.mark.filterwarnings("ignore")


def net(units, edges=None, m_max=512, **kw):
    n = units.shape[1]
    p = oracle.Params(n_max=n + 8, e_max=8 * n + 16, m_max=m_max, **kw)
    o = oracle.Oracle(p, units)
    if edges is not None:
        o.import_state(units, None, np.asarray(edges, np.int32))
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


def nearest_two(w, xi):
    """Lexicographic (d, index) top-2 with the binary32 direct-form distance."""
    d = [((xi[0] - w[i, 0]) * (xi[0] - w[i, 0]) + (xi[1] - w[i, 1]) * (xi[1] - w[i, 1]))
         + (xi[2] - w[i, 2]) * (xi[2] - w[i, 2]) for i in range(w.shape[0])]
    order = sorted(range(w.shape[0]), key=lambda i: (d[i], i))
    return order[0], order[1], np.float32(d[order[0]])


def key_of(mode, d1, j):
    return j if mode == 1 else (int(np.float32(d1).view(np.uint32)) << 32) | j


@pytest.mark.parametrize("key_mode", [0, 1])
@pytest.mark.parametrize("seed,n,e,m", [(0, 30, 40, 25), (1, 80, 150, 120), (2, 12, 0, 40),
                                        (3, 200, 500, 300)])
def test_survivors_update_one_after_another(key_mode, seed, n, e, m):
    rng = np.random.default_rng(seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    edges = random_graph(rng, n, e)
    kw = dict(eps_b=0.2, eps_n=0.05, max_age=3)
    o = net(units, edges, m_max=m, lock_mode=1, key_mode=key_mode, **kw)
    ref = SingleSignalGNG(units, edges, **kw)
    err = np.zeros(n, np.float32)
    for it in range(6):
        sig = rng.standard_normal((3, m)).astype(np.float32)
        w, s, d1, d2, acc = o.iterate(sig)
        # the snapshot: every signal's winner and second on the network before the iteration
        snap = [nearest_two(ref.w, sig[:, j]) for j in range(m)]
        assert [(b, c) for b, c, _ in snap] == list(zip(w.tolist(), s.tolist()))
        # survivors: the smallest key of each winner unit
        best = {}
        for j, (b, c, db) in enumerate(snap):
            k = key_of(key_mode, db, j)
            if b not in best or k < best[b][0]:
                best[b] = (k, j)
        expect = np.zeros(m, np.uint8)
        for _, j in best.values():
            expect[j] = 1
        np.testing.assert_array_equal(acc, expect, err_msg=f"iteration {it}")
        # the survivors' single-signal steps in ascending key order
        for k, j in sorted(best.values()):
            b, c, db = snap[j]
            ref.apply(b, c, sig[:, j])
            err[b] = np.float32(err[b] + db)
        err = (err * np.float32(0.995)).astype(np.float32)
        st = o.export()
        np.testing.assert_array_equal(st["xyz"], ref.w.T, err_msg=f"iteration {it}")
        np.testing.assert_array_equal(st["edges"], ref.edges(), err_msg=f"iteration {it}")
        np.testing.assert_array_equal(st["err"], err, err_msg=f"iteration {it}")


def test_one_signal_per_iteration_is_the_single_signal_algorithm():
    """With m = 1 the paper's rule, like the lock-set rule, is the basic iteration."""
    rng = np.random.default_rng(9)
    n = 40
    units = rng.standard_normal((3, n)).astype(np.float32)
    edges = random_graph(rng, n, 60)
    o = net(units, edges, m_max=1, lock_mode=1, key_mode=1, eps_b=0.2, eps_n=0.05, max_age=3)
    ref = SingleSignalGNG(units, edges, eps_b=0.2, eps_n=0.05, max_age=3)
    for _ in range(60):
        xi = rng.standard_normal((3, 1)).astype(np.float32)
        w, s, d1, d2, acc = o.iterate(xi)
        b, sc, db = ref.step(xi[:, 0])
        assert (w[0], s[0], acc[0]) == (b, sc, 1) and d1[0] == db
        st = o.export()
        np.testing.assert_array_equal(st["xyz"], ref.w.T)
        np.testing.assert_array_equal(st["edges"], ref.edges())


def test_disjoint_lock_sets_give_the_lock_set_result():
    """When every signal's lock set {b, s} + N(b) is disjoint from the others', both rules
    accept every signal and the order of the updates does not matter."""
    rng = np.random.default_rng(4)
    # clusters of three units far apart; one signal next to each cluster's first unit
    centres = rng.standard_normal((3, 20)).astype(np.float32) * 100
    units = np.concatenate([centres + np.float32(0.01) * k for k in range(3)], axis=1)
    n = units.shape[1]
    edges = np.array([list(range(20)), list(range(20, 40)), [1] * 20], np.int32)
    sig = (centres + np.float32(0.001)).astype(np.float32)
    outs = []
    for lock_mode in (0, 1):
        o = net(units, edges, m_max=20, lock_mode=lock_mode, eps_b=0.2, eps_n=0.05, max_age=3)
        w, s, d1, d2, acc = o.iterate(sig)
        assert acc.all()
        outs.append(o.export())
    np.testing.assert_array_equal(outs[0]["xyz"], outs[1]["xyz"])
    np.testing.assert_array_equal(outs[0]["edges"], outs[1]["edges"])
    np.testing.assert_array_equal(outs[0]["err"], outs[1]["err"])


def test_modes_are_validated():
    units = np.zeros((3, 4), np.float32)
    for bad in (dict(lock_mode=3), dict(key_mode=-1)):
        with pytest.raises(oracle.OracleError):
            oracle.Oracle(oracle.Params(n_max=8, e_max=8, m_max=4, **bad), units)
