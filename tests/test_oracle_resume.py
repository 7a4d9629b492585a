"""Pins of the oracle as a whole-run program.

* Checkpoint and resume: a run cut after 50 iterations, exported, imported into a fresh
  network and continued for 50 more ends in the state of 100 iterations straight, bit for
  bit (the state the iteration reads is exactly positions, errors and the edge list with
  ages; Sec. 2.1).
* The implicit winner lock (Sec. 2.2): with signals placed on uniformly drawn units every
  signal's winner is its own unit, so under the winner lock the discarded fraction is the
  birthday statistic of m draws among N units, whose mean is the closed form
  1 - (N/m)(1 - (1 - 1/N)^m).
"""
import numpy as np
import pytest

import oracle
from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream


@pytest.mark.parametrize("lock_mode", [0, 1, 2])
def test_resume_equals_an_uninterrupted_run(lock_mode):
    wl = WORKLOADS["torus_grow"]
    cloud = wl.make_cloud(20_000)
    units = wl.make_units(cloud, 400)
    m, cut, total = 128, 25, 50
    p = oracle.Params(wl.eps_b, wl.eps_n, 3, wl.err_alpha, wl.err_beta, 600, 3_000, m,
                      lock_mode=lock_mode)
    stream = SignalStream(cloud, wl.signal_seed)
    batches = [stream.next(m) for _ in range(total)]
    straight = oracle.Oracle(p, units)
    for t in range(1, total + 1):
        straight.iterate(batches[t - 1], t, 5, True)
    first = oracle.Oracle(p, units)
    for t in range(1, cut + 1):
        first.iterate(batches[t - 1], t, 5, True)
    snap = first.export()
    assert not snap["orphan"].any()        # growth consumed the removal marks
    resumed = oracle.Oracle(p, units)
    resumed.import_state(snap["xyz"], snap["err"], snap["edges"])
    for t in range(cut + 1, total + 1):
        resumed.iterate(batches[t - 1], t, 5, True)
    a, b = straight.export(), resumed.export()
    for k in ("xyz", "err", "edges"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    assert straight.sizes()[0] != 400      # insertion and removal happened


@pytest.mark.parametrize("n,m", [(2_000, 256), (2_000, 2_048), (5_000, 16_384)])
def test_winner_lock_discards_the_birthday_fraction(n, m):
    rng = np.random.default_rng(11)
    units = rng.standard_normal((3, n)).astype(np.float32)
    p = oracle.Params(0.05, 0.0006, 50, 0.5, 0.995, n, 4 * n, m, lock_mode=1)
    o = oracle.Oracle(p, units)
    trials = 8
    rates = []
    for _ in range(trials):
        pick = rng.integers(0, n, m)
        sig = np.ascontiguousarray(units[:, pick])
        w, s, d1, _ = o.find_winners(sig)
        np.testing.assert_array_equal(w, pick)      # a signal on a unit finds that unit
        acc = o.resolve_conflicts(w, s, d1)
        # exactly one survivor per distinct winner (the implicit lock on the winner)
        assert int(acc.sum()) == len(np.unique(pick))
        rates.append(1.0 - acc.sum() / m)
    expected = 1.0 - (n / m) * (1.0 - (1.0 - 1.0 / n) ** m)
    # variance of the number of distinct values among m uniform draws from n
    q1, q2 = (1 - 1 / n) ** m, (1 - 2 / n) ** m
    var_distinct = n * q1 + n * (n - 1) * q2 - (n * q1) ** 2
    sd_mean_rate = np.sqrt(max(var_distinct, 0.0)) / m / np.sqrt(trials)
    assert abs(np.mean(rates) - expected) <= 5 * sd_mean_rate + 1e-12
