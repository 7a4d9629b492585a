"""Pins of the oracle's growing-network schedule (Sec. 3.1: the level of parallelism is the
smallest power of two above the number of units, capped at 8192; GNG insertion at regular
intervals, Sec. 2.1; stop on a threshold on the quantization error, the mean squared
distance between signals and their winners, Sec. 2.1).

The generator is pinned by the published SplitMix64 outputs; the power-of-two rule by hand;
the loop by a reference written here that drives the oracle's single steps (iterate, removal,
one insertion at a time) with signals drawn by the pinned generator and the quantization error
summed in exact integers."""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64_seed1234567.txt")
M64 = (1 << 64) - 1


def golden_outputs():
    return [int(line) for line in open(GOLDEN) if line.strip() and not line.startswith("#")]


def test_generator_matches_the_published_outputs():
    assert [oracle.splitmix64(1234567, c) for c in range(1, 6)] == golden_outputs()


def test_generator_is_counter_based():
    # output c depends only on (seed, c): the c-th output of seed s is the first output of
    # seed s + (c - 1) * gamma
    gamma = 0x9E3779B97F4A7C15
    for c in (1, 2, 17, 1000):
        assert oracle.splitmix64(99, c) == oracle.splitmix64((99 + (c - 1) * gamma) & M64, 1)


@pytest.mark.parametrize("n,m", [(1, 2), (2, 4), (3, 4), (4, 8), (7, 8), (8, 16), (1000, 1024),
                                 (1024, 2048), (4095, 4096), (4096, 8192), (5000, 8192),
                                 (8191, 8192), (8192, 8192), (100000, 8192)])
def test_level_of_parallelism(n, m):
    assert oracle.schedule_m(n, 8192) == m


def test_fixed_level_of_parallelism_and_cap():
    assert oracle.schedule_m(5000, 8192, fixed_m=1) == 1
    assert oracle.schedule_m(5000, 512) == 512
    assert oracle.schedule_m(3, 2) == 2


def torus(n, seed):
    rng = np.random.default_rng(seed)
    th = rng.uniform(0, 2 * np.pi, n)
    ph = rng.uniform(0, 2 * np.pi, n)
    x = (1 + 0.3 * np.cos(ph)) * np.cos(th)
    y = (1 + 0.3 * np.cos(ph)) * np.sin(th)
    z = 0.3 * np.sin(ph)
    return np.ascontiguousarray(np.stack([x, y, z]).astype(np.float32))


def reference_run(o, cloud, sch):
    """The schedule, written out with the oracle's single steps."""
    P = cloud.shape[1]
    it = sig_count = accepted = inserted = 0
    wsum = wcount = 0
    qe = None
    last_partial = None
    converged = False
    while True:
        n = o.sizes()[0]
        m = sch.fixed_m if sch.fixed_m > 0 else min(sch.m_cap, 1 << n.bit_length())
        idx = []
        for j in range(m):
            z = oracle.splitmix64(sch.seed, sig_count + j + 1)
            idx.append(((z >> 32) * P) >> 32)
        sig = np.ascontiguousarray(cloud[:, idx])
        w, s, d1, d2, acc = o.iterate(sig)
        for v in d1:
            f = np.float32(v)
            wsum += int(f * np.float32(2.0 ** 32)) if f < np.float32(4096.0) else 1 << 44
        accepted += int(acc.sum())
        sig_count += m
        wcount += m
        it += 1
        o.grow(0, 0)                       # removal only
        k = (sig_count // sch.insert_every - (sig_count - m) // sch.insert_every
             if sch.insert_every > 0 else 0)
        for _ in range(k):
            before = o.sizes()[0]
            o.grow(1, 1)                   # one insertion
            if o.sizes()[0] == before:
                break
            inserted += 1
        if wcount >= sch.qe_window:
            qe = float(wsum) * 2.0 ** -32 / float(wcount)
            wsum = wcount = 0
            if qe < float(np.float32(sch.qe_threshold)):
                converged = True
                break
        if sig_count >= sch.max_signals:
            break
    if qe is None and wcount > 0:
        qe = float(wsum) * 2.0 ** -32 / float(wcount)
    return dict(iterations=it, signals=sig_count, accepted=accepted, inserted=inserted,
                qe=qe, converged=int(converged))


def start(cloud, lock_mode=0, key_mode=0, n_max=400):
    p = oracle.Params(eps_b=0.05, eps_n=0.0006, max_age=50, n_max=n_max, e_max=4 * n_max,
                      m_max=512, lock_mode=lock_mode, key_mode=key_mode)
    return oracle.Oracle(p, np.ascontiguousarray(cloud[:, :2]))


@pytest.mark.parametrize("lock_mode,key_mode", [(0, 0), (1, 1)])
@pytest.mark.parametrize("sch", [
    oracle.Schedule(m_cap=512, insert_every=50, qe_window=1024, max_signals=30000,
                    qe_threshold=0.004, seed=7),
    oracle.Schedule(m_cap=64, insert_every=37, qe_window=100, max_signals=6000,
                    qe_threshold=0.0, seed=11),
    oracle.Schedule(m_cap=512, fixed_m=1, insert_every=20, qe_window=500, max_signals=1500,
                    qe_threshold=0.0, seed=3),
])
def test_schedule_equals_the_step_by_step_reference(sch, lock_mode, key_mode):
    cloud = torus(5000, 1)
    a = start(cloud, lock_mode, key_mode)
    b = start(cloud, lock_mode, key_mode)
    got = a.run_schedule(cloud, sch)
    want = reference_run(b, cloud, sch)
    for k, v in want.items():
        assert got[k] == v, k
    assert (got["n_units"], got["n_edges"]) == b.sizes()
    sa, sb = a.export(), b.export()
    for k in ("xyz", "err", "edges"):
        np.testing.assert_array_equal(sa[k], sb[k], err_msg=k)


def test_quantization_error_is_the_mean_squared_winner_distance():
    """The fixed-point window mean equals the float64 mean of d1 within the truncation."""
    cloud = torus(5000, 2)
    o = start(cloud)
    sch = oracle.Schedule(m_cap=256, insert_every=10**9, qe_window=256, max_signals=256,
                          qe_threshold=0.0, seed=5)
    # no insertion: 64 iterations at m = 4; recompute every d1 by float64 brute force
    r = o.run_schedule(cloud, sch)
    assert r["iterations"] == 64 and r["signals"] == 256
    o2 = start(cloud)
    d1s = []
    c = 0
    for _ in range(64):
        n = o2.sizes()[0]
        m = min(256, 1 << n.bit_length())
        idx = [((oracle.splitmix64(5, c + j + 1) >> 32) * 5000) >> 32 for j in range(m)]
        c += m
        sig = cloud[:, idx].astype(np.float64)
        w = o2.export()["xyz"].astype(np.float64)
        d = ((sig[:, :, None] - w[:, None, :]) ** 2).sum(axis=0)
        d1s.extend(d.min(axis=1))
        o2.iterate(np.ascontiguousarray(cloud[:, idx]))
    mean = float(np.mean(d1s))
    assert abs(r["qe"] - mean) <= 1e-6 * mean + 2.0 ** -32


def test_stops_on_the_threshold_and_on_the_signal_cap():
    cloud = torus(5000, 3)
    big = start(cloud).run_schedule(cloud, oracle.Schedule(
        m_cap=512, insert_every=20, qe_window=64, max_signals=10**6, qe_threshold=10.0, seed=1))
    assert big["converged"] == 1 and big["signals"] >= 64 and big["qe"] < 10.0
    capped = start(cloud).run_schedule(cloud, oracle.Schedule(
        m_cap=512, insert_every=20, qe_window=64, max_signals=3000, qe_threshold=0.0, seed=1))
    assert capped["converged"] == 0 and 3000 <= capped["signals"] < 3000 + 512
    assert capped["inserted"] > 0 and capped["n_units"] == 2 + capped["inserted"]


def test_invalid_schedules_are_rejected():
    cloud = torus(100, 4)
    for bad in (dict(m_cap=0), dict(m_cap=100000), dict(qe_window=0), dict(max_signals=0),
                dict(insert_every=-1), dict(fixed_m=-2), dict(qe_window=1 << 19)):
        kw = dict(m_cap=64, insert_every=10, qe_window=64, max_signals=100, seed=0)
        kw.update(bad)
        with pytest.raises(oracle.OracleError):
            start(cloud).run_schedule(cloud, oracle.Schedule(**kw))
