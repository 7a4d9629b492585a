"""GPU parity of the growing-network schedule (Sec. 3.1 level of parallelism, GNG insertion
at regular intervals and the quantization-error stop of Sec. 2.1) against the oracle's
schedule: iteration, signal, acceptance and insertion counts, the window mean (bit for bit),
the stop, and the final network (positions, errors and edges bit for bit), in both collision
rules."""
import numpy as np
import pytest

from parity import oracle_threads

pytestmark = pytest.mark.gpu


def torus(n, seed):
    rng = np.random.default_rng(seed)
    th = rng.uniform(0, 2 * np.pi, n)
    ph = rng.uniform(0, 2 * np.pi, n)
    x = (1 + 0.3 * np.cos(ph)) * np.cos(th)
    y = (1 + 0.3 * np.cos(ph)) * np.sin(th)
    z = 0.3 * np.sin(ph)
    return np.ascontiguousarray(np.stack([x, y, z]).astype(np.float32))


def pair(cloud, n_max, m_max, lock_mode, key_mode, max_age=50):
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    units = np.ascontiguousarray(cloud[:, :2])
    kw = dict(eps_b=0.05, eps_n=0.0006, max_age=max_age, err_alpha=0.5, err_beta=0.995)
    g = gsn.Network(gsn.make_params(n_max=n_max, e_max=4 * n_max + 16, m_max=m_max,
                                    lock_mode=lock_mode, key_mode=key_mode, **kw),
                    torch.from_numpy(units).cuda())
    o = oracle.Oracle(oracle.Params(n_max=n_max, e_max=4 * n_max + 16, m_max=m_max,
                                    lock_mode=lock_mode, key_mode=key_mode, **kw),
                      units, threads=oracle_threads())
    return g, o


SCHEDULES = [
    dict(m_cap=512, insert_every=50, qe_window=1024, max_signals=40_000, qe_threshold=0.003,
         seed=7),
    dict(m_cap=64, insert_every=37, qe_window=100, max_signals=6_000, qe_threshold=0.0, seed=11),
    dict(m_cap=512, fixed_m=1, insert_every=20, qe_window=500, max_signals=1_500,
         qe_threshold=0.0, seed=3),
]


@pytest.mark.parametrize("lock_mode,key_mode", [(0, 0), (1, 1), (1, 0)])
@pytest.mark.parametrize("k", range(len(SCHEDULES)))
def test_schedule_matches_the_oracle(k, lock_mode, key_mode):
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    cloud = torus(20_000, 1)
    g, o = pair(cloud, 600, 512, lock_mode, key_mode)
    sch = SCHEDULES[k]
    g.stat(gsn.GSN_STAT_CLEAR)
    got = g.run_schedule(torch.from_numpy(cloud).cuda(), gsn.make_schedule(**sch))
    want = o.run_schedule(cloud, oracle.Schedule(**sch))
    assert got == want
    assert g.stat(gsn.GSN_STAT_ACCEPTED) == got["accepted"]
    assert g.stat(gsn.GSN_STAT_RESOLVED) == got["signals"]
    gs, os_ = g.export(), o.export()
    for f in ("xyz", "err", "edges"):
        np.testing.assert_array_equal(gs[f].numpy(), os_[f], err_msg=f)
    assert g.check() == 0


def test_growth_to_two_thousand_units_with_pruning():
    """A longer run: N grows from 2 to the capacity 2,000, edges age out (max_age 8) and
    orphaned units are removed, m follows the power-of-two rule up to 2,048."""
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    cloud = torus(200_000, 2)
    g, o = pair(cloud, 2_000, 2_048, 0, 0, max_age=8)
    sch = dict(m_cap=2_048, insert_every=60, qe_window=4_096, max_signals=150_000,
               qe_threshold=0.0, seed=5)
    got = g.run_schedule(torch.from_numpy(cloud).cuda(), gsn.make_schedule(**sch))
    want = o.run_schedule(cloud, oracle.Schedule(**sch))
    assert got == want
    assert got["n_units"] > 1_500
    gs, os_ = g.export(), o.export()
    for f in ("xyz", "err", "edges"):
        np.testing.assert_array_equal(gs[f].numpy(), os_[f], err_msg=f)


def test_schedule_arguments_are_checked():
    import torch
    from paper_1503_08294_amd import gsn
    cloud = torus(1_000, 3)
    g, _ = pair(cloud, 100, 64, 0, 0)
    dc = torch.from_numpy(cloud).cuda()
    for bad in (dict(m_cap=0), dict(m_cap=65), dict(qe_window=0), dict(max_signals=0),
                dict(insert_every=-1), dict(fixed_m=-1), dict(fixed_m=65)):
        kw = dict(m_cap=64, insert_every=10, qe_window=64, max_signals=100, seed=0)
        kw.update(bad)
        with pytest.raises(gsn.GsnError) as e:
            g.run_schedule(dc, gsn.make_schedule(**kw))
        assert e.value.code == gsn.GSN_E_INVAL
    sig = dc[:, :8].contiguous()
    g.find_winners(sig)
    with pytest.raises(gsn.GsnError) as e:        # not between iterations
        g.run_schedule(dc, gsn.make_schedule(m_cap=64, max_signals=10))
    assert e.value.code == gsn.GSN_E_STATE


def imported_pair(units, err, edges, n_max, m_max, lock_mode=0):
    """A GPU network and an oracle network holding the same units, errors and edges."""
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    kw = dict(eps_b=0.05, eps_n=0.0006, max_age=50, err_alpha=0.5, err_beta=0.995)
    e_max = edges.shape[1] + 2 * n_max + 16
    g = gsn.Network(gsn.make_params(n_max=n_max, e_max=e_max, m_max=m_max,
                                    lock_mode=lock_mode, **kw), torch.from_numpy(units).cuda())
    o = oracle.Oracle(oracle.Params(n_max=n_max, e_max=e_max, m_max=m_max,
                                    lock_mode=lock_mode, **kw), units,
                      threads=oracle_threads())
    g.import_state(torch.from_numpy(units), torch.from_numpy(err), torch.from_numpy(edges))
    o.import_state(units, err, edges)
    return g, o


def graph(n, rng, hub=None, hub_degree=0):
    """A ring through all units plus chords (degrees about 4), and optionally one hub
    joined to hub_degree other units; (u, v, age) with u < v, sorted."""
    pairs = set()
    for i in range(n):
        pairs.add((min(i, (i + 1) % n), max(i, (i + 1) % n)))
    for u, v in rng.integers(0, n, (n, 2)):
        if u != v:
            pairs.add((min(u, v), max(u, v)))
    if hub is not None:
        for v in rng.choice(np.delete(np.arange(n), hub), hub_degree, replace=False):
            pairs.add((min(hub, v), max(hub, v)))
    pairs = sorted(pairs)
    ages = rng.integers(0, 10, len(pairs))
    return np.array([[p[0] for p in pairs], [p[1] for p in pairs], ages], np.int32)


@pytest.mark.parametrize("case", ["dominant", "equal", "hub", "random", "capacity"])
def test_hundreds_of_insertions_in_one_call(case):
    """One iteration of 600 signals and then 600 insertions (insert_every 1) in one call,
    from imported errors that stress the order of the insertions: one error far above the
    rest (q is taken again and again, and so are the new units), all errors equal (the
    index decides every tie), a hub of 100 neighbours with the largest error (its row is
    too long to be held, and takes the one-wave insertion), plain random errors (several
    selection rounds), and a unit capacity reached in the middle of the call."""
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng({"dominant": 1, "equal": 2, "hub": 3, "random": 4,
                                 "capacity": 5}[case])
    cloud = torus(20_000, 9)
    n = 3_000
    units = np.ascontiguousarray(cloud[:, :n])
    err = rng.uniform(0.0, 1.0, n).astype(np.float32)
    hub = None
    if case == "dominant":
        err[17] = 1e6
    elif case == "equal":
        err[:] = 1.0
    elif case == "hub":
        hub = 1234
        err[hub] = 1e3
    edges = graph(n, rng, hub, 100)
    n_max = n + (250 if case == "capacity" else 700)
    g, o = imported_pair(units, err, edges, n_max, 600)
    sch = dict(m_cap=600, fixed_m=600, insert_every=1, qe_window=100_000,
               max_signals=600, qe_threshold=0.0, seed=13)
    got = g.run_schedule(torch.from_numpy(cloud).cuda(), gsn.make_schedule(**sch))
    want = o.run_schedule(cloud, oracle.Schedule(**sch))
    assert got == want
    assert got["inserted"] == (250 if case == "capacity" else 600)
    gs, os_ = g.export(), o.export()
    for f in ("xyz", "err", "edges"):
        np.testing.assert_array_equal(gs[f].numpy(), os_[f], err_msg=f)
    assert g.check() == 0
