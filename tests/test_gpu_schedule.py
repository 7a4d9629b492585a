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
