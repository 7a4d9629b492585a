"""GPU parity of whole iterations (find -> resolve -> adapt -> update_edges, plus grow
where the workload grows) against the oracle on the seeded synthetic workloads: every
iteration's winner, second, d1, d2 and acceptance bit-exact; edge lists bit-exact and
positions within 1e-6 after the iterations stated."""
import numpy as np
import pytest

from parity import run_workload

pytestmark = pytest.mark.gpu


def test_tiny_sphere_20_iterations():
    pair, _ = run_workload("tiny_sphere")
    n, e = pair.net.sizes()
    assert n == 1000 and e > 0


def test_torus_grow_100_iterations():
    pair, _ = run_workload("torus_grow")
    n, _ = pair.net.sizes()
    assert n > 10_000          # insertions happened


def test_pruning_removal_and_insertion():
    """A dense small network with max_age 2: edges are pruned, units are orphaned and
    removed, and a unit is inserted every 10 iterations."""
    pair, _ = run_workload("torus_grow", iterations=60, n_points=50_000, n_units=1_500, m=1_024,
                           max_age=2)
    # the same state was reached; check that removal and insertion actually occurred
    n, _ = pair.net.sizes()
    assert n != 1_500


def test_spheres_plane_200_iterations():
    pair, _ = run_workload("spheres_plane_prune", compare_every=25)
    assert pair.net.sizes()[0] != 50_000


@pytest.mark.timeout(600)
def test_genus3_100_iterations():
    """The genus-3 workload at its stated length: 100 iterations of N = 200,000 units and
    m = 16,384 signals; every iteration's outputs and the state every 10 iterations equal
    the oracle's bit for bit."""
    pair, _ = run_workload("genus3_200k", compare_every=10)
    n, e = pair.net.sizes()
    assert n == 200_000 and e > 200_000


@pytest.mark.timeout(600)
def test_genus3_separate_calls_against_the_oracle():
    """The four separate calls (find, resolve, adapt, update_edges), not gsn_iterate, on the
    genus-3 workload against the oracle directly."""
    run_workload("genus3_200k", iterations=30, compare_every=10, calls="steps")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("m", [1, 64, 1_024, 16_384, 65_536])
def test_torus_sweep_stated_length(m):
    """The sweep workload at every m at its stated length (10 warm-up iterations + 50):
    N = 100,000 units on the noisy torus."""
    _, rate = run_workload("torus_sweep", iterations=60, m=m, compare_every=10)
    assert 0.0 <= rate < 1.0
    if m == 1:
        assert rate == 0.0


@pytest.mark.parametrize("name,iters", [("tiny_sphere", 20), ("torus_grow", 100)])
def test_separate_calls_against_the_oracle(name, iters):
    run_workload(name, iterations=iters, calls="steps")


@pytest.mark.parametrize("lock_mode", [0, 1, 2])
def test_checkpoint_resume_equals_an_uninterrupted_run(lock_mode):
    """50 iterations, gsn_export, a new handle, gsn_import, 50 more iterations: the state
    equals that of 100 iterations straight, bit for bit, on the GPU and on the oracle (the
    growing torus workload, so insertion and removal run on both sides of the cut)."""
    import torch
    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    from parity import Pair, params_pair, oracle_threads
    import oracle

    wl = WORKLOADS["torus_grow"]
    cloud = wl.make_cloud(100_000)
    units = wl.make_units(cloud, 3_000)
    m, cut, total = 1_024, 50, 100
    kw = dict(eps_b=wl.eps_b, eps_n=wl.eps_n, max_age=4, err_alpha=wl.err_alpha,
              err_beta=wl.err_beta, lock_mode=lock_mode)
    n_max, e_max = 3_400, 16_000
    straight = Pair(units, n_max=n_max, e_max=e_max, m_max=m, **kw)
    first = Pair(units, n_max=n_max, e_max=e_max, m_max=m, **kw)
    batches = []
    stream = SignalStream(cloud, wl.signal_seed)
    for _ in range(total):
        batches.append(stream.next(m))
    for t in range(1, total + 1):
        straight.iterate(batches[t - 1], t, wl.insert_every, True)
    for t in range(1, cut + 1):
        first.iterate(batches[t - 1], t, wl.insert_every, True)
    gs, os_ = first.net.export(), first.orc.export()
    del first
    gp, op = params_pair(n_max, e_max, m, **kw)
    resumed = gsn.Network(gp, torch.from_numpy(units).cuda())
    resumed.import_state(gs["xyz"], gs["err"], gs["edges"])
    orc = oracle.Oracle(op, units, threads=oracle_threads())
    orc.import_state(os_["xyz"], os_["err"], os_["edges"])
    for t in range(cut + 1, total + 1):
        sig = torch.from_numpy(batches[t - 1]).cuda()
        resumed.iterate(sig)
        resumed.grow(t, wl.insert_every)
        orc.iterate(batches[t - 1], t, wl.insert_every, True)
    a, b = straight.net.export(), resumed.export()
    oa, ob = straight.orc.export(), orc.export()
    for k in ("xyz", "err", "edges"):
        assert torch.equal(a[k], b[k]), f"GPU {k}"
        np.testing.assert_array_equal(oa[k], ob[k], err_msg=f"oracle {k}")
        np.testing.assert_array_equal(a[k].numpy(), oa[k], err_msg=f"GPU vs oracle {k}")
    assert straight.net.sizes()[0] != 3_000        # units were inserted or removed
    assert resumed.check() == 0


def test_determinism_of_repeated_runs():
    a, _ = run_workload("torus_grow", iterations=15)
    b, _ = run_workload("torus_grow", iterations=15)
    sa, sb = a.net.export(), b.net.export()
    for k in ("xyz", "err", "edges"):
        assert np.array_equal(sa[k].numpy(), sb[k].numpy()), k


@pytest.mark.parametrize("lock_mode", [0, 1, 2])
def test_fused_iteration_equals_the_four_calls(lock_mode):
    """gsn_iterate (fused update for the lock-set rule) against find, resolve, adapt and
    update_edges called one by one, on two networks from the same state: every output and
    the whole state bit for bit, with pruning, removal and insertion."""
    import torch
    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS["torus_grow"]
    cloud = wl.make_cloud(50_000)
    units = torch.from_numpy(wl.make_units(cloud, 1_500)).cuda()
    p = gsn.make_params(wl.eps_b, wl.eps_n, 2, wl.err_alpha, wl.err_beta, 1_700, 8_000, 1_024,
                        lock_mode, 0)
    a, b = gsn.Network(p, units), gsn.Network(p, units)
    a.stat(gsn.GSN_STAT_CLEAR)
    b.stat(gsn.GSN_STAT_CLEAR)
    stream = SignalStream(cloud, wl.signal_seed)
    accepted = 0
    for t in range(1, 41):
        sig = torch.from_numpy(stream.next(1_024)).cuda()
        ra = [x.clone() for x in a.iterate(sig)]
        rb = [x.clone() for x in b.iterate_steps(sig)]
        for x, y in zip(ra, rb):
            assert torch.equal(x, y), f"iteration {t}"
        accepted += int(ra[4].sum().item())
        a.grow(t, 10)
        b.grow(t, 10)
    # the statistics count every resolved and accepted signal on both paths
    for net in (a, b):
        assert net.stat(gsn.GSN_STAT_RESOLVED) == 40 * 1_024
        assert net.stat(gsn.GSN_STAT_ACCEPTED) == accepted
    sa, sb = a.export(), b.export()
    for k in ("xyz", "err", "edges"):
        assert torch.equal(sa[k], sb[k]), k
    assert a.sizes() == b.sizes() and a.sizes()[0] != 1_500
    assert a.check() == 0 and b.check() == 0


@pytest.mark.parametrize("lock_mode", [0, 1])
def test_network_beyond_the_folded_rewrite(lock_mode):
    """600,000 units: the edge rewrites take more than 2,048 workgroups, so the block
    offsets come from the single-workgroup scan instead of being summed by every writing
    workgroup (the path the smaller workloads never take).  Edges: a path through all units
    plus chords, ages 0-5, max_age 4 so that edges are pruned; signals on top of units, so
    that lock sets collide."""
    import torch
    from parity import Pair, assert_iter_equal
    rng = np.random.default_rng(31)
    n, m = 600_000, 4_096
    units = rng.standard_normal((3, n)).astype(np.float32)
    units /= np.linalg.norm(units, axis=0).astype(np.float32)
    u = np.concatenate([np.arange(n - 1), np.arange(0, n - 7, 3)])
    v = np.concatenate([np.arange(1, n), np.arange(7, n, 3)])
    order = np.lexsort((v, u))
    edges = np.stack([u[order], v[order], rng.integers(0, 6, len(u))]).astype(np.int32)
    pair = Pair(units, e_max=2 * edges.shape[1] + 4 * m, m_max=m, max_age=4,
                lock_mode=lock_mode)
    pair.net.import_state(torch.from_numpy(units), None, torch.from_numpy(edges))
    pair.orc.import_state(units, None, edges)
    for t in range(1, 4):
        pick = rng.integers(0, n, m)
        sig = (units[:, pick] + 1e-3 * rng.standard_normal((3, m))).astype(np.float32)
        g, o = pair.iterate(sig, t, 0, False)
        assert_iter_equal(g, o, f"iteration {t}")
        pair.compare_state(f"iteration {t}")
    assert pair.net.check() == 0
