"""GPU parity of the indexed find winners (the paper's hash index of Sec. 3.1 applied to every
signal: the signal's cube and its 26 neighbours, the exhaustive search when they hold fewer
than two units) against the oracle's indexed search: winner, second, d1, d2 bit-exact."""
import numpy as np
import pytest

from parity import oracle_threads

pytestmark = pytest.mark.gpu


def setup(units, m_max, n_max=None):
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    n = units.shape[1]
    n_max = n_max or n + 8
    g = gsn.Network(gsn.make_params(n_max=n_max, e_max=4 * n_max, m_max=m_max),
                    torch.from_numpy(np.ascontiguousarray(units)).cuda())
    o = oracle.Oracle(oracle.Params(n_max=n_max, e_max=4 * n_max, m_max=m_max), units,
                      threads=oracle_threads())
    return g, o


def compare(g, o, sig, lo, h, dims, where=""):
    import torch
    from paper_1503_08294_amd import gsn
    grid = gsn.make_grid(lo, h, dims)
    ws = g.grid_workspace(grid)
    got = [t.cpu().numpy() for t in g.find_winners_grid(torch.from_numpy(sig).cuda(), grid, ws)]
    want = o.find_winners_grid(sig, lo, h, dims)
    for a, b, nm in zip(got, want[:4], ("winner", "second", "d1", "d2")):
        np.testing.assert_array_equal(a, b, err_msg=f"{where} {nm}")
    return want[4]


@pytest.mark.parametrize("seed,n,m,h", [(0, 500, 700, 0.3), (1, 3000, 4096, 0.12),
                                        (2, 40, 300, 0.5), (3, 2, 64, 0.25),
                                        (4, 20000, 10000, 0.05)])
def test_random_inputs(seed, n, m, h):
    rng = np.random.default_rng(seed)
    units = rng.uniform(-1, 1, (3, n)).astype(np.float32)
    sig = rng.uniform(-1.2, 1.2, (3, m)).astype(np.float32)   # some outside the box
    g, o = setup(units, m)
    dims = tuple(int(np.ceil(2.0 / h)) for _ in range(3))
    fb = compare(g, o, sig, (-1.0, -1.0, -1.0), h, dims, f"seed {seed}")
    assert 0 <= fb <= m


def test_every_signal_falling_back():
    rng = np.random.default_rng(5)
    units = rng.uniform(-1, 1, (3, 300)).astype(np.float32)
    sig = rng.uniform(-1, 1, (3, 200)).astype(np.float32)
    g, o = setup(units, 200)
    # cubes so small that the 27 around a signal hold at most one unit
    fb = compare(g, o, sig, (-1.0, -1.0, -1.0), 0.001, (2000, 2000, 2))
    assert fb > 150


def test_one_cube_is_the_exhaustive_search():
    import torch
    rng = np.random.default_rng(6)
    units = rng.standard_normal((3, 5000)).astype(np.float32)
    sig = rng.standard_normal((3, 3000)).astype(np.float32)
    g, o = setup(units, 3000)
    compare(g, o, sig, (-10.0, -10.0, -10.0), 20.0, (1, 1, 1))
    ex = [t.cpu().numpy() for t in g.find_winners(torch.from_numpy(sig).cuda())]
    want = o.find_winners(sig)
    for a, b in zip(ex, want):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("name,h", [("tiny_sphere", 0.1), ("torus_grow", 0.02),
                                    ("genus3_200k", 0.01), ("genus3_200k", 0.02)])
def test_workloads(name, h):
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS[name]
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    sig = SignalStream(cloud, wl.signal_seed).next(wl.m)
    g, o = setup(units, wl.m)
    lo = cloud.min(axis=0) - np.float32(1e-3)
    hi = cloud.max(axis=0) + np.float32(1e-3)
    dims = tuple(int(np.ceil((hi[a] - lo[a]) / h)) for a in range(3))
    compare(g, o, sig, tuple(float(v) for v in lo), h, dims, name)


def test_iterations_with_the_index_match_the_oracle():
    """find (indexed) -> resolve -> adapt -> update edges, both sides, several iterations."""
    import torch
    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS["torus_grow"]
    cloud = wl.make_cloud(50_000)
    units = wl.make_units(cloud, 2_000)
    g, o = setup(units, 1024, n_max=2_100)
    stream = SignalStream(cloud, wl.signal_seed)
    lo, h = (-1.4, -1.4, -0.4), 0.05
    dims = (56, 56, 16)
    grid = gsn.make_grid(lo, h, dims)
    ws = g.grid_workspace(grid)
    for t in range(8):
        sig = stream.next(1024)
        dsig = torch.from_numpy(sig).cuda()
        g.find_winners_grid(dsig, grid, ws)
        g.resolve_conflicts(1024)
        g.adapt(dsig)
        g.update_edges(1024)
        w, s, d1, d2, _ = o.find_winners_grid(sig, lo, h, dims)
        acc = o.resolve_conflicts(w, s, d1)
        o.adapt(sig, w, s, d1, acc)
        o.update_edges(w, s, acc)
        np.testing.assert_array_equal(g.buf.winner[:1024].cpu().numpy(), w)
        np.testing.assert_array_equal(g.buf.accepted[:1024].cpu().numpy(), acc)
    gs, os_ = g.export(), o.export()
    for f in ("xyz", "err", "edges"):
        np.testing.assert_array_equal(gs[f].numpy(), os_[f], err_msg=f)


@pytest.mark.parametrize("lock_mode", [0, 1, 2])
def test_fused_update_after_the_index_matches_the_oracle(lock_mode):
    """find (indexed) -> gsn_update (resolve, adapt and edges fused as in gsn_iterate) in
    each collision rule, with pruning (max_age 2), against the oracle's four steps."""
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS["torus_grow"]
    cloud = wl.make_cloud(50_000)
    units = wl.make_units(cloud, 2_000)
    kw = dict(n_max=2_100, e_max=8_400, m_max=1024, max_age=2, lock_mode=lock_mode)
    g = gsn.Network(gsn.make_params(**kw), torch.from_numpy(np.ascontiguousarray(units)).cuda())
    o = oracle.Oracle(oracle.Params(**kw), units, threads=oracle_threads())
    stream = SignalStream(cloud, wl.signal_seed)
    lo, h = (-1.4, -1.4, -0.4), 0.05
    dims = (56, 56, 16)
    grid = gsn.make_grid(lo, h, dims)
    ws = g.grid_workspace(grid)
    with pytest.raises(gsn.GsnError) as e:          # an update needs a find first
        g.update(torch.zeros((3, 8), dtype=torch.float32, device="cuda"))
    assert e.value.code == gsn.GSN_E_STATE
    for t in range(10):
        sig = stream.next(1024)
        dsig = torch.from_numpy(sig).cuda()
        g.find_winners_grid(dsig, grid, ws)
        got = g.update(dsig).cpu().numpy()
        w, s, d1, d2, _ = o.find_winners_grid(sig, lo, h, dims)
        acc = o.resolve_conflicts(w, s, d1)
        o.adapt(sig, w, s, d1, acc)
        o.update_edges(w, s, acc)
        np.testing.assert_array_equal(g.buf.winner[:1024].cpu().numpy(), w, err_msg=f"{t}")
        np.testing.assert_array_equal(got, acc, err_msg=f"iteration {t}")
        gs, os_ = g.export(), o.export()
        for f in ("xyz", "err", "edges"):
            np.testing.assert_array_equal(gs[f].numpy(), os_[f], err_msg=f"{t} {f}")
    assert g.check() == 0


def test_grid_arguments_are_checked():
    import torch
    from paper_1503_08294_amd import gsn
    units = np.random.default_rng(7).standard_normal((3, 50)).astype(np.float32)
    g, _ = setup(units, 16)
    sig = torch.zeros((3, 16), dtype=torch.float32, device="cuda")
    good = gsn.make_grid((0, 0, 0), 0.5, (4, 4, 4))
    ws = g.grid_workspace(good)
    for bad in (gsn.make_grid((0, 0, 0), 0.0, (4, 4, 4)), gsn.make_grid((0, 0, 0), -1.0, (4, 4, 4)),
                gsn.make_grid((0, 0, 0), 0.5, (0, 4, 4)),
                gsn.make_grid((0, 0, 0), 0.5, (4096, 4096, 2)),
                gsn.make_grid((float("nan"), 0, 0), 0.5, (4, 4, 4))):
        assert gsn.gsn_grid_workspace_bytes(bad, 58, 16) == 0
        with pytest.raises(gsn.GsnError) as e:
            g.find_winners_grid(sig, bad, ws)
        assert e.value.code == gsn.GSN_E_INVAL
    big = gsn.make_grid((0, 0, 0), 0.01, (400, 400, 4))
    with pytest.raises(gsn.GsnError) as e:        # workspace sized for the small grid
        g.find_winners_grid(sig, big, ws)
    assert e.value.code == gsn.GSN_E_CAPACITY


# ------------------------------------------------------------------ exact mode ----
# With exact = 1 the 27-cube result is kept only where it is certified; the outputs must
# equal the exhaustive search's (the oracle's find_winners) bit for bit.

def compare_exact(g, o, sig, lo, h, dims, where=""):
    import torch
    from paper_1503_08294_amd import gsn
    grid = gsn.make_grid(lo, h, dims, exact=True)
    ws = g.grid_workspace(grid)
    got = [t.cpu().numpy() for t in g.find_winners_grid(torch.from_numpy(sig).cuda(), grid, ws)]
    want = o.find_winners(sig)
    for a, b, nm in zip(got, want, ("winner", "second", "d1", "d2")):
        np.testing.assert_array_equal(a, b, err_msg=f"{where} {nm}")


@pytest.mark.parametrize("seed,n,m,h", [(10, 500, 700, 0.3), (11, 3000, 4096, 0.12),
                                        (12, 40, 300, 0.5), (13, 2, 64, 0.25),
                                        (14, 20000, 10000, 0.05), (15, 20000, 4000, 0.01),
                                        (16, 5000, 3000, 0.2)])
def test_exact_mode_random_inputs(seed, n, m, h):
    rng = np.random.default_rng(seed)
    units = rng.uniform(-1, 1, (3, n)).astype(np.float32)
    sig = rng.uniform(-1.3, 1.3, (3, m)).astype(np.float32)   # some outside the box
    g, o = setup(units, m)
    dims = tuple(int(np.ceil(2.0 / h)) for _ in range(3))
    compare_exact(g, o, sig, (-1.0, -1.0, -1.0), h, dims, f"seed {seed}")


def test_exact_mode_on_cube_faces():
    """Units and signals on and next to cube faces, on a lattice: distances tie often, and
    the nearest outside unit sits right behind the block's faces."""
    rng = np.random.default_rng(17)
    h = 0.125
    ax = np.arange(-1.0, 1.0001, h / 2, dtype=np.float32)
    grid_pts = np.stack(np.meshgrid(ax, ax, ax[:5], indexing="ij")).reshape(3, -1)
    units = grid_pts[:, rng.choice(grid_pts.shape[1], 3000, replace=False)].astype(np.float32)
    jitter = rng.choice(np.array([0.0, 1e-6, -1e-6, h / 4], np.float32), size=(3, 2000))
    sig = (grid_pts[:, rng.choice(grid_pts.shape[1], 2000)] + jitter).astype(np.float32)
    g, o = setup(units, 2000)
    compare_exact(g, o, sig, (-1.0, -1.0, -1.0), h, (16, 16, 3), "lattice")


@pytest.mark.parametrize("h", [0.005, 0.01, 0.02])
def test_exact_mode_genus3(h):
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS["genus3_200k"]
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    sig = SignalStream(cloud, wl.signal_seed).next(wl.m)
    g, o = setup(units, wl.m)
    lo = cloud.min(axis=0) - np.float32(1e-3)
    hi = cloud.max(axis=0) + np.float32(1e-3)
    dims = tuple(int(np.ceil((hi[a] - lo[a]) / h)) for a in range(3))
    compare_exact(g, o, sig, tuple(float(v) for v in lo), h, dims, f"genus3 h={h}")
