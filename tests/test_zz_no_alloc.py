"""gsn_find_winners_grid_noalloc (the indexed find winners on the library's fixed scratch
array, for callers that cannot allocate) against gsn_find_winners_grid with a caller
workspace, and against the oracle's indexed search (Sec. 3.1, "Indexed"), bit for bit: two
calls in a row, the second on a smaller input, in both the paper's approximate mode and the
certified exact mode; a grid too large for the array is rejected on the host."""
import numpy as np
import pytest

from parity import oracle_threads

pytestmark = pytest.mark.gpu


def make(n, m_max, seed):
    import torch
    import oracle
    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import torus_cloud
    cloud = torus_cloud(max(4 * n, 20_000), seed, 1.0, 0.3, 0.005)
    rng = np.random.default_rng(seed + 100)
    units = np.ascontiguousarray(cloud[rng.choice(cloud.shape[0], n, replace=False)].T)
    g = gsn.Network(gsn.make_params(n_max=n, e_max=4 * n, m_max=m_max),
                    torch.from_numpy(units).cuda())
    o = oracle.Oracle(oracle.Params(n_max=n, e_max=4 * n, m_max=m_max), units,
                      threads=oracle_threads())
    return cloud, g, o


def grid_for(cloud, h):
    lo = cloud.min(axis=0) - np.float32(1e-3)
    hi = cloud.max(axis=0) + np.float32(1e-3)
    dims = [int(np.ceil((hi[a] - lo[a]) / h)) for a in range(3)]
    return [float(v) for v in lo], dims


@pytest.mark.parametrize("exact", [False, True])
def test_noalloc_equals_the_workspace_call(exact):
    import torch
    from paper_1503_08294_amd import gsn
    cases = [(20_000, 4_096, 0.05, 0), (5_000, 700, 0.09, 1)]   # second: a smaller input
    for n, m, h, seed in cases:
        cloud, g, o = make(n, m, seed)
        lo, dims = grid_for(cloud, h)
        grid = gsn.make_grid(lo, h, dims, exact=exact)
        assert gsn.gsn_grid_workspace_bytes(grid, n, m) <= gsn.GSN_NOALLOC_SCRATCH_BYTES
        rng = np.random.default_rng(seed + 7)
        sig_h = np.ascontiguousarray(cloud[rng.integers(0, cloud.shape[0], m)].T)
        sig = torch.from_numpy(sig_h).cuda()
        ws = g.grid_workspace(grid)
        want = [t.clone() for t in g.find_winners_grid(sig, grid, ws)]
        got = [t.clone() for t in g.find_winners_grid_noalloc(sig, grid)]
        torch.cuda.synchronize()
        for a, b, nm in zip(got, want, ("winner", "second", "d1", "d2")):
            assert torch.equal(a, b), f"n={n} m={m} exact={exact}: {nm}"
        if exact:
            ref = o.find_winners(sig_h)
        else:
            ref = o.find_winners_grid(sig_h, lo, h, dims)[:4]
        for a, b, nm in zip(got, ref, ("winner", "second", "d1", "d2")):
            np.testing.assert_array_equal(a.cpu().numpy(), b, err_msg=f"oracle {nm}")
        assert g.check() == 0
        g.close()


def test_noalloc_rejects_a_grid_beyond_the_array():
    import torch
    from paper_1503_08294_amd import gsn
    cloud, g, _ = make(2_000, 256, 3)
    grid = gsn.make_grid([-2.0, -2.0, -2.0], 4.0 / 256, [256, 256, 256])
    assert gsn.gsn_grid_workspace_bytes(grid, 2_000, 256) > gsn.GSN_NOALLOC_SCRATCH_BYTES
    sig = torch.from_numpy(np.ascontiguousarray(cloud[:256].T)).cuda()
    with pytest.raises(gsn.GsnError) as e:
        g.find_winners_grid_noalloc(sig, grid)
    assert e.value.code == gsn.GSN_E_CAPACITY
    # nothing was enqueued and the handle is still usable
    lo, dims = grid_for(cloud, 0.2)
    small = gsn.make_grid(lo, 0.2, dims)
    w, s, _, _ = g.find_winners_grid_noalloc(sig, small)
    assert bool((w != s).all().item())
    assert g.check() == 0
