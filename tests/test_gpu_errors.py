"""Error handling through the C ABI on the GPU: call order, capacities, invalid indices,
degenerate sizes.  Every kernel still exits normally; errors are host return codes or the
sticky device status."""
import numpy as np
import pytest

from parity import Pair

pytestmark = pytest.mark.gpu


def small_pair(n=20, m_max=16, **kw):
    rng = np.random.default_rng(0)
    return Pair(rng.standard_normal((3, n)).astype(np.float32), m_max=m_max, **kw), rng


def test_call_order_is_enforced():
    from paper_1503_08294_amd import gsn
    pair, rng = small_pair()
    sig = pair.to_dev(rng.standard_normal((3, 8)).astype(np.float32))
    with pytest.raises(gsn.GsnError) as e:
        pair.net.adapt(sig)
    assert e.value.code == gsn.GSN_E_STATE
    pair.net.find_winners(sig)
    with pytest.raises(gsn.GsnError) as e:
        pair.net.update_edges(8)
    assert e.value.code == gsn.GSN_E_STATE
    pair.net.resolve_conflicts(8)
    pair.net.resolve_conflicts(8)        # repeatable
    pair.net.adapt(sig)
    with pytest.raises(gsn.GsnError):
        pair.net.grow(1, 1)              # grow only between iterations
    pair.net.update_edges(8)
    pair.net.grow(1, 0)
    assert pair.net.check() == 0


def test_signal_capacity_and_empty_batch():
    from paper_1503_08294_amd import gsn
    import torch
    pair, rng = small_pair(m_max=16)
    sig = pair.to_dev(rng.standard_normal((3, 17)).astype(np.float32))
    out = [torch.empty(17, dtype=dt, device="cuda")
           for dt in (torch.int32, torch.int32, torch.float32, torch.float32)]
    with pytest.raises(gsn.GsnError) as e:         # m = 17 > m_max = 16: rejected by the library
        gsn.gsn_find_winners(pair.net.h, sig, 17, *out)
    assert e.value.code == gsn.GSN_E_INVAL
    empty = pair.to_dev(np.zeros((3, 0), np.float32))
    pair.net.iterate(empty)
    assert pair.net.check() == 0


def test_fewer_than_two_units():
    from paper_1503_08294_amd import gsn
    pair = Pair(np.zeros((3, 1), np.float32), n_max=4, m_max=4)
    with pytest.raises(gsn.GsnError) as e:
        pair.net.find_winners(pair.to_dev(np.zeros((3, 2), np.float32)))
    assert e.value.code == gsn.GSN_E_INVAL


def test_invalid_injected_winner_sets_sticky_status():
    import torch
    from paper_1503_08294_amd import gsn
    pair, rng = small_pair()
    sig = pair.to_dev(rng.standard_normal((3, 4)).astype(np.float32))
    pair.net.find_winners(sig)
    w = torch.tensor([0, 99, 2, 3], dtype=torch.int32, device="cuda")
    s = torch.tensor([1, 1, 2, 4], dtype=torch.int32, device="cuda")
    d1 = torch.zeros(4, dtype=torch.float32, device="cuda")
    acc = pair.net.resolve_conflicts(4, w, s, d1)
    assert acc.cpu().tolist() == [1, 0, 0, 1]   # out-of-range and b == s rejected
    assert pair.net.check() == gsn.GSN_E_INVAL


def test_edge_capacity_overflow_is_reported():
    from paper_1503_08294_amd import gsn
    pair, rng = small_pair(n=200, m_max=64, e_max=3)
    sig = pair.to_dev(rng.standard_normal((3, 64)).astype(np.float32))
    pair.net.iterate(sig)
    assert pair.net.check() == gsn.GSN_E_CAPACITY


def test_import_export_round_trip():
    pair, rng = small_pair(n=30, m_max=16)
    import torch
    xyz = torch.from_numpy(rng.standard_normal((3, 25)).astype(np.float32))
    err = torch.from_numpy(rng.random(25).astype(np.float32))
    edges = torch.tensor([[3, 0, 7], [1, 5, 2], [4, 0, 9]], dtype=torch.int32)
    pair.net.import_state(xyz, err, edges)
    st = pair.net.export()
    assert torch.equal(st["xyz"], xyz) and torch.equal(st["err"], err)
    assert st["edges"].tolist() == [[0, 1, 2], [5, 3, 7], [0, 4, 9]]
    pair.orc.import_state(xyz.numpy(), err.numpy(), edges.numpy())
    for t in range(1, 6):
        sig = rng.standard_normal((3, 16)).astype(np.float32)
        pair.iterate(sig)
        pair.compare_state(f"after import, iteration {t}")
