"""gsn_iterate_loop: count iterations recorded into a HIP graph once and replayed.  Every
call leaves the state of count gsn_iterate calls (bit-exact against the oracle stepping
the same batches) and the outputs of the last one, whether the call records a new graph or
replays a cached one; eager calls between the loop calls change the handle's internal
buffer parities, so later calls need other graphs; batch contents change between replays
(the graph reads them when it runs)."""
import numpy as np
import pytest

from parity import Pair, assert_iter_equal

pytestmark = pytest.mark.gpu


def run_loop_case(m, lock, counts, rebucket, seed, n=6_000):
    import torch
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    pair = Pair(units, m_max=m, lock_mode=lock)
    net = pair.net
    if rebucket:
        net.tune(gsn.GSN_TUNE_REBUCKET, rebucket)
    bufs = {}
    for call, count in enumerate(counts):
        sigs = rng.standard_normal((count, 3, m)).astype(np.float32)
        if count not in bufs:
            bufs[count] = torch.empty((count, 3, m), dtype=torch.float32, device="cuda")
        dev = bufs[count]
        dev.copy_(pair.to_dev(sigs))          # same address, new contents
        g = [t.cpu().numpy() for t in net.iterate_loop(dev)]
        for k in range(count):
            o = pair.orc.iterate(sigs[k], 0, 0, False)
        where = f"m={m} lock={lock} call {call} count {count}"
        assert_iter_equal(g, o, where + " (last iteration)")
        pair.compare_state(where)
        if call % 2 == 1:
            # an eager iteration in between: the buffer parities change
            extra = rng.standard_normal((3, m)).astype(np.float32)
            g, o = pair.iterate(extra)
            assert_iter_equal(g, o, where + " eager")
    assert net.check() == 0
    torch.cuda.synchronize()
    return net.stat(gsn.GSN_STAT_LOOP_RECORDS)


@pytest.mark.parametrize("m,lock,counts,rebucket,replays", [
    (2_000, 0, [4, 4, 4, 4, 3, 3, 3], 0, True),   # staged find, lock set; odd counts
    (2_000, 0, [4, 4, 4, 4], 3, True),            # unit order rebuilt at every call's start
    (2_000, 0, [1, 2, 3, 4, 5, 1, 2], 0, False),  # more graphs than the cache holds
    (100, 0, [5, 5, 5, 2], 0, True),              # unit-parallel small-batch find
    (2_000, 1, [4, 4, 3, 3], 0, False),           # winner lock (the paper's rule)
    (2_000, 2, [2, 2, 2], 0, False),              # greedy re-admission
])
def test_loop_matches_the_oracle(m, lock, counts, rebucket, replays):
    records = run_loop_case(m, lock, counts, rebucket, seed=2000 + m + 10 * lock + rebucket)
    assert 1 <= records <= len(counts)
    if replays:
        assert records < len(counts)       # some calls replayed a recorded graph


def test_loop_argument_errors():
    from paper_1503_08294_amd import gsn
    import torch
    rng = np.random.default_rng(7)
    pair = Pair(rng.standard_normal((3, 500)).astype(np.float32), m_max=64)
    b = pair.net.buf
    sigs = torch.zeros((2, 3, 64), dtype=torch.float32, device="cuda")
    import ctypes
    ptrs = [ctypes.c_void_p(t.data_ptr()) for t in (sigs, b.winner, b.second, b.d1, b.d2,
                                                      b.accepted)]
    for count in (0, -1, gsn.GSN_MAX_LOOP + 1):
        # the C call itself (the binding would refuse the tensor size first)
        rc = gsn._lib.gsn_iterate_loop(pair.net.h, ptrs[0], 64, count, *ptrs[1:],
                                       ctypes.c_void_p(0))
        assert rc == gsn.GSN_E_INVAL, count
    # more signals than m_max
    assert gsn._lib.gsn_iterate_loop(pair.net.h, ptrs[0], 65, 1, *ptrs[1:],
                                     ctypes.c_void_p(0)) == gsn.GSN_E_INVAL
    # nothing ran: the state is still the initial one
    pair.compare_state("after rejected loop calls")


@pytest.mark.timeout(600)
def test_loop_genus3_against_the_oracle():
    """The genus-3 workload (200,000 units, 16,384 signals) for 40 iterations through four
    gsn_iterate_loop calls of 10 (the first records, the second records the state after
    10 iterations with the unit order rebuilt or not, later ones replay), every call's
    last outputs and the state after it compared with the oracle."""
    import torch
    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS["genus3_200k"]
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    cap = wl.capacity()
    pair = Pair(units, n_max=cap["n_max"], e_max=cap["e_max"], m_max=wl.m, eps_b=wl.eps_b,
                eps_n=wl.eps_n, max_age=wl.max_age, err_alpha=wl.err_alpha,
                err_beta=wl.err_beta)
    stream = SignalStream(cloud, wl.signal_seed)
    count = 10
    buf = torch.empty((count, 3, wl.m), dtype=torch.float32, device="cuda")
    for call in range(4):
        sigs = np.stack([stream.next(wl.m) for _ in range(count)])
        buf.copy_(pair.to_dev(sigs))
        g = [t.cpu().numpy() for t in pair.net.iterate_loop(buf)]
        for k in range(count):
            o = pair.orc.iterate(sigs[k], 0, 0, False)
        assert_iter_equal(g, o, f"genus3 loop call {call}")
        pair.compare_state(f"genus3 after loop call {call}")
    assert pair.net.check() == 0
    assert pair.net.stat(gsn.GSN_STAT_LOOP_RECORDS) < 4


def test_loop_of_empty_batches_decays_the_errors():
    """Iterations without signals still apply the error decay (and age nothing): a loop of
    empty batches, recorded and replayed, against the oracle."""
    import torch
    rng = np.random.default_rng(11)
    pair = Pair(rng.standard_normal((3, 3_000)).astype(np.float32), m_max=500)
    for _ in range(3):
        g, o = pair.iterate(rng.standard_normal((3, 500)).astype(np.float32))
        assert_iter_equal(g, o, "warm-up")
    empty = torch.zeros((4, 3, 0), dtype=torch.float32, device="cuda")
    for call in range(3):
        pair.net.iterate_loop(empty)
        for _ in range(4):
            pair.orc.iterate(np.zeros((3, 0), np.float32), 0, 0, False)
        pair.compare_state(f"empty loop call {call}")
    assert pair.net.check() == 0
