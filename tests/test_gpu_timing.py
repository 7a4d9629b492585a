"""Measurement hooks: the timers record one event pair per timed launch, give positive
durations, and change no result, for every find-winners variant."""
import numpy as np
import pytest

from parity import Pair, assert_find_equal

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("variant,m", [(4, 1_500), (5, 1_500), (6, 100), (3, 1_500), (2, 1_500),
                                       (1, 300)])
def test_scan_timer_counts_launches_and_changes_nothing(variant, m):
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(variant)
    units = rng.standard_normal((3, 20_000)).astype(np.float32)
    sig = rng.standard_normal((3, m)).astype(np.float32)
    pair = Pair(units, m_max=m)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, variant)
    o = pair.orc.find_winners(sig)
    h = pair.net.h
    for w in range(gsn.GSN_T_COUNT):
        gsn.gsn_timing_read(h, w)
    gsn.gsn_timing_select(h, (1 << gsn.GSN_T_FIND_SCAN) | (1 << gsn.GSN_T_FIND))
    gsn.gsn_timing_enable(h, True)
    calls = 4
    for _ in range(calls):
        g = [t.cpu().numpy() for t in pair.net.find_winners(pair.to_dev(sig))]
        assert_find_equal(g, o, f"variant {variant} timed")
    gsn.gsn_timing_enable(h, False)
    scan_ms, scan_n = gsn.gsn_timing_read(h, gsn.GSN_T_FIND_SCAN)
    find_ms, find_n = gsn.gsn_timing_read(h, gsn.GSN_T_FIND)
    assert scan_n == calls and find_n == calls
    assert 0.0 < scan_ms <= find_ms
    # nothing left to read, and timers off record nothing
    assert gsn.gsn_timing_read(h, gsn.GSN_T_FIND_SCAN) == (0.0, 0)
    pair.net.find_winners(pair.to_dev(sig))
    assert gsn.gsn_timing_read(h, gsn.GSN_T_FIND_SCAN) == (0.0, 0)
