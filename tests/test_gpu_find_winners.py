"""GPU parity of find-winners against the oracle: winner, second, d1, d2 bit-exact, over
sizes that span several tiles, chunks and a ragged tail, tie-heavy inputs, every split of
the unit range, and the full 200k-unit x 16k-signal genus-3 workload."""
import numpy as np
import pytest

from parity import Pair, assert_find_equal

pytestmark = pytest.mark.gpu

CASES = [(2, 1, 0), (3, 7, 1), (100, 33, 2), (1000, 256, 3), (1537, 1000, 4),
         (4099, 2049, 5), (10_000, 2_048, 6), (50_000, 300, 7), (20_000, 8_192, 8),
         (700, 20_000, 9)]


@pytest.mark.parametrize("n,m,seed", CASES)
def test_random_inputs(n, m, seed):
    rng = np.random.default_rng(seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    sig = rng.standard_normal((3, m)).astype(np.float32)
    pair = Pair(units, m_max=m)
    g, o = pair.find(sig)
    assert_find_equal(g, o, f"n={n} m={m}")


@pytest.mark.parametrize("grid,n,m", [(1, 50, 500), (3, 3000, 4000), (2, 9, 64)])
def test_ties_duplicates_and_signals_on_units(grid, n, m):
    rng = np.random.default_rng(grid)
    units = rng.integers(-grid, grid + 1, (3, n)).astype(np.float32)
    sig = rng.integers(-grid, grid + 1, (3, m)).astype(np.float32)
    sig[:, : min(m, n)] = units[:, : min(m, n)]
    pair = Pair(units, m_max=m)
    g, o = pair.find(sig)
    assert_find_equal(g, o, f"grid={grid}")


def test_every_split_gives_the_same_answer():
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(21)
    units = rng.standard_normal((3, 5000)).astype(np.float32)
    units[:, 4000:] = units[:, :1000]                  # exact duplicates across chunks
    sig = rng.standard_normal((3, 3000)).astype(np.float32)
    pair = Pair(units, m_max=3000)
    o = pair.orc.find_winners(sig)
    for split in (1, 2, 3, 7, 16, 64, 0):
        pair.net.tune(gsn.GSN_TUNE_SPLIT, split)
        g = [t.cpu().numpy() for t in pair.net.find_winners(pair.to_dev(sig))]
        assert_find_equal(g, o, f"split={split}")


def test_larger_network_every_split():
    """40,037 units (a ragged last batch) and 2,999 signals (a ragged last signal block):
    chunks of several dozen batches, the XCD order of chunks for splits that are multiples of
    8, exact duplicates in different chunks and signals on top of units."""
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(22)
    n, m = 40037, 2999
    units = rng.standard_normal((3, n)).astype(np.float32)
    units[:, 30000:31000] = units[:, :1000]
    units[:, 20000:20300] = units[:, 20300:20600]
    sig = rng.standard_normal((3, m)).astype(np.float32)
    sig[:, :500] = units[:, 29500:30000]
    pair = Pair(units, m_max=m)
    o = pair.orc.find_winners(sig)
    for split in (16, 24, 40, 56, 64, 0):
        pair.net.tune(gsn.GSN_TUNE_SPLIT, split)
        g = [t.cpu().numpy() for t in pair.net.find_winners(pair.to_dev(sig))]
        assert_find_equal(g, o, f"split={split}")


def test_zero_signals_and_repeat_calls():
    rng = np.random.default_rng(4)
    units = rng.standard_normal((3, 300)).astype(np.float32)
    pair = Pair(units, m_max=64)
    sig = rng.standard_normal((3, 64)).astype(np.float32)
    a = [t.cpu().numpy().copy() for t in pair.net.find_winners(pair.to_dev(sig))]
    pair.net.find_winners(pair.to_dev(np.zeros((3, 0), np.float32)))
    b = [t.cpu().numpy() for t in pair.net.find_winners(pair.to_dev(sig))]
    assert_find_equal(a, b, "repeat")


def test_genus3_full_size():
    """200,000 units and 16,384 signals from the 4M-point genus-3 cloud (the launch
    configuration the benchmark times), every output compared."""
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS["genus3_200k"]
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    sig = SignalStream(cloud, wl.signal_seed).next(wl.m)
    pair = Pair(units, m_max=wl.m)
    g, o = pair.find(sig)
    assert_find_equal(g, o, "genus3_200k")


@pytest.mark.parametrize("variant", [1, 2, 3, 4, 5, 6])
@pytest.mark.parametrize("n,m,seed", [(2, 3, 0), (3, 1, 1), (257, 999, 2), (4000, 16_384, 3),
                                      (30_000, 5_000, 4)])
def test_both_kernel_variants(variant, n, m, seed):
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(100 + seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    sig = rng.standard_normal((3, m)).astype(np.float32)
    pair = Pair(units, m_max=m)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, variant)
    g, o = pair.find(sig)
    assert_find_equal(g, o, f"variant={variant} n={n} m={m}")


@pytest.mark.parametrize("variant", [1, 2, 3, 4, 5, 6])
def test_cancellation_and_near_ties_far_from_the_origin(variant):
    """Units and signals around (1000, -1000, 1000) separated by ~1e-3: the expanded form
    loses about 12 bits to cancellation here, and many distances differ by a few ulps, so a
    screen without a correct rounding margin would drop true winners."""
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(77)
    c = np.array([1000.0, -1000.0, 1000.0])[:, None]
    n, m = 6000, 4096
    off = rng.standard_normal((3, n)) * 1e-3
    units = (c + off).astype(np.float32)
    # a shell of near-equidistant units around some signals
    sig = (c + rng.standard_normal((3, m)) * 1e-3).astype(np.float32)
    for j in range(0, m, 97):
        dirs = rng.standard_normal((3, 8))
        dirs /= np.linalg.norm(dirs, axis=0)
        k = (j // 97) * 8 % (n - 8)
        units[:, k:k + 8] = (sig[:, j:j + 1].astype(np.float64) + 2e-4 * dirs).astype(np.float32)
    pair = Pair(units, m_max=m)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, variant)
    g, o = pair.find(sig)
    assert_find_equal(g, o, f"variant={variant}")


@pytest.mark.parametrize("variant", [2, 3, 4, 5])
def test_screened_variants_ties_on_a_grid(variant):
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(5)
    units = rng.integers(-2, 3, (3, 2000)).astype(np.float32)
    sig = rng.integers(-2, 3, (3, 9000)).astype(np.float32)
    pair = Pair(units, m_max=9000)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, variant)
    for split in (1, 5, 64):
        pair.net.tune(gsn.GSN_TUNE_SPLIT, split)
        g, o = pair.find(sig)
        assert_find_equal(g, o, f"split={split}")


@pytest.mark.parametrize("variant", [1, 2, 3, 4, 5, 6])
@pytest.mark.parametrize("scale", [1e17, 1e20])
def test_huge_signal_coordinates_are_scanned_exactly(variant, scale):
    """Signals far outside the screen's range (margin above 2^90, distances near or past
    binary32 overflow) beside ordinary ones: the screened variants scan such signals
    exactly in the direct form; ties of overflowed distances go to the smaller index."""
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(31)
    units = rng.standard_normal((3, 3000)).astype(np.float32)
    sig = rng.standard_normal((3, 1000)).astype(np.float32)
    far = rng.choice(1000, 120, replace=False)
    sig[:, far] = (rng.standard_normal((3, 120)) * scale).astype(np.float32)
    pair = Pair(units, m_max=1000)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, variant)
    g, o = pair.find(sig)
    assert_find_equal(g, o, f"variant={variant} scale={scale:g}")


@pytest.mark.parametrize("variant", [2, 3, 4, 5])
def test_one_huge_unit_opens_every_signal(variant):
    """A single unit at 1e19 makes the magnitude bounds overflow, so every signal is open
    (scanned exactly); results still match the oracle."""
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(32)
    units = rng.standard_normal((3, 700)).astype(np.float32)
    units[:, 123] = np.float32(1e19)
    sig = rng.standard_normal((3, 300)).astype(np.float32)
    pair = Pair(units, m_max=300)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, variant)
    g, o = pair.find(sig)
    assert_find_equal(g, o, f"variant={variant}")


@pytest.mark.parametrize("variant", [2, 3, 4, 5])
def test_everything_at_1e17_is_scanned_exactly(variant):
    """Units and signals spread at the 1e17 scale: distances are finite and distinct but the
    screen's margin exceeds its range for every signal, so all are scanned exactly."""
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(33)
    units = (rng.standard_normal((3, 900)) * 1e17).astype(np.float32)
    sig = (rng.standard_normal((3, 400)) * 1e17).astype(np.float32)
    pair = Pair(units, m_max=400)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, variant)
    g, o = pair.find(sig)
    assert len(np.unique(o[0])) > 100, "the case must not collapse into ties"
    assert_find_equal(g, o, f"variant={variant}")


@pytest.mark.parametrize("n,m,seed", [(2, 5, 0), (130, 700, 1), (511, 64, 2), (40_037, 2_999, 3),
                                      (200_003, 1_300, 4)])
def test_dynamic_scan_any_grab_and_replica_count(n, m, seed):
    """Variant 5 deals the unit batches out with atomic counters; the answer cannot depend
    on the grab size, the number of replicas (rows of partial keys), or on which wave took
    which batch.  Sizes with fewer batches than lists (2, 130, 511 units), ragged batches
    and signal blocks, duplicates across lists and signals on units."""
    from paper_1503_08294_amd import gsn
    rng = np.random.default_rng(300 + seed)
    units = rng.standard_normal((3, n)).astype(np.float32)
    if n >= 2_000:
        units[:, n - 1_000:] = units[:, :1_000]
    sig = rng.standard_normal((3, m)).astype(np.float32)
    k = min(m, n) // 2
    sig[:, :k] = units[:, n - k:]
    pair = Pair(units, m_max=m)
    o = pair.orc.find_winners(sig)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, 5)
    for split, grab in ((0, 0), (8, 1), (16, 3), (64, 2), (24, 1024), (0, 7)):
        pair.net.tune(gsn.GSN_TUNE_SPLIT, split)
        pair.net.tune(gsn.GSN_TUNE_GRAB, grab)
        g = [t.cpu().numpy() for t in pair.net.find_winners(pair.to_dev(sig))]
        assert_find_equal(g, o, f"n={n} m={m} split={split} grab={grab}")


def test_dynamic_scan_genus3_full_size():
    """Variant 5 on the full 200,000 x 16,384 genus-3 launch, every output compared."""
    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS["genus3_200k"]
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    sig = SignalStream(cloud, wl.signal_seed).next(wl.m)
    pair = Pair(units, m_max=wl.m)
    pair.net.tune(gsn.GSN_TUNE_VARIANT, 5)
    g, o = pair.find(sig)
    assert_find_equal(g, o, "genus3_200k variant 5")


@pytest.mark.parametrize("m", [1, 2, 3, 63, 64, 65, 200, 256, 257, 1024])
@pytest.mark.parametrize("n,kind", [(2, "random"), (3, "grid"), (1_000, "grid"),
                                    (100_000, "random"), (200_003, "random")])
def test_small_batches(m, n, kind):
    """Batches of at most 256 signals take the unit-parallel scan by default (larger ones the
    staged scan): every slot count from 1 to 256, ragged slot groups (3, 63, 65, 200),
    integer grids with many exact ties and duplicated units, signals on top of units."""
    rng = np.random.default_rng(1000 * m + n)
    if kind == "grid":
        units = rng.integers(-3, 4, (3, n)).astype(np.float32)
        sig = rng.integers(-3, 4, (3, m)).astype(np.float32)
    else:
        units = rng.standard_normal((3, n)).astype(np.float32)
        sig = rng.standard_normal((3, m)).astype(np.float32)
        if n >= 4:
            units[:, n // 2:n // 2 + n // 4] = units[:, :n // 4]      # exact duplicates
    k = min(m, n) // 2
    sig[:, :k] = units[:, n - k:]
    pair = Pair(units, m_max=max(m, 256))
    g, o = pair.find(sig)
    assert_find_equal(g, o, f"n={n} m={m} {kind}")
