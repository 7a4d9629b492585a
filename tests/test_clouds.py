"""The seeded input generators: shapes, determinism, and points on their surfaces."""
import numpy as np

from paper_1503_08294_amd import clouds


def test_sphere_points_are_on_the_unit_sphere():
    p = clouds.sphere_cloud(5000, 0).astype(np.float64)
    np.testing.assert_allclose(np.linalg.norm(p, axis=1), 1.0, atol=1e-6)
    assert np.array_equal(p, clouds.sphere_cloud(5000, 0))


def test_torus_points_and_noise():
    p = clouds.torus_cloud(20000, 0, 1.0, 0.3, 0.0).astype(np.float64)
    rho = np.hypot(p[:, 0], p[:, 1])
    np.testing.assert_allclose(np.hypot(rho - 1.0, p[:, 2]), 0.3, atol=1e-6)
    # area-uniform: the outer half (rho > R) holds (pi R + 2 r) / (2 pi R) of the area
    frac = (rho > 1.0).mean()
    assert abs(frac - (np.pi + 0.6) / (2 * np.pi)) < 0.02
    q = clouds.torus_cloud(20000, 0, 1.0, 0.3, 0.005).astype(np.float64)
    rq = np.hypot(np.hypot(q[:, 0], q[:, 1]) - 1.0, q[:, 2]) - 0.3
    assert 0.003 < rq.std() < 0.007


def test_genus3_points_are_on_the_tube_surface():
    p = clouds.genus3_cloud(20000, 0, jitter=0.0)
    d = clouds.genus3_distance(p)
    np.testing.assert_allclose(d, clouds.GENUS3_TUBE, atol=2e-6)
    # every primitive is represented, including the chord tubes
    assert (np.abs(p[:, 0] - 0.35) < 0.13).sum() > 1000
    assert (np.abs(p[:, 0] + 0.35) < 0.13).sum() > 1000


def test_spheres_plane_density_ratio():
    p = clouds.spheres_plane_cloud(60000, 0).astype(np.float64)
    on_patch = np.abs(p[:, 2] + 0.8) < 1e-6
    assert on_patch.any()
    # density (points per area) on the patch vs the heavy sphere region far from others
    c1 = np.array([-0.45, 0.0, 0.0])
    cap = (np.abs(np.linalg.norm(p - c1, axis=1) - 0.6) < 1e-6) & (p[:, 0] < -0.7)
    cap_area = 2 * np.pi * 0.6 * (0.6 - 0.25)        # spherical cap x < -0.7
    ratio = (cap.sum() / cap_area) / (on_patch.sum() / 2.4 ** 2)
    assert 8.0 < ratio < 12.5


def test_signal_stream_is_seeded_and_soa():
    cloud = clouds.sphere_cloud(1000, 0)
    a = clouds.SignalStream(cloud, 2)
    b = clouds.SignalStream(cloud, 2)
    x1, x2 = a.next(64), a.next(64)
    assert x1.shape == (3, 64) and x1.dtype == np.float32 and x1.flags["C_CONTIGUOUS"]
    np.testing.assert_array_equal(x1, b.next(64))
    np.testing.assert_array_equal(x2, b.next(64))
    units = clouds.initial_units(cloud, 100, 1)
    assert units.shape == (3, 100)
    assert len({tuple(c) for c in units.T}) == 100
