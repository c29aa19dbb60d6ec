"""Pins of the fp64 oracle of the analytic three-hit seed and of its per-hit
residual features (Sec. Method, "Analytic seed"), independent of the oracle's
own formulas: truth of noise-free helices, a hand-built circle, a brute-force
circle fit, symmetries, and the residual features of hits moved off the helix
by known amounts along the frame's directions.
"""
import math

import numpy as np
import pytest

import oracle
import tracksynth as ts

KAPPA = ts.KAPPA_GEV_PER_T_M


def _wrap(a):
    return (a + math.pi) % (2 * math.pi) - math.pi


def _noise_free(w, n, seed=5):
    """fp64 hits of noise-free helices and their perigee truth."""
    streams = {k: np.random.default_rng([seed, i])
               for i, k in enumerate(("pt", "eta", "phi", "d0", "z0", "q", "length"))}
    pt, eta, phi, d0, z0, q, _ = ts._draw_params(w, streams, n)
    radii = np.linspace(w.r_min, w.r_max, w.n_det_layers)
    x, y, z, arc = ts.helix_hits(pt, eta, phi, d0, z0, q, radii, w.b_field)
    theta = 2.0 * np.arctan(np.exp(-eta))
    truth = np.stack([d0, z0, phi, theta, q / (pt * np.cosh(eta))], axis=1)
    return x, y, z, arc, truth


@pytest.mark.parametrize("name", ["d128x4_fp32_65k", "deploy_d128x4_bf16_8m", "d256x6_bf16_1m"])
def test_noise_free_helices_give_truth(name):
    """Three exact helix points determine the helix: the seed is the truth."""
    w = ts.WORKLOADS[name]
    x, y, z, _, truth = _noise_free(w, 400)
    for i in range(truth.shape[0]):
        s = oracle.seed_from_points(np.stack([x[i, :3], y[i, :3], z[i, :3]], 1), w.b_field)
        assert abs(s[0] - truth[i, 0]) < 1e-7, (i, s, truth[i])
        assert abs(s[1] - truth[i, 1]) < 1e-7
        assert abs(_wrap(s[2] - truth[i, 2])) < 1e-10
        assert abs(s[3] - truth[i, 3]) < 1e-10
        assert abs(s[4] - truth[i, 4]) <= 1e-8 * abs(truth[i, 4])


def test_features_vanish_on_the_helix_and_give_its_path_length():
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    x, y, z, arc, truth = _noise_free(w, 50, seed=9)
    for i in range(truth.shape[0]):
        s = oracle.seed_from_points(np.stack([x[i, :3], y[i, :3], z[i, :3]], 1), w.b_field)
        for j in range(w.n_det_layers):
            f = oracle.seed_features_hit(s, w.b_field, [x[i, j], y[i, j], z[i, j]])
            assert abs(f[0]) < 1e-8 and abs(f[1]) < 1e-8
            assert abs(f[2] - arc[i, j] / math.sin(truth[i, 3])) < 1e-7


def _circle_centre(x, y):
    """Centre of the circle through three transverse points, from the linear
    system x^2 + y^2 + a x + b y + c = 0 (a brute-force fit, not the oracle's
    conformal map)."""
    A = np.stack([x, y, np.ones(3)], 1)
    a, b, _ = np.linalg.solve(A, -(x ** 2 + y ** 2))
    return -a / 2, -b / 2


@pytest.mark.parametrize("delta", [0.05, -0.7, 3.0])
def test_features_of_a_hit_moved_off_the_helix_radially(delta):
    """A noise-free hit moved by delta along the outward normal of the seed
    circle (away from its centre, in the transverse plane) keeps its turning
    angle, so its helix point and path length are unchanged and its residual
    is delta times that normal.  U = z x T / |z x T| is the transverse tangent
    turned by +90 degrees: it points to the centre for counter-clockwise motion
    (negative charge in a field along +z) and away from it for clockwise
    motion (positive charge).  So dU = q delta and dV = 0: a flipped U, a
    missing or misplaced asinh, or a residual taken the other way would fail.
    Both charges occur among the tracks."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    x, y, z, arc, truth = _noise_free(w, 40, seed=11)
    q = np.sign(truth[:, 4])
    assert (q > 0).any() and (q < 0).any()
    for i in range(truth.shape[0]):
        s = oracle.seed_from_points(np.stack([x[i, :3], y[i, :3], z[i, :3]], 1), w.b_field)
        cx, cy = _circle_centre(x[i, :3], y[i, :3])
        for j in (4, 11, 19):
            nx, ny = x[i, j] - cx, y[i, j] - cy
            nn = math.hypot(nx, ny)
            hit = [x[i, j] + delta * nx / nn, y[i, j] + delta * ny / nn, z[i, j]]
            f = oracle.seed_features_hit(s, w.b_field, hit)
            assert abs(f[0] - math.asinh(q[i] * delta)) < 1e-7, (i, j, f, q[i])
            assert abs(f[1]) < 1e-7
            assert abs(f[2] - arc[i, j] / math.sin(truth[i, 3])) < 1e-7


@pytest.mark.parametrize("dz", [0.02, -1.5, 4.0])
def test_features_of_a_hit_moved_off_the_helix_along_z(dz):
    """A noise-free hit moved by dz along z keeps its transverse position, so
    its helix point and path length are unchanged and its residual is
    (0, 0, dz).  U is transverse, so dU = 0; V = T x U has z component
    sin(theta), so dV = sin(theta) dz.  A missing sin(theta), or a V built as
    U x T, would fail."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    x, y, z, arc, truth = _noise_free(w, 40, seed=12)
    for i in range(truth.shape[0]):
        s = oracle.seed_from_points(np.stack([x[i, :3], y[i, :3], z[i, :3]], 1), w.b_field)
        st = math.sin(truth[i, 3])
        for j in (3, 9, 18):
            f = oracle.seed_features_hit(s, w.b_field, [x[i, j], y[i, j], z[i, j] + dz])
            assert abs(f[0]) < 1e-7, (i, j, f)
            assert abs(f[1] - math.asinh(st * dz)) < 1e-7, (i, j, f, st)
            assert abs(f[2] - arc[i, j] / st) < 1e-7


def test_features_of_a_general_off_helix_move_add_up():
    """The two moves together: outward by a, along z by b gives dU = q a and
    dV = sin(theta) b (the frame is orthonormal, so the components of the
    residual do not mix)."""
    w = ts.WORKLOADS["d128x4_fp32_65k"]
    x, y, z, arc, truth = _noise_free(w, 30, seed=13)
    rng = np.random.default_rng(14)
    for i in range(truth.shape[0]):
        s = oracle.seed_from_points(np.stack([x[i, :3], y[i, :3], z[i, :3]], 1), w.b_field)
        cx, cy = _circle_centre(x[i, :3], y[i, :3])
        j = int(rng.integers(3, w.n_det_layers))
        a, b = rng.uniform(-2, 2, 2)
        nx, ny = x[i, j] - cx, y[i, j] - cy
        nn = math.hypot(nx, ny)
        f = oracle.seed_features_hit(s, w.b_field, [x[i, j] + a * nx / nn, y[i, j] + a * ny / nn, z[i, j] + b])
        st = math.sin(truth[i, 3])
        assert abs(f[0] - math.asinh(math.copysign(1.0, truth[i, 4]) * a)) < 1e-7
        assert abs(f[1] - math.asinh(st * b)) < 1e-7
        assert abs(f[2] - arc[i, j] / st) < 1e-7


def test_hand_built_positive_track():
    """A positive charge in a field along +z turns clockwise: three points on
    the circle of centre (0, -R) through the origin, moving along +x at the
    origin, are a q > 0 track with its perigee at the origin and phi = 0."""
    R, B = 5000.0, 2.0
    al = np.array([0.01, 0.02, 0.035])
    pts = np.stack([R * np.sin(al), -R + R * np.cos(al), 3.0 * R * al], 1)  # cot(theta) = 3
    s = oracle.seed_from_points(pts, B)
    pt = KAPPA * B * R / 1000.0
    theta = math.atan2(1.0, 3.0)
    assert abs(s[0]) < 1e-9 and abs(s[1]) < 1e-9 and abs(s[2]) < 1e-12
    assert abs(s[3] - theta) < 1e-12
    assert abs(s[4] - math.sin(theta) / pt) < 1e-12 * abs(s[4])
    # mirrored in x: the same circle run counter-clockwise is a negative charge
    s2 = oracle.seed_from_points(pts * np.array([-1.0, 1.0, 1.0]), B)
    assert s2[4] < 0 and abs(abs(_wrap(s2[2])) - math.pi) < 1e-12


def test_radius_and_impact_match_a_brute_force_circle():
    """Circle through three smeared points from the 3x3 linear system
    x^2 + y^2 + a x + b y + c = 0: its radius gives pT, its distance from the
    axis |d0|."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hits, offs = ts.make_tracks(w, n_tracks=300)
    for i in range(300):
        p = hits[offs[i]:offs[i] + 3].astype(np.float64)
        A = np.stack([p[:, 0], p[:, 1], np.ones(3)], 1)
        a, b, c = np.linalg.solve(A, -(p[:, 0] ** 2 + p[:, 1] ** 2))
        cx, cy = -a / 2, -b / 2
        R = math.sqrt(cx * cx + cy * cy - c)
        s = oracle.seed_from_points(p, w.b_field)
        pt = abs(math.sin(s[3]) / s[4])
        assert abs(pt - KAPPA * w.b_field * R / 1000.0) < 1e-7 * pt
        assert abs(abs(s[0]) - abs(math.hypot(cx, cy) - R)) < 1e-6


def test_rotation_about_z_shifts_phi_only():
    w = ts.WORKLOADS["d128x4_fp32_65k"]
    hits, offs = ts.make_tracks(w, n_tracks=64)
    for i in range(64):
        p = hits[offs[i]:offs[i] + 3].astype(np.float64)
        s = oracle.seed_from_points(p, w.b_field)
        for ang in (0.4, -2.0, 3.0):
            c, sn = math.cos(ang), math.sin(ang)
            pr = p.copy()
            pr[:, 0], pr[:, 1] = c * p[:, 0] - sn * p[:, 1], sn * p[:, 0] + c * p[:, 1]
            sr = oracle.seed_from_points(pr, w.b_field)
            assert abs(_wrap(sr[2] - s[2] - ang)) < 1e-9
            for k in (0, 1, 3, 4):
                assert abs(sr[k] - s[k]) <= 1e-9 * max(1.0, abs(s[k]))


def test_mirror_in_z():
    w = ts.WORKLOADS["d128x4_fp32_65k"]
    hits, offs = ts.make_tracks(w, n_tracks=64)
    for i in range(64):
        p = hits[offs[i]:offs[i] + 3].astype(np.float64)
        s = oracle.seed_from_points(p, w.b_field)
        sm = oracle.seed_from_points(p * np.array([1.0, 1.0, -1.0]), w.b_field)
        assert abs(sm[3] - (math.pi - s[3])) < 1e-12
        assert abs(sm[1] + s[1]) < 1e-9
        for k in (0, 2, 4):
            assert abs(sm[k] - s[k]) <= 1e-12 * max(1.0, abs(s[k]))


def test_smeared_tracks_land_near_truth():
    """With 10 um smearing the seed is a rough but unbiased estimate."""
    w = ts.WORKLOADS["d128x4_fp32_65k"]
    hits, offs, truth = ts.make_tracks(w, n_tracks=2000, with_truth=True)
    seeds, _, bad = oracle.seed_tracks(hits, offs, w.b_field, features=False)
    assert bad == 0
    assert np.median(np.abs(_wrap(seeds[:, 2] - truth[:, 2]))) < 2e-3
    assert np.median(np.abs(seeds[:, 3] - truth[:, 3])) < 2e-3
    assert np.median(np.abs(seeds[:, 4] / truth[:, 4] - 1.0)) < 0.1


def test_batch_matches_single_track_calls_and_flags_short_tracks():
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hits, offs = ts.make_tracks(w, n_tracks=40)
    # make track 3 two hits long and track 7 one hit long
    L = np.diff(offs)
    L[3], L[7] = 2, 1
    keep = np.concatenate([np.arange(offs[i], offs[i] + L[i]) for i in range(40)])
    h = hits[keep]
    o = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
    seeds, feats, bad = oracle.seed_tracks(h, o, w.b_field)
    assert bad == 2
    assert np.all(np.isnan(seeds[[3, 7]])) and np.all(np.isnan(feats[o[3]:o[4]]))
    for i in (0, 5, 39):
        s = oracle.seed_from_points(h[o[i]:o[i] + 3].astype(np.float64), w.b_field)
        assert np.array_equal(s, seeds[i])
        for j in range(o[i], o[i + 1]):
            assert np.array_equal(oracle.seed_features_hit(s, w.b_field, h[j].astype(np.float64)), feats[j])


def test_collinear_points_have_no_seed():
    s = oracle.seed_from_points([[10.0, 0.0, 0.0], [20.0, 0.0, 1.0], [30.0, 0.0, 2.0]], 2.0)
    assert np.all(np.isnan(s))
