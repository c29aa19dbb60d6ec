"""Checks of the synthetic inputs: helix geometry, hit counts, seeding, weights."""
import dataclasses

import numpy as np
import pytest

import tracksynth as ts


def _noise_free(w, n=500, seed=1):
    rng = np.random.default_rng(seed)
    pt, eta, phi, d0, z0, q, _ = ts._draw_params(w, rng, n)
    radii = np.linspace(w.r_min, w.r_max, w.n_det_layers)
    x, y, z, s = ts.helix_hits(pt, eta, phi, d0, z0, q, radii, w.b_field)
    return (pt, eta, phi, d0, z0, q), radii, x, y, z, s


@pytest.mark.parametrize("name", list(ts.WORKLOADS))
def test_noise_free_hits_lie_on_cylinders(name):
    w = ts.WORKLOADS[name]
    _, radii, x, y, z, s = _noise_free(w)
    np.testing.assert_allclose(np.hypot(x, y), np.broadcast_to(radii, x.shape), rtol=1e-9)
    assert np.all(np.diff(s, axis=1) > 0)          # ordered outwards = time order
    assert np.all(np.abs(z) <= w.z_max)


def test_circle_through_hits_has_the_helix_radius():
    """R = pT / (0.299792458 B): fit a circle exactly through three noise-free hits."""
    w = ts.workload("d128x4_fp32_65k")
    (pt, eta, phi, d0, z0, q), radii, x, y, z, s = _noise_free(w, n=200)
    p1, p2, p3 = (np.stack([x[:, k], y[:, k]], 1) for k in (0, 9, 19))
    a = np.linalg.norm(p2 - p3, axis=1)
    b = np.linalg.norm(p1 - p3, axis=1)
    c = np.linalg.norm(p1 - p2, axis=1)
    cross = np.abs((p2 - p1)[:, 0] * (p3 - p1)[:, 1] - (p2 - p1)[:, 1] * (p3 - p1)[:, 0])
    R_fit = a * b * c / (2.0 * cross)
    R_true = 1000.0 * pt / (ts.KAPPA_GEV_PER_T_M * w.b_field)
    np.testing.assert_allclose(R_fit, R_true, rtol=1e-7)
    # the perigee is at distance |d0| from the axis and z grows as s * sinh(eta)
    slope = (z[:, -1] - z[:, 0]) / (s[:, -1] - s[:, 0])
    np.testing.assert_allclose(slope, np.sinh(eta), rtol=1e-9, atol=1e-12)


def test_charge_sets_turning_direction():
    """A positive track in +B_z turns clockwise: the azimuth of its hits decreases
    relative to the straight line (the cross product of successive steps is negative)."""
    w = ts.workload("d128x4_fp32_65k")
    (pt, eta, phi, d0, z0, q), radii, x, y, z, s = _noise_free(w, n=300)
    v1 = np.stack([x[:, 5] - x[:, 0], y[:, 5] - y[:, 0]], 1)
    v2 = np.stack([x[:, 19] - x[:, 5], y[:, 19] - y[:, 5]], 1)
    cross = v1[:, 0] * v2[:, 1] - v1[:, 1] * v2[:, 0]
    assert np.all(np.sign(cross) == -q)


@pytest.mark.parametrize("name", list(ts.WORKLOADS))
def test_hit_counts_and_packing(name):
    w = ts.WORKLOADS[name]
    hits, offs = ts.make_tracks(w, n_tracks=3000)
    L = np.diff(offs)
    assert offs[0] == 0 and offs[-1] == hits.shape[0]
    assert L.min() >= w.len_min and L.max() <= w.len_max
    if w.len_min != w.len_max:
        assert L.min() == w.len_min and L.max() == w.len_max   # the full range occurs
    r = np.hypot(hits[:, 0].astype(np.float64), hits[:, 1].astype(np.float64))
    radii = np.linspace(w.r_min, w.r_max, w.n_det_layers)
    for i in range(0, 3000, 97):
        np.testing.assert_allclose(r[offs[i]:offs[i + 1]], radii[:L[i]], rtol=2e-7, atol=1e-4)


def test_seeding_is_deterministic_and_chunked():
    w = ts.workload("deploy_d128x4_bf16_8m")
    h1, o1 = ts.make_tracks(w, n_tracks=70000)
    h2, o2 = ts.make_tracks(w, n_tracks=70000)
    assert np.array_equal(h1, h2) and np.array_equal(o1, o2)
    # the second chunk regenerates alone
    hc, lc, _ = ts.make_track_chunk(w, 1, ts.TRACK_CHUNK)
    start = o1[ts.TRACK_CHUNK]
    assert np.array_equal(hc[: o1[70000] - start], h1[start:])
    # the first tracks do not depend on how many are drawn
    h4, o4 = ts.make_tracks(w, n_tracks=100)
    assert np.array_equal(h4, h1[: o1[100]]) and np.array_equal(o4, o1[:101])
    # a different seed gives different tracks
    h3, _ = ts.make_tracks(w, n_tracks=100, seed=5)
    assert not np.array_equal(h3[:50], h1[:50])


def test_smearing_size():
    w = dataclasses.replace(ts.workload("d128x4_fp32_65k"), len_min=20, len_max=20)
    h0, _, _ = ts.make_track_chunk(w, 0, 2000, smear=False)
    h1, _, _ = ts.make_track_chunk(w, 0, 2000, smear=True)
    dz = (h1[:, 2] - h0[:, 2]).astype(np.float64)
    assert 0.008 < dz.std() < 0.012


def test_bf16_rounding():
    v = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.14159265, 1e-20], np.float32)
    r = ts.round_to_bf16(v)
    # ties go to even: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == np.float32(1.0 + 2 ** -6) and r[3] == -2.5
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)
    assert abs(float(r[4]) - 3.14159265) < 2 ** -7 * 2


def test_weights_blob():
    for name, w in ts.WORKLOADS.items():
        b = ts.make_weights(w)
        assert b.dtype == np.float32 and b.size == ts.blob_size(w.n_layers, w.d_model)
        if w.dtype == "bf16":
            assert np.all((b.view(np.uint32) & 0xFFFF) == 0)
    a = ts.make_weights(n_layers=2, d=64, dtype="fp32", seed=3)
    P = ts.split_blob(a, 2, 64)
    assert abs(P["layer0.in.W"].std() - 64 ** -0.5) < 0.01
    assert abs(P["layer1.out.W"].std() - 128 ** -0.5) < 0.01
    assert P["layer0.norm.g"].min() >= 0.5 and P["layer0.norm.g"].max() <= 1.5
    assert np.abs(P["head.b1"]).max() <= 64 ** -0.5
