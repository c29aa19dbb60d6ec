"""Pins of the fp64 oracle of the paper's multi-scale Fourier front end
(Sec. Encoder: 15 per-hit features min-max normalised, expanded at 16 scales
to 480 values, projected by a dense layer to d_model), independent of the
oracle's formulas: exact values at special points, the features rebuilt by
repeated squaring of a unit complex number, single weights that pin the
column order, and the float32 normalisation done with numpy's float32.
"""
import math

import numpy as np
import pytest

import oracle
import tracksynth as ts


def _squaring_features(u):
    """sin and cos of pi 2^s u, s = 0..15, from z = exp(i pi u) squared s times."""
    z = complex(math.cos(math.pi * u), math.sin(math.pi * u))
    sin, cos = [], []
    for _ in range(16):
        sin.append(z.imag)
        cos.append(z.real)
        z = z * z
    return np.array(sin), np.array(cos)


def test_special_points():
    lo = np.array([0.0, -2.0, 10.0], np.float32)
    hi = np.array([2.0, 2.0, 14.0], np.float32)
    # u = 1/2, 0, 1
    phi = oracle.fourier_features([1.0, -2.0, 14.0], lo, hi).reshape(3, 2, 16)
    s = np.arange(16)
    assert np.allclose(phi[0, 0], np.where(s == 0, 1.0, 0.0), atol=1e-15)          # sin(pi 2^s / 2)
    assert np.allclose(phi[0, 1], np.where(s == 0, 0.0, np.where(s == 1, -1.0, 1.0)), atol=1e-15)
    assert np.array_equal(phi[1, 0], np.zeros(16)) and np.array_equal(phi[1, 1], np.ones(16))   # u = 0
    assert np.allclose(phi[2, 0], 0.0, atol=1e-15)                                  # u = 1
    assert np.allclose(phi[2, 1], np.where(s == 0, -1.0, 1.0), atol=1e-15)


def test_features_match_repeated_squaring():
    rng = np.random.default_rng(3)
    lo = np.array([-1000.0, -3000.0, 0.0], np.float32)
    hi = np.array([1000.0, 3000.0, 1.0], np.float32)
    for _ in range(200):
        x = np.array([rng.uniform(-1000, 1000), rng.uniform(-3000, 3000), rng.uniform(0, 1)], np.float32)
        phi = oracle.fourier_features(x, lo, hi).reshape(3, 2, 16)
        for f in range(3):
            u = float((x[f] - lo[f]) * (np.float32(1.0) / (hi[f] - lo[f])))
            sn, cs = _squaring_features(u)
            # squaring doubles the phase error each time: 2^15 * 1e-16
            assert np.allclose(phi[f, 0], sn, atol=1e-10) and np.allclose(phi[f, 1], cs, atol=1e-10)


def test_normalisation_is_float32():
    """u = fl32(fl32(x - lo) * fl32(1 / fl32(hi - lo))): at the finest scale a
    different rounding of u moves the phase by up to pi 2^15 2^-24."""
    rng = np.random.default_rng(4)
    lo = np.array([-1000.0], np.float32)
    hi = np.array([1000.0], np.float32)
    n_diff = 0
    for _ in range(300):
        x = np.float32(rng.uniform(-1000, 1000))
        t = np.float32(x - lo[0])
        inv = np.float32(np.float32(1.0) / np.float32(hi[0] - lo[0]))
        u32 = float(np.float32(t * inv))
        u64 = (float(x) + 1000.0) / 2000.0
        phi = oracle.fourier_features([x], lo, hi)
        assert abs(phi[15] - math.sin(math.pi * math.fmod(u32 * 2.0 ** 15, 2.0))) < 1e-12
        n_diff += abs(math.sin(math.pi * u32 * 2 ** 15) - math.sin(math.pi * u64 * 2 ** 15)) > 1e-9
    assert n_diff > 50   # the float32 reading is visible at this scale


@pytest.mark.parametrize("f,c,s", [(0, 0, 0), (2, 1, 7), (1, 0, 15), (2, 1, 15)])
def test_dense_projection_reads_column_32f_16c_s(f, c, s):
    """With no layers the residual stream is the front end's output: a single
    weight fe.W[j][32 f + 16 c + s] = 1 and bias 0.25 give r_j = 0.25 +
    (sin if c == 0 else cos)(pi 2^s u_f) and 0.25 elsewhere."""
    d, F, j = 4, 3, 2
    lo = np.array([0.0, -5.0, 100.0], np.float32)
    hi = np.array([1.0, 5.0, 300.0], np.float32)
    W = np.zeros((d, 32 * F))
    W[j, 32 * f + 16 * c + s] = 1.0
    rest = np.zeros(ts.blob_size(0, d) - 4 * d)   # head only (no layers)
    blob = np.concatenate([lo, hi, W.ravel(), np.full(d, 0.25), rest]).astype(np.float32)
    assert blob.size == oracle.fourier_blob_size(0, d, F)
    hits = np.array([[0.3, 1.5, 170.0], [0.9, -4.0, 290.0]], np.float32)
    _, _, resid = oracle.track_forward(hits, blob, 0, d, n_features=F)
    for t in range(2):
        u = float((hits[t, f] - lo[f]) * (np.float32(1.0) / (hi[f] - lo[f])))
        sn, cs = _squaring_features(u)
        want = np.full(d, 0.25)
        want[j] += (sn if c == 0 else cs)[s]
        assert np.allclose(resid[t], want, atol=1e-10)


def test_fourier_model_without_layers_is_head_of_mean():
    """n_layers = 0: out = W2 SiLU(W1 mean_t(fe.W phi_t + fe.b) + b1) + b2,
    composed here with the squaring features and numpy products."""
    w = ts.workload("fourier15_tiny_d32_fp32")
    F, d = 15, 8
    rng = np.random.default_rng(9)
    hits, offs = ts.make_tracks(w, n_tracks=3)
    _, sf, _ = oracle.seed_tracks(hits, offs, w.b_field)
    feats = ts.hit_features(w, hits, offs, sf)
    lo, hi = ts.feature_bounds(w)
    fW = rng.normal(0, 0.1, (d, 32 * F)).astype(np.float32)
    fb = rng.normal(0, 0.1, d).astype(np.float32)
    W1 = rng.normal(0, 0.3, (d, d)).astype(np.float32)
    b1 = rng.normal(0, 0.1, d).astype(np.float32)
    W2 = rng.normal(0, 0.3, (5, d)).astype(np.float32)
    b2 = rng.normal(0, 0.1, 5).astype(np.float32)
    blob = np.concatenate([lo, hi, fW.ravel(), fb, W1.ravel(), b1, W2.ravel(), b2])
    out = oracle.fit_tracks(feats, offs, blob, 0, d, n_features=F)
    for i in range(3):
        rows = []
        for t in range(offs[i], offs[i + 1]):
            phi = []
            for f in range(F):
                u = float((feats[t, f] - lo[f]) * (np.float32(1.0) / (hi[f] - lo[f])))
                sn, cs = _squaring_features(u)
                phi += list(sn) + list(cs)
            rows.append(fW.astype(np.float64) @ np.array(phi) + fb)
        p = np.mean(rows, axis=0)
        h = W1.astype(np.float64) @ p + b1
        h = h / (1.0 + np.exp(-h))
        assert np.allclose(out[i], W2.astype(np.float64) @ h + b2, rtol=1e-9, atol=1e-9)


def test_generator_features_lie_in_their_bounds():
    """The bounds cover the generated features (u in [0, 1], up to the seed
    features' rare tails)."""
    w = ts.workload("fourier15_deploy_d128x4_bf16_8m")
    hits, offs = ts.make_tracks(w, n_tracks=2000)
    _, sf, _ = oracle.seed_tracks(hits, offs, w.b_field)
    feats = ts.hit_features(w, hits, offs, sf)
    lo, hi = ts.feature_bounds(w)
    u = (feats - lo) / (hi - lo)
    assert feats.shape[1] == 15
    assert np.all(u[:, :12] >= 0) and np.all(u[:, :12] <= 1)
    assert np.mean((u[:, 12:] >= 0) & (u[:, 12:] <= 1)) > 0.999
