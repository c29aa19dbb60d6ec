"""GPU parity of the encoder with the paper's multi-scale Fourier front end
(15 per-hit features, 16 scales, 480 values projected to d_model) against the
fp64 oracle, element by element: pooled-head outputs and end states, ragged
and fixed lengths on both tile shapes, rejected tracks, tile independence.
The inputs are the generator's 12 measured-feature stand-ins and the oracle's
3 seed residual features.
"""
import dataclasses
import os

import numpy as np
import pytest

import oracle
import tracksynth as ts
from tests.parity import TOL, assert_parity, column_rms

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

THREADS = int(os.environ.get("ORACLE_THREADS", "0"))
N = {"fourier15_tiny_d32_fp32": 256, "fourier15_d128x4_fp32_65k": 1024, "fourier15_deploy_d128x4_bf16_8m": 2048}


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32479_amd as tf
    return tf


def _inputs(w, n):
    """Features of n tracks; tracks too short for a seed (under three hits)
    get zero seed features (the seed leaves them NaN)."""
    hits, offs = ts.make_tracks(w, n_tracks=n)
    _, sf, bad = oracle.seed_tracks(hits, offs, w.b_field)
    assert bad == int(np.sum(np.diff(offs) < 3))
    return ts.hit_features(w, hits, offs, np.nan_to_num(sf, nan=0.0)), offs


def _weights(tf, w, max_hits=None):
    blob = ts.make_fourier_weights(w)
    W = tf.Weights(blob, w.n_layers, w.d_model, tf.MODE_FOR_WEIGHTS[w.dtype],
                   w.len_max if max_hits is None else max_hits, n_features=w.n_features)
    return W, blob


def _gpu(tf, W, feats, offs, states=False, n_tracks=None):
    h = torch.from_numpy(np.ascontiguousarray(feats, dtype=np.float32)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(offs, dtype=np.int32)).cuda()
    out = (tf.fit_tracks_states if states else tf.fit_tracks)(h, o, W, n_tracks=n_tracks)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _ref(w, feats, offs, blob, states=False):
    fn = oracle.track_states if states else oracle.fit_tracks
    return fn(feats, offs, blob, w.n_layers, w.d_model, n_threads=THREADS, n_features=w.n_features)


def _state_err(g, r):
    ok = ~np.isnan(r).any(axis=1)
    rms = np.sqrt(np.mean(r[ok] ** 2, axis=1, keepdims=True))
    return float(np.max(np.abs(g[ok] - r[ok]) / rms))


@pytest.mark.parametrize("name", list(ts.FOURIER_WORKLOADS))
def test_fourier_encoder_matches_oracle(tf, name):
    w = ts.workload(name)
    print(f"[fourier] {name} n={N[name]}", flush=True)
    W, blob = _weights(tf, w)
    feats, offs = _inputs(w, N[name])
    g = _gpu(tf, W, feats, offs)
    r = _ref(w, feats, offs, blob)
    emax, l2 = assert_parity(g, r, TOL[w.dtype], name)
    print(f"[fourier] {name}: max col err {emax.max():.3g} l2 {l2.max():.3g}", flush=True)
    assert tf.device_error(W) == 0


@pytest.mark.parametrize("name", list(ts.FOURIER_WORKLOADS))
def test_fourier_end_states_match_oracle(tf, name):
    w = ts.workload(name)
    W, blob = _weights(tf, w)
    feats, offs = _inputs(w, min(N[name], 1024))
    g = _gpu(tf, W, feats, offs, states=True)
    r = _ref(w, feats, offs, blob, states=True)
    e = _state_err(g, r)
    print(f"[fourier-states] {name}: max err {e:.3g} of the track's state rms", flush=True)
    assert e <= TOL[w.dtype]


@pytest.mark.parametrize("name,L,max_hits", [("fourier15_deploy_d128x4_bf16_8m", 1, 32),
                                             ("fourier15_deploy_d128x4_bf16_8m", 64, 64),
                                             ("fourier15_d128x4_fp32_65k", 32, 32),
                                             ("fourier15_tiny_d32_fp32", 64, 64)])
def test_fourier_fixed_lengths(tf, name, L, max_hits):
    w = dataclasses.replace(ts.workload(name), len_min=L, len_max=L, n_det_layers=max(L, 8))
    print(f"[fourier-fixed] {name} L={L} max_hits={max_hits}", flush=True)
    W, blob = _weights(tf, w, max_hits=max_hits)
    feats, offs = _inputs(w, 200)
    assert_parity(_gpu(tf, W, feats, offs), _ref(w, feats, offs, blob), TOL[w.dtype], f"{name} L={L}")


def test_fourier_ragged_batches_bad_tracks_and_neighbours(tf):
    w0 = ts.workload("fourier15_deploy_d128x4_bf16_8m")
    W, blob = _weights(tf, w0, max_hits=32)
    w = dataclasses.replace(w0, len_min=1, len_max=32, n_det_layers=32)
    feats, offs = _inputs(w, 600)
    r_all = _ref(w, feats, offs, blob)
    for n in (1, 2, 33, 600):
        g = _gpu(tf, W, feats, offs[: n + 1])
        assert_parity(g, r_all[:n], TOL[w.dtype], f"n={n}", rms=column_rms(r_all))
    # track 4 emptied, track 8 too long: NaN rows, the rest unchanged
    Lk = np.diff(offs)
    Lk[4], Lk[8] = 0, 33
    rows = [np.resize(np.arange(offs[i], offs[i + 1]), Lk[i]) if Lk[i] else np.arange(0) for i in range(600)]
    f2 = feats[np.concatenate(rows)]
    o2 = np.concatenate([[0], np.cumsum(Lk)]).astype(np.int32)
    g = _gpu(tf, W, f2, o2)
    assert np.all(np.isnan(g[[4, 8]]))
    good = np.ones(600, bool)
    good[[4, 8]] = False
    assert_parity(g[good], r_all[good], TOL[w.dtype], "neighbours of bad tracks", rms=column_rms(r_all))
    assert tf.device_error(W) == (tf.DEVERR_EMPTY_TRACK | tf.DEVERR_TOO_LONG)
    # a track's result does not depend on its tile neighbours (bitwise)
    a = _gpu(tf, W, feats, offs)
    perm = np.random.default_rng(2).permutation(600)
    L = np.diff(offs)
    fp = np.concatenate([feats[offs[i]:offs[i + 1]] for i in perm])
    op = np.concatenate([[0], np.cumsum(L[perm])]).astype(np.int32)
    assert np.array_equal(_gpu(tf, W, fp, op), a[perm])


def test_fourier_model_rejects_unsupported_shapes(tf):
    blob = np.zeros(tf.blob_size(2, 64, 15), np.float32)
    with pytest.raises(tf.TrackfitError):
        tf.Weights(blob, 2, 64, "bf16", 32, n_features=15)      # d = 64 not built with the front end
    with pytest.raises(tf.TrackfitError):
        tf.Weights(np.zeros(10, np.float32), 2, 128, "bf16", 32, n_features=17)
