"""Pins of the fp64 oracle of the paper's readout and decode (Sec. Encoder,
last paragraph: end states -> RMSNorm -> two-layer head -> 35 quantiles;
Sec. Losses: median point estimate, seed-anchored targets), against an
independent numpy restatement, closed forms and invariances.
"""
import math

import numpy as np
import pytest

import oracle
import tracksynth as ts
from tests import bruteforce


def test_median_of_seven_matches_numpy():
    rng = np.random.default_rng(0)
    for _ in range(300):
        v = rng.normal(size=7)
        if rng.random() < 0.3:
            v[rng.integers(7)] = v[rng.integers(7)]  # ties
        assert oracle.median_odd(v) == np.median(v)
    assert oracle.median_odd(np.arange(7.0)) == 3.0
    assert oracle.median_odd(np.arange(7.0)[::-1]) == 3.0


def test_decode_closed_forms():
    seed = np.array([0.05, -1.0, 3.0, 1.2, -0.4])
    med = np.array([0.01, 0.2, 0.5, -0.1, 0.25])
    out = oracle.decode(seed, med)
    assert out[0] == seed[0] + med[0] and out[1] == seed[1] + med[1] and out[3] == seed[3] + med[3]
    assert abs(out[2] - (3.5 - 2 * math.pi)) < 1e-15          # wrapped into [-pi, pi)
    assert out[4] == seed[4] + 0.25 * (0.4 + 0.02)
    # the scale-free q/p target inverts exactly
    rng = np.random.default_rng(1)
    for _ in range(100):
        s, t = rng.normal(size=2)
        m = (t - s) / (abs(s) + 0.02)
        o = oracle.decode(np.array([0, 0, 0, 0, s]), np.array([0, 0, 0, 0, m]))
        assert abs(o[4] - t) < 1e-12 * max(1.0, abs(t))
    assert oracle.decode(np.zeros(5), np.array([0, 0, -math.pi, 0, 0]))[2] == -math.pi
    assert oracle.decode(np.zeros(5), np.array([0, 0, math.pi, 0, 0]))[2] == -math.pi


@pytest.mark.parametrize("n_layers,d", [(1, 4), (2, 8)])
def test_end_states_match_brute_force(n_layers, d):
    w = ts.Workload("pin", 97, n_layers=n_layers, d_model=d, dtype="fp32", n_tracks=6,
                    len_min=1, len_max=9, n_det_layers=10)
    blob = ts.make_weights(w)
    hits, offs = ts.make_tracks(w)
    st = oracle.track_states(hits, offs, blob, n_layers, d)
    for i in range(6):
        ref = np.empty(2 * d)
        bruteforce.track_forward(hits[offs[i]:offs[i + 1]], blob, n_layers, d, states_out=ref)
        assert np.allclose(st[i], ref, rtol=1e-12, atol=1e-12)
        # length 1: the forward and reverse states coincide at the one hit
        if offs[i + 1] - offs[i] == 1:
            assert np.allclose(st[i, :d], st[i, d:], rtol=0, atol=1e-15)


def test_readout_matches_brute_force():
    for name in ("tiny_d32_fp32", "deploy_d128x4_bf16_8m"):
        w = ts.WORKLOADS[name]
        d = w.d_model
        hb = ts.make_readout_weights(w)
        assert hb.size == oracle.readout_blob_size(d)
        rng = np.random.default_rng(2)
        z = rng.normal(size=(20, 2 * d))
        seeds = np.stack([rng.normal(0, 0.1, 20), rng.normal(0, 1, 20), rng.uniform(-3, 3, 20),
                          rng.uniform(0.5, 2.6, 20), rng.uniform(-1, 1, 20)], 1)
        q, out = oracle.readout_tracks(z, seeds, hb, d)
        for i in range(20):
            rq, ro = bruteforce.readout(z[i], seeds[i], hb, d)
            assert np.allclose(q[i], rq, rtol=1e-12, atol=1e-12)
            assert np.allclose(out[i], ro, rtol=1e-12, atol=1e-12)


def test_readout_is_scale_free_in_the_states():
    """RMSNorm makes the head blind to the scale of the states (up to eps)."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hb = ts.make_readout_weights(w)
    rng = np.random.default_rng(4)
    z = rng.normal(size=(5, 256))
    s = np.zeros((5, 5))
    q1, _ = oracle.readout_tracks(z, s, hb, 128)
    q2, _ = oracle.readout_tracks(1e3 * z, s, hb, 128)
    assert np.allclose(q1, q2, rtol=1e-6, atol=1e-6)


def test_empty_tracks_give_nan_states_and_outputs():
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    blob = ts.make_weights(w)
    hits, offs = ts.make_tracks(w, n_tracks=4)
    offs = np.array([0, offs[1], offs[1], offs[2]], dtype=np.int32)  # track 1 is empty
    st = oracle.track_states(hits, offs, blob, w.n_layers, w.d_model)
    assert np.all(np.isnan(st[1])) and not np.isnan(st[[0, 2]]).any()
    q, out = oracle.readout_tracks(st, np.zeros((3, 5)), ts.make_readout_weights(w), w.d_model)
    assert np.all(np.isnan(out[1])) and not np.isnan(out[[0, 2]]).any()
