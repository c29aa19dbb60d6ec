"""Pins of the fp64 oracle of the paper's readout and decode (Sec. Encoder,
last paragraph: end states -> RMSNorm -> two-layer head -> 35 quantiles;
Sec. Losses: median point estimate, seed-anchored targets): closed forms of
small heads, the median against numpy's, invariances, and the end states
against the brute-force matrix form of the scans.  (The comparison with a
numpy restatement of the head is a cross-check, not a pin.)
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


def _head(d, g, W1, b1, W2, b2):
    return np.concatenate([np.ravel(g), np.ravel(W1), np.ravel(b1), np.ravel(W2), np.ravel(b2)]).astype(np.float32)


def test_zero_head_gives_the_bias_and_medians_group_by_parameter():
    """W1 = 0, b1 = 0: the hidden layer is SiLU(0) = 0, so q = b2 whatever the
    states; outputs 7p .. 7p+6 are parameter p's quantiles, planted out of
    order, and each parameter's median is added to its own seed entry."""
    d = 3
    b2 = np.zeros(35)
    for p in range(5):
        b2[7 * p:7 * p + 7] = np.array([9.0, -3.0, 0.5, 2.0, -7.0, 4.0, 1.0]) + 10.0 * p   # median 1 + 10 p
    hb = _head(d, np.ones(2 * d), np.zeros((d, 2 * d)), np.zeros(d), np.ones((35, d)), b2)
    z = np.random.default_rng(5).normal(size=(4, 2 * d))
    seeds = np.array([[0.1, 0.2, 0.3, 0.4, 0.5]] * 4)
    q, out = oracle.readout_tracks(z, seeds, hb, d)
    assert np.array_equal(q, np.tile(b2, (4, 1)))
    exp = [0.1 + 1.0, 0.2 + 11.0, (0.3 + 21.0 + math.pi) % (2 * math.pi) - math.pi, 0.4 + 31.0,
           0.5 + 41.0 * (0.5 + 0.02)]
    assert np.allclose(out, np.tile(exp, (4, 1)), rtol=0, atol=1e-12)


def test_one_unit_head_in_closed_form():
    """d = 1, z = (3, 4): mean(z^2) = 12.5 over the 2d = 2 entries.  A head that
    reads only z_0 (W1 = (1, 0)) with gain 2 gives pre-activation
    6 / sqrt(12.5 + 1e-6); W1 = (0, 1) with gain 1 reads 4 / sqrt(12.5 + 1e-6).
    W2 sends the hidden unit to output 3 only, with weight -2, b2 = 0.25."""
    W2 = np.zeros((35, 1))
    W2[3, 0] = -2.0
    b2 = np.full(35, 0.25)
    silu = lambda x: x / (1.0 + math.exp(-x))
    for g, W1, pre in (((2.0, 1.0), (1.0, 0.0), 6.0 / math.sqrt(12.5 + 1e-6)),
                       ((1.0, 1.0), (0.0, 1.0), 4.0 / math.sqrt(12.5 + 1e-6)),
                       ((1.0, 3.0), (0.0, 1.0), 12.0 / math.sqrt(12.5 + 1e-6))):
        hb = _head(1, g, np.array([W1]), [0.0], W2, b2)
        q, _ = oracle.readout_tracks(np.array([[3.0, 4.0]]), np.zeros((1, 5)), hb, 1)
        expect = np.full(35, 0.25)
        expect[3] = 0.25 - 2.0 * silu(pre)
        assert np.allclose(q[0], expect, rtol=1e-14, atol=1e-14), (g, W1)


def test_head_matrices_are_row_major_out_by_in():
    """d = 2: a single weight W1[1][2] = 1 makes hidden unit 1 read z_2 only; a
    single W2[20][1] = 1 sends unit 1 to output 20 only.  A transposed read of
    either matrix would move the response to another output or input."""
    d = 2
    W1 = np.zeros((d, 2 * d))
    W1[1, 2] = 1.0
    W2 = np.zeros((35, d))
    W2[20, 1] = 1.0
    hb = _head(d, np.ones(2 * d), W1, np.zeros(d), W2, np.zeros(35))
    rng = np.random.default_rng(6)
    z = rng.normal(size=(6, 2 * d))
    q, _ = oracle.readout_tracks(z, np.zeros((6, 5)), hb, d)
    nz = np.nonzero(np.any(q != 0.0, axis=0))[0]
    assert list(nz) == [20]
    # only z_2 (after the norm) drives it: changing z_0, z_1, z_3 at fixed rms does not
    z2 = z.copy()
    z2[:, [0, 1, 3]] = z[:, [1, 3, 0]]   # a permutation keeps mean(z^2)
    q2, _ = oracle.readout_tracks(z2, np.zeros((6, 5)), hb, d)
    assert np.array_equal(q2, q)
