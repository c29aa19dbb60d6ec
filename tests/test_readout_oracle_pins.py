"""Pins of the fp64 oracle of the paper's readout and decode (Sec. Encoder,
last paragraph: end states -> RMSNorm -> two-layer head of hidden width 128 ->
35 quantiles; Sec. Losses: the median quantile as point estimate,
seed-anchored targets): closed forms of small heads whose hidden width
differs from the state width, the point estimate picked by position,
invariances, and the end states against the brute-force matrix form of the
scans.  (The comparison with a numpy restatement of the head is a
cross-check, not a pin.)
"""
import math

import numpy as np
import pytest

import oracle
import tracksynth as ts
from tests import bruteforce


def test_paper_head_shape_and_size():
    """The paper's head reads the 384-wide end states (two directions of hidden
    width 192) through 128 hidden units into 35 outputs (Sec. Encoder)."""
    w = ts.MINGRU_WORKLOADS["mingru2_h192_fourier15_deploy_bf16_8m"]
    assert ts.readout_dims(w) == (192, 128)
    n = 2 * 192 + 128 * 384 + 128 + 35 * 128 + 35
    assert oracle.readout_blob_size(192, 128) == n == ts.make_readout_weights(w).size


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
    for w in (ts.WORKLOADS["tiny_d32_fp32"], ts.WORKLOADS["deploy_d128x4_bf16_8m"],
              ts.MINGRU_WORKLOADS["mingru2_h192_fourier15_deploy_bf16_8m"]):
        d, nh = ts.readout_dims(w)
        hb = ts.make_readout_weights(w)
        assert hb.size == oracle.readout_blob_size(d, nh)
        rng = np.random.default_rng(2)
        z = rng.normal(size=(20, 2 * d))
        seeds = np.stack([rng.normal(0, 0.1, 20), rng.normal(0, 1, 20), rng.uniform(-3, 3, 20),
                          rng.uniform(0.5, 2.6, 20), rng.uniform(-1, 1, 20)], 1)
        q, out = oracle.readout_tracks(z, seeds, hb, d, nh)
        for i in range(20):
            rq, ro = bruteforce.readout(z[i], seeds[i], hb, d, nh)
            assert np.allclose(q[i], rq, rtol=1e-12, atol=1e-12)
            assert np.allclose(out[i], ro, rtol=1e-12, atol=1e-12)


def test_readout_is_scale_free_in_the_states():
    """RMSNorm makes the head blind to the scale of the states (up to eps)."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hb = ts.make_readout_weights(w)
    rng = np.random.default_rng(4)
    z = rng.normal(size=(5, 256))
    s = np.zeros((5, 5))
    q1, _ = oracle.readout_tracks(z, s, hb, 128, 128)
    q2, _ = oracle.readout_tracks(1e3 * z, s, hb, 128, 128)
    assert np.allclose(q1, q2, rtol=1e-6, atol=1e-6)


def test_empty_tracks_give_nan_states_and_outputs():
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    blob = ts.make_weights(w)
    hits, offs = ts.make_tracks(w, n_tracks=4)
    offs = np.array([0, offs[1], offs[1], offs[2]], dtype=np.int32)  # track 1 is empty
    st = oracle.track_states(hits, offs, blob, w.n_layers, w.d_model)
    assert np.all(np.isnan(st[1])) and not np.isnan(st[[0, 2]]).any()
    q, out = oracle.readout_tracks(st, np.zeros((3, 5)), ts.make_readout_weights(w), *ts.readout_dims(w))
    assert np.all(np.isnan(out[1])) and not np.isnan(out[[0, 2]]).any()


def _head(g, W1, b1, W2, b2):
    return np.concatenate([np.ravel(g), np.ravel(W1), np.ravel(b1), np.ravel(W2), np.ravel(b2)]).astype(np.float32)


def test_zero_head_gives_the_bias_and_the_middle_quantile_is_the_estimate():
    """W1 = 0, b1 = 0: the hidden layer is SiLU(0) = 0, so q = b2 whatever the
    states.  Outputs 7p .. 7p+6 are parameter p's quantiles; the point
    estimate is the median quantile, the fourth of the seven (level 1/2), which
    is what gets added to the seed, not the median of the seven values: they
    are planted so that the two differ (output 3 holds 2.0 + 10 p, the
    sorted middle is 1.0 + 10 p)."""
    d, nh = 3, 5
    b2 = np.zeros(35)
    for p in range(5):
        b2[7 * p:7 * p + 7] = np.array([9.0, -3.0, 0.5, 2.0, -7.0, 4.0, 1.0]) + 10.0 * p
    hb = _head(np.ones(2 * d), np.zeros((nh, 2 * d)), np.zeros(nh), np.ones((35, nh)), b2)
    z = np.random.default_rng(5).normal(size=(4, 2 * d))
    seeds = np.array([[0.1, 0.2, 0.3, 0.4, 0.5]] * 4)
    q, out = oracle.readout_tracks(z, seeds, hb, d, nh)
    assert np.array_equal(q, np.tile(b2, (4, 1)))
    exp = [0.1 + 2.0, 0.2 + 12.0, (0.3 + 22.0 + math.pi) % (2 * math.pi) - math.pi, 0.4 + 32.0,
           0.5 + 42.0 * (0.5 + 0.02)]
    assert np.allclose(out, np.tile(exp, (4, 1)), rtol=0, atol=1e-12)
    # moving the other six outputs of a parameter leaves its estimate alone
    b2s = b2.copy()
    b2s[[0, 1, 2, 4, 5, 6]] = [100.0, -100.0, 50.0, 3.0, 3.0, 3.0]
    hb = _head(np.ones(2 * d), np.zeros((nh, 2 * d)), np.zeros(nh), np.ones((35, nh)), b2s)
    _, out2 = oracle.readout_tracks(z, seeds, hb, d, nh)
    assert np.array_equal(out2, out)


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
        hb = _head(g, np.array([W1]), [0.0], W2, b2)
        q, out = oracle.readout_tracks(np.array([[3.0, 4.0]]), np.zeros((1, 5)), hb, 1, 1)
        expect = np.full(35, 0.25)
        expect[3] = 0.25 - 2.0 * silu(pre)
        assert np.allclose(q[0], expect, rtol=1e-14, atol=1e-14), (g, W1)
        assert abs(out[0, 0] - expect[3]) < 1e-14   # output 3 is d0's estimate


def test_hidden_width_other_than_the_state_width_in_closed_form():
    """d = 1 (z = (3, 4), y = g z / sqrt(12.5 + 1e-6)) with three hidden units:
    unit 0 reads y_0, unit 1 reads y_1, unit 2 reads y_0 - y_1 with bias 0.5.
    W2 row 10 (z0's estimate, output 7 + 3) adds units 0 and 2, row 24 (theta's,
    7 * 3 + 3) takes 3 x unit 1.  A head built as if the hidden width were
    the state width 1, or 2 d = 2, would read the wrong rows and fail."""
    s = 1.0 / math.sqrt(12.5 + 1e-6)
    g = (2.0, 0.5)
    y = (g[0] * 3.0 * s, g[1] * 4.0 * s)
    W1 = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, -1.0]])
    b1 = np.array([0.0, 0.0, 0.5])
    W2 = np.zeros((35, 3))
    W2[10, 0] = W2[10, 2] = 1.0
    W2[24, 1] = 3.0
    b2 = np.zeros(35)
    hb = _head(g, W1, b1, W2, b2)
    assert hb.size == oracle.readout_blob_size(1, 3)
    silu = lambda x: x / (1.0 + math.exp(-x))
    h = (silu(y[0]), silu(y[1]), silu(y[0] - y[1] + 0.5))
    q, out = oracle.readout_tracks(np.array([[3.0, 4.0]]), np.zeros((1, 5)), hb, 1, 3)
    expect = np.zeros(35)
    expect[10] = h[0] + h[2]
    expect[24] = 3.0 * h[1]
    assert np.allclose(q[0], expect, rtol=1e-14, atol=1e-15)
    assert abs(out[0, 1] - expect[10]) < 1e-14 and abs(out[0, 3] - expect[24]) < 1e-14


def test_head_matrices_are_row_major_out_by_in():
    """d = 2 with three hidden units: a single weight W1[2][3] = 1 makes hidden
    unit 2 read z_3 only; a single W2[20][2] = 1 sends unit 2 to output 20 only.
    A transposed read of either matrix would move the response to another
    output or input."""
    d, nh = 2, 3
    W1 = np.zeros((nh, 2 * d))
    W1[2, 3] = 1.0
    W2 = np.zeros((35, nh))
    W2[20, 2] = 1.0
    hb = _head(np.ones(2 * d), W1, np.zeros(nh), W2, np.zeros(35))
    rng = np.random.default_rng(6)
    z = rng.normal(size=(6, 2 * d))
    q, _ = oracle.readout_tracks(z, np.zeros((6, 5)), hb, d, nh)
    nz = np.nonzero(np.any(q != 0.0, axis=0))[0]
    assert list(nz) == [20]
    # only z_3 (after the norm) drives it: changing z_0, z_1, z_2 at fixed rms does not
    z2 = z.copy()
    z2[:, [0, 1, 2]] = z[:, [1, 2, 0]]   # a permutation keeps mean(z^2)
    q2, _ = oracle.readout_tracks(z2, np.zeros((6, 5)), hb, d, nh)
    assert np.allclose(q2, q, rtol=1e-14, atol=0)   # the sum of squares is summed in another order
