"""Pins of the fp64 CPU oracle against closed forms, invariants, library
routines and an independent brute-force restatement (no GPU needed).

Each test names the passage of the paper it pins: Eq. (2) (the gated update),
Sec. Encoder (bidirectional scans, RMSNorm, the head), Sec. Kernel adaptation
(packed, unpadded batches; tracks are independent).
"""
import dataclasses

import numpy as np
import pytest
from scipy.special import expit

import oracle
import tracksynth as ts
from tests import bruteforce as bf

RNG = np.random.default_rng(12345)


def _rand_xa(L, d, rng=RNG):
    x = rng.normal(size=(L, d))
    a = expit(rng.normal(size=(L, d)) * 2.0)
    return x, a


# --------------------------------------------------------------------------
# Eq. (2): the scan alone
# --------------------------------------------------------------------------

@pytest.mark.parametrize("a0", [0.05, 0.3, 0.5, 0.9])
def test_scan_constant_gate_constant_input_closed_form(a0):
    """Constant a and x: h_t = x (1 - (1-a)^t) forward, x (1 - (1-a)^(L-t+1)) backward."""
    L, d = 17, 3
    x0 = np.array([1.5, -0.25, 3.0])
    x = np.tile(x0, (L, 1))
    a = np.full((L, d), a0)
    t = np.arange(1, L + 1)[:, None]
    f_ref = x0 * (1.0 - (1.0 - a0) ** t)
    b_ref = x0 * (1.0 - (1.0 - a0) ** (L - t + 1))
    np.testing.assert_allclose(oracle.scan_forward(x, a), f_ref, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(oracle.scan_backward(x, a), b_ref, rtol=1e-14, atol=1e-14)


def test_scan_constant_gate_geometric_sum():
    """Constant a, any x: f_t = a sum_{k<=t} (1-a)^(t-k) x_k (a geometric-weighted sum)."""
    L, d, a0 = 12, 4, 0.37
    x = RNG.normal(size=(L, d))
    a = np.full((L, d), a0)
    f_ref = np.zeros((L, d))
    for t in range(L):
        w = a0 * (1.0 - a0) ** (t - np.arange(t + 1))
        f_ref[t] = w @ x[: t + 1]
    np.testing.assert_allclose(oracle.scan_forward(x, a), f_ref, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("L", [1, 2, 7, 30])
def test_scan_backward_is_forward_of_reversed(L):
    """The reverse scan is the same scan over the reversed sequence (bitwise)."""
    x, a = _rand_xa(L, 5)
    b = oracle.scan_backward(x, a)
    f_rev = oracle.scan_forward(x[::-1], a[::-1])[::-1]
    assert np.array_equal(b, f_rev)


@pytest.mark.parametrize("L", [1, 2, 3, 5, 8])
def test_scan_matches_matrix_form(L):
    """Brute force: f = M_f x, b = M_b x with explicit products of (1 - a)."""
    x, a = _rand_xa(L, 4)
    f_ref, b_ref = bf.bidir_scan(x, a)
    np.testing.assert_allclose(oracle.scan_forward(x, a), f_ref, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(oracle.scan_backward(x, a), b_ref, rtol=1e-12, atol=1e-14)


def test_scan_gate_one_and_zero():
    """a = 1 copies the input; a = 0 holds the zero initial state."""
    x, _ = _rand_xa(9, 3)
    # h + 1 * (x - h) equals x up to the rounding of the subtraction and the add,
    # which is relative to the previous state, so the bound is absolute
    np.testing.assert_allclose(oracle.scan_forward(x, np.ones_like(x)), x, rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.scan_backward(x, np.ones_like(x)), x, rtol=0, atol=1e-15)
    assert np.all(oracle.scan_forward(x, np.zeros_like(x)) == 0.0)


def test_scan_length_one():
    """L = 1: both directions give a_1 x_1."""
    x, a = _rand_xa(1, 6)
    np.testing.assert_array_equal(oracle.scan_forward(x, a), a * x)
    np.testing.assert_array_equal(oracle.scan_backward(x, a), a * x)


# --------------------------------------------------------------------------
# Library routines: linear, RMSNorm, sigmoid, SiLU
# --------------------------------------------------------------------------

def test_linear_matches_numpy():
    W = RNG.normal(size=(7, 5))
    b = RNG.normal(size=7)
    x = RNG.normal(size=(4, 5))
    np.testing.assert_allclose(oracle.linear(W, b, x), x @ W.T + b, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(oracle.linear(W, None, x), x @ W.T, rtol=1e-14, atol=1e-14)


def test_rmsnorm_matches_numpy_norm():
    r = RNG.normal(size=(6, 16)) * 3.0
    g = RNG.uniform(0.5, 1.5, 16)
    eps = 1e-6
    ref = r / np.sqrt((np.linalg.norm(r, axis=1, keepdims=True) ** 2) / 16 + eps) * g
    np.testing.assert_allclose(oracle.rmsnorm(r, g, eps), ref, rtol=1e-13)
    # unit gain, eps=0: every row has root-mean-square exactly 1
    y = oracle.rmsnorm(r, np.ones(16), 0.0)
    np.testing.assert_allclose(np.sqrt((y ** 2).mean(axis=1)), 1.0, rtol=1e-14)


def test_sigmoid_silu_values():
    assert oracle.sigmoid(0.0) == 0.5
    for v in [-30.0, -2.5, -0.1, 0.7, 4.0, 30.0]:
        assert abs(oracle.sigmoid(v) - expit(v)) < 1e-16
        assert abs(oracle.sigmoid(v) + oracle.sigmoid(-v) - 1.0) < 1e-15
        assert abs(oracle.silu(v) - v * expit(v)) <= 1e-15 * max(1.0, abs(v))
    assert oracle.silu(0.0) == 0.0


# --------------------------------------------------------------------------
# The whole model
# --------------------------------------------------------------------------

def _tiny_model(n_layers, d, seed):
    return ts.make_weights(n_layers=n_layers, d=d, dtype="fp32", seed=seed)


def _helix_track(L, seed=7):
    """The innermost L hits of one 30-layer helix track."""
    w = dataclasses.replace(ts.workload("d256x6_bf16_1m"), len_min=30, len_max=30)
    hits, lengths, _ = ts.make_track_chunk(w, 0, 1, seed=seed)
    return hits[:L]


@pytest.mark.parametrize("n_layers,d,L", [(1, 4, 1), (1, 4, 5), (2, 4, 8), (2, 8, 3), (1, 8, 2)])
def test_model_matches_bruteforce(n_layers, d, L):
    """Whole model vs the independent matrix-form restatement, fp64."""
    blob = _tiny_model(n_layers, d, seed=100 + L)
    hits = _helix_track(L)
    out, pooled, resid = oracle.track_forward(hits, blob, n_layers, d)
    out_bf, pooled_bf, resid_bf = bf.track_forward(hits, blob, n_layers, d)
    np.testing.assert_allclose(resid, resid_bf, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(pooled, pooled_bf, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out, out_bf, rtol=1e-12, atol=1e-12)


def _closed_form_constant_stream(blob, n_layers, d, L, be):
    """Closed form when every hit embeds to the same vector be (embed.W = 0).

    With identical inputs x and gate a at every hit, Eq. (2) gives
    f_t = x (1 - c^t), b_t = x (1 - c^(L-t+1)), c = 1 - a, so the mean over the
    track of either direction is x (1 - S) with the geometric series
    S = (1/L) sum_{t=1..L} c^t = c (1 - c^L) / (L (1 - c)), and the pooled
    vector is be + (W_f + W_b) x (1 - S) + b_out.  After one layer the hits
    differ, so the form is used with a single layer.
    """
    P = ts.split_blob(blob, n_layers, d)
    assert n_layers == 1
    g = P["layer0.norm.g"]
    y = g * be / np.sqrt(np.mean(be ** 2) + 1e-6)
    W, bias = P["layer0.in.W"], P["layer0.in.b"]
    x = W[:d] @ y + bias[:d]
    a = 1.0 / (1.0 + np.exp(-(W[d:2 * d] @ y + bias[d:2 * d])))
    c = 1.0 - a
    S = c * (1.0 - c ** L) / (L * (1.0 - c))
    Wo = P["layer0.out.W"]
    p = be + (Wo[:, :d] + Wo[:, d:]) @ (x * (1.0 - S)) + P["layer0.out.b"]
    h = P["head.W1"] @ p + P["head.b1"]
    h = h / (1.0 + np.exp(-h))
    return P["head.W2"] @ h + P["head.b2"]


@pytest.mark.parametrize("L", [1, 2, 10, 25])
def test_model_constant_embedding_geometric_series(L):
    """embed.W = 0: a one-layer model reduces to a geometric series in c = 1 - a."""
    d = 16
    blob = _tiny_model(1, d, seed=5).copy()
    blob[: d * 3] = 0.0                                   # embed.W
    be = blob[d * 3: d * 4].astype(np.float64)            # embed.b
    hits = _helix_track(L)
    out, _, _ = oracle.track_forward(hits, blob, 1, d)
    ref = _closed_form_constant_stream(blob, 1, d, L, be)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_model_length_one_closed_form():
    """L = 1: f_1 = b_1 = a_1 x_1, so one layer is an explicit composition of maps."""
    d = 8
    blob = _tiny_model(1, d, seed=9)
    P = ts.split_blob(blob, 1, d)
    hit = _helix_track(1).astype(np.float64)[0]
    u = (hit - np.array([-1000.0, -1000.0, -3000.0])) / np.array([2000.0, 2000.0, 6000.0])
    r = P["embed.W"] @ u + P["embed.b"]
    y = P["layer0.norm.g"] * r / np.sqrt(np.mean(r ** 2) + 1e-6)
    z = P["layer0.in.W"] @ y + P["layer0.in.b"]
    ax = expit(z[d:2 * d]) * z[:d]
    r = r + P["layer0.out.W"] @ np.concatenate([ax, ax]) + P["layer0.out.b"]
    h = P["head.W1"] @ r + P["head.b1"]
    ref = P["head.W2"] @ (h * expit(h)) + P["head.b2"]
    out, _, _ = oracle.track_forward(hit[None, :].astype(np.float32), blob, 1, d)
    np.testing.assert_allclose(out, ref, rtol=1e-13, atol=1e-14)


def test_model_identity_layers():
    """out.W = 0 and out.b = 0 make every layer the identity: out = head(mean(embed))."""
    n_layers, d, L = 3, 8, 6
    blob = _tiny_model(n_layers, d, seed=11).copy()
    o = 4 * d
    for _ in range(n_layers):
        o += d + 3 * d * d + 3 * d
        blob[o: o + d * 2 * d + d] = 0.0
        o += d * 2 * d + d
    P = ts.split_blob(blob, n_layers, d)
    hits = _helix_track(L).astype(np.float64)
    u = (hits - np.array([-1000.0, -1000.0, -3000.0])) / np.array([2000.0, 2000.0, 6000.0])
    p = (u @ P["embed.W"].T + P["embed.b"]).mean(axis=0)
    h = P["head.W1"] @ p + P["head.b1"]
    ref = P["head.W2"] @ (h * expit(h)) + P["head.b2"]
    out, _, _ = oracle.track_forward(hits.astype(np.float32), blob, n_layers, d)
    np.testing.assert_allclose(out, ref, rtol=1e-13, atol=1e-14)


def test_model_gate_one_is_order_free():
    """a = 1 everywhere makes each layer act hit by hit, so the output does not
    depend on the order of the hits within a track."""
    n_layers, d, L = 2, 8, 9
    blob = _tiny_model(n_layers, d, seed=13).copy()
    o = 4 * d
    for _ in range(n_layers):
        inW = o + d
        blob[inW + d * d: inW + 2 * d * d] = 0.0           # gate rows of in.W
        inb = inW + 3 * d * d
        blob[inb + d: inb + 2 * d] = 60.0                 # sigmoid(60) == 1.0 in fp64
        o += d + 3 * d * d + 3 * d + d * 2 * d + d
    hits = _helix_track(L)
    out, _, _ = oracle.track_forward(hits, blob, n_layers, d)
    perm = np.random.default_rng(3).permutation(L)
    out_p, _, _ = oracle.track_forward(hits[perm], blob, n_layers, d)
    np.testing.assert_allclose(out_p, out, rtol=1e-13, atol=1e-14)
    # ... while with the drawn gates the order matters
    blob0 = _tiny_model(n_layers, d, seed=13)
    a, _, _ = oracle.track_forward(hits, blob0, n_layers, d)
    b, _, _ = oracle.track_forward(hits[perm], blob0, n_layers, d)
    assert np.max(np.abs(a - b)) > 1e-6


def test_batch_packing_invariances():
    """Sec. Kernel adaptation: packed batches of independent tracks.  Permuting
    tracks permutes outputs, duplicating a track duplicates its output, and
    moving the packed rows (offsets base) changes nothing, all bitwise."""
    w = ts.workload("d128x4_fp32_65k")
    d, n_layers = 16, 2
    blob = _tiny_model(n_layers, d, seed=17)
    hits, offs = ts.make_tracks(w, n_tracks=40)
    out = oracle.fit_tracks(hits, offs, blob, n_layers, d, n_threads=4)
    L = np.diff(offs)
    # permutation
    perm = np.random.default_rng(1).permutation(40)
    hp = np.concatenate([hits[offs[i]:offs[i + 1]] for i in perm])
    op = np.concatenate([[0], np.cumsum(L[perm])]).astype(np.int32)
    assert np.array_equal(oracle.fit_tracks(hp, op, blob, n_layers, d), out[perm])
    # duplication
    idx = np.array([3, 3, 7, 3])
    hd = np.concatenate([hits[offs[i]:offs[i + 1]] for i in idx])
    od = np.concatenate([[0], np.cumsum(L[idx])]).astype(np.int32)
    assert np.array_equal(oracle.fit_tracks(hd, od, blob, n_layers, d), out[idx])
    # offsets base: prepend junk rows
    junk = np.full((13, 3), 777.0, np.float32)
    hj = np.concatenate([junk, hits])
    assert np.array_equal(oracle.fit_tracks(hj, offs + 13, blob, n_layers, d), out)
    # single track alone equals its batch row
    one, _, _ = oracle.track_forward(hits[offs[5]:offs[6]], blob, n_layers, d)
    assert np.array_equal(one, out[5])


def test_zero_length_track_is_nan():
    d = 8
    blob = _tiny_model(1, d, seed=19)
    hits = _helix_track(4)
    offs = np.array([0, 2, 2, 4], np.int32)
    out = oracle.fit_tracks(hits, offs, blob, 1, d)
    assert np.all(np.isnan(out[1])) and np.all(np.isfinite(out[[0, 2]]))


def test_blob_sizes():
    assert oracle.blob_size(1, 32) == ts.blob_size(1, 32) == 6629
    assert oracle.blob_size(4, 128) == ts.blob_size(4, 128) == 347909
    assert oracle.blob_size(6, 256) == ts.blob_size(6, 256) == 2041861
