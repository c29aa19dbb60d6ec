"""GPU parity of the paper's readout path against the fp64 oracle, element by
element: the encoder's last-layer end states (fit_tracks_states), the readout
head with its point estimates and seed-anchored decode (tf_decode_tracks) on the
oracle's own states, and the chain seed -> states -> decode end to end, plus
the edge cases (length 1 and maximum, ragged batches, rejected tracks, NaN
inputs, tile independence).
"""
import dataclasses
import os

import numpy as np
import pytest

import oracle
import tracksynth as ts
from tests.parity import TOL

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

THREADS = int(os.environ.get("ORACLE_THREADS", "0"))
N_STATES = {"tiny_d32_fp32": 256, "d128x4_fp32_65k": 2048, "d256x6_bf16_1m": 512,
            "long64_d128x4_bf16_200k": 512, "deploy_d128x4_bf16_8m": 2048}
# The head and the decode run in fp32 on fp32 states; against the fp64 oracle
# on the same (fp32-valued) states the differences are fp32 roundings.  A
# quantile is the end of two dot products (2d terms, then nh, the hidden
# width), so its rounding is bounded by about u * (2d + nh) relative to the sum
# of the terms' magnitudes (u = 2^-24), which for these random heads is a few
# times the column's scale: the quantiles are held to u * (2d + nh) * 4/3 per
# column.  The decoded parameters are
# held to the fp32 model's output tolerance.
DECODE_TOL = 1e-5


def quantile_tol(d, nh):
    return 2.0 ** -24 * (2 * d + nh) * 4 / 3


# The 16-bit head takes W1 and W2 in bf16 and keeps the activations to ~16
# bits; it is held to the bf16 model's output tolerance.  Its weights are
# bf16 values, as a bf16 model's are (an fp32 model's head blob is rounded
# to bf16 first, for the oracle as well, so that both sides see the same
# weights: `head_blob`).
def head_blob(w, mode, **kw):
    """The workload's readout head blob, rounded to bf16 values for a 16-bit head."""
    hb = ts.make_readout_weights(w, **kw)
    return hb if mode == "fp32" else ts.round_to_bf16(hb)


def head_tols(mode, d, nh):
    """(quantile, decoded) tolerances of a head of this number type."""
    if mode == "fp32":
        return quantile_tol(d, nh), DECODE_TOL
    return TOL["bf16"], TOL["bf16"]


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32479_amd as tf
    return tf


def colerr(g, r, rms=None):
    """Per column: max |g - r| / max(|r|, rms of the column); NaN patterns must
    match.  rms: column scales of a larger sample, for a batch of few tracks."""
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    assert g.shape == r.shape
    assert np.array_equal(np.isnan(g), np.isnan(r))
    ok = ~np.isnan(r).any(axis=1)
    g, r = g[ok], r[ok]
    if r.shape[0] == 0:
        return np.zeros(r.shape[1])
    if rms is None:
        rms = np.sqrt(np.mean(r ** 2, axis=0))
    return np.max(np.abs(g - r) / np.maximum(np.abs(r), np.maximum(rms, 1e-300)), axis=0)


def state_err(g, r):
    """Largest |g - r| over a track's 2d end states, in units of that track's
    state RMS: the scale the readout's RMSNorm divides by, hence the error
    that reaches the head.  NaN rows must match."""
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    assert g.shape == r.shape
    assert np.array_equal(np.isnan(g), np.isnan(r))
    ok = ~np.isnan(r).any(axis=1)
    g, r = g[ok], r[ok]
    if r.shape[0] == 0:
        return 0.0
    rms = np.sqrt(np.mean(r ** 2, axis=1, keepdims=True))
    return float(np.max(np.abs(g - r) / rms))


def wrap_phi(g, r):
    """phi of g brought to the branch of r (2 pi apart is the same angle)."""
    g = np.array(g, dtype=np.float64)
    d = g[:, 2] - r[:, 2]
    g[:, 2] -= np.round(np.nan_to_num(d) / (2 * np.pi)) * 2 * np.pi
    return g


def _weights(tf, w, max_hits=None):
    blob = ts.make_weights(w)
    W = tf.Weights(blob, w.n_layers, w.d_model, tf.MODE_FOR_WEIGHTS[w.dtype],
                   w.len_max if max_hits is None else max_hits)
    return W, blob


def _states(tf, W, hits, offs, n_tracks=None):
    h = torch.from_numpy(np.ascontiguousarray(hits, dtype=np.float32)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(offs, dtype=np.int32)).cuda()
    s = tf.fit_tracks_states(h, o, W, n_tracks=n_tracks)
    torch.cuda.synchronize()
    return s.cpu().numpy()


def _ref_states(w, hits, offs, blob):
    return oracle.track_states(hits, offs, blob, w.n_layers, w.d_model, n_threads=THREADS)


@pytest.mark.parametrize("name", list(ts.WORKLOADS))
def test_states_match_oracle(tf, name):
    w = ts.WORKLOADS[name]
    print(f"[states] {name} n={N_STATES[name]}", flush=True)
    W, blob = _weights(tf, w)
    hits, offs = ts.make_tracks(w, n_tracks=N_STATES[name])
    g = _states(tf, W, hits, offs)
    r = _ref_states(w, hits, offs, blob)
    assert g.shape == (N_STATES[name], 2 * w.d_model)
    e = state_err(g, r)
    print(f"[states] {name}: max err {e:.3g} of the track's state rms", flush=True)
    assert e <= TOL[w.dtype]
    assert tf.device_error(W) == 0


@pytest.mark.parametrize("name,L,max_hits", [("deploy_d128x4_bf16_8m", 1, 32), ("deploy_d128x4_bf16_8m", 32, 32),
                                             ("deploy_d128x4_bf16_8m", 64, 64), ("d128x4_fp32_65k", 1, 64),
                                             ("d128x4_fp32_65k", 64, 64), ("tiny_d32_fp32", 64, 64),
                                             ("d256x6_bf16_1m", 32, 32)])
def test_states_fixed_lengths(tf, name, L, max_hits):
    """Length 1 (forward and reverse state of one step coincide) and the maximum."""
    w = dataclasses.replace(ts.WORKLOADS[name], len_min=L, len_max=L, n_det_layers=max(L, 8))
    print(f"[states-fixed] {name} L={L} max_hits={max_hits}", flush=True)
    W, blob = _weights(tf, w, max_hits=max_hits)
    hits, offs = ts.make_tracks(w, n_tracks=300)
    g = _states(tf, W, hits, offs)
    r = _ref_states(w, hits, offs, blob)
    assert state_err(g, r) <= TOL[w.dtype]
    if L == 1:
        d = w.d_model
        assert np.array_equal(g[:, :d], g[:, d:])


@pytest.mark.parametrize("name,max_hits", [("deploy_d128x4_bf16_8m", 32), ("deploy_d128x4_bf16_8m", 64),
                                           ("d128x4_fp32_65k", 64)])
def test_states_ragged_small_batches_and_bad_tracks(tf, name, max_hits):
    w0 = ts.WORKLOADS[name]
    print(f"[states-ragged] {name} max_hits={max_hits}", flush=True)
    W, blob = _weights(tf, w0, max_hits=max_hits)
    w = dataclasses.replace(w0, len_min=1, len_max=max_hits, n_det_layers=max_hits)
    hits, offs = ts.make_tracks(w, n_tracks=700)
    r_all = _ref_states(w, hits, offs, blob)
    for n in (1, 2, 33, 700):
        g = _states(tf, W, hits, offs[: n + 1])
        assert state_err(g, r_all[:n]) <= TOL[w.dtype], n
    # track 5 emptied, track 9 one hit too long: NaN rows, neighbours unchanged
    Lk = np.diff(offs)
    Lk[5], Lk[9] = 0, max_hits + 1
    rows = []
    for i in range(700):
        src = np.arange(offs[i], offs[i + 1])
        rows.append(np.resize(src, Lk[i]) if Lk[i] else src[:0])
    h2 = hits[np.concatenate(rows)]
    o2 = np.concatenate([[0], np.cumsum(Lk)]).astype(np.int32)
    g = _states(tf, W, h2, o2)
    assert np.all(np.isnan(g[[5, 9]]))
    good = np.ones(700, bool)
    good[[5, 9]] = False
    assert state_err(g[good], r_all[good]) <= TOL[w.dtype]
    assert tf.device_error(W) == (tf.DEVERR_EMPTY_TRACK | tf.DEVERR_TOO_LONG)


def test_states_do_not_depend_on_tile_neighbours(tf):
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    W, _ = _weights(tf, w)
    hits, offs = ts.make_tracks(w, n_tracks=3000)
    a = _states(tf, W, hits, offs)
    assert np.array_equal(a, _states(tf, W, hits, offs))
    perm = np.random.default_rng(3).permutation(3000)
    L = np.diff(offs)
    hp = np.concatenate([hits[offs[i]:offs[i + 1]] for i in perm])
    op = np.concatenate([[0], np.cumsum(L[perm])]).astype(np.int32)
    assert np.array_equal(_states(tf, W, hp, op), a[perm])


def _decode(tf, R, states, seeds, quantiles=True):
    st = torch.from_numpy(np.ascontiguousarray(states, dtype=np.float32)).cuda()
    sd = torch.from_numpy(np.ascontiguousarray(seeds, dtype=np.float64)).cuda()
    out, q = tf.decode_tracks(st, sd, R, quantiles=quantiles)
    torch.cuda.synchronize()
    return out.cpu().numpy(), (q.cpu().numpy() if q is not None else None)


@pytest.mark.parametrize("name,n,mode,nh", [("deploy_d128x4_bf16_8m", 1000, "bf16", None),
                                            ("deploy_d128x4_bf16_8m", 1000, "fp32", None),
                                            ("tiny_d32_fp32", 77, "fp32", None), ("tiny_d32_fp32", 77, "bf16", None),
                                            ("d256x6_bf16_1m", 300, "bf16", None), ("d256x6_bf16_1m", 300, "fp32", None),
                                            ("d128x4_fp32_65k", 500, "fp32", None),
                                            ("deploy_d128x4_bf16_8m", 1, "bf16", None),
                                            ("deploy_d128x4_bf16_8m", 33, "bf16", None),
                                            ("deploy_d128x4_bf16_8m", 33, "fp32", None),
                                            ("deploy_d128x4_bf16_8m", 500, "bf16", 32),
                                            ("deploy_d128x4_bf16_8m", 500, "fp32", 224),
                                            ("d128x4_fp32_65k", 300, "fp32", 64),
                                            ("d256x6_bf16_1m", 300, "bf16", 256)])
def test_decode_matches_oracle_on_the_same_states(tf, name, n, mode, nh):
    """The oracle's states (rounded to fp32, as the library takes them) and
    seeds in; the 35 quantiles and the decoded parameters compared, for both
    number types of the head, with hidden widths equal to and different from
    the state width (nh: None takes the workload's head, 128 or 96)."""
    w = ts.WORKLOADS[name]
    d, nh0 = ts.readout_dims(w)
    nh = nh0 if nh is None else nh
    print(f"[decode] {name} n={n} head {mode} hidden {nh}", flush=True)
    # column scales from at least 300 tracks, the first n of which are decoded
    hits, offs = ts.make_tracks(w, n_tracks=max(n, 300))
    blob = ts.make_weights(w)
    st = _ref_states(w, hits, offs, blob).astype(np.float32)
    seeds, _, bad = oracle.seed_tracks(hits, offs, w.b_field, features=False)
    assert bad == 0
    hb = head_blob(w, mode, hidden=nh)
    R = tf.Readout(hb, d, nh, mode)
    r_q, r_out = oracle.readout_tracks(st.astype(np.float64), seeds, hb, d, nh)
    rms_q, rms_o = (np.sqrt(np.mean(a ** 2, axis=0)) for a in (r_q, r_out))
    st, seeds, r_q, r_out = st[:n], seeds[:n], r_q[:n], r_out[:n]
    g_out, g_q = _decode(tf, R, st, seeds)
    eq = colerr(g_q, r_q, rms_q)
    eo = colerr(wrap_phi(g_out, r_out), r_out, rms_o)
    print(f"[decode] {name} head {mode}: quantile err {eq.max():.3g} decoded err {eo.max():.3g}", flush=True)
    tq, to = head_tols(mode, d, nh)
    assert eq.max() <= tq and eo.max() <= to
    # without the quantile output the decode is the same, bit for bit
    g2, q2 = _decode(tf, R, st, seeds, quantiles=False)
    assert q2 is None and np.array_equal(g2, g_out)


@pytest.mark.parametrize("mode", ["fp32", "bf16"])
def test_decode_point_estimate_and_decode_rules_on_a_planted_head(tf, mode):
    """A head whose quantiles are known in closed form: W1 = 0 and W2 = 0, so
    q = b2 for every track; the seven values of each parameter are planted
    out of order, and the decode adds the median quantile, output 7p + 3 (not
    the middle of the sorted seven), to the seed.  Hidden width 64, states 64."""
    d, nh = 32, 64
    hb = np.zeros(oracle.readout_blob_size(d, nh), np.float32)
    hb[: 2 * d] = 1.0
    b2 = hb[-35:]
    rng = np.random.default_rng(8)
    meds = np.zeros(5)
    for p in range(5):
        v = np.sort(rng.uniform(-4, 4, 7))
        b2[7 * p:7 * p + 7] = rng.permutation(v)
        if b2[7 * p + 3] == np.sort(b2[7 * p:7 * p + 7])[3]:   # make the two readings differ
            b2[7 * p + 3], b2[7 * p] = b2[7 * p], b2[7 * p + 3]
        meds[p] = float(b2[7 * p + 3])   # as stored (float32)
    R = tf.Readout(hb, d, nh, mode)
    n = 40
    states = rng.normal(size=(n, 2 * d)).astype(np.float32)
    seeds = np.stack([rng.uniform(-1, 1, n), rng.uniform(-50, 50, n), rng.uniform(-np.pi, np.pi, n),
                      rng.uniform(0.2, 2.9, n), rng.uniform(-1, 1, n)], axis=1)
    out, q = _decode(tf, R, states, seeds)
    assert np.array_equal(q, np.tile(b2, (n, 1)))
    exp = seeds.copy()
    exp[:, [0, 1, 3]] += meds[[0, 1, 3]]
    exp[:, 2] = (seeds[:, 2] + meds[2] + np.pi) % (2 * np.pi) - np.pi
    exp[:, 4] = seeds[:, 4] + meds[4] * (np.abs(seeds[:, 4]) + 0.02)
    assert np.all(out[:, 2] >= -np.pi) and np.all(out[:, 2] < np.pi)
    assert np.allclose(out, exp, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mode", ["fp32", "bf16"])
def test_decode_nan_inputs_stay_local(tf, mode):
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    d = w.d_model
    rng = np.random.default_rng(4)
    n = 100
    st = rng.normal(size=(n, 2 * d)).astype(np.float32)
    seeds = np.stack([rng.uniform(-1, 1, n), rng.uniform(-50, 50, n), rng.uniform(-3, 3, n),
                      rng.uniform(0.2, 2.9, n), rng.uniform(-1, 1, n)], axis=1)
    st[7] = np.nan          # a rejected track's states
    seeds[40] = np.nan      # a track without a seed
    nh = ts.readout_dims(w)[1]
    hb = ts.make_readout_weights(w)
    R = tf.Readout(hb, d, nh, mode)
    out, q = _decode(tf, R, st, seeds)
    assert np.all(np.isnan(out[[7, 40]])) and np.all(np.isnan(q[7]))
    assert np.all(np.isfinite(q[40]))
    good = np.ones(n, bool)
    good[[7, 40]] = False
    assert np.all(np.isfinite(out[good]))
    r_q, r_out = oracle.readout_tracks(st[good].astype(np.float64), seeds[good], hb, d, nh)
    tq, to = head_tols(mode, d, nh)
    assert colerr(q[good], r_q).max() <= tq
    assert colerr(wrap_phi(out[good], r_out), r_out).max() <= to


@pytest.mark.parametrize("name", ["deploy_d128x4_bf16_8m", "d128x4_fp32_65k"])
def test_seed_states_decode_end_to_end(tf, name):
    """hits -> (seed, end states) -> readout and decode, all on the GPU, against
    the oracle's chain; the encoder's tolerance carries through the head."""
    w = ts.WORKLOADS[name]
    print(f"[chain] {name}", flush=True)
    W, blob = _weights(tf, w)
    hb = ts.make_readout_weights(w)
    mode = tf.MODE_FOR_WEIGHTS[w.dtype]
    d, nh = ts.readout_dims(w)
    R = tf.Readout(hb, d, nh, mode)
    hits, offs = ts.make_tracks(w, n_tracks=1500)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    seeds, _ = tf.seed_tracks(h, o, w.b_field, features=False)
    states = tf.fit_tracks_states(h, o, W)
    out, q = tf.decode_tracks(states, seeds, R, quantiles=True)
    torch.cuda.synchronize()
    r_seeds, _, _ = oracle.seed_tracks(hits, offs, w.b_field, features=False)
    r_q, r_out = oracle.readout_tracks(_ref_states(w, hits, offs, blob), r_seeds, hb, d, nh)
    eq = colerr(q.cpu().numpy(), r_q)
    eo = colerr(wrap_phi(out.cpu().numpy(), r_out), r_out)
    print(f"[chain] {name}: quantile err {eq.max():.3g} decoded err {eo.max():.3g}", flush=True)
    # the quantiles carry the head's own rounding on top of the encoder's
    tq, _ = head_tols(mode, d, nh)
    assert eq.max() <= max(TOL[w.dtype], tq) and eo.max() <= TOL[w.dtype]


def test_readout_chain_graph_replays_match_eager(tf):
    """The readout path per batch (seed, the encoder's end states, readout and
    decode), captured in one HIP graph over three batches (the last one
    ragged) as the readout benchmark runs it: every replay, with eager work
    and cleared outputs between the replays, gives the eager chain's seeds,
    end states of the last batch and decoded outputs bit for bit."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hits, offs = ts.make_tracks(w, n_tracks=5000)
    n, batch, d = offs.size - 1, 2048, w.d_model
    mode = tf.MODE_FOR_WEIGHTS[w.dtype]
    W = tf.Weights(ts.make_weights(w), w.n_layers, d, mode, max_hits=w.len_max)
    R = tf.Readout(ts.make_readout_weights(w), *ts.readout_dims(w), mode)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    seeds = torch.empty((n, 5), dtype=torch.float64, device="cuda")
    out = torch.empty((n, 5), dtype=torch.float64, device="cuda")
    states = torch.empty((batch, 2 * d), dtype=torch.float32, device="cuda")
    starts = list(range(0, n, batch))

    def step(stream=None):
        for s0 in starts:
            k = min(batch, n - s0)
            tf.seed_tracks(h, o[s0:], w.b_field, features=False, seeds=seeds[s0:], n_tracks=k, stream=stream)
            tf.fit_tracks_states(h, o[s0:], W, out=states, n_tracks=k, stream=stream)
            tf.decode_tracks(states[:k], seeds[s0:s0 + k], R, out=out[s0:], stream=stream)

    def clear():
        for t in (seeds, out, states):
            t.fill_(float("nan"))

    step()
    torch.cuda.synchronize()
    ref = [t.cpu().numpy().copy() for t in (seeds, states, out)]
    assert np.isfinite(ref[2]).mean() > 0.99
    side = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        step(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            step(side)
    torch.cuda.synchronize()
    for rep in range(3):
        clear()
        step()  # eager work between the replays
        torch.cuda.synchronize()
        clear()  # everything the replay must write again
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [t.cpu().numpy() for t in (seeds, states, out)]
        for name, a, b in zip(("seeds", "end states", "decoded"), got, ref):
            assert np.array_equal(a, b, equal_nan=True), f"replay {rep}: {name}"
