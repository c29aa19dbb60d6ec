"""GPU parity of the paper's bidirectional minGRU backbone (tf_mingru_states)
against the fp64 oracle, element by element: end states on three workloads
(the (x, y, z) front end at d = 32, H = 64 and the Fourier front end at the
paper's d = 128, H = 192), ragged batches, rejected tracks, a workspace too
small for the batch, tile independence, the chain into the 35-quantile
readout and decode, and that chain replayed from a HIP graph.
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
N = {"mingru2_h64_tiny_d32_fp32": 256, "mingru2_h192_fourier15_d128_fp32_65k": 1024,
     "mingru2_h192_fourier15_deploy_bf16_8m": 2048}


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32479_amd as tf
    return tf


def _inputs(w, n, hits=None, offs=None):
    if hits is None:
        hits, offs = ts.make_tracks(w, n_tracks=n)
    if not w.n_features:
        return hits, offs
    _, sf, _ = oracle.seed_tracks(hits, offs, w.b_field)
    return ts.hit_features(w, hits, offs, np.nan_to_num(sf, nan=0.0)), offs


def _model(tf, w):
    blob = ts.make_mingru_weights(w)
    M = tf.MinGRU(blob, w.n_layers, w.d_model, w.hidden, tf.MODE_FOR_WEIGHTS[w.dtype], w.n_features)
    return M, blob


def _gpu(M, inp, offs, n_tracks=None, ws_rows=None):
    h = torch.from_numpy(np.ascontiguousarray(inp, dtype=np.float32)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(offs, dtype=np.int32)).cuda()
    n = offs.size - 1 if n_tracks is None else n_tracks
    rows = int(offs[n] - offs[0]) if ws_rows is None else ws_rows
    ws = torch.empty(M.workspace_bytes(rows), dtype=torch.uint8, device="cuda")
    st = M.states(h, o, workspace=ws, n_tracks=n_tracks)
    torch.cuda.synchronize()
    return st.cpu().numpy()


def _ref(w, inp, offs, blob):
    return oracle.mingru_states(inp, offs, blob, w.n_layers, w.d_model, w.hidden, n_features=w.n_features,
                                n_threads=THREADS)


def _state_err(g, r):
    assert np.array_equal(np.isnan(g), np.isnan(r))
    ok = ~np.isnan(r).any(axis=1)
    rms = np.sqrt(np.mean(r[ok] ** 2, axis=1, keepdims=True))
    return float(np.max(np.abs(g[ok] - r[ok]) / rms)) if ok.any() else 0.0


@pytest.mark.parametrize("name", list(ts.MINGRU_WORKLOADS))
def test_mingru_states_match_oracle(tf, name):
    w = ts.workload(name)
    print(f"[mingru] {name} n={N[name]}", flush=True)
    M, blob = _model(tf, w)
    inp, offs = _inputs(w, N[name])
    g = _gpu(M, inp, offs)
    r = _ref(w, inp, offs, blob)
    assert g.shape == (N[name], 2 * w.hidden)
    e = _state_err(g, r)
    print(f"[mingru] {name}: max err {e:.3g} of the track's state rms", flush=True)
    assert e <= TOL[w.dtype]
    assert M.device_error() == 0


@pytest.mark.parametrize("name", ["mingru2_h192_fourier15_deploy_bf16_8m", "mingru2_h64_tiny_d32_fp32"])
def test_mingru_ragged_batches_bad_tracks_small_workspace(tf, name):
    w0 = ts.workload(name)
    M, blob = _model(tf, w0)
    w = dataclasses.replace(w0, len_min=1, len_max=32, n_det_layers=32)
    inp, offs = _inputs(w, 500)
    r_all = _ref(w, inp, offs, blob)
    for n in (1, 2, 33, 500):
        g = _gpu(M, inp, offs[: n + 1], n_tracks=n)
        assert _state_err(g, r_all[:n]) <= TOL[w.dtype], n
    assert M.device_error() == 0
    # track 3 emptied, track 7 longer than 32: NaN rows, the rest unchanged
    Lk = np.diff(offs)
    Lk[3], Lk[7] = 0, 33
    rows = [np.resize(np.arange(offs[i], offs[i + 1]), Lk[i]) if Lk[i] else np.arange(0) for i in range(500)]
    inp2 = inp[np.concatenate(rows)]
    o2 = np.concatenate([[0], np.cumsum(Lk)]).astype(np.int32)
    g = _gpu(M, inp2, o2)
    assert np.all(np.isnan(g[[3, 7]]))
    good = np.ones(500, bool)
    good[[3, 7]] = False
    assert _state_err(g[good], r_all[good]) <= TOL[w.dtype]
    assert M.device_error() == (tf.DEVERR_EMPTY_TRACK | tf.DEVERR_TOO_LONG)
    # a workspace for the first 200 tracks' rows only: the later tracks are refused
    g = _gpu(M, inp, offs, ws_rows=int(offs[200] - offs[0]))
    assert _state_err(g[:200], r_all[:200]) <= TOL[w.dtype]
    assert np.all(np.isnan(g[200:]))
    assert M.device_error() & tf.DEVERR_BAD_OFFSETS


def test_mingru_tile_independence_and_absolute_offsets(tf):
    w = ts.workload("mingru2_h192_fourier15_deploy_bf16_8m")
    M, blob = _model(tf, w)
    inp, offs = _inputs(w, 3000)
    a = _gpu(M, inp, offs)
    assert np.array_equal(a, _gpu(M, inp, offs))
    perm = np.random.default_rng(5).permutation(3000)
    L = np.diff(offs)
    ip = np.concatenate([inp[offs[i]:offs[i + 1]] for i in perm])
    op = np.concatenate([[0], np.cumsum(L[perm])]).astype(np.int32)
    assert np.array_equal(_gpu(M, ip, op), a[perm])
    # tracks 1000..1999 through absolute offsets into the whole array
    g = _gpu(M, inp, offs[1000:], n_tracks=1000)
    assert np.array_equal(g, a[1000:2000])


@pytest.mark.parametrize("mode", ["bf16_f16act", "bf16"])
def test_fused_backbone_matches_layered_launches_bitwise(tf, mode):
    """The paper's deployed configuration (16-bit, Fourier front end, d = 128,
    H = 192, two layers) runs as one fused launch by default: its end states
    and error bits are those of the layered launches, bit for bit, on ragged
    lengths 1..32, empty and too-long tracks, absolute offsets and a
    workspace too short for the batch."""
    w0 = ts.workload("mingru2_h192_fourier15_deploy_bf16_8m")
    w = dataclasses.replace(w0, len_min=1, len_max=32, n_det_layers=32)
    blob = ts.make_mingru_weights(w0)
    M = tf.MinGRU(blob, w.n_layers, w.d_model, w.hidden, mode, w.n_features)
    inp, offs = _inputs(w, 3000)
    print(f"[fused] {mode}", flush=True)

    def both(inp, offs, **kw):
        out = []
        for fused in (True, False):
            M.set_fused(fused)
            out += [_gpu(M, inp, offs, **kw), M.device_error()]
        M.set_fused(True)
        return out

    a, ea, b, eb = both(inp, offs)
    assert np.array_equal(a, b) and ea == eb == 0
    assert np.isfinite(a).all()
    a1, ea, b1, eb = both(inp, offs[1000:], n_tracks=1000)
    assert np.array_equal(a1, b1) and np.array_equal(a1, a[1000:2000]) and ea == eb == 0
    Lk = np.diff(offs)
    Lk[3], Lk[7] = 0, 33
    rows = [np.resize(np.arange(offs[i], offs[i + 1]), Lk[i]) if Lk[i] else np.arange(0) for i in range(3000)]
    o2 = np.concatenate([[0], np.cumsum(Lk)]).astype(np.int32)
    a2, ea, b2, eb = both(inp[np.concatenate(rows)], o2)
    assert np.array_equal(a2, b2, equal_nan=True) and ea == eb == (tf.DEVERR_EMPTY_TRACK | tf.DEVERR_TOO_LONG)
    assert np.all(np.isnan(a2[[3, 7]]))
    a3, ea, b3, eb = both(inp, offs, ws_rows=int(offs[200] - offs[0]))
    assert np.array_equal(a3, b3, equal_nan=True) and ea == eb and ea & tf.DEVERR_BAD_OFFSETS
    assert np.array_equal(a3[:200], a[:200]) and np.all(np.isnan(a3[200:]))


@pytest.mark.parametrize("nf", [5, 16])
def test_fused_backbone_other_feature_counts(tf, nf):
    """The fused backbone's front end with other feature counts (a partly
    filled last front-end stage, and the most features): end states bitwise
    those of the layered launches, in both 16-bit modes."""
    rng = np.random.default_rng(11 + nf)
    lo = rng.uniform(-2.0, 0.0, nf).astype(np.float32)
    hi = (lo + rng.uniform(0.5, 3.0, nf)).astype(np.float32)
    parts = []
    for _, shape, fan_in, kind in ts.mingru_layout(2, 128, 192, nf):
        n = int(np.prod(shape))
        if kind == "lo":
            parts.append(lo)
        elif kind == "hi":
            parts.append(hi)
        elif kind == "w":
            parts.append(rng.normal(0.0, fan_in ** -0.5, n))
        else:
            parts.append(rng.uniform(-fan_in ** -0.5, fan_in ** -0.5, n))
    blob = np.concatenate(parts).astype(np.float32)
    w = dataclasses.replace(ts.workload("mingru2_h192_fourier15_deploy_bf16_8m"), len_min=1, len_max=32,
                            n_det_layers=32)
    _, offs = ts.make_tracks(w, n_tracks=700)
    feats = (lo + (hi - lo) * rng.random((int(offs[-1]), nf))).astype(np.float32)
    for mode in ("bf16_f16act", "bf16"):
        print(f"[fused] nf={nf} {mode}", flush=True)
        M = tf.MinGRU(blob, 2, 128, 192, mode, nf)
        a = _gpu(M, feats, offs)
        M.set_fused(False)
        b = _gpu(M, feats, offs)
        assert np.array_equal(a, b) and np.isfinite(a).all()
        assert M.device_error() == 0


def test_fused_backbone_only_for_its_configuration(tf):
    w = ts.workload("mingru2_h192_fourier15_d128_fp32_65k")
    M, _ = _model(tf, w)
    with pytest.raises(tf.TrackfitError):
        M.set_fused(True)
    M.set_fused(False)


@pytest.mark.parametrize("name", ["mingru2_h192_fourier15_deploy_bf16_8m", "mingru2_h192_fourier15_d128_fp32_65k"])
def test_mingru_chain_into_readout_and_decode(tf, name):
    """hits -> seed (features, seeds), backbone end states, the paper's
    35-quantile head (hidden width 128 on the 2H = 384 states; 32 on the tiny
    model's 128), point estimates and decode: against the oracle's chain on
    the same features."""
    w = ts.workload(name)
    M, blob = _model(tf, w)
    hits, offs = ts.make_tracks(w, n_tracks=1500)
    seeds, sf, _ = oracle.seed_tracks(hits, offs, w.b_field)
    feats = ts.hit_features(w, hits, offs, sf)
    mode = tf.MODE_FOR_WEIGHTS[w.dtype]
    hb = ts.make_readout_weights(w)
    d, nh = ts.readout_dims(w)
    R = tf.Readout(hb, d, nh, mode)
    st = _gpu(M, feats, offs)
    out, q = tf.decode_tracks(torch.from_numpy(st).cuda(), torch.from_numpy(seeds).cuda(), R, quantiles=True)
    torch.cuda.synchronize()
    r_q, r_out = oracle.readout_tracks(_ref(w, feats, offs, blob), seeds, hb, d, nh)
    from tests.test_readout_gpu import colerr, wrap_phi, head_tols
    eq = colerr(q.cpu().numpy(), r_q)
    eo = colerr(wrap_phi(out.cpu().numpy(), r_out), r_out)
    print(f"[mingru-chain] {name}: quantile err {eq.max():.3g} decoded err {eo.max():.3g}", flush=True)
    tq, _ = head_tols(mode, d, nh)
    assert eq.max() <= max(TOL[w.dtype], tq) and eo.max() <= TOL[w.dtype]


def test_paper_chain_graph_replays_match_eager(tf):
    """The paper's chain per batch (seed with its hit features, the fused
    backbone, readout and decode), captured in one HIP graph over three
    batches (the last one ragged) as the benchmark runs it: every replay,
    with eager work and synchronisations between the replays, gives the eager
    chain's seeds, features and decoded outputs bit for bit."""
    w = ts.MINGRU_WORKLOADS["mingru2_h192_fourier15_deploy_bf16_8m"]
    hits, offs = ts.make_tracks(w, n_tracks=5000)
    n, batch, H = offs.size - 1, 2048, w.hidden
    mode = tf.MODE_FOR_WEIGHTS[w.dtype]
    M, _ = _model(tf, w)
    M.set_fused(True)
    R = tf.Readout(ts.make_readout_weights(w), *ts.readout_dims(w), mode)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    feats = torch.zeros((int(offs[-1] - offs[0]), w.n_features), dtype=torch.float32, device="cuda")
    feats[:, :ts.N_MEASURED] = torch.from_numpy(ts.measured_features(w, hits, offs)).cuda()
    starts = list(range(0, n, batch))
    rows = max(int(offs[min(s0 + batch, n)] - offs[s0]) for s0 in starts)
    ws = torch.empty(M.workspace_bytes(rows), dtype=torch.uint8, device="cuda")
    seeds = torch.empty((n, 5), dtype=torch.float64, device="cuda")
    out = torch.empty((n, 5), dtype=torch.float64, device="cuda")
    states = torch.empty((batch, 2 * H), dtype=torch.float32, device="cuda")

    def step(stream=None):
        for s0 in starts:
            k = min(batch, n - s0)
            r0 = int(offs[s0] - offs[0])
            tf.seed_tracks(h, o[s0:], w.b_field, seeds=seeds[s0:], n_tracks=k, stream=stream,
                           feats=feats[r0:, ts.N_MEASURED:ts.N_MEASURED + 3])
            M.states(feats, o[s0:], out=states, workspace=ws, n_tracks=k, stream=stream)
            tf.decode_tracks(states[:k], seeds[s0:s0 + k], R, out=out[s0:], stream=stream)

    step()
    torch.cuda.synchronize()
    ref = [t.cpu().numpy().copy() for t in (seeds, feats, out)]
    assert np.isfinite(ref[2]).mean() > 0.99
    side = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        step(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            step(side)
    torch.cuda.synchronize()

    def clear():
        for t in (seeds, out, states):
            t.fill_(float("nan"))
        feats[:, ts.N_MEASURED:].fill_(float("nan"))

    for rep in range(3):
        clear()
        step()  # eager work between the replays
        torch.cuda.synchronize()
        clear()  # everything the replay must write again
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [t.cpu().numpy() for t in (seeds, feats, out)]
        for name, a, b in zip(("seeds", "features", "decoded"), got, ref):
            assert np.array_equal(a, b, equal_nan=True), f"replay {rep}: {name}"
