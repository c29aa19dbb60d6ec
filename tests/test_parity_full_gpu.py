"""GPU parity at every workload's full size, in the launch configuration the
benchmark times (the streamed deployment workload: 32 calls of 262 144 tracks
captured in one HIP graph), checked against the fp64 oracle on a seeded sample
of tracks, track by track: the pooled encoder, the Fourier encoder, the
readout path (seed, end states, quantile head, decode) and the paper's whole
model (seed with features, Fourier front end, minGRU backbone, readout).
"""
import os

import numpy as np
import pytest

import oracle
import tracksynth as ts
from tests.parity import TOL, assert_parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SAMPLE = {"tiny_d32_fp32": 256, "d128x4_fp32_65k": 1024, "d256x6_bf16_1m": 256,
          "long64_d128x4_bf16_200k": 384, "deploy_d128x4_bf16_8m": 2048}
WORKERS = min(16, os.cpu_count() or 1)


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32479_amd as tf
    return tf


def _launch(tf, W, h, o, n_tracks, batch):
    """fit_tracks over the whole batch, as the benchmark launches it."""
    out = torch.full((n_tracks, 5), float("nan"), dtype=torch.float32, device=h.device)
    starts = list(range(0, n_tracks, batch))
    if len(starts) == 1:
        tf.fit_tracks(h, o, W, out=out, n_tracks=n_tracks)
        torch.cuda.synchronize()
        return out
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        tf.fit_tracks(h, o, W, out=out, n_tracks=min(batch, n_tracks), stream=side)  # warm-up
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            for s0 in starts:
                tf.fit_tracks(h, o[s0:], W, out=out[s0:], n_tracks=min(batch, n_tracks - s0), stream=side)
    out.fill_(float("nan"))
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("name", list(ts.WORKLOADS))
def test_full_size_sampled(tf, name):
    w = ts.WORKLOADS[name]
    print(f"[full] {name}: {w.n_tracks} tracks", flush=True)
    hits, offs = ts.make_tracks(w, workers=WORKERS)
    n = offs.size - 1
    blob = ts.make_weights(w)
    W = tf.Weights(blob, w.n_layers, w.d_model, tf.MODE_FOR_WEIGHTS[w.dtype], max_hits=w.len_max)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    out = _launch(tf, W, h, o, n, w.batch or n).cpu().numpy()
    assert tf.device_error(W) == 0
    assert np.all(np.isfinite(out)), "a track was not written"

    # seeded sample, always with the first and last track and a shortest and longest one
    L = np.diff(offs)
    rng = np.random.default_rng(11)
    sel = set(rng.choice(n, size=min(SAMPLE[name], n), replace=False).tolist())
    sel |= {0, n - 1, int(np.argmin(L)), int(np.argmax(L))}
    sel = np.array(sorted(sel))
    sh = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
    so = np.concatenate([[0], np.cumsum(L[sel])]).astype(np.int32)
    ref = oracle.fit_tracks(sh, so, blob, w.n_layers, w.d_model)
    emax, l2 = assert_parity(out[sel], ref, TOL[w.dtype], f"{name} full size, {sel.size} sampled tracks")
    print(f"[full] {name}: {sel.size} sampled, max col err {emax.max():.3g}", flush=True)


def test_fourier_deployment_full_size_sampled(tf):
    """All 8 388 608 tracks through the Fourier front end in the benchmark's
    launch configuration: the seed kernel writes the 3 seed features into the
    feature rows, then 32 captured fit_tracks calls.  A seeded sample is run
    through the oracle's own chain (its seed features, its encoder)."""
    w = ts.workload("fourier15_deploy_d128x4_bf16_8m")
    print(f"[full] {w.name}: {w.n_tracks} tracks", flush=True)
    hits, offs = ts.make_tracks(w, workers=WORKERS)
    n = offs.size - 1
    blob = ts.make_fourier_weights(w)
    W = tf.Weights(blob, w.n_layers, w.d_model, tf.MODE_FOR_WEIGHTS[w.dtype], max_hits=w.len_max,
                   n_features=w.n_features)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    feats = torch.empty((hits.shape[0], 15), dtype=torch.float32, device="cuda")
    step = 1 << 20
    for i0 in range(0, n, step):
        i1 = min(n, i0 + step)
        m = ts.measured_features(w, hits[offs[i0]:offs[i1]], offs[i0:i1 + 1])
        feats[offs[i0]:offs[i1], :12] = torch.from_numpy(m).cuda()
    tf.seed_tracks(h, o, w.b_field, feats=feats[:, 12:15])
    out = _launch(tf, W, feats, o, n, w.batch).cpu().numpy()
    assert tf.device_error(W) == 0
    assert np.all(np.isfinite(out))
    L = np.diff(offs)
    rng = np.random.default_rng(12)
    sel = set(rng.choice(n, size=2048, replace=False).tolist()) | {0, n - 1, int(np.argmin(L)), int(np.argmax(L))}
    sel = np.array(sorted(sel))
    sh = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
    so = np.concatenate([[0], np.cumsum(L[sel])]).astype(np.int32)
    _, sf, bad = oracle.seed_tracks(sh, so, w.b_field)
    assert bad == 0
    ref = oracle.fit_tracks(ts.hit_features(w, sh, so, sf), so, blob, w.n_layers, w.d_model,
                            n_features=w.n_features)
    emax, _ = assert_parity(out[sel], ref, TOL[w.dtype], f"{w.name} full size, {sel.size} sampled tracks")
    print(f"[full] {w.name}: {sel.size} sampled, max col err {emax.max():.3g}", flush=True)


def _device_feature_rows(tf, w, hits, offs, h, o):
    """The 15-feature rows on the device: the generator's 12 measured features,
    the GPU seed's 3 features in columns 12..14 (as the benchmark builds them)."""
    n = offs.size - 1
    feats = torch.empty((hits.shape[0], 15), dtype=torch.float32, device="cuda")
    step = 1 << 20
    for i0 in range(0, n, step):
        i1 = min(n, i0 + step)
        m = ts.measured_features(w, hits[offs[i0]:offs[i1]], offs[i0:i1 + 1])
        feats[offs[i0]:offs[i1], :12] = torch.from_numpy(m).cuda()
    tf.seed_tracks(h, o, w.b_field, feats=feats[:, 12:15])
    return feats


def _captured(fn, starts):
    """Run fn(s0, stream) for every batch start, captured in one HIP graph and
    replayed once, as the benchmark does."""
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        for s0 in starts:
            fn(s0, side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            for s0 in starts:
                fn(s0, side)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()


def _sample(offs, seed, k=2048):
    n = offs.size - 1
    L = np.diff(offs)
    rng = np.random.default_rng(seed)
    sel = set(rng.choice(n, size=k, replace=False).tolist()) | {0, n - 1, int(np.argmin(L)), int(np.argmax(L))}
    return np.array(sorted(sel))


def _decoded_err(g, r):
    g = g.copy()
    g[:, 2] -= np.round((g[:, 2] - r[:, 2]) / (2 * np.pi)) * 2 * np.pi
    rms = np.sqrt(np.mean(r ** 2, axis=0))
    return float(np.max(np.abs(g - r) / np.maximum(np.abs(r), rms)))


def test_readout_path_full_size_sampled(tf):
    """All deployment tracks through seed, end states and the 35-quantile
    readout in 32 graph-captured batches (the readout benchmark's
    configuration); a sample against the oracle's chain."""
    w = ts.workload("deploy_d128x4_bf16_8m")
    print(f"[full] readout path {w.name}: {w.n_tracks} tracks", flush=True)
    hits, offs = ts.make_tracks(w, workers=WORKERS)
    n = offs.size - 1
    mode = tf.MODE_FOR_WEIGHTS[w.dtype]
    blob = ts.make_weights(w)
    hb = ts.make_readout_weights(w)
    W = tf.Weights(blob, w.n_layers, w.d_model, mode, max_hits=w.len_max)
    R = tf.Readout(hb, *ts.readout_dims(w), mode)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    seeds = torch.empty((n, 5), dtype=torch.float64, device="cuda")
    out = torch.full((n, 5), float("nan"), dtype=torch.float64, device="cuda")
    states = torch.empty((w.batch, 2 * w.d_model), dtype=torch.float32, device="cuda")

    def one(s0, stream):
        k = min(w.batch, n - s0)
        tf.seed_tracks(h, o[s0:], w.b_field, features=False, seeds=seeds[s0:], n_tracks=k, stream=stream)
        tf.fit_tracks_states(h, o[s0:], W, out=states, n_tracks=k, stream=stream)
        tf.decode_tracks(states[:k], seeds[s0:s0 + k], R, out=out[s0:], stream=stream)

    _captured(one, list(range(0, n, w.batch)))
    g = out.cpu().numpy()
    assert np.all(np.isfinite(g)) and tf.device_error(W) == 0
    sel = _sample(offs, 13)
    L = np.diff(offs)
    sh = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
    so = np.concatenate([[0], np.cumsum(L[sel])]).astype(np.int32)
    r_seed, _, _ = oracle.seed_tracks(sh, so, w.b_field, features=False)
    r_st = oracle.track_states(sh, so, blob, w.n_layers, w.d_model)
    _, r_out = oracle.readout_tracks(r_st, r_seed, hb, *ts.readout_dims(w))
    err = _decoded_err(g[sel], r_out)
    print(f"[full] readout path: {sel.size} sampled, max decoded column error {err:.3g}", flush=True)
    assert err <= TOL[w.dtype]


def test_paper_model_full_size_sampled(tf):
    """The paper's whole model (seed with features, Fourier front end, two
    minGRU layers, readout, decode) over all deployment tracks in 32
    graph-captured batches (the benchmark's configuration); a sample against
    the oracle's chain (its own seed features)."""
    w = ts.workload("mingru2_h192_fourier15_deploy_bf16_8m")
    print(f"[full] paper model {w.name}: {w.n_tracks} tracks", flush=True)
    hits, offs = ts.make_tracks(w, workers=WORKERS)
    n = offs.size - 1
    mode = tf.MODE_FOR_WEIGHTS[w.dtype]
    blob = ts.make_mingru_weights(w)
    hb = ts.make_readout_weights(w)
    M = tf.MinGRU(blob, w.n_layers, w.d_model, w.hidden, mode, w.n_features)
    R = tf.Readout(hb, *ts.readout_dims(w), mode)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    feats = _device_feature_rows(tf, w, hits, offs, h, o)
    seeds = torch.empty((n, 5), dtype=torch.float64, device="cuda")
    out = torch.full((n, 5), float("nan"), dtype=torch.float64, device="cuda")
    states = torch.empty((w.batch, 2 * w.hidden), dtype=torch.float32, device="cuda")
    starts = list(range(0, n, w.batch))
    rows = max(int(offs[min(s0 + w.batch, n)] - offs[s0]) for s0 in starts)
    ws = torch.empty(M.workspace_bytes(rows), dtype=torch.uint8, device="cuda")

    def one(s0, stream):
        k = min(w.batch, n - s0)
        tf.seed_tracks(h, o[s0:], w.b_field, seeds=seeds[s0:], n_tracks=k, stream=stream,
                       feats=feats[int(offs[s0]):, 12:15])
        M.states(feats, o[s0:], out=states, workspace=ws, n_tracks=k, stream=stream)
        tf.decode_tracks(states[:k], seeds[s0:s0 + k], R, out=out[s0:], stream=stream)

    _captured(one, starts)
    g = out.cpu().numpy()
    assert np.all(np.isfinite(g)) and M.device_error() == 0
    sel = _sample(offs, 14)
    L = np.diff(offs)
    sh = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
    so = np.concatenate([[0], np.cumsum(L[sel])]).astype(np.int32)
    r_seed, sf, _ = oracle.seed_tracks(sh, so, w.b_field)
    r_st = oracle.mingru_states(ts.hit_features(w, sh, so, sf), so, blob, w.n_layers, w.d_model, w.hidden,
                                n_features=w.n_features)
    _, r_out = oracle.readout_tracks(r_st, r_seed, hb, *ts.readout_dims(w))
    err = _decoded_err(g[sel], r_out)
    print(f"[full] paper model: {sel.size} sampled, max decoded column error {err:.3g}", flush=True)
    assert err <= TOL[w.dtype]
