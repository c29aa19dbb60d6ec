"""GPU parity of the analytic three-hit seed and its per-hit residual features
(tf_seed_tracks) against the fp64 oracle, element by element, plus the edge
cases: short tracks, collinear hits, absolute offsets, bad offsets.
"""
import numpy as np
import pytest

import oracle
import tracksynth as ts

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# Both sides are fp64 but compute the circle by different formulas (conformal
# map in the oracle, perpendicular bisectors here), so they differ by the
# rounding of a problem whose conditioning grows with R / sagitta: the radius
# carries a relative error of about eps * 8 R^2 / c^2 (c the chord of the first
# three hits), and d0 = D - R inherits it absolutely.  With R = 16.7 m and
# c = 30 mm (the 64-layer geometry at 10 GeV) that is ~1e-8 mm, i.e. ~1e-7 of
# the d0 spread; the residual features (tens of um) see the same ~1e-8 mm.
SEED_TOL = 1e-6
FEAT_TOL = 1e-5


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32479_amd as tf
    return tf


def _colerr(g, r):
    """Per column: max |g - r| / max(|r|, rms of the column) (NaN rows must match)."""
    assert np.array_equal(np.isnan(g), np.isnan(r))
    ok = ~np.isnan(r).any(axis=1)
    g, r = g[ok], r[ok]
    if r.size == 0:
        return np.zeros(g.shape[1] if g.ndim == 2 else 0)
    rms = np.sqrt(np.mean(r ** 2, axis=0))
    return np.max(np.abs(g - r) / np.maximum(np.abs(r), np.maximum(rms, 1e-300)), axis=0)


def _wrap_phi(g, r):
    """Bring phi of g to the branch of r (a difference of 2 pi is the same angle)."""
    g = g.copy()
    d = g[:, 2] - r[:, 2]
    g[:, 2] -= np.round(d / (2 * np.pi)) * 2 * np.pi
    return g


def _run(tf, hits, offs, b, features=True):
    h = torch.from_numpy(np.ascontiguousarray(hits, dtype=np.float32)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(offs, dtype=np.int32)).cuda()
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    seeds, feats = tf.seed_tracks(h, o, b, features=features, flags=flags)
    torch.cuda.synchronize()
    return seeds.cpu().numpy(), (feats.cpu().numpy() if feats is not None else None), int(flags.item())


@pytest.mark.parametrize("name,n", [("d128x4_fp32_65k", 4096), ("deploy_d128x4_bf16_8m", 8192),
                                    ("long64_d128x4_bf16_200k", 1024), ("d256x6_bf16_1m", 2048),
                                    ("tiny_d32_fp32", 256)])
def test_seed_and_features_match_oracle(tf, name, n):
    w = ts.WORKLOADS[name]
    hits, offs = ts.make_tracks(w, n_tracks=n)
    g_seed, g_feat, flags = _run(tf, hits, offs, w.b_field)
    r_seed, r_feat, bad = oracle.seed_tracks(hits, offs, w.b_field)
    assert flags == 0 and bad == 0
    e = _colerr(_wrap_phi(g_seed, r_seed), r_seed)
    print(f"[seed] {name}: seed col err {e}", flush=True)
    assert np.all(e <= SEED_TOL), e
    ef = _colerr(g_feat.astype(np.float64), r_feat)
    print(f"[seed] {name}: feature col err {ef}", flush=True)
    assert np.all(ef <= FEAT_TOL), ef


def test_short_collinear_and_absolute_offsets(tf):
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hits, offs = ts.make_tracks(w, n_tracks=64)
    L = np.diff(offs).astype(np.int64)
    L[[2, 5, 9]] = [0, 1, 2]              # too short for a seed
    rows = [np.arange(offs[i], offs[i] + L[i]) for i in range(64)]
    h = hits[np.concatenate(rows)].copy()
    o = np.concatenate([[0], np.cumsum(L)])
    # track 11: first three hits on a line through the origin
    h[o[11]:o[11] + 3] = [[30.0, 0.0, 1.0], [60.0, 0.0, 2.0], [90.0, 0.0, 3.0]]
    # absolute offsets: 7 leading rows that belong to no track
    pad = 7
    h = np.concatenate([np.full((pad, 3), 123.0, np.float32), h])
    o = (o + pad).astype(np.int32)
    g_seed, g_feat, flags = _run(tf, h, o, w.b_field)
    r_seed, r_feat, bad = oracle.seed_tracks(h, o, w.b_field)
    assert bad == 4
    assert flags == tf.SEED_TOO_SHORT | tf.SEED_NO_CIRCLE
    for i in (2, 5, 9, 11):
        assert np.all(np.isnan(g_seed[i]))
        assert np.all(np.isnan(g_feat[o[i] - pad:o[i + 1] - pad]))
    assert g_feat.shape == (o[-1] - o[0], 3)
    assert np.all(_colerr(_wrap_phi(g_seed, r_seed), r_seed) <= SEED_TOL)
    assert np.all(_colerr(g_feat.astype(np.float64), r_feat) <= FEAT_TOL)


def test_bad_offsets_write_nothing_outside(tf):
    """A decreasing offset and rows past n_hits give NaN seeds and the flag,
    and no feature row outside the batch's rows is written."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hits, offs = ts.make_tracks(w, n_tracks=32)
    o = offs.astype(np.int32).copy()
    o[10] = o[12] + 3            # track 9 ends past track 10's end, track 10 runs backwards
    h = torch.from_numpy(hits).cuda()
    ot = torch.from_numpy(o).cuda()
    n_rows = int(o[-1] - o[0])
    feats = torch.full((n_rows + 64, 3), 7.0, dtype=torch.float32, device="cuda")  # guard rows after
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    seeds, _ = tf.seed_tracks(h, ot, w.b_field, feats=feats, flags=flags)
    torch.cuda.synchronize()
    s = seeds.cpu().numpy()
    assert int(flags.item()) & tf.SEED_BAD_OFFSETS
    assert np.all(np.isnan(s[10]))
    assert torch.all(feats[n_rows:] == 7.0)
    # a track whose rows leave [0, n_hits)
    o2 = offs.astype(np.int32).copy()
    o2[-1] = hits.shape[0] + 5
    flags.zero_()
    seeds2, _ = tf.seed_tracks(h, torch.from_numpy(o2).cuda(), w.b_field, features=False, flags=flags)
    torch.cuda.synchronize()
    assert int(flags.item()) == tf.SEED_BAD_OFFSETS
    assert np.all(np.isnan(seeds2.cpu().numpy()[-1]))
    assert not np.any(np.isnan(seeds2.cpu().numpy()[:-1]))


def test_full_deployment_batch_sampled(tf):
    """All 8 388 608 deployment tracks in one call; a seeded sample, the first
    and the last track checked against the oracle."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    print(f"[seed-full] {w.n_tracks} tracks", flush=True)
    hits, offs = ts.make_tracks(w, workers=16)
    g_seed, g_feat, flags = _run(tf, hits, offs, w.b_field)
    assert flags == 0 and not np.isnan(g_seed).any()
    rng = np.random.default_rng(17)
    n = offs.size - 1
    sel = np.unique(np.concatenate([rng.choice(n, 4096, replace=False), [0, n - 1]]))
    sh = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
    so = np.concatenate([[0], np.cumsum(np.diff(offs)[sel])]).astype(np.int32)
    r_seed, r_feat, _ = oracle.seed_tracks(sh, so, w.b_field)
    gf = np.concatenate([g_feat[offs[i]:offs[i + 1]] for i in sel])
    assert np.all(_colerr(_wrap_phi(g_seed[sel], r_seed), r_seed) <= SEED_TOL)
    assert np.all(_colerr(gf.astype(np.float64), r_feat) <= FEAT_TOL)


def test_features_into_strided_rows(tf):
    """Features written with a row stride into columns 12..14 of [H, 15] rows
    (the Fourier front end's per-hit feature rows): equal to the packed
    features, the other columns untouched."""
    w = ts.WORKLOADS["deploy_d128x4_bf16_8m"]
    hits, offs = ts.make_tracks(w, n_tracks=500)
    h = torch.from_numpy(hits).cuda()
    o = torch.from_numpy(offs).cuda()
    packed = _run(tf, hits, offs, w.b_field)[1]
    rows = torch.full((hits.shape[0], 15), -5.0, dtype=torch.float32, device="cuda")
    # the second half of the tracks alone: row 0 of the view is the first hit of track 250
    r0 = int(offs[250])
    tf.seed_tracks(h, o[250:], w.b_field, feats=rows[r0:, 12:15])
    torch.cuda.synchronize()
    got = rows.cpu().numpy()
    assert np.array_equal(got[r0:, 12:15], packed[r0:])
    assert np.all(got[:, :12] == -5.0) and np.all(got[:r0, 12:] == -5.0)
