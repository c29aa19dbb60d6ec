"""ctypes wrapper of the fp64 CPU oracle.

TEST INFRASTRUCTURE ONLY.  The oracle checks the GPU library; only the tests,
the smoke check and the benchmark's CPU-baseline leg may import it.  It does
not import the GPU package and the GPU package does not import it.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB, build

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        fp = ctypes.POINTER(ctypes.c_float)
        ip = ctypes.POINTER(ctypes.c_int32)
        L.orc_blob_size.restype = ctypes.c_size_t
        L.orc_blob_size.argtypes = [ctypes.c_int, ctypes.c_int]
        L.orc_sigmoid.restype = ctypes.c_double
        L.orc_sigmoid.argtypes = [ctypes.c_double]
        L.orc_silu.restype = ctypes.c_double
        L.orc_silu.argtypes = [ctypes.c_double]
        L.orc_linear.restype = None
        L.orc_linear.argtypes = [dp, dp, dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, dp]
        L.orc_rmsnorm.restype = None
        L.orc_rmsnorm.argtypes = [dp, dp, ctypes.c_int, ctypes.c_int, ctypes.c_double, dp]
        for fn in (L.orc_scan_forward, L.orc_scan_backward):
            fn.restype = None
            fn.argtypes = [dp, dp, ctypes.c_int, ctypes.c_int, dp]
        L.orc_track_forward.restype = ctypes.c_int
        L.orc_track_forward.argtypes = [fp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, fp, dp, dp,
                                        dp, dp]
        L.orc_track_states.restype = ctypes.c_long
        L.orc_track_states.argtypes = [fp, ctypes.c_int, ip, ctypes.c_int32, ctypes.c_int, ctypes.c_int, fp,
                                       ctypes.c_size_t, dp, ctypes.c_int]
        L.orc_fourier_blob_size.restype = ctypes.c_size_t
        L.orc_fourier_blob_size.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.orc_mingru_blob_size.restype = ctypes.c_size_t
        L.orc_mingru_blob_size.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.orc_mingru_states.restype = ctypes.c_long
        L.orc_mingru_states.argtypes = [fp, ctypes.c_int, ip, ctypes.c_int32, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, fp, ctypes.c_size_t, dp, ctypes.c_int]
        L.orc_fourier_features.restype = None
        L.orc_fourier_features.argtypes = [fp, ctypes.c_int, fp, fp, dp]
        L.orc_readout_blob_size.restype = ctypes.c_size_t
        L.orc_readout_blob_size.argtypes = [ctypes.c_int, ctypes.c_int]
        L.orc_decode.restype = None
        L.orc_decode.argtypes = [dp, dp, dp]
        L.orc_readout_track.restype = None
        L.orc_readout_track.argtypes = [dp, ctypes.c_int, ctypes.c_int, fp, dp, dp, dp]
        L.orc_readout_tracks.restype = ctypes.c_long
        L.orc_readout_tracks.argtypes = [dp, ctypes.c_int32, ctypes.c_int, ctypes.c_int, fp, ctypes.c_size_t, dp,
                                         dp, dp]
        L.orc_fit_tracks.restype = ctypes.c_long
        L.orc_fit_tracks.argtypes = [fp, ctypes.c_int, ip, ctypes.c_int32, ctypes.c_int, ctypes.c_int, fp,
                                     ctypes.c_size_t, dp, ctypes.c_int]
        L.orc_threads.restype = ctypes.c_int
        L.orc_threads.argtypes = [ctypes.c_int]
        L.orc_seed_from_points.restype = ctypes.c_int
        L.orc_seed_from_points.argtypes = [dp, ctypes.c_double, dp]
        L.orc_seed_features_hit.restype = None
        L.orc_seed_features_hit.argtypes = [dp, ctypes.c_double, dp, dp]
        L.orc_seed_tracks.restype = ctypes.c_long
        L.orc_seed_tracks.argtypes = [fp, ip, ctypes.c_int32, ctypes.c_double, dp, dp]
        _lib = L
    return _lib


def _d(a):
    a = np.ascontiguousarray(a, dtype=np.float64)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def blob_size(n_layers: int, d: int) -> int:
    return int(lib().orc_blob_size(n_layers, d))


def sigmoid(v: float) -> float:
    return lib().orc_sigmoid(float(v))


def silu(v: float) -> float:
    return lib().orc_silu(float(v))


def linear(W, b, x):
    """y[t] = b + W x[t] for rows x [n, n_in]; W [n_out, n_in]."""
    W, pW = _d(W)
    x, px = _d(np.atleast_2d(x))
    n_out, n_in = W.shape
    assert x.shape[1] == n_in
    pb = None
    if b is not None:
        b, pb = _d(b)
    y = np.empty((x.shape[0], n_out))
    lib().orc_linear(pW, pb, px, x.shape[0], n_in, n_out, y.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return y


def rmsnorm(r, g, eps=1e-6):
    r, pr = _d(np.atleast_2d(r))
    g, pg = _d(g)
    y = np.empty_like(r)
    lib().orc_rmsnorm(pr, pg, r.shape[0], r.shape[1], eps, y.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return y


def _scan(fn, x, a):
    x, px = _d(x)
    a, pa = _d(a)
    assert x.shape == a.shape and x.ndim == 2
    out = np.empty_like(x)
    fn(px, pa, x.shape[0], x.shape[1], out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return out


def scan_forward(x, a):
    """Eq. (2) forward over rows of x, a [L, d]."""
    return _scan(lib().orc_scan_forward, x, a)


def scan_backward(x, a):
    """Eq. (2) run from the last row to the first."""
    return _scan(lib().orc_scan_backward, x, a)


def _model_size(n_layers, d, n_features):
    return fourier_blob_size(n_layers, d, n_features) if n_features else blob_size(n_layers, d)


def track_forward(hits, blob, n_layers, d, with_states=False, n_features=0):
    """One track: returns (out5, pooled [d], residual stream after the last layer [L, d])
    and, if asked, the last layer's end states [2d] (forward at the last hit,
    reverse at the first hit).  n_features > 0: hits are [L, F] per-hit
    features of the Fourier front end."""
    hits, ph = _f(np.asarray(hits).reshape(-1, n_features or 3))
    blob, pb = _f(blob)
    assert blob.size == _model_size(n_layers, d, n_features)
    L = hits.shape[0]
    out = np.empty(5)
    pooled = np.empty(d)
    resid = np.empty((max(L, 1), d))
    states = np.empty(2 * d)
    dp = ctypes.POINTER(ctypes.c_double)
    rc = lib().orc_track_forward(ph, L, int(n_features), n_layers, d, pb, out.ctypes.data_as(dp),
                                 pooled.ctypes.data_as(dp), resid.ctypes.data_as(dp),
                                 states.ctypes.data_as(dp) if (with_states and n_layers > 0) else None)
    res = (out, pooled, (resid[:L] if rc == 0 else None))
    return res + (states,) if with_states else res


def fit_tracks(hits, offsets, blob, n_layers, d, n_threads=0, n_features=0):
    """Packed batch: returns out [N, 5] float64 (NaN rows for tracks with no hits).
    n_features > 0: hits are [H, F] per-hit features of the Fourier front end."""
    hits, ph = _f(np.asarray(hits).reshape(-1, n_features or 3))
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    blob, pb = _f(blob)
    n = offsets.size - 1
    out = np.empty((max(n, 0), 5))
    rc = lib().orc_fit_tracks(ph, int(n_features), offsets.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n,
                              n_layers, d,
                              pb, blob.size, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), int(n_threads))
    if rc < 0:
        raise ValueError("oracle rejected its arguments")
    return out


def fourier_blob_size(n_layers: int, d: int, n_features: int) -> int:
    return int(lib().orc_fourier_blob_size(n_layers, d, n_features))


def fourier_features(feat, lo, hi):
    """Fourier features [32 F] of one hit's F features (fp64 values; see oracle.c)."""
    f, pf = _f(np.asarray(feat).reshape(-1))
    l, pl = _f(lo)
    h, ph = _f(hi)
    assert l.size == f.size == h.size
    out = np.empty(32 * f.size)
    lib().orc_fourier_features(pf, f.size, pl, ph, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return out


def threads(n_threads=0) -> int:
    return int(lib().orc_threads(int(n_threads)))


# ---------------------------------------------------------------------------
# Analytic three-hit seed and per-hit seed residual features (Sec. Method,
# Analytic seed); fp64.
# ---------------------------------------------------------------------------

def seed_from_points(points, b_tesla):
    """Seed (d0, z0, phi, theta, q/p) from three points [3, 3] (fp64 in mm);
    NaN if no circle passes through them."""
    p, pp = _d(np.asarray(points, dtype=np.float64).reshape(9))
    out = np.empty(5)
    lib().orc_seed_from_points(pp, float(b_tesla), out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return out


def seed_features_hit(seed, b_tesla, hit):
    """(asinh dU, asinh dV, helix path length) of one hit against a seed."""
    s, ps = _d(seed)
    h, ph = _d(np.asarray(hit, dtype=np.float64).reshape(3))
    out = np.empty(3)
    lib().orc_seed_features_hit(ps, float(b_tesla), ph, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return out


def seed_tracks(hits, offsets, b_tesla, features=True):
    """Packed batch (float32 hits): returns (seeds [N, 5], features [H, 3] or
    None, number of tracks without a seed).  Feature row r belongs to hit row
    offsets[0] + r."""
    hits, ph = _f(np.asarray(hits).reshape(-1, 3))
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    n = offsets.size - 1
    seeds = np.empty((max(n, 0), 5))
    dp = ctypes.POINTER(ctypes.c_double)
    feats = np.empty((int(offsets[-1] - offsets[0]) if n > 0 else 0, 3)) if features else None
    rc = lib().orc_seed_tracks(ph, offsets.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n, float(b_tesla),
                               seeds.ctypes.data_as(dp), feats.ctypes.data_as(dp) if features else None)
    if rc < 0:
        raise ValueError("oracle rejected its arguments")
    return seeds, feats, int(rc)


# ---------------------------------------------------------------------------
# The paper's readout and decode (Sec. Encoder, last paragraph; Sec. Losses).
# ---------------------------------------------------------------------------

def track_states(hits, offsets, blob, n_layers, d, n_threads=0, n_features=0):
    """Packed batch: the last layer's end states [N, 2d] (NaN rows for empty tracks)."""
    hits, ph = _f(np.asarray(hits).reshape(-1, n_features or 3))
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    blob, pb = _f(blob)
    n = offsets.size - 1
    st = np.empty((max(n, 0), 2 * d))
    rc = lib().orc_track_states(ph, int(n_features), offsets.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n,
                                n_layers, d,
                                pb, blob.size, st.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), int(n_threads))
    if rc < 0:
        raise ValueError("oracle rejected its arguments")
    return st


def readout_blob_size(d, hidden):
    return int(lib().orc_readout_blob_size(int(d), int(hidden)))


def decode(seed, est):
    """Decode the five point estimates against a seed."""
    s, ps = _d(seed)
    m, pm = _d(est)
    out = np.empty(5)
    lib().orc_decode(ps, pm, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return out


def readout_tracks(states, seeds, head_blob, d, hidden):
    """states [N, 2d], seeds [N, 5], a head of hidden width `hidden` ->
    (quantiles [N, 35], decoded [N, 5])."""
    st, pst = _d(np.asarray(states).reshape(-1, 2 * d))
    sd, psd = _d(np.asarray(seeds).reshape(-1, 5))
    hb, phb = _f(head_blob)
    n = st.shape[0]
    assert sd.shape[0] == n
    q = np.empty((n, 35))
    out = np.empty((n, 5))
    dp = ctypes.POINTER(ctypes.c_double)
    rc = lib().orc_readout_tracks(pst, n, d, int(hidden), phb, hb.size, psd, q.ctypes.data_as(dp),
                                  out.ctypes.data_as(dp))
    if rc < 0:
        raise ValueError("oracle rejected its arguments")
    return q, out


# ---------------------------------------------------------------------------
# The paper's bidirectional minGRU backbone (Sec. Encoder).
# ---------------------------------------------------------------------------

def mingru_blob_size(n_layers, d, H, n_features=0):
    return int(lib().orc_mingru_blob_size(int(n_layers), int(d), int(H), int(n_features)))


def mingru_states(hits, offsets, blob, n_layers, d, H, n_features=0, n_threads=0):
    """Packed batch: the last layer's end states [N, 2H] (NaN rows for empty tracks)."""
    hits, ph = _f(np.asarray(hits).reshape(-1, n_features or 3))
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    blob, pb = _f(blob)
    n = offsets.size - 1
    st = np.empty((max(n, 0), 2 * H))
    rc = lib().orc_mingru_states(ph, int(n_features), offsets.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n,
                                 int(n_layers), int(d), int(H), pb, blob.size,
                                 st.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), int(n_threads))
    if rc < 0:
        raise ValueError("oracle rejected its arguments")
    return st
