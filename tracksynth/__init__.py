"""Seeded synthetic inputs: helix tracks in a solenoid and random encoder weights.

This module is shared by the tests, the benchmark and the CPU oracle's callers.
It holds none of the encoder's arithmetic: it only draws track parameters,
intersects helices with detector cylinders, and draws weight tensors.

Tracks (stand-in for the paper's simulated muon samples, Sec. Data): a charged
particle in a uniform field B along z follows a helix whose transverse radius is
R = pT / (0.299792458 * B) metres (pT in GeV, B in tesla).  Each track is
parameterised at its perigee by (d0, z0, phi, theta, q/p), the five quantities
the method regresses (Sec. Method).  Hits are the intersections of the helix
with barrel cylinders of fixed radius, ordered by increasing radius, which for
these outgoing non-looping tracks is the time order the paper feeds the encoder
(Sec. Data).  Each hit is smeared by 10 um along r*phi and along z.

Packed layout (Sec. Kernel adaptation: packed, unpadded batches): hits of all
tracks are concatenated into one float32 array [H, 3] of (x, y, z) in mm and
track i owns rows offsets[i] .. offsets[i+1]-1 of it.

Weights: one float32 blob in the canonical order documented in
``blob_layout``; for bf16 workloads every value is rounded (round to nearest
even) to a bf16-representable float32 before it is returned, so that the CPU
oracle and the GPU library see identical weights.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "workload", "make_tracks", "make_track_chunk",
    "make_weights", "blob_layout", "blob_size", "round_to_bf16", "TRACK_CHUNK",
    "KAPPA_GEV_PER_T_M", "readout_layout", "readout_dims", "make_readout_weights",
    "FOURIER_WORKLOADS", "N_MEASURED", "measured_features", "feature_bounds", "fourier_layout",
    "make_fourier_weights", "hit_features", "MINGRU_WORKLOADS", "mingru_layout", "make_mingru_weights",
]

# pT [GeV] = KAPPA * B [T] * R [m] for a unit-charge particle.
KAPPA_GEV_PER_T_M = 0.299792458
# Tracks are generated in fixed chunks, each from its own seeded stream, so any
# chunk (and therefore any subset of a large workload) can be regenerated alone.
TRACK_CHUNK = 65536


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: model shape, number type and track sample."""
    name: str
    index: int            # 1-based; data seed 1000+index, weight seed 2000+index
    n_layers: int
    d_model: int
    dtype: str            # "fp32" or "bf16"
    n_tracks: int
    len_min: int          # hits per track ~ U{len_min..len_max}
    len_max: int
    n_det_layers: int     # barrel cylinders, radii linearly spaced r_min..r_max
    r_min: float = 30.0
    r_max: float = 1000.0
    z_max: float = 3000.0
    b_field: float = 2.0  # tesla, along +z
    pt_mode: str = "uniform_pt"   # "uniform_pt": pT~U(1,10); "uniform_invpt": 1/pT~U(0.1,1)
    eta_max: float = 1.5
    batch: int = 0        # tracks per fit_tracks call when the workload is streamed
    n_features: int = 0   # > 0: per-hit features for the Fourier front end (12 measured + 3 seed)
    arch: str = "residual"  # "residual": the layers of blob_layout; "mingru": the paper's backbone
    hidden: int = 0       # minGRU hidden width H (the states are 2H wide)
    head_hidden: int = 128  # hidden width of the paper's readout head (Sec. Encoder: 128)

    @property
    def data_seed(self) -> int:
        return 1000 + self.index

    @property
    def weight_seed(self) -> int:
        return 2000 + self.index


WORKLOADS = {
    w.name: w for w in [
        Workload("tiny_d32_fp32", 1, n_layers=1, d_model=32, dtype="fp32", n_tracks=256,
                 len_min=10, len_max=10, n_det_layers=10, head_hidden=96),
        Workload("d128x4_fp32_65k", 2, n_layers=4, d_model=128, dtype="fp32", n_tracks=65536,
                 len_min=8, len_max=20, n_det_layers=20),
        Workload("d256x6_bf16_1m", 3, n_layers=6, d_model=256, dtype="bf16", n_tracks=1048576,
                 len_min=8, len_max=30, n_det_layers=30),
        Workload("long64_d128x4_bf16_200k", 4, n_layers=4, d_model=128, dtype="bf16",
                 n_tracks=200000, len_min=64, len_max=64, n_det_layers=64),
        Workload("deploy_d128x4_bf16_8m", 5, n_layers=4, d_model=128, dtype="bf16",
                 n_tracks=8388608, len_min=8, len_max=20, n_det_layers=20,
                 pt_mode="uniform_invpt", batch=262144),
    ]
}


# The same tracks and encoders with the paper's front end: 15 per-hit features
# (12 measured stand-ins and the 3 seed residual features), Fourier-expanded.
FOURIER_WORKLOADS = {
    w.name: w for w in [
        dataclasses.replace(WORKLOADS["tiny_d32_fp32"], name="fourier15_tiny_d32_fp32", n_features=15),
        dataclasses.replace(WORKLOADS["d128x4_fp32_65k"], name="fourier15_d128x4_fp32_65k", n_features=15),
        dataclasses.replace(WORKLOADS["deploy_d128x4_bf16_8m"], name="fourier15_deploy_d128x4_bf16_8m",
                            n_features=15),
    ]
}


# The paper's backbone: two bidirectional minGRU layers of hidden width H
# behind the front end (the deployed model: Fourier front end to d = 128,
# H = 192), on the same tracks.
MINGRU_WORKLOADS = {
    w.name: w for w in [
        dataclasses.replace(WORKLOADS["tiny_d32_fp32"], name="mingru2_h64_tiny_d32_fp32", n_layers=2,
                            arch="mingru", hidden=64, head_hidden=32),
        dataclasses.replace(WORKLOADS["d128x4_fp32_65k"], name="mingru2_h192_fourier15_d128_fp32_65k",
                            n_layers=2, arch="mingru", hidden=192, n_features=15),
        dataclasses.replace(WORKLOADS["deploy_d128x4_bf16_8m"], name="mingru2_h192_fourier15_deploy_bf16_8m",
                            n_layers=2, arch="mingru", hidden=192, n_features=15),
    ]
}


def workload(name_or_index) -> Workload:
    if isinstance(name_or_index, Workload):
        return name_or_index
    if isinstance(name_or_index, int):
        for w in WORKLOADS.values():
            if w.index == name_or_index:
                return w
        raise KeyError(name_or_index)
    if name_or_index in FOURIER_WORKLOADS:
        return FOURIER_WORKLOADS[name_or_index]
    if name_or_index in MINGRU_WORKLOADS:
        return MINGRU_WORKLOADS[name_or_index]
    return WORKLOADS[name_or_index]


# ----------------------------------------------------------------------------
# Helix tracks
# ----------------------------------------------------------------------------

def _streams(seed: int, chunk: int):
    """One independent stream per drawn quantity, so that the first n draws of
    every quantity do not depend on how many tracks are drawn."""
    names = ("pt", "eta", "phi", "d0", "z0", "q", "length", "smear_rphi", "smear_z")
    return {k: np.random.default_rng([seed, chunk, i]) for i, k in enumerate(names)}


def _draw_params(w: Workload, rng, n: int):
    if not isinstance(rng, dict):
        rng = _streams(int(rng.integers(2 ** 31)), 0)
    if w.pt_mode == "uniform_pt":
        pt = rng["pt"].uniform(1.0, 10.0, n)
    elif w.pt_mode == "uniform_invpt":
        pt = 1.0 / rng["pt"].uniform(0.1, 1.0, n)
    else:
        raise ValueError(w.pt_mode)
    eta = rng["eta"].uniform(-w.eta_max, w.eta_max, n)
    phi = rng["phi"].uniform(-math.pi, math.pi, n)
    d0 = rng["d0"].normal(0.0, 0.1, n)
    z0 = rng["z0"].normal(0.0, 1.0, n)
    q = np.where(rng["q"].random(n) < 0.5, -1.0, 1.0)
    length = rng["length"].integers(w.len_min, w.len_max + 1, n)
    return pt, eta, phi, d0, z0, q, length


def helix_hits(pt, eta, phi, d0, z0, q, radii, b_field):
    """Noise-free intersections of helices with cylinders.

    Arrays of shape [n] for the track parameters and [m] for the radii; returns
    x, y, z of shape [n, m] (mm) and the transverse arc length s [n, m].
    The circle has radius R and centre C = (d0 + R/k) * n_hat with
    n_hat = (-sin phi, cos phi) and k = -q (sense of rotation), so that the
    perigee is P0 = d0 * n_hat with direction (cos phi, sin phi).  The turning
    angle a at radius r follows from |C + Rot(k a)(P0 - C)| = r.
    """
    R = 1000.0 * pt / (KAPPA_GEV_PER_T_M * b_field)          # mm
    k = -q
    nx, ny = -np.sin(phi), np.cos(phi)
    cs = d0 + R / k                                           # signed centre distance
    cx, cy = cs * nx, cs * ny
    D = np.abs(cs)
    ux, uy = -(R / k) * nx, -(R / k) * ny                     # P0 - C
    r = np.asarray(radii, dtype=np.float64)[None, :]
    cos_a = (D[:, None] ** 2 + R[:, None] ** 2 - r ** 2) / (2.0 * R[:, None] * D[:, None])
    if np.any(np.abs(cos_a) > 1.0):
        raise ValueError("a helix does not reach a detector cylinder")
    a = np.arccos(cos_a)
    th = k[:, None] * a
    c, s = np.cos(th), np.sin(th)
    x = cx[:, None] + ux[:, None] * c - uy[:, None] * s
    y = cy[:, None] + ux[:, None] * s + uy[:, None] * c
    arc = R[:, None] * a
    z = z0[:, None] + arc * np.sinh(eta)[:, None]
    return x, y, z, arc


def make_track_chunk(w: Workload, chunk: int, n: int, seed: int | None = None, smear: bool = True):
    """Generate tracks chunk*TRACK_CHUNK .. +n-1 of a workload.

    Returns (hits float32 [H,3], lengths int32 [n], truth float64 [n,5]) where
    truth holds (d0, z0, phi, theta, q/p) at the perigee.
    """
    seed = w.data_seed if seed is None else seed
    rng = _streams(seed, chunk)
    pt, eta, phi, d0, z0, q, length = _draw_params(w, rng, n)
    radii = np.linspace(w.r_min, w.r_max, w.n_det_layers)
    x, y, z, _ = helix_hits(pt, eta, phi, d0, z0, q, radii, w.b_field)
    if smear:
        rphi = rng["smear_rphi"].normal(0.0, 0.010, x.shape)
        dz = rng["smear_z"].normal(0.0, 0.010, x.shape)
        ang = np.arctan2(y, x) + rphi / radii[None, :]
        x = radii[None, :] * np.cos(ang)
        y = radii[None, :] * np.sin(ang)
        z = z + dz
    if np.any(np.abs(z) > w.z_max):
        raise ValueError("hit outside the detector length")
    keep = np.arange(w.n_det_layers)[None, :] < length[:, None]
    hits = np.stack([x[keep], y[keep], z[keep]], axis=1).astype(np.float32)
    theta = 2.0 * np.arctan(np.exp(-eta))
    p = pt * np.cosh(eta)
    truth = np.stack([d0, z0, phi, theta, q / p], axis=1)
    return hits, length.astype(np.int32), truth


def _chunk_job(args):
    w, chunk, n, seed, smear = args
    return make_track_chunk(w, chunk, n, seed, smear)


def make_tracks(w, n_tracks: int | None = None, seed: int | None = None, smear: bool = True,
                with_truth: bool = False, workers: int = 1):
    """Generate the first ``n_tracks`` tracks of a workload (default: all).

    Returns (hits float32 [H,3], offsets int32 [N+1]) and, if requested, the
    truth perigee parameters float64 [N,5].  ``workers`` > 1 generates the
    fixed-size chunks in that many processes (same result: every chunk has its
    own seeded streams).
    """
    w = workload(w)
    n_tracks = w.n_tracks if n_tracks is None else int(n_tracks)
    jobs = []
    done, chunk = 0, 0
    while done < n_tracks:
        n = min(TRACK_CHUNK, n_tracks - done)
        jobs.append((w, chunk, n, seed, smear))
        done += n
        chunk += 1
    if workers > 1 and len(jobs) > 1:
        from concurrent.futures import ProcessPoolExecutor
        with ProcessPoolExecutor(min(workers, len(jobs))) as ex:
            parts = list(ex.map(_chunk_job, jobs))
    else:
        parts = [_chunk_job(j) for j in jobs]
    hits_parts = [p[0] for p in parts]
    len_parts = [p[1] for p in parts]
    truth_parts = [p[2] for p in parts]
    lengths = np.concatenate(len_parts) if len_parts else np.zeros(0, np.int32)
    offsets = np.zeros(n_tracks + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    if offsets[-1] >= 2 ** 31:
        raise ValueError("too many hits for int32 offsets")
    hits = np.concatenate(hits_parts) if hits_parts else np.zeros((0, 3), np.float32)
    out = (np.ascontiguousarray(hits), offsets.astype(np.int32))
    if with_truth:
        out = out + (np.concatenate(truth_parts) if truth_parts else np.zeros((0, 5)),)
    return out


# ----------------------------------------------------------------------------
# Weights
# ----------------------------------------------------------------------------

def blob_layout(n_layers: int, d: int):
    """Canonical fp32 weight blob: list of (name, shape, fan_in, kind).

    Matrices are row-major [out][in].  kind is "w" (normal, variance 1/fan_in),
    "b" (uniform in +-fan_in^-1/2) or "g" (RMSNorm gain, uniform in [0.5, 1.5]).
    Rows 0..d-1 of in.W/in.b give the candidate x, rows d..2d-1 the gate
    pre-activation, rows 2d..3d-1 are present but unused.  Columns 0..d-1 of
    out.W read the forward-scan state, columns d..2d-1 the backward-scan state.
    Head outputs are ordered (d0, z0, phi, theta, q/p).
    """
    lay = [("embed.W", (d, 3), 3, "w"), ("embed.b", (d,), 3, "b")]
    for l in range(n_layers):
        p = f"layer{l}."
        lay += [(p + "norm.g", (d,), d, "g"),
                (p + "in.W", (3 * d, d), d, "w"), (p + "in.b", (3 * d,), d, "b"),
                (p + "out.W", (d, 2 * d), 2 * d, "w"), (p + "out.b", (d,), 2 * d, "b")]
    lay += [("head.W1", (d, d), d, "w"), ("head.b1", (d,), d, "b"),
            ("head.W2", (5, d), d, "w"), ("head.b2", (5,), d, "b")]
    return lay


def blob_size(n_layers: int, d: int) -> int:
    return int(sum(int(np.prod(s)) for _, s, _, _ in blob_layout(n_layers, d)))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), kept as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def make_weights(w=None, *, n_layers: int | None = None, d: int | None = None,
                 dtype: str | None = None, seed: int | None = None) -> np.ndarray:
    """Draw the canonical weight blob from one PCG64 stream, in blob order."""
    if w is not None:
        w = workload(w)
        n_layers = w.n_layers if n_layers is None else n_layers
        d = w.d_model if d is None else d
        dtype = w.dtype if dtype is None else dtype
        seed = w.weight_seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    parts = []
    for _, shape, fan_in, kind in blob_layout(n_layers, d):
        n = int(np.prod(shape))
        if kind == "w":
            v = rng.normal(0.0, fan_in ** -0.5, n)
        elif kind == "b":
            v = rng.uniform(-fan_in ** -0.5, fan_in ** -0.5, n)
        else:
            v = rng.uniform(0.5, 1.5, n)
        parts.append(v)
    blob = np.concatenate(parts).astype(np.float32)
    if dtype == "bf16":
        blob = round_to_bf16(blob)
    return blob


def split_blob(blob: np.ndarray, n_layers: int, d: int) -> dict:
    """View the blob as named arrays (float64 copies)."""
    out, o = {}, 0
    for name, shape, _, _ in blob_layout(n_layers, d):
        n = int(np.prod(shape))
        out[name] = np.asarray(blob[o:o + n], dtype=np.float64).reshape(shape)
        o += n
    assert o == blob.size
    return out


def readout_layout(d: int, hidden: int):
    """Blob of the paper's readout head (Sec. Encoder, last paragraph): RMSNorm
    gain over the 2d end states, a hidden layer of `hidden` units, 35 quantile
    outputs (seven per parameter, parameter p owning outputs 7p..7p+6)."""
    h = hidden
    return [("ro.norm.g", (2 * d,), 2 * d, "g"), ("ro.W1", (h, 2 * d), 2 * d, "w"), ("ro.b1", (h,), 2 * d, "b"),
            ("ro.W2", (35, h), h, "w"), ("ro.b2", (35,), h, "b")]


def readout_dims(w) -> tuple[int, int]:
    """(d, hidden) of a workload's readout head: the end states are 2d wide
    (d = the minGRU hidden width H for the paper's backbone, d_model for the
    residual encoder) and the head has w.head_hidden hidden units."""
    w = workload(w)
    return (w.hidden if w.arch == "mingru" else w.d_model), w.head_hidden


def make_readout_weights(w, seed: int | None = None, d: int | None = None,
                         hidden: int | None = None) -> np.ndarray:
    """float32 blob of a workload's readout head (dimensions from readout_dims
    unless given), drawn like the encoder's (N(0, 1/fan_in),
    U(+-fan_in^-1/2), gains U(0.5, 1.5)); rounded to bf16 values for a bf16
    workload, as its encoder weights are."""
    w = workload(w)
    d0, h0 = readout_dims(w)
    d = d0 if d is None else d
    hidden = h0 if hidden is None else hidden
    rng = np.random.default_rng(w.weight_seed + 100 if seed is None else seed)
    parts = []
    for _, shape, fan_in, kind in readout_layout(d, hidden):
        n = int(np.prod(shape))
        if kind == "w":
            parts.append(rng.normal(0.0, fan_in ** -0.5, n))
        elif kind == "b":
            parts.append(rng.uniform(-fan_in ** -0.5, fan_in ** -0.5, n))
        else:
            parts.append(rng.uniform(0.5, 1.5, n))
    blob = np.concatenate(parts).astype(np.float32)
    return round_to_bf16(blob) if w.dtype == "bf16" else blob


# ----------------------------------------------------------------------------
# Per-hit features of the paper's front end (inputs only: no arithmetic of the
# method).  The paper's hits carry 12 measured features (position, derived
# angles, detector identifiers) and three seed features; these are seeded
# stand-ins with the same roles, computed from the generated hit positions.
# ----------------------------------------------------------------------------

N_MEASURED = 12
MEASURED_NAMES = ("x", "y", "z", "r", "phi", "cot_theta", "layer", "phi_module", "z_module",
                  "local_u", "local_v", "eta")
Z_MODULE_MM = 100.0      # sensor length along z


def _phi_modules(layer):
    """Sensors around the barrel cylinder: more at larger radius."""
    return 8 * (layer + 2)


def measured_features(w, hits, offs) -> np.ndarray:
    """float32 [H, 12]: x, y, z, r, phi, z/r, layer index, sensor index in phi
    and in z, the hit's offsets from its sensor's centre (along r phi and z),
    and asinh(z/r).  Hit t of a track lies on barrel layer t (tracks keep their
    innermost layers)."""
    w = workload(w)
    h = np.asarray(hits, dtype=np.float64)
    offs = np.asarray(offs, dtype=np.int64)
    H = h.shape[0]
    layer = np.arange(H) - np.repeat(offs[:-1] - offs[0], np.diff(offs))
    x, y, z = h[:, 0], h[:, 1], h[:, 2]
    r = np.hypot(x, y)
    phi = np.arctan2(y, x)
    nmod = _phi_modules(layer)
    pm = np.floor((phi + np.pi) / (2 * np.pi) * nmod)
    pm = np.minimum(pm, nmod - 1)
    phic = -np.pi + (pm + 0.5) * 2 * np.pi / nmod
    zm = np.floor((z + w.z_max) / Z_MODULE_MM)
    zc = -w.z_max + (zm + 0.5) * Z_MODULE_MM
    out = np.stack([x, y, z, r, phi, z / r, layer, pm, zm, r * (phi - phic), z - zc, np.arcsinh(z / r)], axis=1)
    return np.ascontiguousarray(out, dtype=np.float32)


def feature_bounds(w):
    """(lo, hi) float32 [15]: min-max bounds of the 12 measured and the 3 seed
    features (asinh dU, asinh dV of the residual in mm, up to ~27 mm on the
    outer layers of a three-hit seed; helix path length in mm)."""
    w = workload(w)
    cot = np.sinh(w.eta_max + 0.1)
    nmod = _phi_modules(w.n_det_layers - 1)
    radii = np.linspace(w.r_min, w.r_max, w.n_det_layers)
    half_u = 1.05 * float(np.max(np.pi * radii / _phi_modules(np.arange(w.n_det_layers))))
    rb = 1.001 * w.r_max   # float32 rounding of hits on the outermost cylinder
    lo = [-rb, -rb, -w.z_max, 0.0, -np.pi, -cot, 0.0, 0.0, 0.0, -half_u, -Z_MODULE_MM / 2,
          -(w.eta_max + 0.1), -4.0, -4.0, 0.0]
    hi = [rb, rb, w.z_max, rb, np.pi, cot, w.n_det_layers - 1, nmod - 1,
          2 * w.z_max / Z_MODULE_MM - 1, half_u, Z_MODULE_MM / 2, w.eta_max + 0.1, 4.0, 4.0, 2.5 * w.r_max]
    return np.array(lo, np.float32), np.array(hi, np.float32)


def fourier_layout(n_layers: int, d: int, n_features: int):
    """Blob of the model with the Fourier front end: the bounds, the dense
    projection of the 32 F Fourier features (column 32 f + 16 c + s: c = 0
    sine, 1 cosine, of pi 2^s u_f), then the encoder layers and head of
    blob_layout."""
    K = 32 * n_features
    lay = [("fe.lo", (n_features,), 0, "lo"), ("fe.hi", (n_features,), 0, "hi"),
           ("fe.W", (d, K), K, "w"), ("fe.b", (d,), K, "b")]
    return lay + blob_layout(n_layers, d)[2:]


def make_fourier_weights(w, seed: int | None = None) -> np.ndarray:
    """float32 blob for a Fourier workload (bounds from feature_bounds; the rest
    drawn like make_weights; matrices rounded to bf16 for a bf16 workload)."""
    w = workload(w)
    F = w.n_features
    assert F == 15, "the feature generator provides 15 features"
    rng = np.random.Generator(np.random.PCG64(w.weight_seed + 200 if seed is None else seed))
    lo, hi = feature_bounds(w)
    parts = []
    for name, shape, fan_in, kind in fourier_layout(w.n_layers, w.d_model, F):
        n = int(np.prod(shape))
        if kind == "lo":
            parts.append(lo.astype(np.float64))
        elif kind == "hi":
            parts.append(hi.astype(np.float64))
        elif kind == "w":
            parts.append(rng.normal(0.0, fan_in ** -0.5, n))
        elif kind == "b":
            parts.append(rng.uniform(-fan_in ** -0.5, fan_in ** -0.5, n))
        else:
            parts.append(rng.uniform(0.5, 1.5, n))
    blob = np.concatenate(parts).astype(np.float32)
    if w.dtype == "bf16":
        blob[2 * F:] = round_to_bf16(blob[2 * F:])
    return blob


def hit_features(w, hits, offs, seed_features) -> np.ndarray:
    """float32 [H, 15]: the 12 measured features and the 3 given seed
    features (from the seed kernel or its oracle), in the blob's order."""
    sf = np.asarray(seed_features, dtype=np.float32).reshape(-1, 3)
    return np.ascontiguousarray(np.concatenate([measured_features(w, hits, offs), sf], axis=1))


def mingru_layout(n_layers: int, d: int, H: int, n_features: int = 0):
    """Blob of the paper's backbone: the front end ((x, y, z) embedding, or the
    Fourier front end), then per layer W[4H][D_l], b[4H] with D_0 = d and
    D_l = 2H: rows 0..H-1 forward candidate, H..2H-1 forward gate
    pre-activation, 2H..3H-1 reverse candidate, 3H..4H-1 reverse gate; the
    input of a later layer is [f; b] of the one before."""
    if n_features:
        lay = fourier_layout(0, d, n_features)[:4]
    else:
        lay = blob_layout(0, d)[:2]
    for l in range(n_layers):
        din = d if l == 0 else 2 * H
        lay += [(f"mg{l}.W", (4 * H, din), din, "w"), (f"mg{l}.b", (4 * H,), din, "b")]
    return lay


def make_mingru_weights(w, seed: int | None = None) -> np.ndarray:
    """float32 blob for a minGRU workload, drawn like make_weights (bounds from
    feature_bounds for the Fourier front end); rounded to bf16 values for a
    bf16 workload, the bounds excepted."""
    w = workload(w)
    assert w.arch == "mingru"
    F = w.n_features
    rng = np.random.Generator(np.random.PCG64(w.weight_seed + 300 if seed is None else seed))
    lo, hi = feature_bounds(w) if F else (None, None)
    parts = []
    for name, shape, fan_in, kind in mingru_layout(w.n_layers, w.d_model, w.hidden, F):
        n = int(np.prod(shape))
        if kind == "lo":
            parts.append(lo.astype(np.float64))
        elif kind == "hi":
            parts.append(hi.astype(np.float64))
        elif kind == "w":
            parts.append(rng.normal(0.0, fan_in ** -0.5, n))
        else:
            parts.append(rng.uniform(-fan_in ** -0.5, fan_in ** -0.5, n))
    blob = np.concatenate(parts).astype(np.float32)
    if w.dtype == "bf16":
        blob[2 * F:] = round_to_bf16(blob[2 * F:])
    return blob
