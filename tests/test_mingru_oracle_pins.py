"""Pins of the fp64 oracle of the paper's bidirectional minGRU backbone (Sec.
Encoder: per-direction gates and candidates, forward and reverse scans, the
two directions' states concatenated into the next layer), independent of the
oracle's loops: the scans in their brute-force matrix form, the geometric
closed form with constant gates, the time-reversal symmetry, and length 1.
"""
import numpy as np
import pytest
from scipy.special import expit

import oracle
import tracksynth as ts
from tests.bruteforce import scan_matrices


def _tiny(n_layers=2, d=4, H=3, n_tracks=5, len_max=7):
    w = ts.Workload("pin", 96, n_layers=n_layers, d_model=d, dtype="fp32", n_tracks=n_tracks, len_min=1,
                    len_max=len_max, n_det_layers=8, arch="mingru", hidden=H)
    hits, offs = ts.make_tracks(w)
    return w, hits, offs


def _split(blob, n_layers, d, H):
    out, o = {}, 0
    for name, shape, _, _ in ts.mingru_layout(n_layers, d, H):
        n = int(np.prod(shape))
        out[name] = blob[o:o + n].astype(np.float64).reshape(shape)
        o += n
    return out


def _matrix_form(hits, blob, n_layers, d, H):
    """The backbone with every scan as an explicit matrix product."""
    P = _split(blob, n_layers, d, H)
    u = (np.asarray(hits, np.float64) - [-1000.0, -1000.0, -3000.0]) / [2000.0, 2000.0, 6000.0]
    X = u @ P["embed.W"].T + P["embed.b"]
    for l in range(n_layers):
        Z = X @ P[f"mg{l}.W"].T + P[f"mg{l}.b"]
        xf, af, xb, ab = Z[:, :H], expit(Z[:, H:2 * H]), Z[:, 2 * H:3 * H], expit(Z[:, 3 * H:])
        f = np.zeros_like(xf)
        b = np.zeros_like(xb)
        for c in range(H):
            f[:, c] = scan_matrices(af[:, c])[0] @ xf[:, c]
            b[:, c] = scan_matrices(ab[:, c])[1] @ xb[:, c]
        X = np.concatenate([f, b], axis=1)
    return np.concatenate([f[-1], b[0]])


@pytest.mark.parametrize("n_layers,d,H", [(1, 4, 3), (2, 4, 3), (3, 6, 2)])
def test_states_match_matrix_form(n_layers, d, H):
    w, hits, offs = _tiny(n_layers, d, H)
    blob = ts.make_mingru_weights(w)
    st = oracle.mingru_states(hits, offs, blob, n_layers, d, H)
    for i in range(offs.size - 1):
        ref = _matrix_form(hits[offs[i]:offs[i + 1]], blob, n_layers, d, H)
        assert np.allclose(st[i], ref, rtol=1e-12, atol=1e-12)


def test_constant_gates_give_the_geometric_sum():
    """One layer with zero gate weights and gate biases logit(a): each state is
    a sum_k (1 - a)^(t - k) x_k, and with the reverse candidate rows equal to
    the forward ones the reverse state at the first hit mirrors it."""
    w, hits, offs = _tiny(1, 4, 3, n_tracks=3)
    d, H = 4, 3
    P = _split(ts.make_mingru_weights(w), 1, d, H)
    a_f, a_b = 0.3, 0.7
    P["mg0.W"][H:2 * H] = 0.0
    P["mg0.b"][H:2 * H] = np.log(a_f / (1 - a_f))
    P["mg0.W"][3 * H:] = 0.0
    P["mg0.b"][3 * H:] = np.log(a_b / (1 - a_b))
    P["mg0.W"][2 * H:3 * H] = P["mg0.W"][:H]
    P["mg0.b"][2 * H:3 * H] = P["mg0.b"][:H]
    blob = np.concatenate([P[k].ravel() for k, _, _, _ in ts.mingru_layout(1, d, H)]).astype(np.float32)
    st = oracle.mingru_states(hits, offs, blob, 1, d, H)
    for i in range(3):
        h = hits[offs[i]:offs[i + 1]].astype(np.float64)
        u = (h - [-1000.0, -1000.0, -3000.0]) / [2000.0, 2000.0, 6000.0]
        X = u @ P["embed.W"].T.astype(np.float32).astype(np.float64) + P["embed.b"].astype(np.float32)
        x = X @ P["mg0.W"][:H].T.astype(np.float32).astype(np.float64) + P["mg0.b"][:H].astype(np.float32)
        L = h.shape[0]
        af32, ab32 = float(np.float32(np.log(a_f / (1 - a_f)))), float(np.float32(np.log(a_b / (1 - a_b))))
        af_, ab_ = expit(af32), expit(ab32)
        f_last = sum(af_ * (1 - af_) ** (L - 1 - k) * x[k] for k in range(L))
        b_first = sum(ab_ * (1 - ab_) ** k * x[k] for k in range(L))
        assert np.allclose(st[i, :H], f_last, rtol=1e-12, atol=1e-12)
        assert np.allclose(st[i, H:], b_first, rtol=1e-12, atol=1e-12)


def test_time_reversal_swaps_the_directions():
    """Reversing a track's hits while swapping the forward and reverse row
    blocks of every layer (and the [f; b] column halves of the later layers'
    inputs) swaps the end states' halves."""
    n_layers, d, H = 2, 4, 3
    w, hits, offs = _tiny(n_layers, d, H)
    blob = ts.make_mingru_weights(w)
    P = _split(blob, n_layers, d, H)
    Q = {k: v.copy() for k, v in P.items()}
    for l in range(n_layers):
        W, b = P[f"mg{l}.W"], P[f"mg{l}.b"]
        Q[f"mg{l}.W"] = np.concatenate([W[2 * H:], W[:2 * H]])
        Q[f"mg{l}.b"] = np.concatenate([b[2 * H:], b[:2 * H]])
        if l > 0:
            Q[f"mg{l}.W"] = np.concatenate([Q[f"mg{l}.W"][:, H:], Q[f"mg{l}.W"][:, :H]], axis=1)
    blob_q = np.concatenate([Q[k].ravel() for k, _, _, _ in ts.mingru_layout(n_layers, d, H)]).astype(np.float32)
    st = oracle.mingru_states(hits, offs, blob, n_layers, d, H)
    L = np.diff(offs)
    rh = np.concatenate([hits[offs[i]:offs[i + 1]][::-1] for i in range(offs.size - 1)])
    st_r = oracle.mingru_states(rh, offs, blob_q, n_layers, d, H)
    assert np.allclose(st_r[:, :H], st[:, H:], rtol=1e-12, atol=1e-13)
    assert np.allclose(st_r[:, H:], st[:, :H], rtol=1e-12, atol=1e-13)
    assert L.min() >= 1


def test_length_one_gives_gate_times_candidate():
    w, hits, offs = _tiny(1, 4, 3, n_tracks=4, len_max=1)
    d, H = 4, 3
    blob = ts.make_mingru_weights(w)
    P = _split(blob, 1, d, H)
    st = oracle.mingru_states(hits, offs, blob, 1, d, H)
    for i in range(4):
        u = (hits[i].astype(np.float64) - [-1000.0, -1000.0, -3000.0]) / [2000.0, 2000.0, 6000.0]
        z = P["mg0.W"] @ (P["embed.W"] @ u + P["embed.b"]) + P["mg0.b"]
        assert np.allclose(st[i, :H], expit(z[H:2 * H]) * z[:H], rtol=1e-12)
        assert np.allclose(st[i, H:], expit(z[3 * H:]) * z[2 * H:3 * H], rtol=1e-12)


def test_fourier_front_end_and_empty_tracks():
    """The Fourier front end feeds the backbone the same vectors as the pooled
    model's (a 0-layer pooled model exposes them as its residual stream), and an
    empty track gives NaN states."""
    w = ts.workload("mingru2_h64_tiny_d32_fp32")
    import dataclasses
    wf = dataclasses.replace(w, n_features=15, n_layers=1, d_model=8, hidden=2)
    hits, offs = ts.make_tracks(wf, n_tracks=3)
    _, sf, _ = oracle.seed_tracks(hits, offs, wf.b_field)
    feats = ts.hit_features(wf, hits, offs, sf)
    blob = ts.make_mingru_weights(wf)
    F, d, H = 15, 8, 2
    front = blob[:2 * F + d * 32 * F + d]
    W, b = blob[front.size:front.size + 4 * H * d].reshape(4 * H, d), blob[front.size + 4 * H * d:]
    # the pooled model with no layers: the residual stream is the front end's output
    rest = np.zeros(ts.blob_size(0, d) - 4 * d, np.float32)
    for i in range(3):
        f_i = feats[offs[i]:offs[i + 1]]
        _, _, r = oracle.track_forward(f_i, np.concatenate([front, rest]), 0, d, n_features=F)
        z = r @ W.T.astype(np.float64) + b
        L = f_i.shape[0]
        af, ab = expit(z[:, H:2 * H]), expit(z[:, 3 * H:])
        Mf = [scan_matrices(af[:, c])[0] for c in range(H)]
        Mb = [scan_matrices(ab[:, c])[1] for c in range(H)]
        want = np.concatenate([[(Mf[c] @ z[:, c])[L - 1] for c in range(H)],
                               [(Mb[c] @ z[:, 2 * H + c])[0] for c in range(H)]])
        st = oracle.mingru_states(f_i, np.array([0, L], np.int32), blob, 1, d, H, n_features=F)
        assert np.allclose(st[0], want, rtol=1e-11, atol=1e-12)
    st = oracle.mingru_states(feats, np.array([0, 0, offs[1]], np.int32), blob, 1, d, H, n_features=F)
    assert np.all(np.isnan(st[0])) and not np.isnan(st[1]).any()
