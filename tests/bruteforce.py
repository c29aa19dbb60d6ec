"""Independent matrix-form restatement of the encoder, for tiny inputs only.

Used by the tests to pin the oracle.  It shares nothing with the oracle: the
scans are written as explicit lower/upper-triangular matrices built from
products of (1 - a) (the closed form of the recurrence of Eq. (2)), the norm
uses numpy.linalg.norm, the gates scipy.special.expit, the linear maps are
matrix products, and a whole batch is handled with einsum.
"""
import numpy as np
from scipy.special import expit

import tracksynth as ts


def scan_matrices(a):
    """a [L] -> (M_f, M_b) with f = M_f x and b = M_b x for one channel.

    Unrolling h_t = (1 - a_t) h_{t-1} + a_t x_t from h_0 = 0 gives
    f_t = sum_{k<=t} a_k prod_{j=k+1..t} (1 - a_j) x_k; the reverse scan is
    the mirror image, b_t = sum_{k>=t} a_k prod_{j=t..k-1} (1 - a_j) x_k.
    """
    L = a.shape[0]
    Mf = np.zeros((L, L))
    Mb = np.zeros((L, L))
    for t in range(L):
        for k in range(L):
            if k <= t:
                Mf[t, k] = a[k] * np.prod(1.0 - a[k + 1:t + 1])
            if k >= t:
                Mb[t, k] = a[k] * np.prod(1.0 - a[t:k])
    return Mf, Mb


def bidir_scan(x, a):
    """x, a [L, d] -> f, b [L, d] through the matrices, channel by channel."""
    L, d = x.shape
    f = np.zeros((L, d))
    b = np.zeros((L, d))
    for c in range(d):
        Mf, Mb = scan_matrices(a[:, c])
        f[:, c] = Mf @ x[:, c]
        b[:, c] = Mb @ x[:, c]
    return f, b


def track_forward(hits, blob, n_layers, d, eps=1e-6, states_out=None):
    P = ts.split_blob(blob, n_layers, d)
    X = np.asarray(hits, dtype=np.float64).reshape(-1, 3)
    lo = np.array([-1000.0, -1000.0, -3000.0])
    span = np.array([2000.0, 2000.0, 6000.0])
    u = (X - lo) / span
    r = u @ P["embed.W"].T + P["embed.b"]
    for l in range(n_layers):
        p = f"layer{l}."
        rms = np.linalg.norm(r, axis=1, keepdims=True) / np.sqrt(d)
        y = r / np.sqrt(rms ** 2 + eps) * P[p + "norm.g"]
        z = y @ P[p + "in.W"].T + P[p + "in.b"]
        x, gate = z[:, :d], z[:, d:2 * d]
        f, b = bidir_scan(x, expit(gate))
        r = r + np.concatenate([f, b], axis=1) @ P[p + "out.W"].T + P[p + "out.b"]
        last_states = np.concatenate([f[-1], b[0]])
    if states_out is not None and n_layers > 0:
        states_out[:] = last_states
    pooled = r.mean(axis=0)
    h = pooled @ P["head.W1"].T + P["head.b1"]
    h = h * expit(h)
    return h @ P["head.W2"].T + P["head.b2"], pooled, r


def readout(states, seed, head_blob, d, hidden, eps=1e-6):
    """The paper's readout and decode, restated with numpy: RMSNorm over the 2d
    end states, SiLU hidden layer of `hidden` units, 35 quantiles, each
    parameter's median quantile (the middle of its seven outputs) as its point
    estimate, seed-anchored decode (phi wrapped to [-pi, pi), scale-free q/p
    with epsilon 0.02 / GeV)."""
    h_ = hidden
    sizes = [2 * d, h_ * 2 * d, h_, 35 * h_, 35]
    parts = np.split(np.asarray(head_blob, dtype=np.float64), np.cumsum(sizes)[:-1])
    g, W1, b1, W2, b2 = parts[0], parts[1].reshape(h_, 2 * d), parts[2], parts[3].reshape(35, h_), parts[4]
    z = np.asarray(states, dtype=np.float64)
    y = g * z / np.sqrt(np.mean(z * z) + eps)
    h = W1 @ y + b1
    h = h * expit(h)
    q = W2 @ h + b2
    est = q.reshape(5, 7)[:, 3]
    s = np.asarray(seed, dtype=np.float64)
    out = s + est
    out[2] = (out[2] + np.pi) % (2 * np.pi) - np.pi
    out[4] = s[4] + est[4] * (abs(s[4]) + 0.02)
    return q, out
