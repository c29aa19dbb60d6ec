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


def track_forward(hits, blob, n_layers, d, eps=1e-6):
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
    pooled = r.mean(axis=0)
    h = pooled @ P["head.W1"].T + P["head.b1"]
    h = h * expit(h)
    return h @ P["head.W2"].T + P["head.b2"], pooled, r
