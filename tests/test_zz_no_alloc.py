"""tf_mingru_states_noalloc, the allocation-free variant of tf_mingru_states
(its workspace is the library's fixed device array), against the existing
entry point with a caller workspace: the same kernels, so the end states
must agree bit for bit.  Two calls in a row on the shared array, the second
with a smaller batch, so that whatever the first left in the array cannot
reach the second's results; and the capacity check, which refuses a batch
whose hit array is larger than the array holds before launching anything.
"""
import ctypes

import numpy as np
import pytest

import oracle
import tracksynth as ts

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32479_amd as tf
    return tf


def _inputs(w, n, seed_offset):
    hits, offs = ts.make_tracks(w, n_tracks=n + seed_offset)
    # a batch of n tracks starting at track seed_offset, rebased to row 0
    o = (offs[seed_offset:] - offs[seed_offset]).astype(np.int32)
    h = hits[offs[seed_offset]:offs[-1]]
    if w.n_features:
        _, sf, _ = oracle.seed_tracks(h, o, w.b_field)
        h = ts.hit_features(w, h, o, np.nan_to_num(sf, nan=0.0))
    return np.ascontiguousarray(h, dtype=np.float32), o


def _with_workspace(tf, M, h, o, rows):
    n = o.numel() - 1
    ws = torch.empty(M.workspace_bytes(rows), dtype=torch.uint8, device="cuda")
    out = torch.full((n, 2 * M.hidden), float("nan"), dtype=torch.float32, device="cuda")
    rc = tf.lib().tf_mingru_states(h.data_ptr(), h.shape[0], o.data_ptr(), n, M.handle, ws.data_ptr(),
                                   ws.numel(), out.data_ptr(), None)
    assert rc == tf.TF_OK
    return out


def _noalloc(tf, M, h, o):
    n = o.numel() - 1
    out = torch.full((n, 2 * M.hidden), float("nan"), dtype=torch.float32, device="cuda")
    rc = tf.lib().tf_mingru_states_noalloc(h.data_ptr(), h.shape[0], o.data_ptr(), n, M.handle, out.data_ptr(),
                                           None)
    assert rc == tf.TF_OK
    return out


@pytest.mark.parametrize("name", ["mingru2_h192_fourier15_deploy_bf16_8m", "mingru2_h64_tiny_d32_fp32"])
def test_noalloc_states_match_the_workspace_entry_point(tf, name):
    w = ts.workload(name)
    print(f"[noalloc] {name}", flush=True)
    blob = ts.make_mingru_weights(w)
    M = tf.MinGRU(blob, w.n_layers, w.d_model, w.hidden, tf.MODE_FOR_WEIGHTS[w.dtype], w.n_features)
    for n, first in ((3000, 0), (700, 3100)):   # the second call: a smaller batch of other tracks
        hn, on = _inputs(w, n, first)
        h = torch.from_numpy(hn).cuda()
        o = torch.from_numpy(on).cuda()
        ref = _with_workspace(tf, M, h, o, int(on[-1] - on[0]))
        got = _noalloc(tf, M, h, o)
        torch.cuda.synchronize()
        g, r = got.cpu().numpy(), ref.cpu().numpy()
        print(f"[noalloc] {name}: {n} tracks, {hn.shape[0]} rows, identical: {np.array_equal(g, r)}", flush=True)
        assert np.all(np.isfinite(r))
        assert np.array_equal(g, r)
    assert M.device_error() == 0


def test_noalloc_refuses_a_hit_array_beyond_its_capacity(tf):
    w = ts.workload("mingru2_h192_fourier15_deploy_bf16_8m")
    blob = ts.make_mingru_weights(w)
    M = tf.MinGRU(blob, w.n_layers, w.d_model, w.hidden, tf.MODE_FOR_WEIGHTS[w.dtype], w.n_features)
    cap = M.noalloc_max_rows()
    assert cap == ((128 << 20) - 256) // (2 * (w.d_model + 2 * w.hidden))
    hn, on = _inputs(w, 64, 0)
    h = torch.from_numpy(hn).cuda()
    o = torch.from_numpy(on).cuda()
    out = torch.full((64, 2 * w.hidden), -7.0, dtype=torch.float32, device="cuda")
    L = tf.lib()
    # n_hits above the capacity: refused before any launch, out untouched
    rc = L.tf_mingru_states_noalloc(h.data_ptr(), cap + 1, o.data_ptr(), 64, M.handle, out.data_ptr(), None)
    assert rc == tf.TF_ETOOLARGE
    assert L.tf_status_string(rc) == b"request exceeds a fixed capacity of the library"
    torch.cuda.synchronize()
    assert bool((out == -7.0).all())
    # bad arguments
    assert L.tf_mingru_states_noalloc(h.data_ptr(), hn.shape[0], o.data_ptr(), 64, None, out.data_ptr(),
                                      None) == tf.TF_EINVAL
    assert L.tf_mingru_states_noalloc(h.data_ptr(), hn.shape[0], None, 64, M.handle, out.data_ptr(),
                                      None) == tf.TF_EINVAL
    assert L.tf_mingru_states_noalloc(h.data_ptr(), hn.shape[0], o.data_ptr(), 0, M.handle, None,
                                      None) == tf.TF_OK   # no tracks: nothing to do
