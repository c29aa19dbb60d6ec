"""Comparison metric between the GPU library and the fp64 oracle.

The relative tolerance is taken per output column p over the checked tracks:
e_p = max_i |g_ip - r_ip| / max(|r_ip|, rms_p), rms_p = sqrt(mean_i r_ip^2),
so that outputs near zero are measured against the column's scale.
"""
import numpy as np

TOL = {"fp32": 1e-5, "bf16": 2e-2}


def column_rms(ref):
    return np.sqrt(np.mean(np.asarray(ref, dtype=np.float64) ** 2, axis=0))


def column_errors(gpu, ref, rms=None):
    """rms: column scales; by default those of ref itself (pass the scales of a
    larger sample when ref holds only a few tracks)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape and gpu.shape[1] == 5
    rms = column_rms(ref) if rms is None else np.asarray(rms, dtype=np.float64)
    den = np.maximum(np.abs(ref), rms[None, :])
    e = np.abs(gpu - ref) / den
    l2 = np.linalg.norm(gpu - ref, axis=0) / np.linalg.norm(ref, axis=0)
    return e.max(axis=0), l2, e


def assert_parity(gpu, ref, tol, what="", rms=None):
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite GPU outputs"
    emax, l2, e = column_errors(gpu, ref, rms)
    worst = np.unravel_index(np.argmax(e), e.shape)
    assert emax.max() <= tol, (f"{what}: max column error {emax} (l2 {l2}) above {tol}; "
                               f"worst track {worst[0]} col {worst[1]} gpu {gpu[worst]} ref {ref[worst]}")
    return emax, l2
