"""Python binding of libtrackfit (the gfx950 track-fit encoder).

Argument marshalling only: every step of the forward pass runs in the HIP
kernels behind the C ABI declared in include/trackfit.h.  PyTorch supplies
device memory and streams.  There is no fallback: if the library is missing
or the GPU is absent, the calls raise.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  -- load torch's HIP runtime before the library (one runtime per process)

__all__ = ["LIB_PATH", "Config", "Weights", "fit_tracks", "device_error", "blob_size",
           "TF_FP32", "TF_BF16", "TF_BF16_F16ACT", "DTYPES", "MODE_FOR_WEIGHTS", "DEVERR_EMPTY_TRACK", "DEVERR_TOO_LONG", "DEVERR_BAD_OFFSETS", "DEVERR_PAIR",
           "TrackfitError", "lib", "seed_tracks", "fit_tracks_states", "Readout", "decode_tracks",
           "readout_blob_size", "MinGRU", "MinGRUConfig", "SEED_TOO_SHORT", "SEED_NO_CIRCLE", "SEED_BAD_OFFSETS"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtrackfit.so")

TF_OK, TF_EINVAL, TF_ENOMEM, TF_EHIP, TF_EUNSUPPORTED, TF_ETOOLARGE = 0, -1, -2, -3, -4, -5
TF_FP32, TF_BF16, TF_BF16_F16ACT = 0, 1, 2
DTYPES = {"fp32": TF_FP32, "bf16": TF_BF16, "bf16_f16act": TF_BF16_F16ACT}
# Library mode used for a model whose weights are given in the named type:
# bf16 weights run with fp16 activation operands (see include/trackfit.h).
MODE_FOR_WEIGHTS = {"fp32": "fp32", "bf16": "bf16_f16act"}
DEVERR_EMPTY_TRACK, DEVERR_TOO_LONG, DEVERR_BAD_OFFSETS, DEVERR_PAIR = 1, 2, 4, 8
SEED_TOO_SHORT, SEED_NO_CIRCLE, SEED_BAD_OFFSETS = 1, 2, 4

EXPORTED = ("tf_weights_create", "tf_weights_destroy", "tf_blob_size", "tf_fourier_blob_size", "tf_max_hits",
            "fit_tracks", "tf_get_device_error", "tf_status_string", "tf_seed_tracks", "fit_tracks_states",
            "tf_readout_blob_size", "tf_readout_create", "tf_readout_destroy", "tf_decode_tracks",
            "tf_mingru_blob_size", "tf_mingru_create", "tf_mingru_destroy", "tf_mingru_workspace_size",
            "tf_mingru_states", "tf_mingru_device_error", "tf_mingru_states_noalloc", "tf_mingru_noalloc_max_rows",
            "tf_mingru_set_fused")


class TrackfitError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {_status_string(status)} ({status})")
        self.status = status


class MinGRUConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("n_features", ctypes.c_int32)]


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("max_hits", ctypes.c_int32), ("n_features", ctypes.c_int32)]


_lib = None


def lib():
    """Load libtrackfit.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        L.tf_weights_create.restype = ctypes.c_int
        L.tf_weights_create.argtypes = [ctypes.POINTER(Config), vp, ctypes.c_size_t, ctypes.POINTER(vp)]
        L.tf_weights_destroy.restype = None
        L.tf_weights_destroy.argtypes = [vp]
        L.tf_blob_size.restype = ctypes.c_size_t
        L.tf_blob_size.argtypes = [ctypes.c_int32, ctypes.c_int32]
        L.tf_fourier_blob_size.restype = ctypes.c_size_t
        L.tf_fourier_blob_size.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
        L.tf_max_hits.restype = ctypes.c_int32
        L.tf_max_hits.argtypes = [vp]
        L.fit_tracks.restype = ctypes.c_int
        L.fit_tracks.argtypes = [vp, ctypes.c_int64, vp, ctypes.c_int32, vp, vp, vp]
        L.fit_tracks_states.restype = ctypes.c_int
        L.fit_tracks_states.argtypes = [vp, ctypes.c_int64, vp, ctypes.c_int32, vp, vp, vp]
        L.tf_get_device_error.restype = ctypes.c_int
        L.tf_get_device_error.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_int32), ctypes.c_int]
        L.tf_status_string.restype = ctypes.c_char_p
        L.tf_status_string.argtypes = [ctypes.c_int]
        L.tf_seed_tracks.restype = ctypes.c_int
        L.tf_seed_tracks.argtypes = [vp, ctypes.c_int64, vp, ctypes.c_int32, ctypes.c_double, vp, vp, ctypes.c_int32,
                                     vp, vp]
        L.tf_readout_blob_size.restype = ctypes.c_size_t
        L.tf_readout_blob_size.argtypes = [ctypes.c_int32, ctypes.c_int32]
        L.tf_readout_create.restype = ctypes.c_int
        L.tf_readout_create.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, vp, ctypes.c_size_t,
                                        ctypes.POINTER(vp)]
        L.tf_readout_destroy.restype = None
        L.tf_readout_destroy.argtypes = [vp]
        L.tf_mingru_blob_size.restype = ctypes.c_size_t
        L.tf_mingru_blob_size.argtypes = [ctypes.POINTER(MinGRUConfig)]
        L.tf_mingru_create.restype = ctypes.c_int
        L.tf_mingru_create.argtypes = [ctypes.POINTER(MinGRUConfig), vp, ctypes.c_size_t, ctypes.POINTER(vp)]
        L.tf_mingru_destroy.restype = None
        L.tf_mingru_destroy.argtypes = [vp]
        L.tf_mingru_workspace_size.restype = ctypes.c_size_t
        L.tf_mingru_workspace_size.argtypes = [vp, ctypes.c_int64]
        L.tf_mingru_states.restype = ctypes.c_int
        L.tf_mingru_states.argtypes = [vp, ctypes.c_int64, vp, ctypes.c_int32, vp, vp, ctypes.c_size_t, vp, vp]
        L.tf_mingru_states_noalloc.restype = ctypes.c_int
        L.tf_mingru_states_noalloc.argtypes = [vp, ctypes.c_int64, vp, ctypes.c_int32, vp, vp, vp]
        L.tf_mingru_noalloc_max_rows.restype = ctypes.c_int64
        L.tf_mingru_noalloc_max_rows.argtypes = [vp]
        L.tf_mingru_set_fused.restype = ctypes.c_int
        L.tf_mingru_set_fused.argtypes = [vp, ctypes.c_int]
        L.tf_mingru_device_error.restype = ctypes.c_int
        L.tf_mingru_device_error.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_int32), ctypes.c_int]
        L.tf_decode_tracks.restype = ctypes.c_int
        L.tf_decode_tracks.argtypes = [vp, ctypes.c_int32, vp, vp, vp, vp, vp]
        _lib = L
    return _lib


def _status_string(status: int) -> str:
    try:
        return lib().tf_status_string(int(status)).decode()
    except Exception:  # library itself unavailable
        return "unknown"


def _check(status: int, what: str):
    if status != TF_OK:
        raise TrackfitError(status, what)


def blob_size(n_layers: int, d_model: int, n_features: int = 0) -> int:
    if n_features:
        return int(lib().tf_fourier_blob_size(int(n_layers), int(d_model), int(n_features)))
    return int(lib().tf_blob_size(int(n_layers), int(d_model)))


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


class Weights:
    """Device-resident weights (tf_weights handle) on the current device."""

    def __init__(self, blob, n_layers: int, d_model: int, dtype: str = "fp32", max_hits: int = 0,
                 n_features: int = 0):
        """dtype: "fp32", "bf16" or "bf16_f16act" (library modes, include/trackfit.h);
        max_hits: longest track that will be passed (0: the largest supported);
        n_features: per-hit features of the Fourier front end (0: hits are x, y, z)."""
        import numpy as np
        arr = np.ascontiguousarray(np.asarray(blob, dtype=np.float32).reshape(-1))
        cfg = Config(int(n_layers), int(d_model), DTYPES[dtype], int(max_hits), int(n_features))
        h = ctypes.c_void_p()
        _check(lib().tf_weights_create(ctypes.byref(cfg), arr.ctypes.data, arr.size, ctypes.byref(h)),
               "tf_weights_create")
        self._h = h
        self.n_layers, self.d_model, self.dtype = int(n_layers), int(d_model), dtype
        self.n_features = int(n_features)
        self.max_hits = int(lib().tf_max_hits(h))

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None):
            lib().tf_weights_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _batch(hits: torch.Tensor, offsets: torch.Tensor, n_tracks: int | None, width: int = 3) -> int:
    """Check a packed batch's tensors; returns the number of tracks."""
    if not (hits.is_cuda and offsets.is_cuda):
        raise ValueError("hits and offsets must be GPU tensors")
    if hits.dtype != torch.float32 or offsets.dtype != torch.int32:
        raise TypeError("hits must be float32 and offsets int32")
    if not (hits.is_contiguous() and offsets.is_contiguous()):
        raise ValueError("hits and offsets must be contiguous")
    if hits.dim() != 2 or hits.shape[1] != width:
        raise ValueError(f"hits must have shape [H, {width}]")
    n = offsets.numel() - 1 if n_tracks is None else int(n_tracks)
    if n < 0 or n + 1 > offsets.numel():
        raise ValueError("n_tracks does not fit the offsets array")
    return n


def _out(out: torch.Tensor | None, n: int, width: int, device, dtype=torch.float32) -> torch.Tensor:
    if out is None:
        return torch.empty((n, width), dtype=dtype, device=device)
    if not (out.is_cuda and out.dtype == dtype and out.is_contiguous() and out.numel() >= width * n):
        raise ValueError(f"output must be a contiguous {dtype} GPU tensor with room for [N, {width}]")
    return out


def fit_tracks(hits: torch.Tensor, offsets: torch.Tensor, weights: Weights, out: torch.Tensor | None = None,
               n_tracks: int | None = None, stream=None) -> torch.Tensor:
    """Enqueue one fit of a packed batch on ``stream`` (default: current stream).

    hits    float32 [H, 3] on the GPU; offsets int32 [N+1] on the GPU (absolute
    row offsets, may start above 0); returns out float32 [N, 5].  ``n_tracks``
    defaults to offsets.numel() - 1 (a prefix of a longer offsets array may be
    given instead).
    """
    n = _batch(hits, offsets, n_tracks, weights.n_features or 3)
    out = _out(out, n, 5, hits.device)
    _check(lib().fit_tracks(hits.data_ptr(), hits.shape[0], offsets.data_ptr(), n, weights.handle,
                            out.data_ptr(), _stream_handle(stream)), "fit_tracks")
    return out


def fit_tracks_states(hits: torch.Tensor, offsets: torch.Tensor, weights: Weights,
                      out: torch.Tensor | None = None, n_tracks: int | None = None, stream=None) -> torch.Tensor:
    """Enqueue the encoder up to the last layer's scans; returns float32
    [N, 2d]: the forward state at each track's last hit, then the reverse
    state at its first hit (the paper's readout input)."""
    n = _batch(hits, offsets, n_tracks, weights.n_features or 3)
    out = _out(out, n, 2 * weights.d_model, hits.device)
    _check(lib().fit_tracks_states(hits.data_ptr(), hits.shape[0], offsets.data_ptr(), n, weights.handle,
                                   out.data_ptr(), _stream_handle(stream)), "fit_tracks_states")
    return out


def device_error(weights: Weights, stream=None, clear: bool = True) -> int:
    """Sticky device error bits (DEVERR_*) seen since the last clear; syncs the stream."""
    v = ctypes.c_int32(0)
    _check(lib().tf_get_device_error(weights.handle, _stream_handle(stream), ctypes.byref(v), int(clear)),
           "tf_get_device_error")
    return int(v.value)


def seed_tracks(hits: torch.Tensor, offsets: torch.Tensor, b_tesla: float, features: bool = True,
                seeds: torch.Tensor | None = None, feats: torch.Tensor | None = None,
                flags: torch.Tensor | None = None, n_tracks: int | None = None, stream=None):
    """Enqueue the analytic three-hit seed (and the per-hit residual features)
    of a packed batch on ``stream`` (default: current stream).

    hits float32 [H, 3] and offsets int32 [N+1] on the GPU.  Returns
    (seeds float64 [N, 5], features float32 [offsets[N] - offsets[0], 3] or
    None).  ``feats`` may be a row-strided view with three unit-stride columns
    (e.g. columns 12..14 of the Fourier front end's [H, 15] feature rows),
    whose row 0 belongs to hit row offsets[0].  ``flags`` (int32 GPU tensor
    of one element) is OR-ed with the SEED_* bits of tracks without a seed.
    """
    if not (hits.is_cuda and offsets.is_cuda):
        raise ValueError("hits and offsets must be GPU tensors")
    if hits.dtype != torch.float32 or offsets.dtype != torch.int32:
        raise TypeError("hits must be float32 and offsets int32")
    if not (hits.is_contiguous() and offsets.is_contiguous()) or hits.dim() != 2 or hits.shape[1] != 3:
        raise ValueError("hits must be a contiguous [H, 3] tensor and offsets contiguous")
    n = offsets.numel() - 1 if n_tracks is None else int(n_tracks)
    if n < 0 or n + 1 > offsets.numel():
        raise ValueError("n_tracks does not fit the offsets array")
    if seeds is None:
        seeds = torch.empty((n, 5), dtype=torch.float64, device=hits.device)
    elif not (seeds.is_cuda and seeds.dtype == torch.float64 and seeds.is_contiguous() and seeds.numel() >= 5 * n):
        raise ValueError("seeds must be a contiguous float64 GPU tensor with room for [N, 5]")
    fptr, fstride = None, 3
    if features:
        if feats is None:  # sized from the offsets (a device read: pass feats to stay asynchronous)
            rows = int(offsets[n].item() - offsets[0].item()) if n > 0 else 0
            feats = torch.empty((max(rows, 0), 3), dtype=torch.float32, device=hits.device)
        elif not (feats.is_cuda and feats.dtype == torch.float32 and feats.dim() == 2 and feats.shape[1] == 3
                  and feats.stride(1) == 1 and feats.stride(0) >= 3):
            raise ValueError("feats must be a float32 GPU tensor [rows, 3] with unit column stride")
        fptr, fstride = feats.data_ptr(), feats.stride(0)
    else:
        feats = None
    if flags is not None and not (flags.is_cuda and flags.dtype == torch.int32 and flags.numel() >= 1):
        raise ValueError("flags must be an int32 GPU tensor")
    _check(lib().tf_seed_tracks(hits.data_ptr(), hits.shape[0], offsets.data_ptr(), n, float(b_tesla),
                                seeds.data_ptr(), fptr, fstride, flags.data_ptr() if flags is not None else None,
                                _stream_handle(stream)), "tf_seed_tracks")
    return seeds, feats


def readout_blob_size(d: int, hidden: int) -> int:
    return int(lib().tf_readout_blob_size(int(d), int(hidden)))


class Readout:
    """Device-resident readout head (tf_readout handle) on the current device:
    end states of width 2d, a hidden layer of `hidden` units, 35 outputs."""

    def __init__(self, blob, d: int, hidden: int, dtype: str = "fp32"):
        """dtype: "fp32", or "bf16" / "bf16_f16act" for the 16-bit head (include/trackfit.h)."""
        import numpy as np
        arr = np.ascontiguousarray(np.asarray(blob, dtype=np.float32).reshape(-1))
        h = ctypes.c_void_p()
        _check(lib().tf_readout_create(int(d), int(hidden), DTYPES[dtype], arr.ctypes.data, arr.size,
                                       ctypes.byref(h)), "tf_readout_create")
        self._h = h
        self.d, self.hidden, self.dtype = int(d), int(hidden), dtype

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None):
            lib().tf_readout_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def decode_tracks(states: torch.Tensor, seeds: torch.Tensor, readout: Readout, quantiles: bool = False,
                  out: torch.Tensor | None = None, q: torch.Tensor | None = None, stream=None):
    """Enqueue the readout head, the point estimates (each parameter's median
    quantile) and the seed-anchored decode.

    states float32 [N, 2d] (fit_tracks_states), seeds float64 [N, 5]
    (seed_tracks), both on the GPU.  Returns (out float64 [N, 5], quantiles
    float32 [N, 35] or None).
    """
    if not (states.is_cuda and seeds.is_cuda):
        raise ValueError("states and seeds must be GPU tensors")
    if states.dtype != torch.float32 or seeds.dtype != torch.float64:
        raise TypeError("states must be float32 and seeds float64")
    if not (states.is_contiguous() and seeds.is_contiguous()):
        raise ValueError("states and seeds must be contiguous")
    n = states.shape[0]
    if states.dim() != 2 or states.shape[1] != 2 * readout.d:
        raise ValueError(f"states must have shape [N, {2 * readout.d}]")
    if seeds.numel() < 5 * n:
        raise ValueError("seeds must hold [N, 5]")
    out = _out(out, n, 5, states.device, torch.float64)
    qptr = None
    if quantiles:
        q = _out(q, n, 35, states.device)
        qptr = q.data_ptr()
    else:
        q = None
    _check(lib().tf_decode_tracks(states.data_ptr(), n, seeds.data_ptr(), readout.handle, qptr, out.data_ptr(),
                                  _stream_handle(stream)), "tf_decode_tracks")
    return out, q


class MinGRU:
    """The paper's bidirectional minGRU backbone (tf_mingru handle) on the current device."""

    def __init__(self, blob, n_layers: int, d_model: int, hidden: int, dtype: str = "fp32", n_features: int = 0):
        import numpy as np
        arr = np.ascontiguousarray(np.asarray(blob, dtype=np.float32).reshape(-1))
        self.cfg = MinGRUConfig(int(n_layers), int(d_model), int(hidden), DTYPES[dtype], int(n_features))
        h = ctypes.c_void_p()
        _check(lib().tf_mingru_create(ctypes.byref(self.cfg), arr.ctypes.data, arr.size, ctypes.byref(h)),
               "tf_mingru_create")
        self._h = h
        self.n_layers, self.d_model, self.hidden, self.dtype = int(n_layers), int(d_model), int(hidden), dtype
        self.n_features = int(n_features)

    @staticmethod
    def blob_size(n_layers, d_model, hidden, n_features=0) -> int:
        c = MinGRUConfig(int(n_layers), int(d_model), int(hidden), 0, int(n_features))
        return int(lib().tf_mingru_blob_size(ctypes.byref(c)))

    @property
    def handle(self):
        return self._h

    def workspace_bytes(self, n_rows: int) -> int:
        return int(lib().tf_mingru_workspace_size(self._h, int(n_rows)))

    def states(self, hits: torch.Tensor, offsets: torch.Tensor, out: torch.Tensor | None = None,
               workspace: torch.Tensor | None = None, n_rows: int | None = None, n_tracks: int | None = None,
               stream=None) -> torch.Tensor:
        """Enqueue the backbone over a packed batch; returns float32 [N, 2H] end
        states.  ``workspace`` (a byte tensor of workspace_bytes(n_rows)) is
        allocated here when not given, sized from the offsets (a device read)
        unless ``n_rows`` (offsets[N] - offsets[0]) is given."""
        n = _batch(hits, offsets, n_tracks, self.n_features or 3)
        out = _out(out, n, 2 * self.hidden, hits.device)
        if workspace is None:
            if n_rows is None:
                n_rows = int(offsets[n].item() - offsets[0].item()) if n > 0 else 0
            workspace = torch.empty(self.workspace_bytes(n_rows), dtype=torch.uint8, device=hits.device)
        elif not (workspace.is_cuda and workspace.is_contiguous()):
            raise ValueError("workspace must be a contiguous GPU tensor")
        _check(lib().tf_mingru_states(hits.data_ptr(), hits.shape[0], offsets.data_ptr(), n, self._h,
                                      workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                      out.data_ptr(), _stream_handle(stream)), "tf_mingru_states")
        return out

    def set_fused(self, fused: bool) -> None:
        """tf_mingru_set_fused: one fused launch (the default for the paper's
        deployed configuration) or the layered launches."""
        _check(lib().tf_mingru_set_fused(self._h, int(bool(fused))), "tf_mingru_set_fused")

    def noalloc_max_rows(self) -> int:
        return int(lib().tf_mingru_noalloc_max_rows(self._h))

    def states_noalloc(self, hits: torch.Tensor, offsets: torch.Tensor, out: torch.Tensor,
                       n_tracks: int | None = None, stream=None) -> torch.Tensor:
        """tf_mingru_states_noalloc: the backbone over a packed batch with the
        library's fixed device workspace; ``out`` (float32 [N, 2H]) is the
        caller's, so the call allocates nothing."""
        n = _batch(hits, offsets, n_tracks, self.n_features or 3)
        if not (out.is_cuda and out.is_contiguous() and out.dtype == torch.float32 and
                out.numel() >= n * 2 * self.hidden):
            raise ValueError(f"out must be a contiguous float32 GPU tensor of at least [{n}, {2 * self.hidden}]")
        _check(lib().tf_mingru_states_noalloc(hits.data_ptr(), hits.shape[0], offsets.data_ptr(), n, self._h,
                                              out.data_ptr(), _stream_handle(stream)), "tf_mingru_states_noalloc")
        return out

    def device_error(self, stream=None, clear: bool = True) -> int:
        v = ctypes.c_int32(0)
        _check(lib().tf_mingru_device_error(self._h, _stream_handle(stream), ctypes.byref(v), int(clear)),
               "tf_mingru_device_error")
        return int(v.value)

    def close(self):
        if getattr(self, "_h", None):
            lib().tf_mingru_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
