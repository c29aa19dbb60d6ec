"""Host-side pieces of bench.py: the one-GPU contract and the algorithmic
flop counts behind roofline.achieved, against closed forms of the work each
path defines (per hit and layer: the candidate and gate projections d -> 2d
and the merge 2d -> d, Eq. (2) and Sec. Encoder)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import tracksynth as ts  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("n_layers,d,hits_per_track,per_track", [
    (4, 128, 14, 7_384_832),     # 4 x 128 encoder, 14 hits (mean of U{8..20})
    (4, 128, 64, 33_637_632),    # the 64-hit tracks
    (6, 256, 19, 59_931_648),    # 6 x 256 encoder, 19 hits (mean of U{8..30})
    (1, 32, 10, 86_208),         # 1 x 32 encoder, 10 hits
])
def test_encoder_flops_per_track(n_layers, d, hits_per_track, per_track):
    # 2 d 2d + 2 2d d per hit and layer, 6 d per hit for the 3 -> d embedding,
    # 2 d d + 10 d per track for the d -> d -> 5 head
    closed = (4 * d * d + 4 * d * d) * n_layers * hits_per_track + 6 * d * hits_per_track + 2 * d * d + 10 * d
    assert closed == per_track
    assert bench.algorithmic_flops(n_layers, d, hits_per_track, 1) == per_track


def test_fourier_front_end_flops():
    # 16 scales, a sine and a cosine of each of 15 features: 480 inputs to d = 128
    assert bench.front_flops(128, 1, 15) == 2 * 480 * 128


def test_paper_backbone_flops_per_hit():
    w = ts.MINGRU_WORKLOADS["mingru2_h192_fourier15_deploy_bf16_8m"]
    # front end 480 -> 128, then 4 maps of width 192 from 128 and from 384
    assert bench.mingru_algorithmic_flops(w, 1) == 2 * 480 * 128 + 2 * 128 * 4 * 192 + 2 * 384 * 4 * 192


def test_readout_flops_per_track():
    # 384 -> 128 -> 35
    assert bench.readout_algorithmic_flops(192, 128, 1) == 2 * 384 * 128 + 2 * 128 * 35


def test_algorithmic_bytes_per_track():
    # 12 B per hit in, 4 B of offsets and 20 B out per track (plus the closing offset)
    assert bench.algorithmic_bytes(14, 1) == 12 * 14 + 4 * 2 + 20
