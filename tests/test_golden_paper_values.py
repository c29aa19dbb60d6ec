"""The oracle and the deployment workload against the sizes and constants the
paper prints for its deployed model (tests/golden/paper_printed_values.txt,
each value with its passage: Sec. Encoder and Sec. Losses)."""
import os

import numpy as np

import oracle
import tracksynth as ts

HERE = os.path.dirname(os.path.abspath(__file__))


def _printed():
    vals = {}
    with open(os.path.join(HERE, "golden", "paper_printed_values.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = line.split()
            vals[k] = float(v) if "." in v else int(v)
    return vals


P = _printed()
W = ts.MINGRU_WORKLOADS["mingru2_h192_fourier15_deploy_bf16_8m"]


def test_the_deployment_workload_has_the_printed_shape():
    assert (W.n_features, W.d_model, W.n_layers, W.hidden) == (
        P["n_hit_features"], P["d_model"], P["n_layers"], P["hidden"])
    assert ts.readout_dims(W) == (P["hidden"], P["head_hidden"])


def test_fourier_map_width():
    """16 scales, a sine and a cosine each, per feature: 480 values for 15."""
    F = P["n_hit_features"]
    rng = np.random.default_rng(3)
    lo = np.zeros(F)
    hi = np.ones(F)
    out = oracle.fourier_features(rng.uniform(size=F), lo, hi)
    assert out.size == P["fourier_width"] == 2 * P["fourier_scales"] * F


def test_backbone_weight_count_from_the_printed_widths():
    """Front end 480 -> 128 (with the features' min and max), then per layer
    four H-row maps (candidate and gate, both directions) of the layer's input:
    d_model for the first, the 384-wide concatenation after it."""
    F, d, H = P["n_hit_features"], P["d_model"], P["hidden"]
    front = 2 * F + d * P["fourier_width"] + d
    layers = 4 * H * d + 4 * H + 4 * H * P["concat_width"] + 4 * H
    assert oracle.mingru_blob_size(P["n_layers"], d, H, F) == front + layers
    assert ts.make_mingru_weights(W).size == front + layers


def test_backbone_output_is_the_concatenation():
    F, d, H = P["n_hit_features"], P["d_model"], P["hidden"]
    w = ts.MINGRU_WORKLOADS["mingru2_h192_fourier15_deploy_bf16_8m"]
    blob = ts.make_mingru_weights(w)
    rng = np.random.default_rng(5)
    L = np.array([1, 4, 9])
    offs = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
    feats = rng.uniform(-1.0, 1.0, size=(int(offs[-1]), F)).astype(np.float32)
    st = oracle.mingru_states(feats, offs, blob, P["n_layers"], d, H, n_features=F)
    assert st.shape == (3, P["concat_width"]) and np.isfinite(st).all()


def test_head_reads_the_concatenation_into_seven_quantiles_of_five_parameters():
    H, Hh, n_out = P["hidden"], P["head_hidden"], P["head_outputs"]
    assert n_out == 5 * P["quantiles"]
    # RMSNorm gain over the 384 inputs, then 384 -> 128 -> 35 with biases
    size = P["concat_width"] + Hh * P["concat_width"] + Hh + n_out * Hh + n_out
    assert oracle.readout_blob_size(H, Hh) == size
    rng = np.random.default_rng(7)
    head = rng.normal(scale=0.1, size=size).astype(np.float32)
    states = rng.normal(size=(2, P["concat_width"]))
    seeds = np.array([[0.01, -0.5, 0.3, 1.1, 0.2], [0.0, 1.0, -2.0, 2.0, -0.7]])
    q, out = oracle.readout_tracks(states, seeds, head, H, Hh)
    assert q.shape == (2, n_out) and out.shape == (2, 5)


def test_scale_free_qop_epsilon():
    """q/p = q/p_seed + estimate (|q/p_seed| + eps), eps = 0.02 / GeV."""
    eps = P["qop_eps"]
    for s, m in ((0.4, 0.25), (-0.05, -1.5), (0.0, 0.3)):
        got = oracle.decode(np.array([0, 0, 0, 0, s]), np.array([0, 0, 0, 0, m]))[4]
        assert abs(got - (s + m * (abs(s) + eps))) < 1e-15
