#!/usr/bin/env python3
"""Throughput of the fused track-fit encoder on one MI355X.

One step = one pass of the whole forward path (embedding, all encoder layers,
mean pool, head) over the workload's batch stream: for the deployment workload
8,388,608 synthetic helix tracks in 32 fit_tracks calls of 262,144 tracks,
captured once in a HIP graph and replayed.  Inputs are resident in HBM before
the timed region.  Prints one JSON line.

``--path seed`` instead times the analytic three-hit seed with its per-hit
residual features (tf_seed_tracks) over the same tracks, one call per step.

``--path readout`` times the paper's readout path per batch: the seed, the
encoder up to the last layer's end states (fit_tracks_states), and the
35-quantile head with its point estimates and seed-anchored decode (tf_decode_tracks),
three launches per batch, the step again captured in one HIP graph.

``--path paper`` times the paper's own deployed model per batch (workload
mingru2_h192_fourier15_deploy_bf16_8m): the seed writing the three seed
features into the 15-feature rows, the Fourier front end and the two
bidirectional minGRU layers (tf_mingru_states: one fused launch), and the
35-quantile readout with its decode, in one HIP graph.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import tracksynth as ts  # noqa: E402

METRIC = "tracks/sec (encoder+head forward) on 1 MI355X; MFMA util / HBM GB/s vs peak"
PEAK_TFLOPS = {"fp32": 157.3, "bf16": 2516.6, "bf16_f16act": 2516.6}  # dense MFMA, MI355X datasheet
PEAK_HBM_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_2609_32479_amd", "csrc")
COPY_MIB = 256  # plain copy kernel used to calibrate the HBM byte counters

# HBM bytes per launch (per call for the paper's model: its front-end pass and
# two layer launches added up), from two rocprofv3 --pmc runs of this script
# with --no-graph --copy-calibration (FETCH_SIZE, then WRITE_SIZE), each scaled
# by the same counter's reading for a plain device copy of known size
# (profiles/ holds the summaries).  Keyed by (path, workload); a record is used
# only while the SHA-256 of the listed kernel sources, concatenated, is the one
# recorded and the launch shape is the recorded one; otherwise traffic is null.
ENCODER_SRCS = ("trackfit.hip", "common.h")
_ENC_SHA = "03e1d19e9cfae1e6cc4e58be2f7d10039fa15c30ceb82f4b6f7b52c4b856a3d3"
TRAFFIC = {
    # "profile": the summary in profiles/ that these figures come from (its
    # trace, counter runs and bench line were taken on one box in one session)
    ("encoder", "deploy_d128x4_bf16_8m"): {
        "srcs": ENCODER_SRCS, "batch": 262144, "calls_per_step": 32, "sha256": _ENC_SHA,
        "fetch_bytes": 53177331, "write_bytes": 5578880,
        # rocprofv3's derived MfmaUtil (matrix-unit busy cycles over SIMD cycles) and
        # VALUBusy (cycles issuing vector instructions), medians over launches
        "mfma_util": 0.367, "valu_busy": 0.582,
        "profile": "profiles/tf_encoder_kernel_deploy_d128x4_bf16_8m.md"},
    ("encoder", "fourier15_deploy_d128x4_bf16_8m"): {
        "srcs": ENCODER_SRCS, "batch": 262144, "calls_per_step": 32, "sha256": _ENC_SHA,
        "fetch_bytes": 233133847, "write_bytes": 9522144, "mfma_util": 0.383, "valu_busy": 0.559,
        "profile": "profiles/tf_encoder_kernel_fourier15_deploy_d128x4_bf16_8m.md"},
    ("encoder", "d128x4_fp32_65k"): {
        "srcs": ENCODER_SRCS, "batch": 65536, "calls_per_step": 1, "sha256": _ENC_SHA,
        "fetch_bytes": 22474213, "write_bytes": 1520192, "mfma_util": 0.656, "valu_busy": 0.175,
        "profile": "profiles/tf_encoder_kernel_d128x4_fp32_65k.md"},
    ("encoder", "d256x6_bf16_1m"): {
        "srcs": ENCODER_SRCS, "batch": 1048576, "calls_per_step": 1, "sha256": _ENC_SHA,
        "fetch_bytes": 478426450, "write_bytes": 88989104, "mfma_util": 0.434, "valu_busy": 0.351,
        "profile": "profiles/tf_encoder_kernel_d256x6_bf16_1m.md"},
    ("encoder", "long64_d128x4_bf16_200k"): {
        "srcs": ENCODER_SRCS, "batch": 200000, "calls_per_step": 1, "sha256": _ENC_SHA,
        "fetch_bytes": 162485638, "write_bytes": 4057664, "mfma_util": 0.295, "valu_busy": 0.545,
        "profile": "profiles/tf_encoder_kernel_long64_d128x4_bf16_200k.md"},
    ("readout", "deploy_d128x4_bf16_8m"): {
        "srcs": ENCODER_SRCS, "batch": 262144, "calls_per_step": 32, "sha256": _ENC_SHA,
        "fetch_bytes": 59044752, "write_bytes": 270794752, "mfma_util": 0.326, "valu_busy": 0.602,
        "profile": "profiles/readout_path_deploy_d128x4_bf16_8m.md"},
    ("paper", "mingru2_h192_fourier15_deploy_bf16_8m"): {
        # the backbone call: one tf_backbone_kernel launch (front end and both layers)
        "srcs": ENCODER_SRCS + ("mingru.hip",), "batch": 262144, "calls_per_step": 32,
        "sha256": "e4a021b3ba6e36bab6b1991c81e2f8484491bd1bef565a312373c60ec51d6e10",
        "fetch_bytes": 255927980, "write_bytes": 402653184, "mfma_util": 0.332, "valu_busy": 0.360,
        "profile": "profiles/paper_model_mingru2_h192_fourier15_deploy_bf16_8m.md"},
}


def sources_sha256(names):
    import hashlib
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(CSRC, n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def counter_record(path, w, batch, calls):
    """The counter record of this path and workload, when it was taken on these
    kernel sources and this launch shape; else None."""
    rec = TRAFFIC.get((path, w.name))
    if rec is None or calls != rec["calls_per_step"] or batch != rec["batch"]:
        return None
    if sources_sha256(rec["srcs"]) != rec["sha256"]:
        return None
    return rec


def traffic_bytes(path, w, batch, calls):
    """Counter-derived HBM bytes per launch, or None."""
    rec = counter_record(path, w, batch, calls)
    return None if rec is None else rec["fetch_bytes"] + rec["write_bytes"]


def counter_profile(path, w, batch, calls):
    """The profiles/ summary the counter figures come from, or None."""
    rec = counter_record(path, w, batch, calls)
    return None if rec is None else rec["profile"]


def host_cpu():
    """The host CPU model (as lscpu and /proc/cpuinfo name it) and the threads this process may use."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"model": model, "logical_cpus": os.cpu_count(), "usable_cpus": len(os.sched_getaffinity(0))}


def busy_counter(path, w, batch, calls, key):
    """rocprofv3's MfmaUtil ("mfma_util") or VALUBusy ("valu_busy") of the
    dominant kernel, or None."""
    rec = counter_record(path, w, batch, calls)
    return None if rec is None else rec.get(key)


def front_flops(d, n_hits, n_features=0):
    """The front end: 6 d per hit for the 3->d embedding, or 2 x 32 F x d per
    hit for the Fourier front end's dense projection (its sines and cosines
    are not counted)."""
    return (64.0 * n_features * d if n_features else 6.0 * d) * n_hits


def algorithmic_flops(n_layers, d, n_hits, n_tracks, n_features=0):
    """8 d^2 per hit and layer (candidate + gate projections: 2 * d * 2d, merge:
    2 * 2d * d), the front end, 2 d^2 + 10 d per track for the head.  The
    unused third of the input projection is not counted."""
    return 8.0 * d * d * n_layers * n_hits + front_flops(d, n_hits, n_features) + (2.0 * d * d + 10.0 * d) * n_tracks


def algorithmic_bytes(n_hits, n_tracks, n_features=0):
    """12 B per hit read (4 F B with the Fourier front end), 4 B per track of
    offsets, 20 B per track written."""
    return 4.0 * (n_features or 3) * n_hits + 4.0 * (n_tracks + 1) + 20.0 * n_tracks


def model_blob(w):
    return ts.make_fourier_weights(w) if w.n_features else ts.make_weights(w)


def device_features(tf, w, hits, offs, h, o, dev):
    """The Fourier front end's per-hit feature rows on the device: the 12
    measured features from the generator (in chunks of tracks), then the
    GPU seed writes its 3 residual features into columns 12..14."""
    import torch
    n = offs.size - 1
    feats = torch.empty((int(offs[-1] - offs[0]), w.n_features), dtype=torch.float32, device=dev)
    step = 1 << 20
    for i0 in range(0, n, step):
        i1 = min(n, i0 + step)
        a, b = int(offs[i0] - offs[0]), int(offs[i1] - offs[0])
        m = ts.measured_features(w, hits[a:b], offs[i0:i1 + 1])
        feats[a:b, :ts.N_MEASURED] = torch.from_numpy(m).to(dev)
    seeds = torch.empty((n, 5), dtype=torch.float64, device=dev)
    tf.seed_tracks(h, o, w.b_field, seeds=seeds, feats=feats[:, ts.N_MEASURED:ts.N_MEASURED + 3])
    torch.cuda.synchronize()
    return feats


def oracle_inputs(w, hits, offs, sel):
    """A sample's packed hits (or, with the Fourier front end, its feature rows
    with the oracle's own seed features) and offsets, for the CPU baseline."""
    import oracle
    L = offs[sel + 1] - offs[sel]
    h = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
    o = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
    if not w.n_features:
        return h, o
    _, sf, _ = oracle.seed_tracks(h, o, w.b_field)
    return ts.hit_features(w, h, o, np.nan_to_num(sf, nan=0.0)), o


def cpu_baseline(w, blob, hits, offs, seconds, threads, gpu_out):
    """Time the fp64 oracle on a bounded, seeded sample of the same tracks."""
    import oracle
    n_all = offs.size - 1
    rng = np.random.default_rng(7)
    # calibrate on 256 tracks, then size the sample for about `seconds`
    idx = np.sort(rng.choice(n_all, size=min(256, n_all), replace=False))

    def run(sel):
        t0 = time.perf_counter()
        h, o = oracle_inputs(w, hits, offs, sel)   # the oracle's seed features are part of its chain
        out = oracle.fit_tracks(h, o, blob, w.n_layers, w.d_model, n_threads=threads, n_features=w.n_features)
        return out, time.perf_counter() - t0

    _, dt = run(idx)
    n = int(min(n_all, max(256, 256 * seconds / max(dt, 1e-3))))
    sel = np.sort(rng.choice(n_all, size=n, replace=False))
    ref, dt = run(sel)
    g = gpu_out[sel].astype(np.float64)
    rms = np.sqrt(np.mean(ref ** 2, axis=0))
    err = float(np.max(np.abs(g - ref) / np.maximum(np.abs(ref), rms)))
    # the same oracle on one host core, on a smaller sample (about a fifth of the time)
    n1 = int(min(n, max(64, n * seconds / 5.0 / max(dt * oracle.threads(threads), 1e-3))))
    sel1 = np.sort(rng.choice(n_all, size=n1, replace=False))
    t0 = time.perf_counter()
    h1, o1 = oracle_inputs(w, hits, offs, sel1)
    oracle.fit_tracks(h1, o1, blob, w.n_layers, w.d_model, n_threads=1, n_features=w.n_features)
    dt1 = time.perf_counter() - t0
    return {"value": n / dt, "unit": "tracks/s", "cores": oracle.threads(threads), "kind": "oracle",
            "sample": f"{n} tracks drawn without replacement (seed 7) from the {n_all}-track workload, "
                      f"fp64 C oracle, {dt:.1f} s wall",
            "parity_max_col_err_on_sample": err,
            "one_core": {"value": n1 / dt1, "unit": "tracks/s", "cores": 1,
                         "sample": f"{n1} further tracks drawn the same way, {dt1:.1f} s wall"}}


SEED_METRIC = "tracks/sec (fp64 three-hit seed + per-hit residual features) on 1 MI355X; HBM GB/s vs peak"
SEED_SRC = os.path.join(ROOT, "paper_2609_32479_amd", "csrc", "seed.hip")
# HBM bytes of one tf_seed_tracks call over the whole deployment workload, from
# FETCH_SIZE / WRITE_SIZE runs of this script's seed path with --copy-calibration
# (scaled as for the encoder); valid only for the recorded source.
SEED_TRAFFIC = {"workload": "deploy_d128x4_bf16_8m", "n_tracks": 8388608,
                "kernel_sha256": "e1a3819882b73f490ea59aa680513cee1e3ad35b038193b373f2bfb5c83660a4",
                "fetch_bytes": 1460226274, "write_bytes": 1756872480}


def seed_algorithmic_bytes(n_hits, n_tracks):
    """Offsets (4 B per track), every hit read once (12 B), a float32 feature
    triple written per hit (12 B), a float64 seed written per track (40 B)."""
    return 4.0 * (n_tracks + 1) + 24.0 * n_hits + 40.0 * n_tracks


def seed_cpu_baseline(w, hits, offs, seconds, gpu_seeds):
    """Time the fp64 seed oracle (one thread) on a bounded, seeded sample."""
    import oracle
    n_all = offs.size - 1
    rng = np.random.default_rng(7)

    def run(sel):
        L = offs[sel + 1] - offs[sel]
        h = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
        o = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
        t0 = time.perf_counter()
        seeds, _, _ = oracle.seed_tracks(h, o, w.b_field)
        return seeds, time.perf_counter() - t0

    idx = np.sort(rng.choice(n_all, size=min(4096, n_all), replace=False))
    _, dt = run(idx)
    n = int(min(n_all, max(4096, 4096 * seconds / max(dt, 1e-4))))
    sel = np.sort(rng.choice(n_all, size=n, replace=False))
    ref, dt = run(sel)
    g = gpu_seeds[sel]
    g[:, 2] -= np.round((g[:, 2] - ref[:, 2]) / (2 * np.pi)) * 2 * np.pi
    rms = np.sqrt(np.mean(ref ** 2, axis=0))
    err = float(np.max(np.abs(g - ref) / np.maximum(np.abs(ref), rms)))
    return {"value": n / dt, "unit": "tracks/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} tracks drawn without replacement (seed 7) from the {n_all}-track workload, "
                      f"fp64 C oracle with features, {dt:.1f} s wall",
            "parity_max_col_err_on_sample": err}


def seed_traffic_bytes(w, n_tracks):
    import hashlib
    with open(SEED_SRC, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    if w.name != SEED_TRAFFIC["workload"] or n_tracks != SEED_TRAFFIC["n_tracks"] or sha != SEED_TRAFFIC["kernel_sha256"]:
        return None
    return SEED_TRAFFIC["fetch_bytes"] + SEED_TRAFFIC["write_bytes"]


def bench_seed(args, w, hits, offs):
    import torch
    import paper_2609_32479_amd as tf
    dev = torch.device("cuda:0")
    h = torch.from_numpy(hits).to(dev)
    o = torch.from_numpy(offs).to(dev)
    n_tracks = offs.size - 1
    n_hits = int(offs[-1] - offs[0])
    seeds = torch.empty((n_tracks, 5), dtype=torch.float64, device=dev)
    feats = torch.empty((n_hits, 3), dtype=torch.float32, device=dev)
    flags = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        tf.seed_tracks(h, o, w.b_field, seeds=seeds, feats=feats, flags=flags, stream=stream)

    for _ in range(max(args.warmup, 1)):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms_per_step = e0.elapsed_time(e1) / args.steps
    byts = seed_algorithmic_bytes(n_hits, n_tracks)
    gbs = byts / (ms_per_step / 1e3) / 1e9
    res = {
        "metric": SEED_METRIC, "value": n_tracks / (ms_per_step / 1e3), "unit": "tracks/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic helix tracks (2 T solenoid, seeded)",
        "config": {"workload": w.name, "n_tracks": n_tracks, "n_hits": n_hits, "calls_per_step": 1,
                   "b_tesla": w.b_field, "features": True},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": gbs / PEAK_HBM_GBS, "traffic": seed_traffic_bytes(w, n_tracks), "kernel": "tf_seed_kernel",
                     "counters_profile": "profiles/tf_seed_kernel_deploy_8m.md" if seed_traffic_bytes(w, n_tracks) else None,
                     "kernel_avg_ms": ms_per_step, "bytes_per_launch": byts},
        "host_wall_s": wall,
        "device_error_flags": int(flags.item()),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = seed_cpu_baseline(w, hits, offs, args.cpu_seconds, seeds.cpu().numpy())
        res["cpu_baseline"]["host_cpu"] = host_cpu()
    if args.copy_calibration:
        copy_calibration(dev)
    print(json.dumps(res), flush=True)


READOUT_METRIC = ("tracks/sec (seed + encoder end states + 35-quantile readout, point estimate, decode) on 1 MI355X; "
                  "MFMA util vs peak")


def states_algorithmic_flops(n_layers, d, n_hits, n_features=0):
    """Encoder up to the last layer's scans: 8 d^2 per hit for each layer but
    the last, 4 d^2 per hit for the last (candidate and gate projections; its
    merge is not evaluated), and the front end."""
    return 8.0 * d * d * (n_layers - 1) * n_hits + 4.0 * d * d * n_hits + front_flops(d, n_hits, n_features)


def readout_algorithmic_flops(d, nh, n_tracks):
    """Per track: 2 * nh * 2d for W1 (nh hidden units), 2 * 35 * nh for W2."""
    return (4.0 * d * nh + 70.0 * nh) * n_tracks


def readout_cpu_baseline(w, blob, hb, hits, offs, seconds, threads, gpu_out):
    """Time the oracle's chain (seed, end states, readout and decode) on a
    bounded, seeded sample of the same tracks."""
    import oracle
    n_all = offs.size - 1
    rng = np.random.default_rng(7)

    def run(sel):
        L = offs[sel + 1] - offs[sel]
        h = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
        o = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
        t0 = time.perf_counter()
        seeds, sf, _ = oracle.seed_tracks(h, o, w.b_field, features=bool(w.n_features))
        inp = ts.hit_features(w, h, o, np.nan_to_num(sf, nan=0.0)) if w.n_features else h
        st = oracle.track_states(inp, o, blob, w.n_layers, w.d_model, n_threads=threads, n_features=w.n_features)
        _, out = oracle.readout_tracks(st, seeds, hb, *ts.readout_dims(w))
        return out, time.perf_counter() - t0

    idx = np.sort(rng.choice(n_all, size=min(256, n_all), replace=False))
    _, dt = run(idx)
    n = int(min(n_all, max(256, 256 * seconds / max(dt, 1e-3))))
    sel = np.sort(rng.choice(n_all, size=n, replace=False))
    ref, dt = run(sel)
    g = gpu_out[sel].copy()
    g[:, 2] -= np.round((g[:, 2] - ref[:, 2]) / (2 * np.pi)) * 2 * np.pi
    rms = np.sqrt(np.mean(ref ** 2, axis=0))
    err = float(np.max(np.abs(g - ref) / np.maximum(np.abs(ref), rms)))
    return {"value": n / dt, "unit": "tracks/s", "cores": oracle.threads(threads), "kind": "oracle",
            "sample": f"{n} tracks drawn without replacement (seed 7) from the {n_all}-track workload, "
                      f"fp64 C oracle (seed, end states, readout, decode), {dt:.1f} s wall",
            "parity_max_col_err_on_sample": err}


def bench_readout(args, w, hits, offs, mode, batch):
    import torch
    import paper_2609_32479_amd as tf
    dev = torch.device("cuda:0")
    h = torch.from_numpy(hits).to(dev)
    o = torch.from_numpy(offs).to(dev)
    n_tracks = offs.size - 1
    n_hits = int(offs[-1] - offs[0])
    d = w.d_model
    blob = model_blob(w)
    hb = ts.make_readout_weights(w)
    W = tf.Weights(blob, w.n_layers, d, mode, max_hits=args.max_hits or w.len_max, n_features=w.n_features)
    R = tf.Readout(hb, *ts.readout_dims(w), mode)
    # the Fourier front end reads per-hit feature rows: the measured columns are
    # inputs; the seed fills columns 12..14 of each batch's rows inside the step
    feats = device_features(tf, w, hits, offs, h, o, dev) if w.n_features else None
    inp = feats if w.n_features else h
    seeds = torch.empty((n_tracks, 5), dtype=torch.float64, device=dev)
    out = torch.empty((n_tracks, 5), dtype=torch.float64, device=dev)
    states = torch.empty((batch, 2 * d), dtype=torch.float32, device=dev)  # reused by every batch
    starts = list(range(0, n_tracks, batch))

    def one(s0, stream):
        n = min(batch, n_tracks - s0)
        if feats is not None:
            r0 = int(offs[s0] - offs[0])
            tf.seed_tracks(h, o[s0:], w.b_field, seeds=seeds[s0:], n_tracks=n, stream=stream,
                           feats=feats[r0:, ts.N_MEASURED:ts.N_MEASURED + 3])
        else:
            tf.seed_tracks(h, o[s0:], w.b_field, features=False, seeds=seeds[s0:], n_tracks=n, stream=stream)
        tf.fit_tracks_states(inp, o[s0:], W, out=states, n_tracks=n, stream=stream)
        tf.decode_tracks(states[:n], seeds[s0:s0 + n], R, out=out[s0:], stream=stream)

    def step(stream=None):
        for s0 in starts:
            one(s0, stream)

    torch.cuda.synchronize()
    step()
    torch.cuda.synchronize()
    # per-launch time of the dominant kernel (the encoder), eager, events on its stream
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in starts]
    for (a, b), s0 in zip(ev, starts):
        a.record()
        tf.fit_tracks_states(inp, o[s0:], W, out=states, n_tracks=min(batch, n_tracks - s0))
        b.record()
    torch.cuda.synchronize()
    launch_ms = np.array([a.elapsed_time(b) for a, b in ev])

    graph = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            step(side)
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                step(side)
        torch.cuda.synchronize()

    def run_step():
        if graph is not None:
            graph.replay()
        else:
            step()

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        run_step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms_per_step = e0.elapsed_time(e1) / args.steps
    flags = tf.device_error(W)
    gpu_out = out.cpu().numpy()
    per_launch_flops = states_algorithmic_flops(w.n_layers, d, n_hits, w.n_features) / len(starts)
    kernel_ms = float(launch_ms.mean())
    achieved = per_launch_flops / (kernel_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[mode]
    res = {
        "metric": READOUT_METRIC, "value": n_tracks / (ms_per_step / 1e3), "unit": "tracks/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": {"fp32": "f32", "bf16": "bf16",
                  "bf16_f16act": "bf16 weights, f16 activations, f32 accumulate"}[mode]
                 + ("; head f32" if mode == "fp32" else "; head bf16 weights x split-bf16 activations")
                 + ", seed and decode f64",
        "data": "synthetic helix tracks (2 T solenoid, seeded), random-init weights",
        "config": {"workload": w.name, "n_tracks": n_tracks, "batch": batch, "calls_per_step": len(starts),
                   "launches_per_call": 3, "n_hits": n_hits, "n_layers": w.n_layers, "d_model": d, "mode": mode,
                   "n_features": w.n_features,
                   "max_hits": W.max_hits, "hip_graph": graph is not None},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": traffic_bytes("readout", w, batch, len(starts)),
                     "mfma_util_counter": busy_counter("readout", w, batch, len(starts), "mfma_util"),
                     "valu_busy_counter": busy_counter("readout", w, batch, len(starts), "valu_busy"),
                     "counters_profile": counter_profile("readout", w, batch, len(starts)),
                     "kernel": "tf_encoder_kernel (end states)", "kernel_avg_ms": kernel_ms,
                     "flops_per_launch": per_launch_flops},
        "readout_flops_per_step": readout_algorithmic_flops(*ts.readout_dims(w), n_tracks),
        "host_wall_s": wall,
        "device_error_flags": flags,
        "finite_outputs": bool(np.isfinite(gpu_out).all()),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = readout_cpu_baseline(w, blob, hb, hits, offs, args.cpu_seconds, args.cpu_threads,
                                                   gpu_out)
        res["cpu_baseline"]["host_cpu"] = host_cpu()
    if args.copy_calibration:
        copy_calibration(dev)
    print(json.dumps(res), flush=True)


PAPER_METRIC = ("tracks/sec (the paper's deployed model: fp64 seed + Fourier front end + 2 bidirectional minGRU "
                "layers + 35-quantile readout and decode) on 1 MI355X; MFMA util vs peak")
PAPER_H100_TRACKS_PER_S = 5.41e6  # the paper's deployed minGRU on one H100 NVL (context: another device, its data)


def mingru_algorithmic_flops(w, n_hits):
    """Per hit: the front end (2 x 32 F x d, or 6 d) and 2 x D_l x 4H per
    layer (D_0 = d, then 2H).  The sines and cosines are not counted."""
    f = front_flops(w.d_model, n_hits, w.n_features)
    for l in range(w.n_layers):
        din = w.d_model if l == 0 else 2 * w.hidden
        f += 2.0 * din * 4 * w.hidden * n_hits
    return f


def paper_cpu_baseline(w, blob, hb, hits, offs, seconds, threads, gpu_out):
    """The oracle's chain for the paper's model (seed and its features, Fourier
    front end and minGRU layers, readout and decode) on a bounded sample."""
    import oracle
    n_all = offs.size - 1
    rng = np.random.default_rng(7)

    def run(sel):
        L = offs[sel + 1] - offs[sel]
        h = np.concatenate([hits[offs[i]:offs[i + 1]] for i in sel])
        o = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
        t0 = time.perf_counter()
        seeds, sf, _ = oracle.seed_tracks(h, o, w.b_field)
        feats = ts.hit_features(w, h, o, np.nan_to_num(sf, nan=0.0))
        st = oracle.mingru_states(feats, o, blob, w.n_layers, w.d_model, w.hidden, n_features=w.n_features,
                                  n_threads=threads)
        _, out = oracle.readout_tracks(st, seeds, hb, *ts.readout_dims(w))
        return out, time.perf_counter() - t0

    idx = np.sort(rng.choice(n_all, size=min(256, n_all), replace=False))
    _, dt = run(idx)
    n = int(min(n_all, max(256, 256 * seconds / max(dt, 1e-3))))
    sel = np.sort(rng.choice(n_all, size=n, replace=False))
    ref, dt = run(sel)
    g = gpu_out[sel].copy()
    g[:, 2] -= np.round((g[:, 2] - ref[:, 2]) / (2 * np.pi)) * 2 * np.pi
    rms = np.sqrt(np.mean(ref ** 2, axis=0))
    err = float(np.max(np.abs(g - ref) / np.maximum(np.abs(ref), rms)))
    return {"value": n / dt, "unit": "tracks/s", "cores": oracle.threads(threads), "kind": "oracle",
            "sample": f"{n} tracks drawn without replacement (seed 7) from the {n_all}-track workload, "
                      f"fp64 C oracle (seed and features, Fourier front end, minGRU layers, readout, decode), "
                      f"{dt:.1f} s wall",
            "parity_max_col_err_on_sample": err}


def bench_paper(args, w, hits, offs, mode, batch):
    import torch
    import paper_2609_32479_amd as tf
    assert w.arch == "mingru", "--path paper takes a minGRU workload"
    dev = torch.device("cuda:0")
    h = torch.from_numpy(hits).to(dev)
    o = torch.from_numpy(offs).to(dev)
    n_tracks = offs.size - 1
    n_hits = int(offs[-1] - offs[0])
    H = w.hidden
    blob = ts.make_mingru_weights(w)
    hb = ts.make_readout_weights(w)
    M = tf.MinGRU(blob, w.n_layers, w.d_model, H, mode, w.n_features)
    try:
        M.set_fused(True)  # the paper's deployed configuration: one fused backbone launch
        fused = True
    except tf.TrackfitError:
        fused = False
    R = tf.Readout(hb, *ts.readout_dims(w), mode)
    feats = device_features(tf, w, hits, offs, h, o, dev)
    seeds = torch.empty((n_tracks, 5), dtype=torch.float64, device=dev)
    out = torch.empty((n_tracks, 5), dtype=torch.float64, device=dev)
    states = torch.empty((batch, 2 * H), dtype=torch.float32, device=dev)
    starts = list(range(0, n_tracks, batch))
    rows_max = max(int(offs[min(s0 + batch, n_tracks)] - offs[s0]) for s0 in starts)
    ws = torch.empty(M.workspace_bytes(rows_max), dtype=torch.uint8, device=dev)

    def one(s0, stream):
        n = min(batch, n_tracks - s0)
        r0 = int(offs[s0] - offs[0])
        tf.seed_tracks(h, o[s0:], w.b_field, seeds=seeds[s0:], n_tracks=n, stream=stream,
                       feats=feats[r0:, ts.N_MEASURED:ts.N_MEASURED + 3])
        M.states(feats, o[s0:], out=states, workspace=ws, n_tracks=n, stream=stream)
        tf.decode_tracks(states[:n], seeds[s0:s0 + n], R, out=out[s0:], stream=stream)

    def step(stream=None):
        for s0 in starts:
            one(s0, stream)

    torch.cuda.synchronize()
    step()
    torch.cuda.synchronize()
    # per-call time of the dominant call (front end + minGRU layers), eager, events on its stream
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in starts]
    for (a, b), s0 in zip(ev, starts):
        a.record()
        M.states(feats, o[s0:], out=states, workspace=ws, n_tracks=min(batch, n_tracks - s0))
        b.record()
    torch.cuda.synchronize()
    call_ms = np.array([a.elapsed_time(b) for a, b in ev])

    graph = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            step(side)
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                step(side)
        torch.cuda.synchronize()

    def run_step():
        if graph is not None:
            graph.replay()
        else:
            step()

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        run_step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms_per_step = e0.elapsed_time(e1) / args.steps
    flags = M.device_error()
    gpu_out = out.cpu().numpy()
    per_call = mingru_algorithmic_flops(w, n_hits) / len(starts)
    call_avg = float(call_ms.mean())
    achieved = per_call / (call_avg / 1e3) / 1e12
    peak = PEAK_TFLOPS[mode]
    value = n_tracks / (ms_per_step / 1e3)
    res = {
        "metric": PAPER_METRIC, "value": value, "unit": "tracks/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"fp32": "f32", "bf16": "bf16", "bf16_f16act": "bf16 weights, f16 activations, f32 accumulate"}[mode]
                 + "; seed and decode f64",
        "data": "synthetic helix tracks (2 T solenoid, seeded), synthetic per-hit features, random-init weights",
        "config": {"workload": w.name, "n_tracks": n_tracks, "batch": batch, "calls_per_step": len(starts),
                   "launches_per_call": 3 if fused else 3 + w.n_layers, "n_hits": n_hits, "n_layers": w.n_layers,
                   "d_model": w.d_model, "hidden": H, "n_features": w.n_features, "mode": mode,
                   "fused_backbone": fused, "hip_graph": graph is not None},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": traffic_bytes("paper", w, batch, len(starts)),
                     "mfma_util_counter": busy_counter("paper", w, batch, len(starts), "mfma_util"),
                     "valu_busy_counter": busy_counter("paper", w, batch, len(starts), "valu_busy"),
                     "counters_profile": counter_profile("paper", w, batch, len(starts)),
                     "kernel": "tf_mingru_states (" + ("tf_backbone_kernel: front end and both layers fused, 1 launch"
                                                       if fused else f"front end + minGRU layers, {1 + w.n_layers} launches")
                               + ")",
                     "kernel_avg_ms": call_avg, "flops_per_launch": per_call},
        "context": {"paper_h100_nvl_tracks_per_s": PAPER_H100_TRACKS_PER_S,
                    "ratio_to_paper_h100": value / PAPER_H100_TRACKS_PER_S,
                    "note": "the paper's deployed model on its own data and device; not the same inputs"},
        "host_wall_s": wall,
        "device_error_flags": flags,
        "finite_outputs": bool(np.isfinite(gpu_out).all()),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = paper_cpu_baseline(w, blob, hb, hits, offs, args.cpu_seconds, args.cpu_threads, gpu_out)
        res["cpu_baseline"]["host_cpu"] = host_cpu()
    if args.copy_calibration:
        copy_calibration(dev)
    print(json.dumps(res), flush=True)


def copy_calibration(dev):
    """A plain elementwise device copy of known size, for scaling HBM counters."""
    import torch
    src = torch.ones(COPY_MIB * (1 << 20) // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)  # reads and writes COPY_MIB MiB
    torch.cuda.synchronize()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=None,
                    choices=list(ts.WORKLOADS) + list(ts.FOURIER_WORKLOADS) + list(ts.MINGRU_WORKLOADS),
                    help="default: deploy_d128x4_bf16_8m (mingru2_h192_fourier15_deploy_bf16_8m for --path paper)")
    ap.add_argument("--mode", default=None, help="library mode: fp32, bf16 or bf16_f16act")
    ap.add_argument("--n-tracks", type=int, default=None, help="override the workload's track count")
    ap.add_argument("--batch", type=int, default=None, help="tracks per fit_tracks call")
    ap.add_argument("--max-hits", type=int, default=None,
                    help="tf_config.max_hits (default: the workload's longest track)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--cpu-threads", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--path", default="encoder", choices=["encoder", "seed", "readout", "paper"],
                    help="encoder: fit_tracks (default); seed: tf_seed_tracks with features; "
                         "readout: seed + fit_tracks_states + tf_decode_tracks; "
                         "paper: seed + tf_mingru_states + tf_decode_tracks")
    ap.add_argument("--copy-calibration", action="store_true",
                    help=f"after the timed region, run a plain {COPY_MIB} MiB device copy (for counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the forward pass has no cross-track exchange, and "
              "this library has no multi-GPU path (shard the batch by offsets ranges across "
              "processes instead).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_32479_amd as tf

    if args.workload is None:
        args.workload = "mingru2_h192_fourier15_deploy_bf16_8m" if args.path == "paper" else "deploy_d128x4_bf16_8m"
    w = ts.workload(args.workload)
    mode = args.mode or tf.MODE_FOR_WEIGHTS[w.dtype]
    n_tracks = args.n_tracks or w.n_tracks
    batch = args.batch or (w.batch if w.batch else n_tracks)
    workers = min(16, os.cpu_count() or 1)

    t0 = time.perf_counter()
    hits, offs = ts.make_tracks(w, n_tracks=n_tracks, workers=workers)
    print(f"[bench] generated {n_tracks} tracks / {hits.shape[0]} hits in {time.perf_counter() - t0:.1f} s",
          file=sys.stderr, flush=True)
    if args.path == "seed":
        bench_seed(args, w, hits, offs)
        return
    if args.path == "readout":
        bench_readout(args, w, hits, offs, mode, batch)
        return
    if args.path == "paper":
        bench_paper(args, w, hits, offs, mode, batch)
        return
    blob = model_blob(w)

    dev = torch.device("cuda:0")
    h = torch.from_numpy(hits).to(dev)
    o = torch.from_numpy(offs).to(dev)
    out = torch.empty((n_tracks, 5), dtype=torch.float32, device=dev)
    W = tf.Weights(blob, w.n_layers, w.d_model, mode, max_hits=args.max_hits or w.len_max, n_features=w.n_features)
    # with the Fourier front end the kernel reads per-hit feature rows (inputs,
    # resident before the timed region like the hits)
    h = device_features(tf, w, hits, offs, h, o, dev) if w.n_features else h
    starts = list(range(0, n_tracks, batch))

    def step(stream=None):
        for s0 in starts:
            n = min(batch, n_tracks - s0)
            tf.fit_tracks(h, o[s0:], W, out=out[s0:], n_tracks=n, stream=stream)

    # per-launch kernel time, eager, with events on the launch stream: the
    # batches in turn, at least 8 launches (a one-batch workload would
    # otherwise time a single launch, the first after idle)
    torch.cuda.synchronize()
    step()
    torch.cuda.synchronize()
    timed = [starts[i % len(starts)] for i in range(max(len(starts), 8))]
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in timed]
    for (a, b), s0 in zip(ev, timed):
        a.record()
        tf.fit_tracks(h, o[s0:], W, out=out[s0:], n_tracks=min(batch, n_tracks - s0))
        b.record()
    torch.cuda.synchronize()
    launch_ms = np.array([a.elapsed_time(b) for a, b in ev])

    graph = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            step(side)
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                step(side)
        torch.cuda.synchronize()

    def run_step():
        if graph is not None:
            graph.replay()
        else:
            step()

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        run_step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms_total = e0.elapsed_time(e1)
    ms_per_step = ms_total / args.steps
    value = n_tracks / (ms_per_step / 1e3)

    flags = tf.device_error(W)
    gpu_out = out.cpu().numpy()
    n_hits = int(offs[-1] - offs[0])
    flops_step = algorithmic_flops(w.n_layers, w.d_model, n_hits, n_tracks, w.n_features)
    # dominant (only) kernel: algorithmic flops of one launch / its mean duration
    per_launch_flops = flops_step / len(starts)
    kernel_ms = float(launch_ms.mean())
    achieved_tflops = per_launch_flops / (kernel_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[mode]
    bytes_step = algorithmic_bytes(n_hits, n_tracks, w.n_features)

    res = {
        "metric": METRIC, "value": value, "unit": "tracks/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"fp32": "f32", "bf16": "bf16", "bf16_f16act": "bf16 weights, f16 activations, f32 accumulate"}[mode],
        "data": "synthetic helix tracks (2 T solenoid, seeded), random-init weights",
        "config": {"workload": w.name, "n_tracks": n_tracks, "batch": batch, "calls_per_step": len(starts),
                   "n_hits": n_hits, "n_layers": w.n_layers, "d_model": w.d_model, "mode": mode,
                   "max_hits": W.max_hits, "n_features": w.n_features,
                   "hip_graph": graph is not None},
        "roofline": {"bound": "mfma", "achieved": achieved_tflops, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved_tflops / peak, "traffic": traffic_bytes("encoder", w, batch, len(starts)),
                     "mfma_util_counter": busy_counter("encoder", w, batch, len(starts), "mfma_util"),
                     "valu_busy_counter": busy_counter("encoder", w, batch, len(starts), "valu_busy"),
                     "counters_profile": counter_profile("encoder", w, batch, len(starts)),
                     "kernel": "tf_encoder_kernel", "kernel_avg_ms": kernel_ms,
                     "flops_per_launch": per_launch_flops},
        "hbm": {"algorithmic_GBps": bytes_step / (ms_per_step / 1e3) / 1e9, "peak_GBps": PEAK_HBM_GBS,
                "frac": bytes_step / (ms_per_step / 1e3) / 1e9 / PEAK_HBM_GBS},
        "host_wall_s": wall,
        "device_error_flags": flags,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, blob, hits, offs, args.cpu_seconds, args.cpu_threads, gpu_out)
        res["cpu_baseline"]["host_cpu"] = host_cpu()
    if args.copy_calibration:
        copy_calibration(dev)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
