"""Throughput benchmark of the parallel-window decoder on one MI355X.

One step = one decode_windows call over the whole batch of the d=25 workload (8192
windows of 50 rounds, 624 stabilizer tokens, D=256, 4 layers, 8 heads, MLP 4x, bf16),
inputs already resident in HBM. The throughput accounting follows the paper's
(Sec. 4.2): decoding time per round = time / (windows * d).

Prints one JSON line with the metric, the per-stage kernel times (HIP events on the
decode stream), the roofline of the dominant kernel, and the fp64 oracle timed on a
bounded sample of the same workload on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3            # MI355X fp32 vector
HBM_PEAK_GBS = 8000.0
PAPER_US_PER_ROUND = {3: 0.781, 7: 0.789, 11: 0.812, 17: 0.841, 25: 0.979}   # one TPU v6e
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# Kernel names as rocprofv3 reports them for the d=25 workload (tok_kernel<d_model, MLP ratio,
# flags>, flags POST=1, EMBED=2, QKV=4).
STAGE_KERNELS = {
    "embed_qkv": "tok_kernel<256, 4, 6>",
    "attention": "attn_kernel<32, 4>",
    "post_qkv": "tok_kernel<256, 4, 5>",
    "post_embed_qkv": "tok_kernel<256, 4, 7>",
    "post": "tok_kernel<256, 4, 1>",
    "readout": "readout_kernel<256>",
    "fp32_window": "f32_window_kernel",
    "stream_split": "stream_split_kernel",
    "stream_combine": "stream_combine_kernel",
    "resident": "resident_kernel",
}
# the stages that run the Syndrome Transformer blocks (Q/K/V, attention, out-projection,
# feed-forward, LayerNorms), whose MFMA fraction the benchmark spec's target speaks of
TRANSFORMER_STAGES = ("embed_qkv", "attention", "post_qkv", "post_embed_qkv", "post", "resident")
EXTRA_WORKLOADS = ("d7", "d11", "d17")


def stage_flops(wl, B):
    """Algorithmic FLOPs of one launch of each stage (real tokens only)."""
    N, D, F, d = wl.N, wl.D, wl.F, wl.d
    qkv = 6 * N * D * D
    post = 2 * N * D * D + 4 * N * D * F
    attn = 4 * N * N * D
    readout = 8 * d * d * D * D + 2 * d * D
    per_window_all = wl.W * wl.L * (qkv + attn + post) + readout
    return {
        "embed_qkv": B * qkv,
        "attention": B * attn,
        "post_qkv": B * (post + qkv),
        "post_embed_qkv": B * (post + qkv),
        "post": B * post,
        "readout": B * readout,
        "fp32_window": B * per_window_all,
        "resident": B * wl.W * wl.L * (qkv + attn + post),
    }, B * per_window_all


def transformer_blocks(stages, flops, steps):
    """MFMA fraction of the transformer-block kernels alone: their algorithmic FLOPs over their
    summed kernel time (HIP events), against the dense bf16 peak."""
    ms = sum(stages[k][0] for k in TRANSFORMER_STAGES if k in stages)
    fl = sum(flops[k] * stages[k][1] for k in TRANSFORMER_STAGES if k in stages)
    tf = fl / (ms * 1e-3) / 1e12 if ms else 0.0
    return {"stages": [k for k in TRANSFORMER_STAGES if k in stages], "ms_per_step": round(ms / steps, 3),
            "tflops": round(tf, 1), "frac_of_bf16_peak": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)}


def workload_line(name, torch, pwdec, synth, reps=3):
    """Another workload of the same network family at its own batch size, decoded with every
    schedule the decoder supports for it: ms per decode (HIP events over `reps` decodes after a
    warm-up), us per round, rounds/s, MFMA fraction of the whole call and of the transformer
    blocks, and kernel launches per decode."""
    wl = synth.WORKLOADS[name]
    weights = synth.make_weights(wl)
    meas, types = synth.make_windows(wl)
    dev_meas = torch.from_numpy(synth.pack_bits(meas).view(np.int32)).cuda()
    dev_types = torch.from_numpy(types).cuda()
    del meas
    logits = torch.empty(wl.B, dtype=torch.float32, device="cuda")
    bits = torch.empty(wl.B, dtype=torch.uint8, device="cuda")
    dec = pwdec.Decoder.from_workload(wl, weights)
    stream = torch.cuda.current_stream()
    flops, step_flops = stage_flops(wl, wl.B)
    peak = MFMA_BF16_PEAK_TFLOPS if wl.dtype == synth.DTYPE_BF16 else FP32_PEAK_TFLOPS
    out = {"workload": f"{wl.name}: d={wl.d}, {wl.N} tokens, {wl.W}-round windows, {wl.B} windows, D={wl.D}, "
                       f"{wl.L} layers, {wl.H} heads", "flop_per_decode": step_flops}
    for sname, sched in (("layers", pwdec.SCHEDULE_LAYERS), ("resident", pwdec.SCHEDULE_RESIDENT)):
        try:
            dec.schedule(sched)
        except pwdec.PwdError:
            continue
        dec.decode(dev_meas, dev_types, logits, bits, stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            dec.decode(dev_meas, dev_types, logits, bits, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        dec.profile(True)
        dec.decode(dev_meas, dev_types, logits, bits, stream)
        torch.cuda.synchronize()
        stages = dec.profile_read()
        dec.profile(False)
        assert np.isfinite(logits.cpu().numpy()).all()
        out[sname] = {
            "ms_per_decode": round(ms, 3), "us_per_round": ms * 1e3 / (wl.B * wl.d),
            "rounds_per_s": wl.B * wl.d / (ms * 1e-3),
            "mfma_frac_call": round(step_flops / (ms * 1e-3) / 1e12 / peak, 4),
            "transformer_blocks": transformer_blocks(stages, flops, 1),
            "launches_per_decode": int(sum(n for _, n in stages.values())),
            "kernel_ms": {k: round(v[0], 3) for k, v in stages.items()},
        }
    dec.close()
    return out


def mxfp8_measurement(torch, pwdec, synth, names=("d7", "d11", "d25"), reps=3):
    """The MXFP8 option (Q/K/V projections and the first feed-forward matrix on E4M3 operands with
    E8M0 block scales, the rest as bf16) on the full batch of each workload, against the bf16
    decoder of the same network and inputs on the same launch schedule (layer-phased; the only one
    MXFP8 runs on) and on bf16's default schedule. Reported separately from the bf16 headline."""
    out = {}
    for name in names:
        base = synth.WORKLOADS[name]
        weights = synth.make_weights(base)
        meas, types = synth.make_windows(base)
        dev_meas = torch.from_numpy(synth.pack_bits(meas).view(np.int32)).cuda()
        dev_types = torch.from_numpy(types).cuda()
        del meas
        logits = torch.empty(base.B, dtype=torch.float32, device="cuda")
        bits = torch.empty(base.B, dtype=torch.uint8, device="cuda")
        stream = torch.cuda.current_stream()
        flops, step_flops = stage_flops(base, base.B)
        N, D, F = base.N, base.D, base.F
        fp8_share = (6 * N * D * D + 2 * N * D * F) / (6 * N * D * D + 4 * N * N * D + 2 * N * D * D + 4 * N * D * F)

        def timed(dec, sched):
            dec.schedule(sched)
            dec.decode(dev_meas, dev_types, logits, bits, stream)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                dec.decode(dev_meas, dev_types, logits, bits, stream)
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            dec.profile(True)
            dec.decode(dev_meas, dev_types, logits, bits, stream)
            torch.cuda.synchronize()
            stages = dec.profile_read()
            dec.profile(False)
            assert np.isfinite(logits.cpu().numpy()).all()
            return ms, stages

        mx = pwdec.Decoder.from_workload(synth.mxfp8(base), weights)
        ms_mx, st_mx = timed(mx, pwdec.SCHEDULE_LAYERS)
        mx.close()
        bf = pwdec.Decoder.from_workload(base, weights)
        ms_bf, _ = timed(bf, pwdec.SCHEDULE_LAYERS)
        ms_auto, _ = timed(bf, pwdec.SCHEDULE_AUTO)
        bf.close()
        tb = transformer_blocks(st_mx, flops, 1)
        out[name] = {
            "workload": f"{base.name}: d={base.d}, {N} tokens, {base.W}-round windows, {base.B} windows, D={D}, "
                        f"{base.L} layers, {base.H} heads, Q/K/V and W1 in MXFP8",
            "ms_per_decode": round(ms_mx, 3), "us_per_round": ms_mx * 1e3 / (base.B * base.d),
            "rounds_per_s": base.B * base.d / (ms_mx * 1e-3),
            "fp8_flop_share": round(fp8_share, 3),
            "transformer_blocks": tb,
            "kernel_ms": {k: round(v[0], 3) for k, v in st_mx.items()},
            "bf16_layers_ms_per_decode": round(ms_bf, 3), "speedup_vs_bf16_layers": round(ms_bf / ms_mx, 3),
            "bf16_default_ms_per_decode": round(ms_auto, 3), "speedup_vs_bf16_default": round(ms_auto / ms_mx, 3),
        }
    return out


# The sources each profiled stage's kernel is compiled from: its counter figures stay valid
# while these files are unchanged, whatever happens to the other kernels.
STAGE_SOURCES = {
    "post_qkv": ("tok.hip", "common.h", "kernels.h", "pipeline.h"),
    "attention": ("attn.hip", "common.h", "kernels.h"),
}


def source_hash(stage=None):
    """Hash of the kernel sources of `stage` (STAGE_SOURCES), or of every source file."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2601_09921_amd", "csrc")
    for f in (STAGE_SOURCES[stage] if stage else sorted(os.listdir(csrc))):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def load_traffic(stage):
    """HBM bytes per launch of `stage` from committed rocprofv3 counter runs, or None when
    they were taken on other sources of that stage's kernel."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if stage not in STAGE_SOURCES or t.get("source_hashes", {}).get(stage) != source_hash(stage):
        return None
    return t.get("bytes_per_launch", {}).get(stage)


# v_exp_f32 issues at half the VALU rate: 8 cycles per 64-lane instruction on each of the 1024
# SIMDs at the 2.4 GHz the dense peaks assume.
EXP_PEAK_PER_S = 1024 * 64 / 8 * 2.4e9


def attention_bound(st, wl, B, peak):
    """The attention launch against both pipes it uses: its MFMA work as a fraction of the dense
    bf16 peak and its exponentials (one per score, H N^2 per window) as a fraction of the
    transcendental issue rate. On gfx950 a SIMD's exponentials and MFMAs barely overlap, so the
    sum of the two fractions is the launch's share of its bound."""
    exps = B * wl.H * wl.N * wl.N
    exp_frac = exps / (st["avg_ms"] * 1e-3) / EXP_PEAK_PER_S
    mfma_frac = st["tflops"] / peak
    return {"kernel": st["kernel"], "mfma_frac": round(mfma_frac, 4), "exp_per_launch": exps,
            "exp_per_s": exps / (st["avg_ms"] * 1e-3), "exp_peak_per_s": EXP_PEAK_PER_S,
            "exp_frac": round(exp_frac, 4), "sum": round(mfma_frac + exp_frac, 4)}


def stream_measurement(dec, wl, torch, pwdec, synth):
    """One decode_stream of a memory experiment as long as the batch (B windows of d rounds,
    the last one ragged): on-device windowing, decoding and XOR / soft-XOR combination."""
    T = wl.B * wl.d - 7
    R = synth.make_stream(wl.N, T, wl.p, seed=2025)
    rounds = torch.from_numpy(np.ascontiguousarray(synth.pack_bits(R)).view(np.int32)).cuda()
    del R
    bit = torch.zeros(1, dtype=torch.uint8, device="cuda")
    prob = torch.zeros(1, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    dec.decode_stream(rounds, bit, prob, stream=stream)          # warm-up
    torch.cuda.synchronize()
    dec.profile(True)
    t0 = time.perf_counter()
    dec.decode_stream(rounds, bit, prob, stream=stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    stages = dec.profile_read()
    dec.profile(False)
    m = -(-T // wl.d)
    split_ms = stages["stream_split"][0]
    split_bytes = T * wl.words * 4 + m * (wl.W + 1) * wl.words * 4 + m
    return {
        "rounds": T, "windows": m, "ms": round(dt * 1e3, 2), "us_per_round": dt / T * 1e6,
        "split_ms": round(split_ms, 4), "split_GBps": round(split_bytes / (split_ms * 1e-3) / 1e9, 1),
        "combine_ms": round(stages["stream_combine"][0], 4),
        "bit": int(bit.item()), "soft_xor": float(prob.item()),
    }


def recurrent_measurement(dec, wl, torch, dev_meas, dev_types):
    """One decode_windows_recurrent of the batch: the same pass with a readout after each of
    the last d rounds (Algorithm 1, recurrent branch)."""
    logits = torch.empty((wl.B, wl.d), dtype=torch.float32, device="cuda")
    bits = torch.empty((wl.B, wl.d), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    dec.decode_recurrent(dev_meas, dev_types, logits, bits, stream)   # warm-up
    torch.cuda.synchronize()
    dec.profile(True)
    t0 = time.perf_counter()
    dec.decode_recurrent(dev_meas, dev_types, logits, bits, stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    stages = dec.profile_read()
    dec.profile(False)
    ro_ms, ro_n = stages["readout"]
    return {"readouts_per_window": wl.d, "ms": round(dt * 1e3, 2), "us_per_round": dt / (wl.B * wl.d) * 1e6,
            "readout_launches": ro_n, "readout_ms_total": round(ro_ms, 2)}


def grid_measurement(wl, weights, torch, pwdec, dev_meas, dev_types):
    """The same batch through the network with the (d+1)^2 token set (every cell of the
    stabilizer array a token): one warm-up and one timed decode."""
    import dataclasses
    gwl = dataclasses.replace(wl, grid=True)
    dec = pwdec.Decoder.from_workload(gwl, weights)
    logits = torch.empty(wl.B, dtype=torch.float32, device="cuda")
    bits = torch.empty(wl.B, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    dec.decode(dev_meas, dev_types, logits, bits, stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    dec.decode(dev_meas, dev_types, logits, bits, stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    dec.close()
    return {"tokens": (wl.d + 1) ** 2, "ms": round(dt * 1e3, 2), "us_per_round": dt / (wl.B * wl.d) * 1e6}


def paper_variant_measurement(wl, torch, pwdec, synth, dev_meas, dev_types):
    """The same batch through the paper's own network shape (App. A model table) at
    d_model 128: the (d+1)^2 token set, the embedder's residual Conv1d block, feed-forward
    5 d_model, and three dilated 3x3 convolutions per layer (dilations 1, 2, 4) between
    attention and feed-forward, 3 layers, random weights. One warm-up and one timed decode
    with per-stage HIP-event timing; the convolution kernel's rate counts all 9 taps of every
    token (18 D^2 FLOP per token and unit)."""
    import dataclasses
    vwl = dataclasses.replace(wl, name=wl.name + "_paper", D=128, L=3, H=8, mlp_ratio=5, grid=True,
                              resnet=True, dil=(1, 2, 4))
    dec = pwdec.Decoder.from_workload(vwl, synth.make_weights(vwl))
    logits = torch.empty(wl.B, dtype=torch.float32, device="cuda")
    bits = torch.empty(wl.B, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    dec.decode(dev_meas, dev_types, logits, bits, stream)     # warm-up
    torch.cuda.synchronize()
    dec.profile(True)
    t0 = time.perf_counter()
    dec.decode(dev_meas, dev_types, logits, bits, stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    stages = dec.profile_read()
    dec.profile(False)
    dec.close()
    T, D = (wl.d + 1) ** 2, vwl.D
    conv_ms, conv_n = stages["dilated_conv"]
    conv_tf = wl.B * 18 * T * D * D / (conv_ms / conv_n * 1e-3) / 1e12
    return {"network": {"d_model": D, "layers": vwl.L, "heads": vwl.H, "mlp_ratio": vwl.mlp_ratio, "tokens": T,
                        "embedder": "linear + residual Conv1d x2", "dilations": list(vwl.dil)},
            "ms": round(dt * 1e3, 2), "us_per_round": dt / (wl.B * wl.d) * 1e6,
            "stage_ms": {k: round(v[0], 2) for k, v in stages.items()},
            "dilated_conv": {"kernel": "conv_kernel<128>", "launches": conv_n, "avg_ms": round(conv_ms / conv_n, 3),
                             "TFLOPs": round(conv_tf, 1), "frac_of_bf16_peak": round(conv_tf / MFMA_BF16_PEAK_TFLOPS, 3)}}


def input_stage_measurement(dec, wl, torch, dev_meas, dev_types, reps=5):
    """The input stage on its own: decoder_detection_events over the batch (packed measurement
    rounds in, packed detection events out; the same event_word the token kernel fuses),
    timed with HIP events on the stream it runs on."""
    B, W, words = wl.B, wl.W, wl.words
    events = torch.empty((B, W, words), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    dec.detection_events(dev_meas, dev_types, events, stream)     # warm-up
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        dec.detection_events(dev_meas, dev_types, events, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = B * (W + 1) * words * 4 + B + B * W * words * 4
    return {"kernel": "events_kernel", "avg_ms": round(ms, 4), "bytes": nbytes,
            "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1), "frac_of_hbm_peak": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 3)}


def environment(torch):
    props = torch.cuda.get_device_properties(0)
    return {"device": props.name, "arch": getattr(props, "gcnArchName", ""),
            "compute_units": props.multi_processor_count, "torch": torch.__version__,
            "hip": getattr(torch.version, "hip", None)}


def cpu_baseline(wl, weights, sample):
    """The fp64 oracle on the batch's first `sample` windows (window types cycle, so all three
    appear from 3 on) with the host's BLAS threads, and on one window with one thread; the
    rounds/s of each is extrapolated to the batch (windows are independent, so time grows
    linearly with their number)."""
    from oracle import decoder as O
    from paper_2601_09921_amd import synth
    import threadpoolctl
    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
    meas, types = synth.make_windows(wl, B=max(sample, 1))
    t0 = time.perf_counter()
    O.forward_windows(meas[:sample], types[:sample], weights, wl.d, wl.H)
    dt = time.perf_counter() - t0
    with threadpoolctl.threadpool_limits(limits=1, user_api="blas"):
        t1 = time.perf_counter()
        O.forward_windows(meas[1:2], types[1:2], weights, wl.d, wl.H)
        dt1 = time.perf_counter() - t1
    return {
        "value": sample * wl.d / dt,
        "unit": "rounds/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": f"{sample} windows (types {sorted(set(types[:sample].tolist()))}) of the {wl.name} workload, "
                  f"fp64 numpy on {cores} BLAS threads, {dt:.1f} s; the rate is extrapolated to the "
                  f"{wl.B}-window batch",
        "extrapolated": True,
        "batch_seconds_extrapolated": dt / sample * wl.B,
        "us_per_round": dt / (sample * wl.d) * 1e6,
        "one_core": {"value": wl.d / dt1, "unit": "rounds/s", "cores": 1, "seconds": round(dt1, 2),
                     "sample": "1 bulk window, one BLAS thread, extrapolated",
                     "batch_seconds_extrapolated": dt1 * wl.B},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="d25")
    ap.add_argument("--cpu-sample", type=int, default=3, help="oracle windows for the CPU baseline (0: skip)")
    ap.add_argument("--no-extra", action="store_true", help="skip the d7 / d11 / d17 workload lines")
    ap.add_argument("--no-stream", action="store_true", help="skip the decode_stream measurement")
    ap.add_argument("--no-recurrent", action="store_true", help="skip the recurrent-readout measurement")
    ap.add_argument("--no-grid", action="store_true", help="skip the (d+1)^2 token-set measurement")
    ap.add_argument("--no-variant", action="store_true",
                    help="skip the paper-shaped network measurement (d_model 128, convolutions, FFN 5x)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first copy 1 GiB device-to-device 3 times (the known-size reference that "
                         "scales rocprofv3 FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: windows are independent, so more GPUs only split the "
              "batch (see the sharding note in the design); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2601_09921_amd import pwdec, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    pwdec.load_library()
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"copy calibration: 3 copies of {src.numel() * 4} bytes", file=sys.stderr, flush=True)
        del src, dst
    wl = synth.WORKLOADS[args.workload]
    B = wl.B
    weights = synth.make_weights(wl)
    meas, types = synth.make_windows(wl)
    dev_meas = torch.from_numpy(synth.pack_bits(meas).view(np.int32)).cuda()
    dev_types = torch.from_numpy(types).cuda()
    logits = torch.empty(B, dtype=torch.float32, device="cuda")
    bits = torch.empty(B, dtype=torch.uint8, device="cuda")
    dec = pwdec.Decoder.from_workload(wl, weights)
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        dec.decode(dev_meas, dev_types, logits, bits, stream)
    torch.cuda.synchronize()
    if dec.sync_status() != pwdec.PWD_OK:
        raise RuntimeError("decoder reported a device error")

    dec.profile(True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        dec.decode(dev_meas, dev_types, logits, bits, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    stages = dec.profile_read()
    dec.profile(False)
    ev_ms = ev0.elapsed_time(ev1)
    step_s = wall / args.steps
    assert np.isfinite(logits.cpu().numpy()).all()

    flops, step_flops = stage_flops(wl, B)
    stage_stats = {}
    for name, (ms, n) in stages.items():
        avg = ms / n
        stage_stats[name] = {
            "kernel": STAGE_KERNELS[name], "launches_per_step": n // args.steps,
            "avg_ms": round(avg, 4), "share": round(ms / (ev_ms or 1), 4),
            "tflops": round(flops[name] / (avg * 1e-3) / 1e12, 1),
        }
    dom = max(stages, key=lambda k: stages[k][0])
    dom_avg_s = stages[dom][0] / stages[dom][1] * 1e-3
    bf16 = wl.dtype == synth.DTYPE_BF16
    peak = MFMA_BF16_PEAK_TFLOPS if bf16 else FP32_PEAK_TFLOPS
    achieved = flops[dom] / dom_avg_s / 1e12
    rounds = B * wl.d
    out = {
        "metric": "decoding rounds/s (one MI355X), us per round = time/(windows*d)",
        "value": rounds / step_s,
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: rotated surface code d={wl.d}, {wl.N} stabilizer tokens, "
                        f"{wl.W}-round windows ({wl.d}-round core), {B} windows (initial/bulk/final mix), "
                        f"Bernoulli({wl.p}) detection events; decoder D={wl.D}, {wl.L} layers, "
                        f"{wl.H} heads, MLP {wl.mlp_ratio}x, random-init weights",
            "distance": wl.d, "windows": B, "window_rounds": wl.W, "tokens": wl.N,
        },
        "us_per_round": step_s / rounds * 1e6,
        "rnn_steps_per_s": B * wl.W / step_s,
        "event_ms_per_step": ev_ms / args.steps,
        "flop_per_step": step_flops,
        "mfma_frac_call": step_flops / step_s / 1e12 / peak,
        "floor_us_per_round_at_peak": step_flops / (peak * 1e12) / rounds * 1e6,
        "paper_us_per_round_tpu_v6e": PAPER_US_PER_ROUND.get(wl.d),
        "stages": stage_stats,
        "transformer_blocks": transformer_blocks(stages, flops, args.steps),
        "roofline": {
            "bound": "mfma" if bf16 else "alu",
            "kernel": STAGE_KERNELS[dom],
            "achieved": round(achieved, 1),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": load_traffic(dom),
        },
    }
    if bf16 and "attention" in stage_stats:
        out["attention_bound"] = attention_bound(stage_stats["attention"], wl, B, peak)
    out["input_stage"] = input_stage_measurement(dec, wl, torch, dev_meas, dev_types)
    out["env"] = environment(torch)
    if not args.no_stream:
        out["stream"] = stream_measurement(dec, wl, torch, pwdec, synth)
    if not args.no_recurrent:
        out["recurrent"] = recurrent_measurement(dec, wl, torch, dev_meas, dev_types)
    dec.close()
    if not args.no_grid and wl.dtype == synth.DTYPE_BF16:
        out["grid_tokens"] = grid_measurement(wl, weights, torch, pwdec, dev_meas, dev_types)
    if not args.no_variant and wl.dtype == synth.DTYPE_BF16:
        out["paper_variant"] = paper_variant_measurement(wl, torch, pwdec, synth, dev_meas, dev_types)
    if not args.no_extra:
        out["workloads"] = {n: workload_line(n, torch, pwdec, synth) for n in EXTRA_WORKLOADS if n != wl.name}
        out["mxfp8"] = mxfp8_measurement(torch, pwdec, synth)
    if args.cpu_sample > 0:
        out["cpu_baseline"] = cpu_baseline(wl, weights, args.cpu_sample)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
