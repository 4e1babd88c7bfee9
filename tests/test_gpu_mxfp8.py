"""GPU parity of the MXFP8 option (Q/K/V projections and the first feed-forward matrix on OCP
MX FP8 operands; quantization per Sec. 1 and Sec. 5) against the emulated-MXFP8 decoder of
oracle/fp8.py and the fp64 oracle, through the C ABI.

Tolerances. The GPU path and the emulation quantize the same weights identically (both from
the same bf16-representable values) and the activations by the same rule, but from activations
that differ by the bf16 path's rounding elsewhere. So the GPU logits differ from the emulated
ones by (a) that bf16 rounding, bounded by the bf16 tolerance, plus (b) quantization decisions
that flip between neighbouring E4M3 values (or block scales), which at most re-draw the
quantization error the emulation itself shows against fp64. Hence:
  * max |gpu - emulated| <= BF16_ATOL + max |emulated - fp64|, the latter measured on a seeded
    sample per workload (tests/golden/mxfp8_deviation.json, written from the oracle by
    tests/golden/make_mxfp8_deviation.py) or, for the small networks, on the tested windows;
  * the GPU path reproduces the quantization rather than ignoring it: on the workloads, where the
    quantization effect (rms |emulated - fp64| about 0.05) is ten times the bf16 rounding noise,
    rms |gpu - emulated| <= rms |emulated - fp64| / 2; on the small networks the MXFP8 decoder's
    logits lie closer (rms) to the emulated ones than the bf16 decoder's logits for the same
    weights and windows do -- where the quantization effect is at least twice the bf16 decoder's
    own rms deviation from fp64 (below that the two decoders cannot be told apart, and only the
    bound above applies);
  * bits agree with the emulation's on decisive windows.
"""
import dataclasses
import json
import os

import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, check_bits, gpu_decode, inputs, say, spread_sample, weights
from oracle import decoder as O
from oracle import fp8 as MX
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "mxfp8_deviation.json")


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def rms(a):
    return float(np.sqrt(np.mean(np.asarray(a, dtype=np.float64) ** 2)))


def check_mx(g, emu, ora, max_dev, what, g_bf16=None):
    """The tolerances above (g_bf16: the bf16 decoder's logits, for the small networks)."""
    assert np.isfinite(g).all()
    err = np.abs(g - emu)
    rms_g, rms_e = rms(g - emu), rms(emu - ora)
    extra = f", rms |bf16 decoder - emulated| {rms(g_bf16 - emu):.3e}" if g_bf16 is not None else ""
    say(f"  {what}: max |gpu - emulated| {err.max():.3e} (bound {BF16_ATOL + max_dev:.3e}), "
        f"rms {rms_g:.3e} vs rms |emulated - fp64| {rms_e:.3e}{extra}, max |gpu - fp64| {np.abs(g - ora).max():.3e}")
    assert err.max() <= BF16_ATOL + max_dev, (g, emu)
    if g_bf16 is None:
        assert rms_g <= rms_e / 2, (rms_g, rms_e)
    elif rms_e >= 2 * rms(g_bf16 - ora):
        assert rms_g < rms(g_bf16 - emu), (rms_g, rms(g_bf16 - emu))
    else:
        say(f"  quantization effect {rms_e:.2e} below twice the bf16 noise {rms(g_bf16 - ora):.2e}: bound only")


# (d, W, B, D, H, L, mlp_ratio, grid, resnet): d_model 128 and 256 (one and two 128-feature
# slices), heads of 16, 32 and 64, 1 to 3 layers, feed-forward 4 and 5 d_model, both token
# sets, the embedder block; batches that leave the last token-kernel workgroup partly empty.
# The batches hold a few dozen windows: with one logit per window, the rms comparison below
# needs that many to tell a quantization effect of 1.5 times the rounding noise apart (at 9
# windows the rms estimates themselves scatter by a quarter).
SMALL = [
    (3, 6, 41, 128, 8, 1, 4, False, False),
    (5, 10, 43, 256, 8, 2, 4, False, False),
    (5, 10, 37, 256, 4, 2, 5, True, False),
    (3, 6, 38, 128, 4, 3, 4, True, True),
]


@pytest.mark.parametrize("d,W,B,D,H,L,mr,grid,resnet", SMALL,
                         ids=[f"d{s[0]}_D{s[3]}_H{s[4]}_L{s[5]}_r{s[6]}{'_grid' if s[7] else ''}{'_res' if s[8] else ''}"
                              for s in SMALL])
def test_mx_small_networks(d, W, B, D, H, L, mr, grid, resnet):
    wl = synth.Workload(f"m{d}", d, W, B, 0.03, 0.0, D, L, H, mr, synth.DTYPE_MXFP8, grid=grid, resnet=resnet)
    w = synth.make_weights(wl, seed=d + 500 + D)
    meas, types = synth.make_windows(wl, seed=d + 501, realistic_boundaries=False)
    say(f"mxfp8 d={d} W={W} B={B} D={D} H={H} L={L} mr={mr} grid={grid} resnet={resnet}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    ora, _ = O.forward_windows(meas, types, w, d, H, grid=grid)
    emu, _ = MX.forward_windows_mx(meas, types, w, d, H, grid=grid)
    bf = pwdec.Decoder.from_workload(dataclasses.replace(wl, dtype=synth.DTYPE_BF16), w, max_windows=B)
    g_bf16, _, _ = gpu_decode(bf, meas, types)
    bf.close()
    check_mx(logits, emu, ora, float(np.abs(emu - ora).max()), "small", g_bf16)
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))
    check_bits(bits, emu)
    # batch invariance: every window moves to another wavefront and workgroup
    sub, _, _ = gpu_decode(dec, meas[1:], types[1:])
    assert np.array_equal(sub.view(np.uint32), logits[1:].view(np.uint32))
    dec.close()


# windows of the emulated decoder per workload (its CPU cost grows as d^4: a d25 window takes
# about 20 s), the leading ones plus one per XCD residue and the last two of the full batch
LEAD = {"d7": 8, "d11": 2, "d25": 1}
SPREAD = {"d7": True, "d11": True, "d25": False}


@pytest.mark.parametrize("name", ["d7", "d11", "d25"])
def test_mx_workload_full_batch(name):
    """The workload's full batch in the benchmark's launch configuration with the MXFP8 option;
    windows across the batch against the emulated MXFP8 decoder and the fp64 oracle."""
    wl = synth.mxfp8(synth.WORKLOADS[name])
    B = wl.B
    w = weights(name)
    meas, types = inputs(name, B)
    say(f"mxfp8 {name} full batch B={B}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK and np.isfinite(logits).all()
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))
    k = LEAD[name]
    sample = list(range(k)) + (spread_sample(B, k) if SPREAD[name] else [B - 1])
    ora, _ = O.forward_windows(meas[sample], types[sample], w, wl.d, wl.H)
    emu, _ = MX.forward_windows_mx(meas[sample], types[sample], w, wl.d, wl.H)
    with open(GOLDEN) as f:
        max_dev = json.load(f)[name]["max"]
    check_mx(logits[sample], emu, ora, max_dev, f"{name} ({len(sample)} windows)")
    check_bits(bits[sample], emu)
    # a window decoded alone gives the same logit bit for bit
    one, _, _ = gpu_decode(dec, meas[B - 1:B], types[B - 1:B])
    assert one.view(np.uint32)[0] == logits.view(np.uint32)[B - 1]
    dec.close()


def test_mx_uses_the_layer_phased_schedule():
    """MXFP8 runs on the layer-phased token kernels: AUTO picks them, RESIDENT is refused; the
    bf16 and MXFP8 decoders of the same network give different logits (the option is in effect),
    and the recurrent branch's last readout equals the decode."""
    base = synth.WORKLOADS["d7"]
    wl = synth.mxfp8(base)
    B = 16
    meas, types = inputs("d7", B)
    dec = pwdec.Decoder.from_workload(wl, weights("d7"), max_windows=B)
    with pytest.raises(pwdec.PwdError) as e:
        dec.schedule(pwdec.SCHEDULE_RESIDENT)
    assert e.value.code == pwdec.PWD_EUNSUPPORTED
    dec.profile(True)
    logits, _, rc = gpu_decode(dec, meas, types)
    stages = dec.profile_read()
    dec.profile(False)
    assert rc == pwdec.PWD_OK and "attention" in stages and "resident" not in stages
    bf = pwdec.Decoder.from_workload(base, weights("d7"), max_windows=B)
    lb, _, _ = gpu_decode(bf, meas, types)
    assert np.abs(lb - logits).max() > 1e-3
    bf.close()
    meas_t = torch.from_numpy(np.ascontiguousarray(synth.pack_bits(meas)).view(np.int32)).cuda()
    types_t = torch.from_numpy(np.ascontiguousarray(types)).cuda()
    rl = torch.empty((B, wl.d), dtype=torch.float32, device="cuda")
    rb = torch.empty((B, wl.d), dtype=torch.uint8, device="cuda")
    dec.decode_recurrent(meas_t, types_t, rl, rb)
    torch.cuda.synchronize()
    assert np.array_equal(rl.cpu().numpy()[:, -1].view(np.uint32), logits.view(np.uint32))
    dec.close()
