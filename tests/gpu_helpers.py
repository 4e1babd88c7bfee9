"""Shared helpers of the GPU tests: run the HIP decoder through the C ABI and cache oracle
results per (workload, batch, input flavour) so each oracle pass runs once per session."""
import functools
import sys

import numpy as np

from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

FP32_RTOL, FP32_ATOL = 1e-4, 1e-6      # fp32 logits: |g - o| <= 1e-4 |o| + 1e-6
BF16_ATOL = 3e-2                        # bf16 logits: |g - o| <= 3e-2
BIT_MARGIN, BIT_AGREE = 0.1, 0.999      # bits agree on >= 99.9 % of windows with |o| > 0.1


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=None)
def weights(name):
    return synth.make_weights(synth.WORKLOADS[name])


@functools.lru_cache(maxsize=None)
def inputs(name, B, realistic=True, zero=False):
    wl = synth.WORKLOADS[name]
    return synth.make_windows(wl, B=B, realistic_boundaries=realistic, zero=zero)


@functools.lru_cache(maxsize=None)
def oracle(name, B, realistic=True, zero=False):
    wl = synth.WORKLOADS[name]
    meas, types = inputs(name, B, realistic, zero)
    say(f"  oracle {name} B={B} realistic={realistic} zero={zero}")
    return O.forward_windows(meas, types, weights(name), wl.d, wl.H, return_events=True)


@functools.lru_cache(maxsize=None)
def decoder(name, max_windows):
    wl = synth.WORKLOADS[name]
    return pwdec.Decoder.from_workload(wl, weights(name), max_windows=max_windows)


def to_device(meas_bits, types):
    import torch
    words = synth.pack_bits(meas_bits)
    return (torch.from_numpy(np.ascontiguousarray(words).view(np.int32)).cuda(),
            torch.from_numpy(np.ascontiguousarray(types)).cuda())


def gpu_decode(dec, meas_bits, types):
    import torch
    meas_t, types_t = to_device(meas_bits, types)
    n = types.shape[0]
    logits = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    bits = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    dec.decode(meas_t, types_t, logits, bits)
    torch.cuda.synchronize()
    return logits.cpu().numpy(), bits.cpu().numpy(), dec.sync_status()


def gpu_events(dec, meas_bits, types, W, words):
    import torch
    meas_t, types_t = to_device(meas_bits, types)
    ev = torch.full((types.shape[0], W, words), -1, dtype=torch.int32, device="cuda")
    dec.detection_events(meas_t, types_t, ev)
    torch.cuda.synchronize()
    return ev.cpu().numpy().view(np.uint32), dec.sync_status()


def check_logits(name, g, o):
    wl = synth.WORKLOADS[name]
    assert np.isfinite(g).all()
    err = np.abs(g - o)
    if wl.dtype == synth.DTYPE_F32:
        bound = FP32_RTOL * np.abs(o) + FP32_ATOL
    else:
        bound = np.full_like(o, BF16_ATOL)
    worst = int(np.argmax(err - bound))
    say(f"  {name}: max |gpu - oracle| = {err.max():.3e} (bound at worst {bound[worst]:.3e})")
    assert (err <= bound).all(), f"window {worst}: gpu {g[worst]!r} oracle {o[worst]!r}"


def spread_sample(B, k):
    """Windows spread over a batch of B beyond its first k: one per residue mod 8 at evenly
    spaced positions (the readout runs one workgroup per window and workgroups go round-robin
    over the 8 XCDs, so each XCD's share is represented; so are distant token-kernel tiles), and
    the last two windows (the final, partly padded workgroup tiles of every kernel)."""
    base = (k + 7) // 8 * 8
    picks = {base + x * ((B - base) // 8) // 8 * 8 + x for x in range(8)} | {B - 2, B - 1}
    return sorted(w for w in picks if k <= w < B)


def check_bits(g_bits, o_logits):
    sel = np.abs(o_logits) > BIT_MARGIN
    if sel.sum() == 0:
        return
    agree = (g_bits[sel] == (o_logits[sel] > 0)).mean()
    assert agree >= BIT_AGREE, f"bits agree on {agree:.4%} of decisive windows"
