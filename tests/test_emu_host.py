"""CPU runs of the library's own kernel sources on the host SIMT stand-in (tests/emu).

The HIP sources are compiled for the CPU with only device-to-host plumbing substituted
(tests/emu/build_emu.py): every index computation, loop, wait and barrier is the library's.
Each work-item runs as a fiber; cross-lane operations (MFMA, shuffles, ballots) exchange
operands across the 64 lanes of a wavefront exactly as the hardware does; every "device"
allocation sits between 8 GiB of inaccessible address space on either side, so an access
outside it faults on the host and names the allocation, kernel, workgroup and work-item;
LDS is poisoned with a NaN pattern per workgroup and direct-to-LDS loads land only at the
issuing lane's vector-memory wait.

Covered here:
  * the attention kernel alone against softmax attention on the same bf16 operands;
  * whole decodes against the fp64 oracle (stabilizer and grid token sets, dilated
    convolutions at d_model 128);
  * the replay of the one GPU memory fault recorded for this library: the dilated
    convolutions at bf16 d_model 256 (d = 11, 3 windows, 2 layers, dilations 1, 2, 4), whose
    launches -- conv_kernel<256> (four weight chunks per tap), the out-projection-only and the
    feed-forward-only token kernels -- must stay inside every allocation and match the
    oracle. The host stand-in has no wait-state hazards, so it could not show the fault's cause
    (a direct-to-LDS load reading its address register before the v_readfirstlane that wrote
    it had settled); tests/test_wait_counts.py checks the compiled code for that.
"""
import ctypes
import os
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "emu"))

import build_emu  # noqa: E402
import run_emu  # noqa: E402
from oracle import decoder as O  # noqa: E402
from paper_2601_09921_amd import synth  # noqa: E402

BF16_ATOL = 3e-2


def _stale(lib: str) -> bool:
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    deps = [os.path.join(build_emu.CSRC, f) for f in build_emu.sources()]
    deps += [os.path.join(build_emu.HERE, f) for f in ("simt.h", "simt.cpp", "units.cpp", "build_emu.py")]
    deps.append(os.path.join(build_emu.INCLUDE, "pwdec.h"))
    return any(os.path.getmtime(d) > t for d in deps)


@pytest.fixture(scope="module")
def emu():
    if not os.path.exists(build_emu.CLANG):
        pytest.skip("ROCm clang++ is needed for the host build")
    lib = os.path.join(build_emu.OUT, "libpwdec_emu.so")
    if _stale(lib):
        lib = build_emu.build()
    h = run_emu.load(lib)
    h.emu_attention.restype = ctypes.c_int
    h.emu_attention.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int] * 5
    return h


def test_translation_leaves_no_device_only_construct():
    for f in build_emu.sources():
        with open(os.path.join(build_emu.CSRC, f)) as fh:
            build_emu.transform(fh.read())   # raises on anything untranslated


def _bf16(x):
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _f32(b):
    return (np.asarray(b).astype(np.uint32) << 16).view(np.float32)


def _kslot(g, i):
    return 4 * g + i if i < 4 else 16 + 4 * g + (i - 4)


ATTN_CASES = [(8, 256, 8, "normal"), (24, 256, 8, "normal"), (80, 256, 8, "normal"), (120, 256, 8, "normal"),
              (48, 128, 8, "normal"), (48, 256, 4, "normal"),
              (120, 256, 8, "overflow"), (48, 128, 8, "overflow"), (48, 256, 4, "underflow"), (80, 256, 8, "underflow")]


@pytest.mark.parametrize("N,D,H,scores", ATTN_CASES, ids=[f"N{c[0]}_D{c[1]}_H{c[2]}_{c[3]}" for c in ATTN_CASES])
def test_attention_kernel_alone(emu, N, D, H, scores):
    """One window: Q (pre-scaled by log2(e)/sqrt(dh)), K, V written in the Q/K/V projection's
    fragment layouts; the kernel's output against softmax attention in float64 on the same
    bf16 values (heads of 16 run in pairs, 64 in two fragments; N = 80 and 120 run two and
    two wavefronts with padding keys). The kernel exponentiates unshifted scores; "overflow"
    scales Q so that rows reach hundreds of log2 units (exp2 overflows to inf), "underflow"
    gives every head's Q and K opposite shared components so that every score is below -150
    (every exp2 underflows): both go through the running-maximum recomputation."""
    dh, npad = D // H, (N + 15) // 16 * 16
    nbw, ksd = npad // 16, D // 32
    rng = np.random.default_rng(N * 1000 + D + H)
    c = np.log2(np.e) / np.sqrt(dh)
    q = rng.standard_normal((npad, D)) * c
    k = rng.standard_normal((npad, D))
    if scores == "overflow":
        q *= 40.0
    elif scores == "underflow":
        u = np.zeros(D)
        u[::dh] = 1.0                       # the first feature of every head
        q, k = q + 24.0 * u, k - 24.0 * u
    Qb = _bf16(q)
    Kb = _bf16(k)
    Vb = _bf16(rng.standard_normal((npad, D)))
    buf = np.zeros((nbw, 3, ksd, 64, 8), np.uint16)
    lane = np.arange(64)
    for tb in range(nbw):
        tok = tb * 16 + lane % 16
        for f in range(ksd):
            for i in range(8):
                feat = f * 32 + np.array([_kslot(g, i) for g in lane // 16])
                buf[tb, 0, f, :, i] = Qb[tok, feat]
                buf[tb, 1, f, :, i] = Kb[tok, feat]
            vt = buf[tb, 2, f].reshape(2, 64, 4)   # V as 16x16 tiles, tokens as rows
            for h2 in range(2):
                for i in range(4):
                    vt[h2, :, i] = Vb[tb * 16 + 4 * (lane // 16) + i, f * 32 + h2 * 16 + lane % 16]
    qkv = run_emu.Buf(emu, buf)
    y = run_emu.Buf(emu, np.zeros((nbw, ksd, 64, 8), np.uint16))
    assert emu.emu_attention(dh, qkv.ptr, y.ptr, N, npad, nbw, H, 1) == 0
    Y = y.get()
    qkv.free()
    y.free()
    out = np.zeros((npad, D))
    for tb in range(nbw):
        for f in range(ksd):
            for i in range(8):
                feat = f * 32 + np.array([_kslot(g, i) for g in lane // 16])
                out[tb * 16 + lane % 16, feat] = _f32(Y[tb, f, :, i])
    ref = np.zeros((N, D))
    extreme = 0
    for h in range(H):
        sl = slice(h * dh, (h + 1) * dh)
        S = _f32(Qb[:N, sl]).astype(np.float64) @ _f32(Kb[:N, sl]).astype(np.float64).T
        extreme += int((S.max(1) > 128).sum() + (S.max(1) < -130).sum())
        P = np.exp2(S - S.max(1, keepdims=True))
        ref[:, sl] = (P / P.sum(1, keepdims=True)) @ _f32(Vb[:N, sl])
    assert emu.emu_errors() == 0
    assert np.isfinite(out[:N]).all()
    assert np.abs(out[:N] - ref).max() < 1e-2
    # the cases meant to leave the unshifted range do (rows whose largest score is beyond it)
    assert (extreme > 0) == (scores != "normal"), extreme


def _case(d, W, B, D, L, H, r, dil=(), grid=False, seed_base=1100):
    wl = synth.Workload(f"c{d}", d, W, B, 0.05, 0.0, D, L, H, r, synth.DTYPE_BF16, grid=grid or bool(dil),
                        resnet=False, dil=dil)
    w = synth.make_weights(wl, seed=d + seed_base)
    meas, types = synth.make_windows(wl, seed=d + seed_base + 1, realistic_boundaries=False)
    return wl, w, meas, types


@pytest.mark.parametrize("d,W,B,D,L,H,r,dil", [
    (9, 9, 2, 256, 1, 8, 4, ()),            # two attention wavefronts per item
    (5, 10, 6, 128, 2, 8, 4, (1, 2, 4)),    # dilated convolutions at d_model 128 (green on the GPU)
])
def test_decode_matches_oracle(emu, d, W, B, D, L, H, r, dil):
    wl, w, meas, types = _case(d, W, B, D, L, H, r, dil)
    logits, bits, rc = run_emu.decode(emu, wl, w, meas, types)
    o, _ = O.forward_windows(meas, types, w, d, H, grid=wl.grid)
    assert rc == 0 and emu.emu_errors() == 0
    assert np.abs(logits - o).max() <= BF16_ATOL
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))


def test_replay_of_the_recorded_gpu_fault(emu):
    """The configuration whose first GPU run ended in a memory fault: dilated convolutions at
    bf16 d_model 256, d = 11 on the (d+1)^2 grid, 3 windows, 2 layers, dilations 1, 2, 4, feed-
    forward 4x. Every launch of a round -- attention, the out-projection-only token kernel
    (which writes the convolutions' input G), three conv_kernel<256> units with four weight
    chunks per tap, and the feed-forward-only token kernels with the next round's embedding --
    runs here on the CPU with every allocation fenced. One round's launches use the same
    addresses in every round, so the window is cut to its core (11 rounds) to keep the CPU
    time down; the batch, layers, dilations and widths are the recorded ones. Result: no
    access outside any allocation, no LDS error, and logits within the bf16 tolerance of the
    oracle."""
    wl, w, meas, types = _case(11, 11, 3, 256, 2, 8, 4, (1, 2, 4))
    logits, bits, rc = run_emu.decode(emu, wl, w, meas, types)
    o, _ = O.forward_windows(meas, types, w, 11, 8, grid=True)
    assert rc == 0 and emu.emu_errors() == 0
    assert np.abs(logits - o).max() <= BF16_ATOL
