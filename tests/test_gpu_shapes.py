"""GPU parity beyond the five benchmark workloads: other code distances (token padding to a
multiple of 16 at every size), the paper's window of 3d rounds (b = c = d, Sec. 3.1), head
sizes 16, 32 and 64 at d_model 128 and 256, and the fp32 path with one head of 64. Small
seeded batches against the fp64 oracle."""
import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, FP32_ATOL, FP32_RTOL, check_bits, gpu_decode, gpu_events, say
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16 = synth.DTYPE_BF16
# (d, W, B, D, L, H): every odd d not among the benchmark workloads, two window lengths,
# d_model 128 / 256 with head sizes 16 / 32
SHAPES = [
    (5, 10, 7, 128, 2, 8),      # N=24 -> 32 tokens, dh 16
    (5, 15, 5, 256, 1, 8),      # W = 3d
    (9, 18, 5, 128, 2, 4),      # N=80, dh 32
    (13, 26, 4, 256, 2, 8),     # N=168 -> 176
    (15, 45, 3, 128, 1, 8),     # N=224, W = 3d
    (19, 38, 3, 256, 1, 8),     # N=360 -> 368
    (21, 42, 3, 128, 1, 4),     # N=440 -> 448, dh 32
    (23, 23, 3, 256, 1, 8),     # N=528, W = d (no buffers)
    (7, 21, 6, 128, 3, 8),      # d7 network with the paper's W = 3d
    (5, 10, 5, 256, 1, 4),      # head size 64: two fragments per head, one wavefront
    (7, 14, 4, 128, 1, 2),      # dh 64, odd key-block count (zero V block of two fragments)
    (11, 22, 3, 128, 2, 2),     # dh 64, four wavefronts
    (25, 25, 2, 256, 1, 4),     # dh 64 at d25: K and V of one head fill 158 KB of LDS
    (27, 27, 2, 256, 1, 8),     # past the benchmark distances: N = 728
    (35, 35, 1, 128, 1, 8),     # N = 1224, 77 key blocks: 155 KB of K/V in LDS
]


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("d,W,B,D,L,H", SHAPES, ids=[f"d{s[0]}_W{s[1]}_D{s[3]}_H{s[5]}" for s in SHAPES])
def test_shape_parity(d, W, B, D, L, H):
    wl = synth.Workload(f"d{d}", d, W, B, 0.02, 0.0, D, L, H, 4, BF16)
    w = synth.make_weights(wl, seed=d + W)
    meas, types = synth.make_windows(wl, seed=77 + d, realistic_boundaries=False)
    say(f"shape d={d} W={W} B={B} D={D} L={L} H={H}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    ev, rc = gpu_events(dec, meas, types, W, wl.words)
    assert rc == pwdec.PWD_OK
    o_logits, _, o_ev = O.forward_windows(meas, types, w, d, H, return_events=True)
    assert np.array_equal(ev, O.pack_bits(o_ev))
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    err = np.abs(logits - o_logits)
    say(f"  max |gpu - oracle| = {err.max():.3e}")
    assert (err <= BF16_ATOL).all(), (logits, o_logits)
    check_bits(bits, o_logits)
    # a smaller batch on the same handle gives the same bits for the same windows
    sub, _, _ = gpu_decode(dec, meas[1:], types[1:])
    assert np.array_equal(sub.view(np.uint32), logits[1:].view(np.uint32))
    dec.close()


def test_fp32_head_of_64():
    """fp32 path (one workgroup per window, whole recurrence in LDS) with d_model 64 and one
    head: the attention loops run over a head of 64 features."""
    wl = synth.Workload("d3h1", 3, 6, 9, 0.02, 0.0, 64, 2, 1, 4, synth.DTYPE_F32)
    w = synth.make_weights(wl, seed=31)
    meas, types = synth.make_windows(wl, seed=32, realistic_boundaries=False)
    say("fp32 d3 D=64 H=1")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=wl.B)
    logits, bits, rc = gpu_decode(dec, meas, types)
    dec.close()
    assert rc == pwdec.PWD_OK
    o_logits, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    assert (np.abs(logits - o_logits) <= FP32_RTOL * np.abs(o_logits) + FP32_ATOL).all(), (logits, o_logits)
